// Varlen compaction of the retained prompts: sequence rho is
// [n_sys system rows | selected vision rows of tile kept[rho], ascending |
//  contextual rows of rho (optional) | n_qry query rows]; every retained tile
// is its own VLM prompt (Sec. 2.3 Stage 2, App. B Step 5).  With a shared
// prefix the n_sys system rows, identical in every prompt, are written once
// at the front as sequence 0 and each prompt holds only the rows after them
// (positions n_sys onwards).
//
//   compact_rows  two waves per packed row r of [0, packed_rows).  The workgroup
//                 stages sel_offsets in LDS (searched in place when there are
//                 more than 4096 prompts) and each wave finds its prompt by
//                 binary search over the prompt starts rho (n_sys + n_qry) +
//                 sel_offsets[rho] (+ ctx_offsets[rho]), checks it (first
//                 offsets, total against the
//                 capacity, tile id, budget) and copies nothing for a bad one;
//                 otherwise it finds the row's source (system, selected vision
//                 or query row) and copies its half of it with a coalesced
//                 16-byte-per-lane copy, four 1 KB loads in flight before the
//                 first store (plain loads: streaming hints measured slower),
//                 and writes the row's position id.
//                 Workgroup 0 also validates the whole call (every tile id,
//                 budget and selected index), writes cu_seqlens and writes the
//                 status word once, with a plain store, so no other launch has
//                 to clear it first.
#include "launch.h"
#include "rift_common.h"

namespace rift {

// The whole-call check of workgroup (0, 0): 256 threads, a strided pass over
// the tile ids and budgets, then (if those hold, so that the number of
// selected indices is known and within the capacity) over the selected
// indices; the status word is written once.
// base: rows before the first prompt (the shared prefix, or 0); fixed: rows
// of a prompt besides its vision and contextual rows; cu gets one more entry
// (0, the prefix sequence) when base > 0.
__device__ void compact_validate(const int* __restrict__ kept, const int* __restrict__ offs,
                                 const int* __restrict__ coffs, const int* __restrict__ sel, int n_keep,
                                 int n_tiles, int n_v, int base, int fixed, bool shared, long long cap,
                                 int* __restrict__ cu, int* __restrict__ status) {
    __shared__ int bad_shape, bad_sel;
    const int tid = threadIdx.x;
    if (tid == 0) {
        bad_shape = 0;
        bad_sel = 0;
    }
    __syncthreads();
    const int o_first = offs[0];
    const int o_last = offs[n_keep];
    const int c_first = coffs != nullptr ? coffs[0] : 0;
    const int c_last = coffs != nullptr ? coffs[n_keep] : 0;
    const long long total = base + (long long)n_keep * fixed + o_last + c_last;
    int* cup = cu + (shared ? 1 : 0);   // prompt starts
    if (tid == 0) {
        cup[n_keep] = (int)total;
        if (shared) cu[0] = 0;
    }
    for (int i = tid; i < n_keep; i += blockDim.x)
        cup[i] = (int)(base + (long long)i * fixed + offs[i] + (coffs != nullptr ? coffs[i] : 0));
    bool bad = o_first != 0 || c_first != 0 || total > cap;
    for (int i = tid; i < n_keep; i += blockDim.x) {
        const int t = kept[i];
        const int b = offs[i + 1] - offs[i];
        const int kc = coffs != nullptr ? coffs[i + 1] - coffs[i] : 0;
        bad |= t < 0 || t >= n_tiles || b < 0 || b > n_v || kc < 0;
    }
    if (bad) atomicOr(&bad_shape, 1);
    __syncthreads();
    if (!bad_shape) {
        bool bs = false;
        for (int j = tid; j < o_last; j += blockDim.x) {
            const int tok = sel[j];
            bs |= tok < 0 || tok >= n_v;
        }
        if (bs) atomicOr(&bad_sel, 1);
    }
    __syncthreads();
    if (tid == 0) *status = (bad_shape | bad_sel) ? (int)RIFT_ERR_SHAPE : 0;
}

constexpr int kLdsMaxKeep = 4096;

// Half `part` (0 or 1) of packed row r: find its prompt among the offsets `so`
// (LDS or global), check it and copy that half of the row.
// so / sc: sel_offsets and ctx_offsets (sc == nullptr: no contextual rows)
__device__ __forceinline__ void compact_row(const int* so, const int* sc, long long r, int lane, int part,
                                            const u32x4_t* __restrict__ tokens, int n_v, int row_vec,
                                            int n_tiles, const int* __restrict__ kept, int n_keep,
                                            const int* __restrict__ sel, const u32x4_t* __restrict__ ctx,
                                            const u32x4_t* __restrict__ sys, int n_sys,
                                            const u32x4_t* __restrict__ qry, int n_qry, bool shared,
                                            u32x4_t* __restrict__ packed, long long cap,
                                            int* __restrict__ pos_ids) {
    const int base = shared ? n_sys : 0;   // shared prefix rows before the first prompt
    const int pre = shared ? 0 : n_sys;    // system rows inside each prompt
    const int fixed = pre + n_qry;
    const int o_first = so[0];
    const int o_last = so[n_keep];
    const int c_first = sc != nullptr ? sc[0] : 0;
    const int c_last = sc != nullptr ? sc[n_keep] : 0;
    const long long total = base + (long long)n_keep * fixed + o_last + c_last;
    if (o_first != 0 || c_first != 0 || total > cap || r >= total) return;   // reported by workgroup 0
    u32x4_t* dst = packed + (size_t)r * row_vec;
    const int half_vec = row_vec / 2;
    const int vend = part ? row_vec : half_vec;
    auto copy_row = [&](const u32x4_t* src, int position) {
        int v = lane + part * half_vec;
        for (; v + 3 * 64 < vend; v += 256) {
            u32x4_t t[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) t[j] = src[v + 64 * j];
#pragma unroll
            for (int j = 0; j < 4; ++j) dst[v + 64 * j] = t[j];
        }
        for (; v < vend; v += 64) dst[v] = src[v];
        if (lane == 0 && part == 0) pos_ids[r] = position;
    };
    if (r < base) {   // the shared prefix
        copy_row(sys + (size_t)r * row_vec, (int)r);
        return;
    }
    const long long rp = r - base;
    // the last prompt whose start rho * fixed + offs[rho] (+ coffs[rho]) is <= r
    // (starts do not decrease when the offsets are valid; the checks below keep
    // every access in bounds when they are not)
    int lo = 0, hi = n_keep - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        const long long st = (long long)mid * fixed + so[mid] + (sc != nullptr ? sc[mid] : 0);
        if (st <= rp) lo = mid; else hi = mid - 1;
    }
    const int rho = lo;
    const int o0 = so[rho];
    const int o1 = so[rho + 1];
    const int c0 = sc != nullptr ? sc[rho] : 0;
    const int c1 = sc != nullptr ? sc[rho + 1] : 0;
    const int budget = o1 - o0;
    const int kc = c1 - c0;
    const long long pl = rp - ((long long)rho * fixed + o0 + c0);
    // o0 >= 0 and o1 <= o_last keep the reads of sel_idx inside its o_last
    // entries, c0 >= 0 and c1 <= c_last those of the contextual rows
    if (budget < 0 || budget > n_v || o0 < 0 || o1 > o_last || kc < 0 || c0 < 0 || c1 > c_last || pl < 0 ||
        pl >= fixed + budget + kc)
        return;
    const int p = (int)pl;
    const u32x4_t* src;
    if (p < pre) {
        src = sys + (size_t)p * row_vec;
    } else if (p < pre + budget) {
        const int tile = kept[rho];
        const int tok = sel[o0 + (p - pre)];
        if (tok < 0 || tok >= n_v || tile < 0 || tile >= n_tiles) return;   // reported by workgroup 0
        src = tokens + ((size_t)tile * n_v + tok) * row_vec;
    } else if (p < pre + budget + kc) {
        src = ctx + (size_t)(c0 + p - pre - budget) * row_vec;
    } else {
        src = qry + (size_t)(p - pre - budget - kc) * row_vec;
    }
    copy_row(src, p + base);   // positions continue after a shared prefix
}

__global__ void __launch_bounds__(256)
compact_rows_kernel(const u32x4_t* __restrict__ tokens, int n_v, int row_vec, int n_tiles,
                    const int* __restrict__ kept, const int* __restrict__ offs, int n_keep,
                    const int* __restrict__ sel, const u32x4_t* __restrict__ ctx,
                    const int* __restrict__ coffs, const u32x4_t* __restrict__ sys, int n_sys,
                    const u32x4_t* __restrict__ qry, int n_qry, int shared, u32x4_t* __restrict__ packed,
                    long long cap, int* __restrict__ cu, int* __restrict__ pos_ids,
                    int* __restrict__ status) {
    // dynamic LDS: sel_offsets, then ctx_offsets, n_keep + 1 entries each
    // (sized 0 when there are more than kLdsMaxKeep prompts)
    extern __shared__ int offs_dyn[];
    int* offs_lds = offs_dyn;
    int* coffs_lds = offs_dyn + (n_keep + 1);
    if (blockIdx.x == 0)
        compact_validate(kept, offs, coffs, sel, n_keep, n_tiles, n_v, shared ? n_sys : 0,
                         shared ? n_qry : n_sys + n_qry, shared != 0, cap, cu, status);
    const int lane = threadIdx.x & 63;
    const long long r = (long long)blockIdx.x * 2 + (threadIdx.x >> 7);   // two rows per workgroup
    const int part = (threadIdx.x >> 6) & 1;                              // and two waves per row
    if (n_keep <= kLdsMaxKeep) {
        for (int i = threadIdx.x; i <= n_keep; i += blockDim.x) {
            offs_lds[i] = offs[i];
            if (coffs != nullptr) coffs_lds[i] = coffs[i];
        }
        __syncthreads();
        compact_row(offs_lds, coffs != nullptr ? coffs_lds : nullptr, r, lane, part, tokens, n_v, row_vec,
                    n_tiles, kept, n_keep, sel, ctx, sys, n_sys, qry, n_qry, shared != 0, packed, cap, pos_ids);
    } else {
        compact_row(offs, coffs, r, lane, part, tokens, n_v, row_vec, n_tiles, kept, n_keep, sel, ctx, sys,
                    n_sys, qry, n_qry, shared != 0, packed, cap, pos_ids);
    }
}

hipError_t launch_compact(const void* tokens, int elem_bytes, int n_tiles, int n_v, int d,
                          const int* kept, const int* offs, const int* sel, int n_keep,
                          const void* ctx, const int* coffs, const void* sys, int n_sys,
                          const void* qry, int n_qry, bool shared, void* packed, long long cap, int* cu,
                          int* pos_ids, int* status, hipStream_t st) {
    const int row_vec = (int)((size_t)d * elem_bytes / 16);
    // two waves per row of the packed buffer; at least one workgroup, for the
    // status word and cu_seqlens
    const long long g = cap > 0 ? (cap + 1) / 2 : 1;
    const size_t lds = n_keep <= kLdsMaxKeep ? (size_t)(n_keep + 1) * sizeof(int) * (coffs != nullptr ? 2 : 1) : 0;
    hipLaunchKernelGGL(compact_rows_kernel, dim3((unsigned)g), dim3(256), lds, st,
                       static_cast<const u32x4_t*>(tokens), n_v, row_vec, n_tiles, kept, offs, n_keep,
                       sel, static_cast<const u32x4_t*>(ctx), coffs, static_cast<const u32x4_t*>(sys),
                       n_sys, static_cast<const u32x4_t*>(qry),
                       n_qry, shared ? 1 : 0, static_cast<u32x4_t*>(packed), cap, cu, pos_ids, status);
    return hipGetLastError();
}

}  // namespace rift

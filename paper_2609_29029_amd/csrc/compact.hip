// Varlen compaction of the retained prompts: sequence rho is
// [n_sys system rows | selected vision rows of tile kept[rho], ascending |
//  n_qry query rows]; every retained tile is its own VLM prompt (Sec. 2.3
// Stage 2, App. B Step 5).
//
//   compact_meta  one workgroup: cu_seqlens, checks of offsets, budgets, tile
//                 ids and capacity, status word.
//   compact_rows  grid (row group, sequence), one wave per packed row: the
//                 row's source (system, selected vision or query row) from the
//                 sequence's offsets, then a coalesced 16-byte-per-lane copy
//                 with every load of the row in flight before the first store
//                 (a row of d bf16 is d/512 loads of 1 KB per wave), and the
//                 row's position id.
#include "launch.h"
#include "rift_common.h"

namespace rift {

__global__ void __launch_bounds__(1024)
compact_meta_kernel(const int* __restrict__ kept, const int* __restrict__ offs, int n_keep,
                    int n_tiles, int n_v, int fixed, long long cap, int* __restrict__ cu,
                    int* __restrict__ status) {
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    for (int i = threadIdx.x; i <= n_keep; i += blockDim.x) {
        const long long c = (long long)i * fixed + offs[i];
        cu[i] = (int)c;
        if (i < n_keep) {
            const int t = kept[i];
            const int b = offs[i + 1] - offs[i];
            if (t < 0 || t >= n_tiles || b < 0 || b > n_v) atomicOr(&bad, 1);
        }
        if (i == 0 && offs[0] != 0) atomicOr(&bad, 1);
        if (i == n_keep && c > cap) atomicOr(&bad, 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) *status = bad ? (int)RIFT_ERR_SHAPE : 0;
}

__global__ void __launch_bounds__(256)
compact_rows_kernel(const u32x4_t* __restrict__ tokens, int n_v, int row_vec, int n_tiles,
                    const int* __restrict__ kept, const int* __restrict__ offs,
                    const int* __restrict__ sel, const u32x4_t* __restrict__ sys, int n_sys,
                    const u32x4_t* __restrict__ qry, int n_qry, u32x4_t* __restrict__ packed,
                    long long cap, int* __restrict__ pos_ids, int* __restrict__ status) {
    const int rho = blockIdx.y;
    const int p = blockIdx.x * 4 + (threadIdx.x >> 6);   // position in the sequence
    const int lane = threadIdx.x & 63;
    if (*status == (int)RIFT_ERR_SHAPE) return;   // compact_meta rejected the call
    const int o0 = offs[rho];
    const int budget = offs[rho + 1] - o0;
    if (p >= n_sys + budget + n_qry) return;
    const long long row = (long long)rho * (n_sys + n_qry) + o0 + p;
    if (row >= cap) return;
    const u32x4_t* src;
    if (p < n_sys) {
        src = sys + (size_t)p * row_vec;
    } else if (p < n_sys + budget) {
        const int tok = sel[o0 + (p - n_sys)];
        const int tile = kept[rho];
        if (tok < 0 || tok >= n_v || tile < 0 || tile >= n_tiles) {
            if (lane == 0) atomicOr(status, (int)RIFT_ERR_SHAPE);
            return;
        }
        src = tokens + ((size_t)tile * n_v + tok) * row_vec;
    } else {
        src = qry + (size_t)(p - n_sys - budget) * row_vec;
    }
    u32x4_t* dst = packed + (size_t)row * row_vec;
    int v = lane;
    for (; v + 7 * 64 < row_vec; v += 512) {
        u32x4_t t[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) t[j] = __builtin_nontemporal_load(src + v + 64 * j);
#pragma unroll
        for (int j = 0; j < 8; ++j) dst[v + 64 * j] = t[j];
    }
    for (; v < row_vec; v += 64) dst[v] = src[v];
    if (lane == 0) pos_ids[row] = p;
}

hipError_t launch_compact(const void* tokens, int elem_bytes, int n_tiles, int n_v, int d,
                          const int* kept, const int* offs, const int* sel, int n_keep,
                          const void* sys, int n_sys, const void* qry, int n_qry, void* packed,
                          long long cap, int* cu, int* pos_ids, int* status, hipStream_t st) {
    hipLaunchKernelGGL(compact_meta_kernel, dim3(1), dim3(1024), 0, st, kept, offs, n_keep,
                       n_tiles, n_v, n_sys + n_qry, cap, cu, status);
    const int row_vec = (int)((size_t)d * elem_bytes / 16);
    if (cap > 0 && n_keep > 0) {
        // every sequence has at most n_sys + n_v + n_qry rows (budgets <= n_v)
        const unsigned gx = (unsigned)((n_sys + n_v + n_qry + 3) / 4);
        hipLaunchKernelGGL(compact_rows_kernel, dim3(gx, (unsigned)n_keep), dim3(256), 0, st,
                           static_cast<const u32x4_t*>(tokens), n_v, row_vec, n_tiles, kept, offs,
                           sel, static_cast<const u32x4_t*>(sys), n_sys,
                           static_cast<const u32x4_t*>(qry), n_qry, static_cast<u32x4_t*>(packed),
                           cap, pos_ids, status);
    }
    return hipGetLastError();
}

}  // namespace rift

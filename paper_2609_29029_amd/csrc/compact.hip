// Varlen compaction of the retained prompts: sequence rho is
// [n_sys system rows | selected vision rows of tile kept[rho], ascending |
//  n_qry query rows]; every retained tile is its own VLM prompt (Sec. 2.3
// Stage 2, App. B Step 5).
//
//   compact_meta  one workgroup: cu_seqlens, checks of offsets, tile ids and
//                 capacity, status word.
//   compact_rows  one wave per packed row: binary search of the row's
//                 sequence in cu_seqlens, then a coalesced 16-byte-per-lane copy
//                 of the source row (a row of d bf16 is d/512 loads of 1 KB per
//                 wave) and the row's position id.
#include "launch.h"
#include "rift_common.h"

namespace rift {

__global__ void __launch_bounds__(1024)
compact_meta_kernel(const int* __restrict__ kept, const int* __restrict__ offs, int n_keep,
                    int n_tiles, int fixed, long long cap, int* __restrict__ cu,
                    int* __restrict__ status) {
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    for (int i = threadIdx.x; i <= n_keep; i += blockDim.x) {
        const long long c = (long long)i * fixed + offs[i];
        cu[i] = (int)c;
        if (i < n_keep) {
            const int t = kept[i];
            if (t < 0 || t >= n_tiles || offs[i + 1] < offs[i]) atomicOr(&bad, 1);
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
                    const int* __restrict__ sel, int n_keep, const u32x4_t* __restrict__ sys,
                    int n_sys, const u32x4_t* __restrict__ qry, int n_qry,
                    u32x4_t* __restrict__ packed, long long cap, const int* __restrict__ cu,
                    int* __restrict__ pos_ids, int* __restrict__ status) {
    const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= cap) return;
    if (*status == (int)RIFT_ERR_SHAPE) return;
    const int total = cu[n_keep];
    if (row >= total) return;
    // largest rho with cu[rho] <= row
    int lo = 0, hi = n_keep - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu[mid] <= row) lo = mid;
        else hi = mid - 1;
    }
    const int rho = lo;
    const int p = (int)(row - cu[rho]);
    const int budget = offs[rho + 1] - offs[rho];
    const u32x4_t* src;
    if (p < n_sys) {
        src = sys + (size_t)p * row_vec;
    } else if (p < n_sys + budget) {
        const int tok = sel[offs[rho] + (p - n_sys)];
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
    for (; v + 192 < row_vec; v += 256) {
        const u32x4_t a = src[v], b = src[v + 64], c = src[v + 128], e = src[v + 192];
        dst[v] = a;
        dst[v + 64] = b;
        dst[v + 128] = c;
        dst[v + 192] = e;
    }
    for (; v < row_vec; v += 64) dst[v] = src[v];
    if (lane == 0) pos_ids[row] = p;
}

hipError_t launch_compact(const void* tokens, int elem_bytes, int n_tiles, int n_v, int d,
                          const int* kept, const int* offs, const int* sel, int n_keep,
                          const void* sys, int n_sys, const void* qry, int n_qry, void* packed,
                          long long cap, int* cu, int* pos_ids, int* status, hipStream_t st) {
    hipLaunchKernelGGL(compact_meta_kernel, dim3(1), dim3(1024), 0, st, kept, offs, n_keep,
                       n_tiles, n_sys + n_qry, cap, cu, status);
    const int row_vec = (int)((size_t)d * elem_bytes / 16);
    if (cap > 0 && n_keep > 0) {
        const long long blocks = (cap + 3) / 4;
        hipLaunchKernelGGL(compact_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                           static_cast<const u32x4_t*>(tokens), n_v, row_vec, n_tiles, kept, offs,
                           sel, n_keep, static_cast<const u32x4_t*>(sys), n_sys,
                           static_cast<const u32x4_t*>(qry), n_qry, static_cast<u32x4_t*>(packed),
                           cap, cu, pos_ids, status);
    }
    return hipGetLastError();
}

}  // namespace rift

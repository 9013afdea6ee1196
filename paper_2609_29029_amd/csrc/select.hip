// Stage 2 token retention of Rift (Sec. 2.3 Stage 2): each kept tile keeps its
// budget of dominant tokens, ranked by the per-token margin, ties to the lower
// token index, emitted in ascending index order.
//
//   select_offsets  one workgroup: validates budgets and tile ids, writes the
//                   exclusive prefix sums sel_offsets and the status word.
//   select_topk     one workgroup per kept tile: bitonic sort of the tile's
//                   (key, index) pairs in LDS -- descending key, ascending index
//                   -- marks the first `budget` positions, then a ballot/prefix
//                   pass writes the marked indices in ascending order.
#include "launch.h"
#include "rift_common.h"

namespace rift {

__global__ void __launch_bounds__(1024)
select_offsets_kernel(const int* __restrict__ kept, const int* __restrict__ budgets, int n_keep,
                      int n_tiles, int n_v, long long cap, int* __restrict__ offs,
                      int* __restrict__ status) {
    __shared__ int bad;
    __shared__ int scan[1024];
    __shared__ long long carry;
    const int tid = threadIdx.x;
    if (tid == 0) {
        bad = 0;
        carry = 0;
    }
    __syncthreads();
    for (int i = tid; i < n_keep; i += blockDim.x) {
        const int b = budgets[i];
        const int t = kept[i];
        if (b < 0 || b > n_v || t < 0 || t >= n_tiles) atomicOr(&bad, 1);
    }
    for (int base = 0; base < n_keep; base += 1024) {
        const int i = base + tid;
        int v = 0;
        if (i < n_keep) {
            v = budgets[i];
            v = v < 0 ? 0 : (v > n_v ? n_v : v);
        }
        scan[tid] = v;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int add = tid >= off ? scan[tid - off] : 0;
            __syncthreads();
            scan[tid] += add;
            __syncthreads();
        }
        if (i < n_keep) offs[i] = (int)(carry + scan[tid] - v);
        __syncthreads();
        if (tid == 0) carry += scan[1023];
        __syncthreads();
    }
    if (tid == 0 && carry > cap) bad = 1;
    __syncthreads();
    if (bad) {
        for (int i = tid; i <= n_keep; i += blockDim.x) offs[i] = 0;
    } else if (tid == 0) {
        offs[n_keep] = (int)carry;
    }
    if (tid == 0) *status = bad ? (int)RIFT_ERR_BUDGET : 0;
}

__device__ __forceinline__ bool key_before(double ka, int ia, double kb, int ib) {
    return (ka > kb) || (ka == kb && ia < ib);
}

__global__ void __launch_bounds__(256)
select_topk_kernel(const double* __restrict__ token_key, int n_v, const int* __restrict__ kept,
                   const int* __restrict__ offs, const int* __restrict__ status,
                   int* __restrict__ sel_idx) {
    __shared__ double key[1024];
    __shared__ int idx[1024];
    __shared__ unsigned char flag[1024];
    __shared__ int wave_tot[4];
    if (*status != 0) return;
    const int rho = blockIdx.x;
    const int off = offs[rho];
    const int budget = offs[rho + 1] - off;
    if (budget <= 0) return;
    const int tid = threadIdx.x;
    if (budget >= n_v) {
        for (int i = tid; i < n_v; i += blockDim.x) sel_idx[off + i] = i;
        return;
    }
    const double* kt = token_key + (size_t)kept[rho] * n_v;
    int N = 1;
    while (N < n_v) N <<= 1;
    for (int i = tid; i < N; i += blockDim.x) {
        key[i] = i < n_v ? kt[i] : -INFINITY;
        idx[i] = i;
    }
    __syncthreads();
    for (int size = 2; size <= N; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = tid; t < (N >> 1); t += blockDim.x) {
                const int i = 2 * t - (t & (stride - 1));
                const int j = i + stride;
                const bool up = (i & size) == 0;
                const bool sw = up ? key_before(key[j], idx[j], key[i], idx[i])
                                   : key_before(key[i], idx[i], key[j], idx[j]);
                if (sw) {
                    const double tk = key[i];
                    key[i] = key[j];
                    key[j] = tk;
                    const int ti = idx[i];
                    idx[i] = idx[j];
                    idx[j] = ti;
                }
            }
            __syncthreads();
        }
    }
    for (int i = tid; i < 1024; i += blockDim.x) flag[i] = 0;
    __syncthreads();
    for (int p = tid; p < budget; p += blockDim.x) flag[idx[p]] = 1;
    __syncthreads();
    // Ascending emission: thread t owns indices [4t, 4t+4); wave ballots give
    // the prefix of set flags before each thread.
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int mine = 0;
    for (int e = 0; e < 4; ++e) mine += flag[4 * tid + e];
    // inclusive scan of `mine` within the wave
    int incl = mine;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
        const int o = __shfl_up(incl, s);
        if (lane >= s) incl += o;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += wave_tot[w];
    int pos = base + incl - mine;
    for (int e = 0; e < 4; ++e) {
        const int i = 4 * tid + e;
        if (flag[i]) sel_idx[off + pos++] = i;
    }
}

hipError_t launch_select(const double* token_key, int n_tiles, int n_v, const int* kept,
                         const int* budgets, int n_keep, int* sel_offsets, int* sel_idx,
                         long long cap, int* status, hipStream_t st) {
    hipLaunchKernelGGL(select_offsets_kernel, dim3(1), dim3(1024), 0, st, kept, budgets, n_keep,
                       n_tiles, n_v, cap, sel_offsets, status);
    if (n_keep > 0)
        hipLaunchKernelGGL(select_topk_kernel, dim3(n_keep), dim3(256), 0, st, token_key, n_v, kept,
                           sel_offsets, status, sel_idx);
    return hipGetLastError();
}

}  // namespace rift

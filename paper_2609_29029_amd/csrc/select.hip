// Stage 2 token retention of Rift (Sec. 2.3 Stage 2): each kept tile keeps its
// budget of dominant tokens, ranked by the per-token margin, ties to the lower
// token index, emitted in ascending index order.
//
//   select_offsets  one workgroup: validates budgets and tile ids, writes the
//                   exclusive prefix sums sel_offsets (each thread sums a
//                   contiguous run, then one scan over the threads) and the
//                   status word.
//   select_topk     one wave per kept tile, keys in registers: an 8-pass radix
//                   select (8-bit digits, histogram in the wave's own LDS
//                   slice) finds the budget-th pair in (descending key,
//                   ascending index) order, then ballot prefix counts write the
//                   chosen indices in ascending order.
#include "launch.h"
#include "rift_common.h"

namespace rift {

__global__ void __launch_bounds__(1024)
select_offsets_kernel(const int* __restrict__ kept, const int* __restrict__ budgets, int n_keep,
                      int n_tiles, int n_v, long long cap, int* __restrict__ offs,
                      int* __restrict__ status) {
    __shared__ int bad;
    __shared__ long long wave_sum[16];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid == 0) bad = 0;
    __syncthreads();
    // thread t owns budgets [t per, (t + 1) per): validate and sum them
    const int per = (n_keep + 1023) / 1024;
    const int i0 = tid * per;
    long long mine = 0;
    for (int j = 0; j < per; ++j) {
        const int i = i0 + j;
        if (i >= n_keep) break;
        const int b = budgets[i];
        const int t = kept[i];
        if (b < 0 || b > n_v || t < 0 || t >= n_tiles) atomicOr(&bad, 1);
        mine += b < 0 ? 0 : (b > n_v ? n_v : b);
    }
    // exclusive scan over threads: within the wave, then across the 16 waves
    long long incl = mine;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
        const long long o = __shfl_up(incl, s);
        if (lane >= s) incl += o;
    }
    if (lane == 63) wave_sum[wave] = incl;
    __syncthreads();
    long long base = 0, total = 0;
    for (int w = 0; w < 16; ++w) {
        if (w < wave) base += wave_sum[w];
        total += wave_sum[w];
    }
    if (tid == 0 && total > cap) bad = 1;
    __syncthreads();
    if (bad) {
        for (int i = tid; i <= n_keep; i += blockDim.x) offs[i] = 0;
    } else {
        long long run = base + incl - mine;
        for (int j = 0; j < per; ++j) {
            const int i = i0 + j;
            if (i >= n_keep) break;
            offs[i] = (int)run;
            const int b = budgets[i];
            run += b < 0 ? 0 : (b > n_v ? n_v : b);
        }
        if (tid == 0) offs[n_keep] = (int)total;
    }
    if (tid == 0) *status = bad ? (int)RIFT_ERR_BUDGET : 0;
}

// Order-preserving map of a key to an unsigned integer, descending: a larger
// key gives a smaller value.  -0 is first made +0 so that the two compare equal,
// as they do as doubles.
__device__ __forceinline__ uint64_t desc_bits(double x) {
    const uint64_t b = __builtin_bit_cast(uint64_t, x + 0.0);
    const uint64_t asc = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
    return ~asc;
}

constexpr int kSelMaxPerLane = 16;   // n_v <= 1024

__global__ void __launch_bounds__(256)
select_topk_kernel(const double* __restrict__ token_key, int n_v, int n_keep,
                   const int* __restrict__ kept, const int* __restrict__ offs,
                   const int* __restrict__ status, int* __restrict__ sel_idx) {
    __shared__ unsigned hist_all[4][256];
    if (*status != 0) return;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int rho = blockIdx.x * 4 + wave;
    if (rho >= n_keep) return;
    const int off = offs[rho];
    const int budget = offs[rho + 1] - off;
    if (budget <= 0) return;
    if (budget >= n_v) {
        for (int i = lane; i < n_v; i += 64) sel_idx[off + i] = i;
        return;
    }
    unsigned* hist = hist_all[wave];
    const double* kt = token_key + (size_t)kept[rho] * n_v;
    const int ne = (n_v + 63) >> 6;   // elements per lane; element e of lane l is index 64 e + l
    uint64_t u[kSelMaxPerLane];
#pragma unroll
    for (int e = 0; e < kSelMaxPerLane; ++e) {
        const int i = 64 * e + lane;
        u[e] = (e < ne && i < n_v) ? desc_bits(kt[i]) : ~0ull;   // padding sorts last
    }
    // the budget-th smallest value T of u over the valid elements, digit by digit
    uint64_t prefix = 0, mask = 0;
    int k = budget;
    for (int shift = 56; shift >= 0; shift -= 8) {
#pragma unroll
        for (int j = 0; j < 4; ++j) hist[4 * lane + j] = 0;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int e = 0; e < kSelMaxPerLane; ++e) {
            const int i = 64 * e + lane;
            if (e < ne && i < n_v && (u[e] & mask) == prefix)
                atomicAdd(&hist[(unsigned)(u[e] >> shift) & 255u], 1u);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        unsigned c[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) c[j] = hist[4 * lane + j];
        const unsigned mine = c[0] + c[1] + c[2] + c[3];
        unsigned incl = mine;
#pragma unroll
        for (int sft = 1; sft < 64; sft <<= 1) {
            const unsigned o = __shfl_up(incl, sft);
            if (lane >= sft) incl += o;
        }
        unsigned before = incl - mine;   // count in bins < 4 lane
        int hit = -1;
        unsigned hit_before = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (hit < 0 && before < (unsigned)k && (unsigned)k <= before + c[j]) {
                hit = 4 * lane + j;
                hit_before = before;
            }
            before += c[j];
        }
        const uint64_t hits = __ballot(hit >= 0);
        const int src = __builtin_ctzll(hits);   // exactly one lane holds the digit
        const int digit = __shfl(hit, src);
        k -= (int)__shfl(hit_before, src);
        prefix |= (uint64_t)digit << shift;
        mask |= 255ull << shift;
    }
    // take every u < T, and the first k (by index) of u == T; write ascending
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int eq_seen = 0, written = 0;
#pragma unroll
    for (int e = 0; e < kSelMaxPerLane; ++e) {
        if (e >= ne) break;
        const int i = 64 * e + lane;
        const bool valid = i < n_v;
        const bool eq = valid && u[e] == prefix;
        const uint64_t eqm = __ballot(eq);
        const bool take = valid && (u[e] < prefix || (eq && eq_seen + __popcll(eqm & below) < k));
        eq_seen += __popcll(eqm);
        const uint64_t tm = __ballot(take);
        if (take) sel_idx[off + written + __popcll(tm & below)] = i;
        written += __popcll(tm);
    }
}

hipError_t launch_select(const double* token_key, int n_tiles, int n_v, const int* kept,
                         const int* budgets, int n_keep, int* sel_offsets, int* sel_idx,
                         long long cap, int* status, hipStream_t st) {
    hipLaunchKernelGGL(select_offsets_kernel, dim3(1), dim3(1024), 0, st, kept, budgets, n_keep,
                       n_tiles, n_v, cap, sel_offsets, status);
    if (n_keep > 0)
        hipLaunchKernelGGL(select_topk_kernel, dim3((n_keep + 3) / 4), dim3(256), 0, st, token_key, n_v,
                           n_keep, kept, sel_offsets, status, sel_idx);
    return hipGetLastError();
}

}  // namespace rift

// Stage 2 token retention of Rift (Sec. 2.3 Stage 2): each kept tile keeps its
// budget of dominant tokens, ranked by the per-token margin, ties to the lower
// token index, emitted in ascending index order.
//
//   select_offsets  one workgroup: validates budgets and tile ids, writes the
//                   exclusive prefix sums sel_offsets (each thread sums a
//                   contiguous run, then one scan over the threads) and the
//                   status word.
//   select_topk     one wave per kept tile, keys in registers: a radix select
//                   (8-bit digits from the top, histogram in the wave's own
//                   LDS slice; it stops once the bin that holds the
//                   budget-th key is taken whole) finds the budget-th pair in
//                   (descending key, ascending index) order, then ballot
//                   prefix counts write the chosen indices in ascending order.
#include "launch.h"
#include "rift_common.h"

namespace rift {

constexpr int kOffBatch = 8;

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
    // thread t owns budgets [t per, (t + 1) per): validate and sum them, in
    // batches of kOffBatch whose loads are all issued before the first is used
    const int per = (n_keep + 1023) / 1024;
    const int i0 = tid * per;
    const int i1 = min(i0 + per, n_keep);
    long long mine = 0;
    bool bad_mine = false;
    for (int j0 = i0; j0 < i1; j0 += kOffBatch) {
        int bv[kOffBatch], tv[kOffBatch];
#pragma unroll
        for (int j = 0; j < kOffBatch; ++j) {
            const int i = min(j0 + j, i1 - 1);
            bv[j] = budgets[i];
            tv[j] = kept[i];
        }
#pragma unroll
        for (int j = 0; j < kOffBatch; ++j) {
            if (j0 + j >= i1) break;
            const int b = bv[j], t = tv[j];
            bad_mine |= b < 0 || b > n_v || t < 0 || t >= n_tiles;
            mine += b < 0 ? 0 : (b > n_v ? n_v : b);
        }
    }
    if (bad_mine) atomicOr(&bad, 1);
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
        for (int j0 = i0; j0 < i1; j0 += kOffBatch) {
            int bv[kOffBatch];
#pragma unroll
            for (int j = 0; j < kOffBatch; ++j) bv[j] = budgets[min(j0 + j, i1 - 1)];
#pragma unroll
            for (int j = 0; j < kOffBatch; ++j) {
                if (j0 + j >= i1) break;
                offs[j0 + j] = (int)run;
                run += bv[j];   // validated above: 0 <= bv[j] <= n_v
            }
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


// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: shifts by
// 1, 2, 4 and 8 inside each row of 16 lanes (lanes shifted in from outside
// the row contribute 0), then the last lane of row 0 is added to row 1 and row
// 3 gets row 2's, and finally lane 31 is added to rows 2 and 3.
__device__ __forceinline__ unsigned wave_incl_scan(unsigned v) {
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

// NE: keys per lane the kernel is built for (n_v <= 64 NE); 9 covers a 24 x 24
// token tile, 16 the largest n_v (1024).
template <int NE>
__global__ void __launch_bounds__(256)
select_topk_kernel(const double* __restrict__ token_key, int n_v, int n_keep,
                   const int* __restrict__ kept, const int* __restrict__ offs,
                   const int* __restrict__ status, int* __restrict__ sel_idx) {
    __shared__ unsigned hist_all[4][256];
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int rho = blockIdx.x * 4 + wave;
    if (rho >= n_keep) return;
    // the status word, this tile's offsets and its id are loaded together
    const int bad = *status;
    const int off = offs[rho];
    const int off_end = offs[rho + 1];
    const int tile = kept[rho];
    if (bad != 0) return;
    const int budget = off_end - off;
    if (budget <= 0) return;
    if (budget >= n_v) {
        for (int i = lane; i < n_v; i += 64) sel_idx[off + i] = i;
        return;
    }
    unsigned* hist = hist_all[wave];
    const double* kt = token_key + (size_t)tile * n_v;
    const int ne = (n_v + 63) >> 6;   // elements per lane; element e of lane l is index 64 e + l
    // every load in bounds (index clamped to the last key), none behind a branch,
    // so the wave waits for its keys once
    double raw[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) raw[e] = kt[min(64 * e + lane, n_v - 1)];
    uint64_t u[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e)
        u[e] = (64 * e + lane < n_v) ? desc_bits(raw[e]) : ~0ull;   // padding sorts last
    // the budget-th smallest value T of u over the valid elements, digit by digit
    uint64_t prefix = 0, mask = 0;
    int k = budget;
    for (int shift = 56; shift >= 0; shift -= 8) {
#pragma unroll
        for (int j = 0; j < 4; ++j) hist[4 * lane + j] = 0;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int i = 64 * e + lane;
            if (e < ne && i < n_v && (u[e] & mask) == prefix)
                atomicAdd(&hist[(unsigned)(u[e] >> shift) & 255u], 1u);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        unsigned c[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) c[j] = hist[4 * lane + j];
        const unsigned mine = c[0] + c[1] + c[2] + c[3];
        unsigned before = wave_incl_scan(mine) - mine;   // count in bins < 4 lane
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
        unsigned hit_count = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (hit == 4 * lane + j) hit_count = c[j];
        const uint64_t hits = __ballot(hit >= 0);
        const int src = __builtin_ctzll(hits);   // exactly one lane holds the digit
        const int digit = __builtin_amdgcn_readlane(hit, src);
        k -= (int)__builtin_amdgcn_readlane(hit_before, src);
        prefix |= (uint64_t)digit << shift;
        mask |= 255ull << shift;
        // every candidate left in the bin is taken: the digits below no longer matter
        if ((int)__builtin_amdgcn_readlane(hit_count, src) == k) break;
    }
    // take every u whose masked value is below the prefix, and the first k (by
    // index) of those equal to it; write ascending
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int eq_seen = 0, written = 0;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        if (e >= ne) break;
        const int i = 64 * e + lane;
        const bool valid = i < n_v;
        const uint64_t um = u[e] & mask;
        const bool eq = valid && um == prefix;
        const uint64_t eqm = __ballot(eq);
        const bool take = valid && (um < prefix || (eq && eq_seen + __popcll(eqm & below) < k));
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
        if (n_v <= 64 * 9)
            hipLaunchKernelGGL(select_topk_kernel<9>, dim3((n_keep + 3) / 4), dim3(256), 0, st, token_key,
                               n_v, n_keep, kept, sel_offsets, status, sel_idx);
        else
            hipLaunchKernelGGL(select_topk_kernel<16>, dim3((n_keep + 3) / 4), dim3(256), 0, st, token_key,
                               n_v, n_keep, kept, sel_offsets, status, sel_idx);
    return hipGetLastError();
}

}  // namespace rift

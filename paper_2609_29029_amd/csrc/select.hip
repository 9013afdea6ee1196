// Stage 2 token retention of Rift (Sec. 2.3 Stage 2): each kept tile keeps its
// budget of dominant tokens, ranked by the per-token margin, ties to the lower
// token index, emitted in ascending index order.
//
// One launch.  A workgroup of W waves handles W consecutive kept tiles, one
// wave per tile:
//   1. the wave issues the loads of its tile's keys (tile id clamped so every
//      read is in bounds whatever the ids hold);
//   2. meanwhile the workgroup reads every budget and tile id of the call:
//      the call is valid only if all of them are in range and the total fits
//      (then every workgroup reaches the same verdict), and the sum of the
//      budgets before its first tile is its base offset;
//   3. each wave finds the budget-th key of its tile, (key desc, index asc),
//      by deciding the order-preserving key bits one at a time from the
//      highest bit in which its keys differ: per bit, a ballot per element
//      counts the candidates with a 0 there; the side that holds the
//      budget-th key stays candidate, and when that is the 1 side every
//      0-side candidate is taken.  The search ends once the candidates left
//      are exactly the ones still needed (on distinct keys after about
//      log2(n_v) + 2 bits), else after bit 0 with equal keys, of which the
//      lowest indices are taken.  Candidate and taken sets are wave-wide bit
//      masks (lane l, element e = token 64 e + l), so the search is a few
//      vector compares and scalar mask operations per bit, with no shared
//      memory traffic;
//   4. the taken tokens are written in ascending index order (ballot prefix
//      counts).
// Workgroup 0 writes the status word; the workgroup of the last tile writes
// the total offset.
//
// Step 2 costs every workgroup a read of all budgets and ids, which grows with
// the square of the tile count.  Calls of more than 8,192 kept tiles therefore
// run two launches: one workgroup checks the call and writes the offsets and
// the status word (select_scan_kernel), then the selection kernel reads its
// tile's offset and the verdict instead of step 2.
#include "launch.h"
#include "rift_common.h"

namespace rift {

typedef int i32x4_t __attribute__((ext_vector_type(4)));


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

// Sum over the wave (every lane gets it).
__device__ __forceinline__ int wave_sum(int v) {
    return __builtin_amdgcn_readlane((int)wave_incl_scan((unsigned)v), 63);
}

// Minimum and maximum over the wave, by the same DPP steps (lanes shifted in
// from outside contribute the identity), read from lane 63.
__device__ __forceinline__ float wave_min(float v) {
    const int inf = __builtin_bit_cast(int, INFINITY);
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x111, 0xf, 0xf, false)));
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x112, 0xf, 0xf, false)));
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x114, 0xf, 0xf, false)));
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x118, 0xf, 0xf, false)));
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x142, 0xa, 0xf, false)));
    v = fminf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(inf, __builtin_bit_cast(int, v), 0x143, 0xc, 0xf, false)));
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float wave_max(float v) { return -wave_min(-v); }

// Large calls, first launch: one workgroup checks every budget (in [0, n_v])
// and tile id (in [0, n_tiles)) of the call and the total (at most cap), and
// writes the exclusive prefix sums of the budgets, their total and the status
// word.  Chunks of kChunk entries: thread t loads entries t + 1024 j (whole
// cache lines per instruction, the next chunk's loads in flight while this one
// is scanned), the budgets go through LDS so that thread t sums the contiguous
// run [kRun t, kRun (t + 1)), a wave scan and the 16 wave totals give each
// run's base, and the offsets return through LDS to be stored as they were
// loaded.  Offsets are written as they are found and, if the call turns out
// invalid, all set to 0 afterwards.
constexpr int kScanThreads = 1024;
constexpr int kRun = 16;
constexpr int kChunk = kRun * kScanThreads;
// Kept tiles above which the two launches beat one: measured 28 against 25 us
// at 6,400 tiles, 103 against 159 us at 51,200.
constexpr int kScanFrom = 8192;
// LDS word of chunk entry i: run t = i / 16 holds words [16 t, 16 t + 16), its
// 4-entry quads rotated by (t / 4) mod 4 so that 16 consecutive runs' quad
// reads (16 bytes a lane) meet 16 different bank groups.
__device__ __forceinline__ unsigned scan_word(unsigned i) {
    return 16u * (i >> 4) + 4u * ((((i >> 2) & 3u) + ((i >> 6) & 3u)) & 3u) + (i & 3u);
}

__global__ void __launch_bounds__(kScanThreads)
select_scan_kernel(const int* __restrict__ kept, const int* __restrict__ budgets, int n_keep, int n_tiles,
                   int n_v, int cap, int* __restrict__ offs, int* __restrict__ status) {
    __shared__ __align__(16) unsigned lb[kChunk];
    __shared__ unsigned wsum[kScanThreads / 64];
    __shared__ int wbad[kScanThreads / 64];
    const unsigned tid = threadIdx.x;
    const unsigned lane = tid & 63u;
    const unsigned wave = tid >> 6;
    const unsigned n = (unsigned)n_keep;   // indices below n + kChunk < 2^32
    unsigned carry = 0u;   // budgets of the earlier chunks (no wrap-around while they are valid)
    bool bad = false;
    unsigned nb[kRun], nt[kRun];
    auto load = [&](unsigned c) {
#pragma unroll
        for (int j = 0; j < kRun; ++j) {
            const unsigned i = c + (unsigned)j * kScanThreads + tid;
            nb[j] = i < n ? (unsigned)budgets[i] : 0u;
            nt[j] = i < n ? (unsigned)kept[i] : 0u;
        }
    };
    load(0u);
    for (unsigned c = 0; c < n; c += kChunk) {
#pragma unroll
        for (int j = 0; j < kRun; ++j) {
            bad = bad || nb[j] > (unsigned)n_v || nt[j] >= (unsigned)n_tiles;   // negative values are huge
            lb[scan_word((unsigned)j * kScanThreads + tid)] = nb[j];
        }
        if (c + kChunk < n) load(c + kChunk);
        __syncthreads();
        const unsigned rot = (tid >> 2) & 3u;
        unsigned v[kRun];
        unsigned sum = 0u;
#pragma unroll
        for (int q = 0; q < kRun / 4; ++q) {
            const u32x4_t x = *reinterpret_cast<const u32x4_t*>(lb + 16u * tid + 4u * ((q + rot) & 3u));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[4 * q + e] = x[e];
                sum += x[e];
            }
        }
        const unsigned incl = wave_incl_scan(sum);
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        unsigned before = 0u, chunk = 0u;
#pragma unroll
        for (int w = 0; w < kScanThreads / 64; ++w) {
            const unsigned x = wsum[w];
            before += (unsigned)w < wave ? x : 0u;
            chunk += x;
        }
        unsigned run = carry + before + incl - sum;
#pragma unroll
        for (int q = 0; q < kRun / 4; ++q) {
            u32x4_t o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                o[e] = run;
                run += v[4 * q + e];
            }
            *reinterpret_cast<u32x4_t*>(lb + 16u * tid + 4u * ((q + rot) & 3u)) = o;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kRun; ++j) {
            const unsigned i = c + (unsigned)j * kScanThreads + tid;
            if (i < n) offs[i] = (int)lb[scan_word((unsigned)j * kScanThreads + tid)];
        }
        carry += chunk;
        __syncthreads();   // lb and wsum are refilled by the next chunk
    }
    const bool wave_bad = __ballot(bad) != 0ull;
    if (lane == 0) wbad[wave] = wave_bad;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the offsets stored, before any is cleared
    __syncthreads();
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < kScanThreads / 64; ++w) any_bad |= wbad[w];
    // valid budgets keep the total within n_tiles * n_v <= INT32_MAX
    const bool valid = any_bad == 0 && carry <= (unsigned)cap;
    if (!valid) {
        for (unsigned i = tid; i < n; i += kScanThreads) offs[i] = 0;
    }
    if (tid == 0) {
        offs[n_keep] = valid ? (int)carry : 0;
        *status = valid ? 0 : (int)RIFT_ERR_BUDGET;
    }
}

// NE: keys per lane the kernel is built for (n_v <= 64 NE); W: waves (kept
// tiles) per workgroup; PRE: select_scan_kernel has checked the call and
// written the offsets and the status word.
template <int NE, int W, bool PRE>
__global__ void __launch_bounds__(64 * W)
select_kernel(const double* __restrict__ token_key, int n_tiles, int n_v, int n_keep,
              const int* __restrict__ kept, const int* __restrict__ budgets, int cap,
              int* __restrict__ offs, int* __restrict__ sel_idx, int* __restrict__ status) {
    __shared__ int red_before[W], red_total[W], red_bad[W];
    __shared__ __align__(16) unsigned hist_all[W][256];
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave: keeps the masks scalar
    const int lane = tid & 63;
    const int first = blockIdx.x * W;
    const int rho = first + wave;
    const bool has_tile = rho < n_keep;

    // 1. the loads, longest first: this wave's tile id; the first round of
    //    every budget and id of the call (16 bytes at a time when both arrays
    //    allow it); this wave's keys (tile id clamped: every read is in bounds
    //    whatever the ids hold); the budgets of this workgroup's tiles up to
    //    this wave's (uniform, through the scalar cache)
    int tile = has_tile ? kept[rho] : 0;
    const bool vec = ((reinterpret_cast<uintptr_t>(budgets) | reinterpret_cast<uintptr_t>(kept)) & 15u) == 0;
    constexpr int kV = 4;                       // 16-byte vectors per thread per round
    constexpr int kRound = kV * 64 * W;         // vectors per round
    const int n4 = (vec && !PRE) ? n_keep >> 2 : 0;   // whole vectors; the rest one by one
    i32x4_t bv[kV], tv[kV];
    if (n4 > 0) {
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            const int v = min(tid + j * 64 * W, n4 - 1);
            bv[j] = reinterpret_cast<const i32x4_t*>(budgets)[v];
            tv[j] = reinterpret_cast<const i32x4_t*>(kept)[v];
        }
    }
    tile = tile < 0 ? 0 : (tile >= n_tiles ? n_tiles - 1 : tile);
    const char* kb = reinterpret_cast<const char*>(token_key + (size_t)tile * n_v);
    double raw[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        const unsigned i = min((unsigned)(64 * e + lane), (unsigned)(n_v - 1));
        raw[e] = *reinterpret_cast<const double*>(kb + i * 8u);
    }
    int off = 0, budget = 0;
    if constexpr (PRE) {
        // the first launch's verdict, this tile's offset and budget (checked)
        if (!has_tile) return;
        if (__builtin_amdgcn_readfirstlane(*status) != 0) return;
        off = __builtin_amdgcn_readfirstlane(offs[rho]);
        budget = __builtin_amdgcn_readfirstlane(budgets[rho]);
    } else {
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const int bw = first + w < n_keep ? budgets[first + w] : 0;
            off += w < wave ? bw : 0;
            budget = w == wave ? bw : budget;
        }

        // 2. validity, base offset and total of the call: the largest budget and
        //    id as unsigned values (a negative one is huge), the sums
        unsigned bmax = 0u, tmax = 0u, total = 0u, before = 0u;
        auto acc4 = [&](int v, const i32x4_t& b4, const i32x4_t& t4) __attribute__((always_inline)) {
            bmax = max(bmax, max(max((unsigned)b4[0], (unsigned)b4[1]), max((unsigned)b4[2], (unsigned)b4[3])));
            tmax = max(tmax, max(max((unsigned)t4[0], (unsigned)t4[1]), max((unsigned)t4[2], (unsigned)t4[3])));
            const unsigned s = (unsigned)b4[0] + (unsigned)b4[1] + (unsigned)b4[2] + (unsigned)b4[3];
            total += s;
            if (4 * v + 3 < first) {
                before += s;
            } else if (4 * v < first) {
#pragma unroll
                for (int c = 0; c < 4; ++c) before += 4 * v + c < first ? (unsigned)b4[c] : 0u;
            }
        };
#pragma unroll
        for (int j = 0; j < kV; ++j)
            if (tid + j * 64 * W < n4) acc4(tid + j * 64 * W, bv[j], tv[j]);
        for (int v0 = tid + kRound; v0 < n4; v0 += kRound) {   // calls of more than one round
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                const int v = min(v0 + j * 64 * W, n4 - 1);
                bv[j] = reinterpret_cast<const i32x4_t*>(budgets)[v];
                tv[j] = reinterpret_cast<const i32x4_t*>(kept)[v];
            }
#pragma unroll
            for (int j = 0; j < kV; ++j)
                if (v0 + j * 64 * W < n4) acc4(v0 + j * 64 * W, bv[j], tv[j]);
        }
        for (int i = 4 * n4 + tid; i < n_keep; i += 64 * W) {
            const unsigned bi = (unsigned)budgets[i];
            bmax = max(bmax, bi);
            tmax = max(tmax, (unsigned)kept[i]);
            total += bi;
            before += i < first ? bi : 0u;
        }
        before = wave_sum((int)before);
        total = wave_sum((int)total);
        const bool any_bad = __ballot(bmax > (unsigned)n_v || tmax >= (unsigned)n_tiles) != 0ull;
        if (lane == 0) {
            red_before[wave] = (int)before;
            red_total[wave] = (int)total;
            red_bad[wave] = any_bad;
        }
        // only shared memory is waited for at the barrier, so the keys stay in flight
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        before = 0u;
        total = 0u;
        int badw = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            before += (unsigned)red_before[w];
            total += (unsigned)red_total[w];
            badw |= red_bad[w];
        }
        // valid budgets and ids keep every sum within n_tiles * n_v <= INT32_MAX
        if (badw == 0 && total > (unsigned)cap) badw = 1;
        badw = __builtin_amdgcn_readfirstlane(badw);
        if (blockIdx.x == 0 && tid == 0) {
            *status = badw ? (int)RIFT_ERR_BUDGET : 0;
            if (n_keep == 0) offs[0] = 0;
        }
        off = __builtin_amdgcn_readfirstlane((int)before + off);
        if (has_tile && lane == 0) {
            offs[rho] = badw ? 0 : off;
            if (rho == n_keep - 1) offs[n_keep] = badw ? 0 : (int)total;
        }
        if (badw || !has_tile) return;
        budget = __builtin_amdgcn_readfirstlane(budget);
    }
    if (budget <= 0) return;
    int* out = sel_idx + off;
    if (budget >= n_v) {
        for (int i = lane; i < n_v; i += 64) out[i] = i;
        return;
    }

    // 3. which tokens to take.  First, when the keys are finite as float32
    // and not all equal, one histogram pass over 256 value buckets of their
    // float32 range: bucket = trunc((max - f) * (256 / (max - min))), clamped
    // to 255, with f the key rounded to float32.  Each step (the rounding to
    // float32, the subtraction, the product with a positive factor, the
    // truncation) is monotone, so every key of a lower bucket is strictly
    // larger than every key of a higher one.  The buckets before the one that
    // holds the budget-th key are taken whole; that bucket's keys, usually a
    // handful, are the candidates for the rest.
    unsigned* hist = hist_all[wave];
    uint64_t cand[NE], take[NE];
    int k = budget;
    int ncand = n_v;
    bool fin = true;
    float fmn = INFINITY, fmx = -INFINITY;
    float f[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        const int base = 64 * e;
        cand[e] = base >= n_v ? 0ull : (base + 64 <= n_v ? ~0ull : ((1ull << (n_v - base)) - 1ull));
        take[e] = 0ull;
        f[e] = (float)raw[e];
        if (base + lane < n_v) {
            fin = fin && (f[e] - f[e] == 0.0f);   // false for NaN, infinities and float32 overflow
            fmn = fminf(fmn, f[e]);
            fmx = fmaxf(fmx, f[e]);
        }
    }
    fmn = wave_min(fmn);
    fmx = wave_max(fmx);
    const bool all_finite = __ballot(!fin) == 0ull;
    const float range = __fsub_rn(fmx, fmn);
    const float scale = 256.0f / range;
    if (all_finite && range > 0.0f && range - range == 0.0f && scale - scale == 0.0f) {
        int bkt[NE];
        *reinterpret_cast<u32x4_t*>(hist + 4 * lane) = u32x4_t{0u, 0u, 0u, 0u};
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int t = (int)__fmul_rn(__fsub_rn(fmx, f[e]), scale);
            bkt[e] = t < 255 ? t : 255;
            if (64 * e + lane < n_v) atomicAdd(&hist[bkt[e]], 1u);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const u32x4_t c = *reinterpret_cast<const u32x4_t*>(hist + 4 * lane);
        const unsigned mine = c[0] + c[1] + c[2] + c[3];
        unsigned bsum = wave_incl_scan(mine) - mine;   // keys in buckets < 4 lane
        int hit = -1;
        unsigned hit_before = 0, hit_count = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (hit < 0 && bsum < (unsigned)k && (unsigned)k <= bsum + c[j]) {
                hit = 4 * lane + j;
                hit_before = bsum;
                hit_count = c[j];
            }
            bsum += c[j];
        }
        const int src = __builtin_ctzll(__ballot(hit >= 0));   // exactly one lane holds the bucket
        const int B = __builtin_amdgcn_readlane(hit, src);
        k -= (int)__builtin_amdgcn_readlane(hit_before, src);
        ncand = (int)__builtin_amdgcn_readlane(hit_count, src);
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            take[e] = __ballot(bkt[e] < B) & cand[e];
            cand[e] = __ballot(bkt[e] == B) & cand[e];
        }
    }
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (ncand != k && ncand <= 64 && all_finite) {
        // Rank each candidate among the candidates by (key desc, index asc)
        // with plain float64 comparisons (-0 and +0 compare equal); take the
        // first k.  The histogram's slice of shared memory holds them.
        double* cx = reinterpret_cast<double*>(hist);
        int* ci = reinterpret_cast<int*>(hist + 128);
        int* chosen = reinterpret_cast<int*>(hist + 192);
        int slot0 = 0;
        int slot[NE];
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            slot[e] = slot0 + __popcll(cand[e] & below);
            if ((cand[e] >> lane) & 1ull) {
                cx[slot[e]] = raw[e];
                ci[slot[e]] = 64 * e + lane;
            }
            slot0 += __popcll(cand[e]);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (lane < ncand) {
            const double mx = cx[lane];
            const int mi = ci[lane];
            int r = 0;
            for (int j = 0; j < ncand; ++j) {
                const double xj = cx[j];
                const int ij = ci[j];
                r += (xj > mx || (xj == mx && ij < mi)) ? 1 : 0;
            }
            chosen[lane] = r < k ? 1 : 0;
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const bool mine_c = (cand[e] >> lane) & 1ull;
            take[e] |= __ballot(mine_c && chosen[mine_c ? slot[e] : 0] != 0);
            cand[e] = 0ull;
        }
        k = 0;
    } else if (ncand != k) {
        // Many candidates (wide ties, non-finite or extreme keys): decide the
        // order-preserving key bits one at a time from the highest bit in
        // which the candidates differ.  Per bit, a ballot per element counts
        // the candidates with a 0 there; the side holding the k-th stays
        // candidate, and when that is the 1 side the 0 side is taken.  It ends
        // once exactly k candidates remain, else after bit 0 with equal keys.
        uint32_t hi[NE], lo[NE];
        uint32_t ah = ~0u, al = ~0u, oh = 0u, ol = 0u;
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const uint64_t u = desc_bits(raw[e]);
            hi[e] = (uint32_t)(u >> 32);
            lo[e] = (uint32_t)u;
            if ((cand[e] >> lane) & 1ull) {
                ah &= hi[e];
                al &= lo[e];
                oh |= hi[e];
                ol |= lo[e];
            }
        }
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) {
            ah &= __shfl_xor(ah, s);
            al &= __shfl_xor(al, s);
            oh |= __shfl_xor(oh, s);
            ol |= __shfl_xor(ol, s);
        }
        const uint32_t dh = __builtin_amdgcn_readfirstlane(ah ^ oh);
        const uint32_t dl = __builtin_amdgcn_readfirstlane(al ^ ol);
        auto decide = [&](const uint32_t (&word)[NE], int b) __attribute__((always_inline)) {
            uint64_t zero[NE];
            int c0 = 0;
#pragma unroll
            for (int e = 0; e < NE; ++e) {
                zero[e] = __ballot(((word[e] >> b) & 1u) == 0u) & cand[e];
                c0 += __popcll(zero[e]);
            }
            if (k <= c0) {
#pragma unroll
                for (int e = 0; e < NE; ++e) cand[e] = zero[e];
                ncand = c0;
            } else {
                k -= c0;
                ncand -= c0;
#pragma unroll
                for (int e = 0; e < NE; ++e) {
                    take[e] |= zero[e];
                    cand[e] &= ~zero[e];
                }
            }
        };
        if ((dh | dl) != 0u) {
            int b = dh != 0u ? 63 - __builtin_clz(dh) : 31 - __builtin_clz(dl);
            for (; b >= 32 && ncand != k; --b) decide(hi, b - 32);
            for (; b >= 0 && ncand != k; --b) decide(lo, b);
        }
    }
    // the candidates left: all of them when exactly k remain, else (equal
    // keys) the k of lowest index
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        uint64_t c = cand[e];
        const int pc = __popcll(c);
        if (pc <= k) {
            take[e] |= c;
            k -= pc;
        } else {
            while (k > 0) {
                const uint64_t low = c & (~c + 1ull);
                take[e] |= low;
                c ^= low;
                --k;
            }
        }
    }

    // 4. ascending index order: element e before e + 1, lane order within
    int written = 0;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        const uint64_t t = take[e];
        if ((t >> lane) & 1ull) out[written + __popcll(t & below)] = 64 * e + lane;
        written += __popcll(t);
    }
}

hipError_t launch_select(const double* token_key, int n_tiles, int n_v, const int* kept,
                         const int* budgets, int n_keep, int* sel_offsets, int* sel_idx,
                         long long cap, int* status, hipStream_t st) {
    // Up to kScanFrom kept tiles every workgroup reads all budgets (one
    // launch), four tiles a workgroup up to 1,024 tiles to spread a query's
    // tiles over the CUs, eight above (16 left some CUs with twice the work
    // of others); larger calls scan the budgets once first.
    const int c = (int)(cap < 0x7fffffffLL ? cap : 0x7fffffffLL);
    auto go = [&](auto kernel, int W) {
        const unsigned wgs = (unsigned)((n_keep + W - 1) / W);
        hipLaunchKernelGGL(kernel, dim3(wgs > 0 ? wgs : 1u), dim3(64 * W), 0, st, token_key, n_tiles, n_v, n_keep,
                           kept, budgets, c, sel_offsets, sel_idx, status);
    };
    const bool small = n_keep <= 4 * 256;
    const bool scan = n_keep > kScanFrom;
    if (scan) {
        hipLaunchKernelGGL(select_scan_kernel, dim3(1), dim3(kScanThreads), 0, st, kept, budgets, n_keep, n_tiles,
                           n_v, c, sel_offsets, status);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_v <= 64 * 9) {
        if (small) go(select_kernel<9, 4, false>, 4);
        else if (!scan) go(select_kernel<9, 8, false>, 8);
        else go(select_kernel<9, 8, true>, 8);
    } else {
        if (small) go(select_kernel<16, 4, false>, 4);
        else if (!scan) go(select_kernel<16, 8, false>, 8);
        else go(select_kernel<16, 8, true>, 8);
    }
    return hipGetLastError();
}

}  // namespace rift

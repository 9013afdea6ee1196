// Stage 2 token retention of Rift (Sec. 2.3 Stage 2): each kept tile keeps its
// budget of dominant tokens, ranked by the per-token margin, ties to the lower
// token index, emitted in ascending index order.
//
// One wave per kept tile, its keys in registers (lane l, element e = token
// 64 e + l).  Up to 8,192 kept tiles, one launch; a workgroup of W waves
// handles W consecutive kept tiles:
//   1. the wave issues the loads of its tile's keys (tile id clamped so every
//      read is in bounds whatever the ids hold);
//   2. meanwhile the workgroup reads every budget and tile id of the call:
//      the call is valid only if all of them are in range and the total fits
//      (then every workgroup reaches the same verdict), and the sum of the
//      budgets before its first tile is its base offset;
//   3. each wave finds the budget-th key of its tile, (key desc, index asc):
//      one histogram pass over 256 value buckets of the keys' float32 range
//      (a monotone bucket map, so whole buckets before the budget-th key's
//      are taken), then that bucket's few candidates ranked by float64
//      comparisons with index ties; wide ties, infinities or a crowded bucket
//      fall back to deciding the order-preserving key bits one at a time with
//      wave-wide candidate masks;
//   4. the taken tokens are written in ascending index order (ballot prefix
//      counts).
// Workgroup 0 writes the status word; the workgroup of the last tile writes
// the total offset.
//
// Step 2 costs every workgroup a read of all budgets and ids, which grows with
// the square of the tile count.  Calls of more than 8,192 kept tiles therefore
// check the call and find the offsets in two small launches first
// (select_chunk_kernel, select_base_kernel), and the selection kernel
// (select_chunked_kernel, one wave a workgroup) reads its tile's offset and
// the verdict instead of step 2.
#include <climits>
#include <type_traits>

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

// Order-preserving signed integer of a float that is not NaN (-0 just below
// +0), and back: the magnitude bits of negative values are flipped.
__device__ __forceinline__ int ord_f32(float x) {
    const int b = __builtin_bit_cast(int, x);
    return b ^ ((b >> 31) & 0x7fffffff);
}
__device__ __forceinline__ float unord_f32(int i) {
    return __builtin_bit_cast(float, i ^ ((i >> 31) & 0x7fffffff));
}

// Minimum and maximum over the wave, by the same DPP steps (lanes shifted in
// from outside contribute the identity), read from lane 63.  On integers, so
// that each step is one DPP min or max.
__device__ __forceinline__ int wave_min_i32(int v) {
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x111, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x112, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x114, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x118, 0xf, 0xf, false));
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x142, 0xa, 0xf, false));
    v = min(v, __builtin_amdgcn_update_dpp(INT_MAX, v, 0x143, 0xc, 0xf, false));
    return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ int wave_max_i32(int v) {
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x111, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x112, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x114, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x118, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x142, 0xa, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(INT_MIN, v, 0x143, 0xc, 0xf, false));
    return __builtin_amdgcn_readlane(v, 63);
}

// Lane l's bit of a wave-wide mask, as the lane's execution condition.
__device__ __forceinline__ bool lane_in(uint64_t mask) { return __builtin_amdgcn_inverse_ballot_w64(mask); }

// Position of this lane among the lanes of `mask` below it, plus `base`.
__device__ __forceinline__ int rank_in(uint64_t mask, int base) {
    return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)mask, (unsigned)base));
}

// Large calls check the budgets and ids and find the offsets in two small
// launches before the selection, in chunks of kChunkN kept tiles; no launch
// waits on another workgroup and no memory beyond the offsets is needed.
//   select_chunk_kernel, one workgroup per chunk: checks the chunk's budgets
//     (in [0, n_v]) and tile ids (in [0, n_tiles)), writes the chunk-local
//     exclusive prefix sums of its budgets to its offsets, except the first
//     (always 0), whose slot receives the chunk's total instead, or -1 if an
//     entry is out of range;
//   select_base_kernel, one workgroup: reads the chunk totals, decides the
//     call (every chunk valid, total at most cap), and rewrites each chunk's
//     first slot with the chunk's global offset (0 if the call is invalid),
//     the total offset and the status word.
// The selection then finds tile rho's offset as the first slot of its chunk
// plus its local one, and rewrites the local one (a slot read by its own
// wave only; the first slots are only read).
constexpr int kChunkN = 1024;
constexpr int kChunkThreads = 256;   // four entries a thread
// Kept tiles above which the three launches beat one.
constexpr int kScanFrom = 8192;

__global__ void __launch_bounds__(kChunkThreads)
select_chunk_kernel(const int* __restrict__ kept, const int* __restrict__ budgets, int n_keep, int n_tiles,
                    int n_v, int* __restrict__ offs) {
    __shared__ unsigned wsum[kChunkThreads / 64];
    __shared__ int wbad[kChunkThreads / 64];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int c0 = blockIdx.x * kChunkN;
    const int i0 = c0 + 4 * tid;
    const bool vec = ((reinterpret_cast<uintptr_t>(budgets) | reinterpret_cast<uintptr_t>(kept) |
                       reinterpret_cast<uintptr_t>(offs)) & 15u) == 0;
    unsigned b[4], t[4];
    if (vec && i0 + 3 < n_keep) {
        const u32x4_t bv = *reinterpret_cast<const u32x4_t*>(budgets + i0);
        const u32x4_t tv = *reinterpret_cast<const u32x4_t*>(kept + i0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            b[j] = bv[j];
            t[j] = tv[j];
        }
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            b[j] = i0 + j < n_keep ? (unsigned)budgets[i0 + j] : 0u;
            t[j] = i0 + j < n_keep ? (unsigned)kept[i0 + j] : 0u;
        }
    }
    bool bad = false;
    unsigned s = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        bad = bad || b[j] > (unsigned)n_v || t[j] >= (unsigned)n_tiles;   // negative values are huge
        s += b[j];
    }
    const unsigned incl = wave_incl_scan(s);
    const bool wave_bad = __ballot(bad) != 0ull;
    if (lane == 63) wsum[wave] = incl;
    if (lane == 0) wbad[wave] = wave_bad;
    __syncthreads();
    unsigned before = 0u, total = 0u;
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < kChunkThreads / 64; ++w) {
        before += w < wave ? wsum[w] : 0u;
        total += wsum[w];
        any_bad |= wbad[w];
    }
    // valid entries keep the total within kChunkN * 1024 < 2^31
    unsigned o[4];
    unsigned run = before + incl - s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        o[j] = run;
        run += b[j];
    }
    if (tid == 0) o[0] = any_bad ? ~0u : total;
    if (vec && i0 + 3 < n_keep) {
        *reinterpret_cast<u32x4_t*>(offs + i0) = u32x4_t{o[0], o[1], o[2], o[3]};
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (i0 + j < n_keep) offs[i0 + j] = (int)o[j];
    }
}

__global__ void __launch_bounds__(1024)
select_base_kernel(int n_keep, int cap, int* __restrict__ offs, int* __restrict__ status) {
    __shared__ unsigned wsum[16];
    __shared__ int wbad[16];
    const unsigned tid = threadIdx.x;
    const unsigned lane = tid & 63u;
    const unsigned wave = tid >> 6;
    const unsigned n_chunks = ((unsigned)n_keep + kChunkN - 1) / kChunkN;
    unsigned carry = 0u;   // totals of the earlier chunks (no wrap-around while they are valid)
    bool bad = false;
    for (unsigned c = 0; c < n_chunks; c += 1024u) {
        const unsigned k = c + tid;
        const int tot = k < n_chunks ? offs[(size_t)k * kChunkN] : 0;
        bad = bad || tot < 0;
        const unsigned s = tot < 0 ? 0u : (unsigned)tot;
        const unsigned incl = wave_incl_scan(s);
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        unsigned before = 0u, blk = 0u;
#pragma unroll
        for (int w = 0; w < 16; ++w) {
            const unsigned x = wsum[w];
            before += (unsigned)w < wave ? x : 0u;
            blk += x;
        }
        if (k < n_chunks) offs[(size_t)k * kChunkN] = (int)(carry + before + incl - s);
        carry += blk;
        __syncthreads();   // wsum is refilled by the next block
    }
    const bool wave_bad = __ballot(bad) != 0ull;
    if (lane == 0) wbad[wave] = wave_bad;
    __syncthreads();
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) any_bad |= wbad[w];
    // valid budgets keep the total within n_tiles * n_v <= INT32_MAX
    const bool valid = any_bad == 0 && carry <= (unsigned)cap;
    if (!valid) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the bases stored, before any is cleared
        for (unsigned k = tid; k < n_chunks; k += 1024u) offs[(size_t)k * kChunkN] = 0;
    }
    if (tid == 0) {
        offs[n_keep] = valid ? (int)carry : 0;
        *status = valid ? 0 : (int)RIFT_ERR_BUDGET;
    }
}

// Steps 3 and 4 for one tile: its keys raw (lane l, element e = token 64 e + l;
// past the tile's end copies of its last key), its budget (in [0, n_v]), where
// its selection goes, and the wave's 256-word slice of shared memory.
template <int NE, bool FULL>
__device__ __forceinline__ void select_tile(const double (&raw)[NE], int n_v, int budget, int* __restrict__ out,
                                            unsigned* hist, int lane) {
    if (budget <= 0) return;
    if (budget >= n_v) {
        for (int i = lane; i < n_v; i += 64) out[i] = i;
        return;
    }

    // 3. which tokens to take.  First, when the keys are finite as float32
    // and not all equal, one histogram pass over 256 value buckets of their
    // float32 range: bucket = trunc(clamp(fl(hi s - f s), 0, 255)) with f the
    // key rounded to float32, hi the largest such value, s = 256 / range
    // (approximately) and fl(hi s - f s) one fused multiply-add.  Each step
    // (the rounding to float32, the once-rounded decreasing affine map, the
    // clamp, the truncation) is monotone, so every key of a lower bucket is
    // strictly larger than every key of a higher one, whatever s and hi s
    // come to.  The buckets before the one that holds the budget-th key are
    // taken whole; that bucket's keys, usually a handful, are the candidates
    // for the rest.
    uint64_t cand[NE], take[NE];
    int k = budget;
    int ncand = n_v;
    float fmn = INFINITY, fmx = -INFINITY, fsum = 0.0f;
    float f[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        const int base = 64 * e;
        cand[e] = FULL || base + 64 <= n_v ? ~0ull : (base >= n_v ? 0ull : ((1ull << (n_v - base)) - 1ull));
        take[e] = 0ull;
        f[e] = (float)raw[e];
        // copies of the last key past the tile's end change none of these
        fsum += f[e];   // NaN once a key is NaN or infinite as float32
        fmn = fminf(fmn, f[e]);
        fmx = fmaxf(fmx, f[e]);
    }
    // (finiteness by class tests: x - x == 0 on a product may be contracted
    // into the product's rounding error)
    const bool all_finite = __ballot(!__builtin_isfinite(fsum)) == 0ull;
    const float hi = unord_f32(wave_max_i32(ord_f32(fmx)));
    const float range = hi - unord_f32(wave_min_i32(ord_f32(fmn)));
    const float scale = 256.0f * __builtin_amdgcn_rcpf(range);
    const float his = hi * scale;
    if (all_finite && range > 0.0f && scale > 0.0f && __builtin_isfinite(scale) && __builtin_isfinite(his)) {
        int bkt[NE];
        // A wave's shared-memory operations execute in the order issued, so
        // the clearing, the increments and the read-back need no waits in
        // between, only to stay in this order (compiler barriers).
        *reinterpret_cast<u32x4_t*>(hist + 4 * lane) = u32x4_t{0u, 0u, 0u, 0u};
        asm volatile("" ::: "memory");
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            bkt[e] = (int)__builtin_amdgcn_fmed3f(__builtin_fmaf(f[e], -scale, his), 0.0f, 255.0f);
            if (FULL || 64 * e + lane < n_v) atomicAdd(&hist[bkt[e]], 1u);
        }
        asm volatile("" ::: "memory");
        const u32x4_t c = *reinterpret_cast<const u32x4_t*>(hist + 4 * lane);
        const unsigned mine = c[0] + c[1] + c[2] + c[3];
        const unsigned incl = wave_incl_scan(mine);   // keys in buckets < 4 lane + 4
        // the budget-th key lies in the buckets of the first lane whose
        // running count reaches it (1 <= k < n_v); then, on the scalar unit,
        // in the first of that lane's four buckets that reaches it
        const int src = __builtin_ctzll(__ballot(incl >= (unsigned)k));
        unsigned before = (unsigned)__builtin_amdgcn_readlane((int)(incl - mine), src);
        unsigned cs[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) cs[j] = (unsigned)__builtin_amdgcn_readlane((int)c[j], src);
        int B = 4 * src + 3;
#pragma unroll
        for (int j = 2; j >= 0; --j) {
            unsigned upto = before;
#pragma unroll
            for (int i = 0; i <= j; ++i) upto += cs[i];
            if (upto >= (unsigned)k) B = 4 * src + j;
        }
        const int j_hit = B - 4 * src;
#pragma unroll
        for (int i = 0; i < 3; ++i) before += i < j_hit ? cs[i] : 0u;
        k -= (int)before;
        ncand = (int)(j_hit == 0 ? cs[0] : j_hit == 1 ? cs[1] : j_hit == 2 ? cs[2] : cs[3]);
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            take[e] = __ballot(bkt[e] < B) & cand[e];
            cand[e] = __ballot(bkt[e] == B) & cand[e];
        }
    }
    if (ncand != k && ncand <= 64 && all_finite) {
        // Rank each candidate among the candidates by (key desc, index asc)
        // with plain float64 comparisons (-0 and +0 compare equal); take the
        // first k.  The candidates move to lanes 0 .. ncand - 1 through the
        // histogram's slice of shared memory, each lane counts the candidates
        // ahead of its own from register reads of the others, and the chosen
        // slots come back as a wave-wide mask.
        double* cx = reinterpret_cast<double*>(hist);
        int* ci = reinterpret_cast<int*>(hist + 128);
        int slot0[NE];
        int n0 = 0;
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            slot0[e] = n0;
            if (cand[e] != 0ull) {   // uniform: elements without candidates cost nothing
                if (lane_in(cand[e])) {
                    const int slot = rank_in(cand[e], n0);
                    cx[slot] = raw[e];
                    ci[slot] = 64 * e + lane;
                }
                n0 += __popcll(cand[e]);
            }
        }
        asm volatile("" ::: "memory");   // in-order shared memory, as above
        const bool has = lane < ncand;
        const double mx = has ? cx[lane] : 0.0;
        const int mi = has ? ci[lane] : 0;
        const int mhi = __double2hiint(mx), mlo = __double2loint(mx);
        int r = 0;
        for (int j = 0; j < ncand; ++j) {
            const double xj = __hiloint2double(__builtin_amdgcn_readlane(mhi, j), __builtin_amdgcn_readlane(mlo, j));
            const int ij = __builtin_amdgcn_readlane(mi, j);
            r += (xj > mx || (xj == mx && ij < mi)) ? 1 : 0;
        }
        const uint64_t chosen = __ballot(has && r < k);
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            if (cand[e] != 0ull) {
                bool ch = false;
                if (lane_in(cand[e])) ch = ((chosen >> rank_in(cand[e], slot0[e])) & 1ull) != 0ull;
                take[e] |= __ballot(ch);
                cand[e] = 0ull;
            }
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
        if (lane_in(t)) out[rank_in(t, written)] = 64 * e + lane;
        written += __popcll(t);
    }
}

// Loads of a tile's keys into raw (tile id clamped: every read is in bounds
// whatever the ids hold).
template <int NE, bool FULL>
__device__ __forceinline__ void load_keys(double (&raw)[NE], const double* __restrict__ token_key, int tile,
                                          int n_tiles, int n_v, int lane) {
    tile = tile < 0 ? 0 : (tile >= n_tiles ? n_tiles - 1 : tile);
    const char* kb = reinterpret_cast<const char*>(token_key + (size_t)tile * n_v);
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        // past the tile's end a lane reads a copy of its last key
        const unsigned i = FULL ? (unsigned)(64 * e + lane) : min((unsigned)(64 * e + lane), (unsigned)(n_v - 1));
        raw[e] = *reinterpret_cast<const double*>(kb + i * 8u);
    }
}

// One-launch path.  NE: keys per lane the kernel is built for (n_v <= 64 NE);
// W: waves (kept tiles) per workgroup; FULL: n_v == 64 NE (no lane holds a key
// past the tile's end).
template <int NE, int W, bool FULL>
__global__ void __launch_bounds__(64 * W, NE <= 9 && FULL ? 8 : 1)   // 8 waves a SIMD where no spills
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
    //    allow it); this wave's keys; the budgets of this workgroup's tiles up
    //    to this wave's (uniform, through the scalar cache)
    const int tile = has_tile ? kept[rho] : 0;
    const bool vec = ((reinterpret_cast<uintptr_t>(budgets) | reinterpret_cast<uintptr_t>(kept)) & 15u) == 0;
    constexpr int kV = 4;                       // 16-byte vectors per thread per round
    constexpr int kRound = kV * 64 * W;         // vectors per round
    const int n4 = vec ? n_keep >> 2 : 0;   // whole vectors; the rest one by one
    i32x4_t bv[kV], tv[kV];
    if (n4 > 0) {
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            const int v = min(tid + j * 64 * W, n4 - 1);
            bv[j] = reinterpret_cast<const i32x4_t*>(budgets)[v];
            tv[j] = reinterpret_cast<const i32x4_t*>(kept)[v];
        }
    }
    double raw[NE];
    load_keys<NE, FULL>(raw, token_key, tile, n_tiles, n_v, lane);
    int off = 0, budget = 0;
    {
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
    select_tile<NE, FULL>(raw, n_v, budget, sel_idx + off, hist_all[wave], lane);
}

// Chunked path, after select_chunk_kernel and select_base_kernel: one wave
// per kept tile.  A tile's offset is its chunk's global offset plus its local
// one, which the wave replaces (0 if the call is invalid).
template <int NE, int W, bool FULL>
__global__ void __launch_bounds__(64 * W, NE <= 9 ? 8 : 1)   // 8 waves a SIMD (latency-bound)
select_chunked_kernel(const double* __restrict__ token_key, int n_tiles, int n_v, int n_keep,
                      const int* __restrict__ kept, const int* __restrict__ budgets,
                      int* __restrict__ offs, int* __restrict__ sel_idx, const int* __restrict__ status) {
    __shared__ __align__(16) unsigned hist_all[W][256];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int rho = blockIdx.x * W + wave;
    if (rho >= n_keep) return;
    double raw[NE];
    load_keys<NE, FULL>(raw, token_key, kept[rho], n_tiles, n_v, lane);
    const int c0 = rho & ~(kChunkN - 1);
    const int verdict = __builtin_amdgcn_readfirstlane(*status);
    int off = __builtin_amdgcn_readfirstlane(offs[c0]);
    if (rho != c0) {
        off += __builtin_amdgcn_readfirstlane(offs[rho]);
        if (lane == 0) offs[rho] = verdict != 0 ? 0 : off;
    }
    if (verdict != 0) return;
    select_tile<NE, FULL>(raw, n_v, __builtin_amdgcn_readfirstlane(budgets[rho]), sel_idx + off, hist_all[wave],
                          lane);
}

hipError_t launch_select(const double* token_key, int n_tiles, int n_v, const int* kept,
                         const int* budgets, int n_keep, int* sel_offsets, int* sel_idx,
                         long long cap, int* status, hipStream_t st) {
    // Up to kScanFrom kept tiles every workgroup reads all budgets (one
    // launch), four tiles a workgroup up to 1,024 tiles to spread a query's
    // tiles over the CUs, eight above (16 left some CUs with twice the work
    // of others); larger calls find the offsets in two launches first.
    const int c = (int)(cap < 0x7fffffffLL ? cap : 0x7fffffffLL);
    auto go = [&](auto kernel, int W) {
        const unsigned wgs = (unsigned)((n_keep + W - 1) / W);
        hipLaunchKernelGGL(kernel, dim3(wgs > 0 ? wgs : 1u), dim3(64 * W), 0, st, token_key, n_tiles, n_v, n_keep,
                           kept, budgets, c, sel_offsets, sel_idx, status);
    };
    auto go_chunked = [&](auto kernel) {
        constexpr int W = 1;   // a wave's slot is free as soon as its tile is done
        hipLaunchKernelGGL(kernel, dim3((unsigned)((n_keep + W - 1) / W)), dim3(64 * W), 0, st, token_key, n_tiles,
                           n_v, n_keep, kept, budgets, sel_offsets, sel_idx, (const int*)status);
    };
    const bool small = n_keep <= 4 * 256;
    const bool scan = n_keep > kScanFrom;
    if (scan) {
        const unsigned n_chunks = (unsigned)((n_keep + kChunkN - 1) / kChunkN);
        hipLaunchKernelGGL(select_chunk_kernel, dim3(n_chunks), dim3(kChunkThreads), 0, st, kept, budgets, n_keep,
                           n_tiles, n_v, sel_offsets);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(select_base_kernel, dim3(1), dim3(1024), 0, st, n_keep, c, sel_offsets, status);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    auto pick = [&](auto full) {
        constexpr bool F = decltype(full)::value;
        if (n_v <= 64 * 9) {
            if (scan) go_chunked(select_chunked_kernel<9, 1, F>);
            else if (small) go(select_kernel<9, 4, F>, 4);
            else go(select_kernel<9, 8, F>, 8);
        } else {
            if (scan) go_chunked(select_chunked_kernel<16, 1, F>);
            else if (small) go(select_kernel<16, 4, F>, 4);
            else go(select_kernel<16, 8, F>, 8);
        }
    };
    if (n_v == 64 * 9 || n_v == 64 * 16) pick(std::true_type{});
    else pick(std::false_type{});
    return hipGetLastError();
}

}  // namespace rift

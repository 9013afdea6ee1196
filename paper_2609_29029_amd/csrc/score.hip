// Stage 1 of Rift (Sec. 2.3, Eq. 1; Listing 1; App. B Step 3) on gfx950.
//
//   prep_w       w = t - (1/M) sum_j B_j in float64, rounded to float32; also
//                clears the per-tile arrival counters of score_tiles.
//   score_tiles  one wave per 32 tokens of a tile (token sets of all tiles
//                dealt out four to a workgroup, so the work spreads evenly over
//                the CUs whatever the tile count).  bf16 rows are read 512
//                contiguous bytes at a time into a per-wave LDS buffer, the next
//                chunk in flight while the current one is computed.  One pass
//                over the tokens computes, per token,
//                  * the float64 ranking key r = (x.w)/|x| on the VALUs, in the
//                    fixed granule order (8-wide granules, granule g into
//                    accumulator g mod 4, then (a0+a2)+(a1+a3));
//                  * the cosines to t and every B_j with bf16 (or f32) MFMA,
//                    the query-versus-token relevance GEMM.
//                Then, in the same launch: the workgroup that completes a tile
//                (a per-tile arrival counter) pools it, s_i = mean r (64
//                strided partial sums in token order, halving tree, divide by
//                n_v); and the workgroup that completes the last tile ranks
//                the scene: order by (s desc, id asc), min-max normalisation
//                u, retention by top-K or u >= tau.  With smoothing the
//                ranking waits for the smoothed scores and runs on its own
//                (rank_tiles).
//
// Register layout of a wave in score_tiles: lane l = r + 16 q (r = l & 15,
// q = l >> 4).  For token block b (16 tokens) and k-step s (32 elements), lane l
// holds elements [32 s + 8 q, 32 s + 8 q + 8) of token 16 b + r.  That is the
// B-operand layout of v_mfma_f32_16x16x32_bf16 (column r, k-slots 8q..8q+7), so
// the same registers feed the MFMA (A operand = the query bank rows) and the
// float64 accumulators of granule 4 s + q.
#include "launch.h"
#include "rift_common.h"

namespace rift {

__global__ void prep_w_kernel(const void* __restrict__ qbank, int is_bf16, int d, int n_bg,
                              float* __restrict__ w32, int* __restrict__ counters, int n_counters) {
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_counters) counters[i] = 0;
    if (i >= d) return;
    auto at = [&](int row) -> double {
        if (is_bf16) return (double)bf16_to_f32(static_cast<const bf16_t*>(qbank)[(size_t)row * d + i]);
        return (double)static_cast<const float*>(qbank)[(size_t)row * d + i];
    };
    double t = at(0);
    double w = t;
    if (n_bg > 0) {
        double acc = 0.0;
        for (int j = 1; j <= n_bg; ++j) acc = acc + at(j);
        w = t - acc / (double)n_bg;
    }
    w32[i] = (float)w;
}

// a precedes b: larger score first, then lower tile id.
__device__ __forceinline__ bool precedes(double ka, int ia, double kb, int ib) {
    return (ka > kb) || (ka == kb && ia < ib);
}

// Rank the scene's tile scores s[0, n) with the threads of one workgroup
// (blockDim.x threads, a multiple of 64): order by (s desc, id asc), u =
// (s - min)/(max - min) in float64 (1 when max == min), n_keep = top-K or the
// count of u >= tau.  A NaN score (only from a non-finite input) ranks as
// -inf.  Up to 1024 tiles: each tile's position is the number of tiles that
// precede it; more: a bitonic sort.  lds: rank_lds_bytes(n) bytes, 16-byte
// aligned.  With s_copy, s is also copied there.
__device__ void rank_scene(const double* s, int n, int keep_count, double tau, float* __restrict__ u_out,
                           int* __restrict__ order, int* __restrict__ n_keep, double* __restrict__ s_copy,
                           unsigned char* lds) {
    int N = 1;
    while (N < n) N <<= 1;
    double* ext = reinterpret_cast<double*>(lds);          // max, min
    int& kept = *reinterpret_cast<int*>(lds + 16);
    double* key = reinterpret_cast<double*>(lds + 32);
    int* id = reinterpret_cast<int*>(lds + 32 + (size_t)8 * N);
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    for (int i = tid; i < N; i += nt) {
        // agent-coherent load: in the fused pass other workgroups wrote s
        const double si = i < n ? __hip_atomic_load(s + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : -INFINITY;
        key[i] = (si == si) ? si : -INFINITY;
        id[i] = i;
        if (s_copy != nullptr && i < n) s_copy[i] = si;
    }
    if (tid == 0) kept = 0;
    __syncthreads();
    int local = 0;
    if (n <= 1024) {
        int pos[4];   // positions of this thread's tiles i = tid + nt j
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = tid + nt * j;
            pos[j] = 0;
            if (i < n) {
                const double ki = key[i];
                int r = 0;
                for (int m = 0; m < n; ++m) r += precedes(key[m], m, ki, i) ? 1 : 0;
                pos[j] = r;
                if (r == 0) ext[0] = ki;
                if (r == n - 1) ext[1] = ki;
            }
        }
        __syncthreads();
        const double smax = ext[0], smin = ext[1], range = smax - smin;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = tid + nt * j;
            if (i < n) {
                const double u = (smax == smin) ? 1.0 : (key[i] - smin) / range;
                order[pos[j]] = i;
                u_out[i] = (float)u;
                local += (u >= tau) ? 1 : 0;
            }
        }
    } else {
        for (int size = 2; size <= N; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int t = tid; t < (N >> 1); t += nt) {
                    const int i = 2 * t - (t & (stride - 1));
                    const int j = i + stride;
                    const bool up = (i & size) == 0;
                    const bool sw = up ? precedes(key[j], id[j], key[i], id[i])
                                       : precedes(key[i], id[i], key[j], id[j]);
                    if (sw) {
                        const double tk = key[i];
                        key[i] = key[j];
                        key[j] = tk;
                        const int ti = id[i];
                        id[i] = id[j];
                        id[j] = ti;
                    }
                }
                __syncthreads();
            }
        }
        // the pads sort last: the first n entries are the tiles
        const double smax = key[0], smin = key[n - 1], range = smax - smin;
        for (int p = tid; p < n; p += nt) {
            const double u = (smax == smin) ? 1.0 : (key[p] - smin) / range;
            order[p] = id[p];
            u_out[id[p]] = (float)u;
            local += (u >= tau) ? 1 : 0;
        }
    }
    if (keep_count == 0 && local) atomicAdd(&kept, local);
    __syncthreads();
    if (tid == 0) *n_keep = keep_count > 0 ? (keep_count < n ? keep_count : n) : kept;
}

constexpr int kScoreWaves = 4;          // waves per workgroup
constexpr int kScoreTok = 32;           // tokens per wave: two 16-token MFMA column blocks
constexpr int kChunkSteps = 8;          // k-steps (32 elements each) per staged chunk: 512 bytes of a bf16 row
constexpr int kStageBytes = kScoreTok * kChunkSteps * 64;   // one wave's LDS staging buffer (16 KB)

template <bool kBf16>
__global__ void __launch_bounds__(64 * kScoreWaves)
score_tiles_kernel(const void* __restrict__ tokens, int n_tiles, int n_v, int d,
                   const void* __restrict__ qbank, int nq, const float* __restrict__ w32,
                   double* __restrict__ token_key, float* __restrict__ token_sim,
                   double* __restrict__ inv_out, int* __restrict__ arrivals, double* __restrict__ tile_score,
                   int rank, int keep_count, double tau, float* __restrict__ tile_u,
                   int* __restrict__ tile_order, int* __restrict__ n_keep, int ctl_off) {
    extern __shared__ __align__(16) unsigned char smem[];
    float* w_lds = reinterpret_cast<float*>(smem);

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int q = lane >> 4;

    for (int i = threadIdx.x; i < d; i += blockDim.x) w_lds[i] = w32[i];
    __syncthreads();

    const int n_sets = (n_v + kScoreTok - 1) / kScoreTok;
    const long long total_sets = (long long)n_tiles * n_sets;
    const long long gw0 = (long long)blockIdx.x * kScoreWaves;          // the workgroup's first token set
    const long long gw_raw = gw0 + wave;                                 // this wave's token set of all tiles
    const bool active = gw_raw < total_sets;
    const long long gw = active ? gw_raw : total_sets - 1;              // idle waves redo the last set, unstored
    const int tile = (int)(gw / n_sets);
    const int t0 = (int)(gw % n_sets) * kScoreTok;
    const size_t tile_row0 = (size_t)tile * n_v;
    const size_t q_off = (size_t)(r < nq ? r : nq - 1) * d;
    const int steps = d / 32;

    double n2[2] = {0.0, 0.0};
    double g[2] = {0.0, 0.0};
    f32x4_t acc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};

    if constexpr (kBf16) {
        // The wave's 32 token rows are read 512 bytes at a time: load i covers
        // rows 2i and 2i + 1 (lanes 0-31 and 32-63), 16 bytes a lane, so each
        // request is two contiguous 512-byte pieces.  The pieces go through a
        // 16 KB LDS buffer (row lt at lt * 512, 16-byte unit j stored at unit
        // j ^ (lt & 15)) and are read back in the MFMA B layout: for k-step s,
        // lane (r, q) takes unit 4 s + q of row 16 b + r, which the swizzle
        // spreads over distinct banks.  The next chunk's loads are in flight
        // while the current one is computed.
        const unsigned char* Xt = static_cast<const unsigned char*>(tokens) + tile_row0 * (size_t)d * 2;
        const bf16_t* Q = static_cast<const bf16_t*>(qbank);
        unsigned char* stage = smem + (size_t)d * sizeof(float) + (size_t)wave * kStageBytes;
        const unsigned row_bytes = (unsigned)d * 2;
        const int unit = lane & 31;
        unsigned src_row[16];   // byte offset of each loaded row in the tile (n_v * 2 d < 2^31)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int lt = 2 * i + (lane >> 5);
            src_row[i] = (unsigned)(t0 + lt < n_v ? t0 + lt : n_v - 1) * row_bytes;
        }
        const int n_chunks = (steps + kChunkSteps - 1) / kChunkSteps;
        u32x4_t P[16], Qc[kChunkSteps];
        // Issued after the query loads of the chunk being computed, so the
        // waits on those (the counter drains in order) leave these in flight.
        // Nontemporal: each token row is read exactly once.
        auto issue = [&](int c) __attribute__((always_inline)) {
            unsigned off = (unsigned)c * 512 + (unsigned)unit * 16;
            off = off < row_bytes - 16 ? off : row_bytes - 16;   // past the row end in a partial last chunk
#pragma unroll
            for (int i = 0; i < 16; ++i) P[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(Xt + src_row[i] + off));
        };
        auto load_q = [&](int c) __attribute__((always_inline)) {
#pragma unroll
            for (int s = 0; s < kChunkSteps; ++s) {
                int st = c * kChunkSteps + s;
                st = st < steps ? st : steps - 1;
                Qc[s] = *reinterpret_cast<const u32x4_t*>(Q + q_off + st * 32 + q * 8);
            }
        };
        auto stage_write = [&]() __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int lt = 2 * i + (lane >> 5);
                *reinterpret_cast<u32x4_t*>(stage + lt * 512 + ((unit ^ (lt & 15)) << 4)) = P[i];
            }
            __builtin_amdgcn_wave_barrier();
        };
        auto step = [&](int st, int s) __attribute__((always_inline)) {   // global k-step st, slot s of the chunk
            const int k = st * 32 + q * 8;
            const f32x4_t w0 = *reinterpret_cast<const f32x4_t*>(w_lds + k);
            const f32x4_t w1 = *reinterpret_cast<const f32x4_t*>(w_lds + k + 4);
            const double wd[8] = {(double)w0[0], (double)w0[1], (double)w0[2], (double)w0[3],
                                  (double)w1[0], (double)w1[1], (double)w1[2], (double)w1[3]};
            const bf16x8_t qa = __builtin_bit_cast(bf16x8_t, Qc[s]);
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const u32x4_t x =
                    *reinterpret_cast<const u32x4_t*>(stage + (16 * b + r) * 512 + (((4 * s + q) ^ r) << 4));
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double x0 = (double)bf16_lo(x[e]);
                    const double x1 = (double)bf16_hi(x[e]);
                    n2[b] = fma(x0, x0, n2[b]);
                    g[b] = fma(x0, wd[2 * e], g[b]);
                    n2[b] = fma(x1, x1, n2[b]);
                    g[b] = fma(x1, wd[2 * e + 1], g[b]);
                }
                acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, __builtin_bit_cast(bf16x8_t, x), acc[b], 0, 0, 0);
            }
        };
        auto full_chunk = [&](int c) __attribute__((always_inline)) {
#pragma unroll
            for (int s = 0; s < kChunkSteps; ++s) step(c * kChunkSteps + s, s);
            __builtin_amdgcn_wave_barrier();   // reads done before the buffer is refilled
        };
        issue(0);
        for (int c = 0; c + 1 < n_chunks; ++c) {
            stage_write();
            load_q(c);
            issue(c + 1);
            full_chunk(c);
        }
        stage_write();
        load_q(n_chunks - 1);
        const int last = n_chunks - 1;
        const int tail = steps - last * kChunkSteps;
        if (tail == kChunkSteps) {
            full_chunk(last);
        } else {
            for (int s = 0; s < tail; ++s) step(last * kChunkSteps + s, s);
        }
    } else {
        const float* X = static_cast<const float*>(tokens);
        const float* Q = static_cast<const float*>(qbank);
        size_t row_off[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int t = t0 + 16 * b + r < n_v ? t0 + 16 * b + r : n_v - 1;
            row_off[b] = (tile_row0 + t) * (size_t)d;
        }
        for (int s = 0; s < steps; ++s) {
            const int k = s * 32 + q * 8;
            const f32x4_t w0 = *reinterpret_cast<const f32x4_t*>(w_lds + k);
            const f32x4_t w1 = *reinterpret_cast<const f32x4_t*>(w_lds + k + 4);
            const float wv[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
            const f32x4_t qa0 = *reinterpret_cast<const f32x4_t*>(Q + q_off + k);
            const f32x4_t qa1 = *reinterpret_cast<const f32x4_t*>(Q + q_off + k + 4);
            const float qa[8] = {qa0[0], qa0[1], qa0[2], qa0[3], qa1[0], qa1[1], qa1[2], qa1[3]};
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const f32x4_t x0 = *reinterpret_cast<const f32x4_t*>(X + row_off[b] + k);
                const f32x4_t x1 = *reinterpret_cast<const f32x4_t*>(X + row_off[b] + k + 4);
                const float xv[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double xd = (double)xv[e];
                    n2[b] = fma(xd, xd, n2[b]);
                    g[b] = fma(xd, (double)wv[e], g[b]);
                    acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[e], xv[e], acc[b], 0, 0, 0);
                }
            }
        }
    }

    // Fold the four granule accumulators of each token: lanes r, r+16, r+32,
    // r+48 hold a0..a3.  xor 32 pairs a0 with a2 and a1 with a3; xor 16 then
    // adds the two pair sums.  Every lane of the token ends with the same value.
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int tok = t0 + 16 * b + r;
        double nn = n2[b] + __shfl_xor(n2[b], 32);
        nn = nn + __shfl_xor(nn, 16);
        double gg = g[b] + __shfl_xor(g[b], 32);
        gg = gg + __shfl_xor(gg, 16);
        double key = (nn == 0.0) ? 0.0 : gg / sqrt(nn);
        key = key + 0.0;  // -0 -> +0
        const bool valid = active && tok < n_v;
        if (valid && q == 0) {
            // agent-coherent store: the workgroup that completes the tile reads it
            __hip_atomic_store(&token_key[tile_row0 + tok], key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (inv_out != nullptr) inv_out[tile_row0 + tok] = (nn == 0.0) ? 0.0 : 1.0 / sqrt(nn);
        }
        if (token_sim != nullptr && valid) {
            const float inv = (nn > 0.0) ? (float)(1.0 / sqrt(nn)) : 0.0f;
            float* dst = token_sim + (tile_row0 + tok) * (size_t)nq;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                if (m < nq) dst[m] = acc[b][v] * inv;
            }
        }
    }

    // Arrival: the workgroup's token sets cover tiles first_tile..last_tile
    // (n_sets of them make a tile).  The workgroup that brings a tile's count
    // to n_sets pools it: lane l sums keys l, l + 64, ... in token order, then
    // the halving tree, over n_v.  The keys (and the pooled scores the
    // ranking reads) cross workgroups, possibly on other XCDs, whose L2
    // caches are not kept coherent: they are written and read with
    // agent-coherent atomic stores and loads, every wave waits for its stores
    // to complete before the counter update, and the counters are atomic.  So
    // no fence has to write back or invalidate an L2.
    // control words at the end of the dynamic shared memory, free by now and
    // clear of the ranking's region (static shared memory here would push a
    // workgroup past half of the CU's LDS and halve the occupancy)
    int* pool_tile = reinterpret_cast<int*>(smem + ctl_off);   // [kScoreWaves]
    int& n_pool = pool_tile[kScoreWaves];
    int& rank_here = pool_tile[kScoreWaves + 1];
    const long long gw_last = (gw0 + kScoreWaves - 1 < total_sets ? gw0 + kScoreWaves - 1 : total_sets - 1);
    const int first_tile = (int)(gw0 / n_sets);
    const int last_tile = (int)(gw_last / n_sets);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        int np = 0;
        for (int t = first_tile; t <= last_tile; ++t) {
            const long long a = (long long)t * n_sets > gw0 ? (long long)t * n_sets : gw0;
            const long long b = (long long)(t + 1) * n_sets - 1 < gw_last ? (long long)(t + 1) * n_sets - 1 : gw_last;
            const int mine = (int)(b - a + 1);
            if (atomicAdd(&arrivals[t], mine) + mine == n_sets) pool_tile[np++] = t;
        }
        n_pool = np;
        rank_here = 0;
    }
    __syncthreads();
    const int np = n_pool;
    if (np == 0) return;
    if (wave < np) {
        const int t = pool_tile[wave];
        const double* kt = token_key + (size_t)t * n_v;
        double p = 0.0;
        for (int i = lane; i < n_v; i += 64) p = p + __hip_atomic_load(kt + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const double o = __shfl_down(p, sft);
            p = p + o;
        }
        if (lane == 0) __hip_atomic_store(&tile_score[t], p / (double)n_v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!rank) return;
    // The workgroup that pools the scene's last tile ranks it.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        if (atomicAdd(&arrivals[n_tiles], np) + np == n_tiles) rank_here = 1;
    }
    __syncthreads();
    if (!rank_here) return;
    rank_scene(tile_score, n_tiles, keep_count, tau, tile_u, tile_order, n_keep, nullptr, smem);
}

// Ranking on its own, after the optional smoothing (one workgroup).
__global__ void __launch_bounds__(1024)
rank_tiles_kernel(const double* __restrict__ s, int n, int keep_count, double tau,
                  float* __restrict__ u_out, int* __restrict__ order, int* __restrict__ n_keep,
                  double* __restrict__ s_copy) {
    extern __shared__ __align__(16) unsigned char rank_lds[];
    rank_scene(s, n, keep_count, tau, u_out, order, n_keep, s_copy, rank_lds);
}

// LDS of the ranking: max, min and the kept count, then keys and ids of
// pow2ceil(n_tiles) entries.
size_t rank_lds_bytes(int n_tiles) {
    size_t N = 1;
    while ((int)N < n_tiles) N <<= 1;
    return 32 + 12 * N;
}

hipError_t launch_score(const void* tokens, bool bf16, int n_tiles, int n_v, int d,
                        const void* qbank, int n_bg, int keep_count, double tau, int knn_m,
                        double* token_key, float* token_sim, double* tile_score, float* tile_u,
                        int* tile_order, int* n_keep, float* w32, int* arrivals, double* inv, float* emb,
                        double* gram, double* s_smooth, hipStream_t st) {
    const int n_clear = n_tiles + 1;
    const int prep_threads = d > n_clear ? d : n_clear;
    hipLaunchKernelGGL(prep_w_kernel, dim3((prep_threads + 255) / 256), dim3(256), 0, st, qbank, bf16 ? 1 : 0,
                       d, n_bg, w32, arrivals, n_clear);
    const long long sets = (long long)n_tiles * ((n_v + kScoreTok - 1) / kScoreTok);
    const unsigned wgs = (unsigned)((sets + kScoreWaves - 1) / kScoreWaves);
    // w and the staging buffers; at the end the ranking's region and, in the
    // last 64 bytes, the control words (80 KB at d = 4096: two workgroups a CU)
    size_t lds = (size_t)d * sizeof(float) + (bf16 ? (size_t)kScoreWaves * kStageBytes : 0);
    const size_t rl = rank_lds_bytes(n_tiles) + 64;
    if (lds < rl) lds = rl;
    const int ctl_off = (int)(lds - 64);
    double* inv_out = knn_m > 0 ? inv : nullptr;
    const int rank = knn_m > 0 ? 0 : 1;   // with smoothing the ranking waits for the smoothed scores
    if (bf16) {
        hipLaunchKernelGGL(score_tiles_kernel<true>, dim3(wgs), dim3(64 * kScoreWaves), lds, st,
                           tokens, n_tiles, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, inv_out, arrivals,
                           tile_score, rank, keep_count, tau, tile_u, tile_order, n_keep, ctl_off);
    } else {
        hipLaunchKernelGGL(score_tiles_kernel<false>, dim3(wgs), dim3(64 * kScoreWaves), lds, st,
                           tokens, n_tiles, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, inv_out, arrivals,
                           tile_score, rank, keep_count, tau, tile_u, tile_order, n_keep, ctl_off);
    }
    if (knn_m > 0) {
        const hipError_t e = launch_knn_smooth(tokens, bf16, n_tiles, n_v, d, inv, emb, gram, tile_score,
                                               knn_m, s_smooth, st);
        if (e != hipSuccess) return e;
        // the output tile score is the one the ranking used
        hipLaunchKernelGGL(rank_tiles_kernel, dim3(1), dim3(1024), rank_lds_bytes(n_tiles), st, s_smooth, n_tiles,
                           keep_count, tau, tile_u, tile_order, n_keep, tile_score);
    }
    return hipGetLastError();
}

}  // namespace rift

namespace rift {
hipError_t score_init_attributes() {
    const int bytes = 16384 * (int)sizeof(float) + kScoreWaves * kStageBytes;   // >= rank_lds_bytes(4096) + 64
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<true>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<false>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}
}  // namespace rift

// Stage 1 of Rift (Sec. 2.3, Eq. 1; Listing 1; App. B Step 3) on gfx950.
//
//   prep_w       w = t - (1/M) sum_j B_j in float64, rounded to float32.
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
//   tile_pool    one wave per tile: s_i = mean r (64 strided partial sums in
//                token order, halving tree, divide by n_v).
//   rank_tiles   one workgroup: bitonic sort of (s desc, id asc), min-max
//                normalisation u, retention by top-K or u >= tau.
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
                              float* __restrict__ w32) {
    int i = blockIdx.x * blockDim.x + threadIdx.x;
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

constexpr int kScoreWaves = 4;          // waves per workgroup
constexpr int kScoreTok = 32;           // tokens per wave: two 16-token MFMA column blocks
constexpr int kChunkSteps = 8;          // k-steps (32 elements each) per staged chunk: 512 bytes of a bf16 row
constexpr int kStageBytes = kScoreTok * kChunkSteps * 64;   // one wave's LDS staging buffer (16 KB)

template <bool kBf16>
__global__ void __launch_bounds__(64 * kScoreWaves)
score_tiles_kernel(const void* __restrict__ tokens, int n_tiles, int n_v, int d,
                   const void* __restrict__ qbank, int nq, const float* __restrict__ w32,
                   double* __restrict__ token_key, float* __restrict__ token_sim,
                   double* __restrict__ inv_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    float* w_lds = reinterpret_cast<float*>(smem);

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int q = lane >> 4;

    for (int i = threadIdx.x; i < d; i += blockDim.x) w_lds[i] = w32[i];
    __syncthreads();

    const int n_sets = (n_v + kScoreTok - 1) / kScoreTok;
    const long long gw = (long long)blockIdx.x * kScoreWaves + wave;   // this wave's token set of all tiles
    if (gw >= (long long)n_tiles * n_sets) return;
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
        const bool valid = tok < n_v;
        if (valid && q == 0) {
            token_key[tile_row0 + tok] = key;
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
}

// Tile score: 64 strided partial sums of the tile's keys (token order), a
// halving tree, divided by n_v.  One wave per tile, four tiles per workgroup.
__global__ void __launch_bounds__(256)
tile_pool_kernel(const double* __restrict__ token_key, int n_tiles, int n_v, double* __restrict__ tile_score) {
    const int tile = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (tile >= n_tiles) return;
    const double* k = token_key + (size_t)tile * n_v;
    double p = 0.0;
    for (int i = lane; i < n_v; i += 64) p = p + k[i];
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        const double o = __shfl_down(p, s);
        p = p + o;
    }
    if (lane == 0) tile_score[tile] = p / (double)n_v;
}

// a precedes b: larger score first, then lower tile id.
__device__ __forceinline__ bool precedes(double ka, int ia, double kb, int ib) {
    return (ka > kb) || (ka == kb && ia < ib);
}

__global__ void __launch_bounds__(1024)
rank_tiles_kernel(const double* __restrict__ s, int n, int keep_count, double tau,
                  float* __restrict__ u_out, int* __restrict__ order, int* __restrict__ n_keep,
                  double* __restrict__ s_copy) {
    __shared__ double key[4096];
    __shared__ int id[4096];
    __shared__ int kept;
    int N = 1;
    while (N < n) N <<= 1;
    // A NaN score (only from a non-finite input) sorts as -inf: it ties the
    // pads and precedes them by id, so the first n entries are real tile ids.
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
        const double si = i < n ? s[i] : -INFINITY;
        key[i] = (si == si) ? si : -INFINITY;
        id[i] = i;
        if (s_copy != nullptr && i < n) s_copy[i] = s[i];
    }
    if (threadIdx.x == 0) kept = 0;
    __syncthreads();
    for (int size = 2; size <= N; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = threadIdx.x; t < (N >> 1); t += blockDim.x) {
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
    const double smax = key[0];
    const double smin = key[n - 1];
    const double range = smax - smin;
    int local = 0;
    for (int p = threadIdx.x; p < n; p += blockDim.x) {
        const double u = (smax == smin) ? 1.0 : (key[p] - smin) / range;
        order[p] = id[p];
        u_out[id[p]] = (float)u;
        local += (u >= tau) ? 1 : 0;
    }
    if (keep_count == 0 && local) atomicAdd(&kept, local);
    __syncthreads();
    if (threadIdx.x == 0) *n_keep = keep_count > 0 ? (keep_count < n ? keep_count : n) : kept;
}

hipError_t launch_score(const void* tokens, bool bf16, int n_tiles, int n_v, int d,
                        const void* qbank, int n_bg, int keep_count, double tau, int knn_m,
                        double* token_key, float* token_sim, double* tile_score, float* tile_u,
                        int* tile_order, int* n_keep, float* w32, double* inv, float* emb,
                        double* gram, double* s_smooth, hipStream_t st) {
    hipLaunchKernelGGL(prep_w_kernel, dim3((d + 255) / 256), dim3(256), 0, st, qbank, bf16 ? 1 : 0,
                       d, n_bg, w32);
    const long long sets = (long long)n_tiles * ((n_v + kScoreTok - 1) / kScoreTok);
    const unsigned wgs = (unsigned)((sets + kScoreWaves - 1) / kScoreWaves);
    const size_t lds = (size_t)d * sizeof(float) + (bf16 ? (size_t)kScoreWaves * kStageBytes : 0);
    double* inv_out = knn_m > 0 ? inv : nullptr;
    if (bf16) {
        hipLaunchKernelGGL(score_tiles_kernel<true>, dim3(wgs), dim3(64 * kScoreWaves), lds, st,
                           tokens, n_tiles, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, inv_out);
    } else {
        hipLaunchKernelGGL(score_tiles_kernel<false>, dim3(wgs), dim3(64 * kScoreWaves), lds, st,
                           tokens, n_tiles, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, inv_out);
    }
    hipLaunchKernelGGL(tile_pool_kernel, dim3((unsigned)((n_tiles + 3) / 4)), dim3(256), 0, st, token_key, n_tiles,
                       n_v, tile_score);
    const double* s_rank = tile_score;
    double* s_copy = nullptr;
    if (knn_m > 0) {
        const hipError_t e = launch_knn_smooth(tokens, bf16, n_tiles, n_v, d, inv, emb, gram, tile_score,
                                               knn_m, s_smooth, st);
        if (e != hipSuccess) return e;
        s_rank = s_smooth;
        s_copy = tile_score;   // the output tile score is the one the ranking used
    }
    hipLaunchKernelGGL(rank_tiles_kernel, dim3(1), dim3(1024), 0, st, s_rank, n_tiles,
                       keep_count, tau, tile_u, tile_order, n_keep, s_copy);
    return hipGetLastError();
}

}  // namespace rift

namespace rift {
hipError_t score_init_attributes() {
    const int bytes = 16384 * (int)sizeof(float) + kScoreWaves * kStageBytes;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<true>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<false>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}
}  // namespace rift

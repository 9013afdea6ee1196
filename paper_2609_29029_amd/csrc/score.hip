// Stage 1 of Rift (Sec. 2.3, Eq. 1; Listing 1; App. B Step 3) on gfx950.
//
//   prep_w       w = t - (1/M) sum_j B_j in float64, rounded to float32.
//   score_tiles  one workgroup per tile of up to 10 waves, a wave per 64-token
//                group (every 10th group beyond 640 tokens); each token row is
//                read a whole 128-byte line at a time, a line ahead of its use.
//                A single pass over the tile's tokens computes, per token,
//                  * the float64 ranking key r = (x.w)/|x| on the VALUs, in the
//                    fixed granule order (8-wide granules, granule g into
//                    accumulator g mod 4, then (a0+a2)+(a1+a3));
//                  * the cosines to t and every B_j with bf16 (or f32) MFMA,
//                    the query-versus-token relevance GEMM;
//                then pools the tile score s_i = mean r through LDS (64 strided
//                partial sums, halving tree, divide by n_v).
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

template <bool kBf16>
__global__ void __launch_bounds__(640)
score_tiles_kernel(const void* __restrict__ tokens, int n_v, int d,
                   const void* __restrict__ qbank, int nq, const float* __restrict__ w32,
                   double* __restrict__ token_key, float* __restrict__ token_sim,
                   double* __restrict__ tile_score, double* __restrict__ inv_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    float* w_lds = reinterpret_cast<float*>(smem);
    double* r_lds = reinterpret_cast<double*>(smem + (size_t)d * sizeof(float));

    const int tile = blockIdx.x;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int r = lane & 15;
    const int q = lane >> 4;

    for (int i = threadIdx.x; i < d; i += blockDim.x) w_lds[i] = w32[i];
    __syncthreads();

    const int n_groups = (n_v + 63) >> 6;       // 64 tokens per group
    const int n_waves = blockDim.x >> 6;
    for (int grp = wave; grp < n_groups; grp += n_waves) {
    int tok[4];
    size_t row_off[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        tok[b] = grp * 64 + b * 16 + r;
        int t_clamped = tok[b] < n_v ? tok[b] : n_v - 1;
        row_off[b] = ((size_t)tile * n_v + t_clamped) * (size_t)d;
    }
    const size_t q_off = (size_t)(r < nq ? r : nq - 1) * d;
    const int steps = d / 32;

    double n2[4] = {0.0, 0.0, 0.0, 0.0};
    double g[4] = {0.0, 0.0, 0.0, 0.0};
    f32x4_t acc[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if constexpr (kBf16) {
        const bf16_t* X = static_cast<const bf16_t*>(tokens);
        const bf16_t* Q = static_cast<const bf16_t*>(qbank);
        // ring of four register sets.  Two consecutive steps cover the two
        // halves of each token row's 128-byte lines, so their loads are issued
        // together, a line ahead: at even s, the loads of steps s + 2, s + 3.
        u32x4_t xs[4][4], qs[4];
        auto load = [&](int st, int slot) {
            const int k = st * 32 + q * 8;
#pragma unroll
            for (int b = 0; b < 4; ++b) xs[slot][b] = *reinterpret_cast<const u32x4_t*>(X + row_off[b] + k);
            qs[slot] = *reinterpret_cast<const u32x4_t*>(Q + q_off + k);
        };
#pragma unroll
        for (int j = 0; j < 2; ++j)
            if (j < steps) load(j, j);
        for (int s0 = 0; s0 < steps; s0 += 4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int s = s0 + j;
                if (s >= steps) break;
                if ((j & 1) == 0) {
                    if (s + 2 < steps) load(s + 2, (j + 2) & 3);
                    if (s + 3 < steps) load(s + 3, (j + 3) & 3);
                }
                const int k = s * 32 + q * 8;
                const f32x4_t w0 = *reinterpret_cast<const f32x4_t*>(w_lds + k);
                const f32x4_t w1 = *reinterpret_cast<const f32x4_t*>(w_lds + k + 4);
                const double wd[8] = {(double)w0[0], (double)w0[1], (double)w0[2], (double)w0[3],
                                      (double)w1[0], (double)w1[1], (double)w1[2], (double)w1[3]};
                const bf16x8_t qa = __builtin_bit_cast(bf16x8_t, qs[j]);
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const u32x4_t x = xs[j][b];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double x0 = (double)bf16_lo(x[e]);
                        const double x1 = (double)bf16_hi(x[e]);
                        n2[b] = fma(x0, x0, n2[b]);
                        g[b] = fma(x0, wd[2 * e], g[b]);
                        n2[b] = fma(x1, x1, n2[b]);
                        g[b] = fma(x1, wd[2 * e + 1], g[b]);
                    }
                    acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, __builtin_bit_cast(bf16x8_t, x),
                                                                     acc[b], 0, 0, 0);
                }
            }
        }
    } else {
        const float* X = static_cast<const float*>(tokens);
        const float* Q = static_cast<const float*>(qbank);
        for (int s = 0; s < steps; ++s) {
            const int k = s * 32 + q * 8;
            const f32x4_t w0 = *reinterpret_cast<const f32x4_t*>(w_lds + k);
            const f32x4_t w1 = *reinterpret_cast<const f32x4_t*>(w_lds + k + 4);
            const float wv[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
            const f32x4_t qa0 = *reinterpret_cast<const f32x4_t*>(Q + q_off + k);
            const f32x4_t qa1 = *reinterpret_cast<const f32x4_t*>(Q + q_off + k + 4);
            const float qa[8] = {qa0[0], qa0[1], qa0[2], qa0[3], qa1[0], qa1[1], qa1[2], qa1[3]};
#pragma unroll
            for (int b = 0; b < 4; ++b) {
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
    const size_t key_base = (size_t)tile * n_v;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        double nn = n2[b] + __shfl_xor(n2[b], 32);
        nn = nn + __shfl_xor(nn, 16);
        double gg = g[b] + __shfl_xor(g[b], 32);
        gg = gg + __shfl_xor(gg, 16);
        double key = (nn == 0.0) ? 0.0 : gg / sqrt(nn);
        key = key + 0.0;  // -0 -> +0
        const bool valid = tok[b] < n_v;
        if (valid && q == 0) {
            token_key[key_base + tok[b]] = key;
            r_lds[tok[b]] = key;
            if (inv_out != nullptr) inv_out[key_base + tok[b]] = (nn == 0.0) ? 0.0 : 1.0 / sqrt(nn);
        }
        if (token_sim != nullptr && valid) {
            const float inv = (nn > 0.0) ? (float)(1.0 / sqrt(nn)) : 0.0f;
            float* dst = token_sim + (key_base + tok[b]) * (size_t)nq;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                if (m < nq) dst[m] = acc[b][v] * inv;
            }
        }
    }
    }   // token groups
    __syncthreads();

    // Tile score: 64 strided partial sums of r, halving tree, divide by n_v.
    if (wave == 0) {
        double p = 0.0;
        for (int i = lane; i < n_v; i += 64) p = p + r_lds[i];
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) {
            const double o = __shfl_down(p, s);
            p = p + o;
        }
        if (lane == 0) tile_score[tile] = p / (double)n_v;
    }
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
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
        key[i] = i < n ? s[i] : -INFINITY;
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
        if (id[p] < n) u_out[id[p]] = (float)u;  // only a NaN score could sort a pad this early
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
    const int groups = (n_v + 63) / 64;
    const int waves = groups < 10 ? groups : 10;   // a wave takes every 10th group beyond 640 tokens
    const size_t lds = (size_t)d * sizeof(float) + (size_t)groups * 64 * sizeof(double);
    double* inv_out = knn_m > 0 ? inv : nullptr;
    if (bf16) {
        hipLaunchKernelGGL(score_tiles_kernel<true>, dim3(n_tiles), dim3(waves * 64), lds, st,
                           tokens, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, tile_score, inv_out);
    } else {
        hipLaunchKernelGGL(score_tiles_kernel<false>, dim3(n_tiles), dim3(waves * 64), lds, st,
                           tokens, n_v, d, qbank, 1 + n_bg, w32, token_key, token_sim, tile_score, inv_out);
    }
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
    const int bytes = 16384 * (int)sizeof(float) + 1024 * (int)sizeof(double);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<true>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&score_tiles_kernel<false>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}
}  // namespace rift

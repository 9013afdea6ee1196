// Optional Stage-1 score smoothing (Listing 1's note, App. B Step 3): each
// tile's score is averaged with those of its m most visually similar tiles.
//
//   pool_embed    E_i = fp32(sum over tokens t, ascending, of x_t * inv_t):
//                 one thread per 8 consecutive elements of a tile, the product
//                 and the sum each rounded on its own (no fused multiply-add),
//                 so the sum is the same sequence of float64 operations
//                 whatever the launch shape.
//   tile_gram     G_ij = the canonical float64 dot product of E_i and E_j
//                 (8-element granules, granule g into accumulator g mod 4, then
//                 (a0 + a2) + (a1 + a3)); the float32 products are exact in
//                 float64, so fused multiply-adds change nothing.  16 x 16 pairs
//                 per workgroup, 32-element chunks of both rows through LDS.
//   knn_smooth    one wave per tile: cosines G_ij / sqrt(G_ii G_jj) (0 when
//                 that is 0) in LDS, m rounds of a wave arg-max (largest
//                 cosine, then the lower tile), then
//                 s'_i = (s_i + s_j1 + ... + s_jm) / (1 + m) in that order.
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

template <bool kBf16>
__global__ void __launch_bounds__(64)
pool_embed_kernel(const void* __restrict__ tokens, int n_v, int d, const double* __restrict__ inv,
                  float* __restrict__ emb) {
    const int tile = blockIdx.y;
    const int k0 = (blockIdx.x * 64 + threadIdx.x) * 8;
    if (k0 >= d) return;
    const double* it = inv + (size_t)tile * n_v;
    double P[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) P[e] = 0.0;
    auto load = [&](int t, double (&x)[8]) {
        const size_t off = ((size_t)tile * n_v + t) * (size_t)d + k0;
        if constexpr (kBf16) {
            const u32x4_t v = *reinterpret_cast<const u32x4_t*>(static_cast<const bf16_t*>(tokens) + off);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[2 * e] = (double)bf16_lo(v[e]);
                x[2 * e + 1] = (double)bf16_hi(v[e]);
            }
        } else {
            const f32x4_t a = *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(tokens) + off);
            const f32x4_t b = *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(tokens) + off + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[e] = (double)a[e];
                x[4 + e] = (double)b[e];
            }
        }
    };
    int t = 0;
    for (; t + 4 <= n_v; t += 4) {   // four rows in flight
        double x[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) load(t + u, x[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const double s = it[t + u];
#pragma unroll
            for (int e = 0; e < 8; ++e) P[e] = __dadd_rn(P[e], __dmul_rn(x[u][e], s));
        }
    }
    for (; t < n_v; ++t) {
        double x[8];
        load(t, x);
        const double s = it[t];
#pragma unroll
        for (int e = 0; e < 8; ++e) P[e] = __dadd_rn(P[e], __dmul_rn(x[e], s));
    }
    float* out = emb + (size_t)tile * d + k0;
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (float)P[e];
}

__global__ void __launch_bounds__(256)
tile_gram_kernel(const float* __restrict__ emb, int n, int d, double* __restrict__ G) {
    __shared__ float A[16][33];
    __shared__ float B[16][33];
    const int tid = threadIdx.x;
    const int ti = tid & 15, tj = tid >> 4;
    const int i0 = blockIdx.x * 16, j0 = blockIdx.y * 16;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int k = 0; k < d; k += 32) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int idx = 2 * tid + u;          // 0..511: row idx / 32, column idx % 32
            const int r = idx >> 5, c = idx & 31;
            const int ia = (i0 + r) < n ? (i0 + r) : n - 1;
            const int jb = (j0 + r) < n ? (j0 + r) : n - 1;
            A[r][c] = emb[(size_t)ia * d + k + c];
            B[r][c] = emb[(size_t)jb * d + k + c];
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc[q] = fma((double)A[ti][8 * q + e], (double)B[tj][8 * q + e], acc[q]);
        __syncthreads();
    }
    const int i = i0 + ti, j = j0 + tj;
    if (i < n && j < n) G[(size_t)i * n + j] = (acc[0] + acc[2]) + (acc[1] + acc[3]);
}

__global__ void __launch_bounds__(64)
knn_smooth_kernel(const double* __restrict__ G, int n, const double* __restrict__ s_raw, int m,
                  double* __restrict__ s_out) {
    extern __shared__ double cosL[];   // [n] cosines, then [n] taken flags
    unsigned char* taken = reinterpret_cast<unsigned char*>(cosL + n);
    const int i = blockIdx.x;
    const int lane = threadIdx.x;
    const double gii = G[(size_t)i * n + i];
    for (int j = lane; j < n; j += 64) {
        const double den = sqrt(gii * G[(size_t)j * n + j]);
        const double c = (den == 0.0) ? 0.0 : G[(size_t)i * n + j] / den;
        // A NaN cosine (only from a non-finite input) ranks below every other
        // candidate; it stays a candidate, so every round picks some tile.
        cosL[j] = (c == c) ? c : -INFINITY;
        taken[j] = (j == i) ? 1 : 0;
    }
    __syncthreads();
    const int m_eff = m < n - 1 ? m : n - 1;
    double acc = s_raw[i];
    for (int r = 0; r < m_eff; ++r) {
        // arg-max over the tiles not yet taken: (cosine desc, id asc).  At least
        // n - 1 - r >= 1 tiles are left, and any of them beats the start value
        // (a -inf cosine ties -inf and has the lower id), so bj ends in [0, n).
        double bv = -INFINITY;
        int bj = 0x7fffffff;
        for (int j = lane; j < n; j += 64) {
            const double v = cosL[j];
            if (!taken[j] && (v > bv || (v == bv && j < bj))) {
                bv = v;
                bj = j;
            }
        }
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const double ov = __shfl_xor(bv, sft);
            const int oj = __shfl_xor(bj, sft);
            if (ov > bv || (ov == bv && oj < bj)) {
                bv = ov;
                bj = oj;
            }
        }
        __syncthreads();
        if ((bj & 63) == lane) taken[bj] = 1;
        __syncthreads();
        acc = acc + s_raw[bj];
    }
    if (lane == 0) s_out[i] = acc / (double)(1 + m_eff);
}

}  // namespace

hipError_t launch_knn_smooth(const void* tokens, bool bf16, int n_tiles, int n_v, int d,
                             const double* inv, float* emb, double* gram, const double* s_raw,
                             int m, double* s_out, hipStream_t st) {
    const dim3 pgrid((d + 511) / 512, n_tiles);
    if (bf16)
        hipLaunchKernelGGL(pool_embed_kernel<true>, pgrid, dim3(64), 0, st, tokens, n_v, d, inv, emb);
    else
        hipLaunchKernelGGL(pool_embed_kernel<false>, pgrid, dim3(64), 0, st, tokens, n_v, d, inv, emb);
    const dim3 ggrid((n_tiles + 15) / 16, (n_tiles + 15) / 16);
    hipLaunchKernelGGL(tile_gram_kernel, ggrid, dim3(256), 0, st, emb, n_tiles, d, gram);
    hipLaunchKernelGGL(knn_smooth_kernel, dim3(n_tiles), dim3(64), (size_t)n_tiles * (sizeof(double) + 1), st,
                       gram, n_tiles, s_raw, m, s_out);
    return hipGetLastError();
}

}  // namespace rift

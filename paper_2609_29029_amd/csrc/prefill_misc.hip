// Elementwise and normalisation kernels of the decoder prefill, plus the plain
// float32 path used by small (f32) models.
//   rope_table  (cos, sin)(p * base^(-2j/hd)) computed in float64, stored f32
//   rmsnorm     h = x / sqrt(mean(x^2) + eps) * g, one wave per row, float32 math
//   gemm_f32    C = A B^T (+C), 64x64 tiles through LDS
//   rope_apply_f32, swiglu_f32, to_f32
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

__global__ void rope_table_kernel(float2* __restrict__ tab, int n_pos, int half, int hd,
                                  double base) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long long)n_pos * half) return;
    const int p = (int)(i / half);
    const int j = (int)(i % half);
    const double theta = pow(base, -2.0 * (double)j / (double)hd);
    const double ang = (double)p * theta;
    tab[i] = make_float2((float)cos(ang), (float)sin(ang));
}

template <bool XBF16, bool GBF16, bool HBF16>
__global__ void __launch_bounds__(256)
rmsnorm_kernel(const void* __restrict__ x, float* __restrict__ resid, const void* __restrict__ g,
               void* __restrict__ h, int rows, int d, float eps) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const size_t base = (size_t)row * d;
    auto load4 = [&](int i) -> f32x4_t {
        if constexpr (XBF16) {
            const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(x) + base + i);
            return f32x4_t{bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y)};
        } else {
            return *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(x) + base + i);
        }
    };
    float ss = 0.f;
    for (int i = lane * 4; i < d; i += 256) {
        const f32x4_t v = load4(i);
        ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
        if (resid != nullptr) *reinterpret_cast<f32x4_t*>(resid + base + i) = v;
    }
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    for (int i = lane * 4; i < d; i += 256) {
        const f32x4_t v = load4(i);
        float gv[4];
        if constexpr (GBF16) {
            const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(g) + i);
            gv[0] = bf16_lo(w.x); gv[1] = bf16_hi(w.x); gv[2] = bf16_lo(w.y); gv[3] = bf16_hi(w.y);
        } else {
            const f32x4_t w = *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(g) + i);
            gv[0] = w[0]; gv[1] = w[1]; gv[2] = w[2]; gv[3] = w[3];
        }
        const float y0 = v[0] * inv * gv[0], y1 = v[1] * inv * gv[1];
        const float y2 = v[2] * inv * gv[2], y3 = v[3] * inv * gv[3];
        if constexpr (HBF16) {
            uint2 o;
            o.x = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
            o.y = (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16);
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(h) + base + i) = o;
        } else {
            *reinterpret_cast<f32x4_t*>(static_cast<float*>(h) + base + i) = f32x4_t{y0, y1, y2, y3};
        }
    }
}

// Same operation with the row held in registers (d = 256 NCH): every load of
// the row is issued before the first use, the row is read from memory once,
// and the squares are summed in the same lane-strided order as above.
template <bool XBF16, bool GBF16, bool HBF16, int NCH>
__global__ void __launch_bounds__(256)
rmsnorm_reg_kernel(const void* __restrict__ x, float* __restrict__ resid, const void* __restrict__ g,
                   void* __restrict__ h, int rows, float eps) {
    constexpr int d = 256 * NCH;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const size_t base = (size_t)row * d + lane * 4;
    f32x4_t v[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if constexpr (XBF16) {
            const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(x) + base + 256 * c);
            v[c] = f32x4_t{bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y)};
        } else {
            v[c] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(static_cast<const float*>(x) + base + 256 * c));
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) ss += v[c][0] * v[c][0] + v[c][1] * v[c][1] + v[c][2] * v[c][2] + v[c][3] * v[c][3];
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int i = lane * 4 + 256 * c;
        if (resid != nullptr) *reinterpret_cast<f32x4_t*>(resid + base + 256 * c) = v[c];
        float gv[4];
        if constexpr (GBF16) {
            const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(g) + i);
            gv[0] = bf16_lo(w.x); gv[1] = bf16_hi(w.x); gv[2] = bf16_lo(w.y); gv[3] = bf16_hi(w.y);
        } else {
            const f32x4_t w = *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(g) + i);
            gv[0] = w[0]; gv[1] = w[1]; gv[2] = w[2]; gv[3] = w[3];
        }
        const float y0 = v[c][0] * inv * gv[0], y1 = v[c][1] * inv * gv[1];
        const float y2 = v[c][2] * inv * gv[2], y3 = v[c][3] * inv * gv[3];
        if constexpr (HBF16) {
            uint2 o;
            o.x = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
            o.y = (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16);
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(h) + base + 256 * c) = o;
        } else {
            *reinterpret_cast<f32x4_t*>(static_cast<float*>(h) + base + 256 * c) = f32x4_t{y0, y1, y2, y3};
        }
    }
}

// C[M][N] = A[M][K] B[N][K]^T (+ C).  64x64 tile, 16x16 threads of 4x4 outputs.
__global__ void __launch_bounds__(256)
gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ B, float* __restrict__ C,
                int M, int N, int K, int accumulate) {
    __shared__ float As[16][64 + 1];
    __shared__ float Bs[16][64 + 1];
    const int m0 = blockIdx.y * 64;
    const int n0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 15;
    const int ty = threadIdx.x >> 4;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
        for (int e = threadIdx.x; e < 64 * 16; e += 256) {
            const int r = e >> 4;
            const int c = e & 15;
            const int kk = k0 + c;
            const int am = m0 + r, bn = n0 + r;
            As[c][r] = (am < M && kk < K) ? A[(size_t)am * K + kk] : 0.f;
            Bs[c][r] = (bn < N && kk < K) ? B[(size_t)bn * K + kk] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[c][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[c][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = m0 + ty * 4 + i;
        if (r >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = n0 + tx * 4 + j;
            if (c >= N) continue;
            float* dst = C + (size_t)r * N + c;
            *dst = accumulate ? *dst + acc[i][j] : acc[i][j];
        }
    }
}

__global__ void rope_apply_f32_kernel(float* __restrict__ x, const float2* __restrict__ tab,
                                      const int* __restrict__ pos, int n_pos, int M, int H,
                                      int hd) {
    const int half = hd / 2;
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long long)M * H * half) return;
    const int j = (int)(i % half);
    const long long rh = i / half;
    const int row = (int)(rh / H);
    const int head = (int)(rh % H);
    int p = pos[row];
    p = p < 0 ? 0 : (p >= n_pos ? n_pos - 1 : p);
    const float2 cs = tab[(size_t)p * half + j];
    float* base = x + (size_t)row * H * hd + (size_t)head * hd;
    const float x1 = base[j], x2 = base[j + half];
    base[j] = x1 * cs.x - x2 * cs.y;
    base[j + half] = x2 * cs.x + x1 * cs.y;
}

__global__ void swiglu_f32_kernel(const float* __restrict__ g, const float* __restrict__ u,
                                  float* __restrict__ a, long long n) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float gv = g[i];
    a[i] = gv / (1.0f + expf(-gv)) * u[i];
}

__global__ void to_f32_kernel(const void* __restrict__ x, int x_bf16, float* __restrict__ out,
                              long long n) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    out[i] = x_bf16 ? bf16_to_f32(static_cast<const bf16_t*>(x)[i]) : static_cast<const float*>(x)[i];
}

__global__ void copy_f32_kernel(const float* __restrict__ x, float* __restrict__ out, long long n) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    out[i] = x[i];
}

inline unsigned blocks_for(long long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t launch_rope_table(float2* tab, int n_pos, int hd, float base, hipStream_t st) {
    const long long n = (long long)n_pos * (hd / 2);
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(rope_table_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, tab, n_pos,
                       hd / 2, hd, (double)base);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(const void* x, bool x_bf16, float* resid, const void* g, bool g_bf16,
                          void* h, bool h_bf16, int rows, int d, float eps, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    const dim3 grid(blocks_for(rows, 4)), blk(256);
#define RIFT_RMS_REG(NCH)                                                                              \
    if (d == 256 * NCH) {                                                                              \
        if (x_bf16 && g_bf16 && h_bf16)                                                                \
            hipLaunchKernelGGL((rmsnorm_reg_kernel<true, true, true, NCH>), grid, blk, 0, st, x, resid, g, h, rows, eps); \
        else if (!x_bf16 && g_bf16 && h_bf16)                                                          \
            hipLaunchKernelGGL((rmsnorm_reg_kernel<false, true, true, NCH>), grid, blk, 0, st, x, resid, g, h, rows, eps); \
        else if (!x_bf16 && !g_bf16 && !h_bf16)                                                        \
            hipLaunchKernelGGL((rmsnorm_reg_kernel<false, false, false, NCH>), grid, blk, 0, st, x, resid, g, h, rows, eps); \
        else                                                                                           \
            return hipErrorInvalidValue;                                                               \
        return hipGetLastError();                                                                      \
    }
    RIFT_RMS_REG(1)
    RIFT_RMS_REG(2)
    RIFT_RMS_REG(4)
    RIFT_RMS_REG(8)
    RIFT_RMS_REG(16)
    RIFT_RMS_REG(32)
#undef RIFT_RMS_REG
    if (x_bf16 && g_bf16 && h_bf16)
        hipLaunchKernelGGL((rmsnorm_kernel<true, true, true>), grid, blk, 0, st, x, resid, g, h, rows, d, eps);
    else if (!x_bf16 && g_bf16 && h_bf16)
        hipLaunchKernelGGL((rmsnorm_kernel<false, true, true>), grid, blk, 0, st, x, resid, g, h, rows, d, eps);
    else if (!x_bf16 && !g_bf16 && !h_bf16)
        hipLaunchKernelGGL((rmsnorm_kernel<false, false, false>), grid, blk, 0, st, x, resid, g, h, rows, d, eps);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_gemm_f32(const float* a, const float* b, float* c, int M, int N, int K,
                           bool accumulate, hipStream_t st) {
    if (M <= 0 || N <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(blocks_for(N, 64), blocks_for(M, 64)), dim3(256), 0,
                       st, a, b, c, M, N, K, accumulate ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_rope_apply_f32(float* x, const float2* rope, const int* pos, int n_pos, int M,
                                 int n_heads, int hd, hipStream_t st) {
    const long long n = (long long)M * n_heads * (hd / 2);
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(rope_apply_f32_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, rope,
                       pos, n_pos, M, n_heads, hd);
    return hipGetLastError();
}

hipError_t launch_swiglu_f32(const float* g, const float* u, float* a, long long n,
                             hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(swiglu_f32_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, g, u, a, n);
    return hipGetLastError();
}

hipError_t launch_to_f32(const void* x, bool x_bf16, float* out, long long n, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(to_f32_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, x_bf16 ? 1 : 0,
                       out, n);
    return hipGetLastError();
}

hipError_t launch_copy_f32(const float* x, float* out, long long n, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(copy_f32_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, out, n);
    return hipGetLastError();
}

}  // namespace rift

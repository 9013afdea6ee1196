// Measurement aid, not part of the Rift path: the bf16 MFMA throughput the chip
// sustains when it does nothing else, the ceiling the prefill GEMMs are
// compared with beside the nominal peak.  Every wave of 512-thread workgroups
// (one per CU) issues independent MFMAs from registers; the operands rotate
// over eight register pairs so consecutive instructions see new inputs, as in
// a GEMM (constant operands draw less power and run faster).
//
//   form 0: v_mfma_f32_16x16x32_bf16, 16 accumulators of 4 floats per wave
//   form 1: v_mfma_f32_32x32x16_bf16,  8 accumulators of 16 floats per wave
//   form 2: as form 0 with 256-thread workgroups that reserve 96 KB of LDS, so
//           one wave per SIMD issues the MFMAs (the issue rate of a lone wave)
//
// One call runs blocks x W waves x iters x 262144 flop (iters a multiple of 8;
// W = 8 for forms 0 and 1, 4 for form 2).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// eight A and eight B fragments of 8 bf16 per lane from a table of 65536 values
__device__ __forceinline__ void load_operands(const uint16_t* __restrict__ src, int t, bf16x8_t (&a)[8],
                                              bf16x8_t (&b)[8]) {
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            a[r][j] = __builtin_bit_cast(__bf16, src[(t * 128 + r * 16 + j) & 65535]);
            b[r][j] = __builtin_bit_cast(__bf16, src[(t * 128 + r * 16 + 8 + j) & 65535]);
        }
}

template <int NT>
__global__ void __launch_bounds__(NT) ceiling_16x16x32(const uint16_t* __restrict__ src, float* __restrict__ out,
                                                       int iters) {
    // with 256 threads, 96 KB of LDS keeps a second workgroup off the CU
    __shared__ float reserve[NT == 256 ? 24 * 1024 : 1];
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    bf16x8_t a[8], b[8];
    load_operands(src, t, a, b);
    f32x4_t acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; it += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int j = 0; j < 16; ++j)
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j & 7], b[(j + u + (j >> 3)) & 7], acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    if (threadIdx.x == 0) reserve[0] = s;
    __syncthreads();
    out[t] = s + 0.f * reserve[0];
}

__global__ void __launch_bounds__(512) ceiling_32x32x16(const uint16_t* __restrict__ src, float* __restrict__ out,
                                                        int iters) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    bf16x8_t a[8], b[8];
    load_operands(src, t, a, b);
    f32x16_t acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
    for (int it = 0; it < iters; it += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j], b[(j + u) & 7], acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) s += acc[j][i];
    out[t] = s;
}

}  // namespace

// src: device, 65536 bf16 values; out: device, blocks * 512 floats (form 2
// writes the first blocks * 256).
// Returns 0, -1 for bad arguments, or the HIP error code of the launch.
extern "C" __attribute__((visibility("default"))) int rift_calib_mfma_bf16(int form, const uint16_t* src,
                                                                           float* out, int blocks, int iters,
                                                                           hipStream_t stream) {
    if (src == nullptr || out == nullptr || blocks < 1 || iters < 8 || iters % 8 != 0 || form < 0 || form > 2)
        return -1;
    if (form == 0)
        hipLaunchKernelGGL(ceiling_16x16x32<512>, dim3(blocks), dim3(512), 0, stream, src, out, iters);
    else if (form == 2)
        hipLaunchKernelGGL(ceiling_16x16x32<256>, dim3(blocks), dim3(256), 0, stream, src, out, iters);
    else
        hipLaunchKernelGGL(ceiling_32x32x16, dim3(blocks), dim3(512), 0, stream, src, out, iters);
    return (int)hipGetLastError();
}

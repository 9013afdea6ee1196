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
//
// rift_calib_mfma_bf16_moves: form 0 plus the data movement of the gate/up
// GEMM's main loop, without its waits and barriers: per 16 MFMAs a wave reads
// 6 x 16 bytes a lane from LDS into the operand registers of its next 16 MFMAs
// (384 bytes per MFMA, as a 128 x 64 wave tile reads its A and B fragments)
// and issues 2 LDS DMA loads of 16 bytes a lane from a 2.5 MiB buffer that
// stays in L2 (128 bytes per MFMA, as the stages of a 256 x 256 tile move them
// into LDS).  blocks x 8 waves x iters x 16 MFMAs (iters a multiple of 16).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

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

// 96 KB of LDS: [0, 64 KB) read back as operands, [64 KB, 96 KB) the DMA
// destination; one workgroup per CU, two waves per SIMD.
__global__ void __launch_bounds__(512) ceiling_moves(const uint16_t* __restrict__ src,
                                                     const u32x4_t* __restrict__ dsrc, float* __restrict__ out,
                                                     int iters) {
    constexpr int R = 6;   // LDS reads per 16 MFMAs
    constexpr int D = 2;   // LDS DMA loads per 16 MFMAs
    __shared__ __align__(16) u32x4_t lds[6144];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < 6144; i += 512) {
        u32x4_t v;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (uint32_t)src[(blockIdx.x * 977 + i * 8 + 2 * e) & 65535] |
                   ((uint32_t)src[(blockIdx.x * 977 + i * 8 + 2 * e + 1) & 65535] << 16);
        lds[i] = v;
    }
    __syncthreads();
    const int t = blockIdx.x * 512 + tid;
    bf16x8_t a[2][8], b[2][8];
    load_operands(src, t, a[0], b[0]);
    load_operands(src, t + 4099, a[1], b[1]);
    f32x4_t acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
    const uint64_t dbase = (uint64_t)(uintptr_t)dsrc;
    for (int it = 0; it < iters; it += 16) {
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int s = u & 1;   // set s feeds the MFMAs, set s ^ 1 is refilled
            asm volatile("" ::: "memory");
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s][j & 7], b[s][(j + u + (j >> 3)) & 7], acc[j],
                                                                 0, 0, 0);
                if (j < R) {
                    const int f = (u * R + j) % 16;
                    const int idx = (wave * 64 + lane + ((it + u) * 16 + j) * 576) & 4095;
                    const bf16x8_t v = __builtin_bit_cast(bf16x8_t, lds[idx]);
                    if (f < 8) a[s ^ 1][f] = v; else b[s ^ 1][f - 8] = v;
                }
                if (j >= 8 && j - 8 < D) {
                    const int jj = j - 8;
                    // byte offsets: lane part < 512 KiB, block part < 2 MiB
                    const uint32_t voff = (uint32_t)(lane * 16 + jj * 1024 + wave * 2048 + (blockIdx.x & 31) * 16384);
                    const uint64_t base = dbase + (uint64_t)((((it + u) * D + jj) * 4096) & 2097151);
                    const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)base) |
                                        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(base >> 32)) << 32);
                    const uint32_t m0 = lds0 + 65536u + (uint32_t)wave * 4096u + (uint32_t)((u * D + jj) & 3) * 1024u;
                    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                                 :: "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(ub) : "memory", "m0");
                }
            }
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) sum += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    out[t] = sum;
}

}  // namespace

// src: device, 65536 bf16 values; dsrc: device, dsrc_bytes >= 2.5 MiB (only
// its first 2.5 MiB are read); out: device, blocks * 512 floats.
// Returns 0, -1 for bad arguments, or the HIP error code of the launch.
extern "C" __attribute__((visibility("default"))) int rift_calib_mfma_bf16_moves(const uint16_t* src,
                                                                                 const void* dsrc,
                                                                                 long long dsrc_bytes, float* out,
                                                                                 int blocks, int iters,
                                                                                 hipStream_t stream) {
    if (src == nullptr || dsrc == nullptr || out == nullptr || dsrc_bytes < 2621440 || blocks < 1 || iters < 16 ||
        iters % 16 != 0)
        return -1;
    hipLaunchKernelGGL(ceiling_moves, dim3(blocks), dim3(512), 0, stream, src,
                       static_cast<const u32x4_t*>(dsrc), out, iters);
    return (int)hipGetLastError();
}

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

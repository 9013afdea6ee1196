// Device-side check for non-finite values (NaN or infinity) in a caller's
// floating-point buffer: the checks of the library's debug mode and of
// rift_check_finite.  An element is non-finite when every exponent bit is set
// (bfloat16: bits 7-14 of 16; float32: bits 23-30; float64: bits 52-62).
//
//   nonfinite_clear  one thread: the flag word := 0
//   nonfinite_scan   grid-stride over 16-byte words when the buffer is 16-byte
//                    aligned (element by element otherwise, and for the tail);
//                    a thread that sees a non-finite element stores
//                    RIFT_ERR_NONFINITE into the flag (every writer stores the
//                    same value, so the stores need no ordering).
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

template <int KIND>   // 0 bfloat16, 1 float32, 2 float64
__device__ __forceinline__ bool bad_word16(const u32x4_t w) {
    bool bad = false;
    if constexpr (KIND == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            bad |= ((w[i] & 0x7f80u) == 0x7f80u) | ((w[i] & 0x7f800000u) == 0x7f800000u);
    } else if constexpr (KIND == 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) bad |= (w[i] & 0x7f800000u) == 0x7f800000u;
    } else {
        bad = ((w[1] & 0x7ff00000u) == 0x7ff00000u) | ((w[3] & 0x7ff00000u) == 0x7ff00000u);
    }
    return bad;
}

template <int KIND>
__device__ __forceinline__ bool bad_elem(const unsigned char* x, long long i) {
    if constexpr (KIND == 0) {
        const uint16_t b = reinterpret_cast<const uint16_t*>(x)[i];
        return (b & 0x7f80u) == 0x7f80u;
    } else if constexpr (KIND == 1) {
        const uint32_t b = reinterpret_cast<const uint32_t*>(x)[i];
        return (b & 0x7f800000u) == 0x7f800000u;
    } else {
        const uint64_t b = reinterpret_cast<const uint64_t*>(x)[i];
        return (b & 0x7ff0000000000000ull) == 0x7ff0000000000000ull;
    }
}

__global__ void nonfinite_clear_kernel(int* flag) { *flag = 0; }

template <int KIND>
__global__ void __launch_bounds__(256) nonfinite_scan_kernel(const unsigned char* __restrict__ x, long long n,
                                                             int* __restrict__ flag) {
    constexpr int EB = KIND == 0 ? 2 : (KIND == 1 ? 4 : 8);
    const long long tid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long stride = (long long)gridDim.x * blockDim.x;
    bool bad = false;
    long long first_elem = 0;   // first element not covered by the 16-byte pass
    if ((reinterpret_cast<uintptr_t>(x) & 15) == 0) {
        const long long nw = (n * EB) / 16;
        const u32x4_t* xw = reinterpret_cast<const u32x4_t*>(x);
        for (long long i = tid; i < nw; i += stride) bad |= bad_word16<KIND>(xw[i]);
        first_elem = nw * 16 / EB;
    }
    for (long long i = first_elem + tid; i < n; i += stride) bad |= bad_elem<KIND>(x, i);
    if (bad) *flag = (int)RIFT_ERR_NONFINITE;
}

}  // namespace

hipError_t launch_nonfinite_clear(int* flag, hipStream_t st) {
    hipLaunchKernelGGL(nonfinite_clear_kernel, dim3(1), dim3(1), 0, st, flag);
    return hipGetLastError();
}

hipError_t launch_nonfinite_scan(const void* x, int kind, long long n, int* flag, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const int eb = kind == 0 ? 2 : (kind == 1 ? 4 : 8);
    const long long words = (n * eb + 15) / 16;
    long long blocks = (words + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    const unsigned char* p = static_cast<const unsigned char*>(x);
    if (kind == 0)
        hipLaunchKernelGGL(nonfinite_scan_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, st, p, n, flag);
    else if (kind == 1)
        hipLaunchKernelGGL(nonfinite_scan_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, st, p, n, flag);
    else
        hipLaunchKernelGGL(nonfinite_scan_kernel<2>, dim3((unsigned)blocks), dim3(256), 0, st, p, n, flag);
    return hipGetLastError();
}

}  // namespace rift

// Decode after prefill: one generated token per prompt and call.  Token
// `step` of prompt i sits at position L_i + step and attends causally to the
// prompt's keys and values, kept by the prefill (kv_cache, rotated keys), and
// to the generated tokens' own, kept in a decode cache slot per step.  With a
// shared prefix of P rows (the prefill's sequence 0), a prompt's keys are the
// P prefix rows followed by its own rows, and L_i counts both.  The
// decoder layers are those of the prefill (Sec. 2.1; LLaMA-7B shape); the
// per-token GEMMs run on the prefill's kernels with M = n_seq.
//
//   decode_pos     position of each prompt's new token, L_i + step
//   kv_append      this step's rotated key and value rows into slot `step`
//   decode_attn    one workgroup (4 waves) per (prompt, head), the HD / 8
//                  lanes of each row group reading one key or value row of
//                  2 HD bytes whole (HD = 128: 16 lanes, 16 groups; HD = 64: 8
//                  lanes, 32 groups): scores of every key in LDS (a dot
//                  product per group, summed over its lanes); the max and the
//                  sum of 2^(s - max) over the workgroup; then the weighted sum
//                  of the values, each lane 8 of the HD dimensions over its
//                  group's keys, the group sums added in fixed order; output
//                  rounded to bfloat16.
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

// cu: the prompts' own row offsets (after the shared prefix sequence when
// n_prefix > 0)
__global__ void decode_pos_kernel(const int* __restrict__ cu, int n_seq, int n_prefix, int step,
                                  int* __restrict__ pos) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_seq) pos[i] = n_prefix + (cu[i + 1] - cu[i]) + step;
}

// 16-byte words of row i of k and v into slot `step` of prompt i
__global__ void kv_append_kernel(const u32x4_t* __restrict__ k, const u32x4_t* __restrict__ v,
                                 u32x4_t* __restrict__ kc, u32x4_t* __restrict__ vc, int n_seq, int row_vec,
                                 int max_new, int step) {
    const long long w = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= (long long)n_seq * row_vec) return;
    const int i = (int)(w / row_vec), c = (int)(w % row_vec);
    const size_t dst = ((size_t)i * max_new + step) * row_vec + c;
    kc[dst] = k[w];
    vc[dst] = v[w];
}

// Sum over the G (16 or 8) lanes of each row group of the wave, every lane
// receiving the same sum: pairs, quads (quad_perm), halves (row_half_mirror)
// and, for G = 16, rows (row_mirror).  Each step adds two values that every
// lane of the group sees in one of two orders, so the lanes agree bit for bit.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xf, 0xf, false));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xf, 0xf, false));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xf, 0xf, false));
    if constexpr (G == 16)
        v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xf, 0xf, false));
    return v;
}

// Keys are visited in blocks of NS kDecU keys: slot s = (64 / G) wave +
// lane / G of the NS = 256 / G row groups takes keys j0 + NS u + s, u < kDecU,
// and the G lanes of a group read one row, lane c its bytes 16 c .. 16 c + 15
// (dims 8 c .. 8 c + 7).
constexpr int kDecU = 4;

template <int HD>
__global__ void __launch_bounds__(256)
decode_attn_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ kp, const bf16_t* __restrict__ vp,
                   const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn, const int* __restrict__ cu,
                   int n_seq, int T, int n_prefix, int H, int max_keys, int max_new, int step, float scale_log2,
                   bf16_t* __restrict__ o) {
    constexpr int G = HD / 8;        // lanes per row group
    constexpr int NS = 256 / G;      // row groups (key slots) per workgroup
    extern __shared__ float sc[];   // one score per key
    __shared__ float red[4];
    __shared__ float part[4][HD];
    const int seq = blockIdx.x / H;
    const int head = blockIdx.x % H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = lane % G;
    const int slot = (64 / G) * wave + lane / G;
    int s0 = cu[seq];
    int L = cu[seq + 1] - s0;
    if (s0 < 0 || L < 0 || s0 + L > T) s0 = L = 0;   // offsets outside the prefill cache: no prompt keys
    const int P = n_prefix;                           // shared prefix rows [0, P) of the cache
    // prefix keys, the prompt's own keys, then the generated ones (at most
    // max_keys, the LDS size)
    const int nk = min(P + L + step + 1, max_keys);
    const int ld = H * HD;
    const size_t hoff = (size_t)head * HD + 8 * c;
    auto row = [&](int j, const bf16_t* prompt_base, const bf16_t* new_base) -> const u32x4_t* {
        return reinterpret_cast<const u32x4_t*>(
            j < P ? prompt_base + (size_t)j * ld + hoff
                  : (j < P + L ? prompt_base + (size_t)(s0 + j - P) * ld + hoff
                               : new_base + ((size_t)seq * max_new + (j - P - L)) * ld + hoff));
    };
    float qf[8];
    {
        const u32x4_t qw = *reinterpret_cast<const u32x4_t*>(q + (size_t)seq * ld + hoff);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            qf[2 * e] = bf16_lo(qw[e]);
            qf[2 * e + 1] = bf16_hi(qw[e]);
        }
    }
    // scores (base-2 logits), and the running max of this lane's keys
    float mx = -INFINITY;
    for (int j0 = 0; j0 < nk; j0 += NS * kDecU) {
        u32x4_t kw[kDecU];
#pragma unroll
        for (int u = 0; u < kDecU; ++u)
            kw[u] = __builtin_nontemporal_load(row(min(j0 + NS * u + slot, nk - 1), kp, kn));
#pragma unroll
        for (int u = 0; u < kDecU; ++u) {
            float acc = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc = fmaf(bf16_lo(kw[u][e]), qf[2 * e], acc);
                acc = fmaf(bf16_hi(kw[u][e]), qf[2 * e + 1], acc);
            }
            const float sl = group_sum<G>(acc) * scale_log2;
            const int j = j0 + NS * u + slot;
            if (j < nk) {
                mx = fmaxf(mx, sl);
                if (c == 0) sc[j] = sl;
            }
        }
    }
    for (int s = 32; s >= 1; s >>= 1) mx = fmaxf(mx, __shfl_xor(mx, s));
    if (lane == 0) red[wave] = mx;
    __syncthreads();
    const float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    float sum = 0.f;
    for (int j = tid; j < nk; j += blockDim.x) {
        const float p = __builtin_amdgcn_exp2f(sc[j] - m);
        sc[j] = p;
        sum += p;
    }
    for (int s = 32; s >= 1; s >>= 1) sum += __shfl_xor(sum, s);
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    const float inv = 1.0f / ((red[0] + red[1]) + (red[2] + red[3]));
    // weighted values over the same key slots; lane c accumulates dims 8 c .. 8 c + 7
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int j0 = 0; j0 < nk; j0 += NS * kDecU) {
        u32x4_t vw[kDecU];
#pragma unroll
        for (int u = 0; u < kDecU; ++u)
            vw[u] = __builtin_nontemporal_load(row(min(j0 + NS * u + slot, nk - 1), vp, vn));
#pragma unroll
        for (int u = 0; u < kDecU; ++u) {
            const int j = j0 + NS * u + slot;
            if (j < nk) {
                const float p = sc[j];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] = fmaf(p, bf16_lo(vw[u][e]), acc[2 * e]);
                    acc[2 * e + 1] = fmaf(p, bf16_hi(vw[u][e]), acc[2 * e + 1]);
                }
            }
        }
    }
    // the row groups of a wave, then the four waves, in fixed order
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int sh = G; sh < 64; sh <<= 1) acc[e] += __shfl_xor(acc[e], sh);
    if (lane < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) part[wave][8 * c + e] = acc[e];
    }
    __syncthreads();
    if (tid < HD) {
        const float r = ((part[0][tid] + part[1][tid]) + part[2][tid]) + part[3][tid];
        o[(size_t)seq * ld + (size_t)head * HD + tid] = f32_to_bf16(r * inv);
    }
}

}  // namespace

hipError_t launch_decode_pos(const int* cu, int n_seq, int n_prefix, int step, int* pos, hipStream_t st) {
    hipLaunchKernelGGL(decode_pos_kernel, dim3((n_seq + 255) / 256), dim3(256), 0, st, cu, n_seq, n_prefix, step,
                       pos);
    return hipGetLastError();
}

hipError_t launch_kv_append(const uint16_t* k, const uint16_t* v, uint16_t* kc, uint16_t* vc, int n_seq, int d,
                            int max_new, int step, hipStream_t st) {
    const int row_vec = d / 8;
    const long long n = (long long)n_seq * row_vec;
    hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       reinterpret_cast<const u32x4_t*>(k), reinterpret_cast<const u32x4_t*>(v),
                       reinterpret_cast<u32x4_t*>(kc), reinterpret_cast<u32x4_t*>(vc), n_seq, row_vec, max_new, step);
    return hipGetLastError();
}

hipError_t launch_decode_attention(const uint16_t* q, const uint16_t* kp, const uint16_t* vp, const uint16_t* kn,
                                   const uint16_t* vn, const int* cu, int n_seq, int T, int n_prefix, int n_heads,
                                   int hd, int max_keys, int max_new, int step, uint16_t* o, hipStream_t st) {
    if (hd != 64 && hd != 128) return hipErrorInvalidValue;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    const dim3 grid((unsigned)(n_seq * n_heads));
    const size_t lds = (size_t)max_keys * sizeof(float);
    if (hd == 128)
        hipLaunchKernelGGL(decode_attn_kernel<128>, grid, dim3(256), lds, st, q, kp, vp, kn, vn, cu, n_seq, T,
                           n_prefix, n_heads, max_keys, max_new, step, scale_log2, o);
    else
        hipLaunchKernelGGL(decode_attn_kernel<64>, grid, dim3(256), lds, st, q, kp, vp, kn, vn, cu, n_seq, T,
                           n_prefix, n_heads, max_keys, max_new, step, scale_log2, o);
    return hipGetLastError();
}

}  // namespace rift

// Decode after prefill: one generated token per prompt and call.  Token
// `step` of prompt i sits at position L_i + step and attends causally to the
// prompt's keys and values, kept by the prefill (kv_cache, rotated keys), and
// to the generated tokens' own, kept in a decode cache slot per step.  The
// decoder layers are those of the prefill (Sec. 2.1; LLaMA-7B shape); the
// per-token GEMMs run on the prefill's kernels with M = n_seq.
//
//   decode_pos     position of each prompt's new token, L_i + step
//   kv_append      this step's rotated key and value rows into slot `step`
//   decode_attn    one workgroup (4 waves) per (prompt, head): the query in
//                  LDS; scores of every key (one key per lane, four waves
//                  splitting the keys) in LDS; the max and the sum of
//                  2^(s - max) over the workgroup; then the weighted sum of
//                  the values, each wave a quarter of the keys with every lane
//                  two of the 128 dimensions, the four partial sums added in
//                  wave order; output rounded to bfloat16.
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int DHD = 128;

__global__ void decode_pos_kernel(const int* __restrict__ cu, int n_seq, int step, int* __restrict__ pos) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_seq) pos[i] = (cu[i + 1] - cu[i]) + step;
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

__global__ void __launch_bounds__(256)
decode_attn_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ kp, const bf16_t* __restrict__ vp,
                   const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn, const int* __restrict__ cu,
                   int n_seq, int T, int H, int max_keys, int max_new, int step, float scale_log2,
                   bf16_t* __restrict__ o) {
    extern __shared__ float sc[];   // one score per key
    __shared__ float qs[DHD];
    __shared__ float red[4];
    __shared__ float part[4][DHD];
    const int seq = blockIdx.x / H;
    const int head = blockIdx.x % H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int s0 = cu[seq];
    int L = cu[seq + 1] - s0;
    if (s0 < 0 || L < 0 || s0 + L > T) s0 = L = 0;   // offsets outside the prefill cache: no prompt keys
    // prompt keys, then the generated ones (at most max_keys, the LDS size)
    const int nk = min(L + step + 1, max_keys);
    const int ld = H * DHD;
    const size_t hoff = (size_t)head * DHD;
    if (tid < DHD) qs[tid] = bf16_to_f32(q[(size_t)seq * ld + hoff + tid]);
    __syncthreads();
    auto key_row = [&](int j, const bf16_t* prompt_base, const bf16_t* new_base) -> const bf16_t* {
        return j < L ? prompt_base + (size_t)(s0 + j) * ld + hoff
                     : new_base + ((size_t)seq * max_new + (j - L)) * ld + hoff;
    };
    // scores, and the running max of this thread's keys
    float mx = -INFINITY;
    for (int j = tid; j < nk; j += blockDim.x) {
        const u32x4_t* kr = reinterpret_cast<const u32x4_t*>(key_row(j, kp, kn));
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < DHD / 8; ++c) {
            const u32x4_t w = kr[c];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc = fmaf(bf16_lo(w[e]), qs[8 * c + 2 * e], acc);
                acc = fmaf(bf16_hi(w[e]), qs[8 * c + 2 * e + 1], acc);
            }
        }
        const float sl = acc * scale_log2;
        sc[j] = sl;
        mx = fmaxf(mx, sl);
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
    // weighted values: wave w takes keys w, w + 4, ...; lane holds dims 2 lane, 2 lane + 1
    float o0 = 0.f, o1 = 0.f;
    for (int j = wave; j < nk; j += 4) {
        const uint32_t w = reinterpret_cast<const uint32_t*>(key_row(j, vp, vn))[lane];
        const float p = sc[j];
        o0 = fmaf(p, bf16_lo(w), o0);
        o1 = fmaf(p, bf16_hi(w), o1);
    }
    part[wave][2 * lane] = o0;
    part[wave][2 * lane + 1] = o1;
    __syncthreads();
    if (tid < DHD) {
        const float r = ((part[0][tid] + part[1][tid]) + part[2][tid]) + part[3][tid];
        o[(size_t)seq * ld + hoff + tid] = f32_to_bf16(r * inv);
    }
}

}  // namespace

hipError_t launch_decode_pos(const int* cu, int n_seq, int step, int* pos, hipStream_t st) {
    hipLaunchKernelGGL(decode_pos_kernel, dim3((n_seq + 255) / 256), dim3(256), 0, st, cu, n_seq, step, pos);
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
                                   const uint16_t* vn, const int* cu, int n_seq, int T, int n_heads, int max_keys,
                                   int max_new, int step, uint16_t* o, hipStream_t st) {
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)DHD);
    hipLaunchKernelGGL(decode_attn_kernel, dim3((unsigned)(n_seq * n_heads)), dim3(256),
                       (size_t)max_keys * sizeof(float), st, q, kp, vp, kn, vn, cu, n_seq, T, n_heads, max_keys,
                       max_new, step, scale_log2, o);
    return hipGetLastError();
}

}  // namespace rift

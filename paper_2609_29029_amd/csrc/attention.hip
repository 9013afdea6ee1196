// Varlen causal softmax attention of the packed prompts (each retained tile is
// an independent sequence; Sec. 2.3 Stage 2).  Query i of a sequence attends
// to keys 0..i of the same sequence, scale 1/sqrt(head_dim).
//
// bf16, head_dim 128, on MFMA.  One workgroup (4 waves) per (sequence, head),
// looping over the sequence's 128-query blocks (no workgroup is launched for a
// block past the end of a short prompt; workgroups are numbered sequence by
// sequence, so prompts packed longest first start first); wave w owns queries
// [32 w, 32 w + 32) of the block.  Keys
// and values stream through two LDS buffers 64 at a time, both row-major; the
// next block's rows are loaded into registers while the current one is used.
// The wave computes S^T = K Q^T (v_mfma_f32_32x32x16_bf16, M = keys,
// N = queries), so each lane holds one query's scores in registers; the online
// softmax runs in float32 (running max and sum per query); the unnormalised
// probabilities, rounded to bf16, are already in the B-operand layout of
// O^T = V^T P^T, whose A operand (V^T) comes from transposing LDS reads.
// Key blocks start at the sequence start, so a sequence's result does not
// depend on how it is packed.
//
// Shared prefix (n_prefix > 0): sequence 0 is rows [0, n_prefix), a prefix of
// every other sequence, computed once.  Sequence s > 0 then holds only its own
// rows; its logical keys are the prefix rows followed by its rows, and its
// queries sit at logical positions n_prefix onwards.  Key blocks still start
// at logical key 0, so the result is the same, bit for bit, as with the prefix
// packed into every sequence.
//
// The float32 path (small models) is a plain per-query loop.
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int HD = 128;
constexpr int BQ = 128;
constexpr int BKV = 64;
constexpr int KPAD = HD + 8;    // K tile row stride (elements): 272 B, b128 reads of 32 rows 2-way
constexpr int VPAD = HD + 32;   // V tile row stride (elements): 320 B, transposing reads 2-way

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// ds_read_b64_tr_b16: lane i of each 16-lane group g gets, in component j, the
// 16-bit element at (address passed by lane 16 g + 4 j + i / 4) + i % 4.
__device__ __forceinline__ v4s_t lds_read_tr16(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p));
}

__global__ void __launch_bounds__(256, 2)
attn_bf16_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                 const bf16_t* __restrict__ v, bf16_t* __restrict__ o,
                 const int* __restrict__ cu, int n_seq, int H, int n_prefix, float scale_log2) {
    __shared__ __align__(16) bf16_t Ks[2][BKV * KPAD];
    __shared__ __align__(16) bf16_t Vs[2][BKV * VPAD];

    const int seq = blockIdx.x / H;
    const int head = blockIdx.x % H;
    const int s0 = cu[seq];
    const int L = cu[seq + 1] - s0;
    const int pre = seq > 0 ? n_prefix : 0;   // logical keys before the sequence's own rows

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int col = lane & 31;
    const int ld = H * HD;
    const size_t head_off = (size_t)head * HD;

    // query blocks, the longest-running (last) first
    for (int qb = (L + BQ - 1) / BQ - 1; qb >= 0; --qb) {
    const int q0 = qb * BQ;
    __syncthreads();   // the previous block's reads of the K/V buffers are done
    const int qw = q0 + wave * 32;            // first query of this wave
    const int qidx = qw + col;                // this lane's query
    const int q_eff = qidx < L ? qidx : L - 1;

    // Q^T B-operand fragments: lane holds Q[query][16 kk + 8 h .. + 8]
    bf16x8_t qf[8];
    {
        const bf16_t* qrow = q + (size_t)(s0 + q_eff) * ld + head_off + 8 * h;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) qf[kk] = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * kk);
    }

    f32x16_t oacc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[t][i] = 0.f;
    float m_run = -INFINITY;
    float l_run = 0.f;

    // logical key range of this block and the logical position of the wave's last query
    const int kv_end = pre + ((q0 + BQ) < L ? (q0 + BQ) : L);
    const int nkv = (kv_end + BKV - 1) / BKV;
    const int wave_last = pre + ((qw + 31) < (L - 1) ? (qw + 31) : (L - 1));

    // K and V rows of a key block (clamped to the sequence): thread moves
    // 16 bytes of rows rr = (tid + 256 it) / 16 of both, into registers first
    u32x4_t kr[4], vr[4];
    auto load_block = [&](int kv0) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int vec = tid + 256 * it;
            int key = kv0 + (vec >> 4);
            key = key < pre + L ? key : pre + L - 1;
            const int row = key < pre ? key : s0 + key - pre;
            const size_t g = (size_t)row * ld + head_off + (vec & 15) * 8;
            kr[it] = *reinterpret_cast<const u32x4_t*>(k + g);
            vr[it] = *reinterpret_cast<const u32x4_t*>(v + g);
        }
    };
    auto store_block = [&](int buf) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int vec = tid + 256 * it;
            const int rr = vec >> 4;
            const int cc = (vec & 15) * 8;
            *reinterpret_cast<u32x4_t*>(&Ks[buf][rr * KPAD + cc]) = kr[it];
            *reinterpret_cast<u32x4_t*>(&Vs[buf][rr * VPAD + cc]) = vr[it];
        }
    };

    // transposing-read addresses of this lane as a source lane: group g,
    // component j, quad u -> key 4 (g >> 1) + j (+ 8), dims 16 (g & 1) + 4 u
    const int tg = lane >> 4, tj = (lane >> 2) & 3, tu = lane & 3;
    const int v_off = (4 * (tg >> 1) + tj) * VPAD + 16 * (tg & 1) + 4 * tu;

    load_block(0);
    store_block(0);
    __syncthreads();
    for (int kb_i = 0; kb_i < nkv; ++kb_i) {
        const int kv0 = kb_i * BKV;
        const int cur = kb_i & 1;
        if (kb_i + 1 < nkv) load_block(kv0 + BKV);
        if (kv0 <= wave_last) {
            // scores for two 32-key sub-blocks; their MFMA chains interleaved
            f32x16_t s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 8; ++kk)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    const bf16x8_t kf =
                        *reinterpret_cast<const bf16x8_t*>(&Ks[cur][(kb * 32 + col) * KPAD + 8 * h + 16 * kk]);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[kb], 0, 0, 0);
                }
            // raw scores; keys past a query are masked only in blocks that
            // cross the wave's diagonal.  The running max is kept on the raw
            // scale (scale_log2 > 0 commutes with max), and p = 2^(s scale - m)
            // takes one fma and the hardware exp2 (its flush of results below
            // 2^-126 to zero drops terms far below the row sum's precision).
            float sc[2][16];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) sc[kb][i] = s[kb][i];
            if (kv0 + BKV - 1 > pre + qw) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int key = kv0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                        sc[kb][i] = (key <= pre + q_eff) ? sc[kb][i] : -INFINITY;
                    }
            }
            float bmax = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) bmax = fmaxf(bmax, sc[kb][i]);
            bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
            const float m_new = fmaxf(m_run, bmax * scale_log2);
            const float neg_m = -m_new;
            float rsum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float pv = __builtin_amdgcn_exp2f(fmaf(sc[kb][i], scale_log2, neg_m));
                    sc[kb][i] = pv;
                    rsum += pv;
                }
            rsum += __shfl_xor(rsum, 32);
            // rescale the sums only when some query's max moved (exact skip)
            if (__any(m_new != m_run)) {
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                l_run *= alpha;
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int i = 0; i < 16; ++i) oacc[t][i] *= alpha;
            }
            l_run += rsum;
            m_run = m_new;

            // O^T += V^T P^T.  MFMA step ks of sub-block kb contracts keys
            // 16 ks + 4 h + {0..3} (slots 0..3) and 16 ks + 8 + 4 h + {0..3}
            // (slots 4..7) of lane half h: the P values this lane holds, and two
            // transposing reads of the row-major V tile give the same keys.
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    bf16x8_t pf;
#pragma unroll
                    for (int jj = 0; jj < 8; ++jj) pf[jj] = (__bf16)sc[kb][8 * ks + jj];
                    const bf16_t* vb = &Vs[cur][(kb * 32 + 16 * ks) * VPAD + v_off];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const v4s_t lo = lds_read_tr16(vb + 32 * t);
                        const v4s_t hi = lds_read_tr16(vb + 32 * t + 8 * VPAD);
                        const u32x4_t vv = {__builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1)),
                                            __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3)),
                                            __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1)),
                                            __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3))};
                        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv),
                                                                          pf, oacc[t], 0, 0, 0);
                    }
                }
        }
        // the other buffer was last read before the previous barrier
        if (kb_i + 1 < nkv) store_block(cur ^ 1);
        __syncthreads();
    }

    if (qidx < L) {
        const float inv = 1.0f / l_run;
        bf16_t* orow = o + (size_t)(s0 + qidx) * ld + head_off;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int dcol = t * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                orow[dcol] = f32_to_bf16(oacc[t][i] * inv);
            }
    }
    }   // query blocks
}

template <int D>
__global__ void __launch_bounds__(128)
attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                const float* __restrict__ v, float* __restrict__ o, const int* __restrict__ cu,
                int n_seq, int H, int n_prefix, float scale) {
    const int seq = blockIdx.x % n_seq;
    const int head = blockIdx.x / n_seq;
    const int s0 = cu[seq];
    const int L = cu[seq + 1] - s0;
    const int pre = seq > 0 ? n_prefix : 0;   // shared prefix rows [0, pre) come first
    const int ld = H * D;
    for (int i = threadIdx.x; i < L; i += blockDim.x) {
        const float* qi = q + (size_t)(s0 + i) * ld + head * D;
        float acc[D];
#pragma unroll
        for (int c = 0; c < D; ++c) acc[c] = 0.f;
        float m = -INFINITY, l = 0.f;
        for (int jl = 0; jl <= pre + i; ++jl) {
            const size_t row = jl < pre ? (size_t)jl : (size_t)(s0 + jl - pre);
            const float* kj = k + row * ld + head * D;
            float s = 0.f;
#pragma unroll
            for (int c = 0; c < D; ++c) s = fmaf(qi[c], kj[c], s);
            s *= scale;
            const float mn = fmaxf(m, s);
            const float a = expf(m - mn);
            const float p = expf(s - mn);
            l = l * a + p;
            const float* vj = v + row * ld + head * D;
#pragma unroll
            for (int c = 0; c < D; ++c) acc[c] = acc[c] * a + p * vj[c];
            m = mn;
        }
        float* oi = o + (size_t)(s0 + i) * ld + head * D;
#pragma unroll
        for (int c = 0; c < D; ++c) oi[c] = acc[c] / l;
    }
}

}  // namespace

hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, const int* cu, int n_seq, int max_seqlen,
                                 int n_heads, int n_prefix, hipStream_t st) {
    if (n_seq <= 0 || max_seqlen <= 0) return hipSuccess;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)HD);
    const long long blocks = (long long)n_seq * n_heads;
    hipLaunchKernelGGL(attn_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, st, q, k, v, o, cu,
                       n_seq, n_heads, n_prefix, scale_log2);
    return hipGetLastError();
}

hipError_t launch_attention_f32(const float* q, const float* k, const float* v, float* o,
                                const int* cu, int n_seq, int max_seqlen, int n_heads, int hd,
                                int n_prefix, hipStream_t st) {
    if (n_seq <= 0 || max_seqlen <= 0) return hipSuccess;
    const float scale = 1.0f / sqrtf((float)hd);
    const dim3 grid((unsigned)(n_seq * n_heads));
    if (hd == 64)
        hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(128), 0, st, q, k, v, o, cu, n_seq,
                           n_heads, n_prefix, scale);
    else
        hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(128), 0, st, q, k, v, o, cu, n_seq,
                           n_heads, n_prefix, scale);
    return hipGetLastError();
}

}  // namespace rift

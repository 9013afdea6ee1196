// Decode-shaped bf16 GEMMs on gfx950 MFMA: C = A B^T with one row per prompt,
// A [M][K] and B [N][K] both K-contiguous (activations and nn.Linear weights).
// At such M the product is bound by reading B, the weights, once; a 256 x 256
// output tile per workgroup would leave most of the chip idle, so K is split:
//
//   skinny_gemm     workgroup (chunk s, 128-column tile, 128-row tile)
//                   multiplies K chunk s of its tile and writes the float32
//                   partial product to part[s][M][N] with
//                   v_mfma_f32_32x32x16_bf16 blocks, each wave 32 columns.
//                   Both operands reach LDS by LDS DMA in whole 128-byte row
//                   segments, into a ring of 64-deep stages.  When the launch
//                   is one round over the CUs, eight waves split the tile 2 x 4
//                   and the ring holds three stages (two in flight); otherwise
//                   two four-wave workgroups share each CU with two-stage rings.
//   reduce kernels  add the S partials of every output in chunk order and do
//                   the layer's elementwise work: residual add then RMSNorm of
//                   the updated row; rotate-half RoPE of q and k, with k and v
//                   written into their decode-cache slot; SiLU(gate) * up.
//
// S depends on N and K only, and each chunk is one fixed sequence of MFMA
// accumulations, so a row's result does not depend on the other rows of the
// batch.  Chunk s of a launch runs on XCD s mod 8 (the hardware hands workgroup
// b to XCD b mod 8), so each XCD's L2 holds only its chunks of A.
#include <type_traits>

#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int SK_BM = 128;   // rows per tile
constexpr int SK_BN = 128;   // columns per workgroup (4 waves x 32)
constexpr int SK_KS = 64;    // k per stage
constexpr int SK_RB = 128;   // bytes of one operand row of a stage
constexpr int kSkinnyTargetWg = 256;   // split K until this many workgroups
constexpr int kSkinnyMaxSplit = 8;
constexpr int kSkinnyMinStages = 4;   // chunks of at least 256 k

struct SkinnyParams {
    const bf16_t* a;
    const bf16_t* b0;
    const bf16_t* b1;
    const bf16_t* b2;
    int nr;      // rows of each weight region: column n is row n mod nr of region n / nr
    int M, N, K;
    int S;       // K chunks
    int num_m;   // 128-row tiles
    float* part; // [S][M][N]
};

template <typename T>
__device__ __forceinline__ T* pick_region(int i, T* x, T* y, T* z) {
    const uintptr_t a = (uintptr_t)x, b = (uintptr_t)y, c = (uintptr_t)z;
    uintptr_t r = i == 1 ? b : a;
    r = i == 2 ? c : r;
    return (T*)r;
}

// LDS DMA (global_load_lds_dwordx4): 16 bytes per lane from base + voff to
// LDS address lds_addr + 16 lane (base and lds_addr wave-uniform).
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds_addr) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    // through uint32_t so that the low word is zero-extended
    const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b) |
                        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(ub) : "memory", "m0");
}

// Slot of 16-byte chunk c in an LDS operand row (128 bytes, 8 chunks):
// c ^ sk_swz(row), so that the operand reads of 8 and of 16 consecutive rows at
// one chunk hit distinct banks.
__device__ __forceinline__ int sk_swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// A stage (64 k) in LDS: A (activation) rows 0..127, then B (weight) rows
// 0..127, SK_RB bytes each; one LDS DMA instruction moves 8 rows (1 KB).
constexpr int kStageBytes = 2 * SK_BM * SK_RB;

// RING stages in LDS; 4 WM waves, wave w taking columns 32 (w % 4) .. + 31 and
// rows 128 / WM (w / 4) .. + 128 / WM - 1 of the tile.
//
// MFMA operands of v_mfma_f32_32x32x16_bf16 (lane l = r + 32 h): the A
// fragment of row block mb at 16-deep step t is row 32 mb + r, k = 16 t + 8 h
// .. + 7; the B fragment column r of the wave's 32 columns, same k.  Result
// element i is row 8 (i / 4) + 4 h + i % 4, column r.
//
// Stage j of the chunk is in ring slot j mod RING.  At the top of stage j
// every wave waits for its own DMA of stage j, the barrier makes every wave's
// visible (and frees slot j - 1, read in stage j - 1), and the DMA of stage
// j + RING - 1 goes into that slot.
template <int RING, int WM>
__global__ void __launch_bounds__(256 * WM)
skinny_gemm_kernel(SkinnyParams p) {
    constexpr int NW = 4 * WM;              // waves
    constexpr int DPW = 16 / NW;            // DMA instructions per operand, wave and stage
    constexpr int MB = 4 / WM;              // 32-row blocks per wave
    __shared__ __align__(16) unsigned char ring[RING * kStageBytes];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave & 3, wm = wave >> 2;
    const int bid = blockIdx.x;
    const int s = bid % p.S;
    const int tile = bid / p.S;
    const int m0 = (tile % p.num_m) * SK_BM;
    const int n0 = (tile / p.num_m) * SK_BN;
    const int nst_all = p.K / SK_KS;
    const int st0 = (int)((long long)s * nst_all / p.S);
    const int nst = (int)((long long)(s + 1) * nst_all / p.S) - st0;
    const int region = n0 / p.nr;
    const bf16_t* bmat = pick_region(region, p.b0, p.b1, p.b2);
    const int brow0 = n0 - region * p.nr;
    // DMA instruction j of this wave moves rows 8 (DPW wave + j) + lane / 8 of A
    // and of B; lane takes global chunk (lane % 8) ^ sk_swz(row) of the row
    uint32_t aoff[DPW], boff[DPW];
#pragma unroll
    for (int j = 0; j < DPW; ++j) {
        const int row = 8 * (DPW * wave + j) + (lane >> 3);
        const int c = (lane & 7) ^ sk_swz(row);
        const int ar = min(m0 + row, p.M - 1);   // rows past M repeat the last one
        aoff[j] = ((uint32_t)ar * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
        boff[j] = ((uint32_t)(brow0 + row) * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
    }
    const uint32_t ring_wave = (uint32_t)(uintptr_t)ring + (uint32_t)wave * (DPW * 1024u);
    auto dma_stage = [&](int j) {
        const uint32_t sb = ring_wave + (uint32_t)(j % RING) * kStageBytes;
        const size_t ko = (size_t)(st0 + j) * SK_KS;
#pragma unroll
        for (int q = 0; q < DPW; ++q) dma16(p.a + ko, aoff[q], sb + q * 1024u);
#pragma unroll
        for (int q = 0; q < DPW; ++q) dma16(bmat + ko, boff[q], sb + SK_BM * SK_RB + q * 1024u);
    };
    // operand read offsets (bytes within a stage) at step t: A of the wave's
    // first row block (each further block adds 32 rows, which keeps the
    // swizzle), B of the wave's columns
    const int r = lane & 31, h = lane >> 5;
    uint32_t ard[4], brd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int ar = 32 * MB * wm + r;
        ard[t] = (uint32_t)(ar * SK_RB + 16 * ((2 * t + h) ^ sk_swz(ar)));
        const int br = 32 * wn + r;
        brd[t] = (uint32_t)(SK_BM * SK_RB + br * SK_RB + 16 * ((2 * t + h) ^ sk_swz(br)));
    }

    f32x16_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mb][i] = 0.f;
    for (int j = 0; j < RING - 1 && j < nst; ++j) dma_stage(j);
    for (int j = 0; j < nst; ++j) {
        // DMAs issued after stage j: stages j + 1 .. min(nst, j + RING - 1) - 1, 2 DPW each
        const int later = min(nst - 1 - j, RING - 2);
        if (later >= 2) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(4 * DPW) : "memory");
        else if (later == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * DPW) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (j + RING - 1 < nst) dma_stage(j + RING - 1);
        const unsigned char* st = ring + (j % RING) * kStageBytes;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            bf16x8_t fa[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                fa[mb] = *reinterpret_cast<const bf16x8_t*>(st + ard[t] + 32 * mb * SK_RB);
            const bf16x8_t fb = *reinterpret_cast<const bf16x8_t*>(st + brd[t]);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mb], fb, acc[mb], 0, 0, 0);
        }
    }
    // partial products: 32 consecutive columns of one row per store
    const int col = n0 + 32 * wn + r;
    float* out = p.part + (size_t)s * p.M * p.N + col;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int row = m0 + 32 * (MB * wm + mb) + 8 * (i >> 2) + 4 * h + (i & 3);
            if (row < p.M) out[(size_t)row * p.N] = acc[mb][i];
        }
}

// x[row] += sum_s part[s][row] (chunk order); then, with h, the RMSNorm of the
// updated row times g, rounded to bfloat16.  One workgroup of T threads per
// row, thread t holding columns 4 t + 4 T c .. + 3, c < NCH; every partial of
// a thread is loaded before the first is added.
template <int T, int NCH>
__global__ void __launch_bounds__(T)
skinny_resid_norm_kernel(const float* __restrict__ part, int S, int M, float* __restrict__ x,
                         const bf16_t* __restrict__ g, bf16_t* __restrict__ h, float eps) {
    constexpr int d = 4 * T * NCH;
    constexpr int kMaxS = kSkinnyMaxSplit;
    __shared__ float red[T / 64];
    const int row = blockIdx.x;
    const int tid = threadIdx.x;
    const size_t base = (size_t)row * d + 4 * tid;
    f32x4_t w[kMaxS][NCH];
#pragma unroll
    for (int s = 0; s < kMaxS; ++s)
        if (s < S)
#pragma unroll
            for (int c = 0; c < NCH; ++c)
                w[s][c] = *reinterpret_cast<const f32x4_t*>(part + (size_t)s * M * d + base + 4 * T * c);
    f32x4_t v[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        v[c] = w[0][c];
#pragma unroll
        for (int s = 1; s < kMaxS; ++s)
            if (s < S) v[c] += w[s][c];
        f32x4_t* xp = reinterpret_cast<f32x4_t*>(x + base + 4 * T * c);
        v[c] = *xp + v[c];
        *xp = v[c];
    }
    if (h == nullptr) return;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) ss += v[c][0] * v[c][0] + v[c][1] * v[c][1] + v[c][2] * v[c][2] + v[c][3] * v[c][3];
    ss = wave_sum(ss);
    if ((tid & 63) == 0) red[tid >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < T / 64; ++i) tot += red[i];
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int i = 4 * tid + 4 * T * c;
        const uint2 gw = *reinterpret_cast<const uint2*>(g + i);
        const float y0 = v[c][0] * inv * bf16_lo(gw.x), y1 = v[c][1] * inv * bf16_hi(gw.x);
        const float y2 = v[c][2] * inv * bf16_lo(gw.y), y3 = v[c][3] * inv * bf16_hi(gw.y);
        uint2 o;
        o.x = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
        o.y = (uint32_t)f32_to_bf16(y2) | ((uint32_t)f32_to_bf16(y3) << 16);
        *reinterpret_cast<uint2*>(h + (size_t)row * d + i) = o;
    }
}

// q | k | v of row m from the partials of [wq | wk | wv] (N = 3 d): with
// half = hd / 2, thread (m, region, head, j4 < half / 4) owns columns
// j = 4 j4 .. + 3 of its head and their rotate-half partners j + half; q goes
// to q[m], k and v to slot `step` of prompt m in the decode cache.
__global__ void __launch_bounds__(256)
skinny_qkv_kernel(const float* __restrict__ part, int S, int M, int d, int hd, const float2* __restrict__ rope,
                  const int* __restrict__ pos, int n_pos, bf16_t* __restrict__ q, bf16_t* __restrict__ kc,
                  bf16_t* __restrict__ vc, int max_new, int step) {
    const int per_region = d >> 3;   // (head, j4) pairs
    const int half = hd >> 1;
    const int q4 = half >> 2;        // j4 per head
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)M * 3 * per_region) return;
    const int m = (int)(idx / (3 * per_region));
    const int rem = (int)(idx % (3 * per_region));
    const int region = rem / per_region;
    const int w = rem % per_region;
    const int j = 4 * (w % q4);
    const int hc = hd * (w / q4) + j;   // column of j within q, k or v
    const size_t N = 3 * (size_t)d;
    const float* p0 = part + (size_t)m * N + (size_t)region * d + hc;
    f32x4_t x1 = *reinterpret_cast<const f32x4_t*>(p0);
    f32x4_t x2 = *reinterpret_cast<const f32x4_t*>(p0 + half);
    for (int s = 1; s < S; ++s) {
        const float* ps = p0 + (size_t)s * M * N;
        x1 += *reinterpret_cast<const f32x4_t*>(ps);
        x2 += *reinterpret_cast<const f32x4_t*>(ps + half);
    }
    f32x4_t y1 = x1, y2 = x2;
    if (region < 2) {
        int ps = pos[m];
        ps = ps < 0 ? 0 : (ps >= n_pos ? n_pos - 1 : ps);
        const f32x4_t* cs = reinterpret_cast<const f32x4_t*>(rope + (size_t)ps * half + j);
        const f32x4_t c01 = cs[0], c23 = cs[1];   // (cos, sin) of j, j+1 and of j+2, j+3
        const float cv[4] = {c01[0], c01[2], c23[0], c23[2]};
        const float sv[4] = {c01[1], c01[3], c23[1], c23[3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            y1[e] = x1[e] * cv[e] - x2[e] * sv[e];
            y2[e] = x2[e] * cv[e] + x1[e] * sv[e];
        }
    }
    bf16_t* dst = region == 0 ? q + (size_t)m * d
                              : (region == 1 ? kc : vc) + ((size_t)m * max_new + step) * d;
    uint2 o1, o2;
    o1.x = (uint32_t)f32_to_bf16(y1[0]) | ((uint32_t)f32_to_bf16(y1[1]) << 16);
    o1.y = (uint32_t)f32_to_bf16(y1[2]) | ((uint32_t)f32_to_bf16(y1[3]) << 16);
    o2.x = (uint32_t)f32_to_bf16(y2[0]) | ((uint32_t)f32_to_bf16(y2[1]) << 16);
    o2.y = (uint32_t)f32_to_bf16(y2[2]) | ((uint32_t)f32_to_bf16(y2[3]) << 16);
    *reinterpret_cast<uint2*>(dst + hc) = o1;
    *reinterpret_cast<uint2*>(dst + hc + half) = o2;
}

// a[m][f] = silu(gate) * up from the partials of [wg | wu] (N = 2 F), four
// columns per thread; silu(g) = g / (1 + 2^(-g log2 e)) with the hardware exp2
// and reciprocal, as in the prefill's SwiGLU epilogue.
__global__ void __launch_bounds__(256)
skinny_swiglu_kernel(const float* __restrict__ part, int S, int M, int F, bf16_t* __restrict__ a) {
    const int q4 = F >> 2;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)M * q4) return;
    const int m = (int)(idx / q4);
    const int f = 4 * (int)(idx % q4);
    const size_t N = 2 * (size_t)F;
    const float* p0 = part + (size_t)m * N + f;
    f32x4_t gt = *reinterpret_cast<const f32x4_t*>(p0);
    f32x4_t up = *reinterpret_cast<const f32x4_t*>(p0 + F);
    for (int s = 1; s < S; ++s) {
        const float* ps = p0 + (size_t)s * M * N;
        gt += *reinterpret_cast<const f32x4_t*>(ps);
        up += *reinterpret_cast<const f32x4_t*>(ps + F);
    }
    bf16_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float ex = __builtin_amdgcn_exp2f(gt[e] * -1.4426950408889634f);
        o[e] = f32_to_bf16(gt[e] * __builtin_amdgcn_rcpf(1.0f + ex) * up[e]);
    }
    uint2 w;
    w.x = (uint32_t)o[0] | ((uint32_t)o[1] << 16);
    w.y = (uint32_t)o[2] | ((uint32_t)o[3] << 16);
    *reinterpret_cast<uint2*>(a + (size_t)m * F + f) = w;
}

}  // namespace

namespace {
int skinny_cu_count() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}
}  // namespace

int skinny_splits(int N, int K) {
    const int tiles = N / SK_BN;
    const int nst = K / SK_KS;
    int S = 1;
    while (S < kSkinnyMaxSplit && (long long)tiles * S < kSkinnyTargetWg && nst >= kSkinnyMinStages * 2 * S) S *= 2;
    return S;
}

bool skinny_supported(int N, int K, int nr) {
    return N > 0 && K > 0 && nr > 0 && N % SK_BN == 0 && K % SK_KS == 0 && nr % SK_BN == 0 && N % nr == 0 &&
           N / nr <= 3;
}

hipError_t launch_skinny_gemm(const uint16_t* a, const uint16_t* b0, const uint16_t* b1, const uint16_t* b2,
                              int nr, int M, int N, int K, float* part, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (!skinny_supported(N, K, nr)) return hipErrorInvalidValue;
    SkinnyParams p{};
    p.a = a;
    p.b0 = b0;
    p.b1 = b1 ? b1 : b0;
    p.b2 = b2 ? b2 : b0;
    p.nr = nr;
    p.M = M;
    p.N = N;
    p.K = K;
    p.S = skinny_splits(N, K);
    p.num_m = (M + SK_BM - 1) / SK_BM;
    p.part = part;
    const long long grid = (long long)p.S * p.num_m * (N / SK_BN);
    // one round of workgroups over the CUs: eight waves each (two per SIMD) and
    // a three-stage ring; more: two four-wave workgroups per CU, two-stage ring
    if (grid <= skinny_cu_count())
        hipLaunchKernelGGL((skinny_gemm_kernel<3, 2>), dim3((unsigned)grid), dim3(512), 0, st, p);
    else
        hipLaunchKernelGGL((skinny_gemm_kernel<2, 1>), dim3((unsigned)grid), dim3(256), 0, st, p);
    return hipGetLastError();
}

bool skinny_norm_supported(int d) {
    return d % 1024 == 0 && (d / 1024 == 1 || d / 1024 == 2 || d / 1024 == 4 || d / 1024 == 8 || d / 1024 == 16);
}

hipError_t launch_skinny_resid_norm(const float* part, int S, int M, int d, float* x, const uint16_t* g,
                                    uint16_t* h, float eps, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (S < 1 || S > kSkinnyMaxSplit) return hipErrorInvalidValue;
#define RIFT_SK_NORM(T, NCH)                                                                           \
    if (d == 4 * T * NCH) {                                                                            \
        hipLaunchKernelGGL((skinny_resid_norm_kernel<T, NCH>), dim3(M), dim3(T), 0, st, part, S, M, x, g, h, \
                           eps);                                                                       \
        return hipGetLastError();                                                                      \
    }
    RIFT_SK_NORM(256, 1)
    RIFT_SK_NORM(512, 1)
    RIFT_SK_NORM(1024, 1)
    RIFT_SK_NORM(1024, 2)
    RIFT_SK_NORM(1024, 4)
#undef RIFT_SK_NORM
    return hipErrorInvalidValue;
}

hipError_t launch_skinny_qkv(const float* part, int S, int M, int d, int hd, const float2* rope, const int* pos,
                             int n_pos, uint16_t* q, uint16_t* kc, uint16_t* vc, int max_new, int step,
                             hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (hd != 64 && hd != 128) return hipErrorInvalidValue;
    const long long n = (long long)M * 3 * (d / 8);
    hipLaunchKernelGGL(skinny_qkv_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, S, M, d, hd,
                       rope, pos, n_pos, q, kc, vc, max_new, step);
    return hipGetLastError();
}

hipError_t launch_skinny_swiglu(const float* part, int S, int M, int F, uint16_t* a, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    const long long n = (long long)M * (F / 4);
    hipLaunchKernelGGL(skinny_swiglu_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, S, M, F, a);
    return hipGetLastError();
}

}  // namespace rift

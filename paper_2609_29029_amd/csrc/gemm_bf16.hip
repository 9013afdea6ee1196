// bf16 GEMMs of the LLaMA decoder prefill on gfx950 MFMA, C = A B^T with A
// [M][K] and B [N][K] both K-contiguous (activations and nn.Linear weights),
// float32 accumulation, and the layer's elementwise work fused into the
// epilogue:
//   QKV   q|k|v = h [wq|wk|wv]^T, rotate-half RoPE on q and k, bf16 out
//   RESID x += A B^T in float32 (attention output and FFN down projections)
//   SWIGLU a = silu(h wg^T) * (h wu^T), bf16 out
//
// Tiling: a 256x256 output tile per workgroup of 8 waves (2 in M x 4 in N),
// each wave a 128x64 block of 8x4 v_mfma_f32_16x16x32_bf16 tiles (under the
// board power limit this instruction sustains more throughput than the
// 32x32x16 form on the same data).  K advances 64 per stage through two LDS
// buffers of 64 KB that LDS DMA (global_load_lds) fills a stage ahead.  The
// whole tiles run the ping-pong loop (the two waves on a SIMD alternate
// between a whole stage of MFMAs and the LDS reads of the next stage); the
// last tiles of a GEMM can run as 256x128 halves on 4 waves, each of which
// reads its operands for the next 32-deep sub-step while it runs the MFMAs of
// the current one.
//
// Every output element is one fixed sequence of MFMA accumulations over K, no
// matter which tile or batch row holds it, so a row's result does not depend on
// what else is packed with it.
//
// Tile order: tile ids walk 8 M-tiles per N-tile.  The hardware hands
// workgroup b to XCD b mod 8, and one workgroup fits a CU, so the 256
// workgroups of a round run together: in each round every XCD takes 32
// consecutive tile ids (8 M-tiles x 4 N-tiles, sharing A and B panels in its
// L2) of the same block of 256, so all XCDs stream the same 8 A panels at the
// same time, and the A panels of one M-group plus all of B stay in the
// memory-side cache while the group's rounds walk N.  With `reverse` a launch
// walks the same order from its last whole tile to its first.
#include <type_traits>

#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int kGroupM = 8;

enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };


struct GemmParams {
    const bf16_t* a;
    const bf16_t* b0;
    const bf16_t* b1;
    const bf16_t* b2;
    int M, N, K;
    int d;            // QKV: width of each of q, k, v;  SWIGLU: ffn width
    int hd;           // QKV: head dim, 128 or 64
    bf16_t* o0;
    bf16_t* o1;
    bf16_t* o2;
    float* resid;
    const float2* rope;
    const int* pos;
    int n_pos;
    int num_m, num_n;   // 256x256 output tiles
    int n_full;         // tiles 0 .. n_full-1 (grouped order) run as whole tiles,
                        // the rest as two 256x128 halves each
    int reverse;        // walk the whole tiles from the last to the first
};

// Workgroup bid of a launch of `count` workgroups -> its index in that launch,
// so that the hardware's round-robin of workgroups over the 8 XCDs gives each
// XCD a contiguous range of indices.
__device__ __forceinline__ int xcd_remap(int bid, int count) {
    const int xcd = bid & 7;
    const int slot = bid >> 3;
    const int base = count >> 3;
    const int extra = count & 7;
    return xcd * base + (xcd < extra ? xcd : extra) + slot;
}

// Workgroup bid of a launch of `count` whole tiles -> tile id: within each
// block of 256 workgroups, XCD bid mod 8 takes ids 32 (bid mod 8) + [0, 32) of
// the block; the last partial block is spread over the XCDs by xcd_remap.
__device__ __forceinline__ int round_remap(int bid, int count) {
    const int full = count & ~255;
    if (bid >= full) return full + xcd_remap(bid - full, count - full);
    return (bid & ~255) + (bid & 7) * 32 + ((bid >> 3) & 31);
}

// Tile t of the grouped order: 8 M-tiles per N-tile, so tiles with nearby t
// share A and B panels.
__device__ __forceinline__ void group_coords(int t, int num_m, int num_n, int& bm, int& bn) {
    const int group = t / (kGroupM * num_n);
    const int first_m = group * kGroupM;
    const int gm = (num_m - first_m) < kGroupM ? (num_m - first_m) : kGroupM;
    const int in_group = t - group * kGroupM * num_n;
    bm = first_m + in_group % gm;
    bn = in_group / gm;
}

// B operand of tile bn, row r (0..255): b_base_row is the matrix it is read
// from and b_row the row inside that matrix.
//   QKV:    one of wq | wk | wv per tile (d % 256 == 0), row bn*256 + r - region*d
//   SWIGLU: tile rows [0,64) gate, [64,128) up for output columns bn*128 + [0,64),
//           rows [128,192) gate, [192,256) up for columns bn*128 + [64,128)
//   RESID:  row bn*256 + r
// One of three pointers by a wave-uniform index, as selects on values (an
// indexed read of the kernel-argument struct would put it in scratch memory).
template <typename T>
__device__ __forceinline__ T* pick3(int i, T* x, T* y, T* z) {
    const uintptr_t a = (uintptr_t)x, b = (uintptr_t)y, c = (uintptr_t)z;
    uintptr_t r = i == 1 ? b : a;
    r = i == 2 ? c : r;
    return (T*)r;
}

template <int EPI>
__device__ __forceinline__ const bf16_t* b_base_row(const GemmParams& p, int bn, int r) {
    if constexpr (EPI == EPI_QKV) {
        const int region = __builtin_amdgcn_readfirstlane((bn * BN) / p.d);
        return pick3(region, p.b0, p.b1, p.b2);
    } else if constexpr (EPI == EPI_SWIGLU) {
        return ((r & 127) < 64) ? p.b0 : p.b1;
    } else {
        return p.b0;
    }
}

template <int EPI>
__device__ __forceinline__ int b_row(const GemmParams& p, int bn, int r) {
    if constexpr (EPI == EPI_QKV) {
        const int region = (bn * BN) / p.d;
        return bn * BN + r - region * p.d;
    } else if constexpr (EPI == EPI_SWIGLU) {
        return bn * 128 + (r >> 7) * 64 + (r & 63);
    } else {
        return bn * BN + r;
    }
}

// Same, saddr form: 64-bit wave-uniform base plus a 32-bit per-lane byte
// offset (the hardware adds them; offsets stay below 2^31 by the host checks).
__device__ __forceinline__ void dma16s(const void* base, uint32_t voff, uint32_t lds_addr) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    // readfirstlane returns a signed int: go through uint32_t so the low word is
    // zero-extended (sign extension would corrupt the upper half of the address)
    const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b) |
                        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(ub) : "memory", "m0");
}
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// ---------------------------------------------------------------------------
// Stages are 64 deep: two LDS buffers of 64 KB (A and B tiles, rows of 128
// bytes = one cache line of a K-contiguous operand row, so every LDS DMA
// request reads whole lines).  LDS rows hold 8 chunks of 16 bytes; chunk c of
// row r sits at c ^ swz8(r), conflict-free for the operand reads.
constexpr int BK3 = 64;
constexpr int kStage3 = 2 * BM * BK3;   // elements per stage (A then B)

__device__ __forceinline__ int swz8(int r) { return ((r >> 1) ^ ((r & 1) << 2)) & 7; }

// ---------------------------------------------------------------------------
// Wave layout: 2 (M) x 4 (N) waves, each 128 rows x 64 columns: eight 16-row
// blocks mb and four 16-column blocks nb at tile columns
// c0 + 16 (nb & 1) + 64 (nb >> 1) with c0 = 128 (wn >> 1) + 32 (wn & 1), so the
// RoPE pairs (j, j + 64) of a head and the gate/up pairs of SwiGLU (blocks nb
// and nb + 2) sit in the same lane.
//
// MFMA operands (lane l = r + 16 q): the A fragment of block mb in 32-deep
// sub-step s is row 16 mb + r, k = 32 s + 8 q .. + 7, the B fragment of block
// nb column r of the block, same k; result element v of the block is row
// 4 q + v, column r.
__device__ __forceinline__ int w8_c0(int wn) { return 128 * (wn >> 1) + 32 * (wn & 1); }
__device__ __forceinline__ int w8_col(int wn, int nb) { return w8_c0(wn) + 16 * (nb & 1) + 64 * (nb >> 1); }

// MFMA order inside a 32-deep sub-step: row block mb = i / 4 outer, column
// block nb inner, in snake order (0 1 2 3, 3 2 1 0, ...) so that consecutive
// MFMAs change only one operand (fewer input toggles under the power limit).
// The order of accumulation of any one output is unchanged.
__device__ __forceinline__ int snake_nb(int i) { return ((i >> 2) & 1) ? 3 - (i & 3) : (i & 3); }

// Epilogue.  For the bf16 outputs the stage buffers, free after the main loop,
// hold the tile: each wave writes its outputs (SiLU(gate)*up, RoPE'd q/k, v)
// into a row-major tile in LDS, then every thread of the workgroup moves 16
// contiguous bytes of a row, so global stores are whole row segments.  The
// residual GEMMs read, add and write float32 straight from the lanes (16
// consecutive columns of 4 rows per instruction).  acc[mb][nb][v] is tile row
// 128 wm + 16 mb + 4 (lane/16) + v, tile column w8_col(wn, nb) + lane%16.  A
// half-tile workgroup (HALF) holds logical tile columns [128 h, 128 h + 128).
constexpr int kStagingBytes = 256 * (256 + 8) * 2;   // largest staging tile (QKV, bf16)

template <int EPI, bool HALF>
__device__ __forceinline__ void epilogue_staged(const GemmParams& p, f32x4_t (&acc)[8][4], int m0, int bn,
                                                int h, int wm, int wn, int lane, const int* pos_lds,
                                                unsigned char* stage) {
    constexpr int NT = HALF ? 256 : 512;
    const int tid = threadIdx.x;
    const int col_in = lane & 15;
    const int row_hi = 4 * (lane >> 4);
    const int cbase = HALF ? 128 * h : 0;
    // No barrier here: in both kernels every wave's last operand read of the
    // stage buffers completes before a workgroup barrier that every wave has
    // passed before its last MFMAs (the ping-pong kernel: the end of group 1's
    // last read turn; the half-tile kernel: the barrier before the last
    // sub-step), so the buffers are free, and group 0 of the ping-pong kernel
    // starts its epilogue while group 1 runs its last MFMA turn.
    if constexpr (EPI == EPI_SWIGLU) {
        constexpr int OC = HALF ? 64 : 128;   // outputs per row of this workgroup
        constexpr int LD = OC + 8;
        bf16_t* S = reinterpret_cast<bf16_t*>(stage);
        const int sc = 64 * (wn >> 1) + 32 * (wn & 1) + col_in - (HALF ? 64 * h : 0);
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int r = wm * 128 + mb * 16 + row_hi + v;
                    const float gt = acc[mb][nb][v];
                    const float up = acc[mb][nb + 2][v];
                    // silu(g) = g / (1 + e^-g) with the hardware exp2 and reciprocal
                    // (about 1 ulp each; the result is rounded to bf16)
                    const float e = __builtin_amdgcn_exp2f(gt * -1.4426950408889634f);
                    S[r * LD + sc + 16 * nb] = f32_to_bf16(gt * __builtin_amdgcn_rcpf(1.0f + e) * up);
                }
        __syncthreads();
        constexpr int VPR = OC / 8;
        bf16_t* out = p.o0 + bn * 128 + (HALF ? 64 * h : 0);
        for (int v = tid; v < 256 * VPR; v += NT) {
            const int r = v / VPR;
            const int cv = (v % VPR) * 8;
            const int row = m0 + r;
            if (row < p.M)
                *reinterpret_cast<u32x4_t*>(out + (size_t)row * p.d + cv) =
                    *reinterpret_cast<const u32x4_t*>(S + r * LD + cv);
        }
    } else if constexpr (EPI == EPI_QKV) {
        constexpr int OC = HALF ? 128 : 256;
        constexpr int LD = OC + 8;
        bf16_t* S = reinterpret_cast<bf16_t*>(stage);
        const int region = __builtin_amdgcn_readfirstlane((bn * BN) / p.d);
        const int j = 32 * (wn & 1) + col_in;            // block nb = 0 column within the head (+16 for nb = 1)
        const int sc = 128 * (wn >> 1) + j - cbase;      // staging column of j; j + 64 at sc + 64
        // Head dim 64: the rotate-half partner of column c (c mod 64 < 32) is
        // c + 32, held by the same lane and accumulator slot of wave wn ^ 1
        // (wave index ^ 1, in whole and half tiles alike).  The two waves
        // swap their float32 values through LDS one row block at a time; each
        // keeps its own rotated half in acc, and the tile is then staged as v
        // is.  Angle index of (nb, lane): 16 (nb & 1) + col_in.
        const bool rope64 = p.hd == 64 && region < 2;
        if (rope64) {
            float* X = reinterpret_cast<float*>(stage);   // [wave][16 values][64 lanes] per row block
            const int wave = threadIdx.x >> 6;
            const bool first = (wn & 1) == 0;             // holds j < 32 of its head
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) {
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) X[(wave * 16 + nb * 4 + v) * 64 + lane] = acc[mb][nb][v];
                __syncthreads();
                const int r0 = wm * 128 + mb * 16 + row_hi;
#pragma unroll
                for (int nb = 0; nb < 4; ++nb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float other = X[((wave ^ 1) * 16 + nb * 4 + v) * 64 + lane];
                        const float2 cs = p.rope[(size_t)pos_lds[r0 + v] * 32 + 16 * (nb & 1) + col_in];
                        const float own = acc[mb][nb][v];
                        acc[mb][nb][v] = first ? own * cs.x - other * cs.y : own * cs.x + other * cs.y;
                    }
                __syncthreads();
            }
        }
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) {
            __builtin_amdgcn_sched_barrier(0);
            const int r0 = wm * 128 + mb * 16 + row_hi;
            if (region == 2 || rope64) {
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int r = r0 + v;
                        S[r * LD + sc + 16 * nb] = f32_to_bf16(acc[mb][nb][v]);
                        S[r * LD + sc + 16 * nb + 64] = f32_to_bf16(acc[mb][nb + 2][v]);
                    }
            } else {
                float2 cs[2][4];
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) cs[nb][v] = p.rope[(size_t)pos_lds[r0 + v] * 64 + j + 16 * nb];
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int r = r0 + v;
                        const float x1 = acc[mb][nb][v];
                        const float x2 = acc[mb][nb + 2][v];
                        S[r * LD + sc + 16 * nb] = f32_to_bf16(x1 * cs[nb][v].x - x2 * cs[nb][v].y);
                        S[r * LD + sc + 16 * nb + 64] = f32_to_bf16(x2 * cs[nb][v].x + x1 * cs[nb][v].y);
                    }
            }
        }
        __syncthreads();
        constexpr int VPR = OC / 8;
        bf16_t* out = pick3(region, p.o0, p.o1, p.o2) + (bn * BN - region * p.d) + cbase;
        for (int v = tid; v < 256 * VPR; v += NT) {
            const int r = v / VPR;
            const int cv = (v % VPR) * 8;
            const int row = m0 + r;
            if (row < p.M)
                *reinterpret_cast<u32x4_t*>(out + (size_t)row * p.d + cv) =
                    *reinterpret_cast<const u32x4_t*>(S + r * LD + cv);
        }
    } else {   // RESID: x += A B^T in float32, read-modify-write straight from the lanes
        const int c0 = w8_c0(wn);
#pragma unroll
        for (int mp = 0; mp < 8; mp += 2) {   // two row blocks at a time
            __builtin_amdgcn_sched_barrier(0);
            float old[2][4][4];
#pragma unroll
            for (int e = 0; e < 2; ++e)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int row = m0 + wm * 128 + (mp + e) * 16 + row_hi + v;
                    const float* src = p.resid + (size_t)(row < p.M ? row : p.M - 1) * p.N + bn * BN + c0 + col_in;
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) old[e][v][nb] = src[16 * (nb & 1) + 64 * (nb >> 1)];
                }
#pragma unroll
            for (int e = 0; e < 2; ++e)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int row = m0 + wm * 128 + (mp + e) * 16 + row_hi + v;
                    if (row >= p.M) continue;
                    float* dst = p.resid + (size_t)row * p.N + bn * BN + c0 + col_in;
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb)
                        dst[16 * (nb & 1) + 64 * (nb >> 1)] = old[e][v][nb] + acc[mp + e][nb][v];
                }
        }
        (void)stage;
        (void)cbase;
    }
}

// Half-tile kernel: a workgroup of 4 waves computes one half (128 columns,
// h = 0 or 1) of a 256x256 tile, as waves (wm, 2h + (wave & 1)) of the
// whole-tile layout would; only those 128 B rows are loaded.  Used for the last
// tiles of a GEMM so that the final round over the CUs is half as long.  Each
// wave reads its operands for the next 32-deep sub-step while it runs the 32
// MFMAs of the current one.  The barrier sits before sub-step 1: by then stage
// kt+1 has landed and every wave has read the whole of stage kt, so sub-step 1
// also issues the DMA of stage kt+2 into the buffer stage kt used, a stage
// before it is needed.
template <int EPI>
__global__ void __launch_bounds__(256, 1) gemm_bf16_half_kernel(GemmParams p) {
    __shared__ __align__(16) bf16_t lds[kStagingBytes / 2];   // two stages, then the epilogue tile
    __shared__ int pos_lds[BM];   // QKV: clamped position of each tile row
    int bm, bn, h;
    {
        const int i = xcd_remap(blockIdx.x, 2 * (p.num_m * p.num_n - p.n_full));
        h = i & 1;
        group_coords(p.n_full + (i >> 1), p.num_m, p.num_n, bm, bn);
    }
    const int m0 = bm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1;
    const int wn = 2 * h + (wave & 1);

    // DMA: instructions 0..7 of this wave move A rows 8 (8 wave + j) +
    // (lane >> 3), instructions 8..11 B rows 128 h + 8 (4 wave + j) +
    // (lane >> 3).  Per-lane byte offsets are fixed for the whole K loop; the
    // stage's K offset goes into the wave-uniform base.  LDS rows sit where
    // the whole-tile kernel puts them.
    constexpr int NA = 8;
    constexpr int NB = 4;
    constexpr int NQ = NA + NB;
    uint32_t aoff[NA], boff[NB];
    const bf16_t* bbase[NB];
    int arow0[NA], brow0[NB];
#pragma unroll
    for (int j = 0; j < NA; ++j) {
        arow0[j] = 8 * (NA * wave + j);
        const int row = arow0[j] + (lane >> 3);
        const int c = (lane & 7) ^ swz8(row);
        int ar = m0 + row;
        ar = ar < p.M ? ar : p.M - 1;
        aoff[j] = ((uint32_t)ar * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        brow0[j] = 128 * h + 8 * (4 * wave + j);
        const int row = brow0[j] + (lane >> 3);
        const int c = (lane & 7) ^ swz8(row);
        boff[j] = ((uint32_t)b_row<EPI>(p, bn, row) * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
        bbase[j] = b_base_row<EPI>(p, bn, brow0[j]);   // one matrix per 8-row group
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
    auto dma_one = [&](int buf, int kt, int q) {   // q = 0..NQ-1: A chunks then B chunks
        const uint32_t sb = lds0 + (uint32_t)buf * (kStage3 * 2);
        const size_t ko = (size_t)kt * BK3;
        if (q < NA) dma16s(p.a + ko, aoff[q], sb + (uint32_t)arow0[q] * 128u);
        else dma16s(bbase[q - NA] + ko, boff[q - NA], sb + BM * BK3 * 2 + (uint32_t)brow0[q - NA] * 128u);
    };

    if constexpr (EPI == EPI_QKV) {
        for (int i = tid; i < BM; i += 256) {
            int r = m0 + i;
            r = r < p.M ? r : p.M - 1;
            int ps = p.pos[r];
            pos_lds[i] = ps < 0 ? 0 : (ps >= p.n_pos ? p.n_pos - 1 : ps);
        }
    }

    f32x4_t acc[8][4];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nk = p.K / BK3;
    const int rd_a = (wm * 128 + (lane & 15)) * BK3;
    const int rd_b = BM * BK3 + (w8_c0(wn) + (lane & 15)) * BK3;
    const int key = swz8(lane & 15);
    const int qsel = lane >> 4;
    bf16x8_t fa[2][8], fb[2][4];
    // LDS read q (0..11) of sub-step s of buffer buf, in the order the MFMAs
    // consume them: a[0], b[0..3], a[1..7]
    auto read_one = [&](int slot, int buf, int s, int q) {
        const bf16_t* sA = lds + buf * kStage3;
        const int sw = ((4 * s + qsel) ^ key) << 3;
        if (q == 0) {
            fa[slot][0] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw);
        } else if (q <= 4) {
            const int nb = q - 1;
            fb[slot][nb] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + (16 * (nb & 1) + 64 * (nb >> 1)) * BK3);
        } else {
            fa[slot][q - 4] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + (q - 4) * 16 * BK3);
        }
    };
    auto mfma_one = [&](int slot, int i) {   // i = 0..31: (mb, nb) = (i >> 2, snake(i))
        const int mb = i >> 2, nb = snake_nb(i);
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[slot][mb], fb[slot][nb], acc[mb][nb], 0, 0, 0);
    };

#pragma unroll
    for (int q = 0; q < NQ; ++q) dma_one(0, 0, q);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    wg_barrier();
    if (nk > 1) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) dma_one(1, 1, q);
    }
#pragma unroll
    for (int q = 0; q < 12; ++q) read_one(0, 0, 0, q);

    // sub-step 0 reads sub-step 1 of the stage; sub-step 1 issues the DMA of
    // stage kt + 2 and reads sub-step 0 of stage kt + 1
    auto stage = [&](int kt, auto kDma, auto kMore) {
        const int cur = kt & 1;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            mfma_one(0, i);
            if ((i & 1) == 0 && (i >> 1) < 12) read_one(1, cur, 1, i >> 1);
            __builtin_amdgcn_sched_barrier(0);
        }
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
        wg_barrier();
#pragma unroll
        for (int m = 0; m < 8; ++m) asm volatile("" : "+v"(fa[1][m]));
#pragma unroll
        for (int n = 0; n < 4; ++n) asm volatile("" : "+v"(fb[1][n]));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            mfma_one(1, i);
            if constexpr (decltype(kDma)::value) {
                if ((i & 1) == 1 && (i >> 1) < NQ) dma_one(cur, kt + 2, i >> 1);
            }
            if constexpr (decltype(kMore)::value) {
                if ((i & 1) == 0 && (i >> 1) < 12) read_one(0, cur ^ 1, 0, i >> 1);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    int kt = 0;
    for (; kt + 2 < nk; ++kt) stage(kt, T_{}, T_{});
    if (kt + 1 < nk) stage(kt++, F_{}, T_{});
    stage(kt, F_{}, F_{});
    epilogue_staged<EPI, true>(p, acc, m0, bn, h, wm, wn, lane, pos_lds, reinterpret_cast<unsigned char*>(lds));
}

// ---------------------------------------------------------------------------
// Ping-pong kernel (every whole tile).  The 2 x 4 wave layout above, with the
// same LDS stages and order of accumulation as the half-tile kernel; the two
// waves that share a SIMD take turns: while one issues the 64 MFMAs of a whole 64-deep stage from
// registers, the other reads its operands for the next stage from LDS, and a
// workgroup barrier separates the turns.  Waves 0-3 (rows 0-127 of the tile)
// run one turn ahead of waves 4-7 (rows 128-255); the hardware places waves w
// and w + 4 of a 512-thread workgroup on the same SIMD, so every SIMD holds one
// wave of each group and its MFMA pipe is fed by one of them at every moment.
//
// Turn t (each ends with a barrier of all eight waves):
//   group 0: t = 2j   reads stage j          t = 2j+1  MFMAs of stage j
//   group 1: t = 2j+1 reads stage j          t = 2j+2  MFMAs of stage j
// Stage j sits in buffer j mod 2 and is last read in turn 2j+1, so the LDS
// DMA of stage j+2 is issued in turn 2j+2, all of it by group 0 while it reads
// stage j+1 (wave w moves its own rows and those of wave w + 4): the MFMA turns
// issue nothing but MFMAs, and the read turns have time to spare.  Group 0
// waits for that DMA at the end of turn 2j+3, before it reads stage j+2.
template <int EPI>
__global__ void __launch_bounds__(512, 1) gemm_bf16_pp_kernel(GemmParams p) {
    __shared__ __align__(16) bf16_t lds[kStagingBytes / 2];   // two stages, then the epilogue tile
    __shared__ int pos_lds[BM];   // QKV: clamped position of each tile row
    int bm, bn;
    {
        int t = round_remap(blockIdx.x, p.n_full);
        if (p.reverse) t = p.n_full - 1 - t;
        group_coords(t, p.num_m, p.num_n, bm, bn);
    }
    const int m0 = bm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2;   // also the group
    const int wn = wave & 3;

    // DMA: instruction j (0..3) of a wave moves A-tile rows and B-tile rows
    // 8 (4 wave + j) + (lane >> 3) of the stage.
    uint32_t aoff[4], boff[4];
    const bf16_t* bbase[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int row = 8 * (4 * wave + j) + (lane >> 3);
        const int c = (lane & 7) ^ swz8(row);
        int ar = m0 + row;
        ar = ar < p.M ? ar : p.M - 1;
        aoff[j] = ((uint32_t)ar * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
        boff[j] = ((uint32_t)b_row<EPI>(p, bn, row) * (uint32_t)p.K + (uint32_t)c * 8u) * 2u;
        bbase[j] = b_base_row<EPI>(p, bn, 8 * (4 * wave + j));
    }
    const uint32_t ring_wave = (uint32_t)(uintptr_t)lds + (uint32_t)wave * 4096u;
    auto dma_one = [&](int kt, int q) {   // q = 0..7: A chunks 0..3 then B chunks 0..3
        const uint32_t sb = ring_wave + (uint32_t)(kt & 1) * (kStage3 * 2);
        const size_t ko = (size_t)kt * BK3;
        if (q < 4) dma16s(p.a + ko, aoff[q], sb + q * 1024u);
        else dma16s(bbase[q - 4] + ko, boff[q - 4], sb + BM * BK3 * 2 + (q - 4) * 1024u);
    };
    // the share of wave w + 4 (rows + 128), issued by wave w of group 0; the B
    // row of tile row r + 128 is that of r plus 128 (64 for SWIGLU), same matrix
    const uint32_t bdelta = (uint32_t)(EPI == EPI_SWIGLU ? 64 : 128) * (uint32_t)p.K * 2u;
    auto dma_partner = [&](int kt, int q) {
        const uint32_t sb = ring_wave + 4u * 4096u + (uint32_t)(kt & 1) * (kStage3 * 2);
        const size_t ko = (size_t)kt * BK3;
        if (q < 4) {
            const int row = 8 * (4 * (wave + 4) + q) + (lane >> 3);
            const int c = (lane & 7) ^ swz8(row);
            int ar = m0 + row;
            ar = ar < p.M ? ar : p.M - 1;
            dma16s(p.a + ko, ((uint32_t)ar * (uint32_t)p.K + (uint32_t)c * 8u) * 2u, sb + q * 1024u);
        } else {
            dma16s(bbase[q - 4] + ko, boff[q - 4] + bdelta, sb + BM * BK3 * 2 + (q - 4) * 1024u);
        }
    };

    if constexpr (EPI == EPI_QKV) {
        if (tid < BM) {
            int r = m0 + tid;
            r = r < p.M ? r : p.M - 1;
            int ps = p.pos[r];
            pos_lds[tid] = ps < 0 ? 0 : (ps >= p.n_pos ? p.n_pos - 1 : ps);
        }
    }

    f32x4_t acc[8][4];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nk = p.K / BK3;
    const int rd_a = (wm * 128 + (lane & 15)) * BK3;
    const int rd_b = BM * BK3 + (w8_c0(wn) + (lane & 15)) * BK3;
    const int key = swz8(lane & 15);
    const int qsel = lane >> 4;
    bf16x8_t fa[2][8], fb[2][4];   // [32-deep sub-step][mb or nb]: one whole stage
    auto read_one = [&](int kt, int r) {   // r = 0..23: sub-step r / 12, operand r % 12
        const bf16_t* sA = lds + (kt & 1) * kStage3;
        const int s = r / 12, q = r % 12;
        const int sw = ((4 * s + qsel) ^ key) << 3;
        if (q < 8) {
            fa[s][q] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + q * 16 * BK3);
        } else {
            const int nb = q - 8;
            fb[s][nb] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + (16 * (nb & 1) + 64 * (nb >> 1)) * BK3);
        }
    };
    auto mfma_one = [&](int i) {   // i = 0..63: sub-step i / 32, (mb, nb) = ((i >> 2) & 7, snake(i))
        const int s = i >> 5, mb = (i >> 2) & 7, nb = snake_nb(i);
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[s][mb], fb[s][nb], acc[mb][nb], 0, 0, 0);
    };
    auto turn_end = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        wg_barrier();
        __builtin_amdgcn_sched_barrier(0);
    };
    // reads of stage kt; with kDma (group 0 only), the DMA of stage kt + 1 for
    // this wave's rows and for those of wave + 4
    auto read_turn = [&](int kt, auto kDma) {
#pragma unroll
        for (int r = 0; r < 24; ++r) {
            read_one(kt, r);
            if constexpr (decltype(kDma)::value) {
                if (r % 3 == 2) dma_one(kt + 1, r / 3);
                if (r % 3 == 0) dma_partner(kt + 1, r / 3);
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    };
    // MFMAs of stage kt
    auto mfma_turn = [&]() {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int i = 0; i < 64; ++i) {
            mfma_one(i);
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_setprio(0);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;

    // prologue: stages 0 and 1 in flight, wait for stage 0
#pragma unroll
    for (int q = 0; q < 8; ++q) dma_one(0, q);
    if (nk > 1) {
#pragma unroll
        for (int q = 0; q < 8; ++q) dma_one(1, q);
        asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    } else {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    turn_end();

    if (wm == 0) {
        // stage 1 was issued by the prologue; stages 2 .. nk-1 here
        auto step = [&](int kt, auto kDma) {
            read_turn(kt, kDma);
            turn_end();
            mfma_turn();
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            turn_end();
        };
        step(0, F_{});
        int kt = 1;
        for (; kt + 1 < nk; ++kt) step(kt, T_{});
        if (kt < nk) step(kt, F_{});
    } else {
        turn_end();
        for (int kt = 0; kt < nk; ++kt) {
            read_turn(kt, F_{});
            // only the prologue's DMA of stage 1 can still be in flight here
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            turn_end();
            mfma_turn();
            if (kt + 1 < nk) turn_end();
        }
    }
    epilogue_staged<EPI, false>(p, acc, m0, bn, 0, wm, wn, lane, pos_lds, reinterpret_cast<unsigned char*>(lds));
}

int cu_count() {
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

// Whole 256x256 tiles first (ping-pong kernel), then, if the tiles of the last
// round over the CUs fill at most half of it, those tiles as two 256x128
// halves each (half-tile kernel), so that round takes about half as long.
// Every output element is accumulated in the same order by both kernels.
template <int EPI>
hipError_t launch_gemm(GemmParams p, int num_n, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    p.num_m = (p.M + BM - 1) / BM;
    p.num_n = num_n;
    const int nt = p.num_m * num_n;
    const int cus = cu_count();
    const int rem = nt % cus;
    p.n_full = (2 * rem <= cus) ? nt - rem : nt;
    if (p.n_full > 0) {
        hipLaunchKernelGGL(gemm_bf16_pp_kernel<EPI>, dim3(p.n_full), dim3(512), 0, st, p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (nt > p.n_full)
        hipLaunchKernelGGL(gemm_bf16_half_kernel<EPI>, dim3(2 * (nt - p.n_full)), dim3(256), 0, st, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_qkv_rope(const QkvArgs& a, hipStream_t st, bool reverse) {
    GemmParams p{};
    p.a = a.a;
    p.b0 = a.wq;
    p.b1 = a.wk;
    p.b2 = a.wv;
    p.M = a.M;
    p.N = 3 * a.d;
    p.K = a.d;
    p.d = a.d;
    p.o0 = a.q;
    p.o1 = a.k;
    p.o2 = a.v;
    p.rope = a.rope;
    p.pos = a.pos;
    p.n_pos = a.n_pos;
    p.hd = a.hd;
    p.reverse = reverse ? 1 : 0;
    return launch_gemm<EPI_QKV>(p, p.N / BN, st);
}

hipError_t launch_gemm_resid(const uint16_t* a, const uint16_t* b, float* resid, int M, int N,
                             int K, hipStream_t st, bool reverse) {
    GemmParams p{};
    p.a = a;
    p.b0 = b;
    p.M = M;
    p.N = N;
    p.K = K;
    p.resid = resid;
    p.reverse = reverse ? 1 : 0;
    return launch_gemm<EPI_RESID>(p, N / BN, st);
}

hipError_t launch_gemm_swiglu(const uint16_t* a, const uint16_t* wg, const uint16_t* wu,
                              uint16_t* out, int M, int F, int K, hipStream_t st, bool reverse) {
    GemmParams p{};
    p.a = a;
    p.b0 = wg;
    p.b1 = wu;
    p.M = M;
    p.N = 2 * F;
    p.K = K;
    p.d = F;
    p.o0 = out;
    p.reverse = reverse ? 1 : 0;
    return launch_gemm<EPI_SWIGLU>(p, F / 128, st);
}

}  // namespace rift

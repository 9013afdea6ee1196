// bf16 GEMMs of the LLaMA decoder prefill on gfx950 MFMA, C = A B^T with A
// [M][K] and B [N][K] both K-contiguous (activations and nn.Linear weights),
// float32 accumulation, and the layer's elementwise work fused into the
// epilogue:
//   QKV   q|k|v = h [wq|wk|wv]^T, rotate-half RoPE on q and k, bf16 out
//   RESID x += A B^T in float32 (attention output and FFN down projections)
//   SWIGLU a = silu(h wg^T) * (h wu^T), bf16 out
//
// Tiling: a 256x256 output tile per workgroup of 4 waves (2x2), each wave a
// 128x128 block of 4x4 v_mfma_f32_32x32x16_bf16 tiles (256 accumulator
// registers).  K advances 32 per stage through a ring of four LDS stages
// (128 KB) that LDS DMA fills three stages ahead (see the kernel).
//
// Every output element is one fixed sequence of MFMA accumulations over K, no
// matter which tile or batch row holds it, so a row's result does not depend on
// what else is packed with it.
//
// Tile order: the hardware hands workgroup b to XCD b mod 8; each XCD gets a
// contiguous range of tile ids, and tile ids walk 8 M-tiles per N-tile, so the
// workgroups resident on one XCD share A and B panels in that XCD's L2.
#include <type_traits>

#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int kGroupM = 8;

enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

#ifndef RIFT_GEMM_K64
#define RIFT_GEMM_K64 1
#endif
#ifndef RIFT_GEMM_W8
#define RIFT_GEMM_W8 1
#endif

struct GemmParams {
    const bf16_t* a;
    const bf16_t* b0;
    const bf16_t* b1;
    const bf16_t* b2;
    int M, N, K;
    int d;            // QKV: width of each of q, k, v;  SWIGLU: ffn width
    bf16_t* o0;
    bf16_t* o1;
    bf16_t* o2;
    float* resid;
    const float2* rope;
    const int* pos;
    int n_pos;
};

__device__ __forceinline__ void tile_coords(int bid, int num_m, int num_n, int& bm, int& bn) {
    const int nt = num_m * num_n;
    const int xcd = bid & 7;
    const int slot = bid >> 3;
    const int base = nt >> 3;
    const int extra = nt & 7;
    const int t = xcd * base + (xcd < extra ? xcd : extra) + slot;
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
template <int EPI>
__device__ __forceinline__ const bf16_t* b_base_row(const GemmParams& p, int bn, int r) {
    if constexpr (EPI == EPI_QKV) {
        const int region = (bn * BN) / p.d;
        return region == 0 ? p.b0 : (region == 1 ? p.b1 : p.b2);
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

// Epilogue.  acc[m][n][i] is row 8 (i/4) + 4 (lane/32) + (i%4) and column
// lane%32 of the 32x32 tile (m, n) of wave (wm, wn).  Rows are handled 32 at a
// time (one m) so that every global load of a block is in flight at once.
// pos_lds holds the clamped position of each of the tile's 256 rows (QKV).
template <int EPI>
__device__ __forceinline__ void epilogue(const GemmParams& p, f32x16_t (&acc)[4][4], int m0, int bn,
                                         int wm, int wn, int lane, const int* pos_lds) {
    const int col_in = lane & 31;
    const int row_hi = 4 * (lane >> 5);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        __builtin_amdgcn_sched_barrier(0);
        const int r0 = wm * 128 + m * 32 + row_hi;   // tile row of i = 0
        if constexpr (EPI == EPI_RESID) {
            float old[16][4];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                const float* src = p.resid + (size_t)(row < p.M ? row : p.M - 1) * p.N +
                                   bn * BN + wn * 128 + col_in;
#pragma unroll
                for (int n = 0; n < 4; ++n) old[i][n] = src[n * 32];
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                if (row >= p.M) continue;
                float* dst = p.resid + (size_t)row * p.N + bn * BN + wn * 128 + col_in;
#pragma unroll
                for (int n = 0; n < 4; ++n) dst[n * 32] = old[i][n] + acc[m][n][i];
            }
        } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                if (row >= p.M) continue;
                bf16_t* dst = p.o0 + (size_t)row * p.d + bn * 128 + wn * 64 + col_in;
#pragma unroll
                for (int n = 0; n < 2; ++n) {
                    const float gt = acc[m][n][i];
                    const float up = acc[m][n + 2][i];
                    dst[n * 32] = f32_to_bf16(gt / (1.0f + expf(-gt)) * up);
                }
            }
        } else {  // QKV
            const int region = (bn * BN) / p.d;
            const int head_col = (bn * BN - region * p.d) + wn * 128;  // first column of the head
            bf16_t* outb = (region == 0 ? p.o0 : (region == 1 ? p.o1 : p.o2)) + head_col + col_in;
            if (region == 2) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                    if (row >= p.M) continue;
#pragma unroll
                    for (int n = 0; n < 4; ++n) outb[(size_t)row * p.d + n * 32] = f32_to_bf16(acc[m][n][i]);
                }
            } else {
#pragma unroll
                for (int half = 0; half < 2; ++half) {   // 8 rows at a time
                    __builtin_amdgcn_sched_barrier(0);
                    float2 cs[8][2];
#pragma unroll
                    for (int ii = 0; ii < 8; ++ii) {
                        const int i = 8 * half + ii;
                        const int ps = pos_lds[r0 + 8 * (i >> 2) + (i & 3)];
#pragma unroll
                        for (int n = 0; n < 2; ++n) cs[ii][n] = p.rope[(size_t)ps * 64 + n * 32 + col_in];
                    }
#pragma unroll
                    for (int ii = 0; ii < 8; ++ii) {
                        const int i = 8 * half + ii;
                        const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                        if (row >= p.M) continue;
                        bf16_t* out = outb + (size_t)row * p.d;
#pragma unroll
                        for (int n = 0; n < 2; ++n) {
                            const float x1 = acc[m][n][i];
                            const float x2 = acc[m][n + 2][i];
                            out[n * 32] = f32_to_bf16(x1 * cs[ii][n].x - x2 * cs[ii][n].y);
                            out[n * 32 + 64] = f32_to_bf16(x2 * cs[ii][n].x + x1 * cs[ii][n].y);
                        }
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Main loop: a 4-stage LDS ring filled by global_load_lds_dwordx4 (LDS DMA).
// K advances 32 per stage; a stage holds the A and B tiles (256 rows x 64
// bytes each, 32 KB).  Loads for stage k+3 are issued right after the barrier
// that opens stage k, so each load has about three stages of MFMA work to land;
// no registers stage the data.  Rows are 64 bytes (4 chunks of 16 bytes);
// chunk c of row r sits at position c ^ swz4(r), which keeps the operand reads
// of any 8 consecutive rows, and of the 4 rows r, r+4, r+8, r+12, on distinct
// banks.  The loads are issued with inline assembly and the waits are explicit
// (s_waitcnt vmcnt before every barrier), because the compiler would otherwise
// wait for every outstanding LDS DMA before each LDS read.
constexpr int BK2 = 32;
constexpr int NST = 4;
constexpr int kStageElems = 2 * BM * BK2;   // A tile then B tile

__device__ __forceinline__ int swz4(int r) { return ((r >> 2) ^ (r & 2)) & 3; }

// 16 bytes per lane from global memory to LDS address lds_addr + 16 * lane.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(g) : "memory", "m0");
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
template <int N>
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory"); }

template <int EPI>
__global__ void __launch_bounds__(256, 1) gemm_bf16_dma_kernel(GemmParams p) {
    __shared__ __align__(16) bf16_t lds[NST * kStageElems];
    __shared__ int pos_lds[BM];   // QKV: clamped position of each tile row
    const int num_m = (p.M + BM - 1) / BM;
    const int num_n = (EPI == EPI_SWIGLU) ? p.d / 128 : p.N / BN;
    int bm, bn;
    tile_coords(blockIdx.x, num_m, num_n, bm, bn);
    const int m0 = bm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1;
    const int wn = wave & 1;

    // DMA sources: instruction j (0..3) of this wave moves tile rows
    // 16 (4 wave + j) + (lane >> 2); the lane fetches logical chunk cl.
    const int rsub = lane >> 2;
    const int cl = (lane & 3) ^ swz4(rsub);
    const bf16_t* asrc[4];
    const bf16_t* bsrc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int row = 16 * (4 * wave + j) + rsub;
        int ar = m0 + row;
        ar = ar < p.M ? ar : p.M - 1;
        asrc[j] = p.a + (size_t)ar * p.K + cl * 8;
        bsrc[j] = b_base_row<EPI>(p, bn, row) + (size_t)b_row<EPI>(p, bn, row) * p.K + cl * 8;
    }
    const uint32_t ring = (uint32_t)(uintptr_t)lds;
    auto issue = [&](int stage, int kt) {
        const uint32_t sb = ring + (uint32_t)stage * (kStageElems * 2) + (uint32_t)wave * 4096u;
        const size_t ko = (size_t)kt * BK2;
#pragma unroll
        for (int j = 0; j < 4; ++j) dma16(asrc[j] + ko, sb + j * 1024u);
#pragma unroll
        for (int j = 0; j < 4; ++j) dma16(bsrc[j] + ko, sb + BM * BK2 * 2 + j * 1024u);
    };

    f32x16_t acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[m][n][i] = 0.f;

    if constexpr (EPI == EPI_QKV) {
        int r = m0 + tid;
        r = r < p.M ? r : p.M - 1;
        int ps = p.pos[r];
        pos_lds[tid] = ps < 0 ? 0 : (ps >= p.n_pos ? p.n_pos - 1 : ps);
    }   // read only after the main loop's barriers

    const int nk = p.K / BK2;
    for (int s = 0; s < 3 && s < nk; ++s) issue(s, s);

    // operand reads: row & 15 == lane & 15 for every (m, n), so one swizzle key
    const int rd_a = (wm * 128 + (lane & 31)) * BK2;
    const int rd_b = BM * BK2 + (wn * 128 + (lane & 31)) * BK2;
    const int key = swz4(lane & 15);
    const int hsel = lane >> 5;
    const int sw0 = ((0 + hsel) ^ key) << 3;   // k sub-step 0: logical chunks 0, 1
    const int sw1 = ((2 + hsel) ^ key) << 3;   // k sub-step 1: logical chunks 2, 3

    bf16x8_t a0[4], b0[4], a1[4], b1[4];
    auto read = [&](bf16x8_t (&af)[4], bf16x8_t (&bf)[4], int stage, int sw) {
        const bf16_t* sA = lds + stage * kStageElems;
#pragma unroll
        for (int m = 0; m < 4; ++m)
            af[m] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + m * 32 * BK2);
#pragma unroll
        for (int n = 0; n < 4; ++n)
            bf[n] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + n * 32 * BK2);
    };
    auto mma = [&](const bf16x8_t (&af)[4], const bf16x8_t (&bf)[4]) {
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int n = 0; n < 4; ++n)
                acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[m], bf[n], acc[m][n], 0, 0, 0);
    };
    // Wait until this wave's DMA for stage s has landed, given that the
    // stages after s up to min(s + 2, nk - 1) have been issued, then barrier.
    auto open_stage = [&](int s) {
        const int after = nk - 1 - s;
        if (after >= 2) asm volatile("s_waitcnt vmcnt(16) lgkmcnt(0)" ::: "memory");
        else if (after == 1) asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
        wg_barrier();
    };

    // Software pipeline: sub-step 1 of stage kt is read while sub-step 0
    // computes; stage kt+1 opens (wait, barrier, DMA of stage kt+4 into the
    // buffer stage kt used) between the two MFMA groups, and its sub-step 0 is
    // read while sub-step 1 of stage kt computes.
    open_stage(0);
    if (nk > 3) issue(3, 3);
    read(a0, b0, 0, sw0);
    int kt = 0;
    // steady state, branch-free: when stage kt+1 opens, stages kt+2 and kt+3
    // are in flight (16 DMA instructions per lane), and stage kt+4 exists
    // Steady state.  Each phase runs 16 MFMAs; in the shadow of each of its
    // first 8 MFMAs it issues one LDS read for the next phase (and, in phase 2,
    // one DMA instruction for stage kt+4), so neither reads nor DMA issue
    // stall the MFMA pipe.  Reads come in the order a[0], b[0..3], a[1..3], the
    // order in which the next phase's MFMAs need them.  sched_barrier pins the
    // order.
    auto read_one = [&](bf16x8_t (&af)[4], bf16x8_t (&bf)[4], int stage, int sw, int q) {
        const bf16_t* sA = lds + stage * kStageElems;
        if (q == 0) af[0] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw);
        else if (q <= 4) bf[q - 1] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + (q - 1) * 32 * BK2);
        else af[q - 4] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + (q - 4) * 32 * BK2);
    };
    const uint32_t ring_wave = ring + (uint32_t)wave * 4096u;
    for (; kt + 4 < nk; ++kt) {
        const int cur = kt & (NST - 1);
        const int nxt = (kt + 1) & (NST - 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            acc[q >> 2][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[q >> 2], b0[q & 3],
                                                                          acc[q >> 2][q & 3], 0, 0, 0);
            if (q < 8) read_one(a1, b1, cur, sw1, q);
            __builtin_amdgcn_sched_barrier(0);
        }
        asm volatile("s_waitcnt vmcnt(16) lgkmcnt(0)" ::: "memory");
        wg_barrier();
        // a1/b1 are complete (lgkmcnt(0) above); an empty asm that redefines
        // them tells the compiler so, and keeps it from waiting on the reads
        // issued below before using them
#pragma unroll
        for (int m = 0; m < 4; ++m) asm volatile("" : "+v"(a1[m]), "+v"(b1[m]));
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t sb = ring_wave + (uint32_t)cur * (kStageElems * 2);
        const size_t ko = (size_t)(kt + 4) * BK2;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            acc[q >> 2][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[q >> 2], b1[q & 3],
                                                                          acc[q >> 2][q & 3], 0, 0, 0);
            if (q < 4) dma16(asrc[q] + ko, sb + q * 1024u);
            else if (q < 8) dma16(bsrc[q - 4] + ko, sb + BM * BK2 * 2 + (q - 4) * 1024u);
            if (q < 8) read_one(a0, b0, nxt, sw0, q);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // last stages
    for (; kt < nk; ++kt) {
        const int cur = kt & (NST - 1);
        read(a1, b1, cur, sw1);
        mma(a0, b0);
        if (kt + 1 < nk) {
            open_stage(kt + 1);
            read(a0, b0, (kt + 1) & (NST - 1), sw0);
        }
        mma(a1, b1);
    }
    epilogue<EPI>(p, acc, m0, bn, wm, wn, lane, pos_lds);
}

// ---------------------------------------------------------------------------
// Main loop, 64-deep stages: two LDS buffers of 64 KB (A and B tiles, rows of
// 128 bytes = one cache line of a K-contiguous operand row, so every LDS DMA
// request reads whole lines).  Within a stage the four 16-deep sub-steps each
// run 16 MFMAs while the next sub-step's operands are read from LDS.  The
// barrier sits before sub-step 3: by then stage kt+1 has landed and every wave
// has read the whole of stage kt, so sub-step 3 also issues the DMA of stage
// kt+2 into the buffer stage kt used (one instruction per MFMA), about 64
// MFMAs before it is needed.  LDS rows hold 8 chunks of 16 bytes; chunk c of
// row r sits at c ^ swz8(r), conflict-free for the operand reads.
constexpr int BK3 = 64;
constexpr int kStage3 = 2 * BM * BK3;   // elements per stage (A then B)

__device__ __forceinline__ int swz8(int r) { return ((r >> 1) ^ ((r & 1) << 2)) & 7; }

template <int EPI>
__global__ void __launch_bounds__(256, 1) gemm_bf16_k64_kernel(GemmParams p) {
    __shared__ __align__(16) bf16_t lds[2 * kStage3];
    __shared__ int pos_lds[BM];   // QKV: clamped position of each tile row
    const int num_m = (p.M + BM - 1) / BM;
    const int num_n = (EPI == EPI_SWIGLU) ? p.d / 128 : p.N / BN;
    int bm, bn;
    tile_coords(blockIdx.x, num_m, num_n, bm, bn);
    const int m0 = bm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1;
    const int wn = wave & 1;

    // DMA: instruction j (0..7) of this wave moves tile rows 8 (8 wave + j) +
    // (lane >> 3), lane fetching logical chunk (lane & 7) ^ swz8(row).
    const bf16_t* asrc[8];
    const bf16_t* bsrc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int row = 8 * (8 * wave + j) + (lane >> 3);
        const int c = (lane & 7) ^ swz8(row);
        int ar = m0 + row;
        ar = ar < p.M ? ar : p.M - 1;
        asrc[j] = p.a + (size_t)ar * p.K + c * 8;
        bsrc[j] = b_base_row<EPI>(p, bn, row) + (size_t)b_row<EPI>(p, bn, row) * p.K + c * 8;
    }
    const uint32_t ring_wave = (uint32_t)(uintptr_t)lds + (uint32_t)wave * 8192u;
    auto dma_one = [&](int buf, int kt, int q) {   // q = 0..15: A chunks 0..7 then B chunks 0..7
        const uint32_t sb = ring_wave + (uint32_t)buf * (kStage3 * 2);
        const size_t ko = (size_t)kt * BK3;
        if (q < 8) dma16(asrc[q] + ko, sb + q * 1024u);
        else dma16(bsrc[q - 8] + ko, sb + BM * BK3 * 2 + (q - 8) * 1024u);
    };

    if constexpr (EPI == EPI_QKV) {
        int r = m0 + tid;
        r = r < p.M ? r : p.M - 1;
        int ps = p.pos[r];
        pos_lds[tid] = ps < 0 ? 0 : (ps >= p.n_pos ? p.n_pos - 1 : ps);
    }

    f32x16_t acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[m][n][i] = 0.f;

    const int nk = p.K / BK3;
    const int rd_a = (wm * 128 + (lane & 31)) * BK3;
    const int rd_b = BM * BK3 + (wn * 128 + (lane & 31)) * BK3;
    const int key = swz8(lane & 15);
    const int hsel = lane >> 5;
    // logical chunk of sub-step kk for this lane: 2 kk + hsel
    auto swk = [&](int kk) { return ((2 * kk + hsel) ^ key) << 3; };
    bf16x8_t fa[2][4], fb[2][4];
    // one LDS read (order a[0], b[0..3], a[1..3]) of sub-step kk of buffer buf
    auto read_one = [&](int slot, int buf, int kk, int q) {
        const bf16_t* sA = lds + buf * kStage3;
        const int sw = swk(kk);
        if (q == 0) fa[slot][0] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw);
        else if (q <= 4) fb[slot][q - 1] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + (q - 1) * 32 * BK3);
        else fa[slot][q - 4] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + (q - 4) * 32 * BK3);
    };
    auto mfma_one = [&](int slot, int q) {
        acc[q >> 2][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][q >> 2], fb[slot][q & 3],
                                                                      acc[q >> 2][q & 3], 0, 0, 0);
    };

    // prologue: stage 0 (and stage 1 when it exists) in flight, stage 0 landed
#pragma unroll
    for (int q = 0; q < 16; ++q) dma_one(0, 0, q);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    wg_barrier();
    if (nk > 1) {
#pragma unroll
        for (int q = 0; q < 16; ++q) dma_one(1, 1, q);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) read_one(0, 0, 0, q);

    // one stage; kDma / kMore say whether stage kt+2 gets loaded and whether
    // sub-step 0 of stage kt+1 gets read (both true except in the last two)
    auto stage = [&](int kt, auto kDma, auto kMore) {
        const int cur = kt & 1;
#pragma unroll
        for (int kk = 0; kk < 3; ++kk) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                mfma_one(kk & 1, q);
                if (q < 8) read_one((kk + 1) & 1, cur, kk + 1, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // stage kt+1 landed (its DMA is the only one outstanding) and every
        // wave has read all of stage kt
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
        wg_barrier();
#pragma unroll
        for (int m = 0; m < 4; ++m) asm volatile("" : "+v"(fa[1][m]), "+v"(fb[1][m]));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            mfma_one(1, q);
            if constexpr (decltype(kDma)::value) dma_one(cur, kt + 2, q);
            if constexpr (decltype(kMore)::value) { if (q < 8) read_one(0, cur ^ 1, 0, q); }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    int kt = 0;
    for (; kt + 2 < nk; ++kt) stage(kt, T_{}, T_{});
    if (kt + 1 < nk) stage(kt++, F_{}, T_{});
    stage(kt, F_{}, F_{});
    epilogue<EPI>(p, acc, m0, bn, wm, wn, lane, pos_lds);
}

// ---------------------------------------------------------------------------
// Eight-wave variant (two waves per SIMD, so one wave's LDS or DMA issue
// stalls are covered by the other's MFMAs).  Same tile, stages and order of
// accumulation; waves are 2 (M) x 4 (N), each 128 rows x 64 columns, its two
// 32-column blocks at tile columns c0 and c0 + 64 with
// c0 = 128 (wn >> 1) + 32 (wn & 1), so the RoPE pairs (j, j + 64) of a head and
// the gate/up pairs of SwiGLU sit in the same lane.
__device__ __forceinline__ int w8_c0(int wn) { return 128 * (wn >> 1) + 32 * (wn & 1); }

template <int EPI>
__device__ __forceinline__ void epilogue_w8(const GemmParams& p, f32x16_t (&acc)[4][2], int m0, int bn,
                                            int wm, int wn, int lane, const int* pos_lds) {
    const int col_in = lane & 31;
    const int row_hi = 4 * (lane >> 5);
    const int c0 = w8_c0(wn);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        __builtin_amdgcn_sched_barrier(0);
        const int r0 = wm * 128 + m * 32 + row_hi;   // tile row of i = 0
        if constexpr (EPI == EPI_RESID) {
            float old[16][2];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                const float* src = p.resid + (size_t)(row < p.M ? row : p.M - 1) * p.N + bn * BN + c0 + col_in;
#pragma unroll
                for (int n = 0; n < 2; ++n) old[i][n] = src[n * 64];
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                if (row >= p.M) continue;
                float* dst = p.resid + (size_t)row * p.N + bn * BN + c0 + col_in;
#pragma unroll
                for (int n = 0; n < 2; ++n) dst[n * 64] = old[i][n] + acc[m][n][i];
            }
        } else if constexpr (EPI == EPI_SWIGLU) {
            const int oc = bn * 128 + 64 * (wn >> 1) + 32 * (wn & 1) + col_in;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                if (row >= p.M) continue;
                const float gt = acc[m][0][i];
                const float up = acc[m][1][i];
                p.o0[(size_t)row * p.d + oc] = f32_to_bf16(gt / (1.0f + expf(-gt)) * up);
            }
        } else {  // QKV
            const int region = (bn * BN) / p.d;
            const int j = 32 * (wn & 1) + col_in;                                     // 0..63 in the head
            bf16_t* outb = (region == 0 ? p.o0 : (region == 1 ? p.o1 : p.o2)) +
                           (bn * BN - region * p.d) + 128 * (wn >> 1) + j;
            if (region == 2) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                    if (row >= p.M) continue;
#pragma unroll
                    for (int n = 0; n < 2; ++n) outb[(size_t)row * p.d + n * 64] = f32_to_bf16(acc[m][n][i]);
                }
            } else {
                float2 cs[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) cs[i] = p.rope[(size_t)pos_lds[r0 + 8 * (i >> 2) + (i & 3)] * 64 + j];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int row = m0 + r0 + 8 * (i >> 2) + (i & 3);
                    if (row >= p.M) continue;
                    const float x1 = acc[m][0][i];
                    const float x2 = acc[m][1][i];
                    bf16_t* out = outb + (size_t)row * p.d;
                    out[0] = f32_to_bf16(x1 * cs[i].x - x2 * cs[i].y);
                    out[64] = f32_to_bf16(x2 * cs[i].x + x1 * cs[i].y);
                }
            }
        }
    }
}

template <int EPI>
__global__ void __launch_bounds__(512, 1) gemm_bf16_w8_kernel(GemmParams p) {
    __shared__ __align__(16) bf16_t lds[2 * kStage3];
    __shared__ int pos_lds[BM];   // QKV: clamped position of each tile row
    const int num_m = (p.M + BM - 1) / BM;
    const int num_n = (EPI == EPI_SWIGLU) ? p.d / 128 : p.N / BN;
    int bm, bn;
    tile_coords(blockIdx.x, num_m, num_n, bm, bn);
    const int m0 = bm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2;
    const int wn = wave & 3;

    // DMA: instruction j (0..3) of this wave moves A-tile rows 8 (4 wave + j) +
    // (lane >> 3) and instruction 4 + j the same B-tile rows.
    // Per-lane byte offsets are fixed for the whole K loop; the stage's K
    // offset goes into the wave-uniform base.
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
        bbase[j] = b_base_row<EPI>(p, bn, 8 * (4 * wave + j));   // one matrix per 8-row group
    }
    const uint32_t ring_wave = (uint32_t)(uintptr_t)lds + (uint32_t)wave * 4096u;
    auto dma_one = [&](int buf, int kt, int q) {   // q = 0..7: A chunks 0..3 then B chunks 0..3
        const uint32_t sb = ring_wave + (uint32_t)buf * (kStage3 * 2);
        const size_t ko = (size_t)kt * BK3;
        if (q < 4) dma16s(p.a + ko, aoff[q], sb + q * 1024u);
        else dma16s(bbase[q - 4] + ko, boff[q - 4], sb + BM * BK3 * 2 + (q - 4) * 1024u);
    };

    if constexpr (EPI == EPI_QKV) {
        if (tid < BM) {
            int r = m0 + tid;
            r = r < p.M ? r : p.M - 1;
            int ps = p.pos[r];
            pos_lds[tid] = ps < 0 ? 0 : (ps >= p.n_pos ? p.n_pos - 1 : ps);
        }
    }

    f32x16_t acc[4][2];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[m][n][i] = 0.f;

    const int nk = p.K / BK3;
    const int rd_a = (wm * 128 + (lane & 31)) * BK3;
    const int rd_b = BM * BK3 + (w8_c0(wn) + (lane & 31)) * BK3;
    const int key = swz8(lane & 15);
    const int hsel = lane >> 5;
    auto swk = [&](int kk) { return ((2 * kk + hsel) ^ key) << 3; };
    bf16x8_t fa[2][4], fb[2][2];
    // one LDS read (order a[0], b[0], b[1], a[1..3]) of sub-step kk of buffer buf
    auto read_one = [&](int slot, int buf, int kk, int q) {
        const bf16_t* sA = lds + buf * kStage3;
        const int sw = swk(kk);
        if (q == 0) fa[slot][0] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw);
        else if (q <= 2) fb[slot][q - 1] = *reinterpret_cast<const bf16x8_t*>(sA + rd_b + sw + (q - 1) * 64 * BK3);
        else fa[slot][q - 2] = *reinterpret_cast<const bf16x8_t*>(sA + rd_a + sw + (q - 2) * 32 * BK3);
    };
    auto mfma_one = [&](int slot, int q) {   // q = 0..7: (m, n) = (q >> 1, q & 1)
        acc[q >> 1][q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][q >> 1], fb[slot][q & 1],
                                                                      acc[q >> 1][q & 1], 0, 0, 0);
    };

#pragma unroll
    for (int q = 0; q < 8; ++q) dma_one(0, 0, q);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    wg_barrier();
    if (nk > 1) {
#pragma unroll
        for (int q = 0; q < 8; ++q) dma_one(1, 1, q);
    }
#pragma unroll
    for (int q = 0; q < 6; ++q) read_one(0, 0, 0, q);

    auto stage = [&](int kt, auto kDma, auto kMore) {
        const int cur = kt & 1;
#pragma unroll
        for (int kk = 0; kk < 3; ++kk) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                mfma_one(kk & 1, q);
                if (q < 6) read_one((kk + 1) & 1, cur, kk + 1, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
        wg_barrier();
#pragma unroll
        for (int m = 0; m < 4; ++m) asm volatile("" : "+v"(fa[1][m]));
#pragma unroll
        for (int n = 0; n < 2; ++n) asm volatile("" : "+v"(fb[1][n]));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            mfma_one(1, q);
            if constexpr (decltype(kDma)::value) dma_one(cur, kt + 2, q);
            if constexpr (decltype(kMore)::value) { if (q < 6) read_one(0, cur ^ 1, 0, q); }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    int kt = 0;
    for (; kt + 2 < nk; ++kt) stage(kt, T_{}, T_{});
    if (kt + 1 < nk) stage(kt++, F_{}, T_{});
    stage(kt, F_{}, F_{});
    epilogue_w8<EPI>(p, acc, m0, bn, wm, wn, lane, pos_lds);
}

template <int EPI>
hipError_t launch_gemm(const GemmParams& p, int num_n, hipStream_t st) {
    const int num_m = (p.M + BM - 1) / BM;
    if (p.M <= 0) return hipSuccess;
#if RIFT_GEMM_W8
    hipLaunchKernelGGL(gemm_bf16_w8_kernel<EPI>, dim3(num_m * num_n), dim3(512), 0, st, p);
#elif RIFT_GEMM_K64
    hipLaunchKernelGGL(gemm_bf16_k64_kernel<EPI>, dim3(num_m * num_n), dim3(256), 0, st, p);
#else
    hipLaunchKernelGGL(gemm_bf16_dma_kernel<EPI>, dim3(num_m * num_n), dim3(256), 0, st, p);
#endif
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_qkv_rope(const QkvArgs& a, hipStream_t st) {
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
    return launch_gemm<EPI_QKV>(p, p.N / BN, st);
}

hipError_t launch_gemm_resid(const uint16_t* a, const uint16_t* b, float* resid, int M, int N,
                             int K, hipStream_t st) {
    GemmParams p{};
    p.a = a;
    p.b0 = b;
    p.M = M;
    p.N = N;
    p.K = K;
    p.resid = resid;
    return launch_gemm<EPI_RESID>(p, N / BN, st);
}

hipError_t launch_gemm_swiglu(const uint16_t* a, const uint16_t* wg, const uint16_t* wu,
                              uint16_t* out, int M, int F, int K, hipStream_t st) {
    GemmParams p{};
    p.a = a;
    p.b0 = wg;
    p.b1 = wu;
    p.M = M;
    p.N = 2 * F;
    p.K = K;
    p.d = F;
    p.o0 = out;
    return launch_gemm<EPI_SWIGLU>(p, F / 128, st);
}

}  // namespace rift

// Varlen causal softmax attention of the packed prompts (each retained tile is
// an independent sequence; Sec. 2.3 Stage 2).  Query i of a sequence attends
// to keys 0..i of the same sequence, scale 1/sqrt(head_dim).
//
// bf16, head_dim 128 or 64, on MFMA.  With a head count that is a multiple of
// 8, one workgroup of W = 4 waves per (sequence, head, 128-query block), from
// a work list built once per prefill: workgroup b runs entry b / 8 (sequence,
// group of 8 heads, block) for head 8 g + b mod 8, so all blocks of one
// (sequence, head) run on one XCD at about the same time and read its keys
// and values from that XCD's L2 after the first fetch (HBM-side fetch per
// layer 0.46 GB, the q, k and v bytes, against 0.79 GB when one workgroup
// loops over a sequence's blocks and its later passes miss the L2).
// Otherwise one workgroup per (sequence, head), looping over the sequence's
// 128-query blocks, the last (longest-running) first.  Wave w owns queries
// [32 w, 32 w + 32) of a block (sequences in packing order, so prompts packed
// longest first start first).  Keys and values stream 64 at a time through a ring of
// S = 2 LDS stages that LDS DMA fills a block ahead, one barrier per block,
// and two workgroups share a CU; the last key block of a query block loads
// the first one of the next query block.  Tile rows are 256 bytes, unpadded; the
// 16-byte chunks of row r sit at chunk ^ (r & 15) for keys and chunk ^
// 4 (r & 3) for values, which keeps both the key-row reads and the
// transposing value reads free of bank conflicts.  (The kernel also runs
// with W = 8, two query blocks sharing each key/value tile, and with deeper
// rings; on the 400-tile query those were slower: one workgroup a CU leaves
// the SIMDs half idle on prompts of a single query block.)
// The wave computes S^T = K Q^T (v_mfma_f32_32x32x16_bf16, M = keys,
// N = queries), so each lane holds one query's scores in registers; the online
// softmax runs in float32 (a running reference and sum per query); the unnormalised
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

constexpr int kLdsDims = 128;                   // dimensions of an LDS key or value row
constexpr int BQ = 128;
constexpr int BKV = 64;
constexpr int kRowBytes = kLdsDims * 2;         // one key or value row
constexpr int kTileBytes = BKV * kRowBytes;     // 16 KB
constexpr int kStageBytes = 2 * kTileBytes;     // keys, then values
constexpr float kLazy = 8.0f;                   // softmax reference slack (log2 units)

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// ds_read_b64_tr_b16: lane i of each 16-lane group g gets, in component j, the
// 16-bit element at (address passed by lane 16 g + 4 j + i / 4) + i % 4.
__device__ __forceinline__ v4s_t lds_read_tr16(const void* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p));
}

// LDS DMA of 16 bytes per lane from a per-lane global address into
// LDS[m0 + 16 lane] (m0 wave-uniform).
__device__ __forceinline__ void dma16v(const void* gaddr, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(gaddr) : "memory", "m0");
}

// Same, saddr form: 64-bit wave-uniform base plus a 32-bit per-lane byte
// offset.
__device__ __forceinline__ void dma16s(const void* base, uint32_t voff, uint32_t lds_addr) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b) |
                        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(ub) : "memory", "m0");
}

// wait until at most n of this wave's vector memory operations are outstanding
__device__ __forceinline__ void wait_vm(int n) {
    switch (n) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
        case 8: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
        case 16: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}

// W waves (W / 4 query blocks per pass), S ring stages, head dim HD (128 or
// 64).  With HD = 64 the tiles keep their 256-byte rows: the DMA fills only
// the head's 8 chunks of each row, and the score and output MFMAs stop at the
// head's dimensions (the other chunks are never read).
template <int W, int S, int HD, bool LIST>
__global__ void __launch_bounds__(64 * W, W == 8 ? 1 : 2)
attn_bf16_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                 const bf16_t* __restrict__ v, bf16_t* __restrict__ o,
                 const int* __restrict__ cu, int n_seq, int H, int n_prefix, float scale_log2,
                 const int2* __restrict__ list) {
    constexpr int G = W / 4;                 // query blocks per pass
    constexpr int NDMA = 32 / W;             // DMA instructions per wave per key block
    static_assert(!LIST || W == 4, "the query-block kernel runs one block per pass");
    __shared__ __align__(16) unsigned char ring[S * kStageBytes];

    int seq, head, qb_top = -1;
    if constexpr (LIST) {
        // entry blockIdx / 8: sequence, group of 8 heads, query block; the
        // head within the group is blockIdx mod 8, the XCD the workgroup runs
        // on, so one XCD runs every query block of a (sequence, head)
        const int2 it = list[blockIdx.x >> 3];
        if (it.x < 0) return;
        seq = it.x;
        head = (it.y >> 16) * 8 + (int)(blockIdx.x & 7);
        qb_top = it.y & 0xffff;
    } else {
        seq = blockIdx.x / H;
        head = blockIdx.x % H;
    }
    const int s0 = cu[seq];
    const int L = cu[seq + 1] - s0;
    const int pre = seq > 0 ? n_prefix : 0;   // logical keys before the sequence's own rows

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2;                // with W = 8: 0 the upper block of a pass, 1 the lower
    const int wq = wave & 3;                  // wave within its block
    const int h = lane >> 5;
    const int col = lane & 31;
    const int ld = H * HD;
    const size_t head_off = (size_t)head * HD;
    const uint32_t ring0 = (uint32_t)(uintptr_t)ring;

    // DMA of logical key block `blk` into ring stage slot % S: 32 instructions
    // of four 256-byte rows each (0..15 keys, 16..31 values); wave w issues
    // NDMA = 32 / W of them (the first W / 2 waves keys, the others values).
    // Lane l moves chunk position l % 16 of row 4 jj + l / 16, i.e. global
    // chunk position ^ swz.
    const bool dma_v = wave >= W / 2;
    const bf16_t* dma_src = dma_v ? v : k;
    const int dma_row_lo = lane >> 4;
    // Per-lane part of each instruction's source, for blocks that lie inside
    // the sequence's own rows: byte offset of (row, chunk) from the block's
    // first row; the wave-uniform rest goes into the scalar base.
    uint32_t dma_off[NDMA];
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
        const int jj = NDMA * (wave % (W / 2)) + i;
        const int row = 4 * jj + dma_row_lo;
        const int swz = dma_v ? 4 * (row & 3) : (row & 15);
        const int c = (lane & 15) ^ swz;
        dma_off[i] = ((uint32_t)row * (uint32_t)ld + (uint32_t)c * 8u) * 2u;
    }
    auto dma_block = [&](int blk, int slot) {
        const uint32_t sb = ring0 + (uint32_t)(slot % S) * kStageBytes + (dma_v ? kTileBytes : 0);
        const int k0 = blk * BKV;
        if (k0 >= pre && k0 + BKV <= pre + L) {
            const bf16_t* base = dma_src + (size_t)(s0 + k0 - pre) * ld + head_off;
#pragma unroll
            for (int i = 0; i < NDMA; ++i) {
                const int jj = NDMA * (wave % (W / 2)) + i;
                const int row = 4 * jj + dma_row_lo;
                const int swz = dma_v ? 4 * (row & 3) : (row & 15);
                const int c = (lane & 15) ^ swz;
                if (HD == kLdsDims || c < HD / 8) dma16s(base, dma_off[i], sb + (uint32_t)jj * 1024u);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < NDMA; ++i) {
            const int jj = NDMA * (wave % (W / 2)) + i;
            const int row = 4 * jj + dma_row_lo;
            int key = blk * BKV + row;
            key = key < pre + L ? key : pre + L - 1;
            const int grow = key < pre ? key : s0 + key - pre;
            const int swz = dma_v ? 4 * (row & 3) : (row & 15);
            const int c = (lane & 15) ^ swz;
            if (HD == kLdsDims || c < HD / 8)
                dma16v(dma_src + (size_t)grow * ld + head_off + c * 8, sb + (uint32_t)jj * 1024u);
        }
    };

    // per-lane byte offsets of the operand reads within a stage
    //   keys: row kb*32 + col, chunk 2 kk + h at (2 kk + h) ^ (col & 15)
    //   values (transposing): source lane (tg, tj, tu) passes key row
    //   4 (tg >> 1) + tj (+ 16 ks + 32 kb, + 8 for the upper half) and
    //   dimensions 16 (tg & 1) + 4 tu + 32 t: chunk (2 (tg & 1) + tu / 2) | 4 t
    //   at chunk ^ 4 tj, byte 8 (tu & 1) within it
    const int tg = lane >> 4, tj = (lane >> 2) & 3, tu = lane & 3;
    const int k_row_off = col * kRowBytes;
    const int v_off = (4 * (tg >> 1) + tj) * kRowBytes + (2 * (tg & 1) + (tu >> 1)) * 16 + 8 * (tu & 1);

    const int nqb = (L + BQ - 1) / BQ;
    const int top = LIST ? qb_top : nqb - 1;            // the first pass's upper block
    const int n_pass = LIST ? 1 : (nqb + G - 1) / G;
    // Ring position of each pass's first key block: positions run on across
    // passes, so the last block of a pass can load the next pass's first block
    // into the stage that is free by then.
    int g0 = 0;
    bool first_issued = false;
    for (int pr = 0; pr < n_pass; ++pr) {
        const int qb_hi = top - G * pr;
        const int qb = qb_hi - grp;               // -1: the lower half has no block
        const int q0 = qb >= 0 ? qb * BQ : 0;
        const int qw = q0 + wq * 32;              // first query of this wave
        const int qidx = qw + col;                // this lane's query
        const int q_eff = qidx < L ? qidx : L - 1;
        // logical position of the wave's last query, -1 when it has none
        const int wave_last = (qb >= 0 && qw < L) ? pre + ((qw + 31) < (L - 1) ? (qw + 31) : (L - 1)) : -1;

        asm volatile("s_barrier" ::: "memory");   // every wave is done with the ring
        // Q^T B-operand fragments: lane holds Q[query][16 kk + 8 h .. + 8]
        constexpr int NKK = HD / 16;             // 16-dimension steps of the score MFMAs
        constexpr int NT = HD / 32;              // 32-dimension output blocks
        bf16x8_t qf[NKK];
        {
            const bf16_t* qrow = q + (size_t)(s0 + q_eff) * ld + head_off + 8 * h;
#pragma unroll
            for (int kk = 0; kk < NKK; ++kk) qf[kk] = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * kk);
        }

        f32x16_t oacc[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[t][i] = 0.f;
        float m_run = -INFINITY;
        float l_run = 0.f;

        // key blocks of the pair: up to the end of the upper query block
        const int kv_end = pre + ((qb_hi + 1) * BQ < L ? (qb_hi + 1) * BQ : L);
        const int nkv = (kv_end + BKV - 1) / BKV;
        const int pro = nkv < S - 1 ? nkv : S - 1;
        for (int b = first_issued ? 1 : 0; b < pro; ++b) dma_block(b, g0 + b);
        const bool has_next = pr + 1 < n_pass;
        bool issued_next = false;
        // The compiler waits for the Q loads here, once per pair (with them,
        // for the ring's first blocks, issued just after); in the loop it then
        // has no load of its own outstanding, and the explicit waits below
        // keep up to two blocks in flight.
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) asm volatile("" : "+v"(qf[kk]));

        for (int b = 0; b < nkv; ++b) {
            // block b has landed (the Q loads, issued earlier, too) once at
            // most the DMA of blocks b+1, b+2 is outstanding; after the barrier
            // every wave's share has, and every wave is done with block b-1
            const int later = (nkv - 1 < b + S - 2 ? nkv - 1 : b + S - 2) - b;
            wait_vm(NDMA * later);
            asm volatile("s_barrier" ::: "memory");
            if (b + S - 1 < nkv) {
                dma_block(b + S - 1, g0 + b + S - 1);    // into the stage block b-1 used
            } else if (b == nkv - 1 && has_next) {
                dma_block(0, g0 + nkv);                  // the next pass's first block
                issued_next = true;
            }

            const int kv0 = b * BKV;
            if (kv0 <= wave_last) {
                const unsigned char* Kb = ring + ((g0 + b) % S) * kStageBytes;
                const unsigned char* Vb = Kb + kTileBytes;
                // scores for two 32-key sub-blocks; their MFMA chains interleaved
                f32x16_t s[2];
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
                for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb) {
                        const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(
                            Kb + kb * 32 * kRowBytes + k_row_off + (((2 * kk + h) ^ (col & 15)) << 4));
                        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[kb], 0, 0, 0);
                    }
                // raw scores; keys past a query are masked only in blocks that
                // cross the wave's diagonal.  The block max is taken on the raw
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
                // The reference m_run moves only when a query's block max
                // passes it by more than kLazy (log2 units); until then the
                // probabilities 2^(s scale - m_run) stay below 2^kLazy, and
                // the sums and the output need no rescaling (on most blocks
                // after the first).  The normalisation by the row sum at the
                // end is the same whatever the reference.
                const float m_blk = bmax * scale_log2;
                const float m_new = m_blk > m_run + kLazy ? m_blk : m_run;
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
                // rescale the sums only when some query's reference moved
                if (__any(m_new != m_run)) {
                    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                    l_run *= alpha;
#pragma unroll
                    for (int t = 0; t < NT; ++t)
#pragma unroll
                        for (int i = 0; i < 16; ++i) oacc[t][i] *= alpha;
                }
                l_run += rsum;
                m_run = m_new;

                // O^T += V^T P^T.  MFMA step ks of sub-block kb contracts keys
                // 16 ks + 4 h + {0..3} (slots 0..3) and 16 ks + 8 + 4 h + {0..3}
                // (slots 4..7) of lane half h: the P values this lane holds, and
                // two transposing reads of the value tile give the same keys.
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) {
                        bf16x8_t pf;
#pragma unroll
                        for (int jj = 0; jj < 8; ++jj) pf[jj] = (__bf16)sc[kb][8 * ks + jj];
                        const unsigned char* vb = Vb + (kb * 32 + 16 * ks) * kRowBytes + v_off;
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const int tsw = ((t ^ tj) << 6);   // chunk group t moved by the row's swizzle
                            const v4s_t lo = lds_read_tr16(vb + tsw);
                            const v4s_t hi = lds_read_tr16(vb + tsw + 8 * kRowBytes);
                            const u32x4_t vv = {__builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1)),
                                                __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3)),
                                                __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1)),
                                                __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3))};
                            oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv),
                                                                              pf, oacc[t], 0, 0, 0);
                        }
                    }
            }
        }

        // Output row of this lane's query: slots 4 g .. 4 g + 3 of block t are
        // dimensions 32 t + 8 g + 4 h + {0..3}.  Lanes h = 0 and 1 of a query
        // swap the 8-byte halves of each 16-dimension group pair, so that
        // each writes 16 contiguous bytes: h = 0 dimensions 32 t + 16 j + [0, 8),
        // h = 1 dimensions 32 t + 16 j + [8, 16).
        {
            const float inv = 1.0f / l_run;
            const bool store = qb >= 0 && qidx < L;
            bf16_t* orow = o + (size_t)(s0 + q_eff) * ld + head_off;
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    uint32_t a[2], b[2];
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        a[e] = (uint32_t)f32_to_bf16(oacc[t][8 * j + 2 * e] * inv) |
                               ((uint32_t)f32_to_bf16(oacc[t][8 * j + 2 * e + 1] * inv) << 16);
                        b[e] = (uint32_t)f32_to_bf16(oacc[t][8 * j + 4 + 2 * e] * inv) |
                               ((uint32_t)f32_to_bf16(oacc[t][8 * j + 4 + 2 * e + 1] * inv) << 16);
                    }
                    uint32_t r[2];
#pragma unroll
                    for (int e = 0; e < 2; ++e) r[e] = (uint32_t)__shfl_xor((int)(h ? a[e] : b[e]), 32);
                    const u32x4_t v = h ? u32x4_t{r[0], r[1], b[0], b[1]} : u32x4_t{a[0], a[1], r[0], r[1]};
                    if (store) *reinterpret_cast<u32x4_t*>(orow + t * 32 + 16 * j + 8 * h) = v;
                }
        }
        g0 += nkv;
        first_issued = issued_next;
    }   // query block pairs
}

// Work list of the query-block kernel: for each sequence s in order, for each
// group g of 8 heads, its query blocks from the last (longest) to the first,
// entry {s, (g << 16) | block}; entries past the list up to n_list: {-1, 0}.
// One workgroup; sequences 1,024 at a time, their entry counts scanned.
__global__ void __launch_bounds__(1024)
attn_worklist_kernel(const int* __restrict__ cu, int n_seq, int hs, int2* __restrict__ list, int n_list) {
    __shared__ int wsum[16];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int carry = 0;
    for (int base = 0; base < n_seq; base += 1024) {
        const int s = base + tid;
        int len = s < n_seq ? cu[s + 1] - cu[s] : 0;
        len = len > 0 ? len : 0;
        const int nqb = (len + BQ - 1) / BQ;
        const int cnt = hs * nqb;
        int incl = cnt;   // inclusive scan over the wave
#pragma unroll
        for (int sh = 1; sh < 64; sh <<= 1) {
            const int x = __shfl_up(incl, sh);
            incl += lane >= sh ? x : 0;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        int before = 0, blk = 0;
#pragma unroll
        for (int w = 0; w < 16; ++w) {
            before += w < wave ? wsum[w] : 0;
            blk += wsum[w];
        }
        const int start = carry + before + incl - cnt;
        for (int r = 0; r < cnt; ++r) {
            const int i = start + r;
            if (i < n_list) list[i] = int2{s, ((r / nqb) << 16) | (nqb - 1 - r % nqb)};
        }
        carry += blk;
        __syncthreads();   // wsum is refilled by the next round
    }
    for (int i = carry + tid; i < n_list; i += 1024) list[i] = int2{-1, 0};
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

int attention_worklist_entries(int T, int n_seq, int n_heads) {
    // sum over sequences of ceil(len / BQ) <= ceil(T / BQ) + (non-empty sequences)
    const long long e = (long long)(n_heads / 8) * ((T + BQ - 1) / BQ + (n_seq < T ? n_seq : T));
    return e < (1 << 28) ? (int)e : (1 << 28);
}

hipError_t launch_attention_worklist(const int* cu, int n_seq, int n_heads, int2* list, int n_list,
                                     hipStream_t st) {
    if (n_heads % 8 != 0 || n_heads / 8 > 0x7fff || n_list <= 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(attn_worklist_kernel, dim3(1), dim3(1024), 0, st, cu, n_seq, n_heads / 8, list, n_list);
    return hipGetLastError();
}

hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, const int* cu, int n_seq, int max_seqlen,
                                 int n_heads, int hd, int n_prefix, const int2* list, int n_list,
                                 hipStream_t st) {
    if (n_seq <= 0 || max_seqlen <= 0) return hipSuccess;
    if (hd != 64 && hd != 128) return hipErrorInvalidValue;
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    if (list != nullptr) {
        if (n_heads % 8 != 0 || n_list <= 0) return hipErrorInvalidValue;
        const dim3 grid((unsigned)n_list * 8u);
        if (hd == 128)
            hipLaunchKernelGGL((attn_bf16_kernel<4, 2, 128, true>), grid, dim3(256), 0, st, q, k, v, o, cu, n_seq,
                               n_heads, n_prefix, scale_log2, list);
        else
            hipLaunchKernelGGL((attn_bf16_kernel<4, 2, 64, true>), grid, dim3(256), 0, st, q, k, v, o, cu, n_seq,
                               n_heads, n_prefix, scale_log2, list);
        return hipGetLastError();
    }
    const long long blocks = (long long)n_seq * n_heads;
    if (hd == 128)
        hipLaunchKernelGGL((attn_bf16_kernel<4, 2, 128, false>), dim3((unsigned)blocks), dim3(256), 0, st, q, k, v,
                           o, cu, n_seq, n_heads, n_prefix, scale_log2, nullptr);
    else
        hipLaunchKernelGGL((attn_bf16_kernel<4, 2, 64, false>), dim3((unsigned)blocks), dim3(256), 0, st, q, k, v,
                           o, cu, n_seq, n_heads, n_prefix, scale_log2, nullptr);
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

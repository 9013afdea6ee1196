// Internal launchers of the Rift kernels (host side).  The C ABI in capi.hip
// validates arguments and calls these; every launcher only enqueues work.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rift {

hipError_t launch_score(const void* tokens, bool bf16, int n_tiles, int n_v, int d,
                        const void* qbank, int n_bg, int keep_count, double tau, int knn_m,
                        double* token_key, float* token_sim, double* tile_score, float* tile_u,
                        int* tile_order, int* n_keep, float* w32, int* arrivals, double* inv, float* emb,
                        double* gram, double* s_smooth, hipStream_t st);
// optional score smoothing over each tile's knn_m most similar tiles
hipError_t launch_knn_smooth(const void* tokens, bool bf16, int n_tiles, int n_v, int d,
                             const double* inv, float* emb, double* gram, const double* s_raw,
                             int m, double* s_out, hipStream_t st);

// non-finite scan: clear the flag word, then scan buffers into it (kind 0
// bfloat16, 1 float32, 2 float64; n elements)
hipError_t launch_nonfinite_clear(int* flag, hipStream_t st);
hipError_t launch_nonfinite_scan(const void* x, int kind, long long n, int* flag, hipStream_t st);

hipError_t launch_select(const double* token_key, int n_tiles, int n_v, const int* kept,
                         const int* budgets, int n_keep, int* sel_offsets, int* sel_idx,
                         long long cap, int* status, hipStream_t st);

// ctx / coffs: optional contextual rows and their per-prompt offsets (nullptr: none)
hipError_t launch_compact(const void* tokens, int elem_bytes, int n_tiles, int n_v, int d,
                          const int* kept, const int* offs, const int* sel, int n_keep,
                          const void* ctx, const int* coffs, const void* sys, int n_sys,
                          const void* qry, int n_qry, bool shared, void* packed, long long cap, int* cu,
                          int* pos_ids, int* status, hipStream_t st);

// optional merge of the remainder into contextual tokens; workspace arrays
// grp, tgt [n_keep][n_v] int, inv [n_keep][n_v] double, ok [n_keep] int
hipError_t launch_merge(const void* tokens, bool bf16, int n_tiles, int n_v, int d, const int* kept,
                        const int* offs, const int* sel, const int* coffs, int n_keep, void* ctx_rows,
                        long long ctx_cap, int* status, int* grp, int* tgt, double* inv, int* ok,
                        hipStream_t st);

// ---------------------------------------------------------------- prefill pieces
// RoPE table: tab[p * (hd/2) + j] = (cos, sin)(p * base^(-2j/hd)), p < n_pos.
hipError_t launch_rope_table(float2* tab, int n_pos, int hd, float base, hipStream_t st);

// h = RMSNorm(x) * g, one row per wave.  x is f32 (x_bf16 == false) or bf16;
// when resid != nullptr the f32 value of x is also stored there.  h is bf16
// (h_bf16) or f32.
hipError_t launch_rmsnorm(const void* x, bool x_bf16, float* resid, const void* g, bool g_bf16,
                          void* h, bool h_bf16, int rows, int d, float eps, hipStream_t st);

// bf16 MFMA GEMMs, C = A B^T (A [M][K], B rows [N][K], K contiguous).
struct QkvArgs {
    const uint16_t* a;  // h [M][d]
    const uint16_t* wq;
    const uint16_t* wk;
    const uint16_t* wv;
    uint16_t* q;  // [M][d]
    uint16_t* k;
    uint16_t* v;
    const float2* rope;  // [n_pos][hd/2]
    const int* pos;      // [M]
    int n_pos;
    int M, d;
    int hd;              // head dim: 128, or 64
};
// The GEMMs walk their output tiles from the first row block to the last, or
// with `reverse` from the last to the first.  The order changes no result; it
// decides which rows of A a GEMM reads first, and the rows its producer wrote
// last are still in the memory-side cache.
hipError_t launch_gemm_qkv_rope(const QkvArgs& a, hipStream_t st, bool reverse = false);

// resid[M][N] += A[M][K] B[N][K]^T  (attention output and FFN down projections)
hipError_t launch_gemm_resid(const uint16_t* a, const uint16_t* b, float* resid, int M, int N,
                             int K, hipStream_t st, bool reverse = false);

// out[M][F] = silu(A Wg^T) * (A Wu^T), A [M][K], Wg, Wu [F][K]
hipError_t launch_gemm_swiglu(const uint16_t* a, const uint16_t* wg, const uint16_t* wu,
                              uint16_t* out, int M, int F, int K, hipStream_t st, bool reverse = false);

// Varlen causal attention, bf16, head_dim hd (128 or 64).  q, k, v, o: [T][H*hd].
// With `list` (from launch_attention_worklist, n_list entries) one workgroup
// runs one 128-query block; without it one workgroup runs a whole sequence.
hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, const int* cu, int n_seq, int max_seqlen,
                                 int n_heads, int hd, int n_prefix, const int2* list, int n_list,
                                 hipStream_t st);
// Work list of the query-block attention for n_heads a multiple of 8 (one
// entry per sequence, group of 8 heads and query block; unused entries up to
// n_list are marked empty); n_list >= attention_worklist_entries(T, n_seq, H).
int attention_worklist_entries(int T, int n_seq, int n_heads);
hipError_t launch_attention_worklist(const int* cu, int n_seq, int n_heads, int2* list, int n_list,
                                     hipStream_t st);

// ---------------------------------------------------------------- decode (bf16)
// pos[i] = (cu[i+1] - cu[i]) + step
hipError_t launch_decode_pos(const int* cu, int n_seq, int n_prefix, int step, int* pos, hipStream_t st);
// rows of k, v [n_seq][d] into slot `step` of kc, vc [n_seq][max_new][d]
hipError_t launch_kv_append(const uint16_t* k, const uint16_t* v, uint16_t* kc, uint16_t* vc, int n_seq, int d,
                            int max_new, int step, hipStream_t st);
// one query per prompt over its prefill keys kp/vp [T][H*128] and slots 0..step of kn/vn
hipError_t launch_decode_attention(const uint16_t* q, const uint16_t* kp, const uint16_t* vp, const uint16_t* kn,
                                   const uint16_t* vn, const int* cu, int n_seq, int T, int n_prefix, int n_heads,
                                   int hd, int max_keys, int max_new, int step, uint16_t* o, hipStream_t st);

// Decode-shaped GEMMs (few rows): K split into S chunks (S from N and K only),
// float32 partials part[S][M][N] of A [M][K] times the weight regions b0|b1|b2
// (each [nr][K], N = regions * nr), then reduce kernels that add the partials
// in chunk order and finish the layer's elementwise work.
int skinny_splits(int N, int K);
bool skinny_supported(int N, int K, int nr);
bool skinny_norm_supported(int d);
hipError_t launch_skinny_gemm(const uint16_t* a, const uint16_t* b0, const uint16_t* b1, const uint16_t* b2,
                              int nr, int M, int N, int K, float* part, hipStream_t st);
// x += sum of partials [S][M][d]; with h, h = bf16(RMSNorm(x) * g)
hipError_t launch_skinny_resid_norm(const float* part, int S, int M, int d, float* x, const uint16_t* g,
                                    uint16_t* h, float eps, hipStream_t st);
// q to q[M][d], k and v to slot `step` of kc, vc [M][max_new][d], RoPE at
// pos[m] over heads of hd (128 or 64) dimensions
hipError_t launch_skinny_qkv(const float* part, int S, int M, int d, int hd, const float2* rope, const int* pos,
                             int n_pos, uint16_t* q, uint16_t* kc, uint16_t* vc, int max_new, int step,
                             hipStream_t st);
// a[M][F] = silu(gate) * up
hipError_t launch_skinny_swiglu(const float* part, int S, int M, int F, uint16_t* a, hipStream_t st);

// ---------------------------------------------------------------- f32 path
// C[M][N] = A[M][K] B[N][K]^T (+ C when accumulate)
hipError_t launch_gemm_f32(const float* a, const float* b, float* c, int M, int N, int K,
                           bool accumulate, hipStream_t st);
// in-place rotate-half RoPE on x [M][H*hd] (f32)
hipError_t launch_rope_apply_f32(float* x, const float2* rope, const int* pos, int n_pos, int M,
                                 int n_heads, int hd, hipStream_t st);
// a[M][F] = silu(g) * u  (f32, separate gate/up buffers; a may alias g)
hipError_t launch_swiglu_f32(const float* g, const float* u, float* a, long long n,
                             hipStream_t st);
hipError_t launch_attention_f32(const float* q, const float* k, const float* v, float* o,
                                const int* cu, int n_seq, int max_seqlen, int n_heads, int hd,
                                int n_prefix, hipStream_t st);
// elementwise widening copy of a [rows][d] matrix into f32
hipError_t launch_to_f32(const void* x, bool x_bf16, float* out, long long n, hipStream_t st);
// copy f32 -> storage type (for KV-cache output of the f32 path / bf16 keys)
hipError_t launch_copy_f32(const float* x, float* out, long long n, hipStream_t st);

// kernels that need more than the default dynamic LDS are registered here
hipError_t init_kernel_attributes();

}  // namespace rift

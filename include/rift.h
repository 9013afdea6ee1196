/*
 * rift.h -- C ABI of the Rift hot path on AMD Instinct MI355X (gfx950).
 *
 * The four stages of one scene-query, in the order the paper applies them:
 *   1. rift_score_tiles    query-conditioned tile relevance and pruning
 *                          (Sec. 2.3 Stage 1, Eq. 1, Listing 1, App. B Step 3)
 *   2. rift_select_tokens  per-tile dominant-token selection under elastic
 *                          budgets (Sec. 2.3 Stage 2)
 *   (optional) rift_merge_context: the non-selected tokens of each kept
 *                          tile merged into contextual tokens (VisionZip's
 *                          merge of the remaining tokens, Sec. 2.3 Stage 2)
 *   3. rift_compact        packing of each retained tile's prompt into one
 *                          varlen batch (each tile is its own VLM call,
 *                          Sec. 2.3 Stage 2 and App. B Step 5)
 *   4. rift_prefill        LLaMA-7B-shaped decoder prefill of the packed
 *                          prompts (Sec. 2.1; LLaVA-1.5-7B, Sec. 3)
 * plus the host-side budget assignment rift_assign_budgets, and
 *   5. rift_decode_step    one generated token per prompt after the prefill,
 *                          reusing the prefill's key/value cache (the answers
 *                          are a few words, Sec. 2.2).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless the comment says [host].
 *   - The caller owns every buffer (inputs, outputs, workspace).  The library
 *     allocates no device memory and keeps no per-call state.
 *   - Calls are asynchronous and ordered on `stream` (a hipStream_t; NULL is
 *     the null stream).  The library never synchronises the device.
 *   - Arguments are validated on the host first; on failure a call returns a
 *     non-OK status and enqueues nothing.  Errors that only the device can see
 *     (a budget out of range, an index out of bounds) are reported through a
 *     device status word, and the kernels then write nothing out of bounds.
 *   - Storage types: RIFT_BF16 (bfloat16) or RIFT_F32.  One dtype is shared by
 *     tokens, query bank, system/query embeddings and weights of a call chain.
 *   - Debug mode (environment variable RIFT_DEBUG=1 when the library is first
 *     used, or rift_set_debug): rift_score_tiles, rift_select_tokens and
 *     rift_prefill first scan their floating-point inputs on the device for
 *     NaN or infinity, wait for the scan (the one place the library
 *     synchronises its stream) and return RIFT_ERR_NONFINITE, with nothing
 *     else enqueued, when one is found.  Index bounds are checked on the device
 *     in every mode (the status words of select and compact).
 */
#ifndef RIFT_H
#define RIFT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RIFT_ABI_VERSION 7

#if defined(__GNUC__) || defined(__clang__)
#define RIFT_API __attribute__((visibility("default")))
#else
#define RIFT_API
#endif

typedef enum {
    RIFT_OK = 0,
    RIFT_ERR_NULL = 1,        /* a required pointer is NULL                       */
    RIFT_ERR_SHAPE = 2,       /* a size breaks the shape rules of the call        */
    RIFT_ERR_DTYPE = 3,       /* unknown or mismatched storage type               */
    RIFT_ERR_BUDGET = 4,      /* budget, level or tier out of range               */
    RIFT_ERR_WORKSPACE = 5,   /* workspace too small or not 256-byte aligned      */
    RIFT_ERR_HIP = 6,         /* a HIP runtime call or a kernel launch failed     */
    RIFT_ERR_NONFINITE = 7,   /* a floating-point input holds NaN or infinity     */
    RIFT_ERR_UNSUPPORTED = 8  /* valid request outside what this library implements */
} rift_status;

typedef enum { RIFT_F32 = 0, RIFT_BF16 = 1 } rift_dtype;

typedef void* rift_stream; /* hipStream_t */

/* ABI version of the loaded library (RIFT_ABI_VERSION it was built with). */
RIFT_API int32_t rift_abi_version(void);

/* Static text for a status code. */
RIFT_API const char* rift_status_string(rift_status s);

/*
 * rift_set_debug -- switch the debug mode of the process on (on != 0) or off;
 * returns the previous setting (1 or 0).  The first use of the library reads
 * the initial setting from RIFT_DEBUG.  Calls that are already running keep
 * the mode they started with.
 */
RIFT_API int32_t rift_set_debug(int32_t on);

/*
 * rift_check_finite -- device check that x holds no NaN or infinity, the
 * check the debug mode runs on the inputs (usable on its own, e.g. on weights
 * once after loading them).  Asynchronous like every call.
 * x       [count] dt, any alignment
 * status  [1] i32 out  0, or RIFT_ERR_NONFINITE
 * Errors: RIFT_ERR_NULL (status, or x with count > 0), RIFT_ERR_DTYPE,
 * RIFT_ERR_SHAPE (count < 0).
 */
RIFT_API rift_status rift_check_finite(const void* x, rift_dtype dt, int64_t count, int32_t* status,
                                       rift_stream stream);

/* ------------------------------------------------------------------ Stage 1 */

/* Workspace bytes rift_score_tiles needs for a scene of this shape and knn_m
 * (0 if the call does not smooth; a smoothing call needs about
 * 8 n_tiles (n_v + n_tiles) + 4 n_tiles d bytes more). */
RIFT_API size_t rift_score_workspace_size(int32_t n_tiles, int32_t n_v, int32_t d, int32_t knn_m);

/*
 * rift_score_tiles -- Stage 1 of Sec. 2.3: Eq. 1 background-margin relevance,
 * per-scene min-max normalisation and retention (Listing 1; App. B Step 3).
 *
 * tokens      [n_tiles][n_v][d] dt   vision tokens of every tile (row-major)
 * query_bank  [1 + n_bg][d]     dt   row 0 = query object t, rows 1..n_bg =
 *                                    background phrases B_j; unit norm before
 *                                    rounding to dt (the rounded values count)
 * keep_count  > 0: keep the top min(keep_count, n_tiles) tiles by score;
 *             == 0: keep every tile with u >= tau (tau is compared in float64)
 * knn_m       0: no smoothing.  > 0: before normalisation each tile score is
 *             averaged with the scores of its knn_m most visually similar tiles
 *             (the optional smoothing of Listing 1's note and App. B Step 3,
 *             which the paper runs with six neighbours).  The tile embedding
 *             is the float32-rounded sum of its unit tokens, accumulated over
 *             tokens in ascending order with
 *             each product and sum rounded on its own; similarity is the cosine
 *             of the canonical dot products; neighbours are the knn_m (at most
 *             n_tiles - 1) largest over the other tiles, ties to the lower id;
 *             s' = (s + neighbour scores in neighbour order) / (1 + knn_m).
 * Outputs (all device):
 * token_key   [n_tiles*n_v] f64  per-token margin of the unit token,
 *                                r = (x.w)/|x| with w = t - mean_j B_j rounded
 *                                to f32 (Eq. 1 is linear in the tile
 *                                embedding); a fixed float64 summation order
 *                                makes r reproducible bit for bit: elements in
 *                                8-wide granules, granule g into accumulator
 *                                g mod 4, ascending, then (a0+a2)+(a1+a3).
 *                                All-zero token -> +0.
 * token_sim   [n_tiles*n_v][1+n_bg] f32 cosine of each token to t and each
 *                                B_j (MFMA relevance GEMM), or NULL to skip
 * tile_score  [n_tiles] f64      s_i = mean of the tile's token margins: 64
 *                                strided partial sums then a halving tree,
 *                                divided by n_v; the smoothed score when
 *                                knn_m > 0 (the score u and the order use)
 * tile_u      [n_tiles] f32      (s - min s)/(max s - min s) in float64,
 *                                rounded to f32; all 1 when max == min
 * tile_order  [n_tiles] i32      tile ids by (s descending, id ascending); the
 *                                first *n_keep entries are the kept tiles
 * n_keep      [1] i32            number of kept tiles
 * Shape rules: 1 <= n_tiles <= 4096, 1 <= n_v <= 1024, d % 32 == 0,
 * 32 <= d <= 16384, 0 <= n_bg <= 15, 0 <= tau (any double), knn_m >= 0.
 * workspace   >= rift_score_workspace_size(...) bytes, 256-byte aligned.
 */
RIFT_API rift_status rift_score_tiles(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                             int32_t d, const void* query_bank, int32_t n_bg,
                             int32_t keep_count, double tau, int32_t knn_m,
                             double* token_key, float* token_sim, double* tile_score,
                             float* tile_u, int32_t* tile_order, int32_t* n_keep,
                             void* workspace, size_t ws_bytes, rift_stream stream);

/*
 * rift_score_tiles_noalloc -- rift_score_tiles without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation).  Same arguments, outputs,
 * shape rules and errors as rift_score_tiles; the workspace is a static
 * device array of RIFT_SCORE_SCRATCH_BYTES that the library holds on each GPU
 * it runs on until the process ends.  The call runs on the current device;
 * `stream` must belong to it.  Nothing is allocated (no hipMalloc, no
 * allocating library routine).
 * Limit: calls whose rift_score_workspace_size(n_tiles, n_v, d, knn_m)
 * exceeds RIFT_SCORE_SCRATCH_BYTES return RIFT_ERR_WORKSPACE and enqueue
 * nothing (every call without smoothing fits; with smoothing, e.g. 400 tiles
 * x 576 tokens at d = 4096 needs about 9.7 MB).
 * Every call on a GPU shares that GPU's array: calls that overlap in time on
 * one GPU (different streams or threads, or another host thread's call that
 * has not finished) race on it and must be ordered by the caller.  Nothing in
 * the array needs to start at zero: every word a call reads, the same call
 * writes first.
 */
#define RIFT_SCORE_SCRATCH_BYTES (16u << 20)
RIFT_API rift_status rift_score_tiles_noalloc(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                                              int32_t d, const void* query_bank, int32_t n_bg,
                                              int32_t keep_count, double tau, int32_t knn_m,
                                              double* token_key, float* token_sim, double* tile_score,
                                              float* tile_u, int32_t* tile_order, int32_t* n_keep,
                                              rift_stream stream);

/* ------------------------------------------------------------------ Stage 2 */

/*
 * rift_assign_budgets -- [host only] per-tile token budgets from the discrete
 * set C of Sec. 2.3 Stage 2, assigned by score rank: the kept tile of rank rho
 * gets levels[j] for the tier j containing rho; tier j < n_levels-1 holds
 * floor(n_keep * tier_num[j] / tier_den) tiles and the last tier the rest.
 * levels    [host] n_levels budgets, strictly descending, each in [1, n_v]
 * tier_num  [host] n_levels-1 numerators (>= 0; sum <= tier_den), or NULL for
 *           the default {1, 3, 4}/16 (requires n_levels == 4)
 * budgets   [host] out [n_keep];  total [host] out: sum of budgets (may be NULL)
 */
RIFT_API rift_status rift_assign_budgets(int32_t n_keep, int32_t n_v, const int32_t* levels,
                                int32_t n_levels, const int32_t* tier_num, int32_t tier_den,
                                int32_t* budgets, int64_t* total);

/*
 * rift_assign_budgets_utility -- [host only] the elastic-prefill policy of
 * Eq. 2 (Sec. 2.3 Stage 2): for each kept tile the budget c of the candidate
 * set maximising U(c) = p a+_c + (1 - p) a-_c - lambda E_c, where p is the
 * probability that the tile holds the object (the paper's trained predictor is
 * outside this library: the caller supplies p), a+_c / a-_c the profiled answer
 * accuracy with / without the object and E_c the profiled energy of budget c.
 * U is evaluated in float64 as ((p a+) + ((1 - p) a-)) - (lambda E), each
 * operation rounded on its own; ties go to the smaller budget.
 * levels     [host] n_c candidate budgets, each in [1, n_v], any order
 * alpha_pos, alpha_neg, energy  [host] n_c finite values, same order
 * lambda     finite accuracy-energy trade-off
 * p          [host] n_keep values in [0, 1] (f32)
 * budgets    [host] out [n_keep];  total [host] out: sum of budgets (may be NULL)
 * Errors: RIFT_ERR_NULL, RIFT_ERR_SHAPE (n_keep < 0, n_v < 1, n_c outside
 * [1, 64]), RIFT_ERR_BUDGET (a value out of range or not finite).
 */
RIFT_API rift_status rift_assign_budgets_utility(int32_t n_keep, int32_t n_v, int32_t n_c,
                                        const int32_t* levels, const double* alpha_pos,
                                        const double* alpha_neg, const double* energy,
                                        double lambda, const float* p, int32_t* budgets,
                                        int64_t* total);

/*
 * rift_select_tokens -- VisionZip-style dominant-token retention (Sec. 2.3
 * Stage 2) under per-tile budgets: for kept tile rho (id kept_tiles[rho]), keep
 * the budgets[rho] tokens with the largest token_key, ties to the lower token
 * index, and emit their indices in ascending order.
 * token_key   [n_tiles*n_v] f64   from rift_score_tiles
 * kept_tiles  [n_keep] i32        tile ids (e.g. the head of tile_order)
 * budgets     [n_keep] i32        each in [0, n_v]
 * sel_offsets [n_keep+1] i32 out  exclusive prefix sums of budgets
 * sel_idx     [sel_capacity] i32 out   the kept indices, tile after tile
 * status      [1] i32 out         0, or RIFT_ERR_BUDGET if a budget is out of
 *                                 range, a tile id is out of range or the total
 *                                 exceeds sel_capacity (then nothing is written
 *                                 to sel_idx and all offsets are 0)
 * Shape rules: 1 <= n_v <= 1024, n_tiles >= 1, n_tiles * n_v <= INT32_MAX,
 *              0 <= n_keep <= n_tiles, sel_capacity <= INT32_MAX.
 */
RIFT_API rift_status rift_select_tokens(const double* token_key, int32_t n_tiles, int32_t n_v,
                               const int32_t* kept_tiles, const int32_t* budgets,
                               int32_t n_keep, int32_t* sel_offsets, int32_t* sel_idx,
                               int64_t sel_capacity, int32_t* status, rift_stream stream);

/*
 * rift_split_budgets -- [host] split each budget c into dominant and
 * contextual tokens for rift_merge_context: k_c = min(floor(c num / den),
 * n_v - c), k_d = c - k_c (num/den = 10/64 gives VisionZip's 54 + 10 at 64
 * tokens; at the full budget k_c = 0).
 * budgets [host] [n_keep] in [0, n_v];  dominant, context [host] out [n_keep]
 * Errors: RIFT_ERR_NULL, RIFT_ERR_SHAPE (n_keep < 0, n_v < 1, num < 0,
 * den < 1, num > den), RIFT_ERR_BUDGET (a budget out of range).
 */
RIFT_API rift_status rift_split_budgets(int32_t n_keep, int32_t n_v, const int32_t* budgets, int32_t num,
                                        int32_t den, int32_t* dominant, int32_t* context);

/* Workspace bytes of rift_merge_context (256-byte aligned). */
RIFT_API size_t rift_merge_workspace_size(int32_t n_keep, int32_t n_v);

/*
 * rift_merge_context -- merge each kept tile's non-selected tokens into
 * contextual tokens (Sec. 2.3 Stage 2: VisionZip keeps the dominant tokens and
 * merges the remainder; the scheme is VisionZip's).  For kept tile rho with
 * dominant tokens sel_idx[sel_offsets[rho] .. sel_offsets[rho + 1]) (from
 * rift_select_tokens with the dominant budgets) and
 * k_c = ctx_offsets[rho + 1] - ctx_offsets[rho]: the remainder R is the other
 * tokens in ascending order; target j is R[floor(j |R| / k_c)]; every other
 * token of R joins the target j of largest cdot(x_r, x_j) / |x_j| (the cosine
 * up to 1/|x_r|, with cdot the float64 dot product in the order described for
 * token_key and |x_j| = sqrt(cdot(x_j, x_j)), a zero token scoring 0), ties to
 * the lower j; contextual row ctx_offsets[rho] + j is the float64 sum of the
 * group (target and members) in ascending token order over the group size,
 * rounded to float32 and then to dt.
 * tokens       [n_tiles][n_v][d] dt
 * kept_tiles, sel_offsets, sel_idx   as for rift_compact (the dominant tokens;
 *              distinct, any order)
 * ctx_offsets  [n_keep+1] i32       prefix sums of k_c (k_c <= n_v - k_d)
 * ctx_rows     [ctx_capacity][d] dt out
 * status       [1] i32 out  0, or RIFT_ERR_SHAPE if an offset, count or tile
 *              id is out of range, ctx_offsets[n_keep] > ctx_capacity, or a
 *              dominant index is out of range or repeated (that tile's rows are
 *              then not written)
 * workspace    >= rift_merge_workspace_size(n_keep, n_v) bytes, 256-aligned
 * Shape rules: d % 32 == 0, 32 <= d <= 16384, 1 <= n_v <= 1024,
 *              0 <= n_keep <= 65535, 0 <= ctx_capacity <= 2^24.
 */
RIFT_API rift_status rift_merge_context(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                                        int32_t d, const int32_t* kept_tiles, const int32_t* sel_offsets,
                                        const int32_t* sel_idx, const int32_t* ctx_offsets, int32_t n_keep,
                                        void* ctx_rows, int64_t ctx_capacity, int32_t* status,
                                        void* workspace, size_t ws_bytes, rift_stream stream);

/*
 * rift_compact -- pack every kept tile's prompt [n_sys system rows | selected
 * vision rows of the tile, ascending | contextual rows of the tile (optional)
 * | n_qry query rows] into one varlen batch.
 * shared_prefix 0: every prompt holds its own copy of the system rows.
 *              1: the system rows, identical in every prompt, are written once
 *              at rows [0, n_sys) as sequence 0 and prompt i holds only its
 *              rows after them, positions n_sys onwards; rift_prefill and
 *              rift_decode_step then take n_prefix = n_sys.  Under causal
 *              attention the prefix's states do not depend on what follows,
 *              so the prefill's results are those of the unshared layout.
 * tokens   [n_tiles][n_v][d] dt;  sys_emb [n_sys][d] dt;  qry_emb [n_qry][d] dt
 * kept_tiles, sel_offsets, sel_idx as produced for rift_select_tokens
 * ctx_rows, ctx_offsets   optional (both NULL: none): rows of rift_merge_context
 *              and their prefix sums [n_keep+1] per kept tile
 * packed       [packed_rows][d] dt out, total rows
 *              T = n_keep*(n_sys+n_qry) + sel_offsets[n_keep] (+ ctx_offsets[n_keep]),
 *              or with shared_prefix n_sys + n_keep*n_qry + sel_offsets[n_keep]
 *              (+ ctx_offsets[n_keep]); must be <= packed_rows
 * cu_seqlens   [n_keep+1] i32 out  prefix sums of sequence lengths ([n_keep+2]
 *              with shared_prefix: 0, n_sys, then the prompts' ends)
 * position_ids [packed_rows] i32 out  0..L-1 within each sequence (a prompt
 *              after a shared prefix: n_sys..n_sys+L-1)
 * status       [1] i32 out  0, or RIFT_ERR_SHAPE if a tile id or selected index is
 *              out of range, a budget (sel_offsets step) is outside [0, n_v], a
 *              ctx_offsets step is negative, a first offset is not 0 or
 *              T > packed_rows; a bad first offset or total stops every row
 *              from being written, a bad tile id or budget the rows of that
 *              prompt (and of any prompt whose offsets reach past the last
 *              offset), a bad selected index only its own row.  sel_idx must
 *              hold sel_offsets[n_keep] entries and ctx_rows ctx_offsets[n_keep]
 *              rows.
 * Shape rules: d * sizeof(dt) % 16 == 0; n_sys, n_qry >= 0; 0 <= n_keep <= 65535;
 *              packed_rows <= 2^25 (two waves per packed row); shared_prefix
 *              0 or 1.
 */
RIFT_API rift_status rift_compact(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                         int32_t d, const int32_t* kept_tiles, const int32_t* sel_offsets,
                         const int32_t* sel_idx, int32_t n_keep, const void* ctx_rows,
                         const int32_t* ctx_offsets, const void* sys_emb, int32_t n_sys,
                         const void* qry_emb, int32_t n_qry, int32_t shared_prefix, void* packed,
                         int64_t packed_rows, int32_t* cu_seqlens, int32_t* position_ids,
                         int32_t* status, rift_stream stream);

/* ------------------------------------------------------------------ prefill */

/* Weights of one decoder layer, nn.Linear layout [out][in], storage type
 * cfg->dt: wq, wk, wv, wo [d][d]; w_gate, w_up [ffn][d]; w_down [d][ffn];
 * RMSNorm gains g_attn, g_ffn [d]. */
typedef struct {
    const void* wq;
    const void* wk;
    const void* wv;
    const void* wo;
    const void* w_gate;
    const void* w_up;
    const void* w_down;
    const void* g_attn;
    const void* g_ffn;
} rift_layer_weights;

typedef struct {
    int32_t d;          /* hidden size                       */
    int32_t n_heads;    /* attention heads (no grouped KV)   */
    int32_t head_dim;   /* n_heads * head_dim == d           */
    int32_t ffn;        /* SwiGLU inner size                 */
    int32_t n_layers;
    float rms_eps;      /* RMSNorm epsilon                   */
    float rope_base;    /* rotary base (10000 for LLaMA)     */
    rift_dtype dt;      /* storage type of weights and activations */
} rift_model_cfg;

/* Workspace bytes rift_prefill needs for this model and batch. */
RIFT_API size_t rift_prefill_workspace_size(const rift_model_cfg* cfg, int32_t total_tokens,
                                   int32_t max_seqlen);

/*
 * rift_prefill -- prefill of n_seq independent prompts packed back to back
 * (Sec. 2.1: prefill reads the whole input and builds the KV cache; each
 * retained tile is its own call, Sec. 2.3).  Per layer, on each sequence:
 *   h = RMSNorm(x) g_attn;  q,k,v = h Wq^T, h Wk^T, h Wv^T;
 *   rotate-half RoPE on q, k (angle pos * base^(-2j/head_dim));
 *   causal softmax attention within the sequence, scale 1/sqrt(head_dim);
 *   x += o Wo^T;  h2 = RMSNorm(x) g_ffn;  x += (silu(h2 Wg^T) * (h2 Wu^T)) Wd^T.
 * cfg, layers  [host] model shape and n_layers weight sets
 * x_in         [total_tokens][d]: packed prompt tokens in cfg->dt, or, with
 *              x_dt == RIFT_F32, a float32 residual stream (e.g. the output of
 *              an earlier call); may alias hidden_out when x_dt == RIFT_F32
 * cu_seqlens   [n_seq+1] i32, cu_seqlens[0] = 0, non-decreasing, last =
 *              total_tokens, every length <= max_seqlen
 * position_ids [total_tokens] i32, each in [0, max_seqlen)  (values outside
 *              are clamped)
 * n_prefix     0, or the length of a prefix shared by every prompt: sequence 0
 *              is then rows [0, n_prefix) (cu_seqlens[1] == n_prefix) and each
 *              other sequence holds only its rows after the prefix (positions
 *              from n_prefix) and attends to the prefix rows first, exactly as
 *              if they were packed in front of it (rift_compact with
 *              shared_prefix); max_seqlen bounds n_prefix + each length.
 * hidden_out   [total_tokens][d] f32 out: residual stream after the last layer
 *              (no final norm, no vocabulary projection)
 * kv_cache     optional out [n_layers][2][total_tokens][d] cfg->dt: per layer
 *              the rotated keys, then the values; NULL to skip
 * events       optional [host] array of 10 * n_layers hipEvent_t (created by the
 *              caller), or NULL.  For benchmarks: events[10 l + 2 g] and
 *              events[10 l + 2 g + 1] are recorded on `stream` right before and
 *              after stage g of layer l -- g = 0 QKV projection (+RoPE),
 *              1 attention, 2 output projection, 3 gate/up projection (+SwiGLU),
 *              4 down projection.  A NULL entry is skipped (each recorded
 *              event adds a marker between kernels, so a benchmark records only
 *              the pairs it needs).
 * Implemented: bf16 with head_dim in {64, 128}, d % 256 == 0, ffn % 128 == 0;
 *              f32 with head_dim in {64, 128}, d % 64 == 0, ffn % 16 == 0;
 *              anything else returns RIFT_ERR_UNSUPPORTED.
 * Shape rules: 1 <= max_seqlen <= 65536, total_tokens >= 0, n_seq >= 0;
 *              0 <= n_prefix <= min(total_tokens, max_seqlen), n_seq >= 1 when
 *              n_prefix > 0.
 */
RIFT_API rift_status rift_prefill(const rift_model_cfg* cfg, const rift_layer_weights* layers,
                         const void* x_in, rift_dtype x_dt, const int32_t* cu_seqlens,
                         const int32_t* position_ids, int32_t n_seq, int32_t total_tokens,
                         int32_t max_seqlen, int32_t n_prefix, float* hidden_out, void* kv_cache,
                         void* workspace, size_t ws_bytes, void* const* events,
                         rift_stream stream);

/*
 * rift_decode_workspace_size -- bytes of workspace for rift_decode_step.
 */
RIFT_API size_t rift_decode_workspace_size(const rift_model_cfg* cfg, int32_t n_seq, int32_t max_seqlen,
                                           int32_t max_new);

/*
 * rift_decode_step -- one generated token per prompt after rift_prefill: the
 * token `step` of prompt i (input embedding row i of x_new) sits at position
 * L_i + step, L_i = cu_seqlens[i+1] - cu_seqlens[i], and attends causally to
 * the prompt's keys and values (kv_cache, as rift_prefill wrote it for these
 * cu_seqlens) and to those of the prompt's tokens 0..step, which this call and
 * the earlier steps keep in kv_new.  Same decoder layers as rift_prefill;
 * bfloat16 models only.  Decode attention keeps scores and probabilities in
 * float32 (the prefill rounds probabilities to bf16 for its MFMA).
 * x_new       [n_seq][d] bf16   input embeddings of this step's tokens
 * cu_seqlens  [n_seq+1] i32     the prefill's prompt offsets ([n_seq+2] with
 *             n_prefix > 0: the prefill's sequence 0 is the shared prefix and
 *             prompt i is its sequence i+1; its keys are the n_prefix prefix
 *             rows, then its own rows, and L_i counts both)
 * kv_cache    [n_layers][2][total_tokens][d] bf16 (rift_prefill's kv_cache)
 * kv_new      [n_layers][2][n_seq][max_new][d] bf16: slot `step` is written,
 *             slots < step are read (caller-owned, kept across steps)
 * max_seqlen  >= every L_i (positions up to max_seqlen + max_new - 1)
 * hidden_out  [n_seq][d] f32 out  residual stream of the new tokens after the
 *             last layer (before any final norm)
 * Shape rules: 0 <= step < max_new, max_seqlen + max_new <= 16384,
 * 0 <= n_prefix <= min(total_tokens, max_seqlen); the model rules of
 * rift_prefill.  Errors: RIFT_ERR_UNSUPPORTED for float32 models.
 */
RIFT_API rift_status rift_decode_step(const rift_model_cfg* cfg, const rift_layer_weights* layers,
                                      const void* x_new, const int32_t* cu_seqlens, int32_t n_seq,
                                      int32_t total_tokens, int32_t max_seqlen, int32_t n_prefix,
                                      const void* kv_cache, void* kv_new, int32_t max_new, int32_t step,
                                      float* hidden_out, void* workspace, size_t ws_bytes,
                                      rift_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* RIFT_H */

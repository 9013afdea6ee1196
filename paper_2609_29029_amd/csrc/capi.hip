// C ABI of the Rift hot path: argument validation, workspace carving and
// kernel launches.  Nothing here allocates device memory; only the debug mode
// synchronises (to read the result of its input scan).
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <cmath>

#include <mutex>

#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

std::once_flag g_init_flag;
hipError_t g_init_err = hipSuccess;

}  // namespace

// score_tiles_kernel is defined in score.hip; its LDS need grows with d.
hipError_t score_init_attributes();

hipError_t init_kernel_attributes() {
    std::call_once(g_init_flag, [] {
        g_init_err = score_init_attributes();
    });
    return g_init_err;
}

}  // namespace rift

using namespace rift;

namespace {

constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

inline bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & (kAlign - 1)) != 0; }

inline size_t dt_bytes(rift_dtype dt) { return dt == RIFT_BF16 ? 2 : 4; }

// A caller may pass any integer as an enum: its first inspection reads the
// bits (loading an enum outside its range would be undefined behaviour).
template <typename E>
inline int enum_bits(const E& e) {
    int v = 0;
    memcpy(&v, &e, sizeof v);
    return v;
}

inline bool dt_valid(const rift_dtype& dt) {
    const int v = enum_bits(dt);
    return v == (int)RIFT_BF16 || v == (int)RIFT_F32;
}

inline rift_status hip_status(hipError_t e) { return e == hipSuccess ? RIFT_OK : RIFT_ERR_HIP; }

// debug mode: -1 until first read from RIFT_DEBUG
std::atomic<int> g_debug{-1};

bool debug_on() {
    int v = g_debug.load(std::memory_order_relaxed);
    if (v < 0) {
        const char* e = getenv("RIFT_DEBUG");
        const int want = (e != nullptr && e[0] == '1') ? 1 : 0;
        int expected = -1;
        g_debug.compare_exchange_strong(expected, want);
        v = g_debug.load(std::memory_order_relaxed);
    }
    return v == 1;
}

// A floating-point input of a debug-mode check: elements and kind (0 bfloat16,
// 1 float32, 2 float64).
struct DebugInput {
    const void* x;
    int kind;
    long long n;
};

// Scan the inputs into flag (device) and wait for the answer.
rift_status debug_scan(const DebugInput* in, int count, int* flag, hipStream_t st) {
    if (launch_nonfinite_clear(flag, st) != hipSuccess) return RIFT_ERR_HIP;
    for (int i = 0; i < count; ++i)
        if (launch_nonfinite_scan(in[i].x, in[i].kind, in[i].n, flag, st) != hipSuccess) return RIFT_ERR_HIP;
    int h = 0;
    if (hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return RIFT_ERR_HIP;
    return h == (int)RIFT_ERR_NONFINITE ? RIFT_ERR_NONFINITE : RIFT_OK;
}

inline int dt_kind(rift_dtype dt) { return dt == RIFT_BF16 ? 0 : 1; }

struct PrefillLayout {
    size_t rope, h, q, k, v, a, gate2, alist, dbg, total;
};

// Entries of the query-block attention's work list the workspace holds (any
// number of sequences; 0 where that kernel does not run).
int64_t attention_list_capacity(const rift_model_cfg& c, int64_t T) {
    if (c.dt != RIFT_BF16 || c.n_heads % 8 != 0 || T <= 0) return 0;
    return attention_worklist_entries((int)T, (int)T, c.n_heads);
}

PrefillLayout prefill_layout(const rift_model_cfg& c, int64_t T, int64_t P) {
    PrefillLayout L{};
    const size_t e = dt_bytes(c.dt);
    size_t off = 0;
    L.rope = off;
    off += align_up((size_t)P * (size_t)(c.head_dim / 2) * sizeof(float2));
    L.h = off;
    off += align_up((size_t)T * c.d * e);
    L.q = off;
    off += align_up((size_t)T * c.d * e);
    L.k = off;
    off += align_up((size_t)T * c.d * e);
    L.v = off;
    off += align_up((size_t)T * c.d * e);
    L.a = off;
    off += align_up((size_t)T * c.ffn * e);
    L.gate2 = off;
    if (c.dt == RIFT_F32) off += align_up((size_t)T * c.ffn * e);
    L.alist = off;
    off += align_up((size_t)attention_list_capacity(c, T) * sizeof(int2));
    L.dbg = off;   // debug mode: flag word of the input scan
    off += kAlign;
    L.total = off;
    return L;
}

rift_status check_cfg(const rift_model_cfg* cfg) {
    if (cfg == nullptr) return RIFT_ERR_NULL;
    if (!dt_valid(cfg->dt)) return RIFT_ERR_DTYPE;
    if (cfg->d <= 0 || cfg->n_heads <= 0 || cfg->head_dim <= 0 || cfg->ffn <= 0 ||
        cfg->n_layers < 0 || (int64_t)cfg->n_heads * cfg->head_dim != cfg->d)
        return RIFT_ERR_SHAPE;
    if (!(cfg->rms_eps >= 0.0f) || !(cfg->rope_base > 0.0f)) return RIFT_ERR_SHAPE;
    if (cfg->dt == RIFT_BF16) {
        if ((cfg->head_dim != 64 && cfg->head_dim != 128) || cfg->d % 256 != 0 || cfg->ffn % 128 != 0)
            return RIFT_ERR_UNSUPPORTED;
        if ((uint64_t)cfg->d * cfg->ffn >= (1ull << 31)) return RIFT_ERR_UNSUPPORTED;
    } else {
        if ((cfg->head_dim != 64 && cfg->head_dim != 128) || cfg->d % 64 != 0 || cfg->ffn % 16 != 0)
            return RIFT_ERR_UNSUPPORTED;
    }
    return RIFT_OK;
}

}  // namespace

extern "C" {

int32_t rift_abi_version(void) { return RIFT_ABI_VERSION; }

const char* rift_status_string(rift_status s) {
    switch (enum_bits(s)) {
        case RIFT_OK: return "ok";
        case RIFT_ERR_NULL: return "a required pointer is NULL";
        case RIFT_ERR_SHAPE: return "a size breaks the shape rules of the call";
        case RIFT_ERR_DTYPE: return "unknown or mismatched storage type";
        case RIFT_ERR_BUDGET: return "budget, level or tier out of range";
        case RIFT_ERR_WORKSPACE: return "workspace too small or not 256-byte aligned";
        case RIFT_ERR_HIP: return "a HIP runtime call or kernel launch failed";
        case RIFT_ERR_UNSUPPORTED: return "valid request outside what this library implements";
        case RIFT_ERR_NONFINITE: return "a floating-point input holds NaN or infinity";
    }
    return "unknown status";
}

int32_t rift_set_debug(int32_t on) {
    const int prev = debug_on() ? 1 : 0;
    g_debug.store(on != 0 ? 1 : 0, std::memory_order_relaxed);
    return prev;
}

rift_status rift_check_finite(const void* x, rift_dtype dt, int64_t count, int32_t* status,
                              rift_stream stream) {
    if (status == nullptr || (count > 0 && x == nullptr)) return RIFT_ERR_NULL;
    if (!dt_valid(dt)) return RIFT_ERR_DTYPE;
    if (count < 0) return RIFT_ERR_SHAPE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = launch_nonfinite_clear(status, st);
    if (e == hipSuccess) e = launch_nonfinite_scan(x, dt_kind(dt), (long long)count, status, st);
    return hip_status(e);
}

namespace {
// score workspace: w (float32 [d]), the per-tile arrival counters and the
// pooled-tile counter (int32 [n_tiles + 1], cleared by the call itself); with
// smoothing, then inverse token norms (float64 [n_tiles n_v]), tile
// embeddings (float32 [n_tiles][d]), their dot products (float64
// [n_tiles][n_tiles]) and the smoothed scores.
struct ScoreLayout {
    size_t w, cnt, inv, emb, gram, smooth, dbg, total;
};
ScoreLayout score_layout(int32_t n_tiles, int32_t n_v, int32_t d, int32_t knn_m) {
    ScoreLayout L{};
    size_t off = 0;
    L.w = off;
    off += align_up((size_t)d * sizeof(float));
    L.cnt = off;
    off += align_up((size_t)(n_tiles + 1) * sizeof(int));
    if (knn_m > 0) {
        L.inv = off;
        off += align_up((size_t)n_tiles * n_v * sizeof(double));
        L.emb = off;
        off += align_up((size_t)n_tiles * d * sizeof(float));
        L.gram = off;
        off += align_up((size_t)n_tiles * n_tiles * sizeof(double));
        L.smooth = off;
        off += align_up((size_t)n_tiles * sizeof(double));
    }
    L.dbg = off;   // debug mode: flag word of the input scan
    off += kAlign;
    L.total = off;
    return L;
}
}  // namespace

size_t rift_score_workspace_size(int32_t n_tiles, int32_t n_v, int32_t d, int32_t knn_m) {
    if (d <= 0 || n_tiles <= 0 || n_v <= 0 || knn_m < 0) return 0;
    return score_layout(n_tiles, n_v, d, knn_m).total;
}

}  // extern "C"

namespace {

// Argument checks of rift_score_tiles that do not involve the workspace.
rift_status score_check(const void* tokens, const rift_dtype& dt, int32_t n_tiles, int32_t n_v, int32_t d,
                        const void* query_bank, int32_t n_bg, int32_t keep_count, double tau, int32_t knn_m,
                        const double* token_key, const double* tile_score, const float* tile_u,
                        const int32_t* tile_order, const int32_t* n_keep) {
    if (tokens == nullptr || query_bank == nullptr || token_key == nullptr ||
        tile_score == nullptr || tile_u == nullptr || tile_order == nullptr || n_keep == nullptr)
        return RIFT_ERR_NULL;
    if (!dt_valid(dt)) return RIFT_ERR_DTYPE;
    if (n_tiles < 1 || n_tiles > 4096 || n_v < 1 || n_v > 1024 || d < 32 || d > 16384 ||
        d % 32 != 0 || n_bg < 0 || n_bg > 15 || keep_count < 0 || isnan(tau) || knn_m < 0)
        return RIFT_ERR_SHAPE;
    return RIFT_OK;
}

// Enqueue the scoring of a validated call on a workspace laid out by
// score_layout (device memory of at least L.total bytes, 256-byte aligned).
rift_status score_enqueue(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v, int32_t d,
                          const void* query_bank, int32_t n_bg, int32_t keep_count, double tau, int32_t knn_m,
                          double* token_key, float* token_sim, double* tile_score, float* tile_u,
                          int32_t* tile_order, int32_t* n_keep, unsigned char* ws, const ScoreLayout& L,
                          hipStream_t st) {
    if (init_kernel_attributes() != hipSuccess) return RIFT_ERR_HIP;
    if (debug_on()) {
        const DebugInput in[2] = {{tokens, dt_kind(dt), (long long)n_tiles * n_v * d},
                                  {query_bank, dt_kind(dt), (long long)(1 + n_bg) * d}};
        const rift_status ds = debug_scan(in, 2, reinterpret_cast<int*>(ws + L.dbg), st);
        if (ds != RIFT_OK) return ds;
    }
    hipError_t e = launch_score(tokens, dt == RIFT_BF16, n_tiles, n_v, d, query_bank, n_bg,
                                keep_count, tau, knn_m, token_key, token_sim, tile_score, tile_u,
                                tile_order, n_keep, reinterpret_cast<float*>(ws + L.w),
                                reinterpret_cast<int*>(ws + L.cnt), reinterpret_cast<double*>(ws + L.inv), reinterpret_cast<float*>(ws + L.emb),
                                reinterpret_cast<double*>(ws + L.gram), reinterpret_cast<double*>(ws + L.smooth), st);
    return hip_status(e);
}

// Scratch of rift_score_tiles_noalloc: one copy per GPU, resident until the
// process ends.  In host code `scratch` only names the symbol; its device
// address on each GPU comes from hipGetSymbolAddress with that GPU current.
constexpr size_t kScoreScratchBytes = (size_t)RIFT_SCORE_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScoreScratchBytes];
std::mutex g_scratch_mu;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// The current GPU's address of `scratch`, looked up once per device.
rift_status scratch_address(unsigned char** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return RIFT_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return RIFT_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return RIFT_ERR_HIP;
        g_scratch_ptr[dev] = static_cast<unsigned char*>(p);
    }
    *out = g_scratch_ptr[dev];
    return RIFT_OK;
}

}  // namespace

extern "C" {

rift_status rift_score_tiles(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                             int32_t d, const void* query_bank, int32_t n_bg, int32_t keep_count,
                             double tau, int32_t knn_m, double* token_key, float* token_sim,
                             double* tile_score, float* tile_u, int32_t* tile_order, int32_t* n_keep,
                             void* workspace, size_t ws_bytes, rift_stream stream) {
    rift_status c = score_check(tokens, dt, n_tiles, n_v, d, query_bank, n_bg, keep_count, tau, knn_m, token_key,
                                tile_score, tile_u, tile_order, n_keep);
    if (c != RIFT_OK) return c;
    if (workspace == nullptr) return RIFT_ERR_NULL;
    const ScoreLayout L = score_layout(n_tiles, n_v, d, knn_m);
    if (misaligned(workspace) || ws_bytes < L.total) return RIFT_ERR_WORKSPACE;
    return score_enqueue(tokens, dt, n_tiles, n_v, d, query_bank, n_bg, keep_count, tau, knn_m, token_key,
                         token_sim, tile_score, tile_u, tile_order, n_keep, static_cast<unsigned char*>(workspace),
                         L, static_cast<hipStream_t>(stream));
}

rift_status rift_score_tiles_noalloc(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                                     int32_t d, const void* query_bank, int32_t n_bg, int32_t keep_count,
                                     double tau, int32_t knn_m, double* token_key, float* token_sim,
                                     double* tile_score, float* tile_u, int32_t* tile_order, int32_t* n_keep,
                                     rift_stream stream) {
    rift_status c = score_check(tokens, dt, n_tiles, n_v, d, query_bank, n_bg, keep_count, tau, knn_m, token_key,
                                tile_score, tile_u, tile_order, n_keep);
    if (c != RIFT_OK) return c;
    const ScoreLayout L = score_layout(n_tiles, n_v, d, knn_m);
    if (L.total > kScoreScratchBytes) return RIFT_ERR_WORKSPACE;
    unsigned char* ws = nullptr;
    c = scratch_address(&ws);
    if (c != RIFT_OK) return c;
    return score_enqueue(tokens, dt, n_tiles, n_v, d, query_bank, n_bg, keep_count, tau, knn_m, token_key,
                         token_sim, tile_score, tile_u, tile_order, n_keep, ws, L, static_cast<hipStream_t>(stream));
}

rift_status rift_assign_budgets(int32_t n_keep, int32_t n_v, const int32_t* levels,
                                int32_t n_levels, const int32_t* tier_num, int32_t tier_den,
                                int32_t* budgets, int64_t* total) {
    static const int32_t kDefaultNum[3] = {1, 3, 4};
    if (levels == nullptr || (n_keep > 0 && budgets == nullptr)) return RIFT_ERR_NULL;
    if (n_keep < 0 || n_v < 1 || n_levels < 1 || n_levels > 64) return RIFT_ERR_SHAPE;
    if (tier_num == nullptr) {
        if (n_levels != 4) return RIFT_ERR_BUDGET;
        tier_num = kDefaultNum;
        tier_den = 16;
    }
    if (tier_den < 1) return RIFT_ERR_BUDGET;
    int64_t num_sum = 0;
    for (int j = 0; j < n_levels; ++j) {
        if (levels[j] < 1 || levels[j] > n_v) return RIFT_ERR_BUDGET;
        if (j > 0 && levels[j] >= levels[j - 1]) return RIFT_ERR_BUDGET;
        if (j < n_levels - 1) {
            if (tier_num[j] < 0) return RIFT_ERR_BUDGET;
            num_sum += tier_num[j];
        }
    }
    if (num_sum > tier_den) return RIFT_ERR_BUDGET;
    int64_t rho = 0, sum = 0;
    for (int j = 0; j < n_levels; ++j) {
        int64_t cnt;
        if (j < n_levels - 1) cnt = ((int64_t)n_keep * tier_num[j]) / tier_den;
        else cnt = (int64_t)n_keep - rho;
        for (int64_t c = 0; c < cnt; ++c) {
            budgets[rho++] = levels[j];
            sum += levels[j];
        }
    }
    if (total != nullptr) *total = sum;
    return RIFT_OK;
}

rift_status rift_assign_budgets_utility(int32_t n_keep, int32_t n_v, int32_t n_c,
                                        const int32_t* levels, const double* alpha_pos,
                                        const double* alpha_neg, const double* energy, double lambda,
                                        const float* p, int32_t* budgets, int64_t* total) {
#pragma clang fp contract(off)
    if (levels == nullptr || alpha_pos == nullptr || alpha_neg == nullptr || energy == nullptr)
        return RIFT_ERR_NULL;
    if (n_keep > 0 && (p == nullptr || budgets == nullptr)) return RIFT_ERR_NULL;
    if (n_keep < 0 || n_v < 1 || n_c < 1 || n_c > 64) return RIFT_ERR_SHAPE;
    if (!std::isfinite(lambda)) return RIFT_ERR_BUDGET;
    for (int c = 0; c < n_c; ++c) {
        if (levels[c] < 1 || levels[c] > n_v) return RIFT_ERR_BUDGET;
        if (!std::isfinite(alpha_pos[c]) || !std::isfinite(alpha_neg[c]) || !std::isfinite(energy[c]))
            return RIFT_ERR_BUDGET;
    }
    for (int i = 0; i < n_keep; ++i)
        if (!(p[i] >= 0.0f && p[i] <= 1.0f)) return RIFT_ERR_BUDGET;
    int64_t sum = 0;
    for (int i = 0; i < n_keep; ++i) {
        const double pi = (double)p[i];
        int best_c = 0;
        double best_u = 0.0;
        for (int c = 0; c < n_c; ++c) {
            // each operation rounded on its own (no contraction in this function)
            const double u = ((pi * alpha_pos[c]) + ((1.0 - pi) * alpha_neg[c])) - (lambda * energy[c]);
            if (c == 0 || u > best_u || (u == best_u && levels[c] < best_c)) {
                best_c = levels[c];
                best_u = u;
            }
        }
        budgets[i] = best_c;
        sum += best_c;
    }
    if (total != nullptr) *total = sum;
    return RIFT_OK;
}

rift_status rift_select_tokens(const double* token_key, int32_t n_tiles, int32_t n_v,
                               const int32_t* kept_tiles, const int32_t* budgets, int32_t n_keep,
                               int32_t* sel_offsets, int32_t* sel_idx, int64_t sel_capacity,
                               int32_t* status, rift_stream stream) {
    if (sel_offsets == nullptr || status == nullptr) return RIFT_ERR_NULL;
    if (n_keep > 0 && (token_key == nullptr || kept_tiles == nullptr || budgets == nullptr))
        return RIFT_ERR_NULL;
    if (sel_capacity > 0 && sel_idx == nullptr) return RIFT_ERR_NULL;
    if (n_v < 1 || n_v > 1024 || n_tiles < 1 || (int64_t)n_tiles * n_v > (int64_t)INT32_MAX ||
        n_keep < 0 || n_keep > n_tiles || sel_capacity < 0 || sel_capacity > (int64_t)INT32_MAX)
        return RIFT_ERR_SHAPE;
    if (debug_on() && n_keep > 0) {   // every key of the scene; the status word holds the flag
        const DebugInput in[1] = {{token_key, 2, (long long)n_tiles * n_v}};
        const rift_status ds = debug_scan(in, 1, status, static_cast<hipStream_t>(stream));
        if (ds != RIFT_OK) return ds;
    }
    hipError_t e = launch_select(token_key, n_tiles, n_v, kept_tiles, budgets, n_keep, sel_offsets,
                                 sel_idx, sel_capacity, status, static_cast<hipStream_t>(stream));
    return hip_status(e);
}

rift_status rift_split_budgets(int32_t n_keep, int32_t n_v, const int32_t* budgets, int32_t num,
                               int32_t den, int32_t* dominant, int32_t* context) {
    if (n_keep > 0 && (budgets == nullptr || dominant == nullptr || context == nullptr)) return RIFT_ERR_NULL;
    if (n_keep < 0 || n_v < 1 || num < 0 || den < 1 || num > den) return RIFT_ERR_SHAPE;
    for (int i = 0; i < n_keep; ++i)
        if (budgets[i] < 0 || budgets[i] > n_v) return RIFT_ERR_BUDGET;
    for (int i = 0; i < n_keep; ++i) {
        const int64_t c = budgets[i];
        int64_t kc = c * num / den;
        if (kc > n_v - c) kc = n_v - c;
        context[i] = (int32_t)kc;
        dominant[i] = (int32_t)(c - kc);
    }
    return RIFT_OK;
}

namespace {
// merge workspace: group of each token, targets, their inverse norms, tile flags
struct MergeLayout {
    size_t grp, tgt, inv, ok, total;
};
MergeLayout merge_layout(int32_t n_keep, int32_t n_v) {
    MergeLayout L{};
    const size_t nk = n_keep > 0 ? (size_t)n_keep : 1;
    size_t off = 0;
    L.grp = off;
    off += align_up(nk * n_v * sizeof(int));
    L.tgt = off;
    off += align_up(nk * n_v * sizeof(int));
    L.inv = off;
    off += align_up(nk * n_v * sizeof(double));
    L.ok = off;
    off += align_up(nk * sizeof(int));
    L.total = off;
    return L;
}
}  // namespace

size_t rift_merge_workspace_size(int32_t n_keep, int32_t n_v) {
    if (n_keep < 0 || n_v < 1) return 0;
    return merge_layout(n_keep, n_v).total;
}

rift_status rift_merge_context(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                               int32_t d, const int32_t* kept_tiles, const int32_t* sel_offsets,
                               const int32_t* sel_idx, const int32_t* ctx_offsets, int32_t n_keep,
                               void* ctx_rows, int64_t ctx_capacity, int32_t* status,
                               void* workspace, size_t ws_bytes, rift_stream stream) {
    if (sel_offsets == nullptr || ctx_offsets == nullptr || status == nullptr || workspace == nullptr)
        return RIFT_ERR_NULL;
    if (n_keep > 0 && (tokens == nullptr || kept_tiles == nullptr || sel_idx == nullptr)) return RIFT_ERR_NULL;
    if (ctx_capacity > 0 && ctx_rows == nullptr) return RIFT_ERR_NULL;
    if (!dt_valid(dt)) return RIFT_ERR_DTYPE;
    if (n_tiles < 1 || n_v < 1 || n_v > 1024 || d < 32 || d > 16384 || d % 32 != 0 || n_keep < 0 ||
        n_keep > 65535 || ctx_capacity < 0 || ctx_capacity > ((int64_t)1 << 24))
        return RIFT_ERR_SHAPE;
    const MergeLayout L = merge_layout(n_keep, n_v);
    if (misaligned(workspace) || ws_bytes < L.total) return RIFT_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    hipError_t e = launch_merge(tokens, dt == RIFT_BF16, n_tiles, n_v, d, kept_tiles, sel_offsets, sel_idx,
                                ctx_offsets, n_keep, ctx_rows, ctx_capacity, status,
                                reinterpret_cast<int*>(ws + L.grp), reinterpret_cast<int*>(ws + L.tgt),
                                reinterpret_cast<double*>(ws + L.inv), reinterpret_cast<int*>(ws + L.ok),
                                static_cast<hipStream_t>(stream));
    return hip_status(e);
}

rift_status rift_compact(const void* tokens, rift_dtype dt, int32_t n_tiles, int32_t n_v,
                         int32_t d, const int32_t* kept_tiles, const int32_t* sel_offsets,
                         const int32_t* sel_idx, int32_t n_keep, const void* ctx_rows,
                         const int32_t* ctx_offsets, const void* sys_emb, int32_t n_sys,
                         const void* qry_emb, int32_t n_qry, int32_t shared_prefix, void* packed,
                         int64_t packed_rows, int32_t* cu_seqlens, int32_t* position_ids, int32_t* status,
                         rift_stream stream) {
    if (sel_offsets == nullptr || cu_seqlens == nullptr || status == nullptr) return RIFT_ERR_NULL;
    if (n_keep > 0 && (tokens == nullptr || kept_tiles == nullptr)) return RIFT_ERR_NULL;
    if (packed_rows > 0 && (packed == nullptr || position_ids == nullptr)) return RIFT_ERR_NULL;
    if ((n_sys > 0 && sys_emb == nullptr) || (n_qry > 0 && qry_emb == nullptr)) return RIFT_ERR_NULL;
    if ((ctx_rows == nullptr) != (ctx_offsets == nullptr)) return RIFT_ERR_NULL;
    if (!dt_valid(dt)) return RIFT_ERR_DTYPE;
    if (n_tiles < 1 || n_v < 1 || d < 1 || n_keep < 0 || n_keep > 65535 || n_sys < 0 || n_qry < 0 ||
        packed_rows < 0 || ((size_t)d * dt_bytes(dt)) % 16 != 0 || packed_rows > ((int64_t)1 << 25) ||
        (shared_prefix != 0 && shared_prefix != 1))
        return RIFT_ERR_SHAPE;
    hipError_t e = launch_compact(tokens, (int)dt_bytes(dt), n_tiles, n_v, d, kept_tiles,
                                  sel_offsets, sel_idx, n_keep, ctx_rows, ctx_offsets, sys_emb, n_sys,
                                  qry_emb, n_qry, shared_prefix != 0, packed, packed_rows, cu_seqlens,
                                  position_ids, status, static_cast<hipStream_t>(stream));
    return hip_status(e);
}

size_t rift_prefill_workspace_size(const rift_model_cfg* cfg, int32_t total_tokens,
                                   int32_t max_seqlen) {
    if (check_cfg(cfg) != RIFT_OK || total_tokens < 0 || max_seqlen < 0) return 0;
    return prefill_layout(*cfg, total_tokens, max_seqlen).total;
}

rift_status rift_prefill(const rift_model_cfg* cfg, const rift_layer_weights* layers,
                         const void* x_in, rift_dtype x_dt, const int32_t* cu_seqlens,
                         const int32_t* position_ids, int32_t n_seq, int32_t total_tokens,
                         int32_t max_seqlen, int32_t n_prefix, float* hidden_out, void* kv_cache,
                         void* workspace, size_t ws_bytes, void* const* events, rift_stream stream) {
    rift_status cs = check_cfg(cfg);
    if (cs != RIFT_OK) return cs;
    const rift_model_cfg c = *cfg;
    if (!dt_valid(x_dt) || (x_dt != c.dt && x_dt != RIFT_F32)) return RIFT_ERR_DTYPE;
    if (total_tokens < 0 || n_seq < 0 || max_seqlen < 1 || max_seqlen > 65536 || n_prefix < 0 ||
        n_prefix > total_tokens || n_prefix > max_seqlen || (n_prefix > 0 && n_seq < 1))
        return RIFT_ERR_SHAPE;
    // the bf16 GEMMs address operands with 32-bit byte offsets
    if (c.dt == RIFT_BF16 && (uint64_t)total_tokens * (uint64_t)(c.d > c.ffn ? c.d : c.ffn) >=
                                 (1ull << 31))
        return RIFT_ERR_UNSUPPORTED;
    if (total_tokens == 0) return RIFT_OK;
    if (x_in == nullptr || cu_seqlens == nullptr || position_ids == nullptr ||
        hidden_out == nullptr || workspace == nullptr || (c.n_layers > 0 && layers == nullptr))
        return RIFT_ERR_NULL;
    for (int l = 0; l < c.n_layers; ++l) {
        const rift_layer_weights& w = layers[l];
        if (!w.wq || !w.wk || !w.wv || !w.wo || !w.w_gate || !w.w_up || !w.w_down || !w.g_attn ||
            !w.g_ffn)
            return RIFT_ERR_NULL;
    }
    const PrefillLayout L = prefill_layout(c, total_tokens, max_seqlen);
    if (misaligned(workspace) || ws_bytes < L.total) return RIFT_ERR_WORKSPACE;
    if (init_kernel_attributes() != hipSuccess) return RIFT_ERR_HIP;

    hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    if (debug_on()) {   // the packed input and every weight and gain
        const int wk = dt_kind(c.dt);
        const long long dd = (long long)c.d * c.d, df = (long long)c.d * c.ffn;
        rift_status ds = RIFT_OK;
        {
            const DebugInput in[1] = {{x_in, x_dt == RIFT_BF16 ? 0 : 1, (long long)total_tokens * c.d}};
            ds = debug_scan(in, 1, reinterpret_cast<int*>(ws + L.dbg), st);
        }
        for (int l = 0; l < c.n_layers && ds == RIFT_OK; ++l) {
            const rift_layer_weights& w = layers[l];
            const DebugInput in[9] = {{w.wq, wk, dd},     {w.wk, wk, dd},     {w.wv, wk, dd},
                                      {w.wo, wk, dd},     {w.w_gate, wk, df}, {w.w_up, wk, df},
                                      {w.w_down, wk, df}, {w.g_attn, wk, c.d}, {w.g_ffn, wk, c.d}};
            ds = debug_scan(in, 9, reinterpret_cast<int*>(ws + L.dbg), st);
        }
        if (ds != RIFT_OK) return ds;
    }
    float2* rope = reinterpret_cast<float2*>(ws + L.rope);
    const int T = total_tokens;
    const int d = c.d;
    const size_t td = (size_t)T * d;
    const bool bf = c.dt == RIFT_BF16;
    const size_t e = dt_bytes(c.dt);
    hipError_t err = hipSuccess;
#define RIFT_TRY(x)                        \
    do {                                   \
        err = (x);                         \
        if (err != hipSuccess) return RIFT_ERR_HIP; \
    } while (0)

    if (c.n_layers == 0) {
        if (x_dt == RIFT_F32) {
            if (static_cast<const void*>(hidden_out) != x_in)
                RIFT_TRY(launch_copy_f32(static_cast<const float*>(x_in), hidden_out, (long long)td, st));
        } else {
            RIFT_TRY(launch_to_f32(x_in, true, hidden_out, (long long)td, st));
        }
        return RIFT_OK;
    }
    RIFT_TRY(launch_rope_table(rope, max_seqlen, c.head_dim, c.rope_base, st));
    // attention work list (one entry per sequence, group of 8 heads and
    // 128-query block), built once for every layer
    int2* alist = nullptr;
    int n_alist = 0;
    if (attention_list_capacity(c, T) > 0) {
        alist = reinterpret_cast<int2*>(ws + L.alist);
        n_alist = attention_worklist_entries(T, n_seq, c.n_heads);
        RIFT_TRY(launch_attention_worklist(cu_seqlens, n_seq, c.n_heads, alist, n_alist, st));
    }
    // benchmark hook: event pair around stage g of layer l (NULL entries skipped)
    auto mark = [&](int l, int g, int end) -> hipError_t {
        if (events == nullptr || events[10 * l + 2 * g + end] == nullptr) return hipSuccess;
        return hipEventRecord(static_cast<hipEvent_t>(events[10 * l + 2 * g + end]), st);
    };

    for (int l = 0; l < c.n_layers; ++l) {
        const rift_layer_weights& w = layers[l];
        void* h = ws + L.h;
        void* qb = ws + L.q;
        void* kb = ws + L.k;
        void* vb = ws + L.v;
        if (kv_cache != nullptr) {
            kb = static_cast<unsigned char*>(kv_cache) + (size_t)(2 * l) * td * e;
            vb = static_cast<unsigned char*>(kv_cache) + (size_t)(2 * l + 1) * td * e;
        }
        // attention input norm; the first layer also lays down the f32 residual
        if (l == 0) {
            const bool in_bf16 = (x_dt == RIFT_BF16);
            float* resid = (in_bf16 || static_cast<const void*>(hidden_out) != x_in) ? hidden_out : nullptr;
            RIFT_TRY(launch_rmsnorm(x_in, in_bf16, resid, w.g_attn, bf, h, bf, T, d, c.rms_eps, st));
        } else {
            RIFT_TRY(launch_rmsnorm(hidden_out, false, nullptr, w.g_attn, bf, h, bf, T, d, c.rms_eps, st));
        }
        if (bf) {
            QkvArgs qa{};
            qa.a = static_cast<const uint16_t*>(h);
            qa.wq = static_cast<const uint16_t*>(w.wq);
            qa.wk = static_cast<const uint16_t*>(w.wk);
            qa.wv = static_cast<const uint16_t*>(w.wv);
            qa.q = static_cast<uint16_t*>(qb);
            qa.k = static_cast<uint16_t*>(kb);
            qa.v = static_cast<uint16_t*>(vb);
            qa.rope = rope;
            qa.pos = position_ids;
            qa.n_pos = max_seqlen;
            qa.M = T;
            qa.d = d;
            qa.hd = c.head_dim;
            // Tile walk directions: each GEMM starts with the rows its input's
            // producer wrote last (norms and attention write rows in ascending
            // order), so its first A panels come from the memory-side cache:
            // QKV, out and gate/up walk backwards, down (after the backward
            // gate/up) forwards.  Results do not depend on the order.
            RIFT_TRY(mark(l, 0, 0));
            RIFT_TRY(launch_gemm_qkv_rope(qa, st, true));
            RIFT_TRY(mark(l, 0, 1));
            // attention output reuses the h buffer (h is consumed by the QKV GEMM)
            RIFT_TRY(mark(l, 1, 0));
            RIFT_TRY(launch_attention_bf16(static_cast<const uint16_t*>(qb), static_cast<const uint16_t*>(kb),
                                           static_cast<const uint16_t*>(vb), static_cast<uint16_t*>(h),
                                           cu_seqlens, n_seq, max_seqlen, c.n_heads, c.head_dim, n_prefix, alist,
                                           n_alist, st));
            RIFT_TRY(mark(l, 1, 1));
            RIFT_TRY(mark(l, 2, 0));
            RIFT_TRY(launch_gemm_resid(static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w.wo),
                                       hidden_out, T, d, d, st, true));
            RIFT_TRY(mark(l, 2, 1));
            RIFT_TRY(launch_rmsnorm(hidden_out, false, nullptr, w.g_ffn, true, h, true, T, d, c.rms_eps, st));
            uint16_t* a = reinterpret_cast<uint16_t*>(ws + L.a);
            RIFT_TRY(mark(l, 3, 0));
            RIFT_TRY(launch_gemm_swiglu(static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w.w_gate),
                                        static_cast<const uint16_t*>(w.w_up), a, T, c.ffn, d, st, true));
            RIFT_TRY(mark(l, 3, 1));
            RIFT_TRY(mark(l, 4, 0));
            RIFT_TRY(launch_gemm_resid(a, static_cast<const uint16_t*>(w.w_down), hidden_out, T, d, c.ffn, st,
                                       false));
            RIFT_TRY(mark(l, 4, 1));
        } else {
            float* hf = static_cast<float*>(h);
            float* qf = static_cast<float*>(qb);
            float* kf = static_cast<float*>(kb);
            float* vf = static_cast<float*>(vb);
            RIFT_TRY(mark(l, 0, 0));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.wq), qf, T, d, d, false, st));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.wk), kf, T, d, d, false, st));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.wv), vf, T, d, d, false, st));
            RIFT_TRY(launch_rope_apply_f32(qf, rope, position_ids, max_seqlen, T, c.n_heads, c.head_dim, st));
            RIFT_TRY(launch_rope_apply_f32(kf, rope, position_ids, max_seqlen, T, c.n_heads, c.head_dim, st));
            RIFT_TRY(mark(l, 0, 1));
            RIFT_TRY(mark(l, 1, 0));
            RIFT_TRY(launch_attention_f32(qf, kf, vf, hf, cu_seqlens, n_seq, max_seqlen, c.n_heads,
                                          c.head_dim, n_prefix, st));
            RIFT_TRY(mark(l, 1, 1));
            RIFT_TRY(mark(l, 2, 0));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.wo), hidden_out, T, d, d, true, st));
            RIFT_TRY(mark(l, 2, 1));
            RIFT_TRY(launch_rmsnorm(hidden_out, false, nullptr, w.g_ffn, false, hf, false, T, d, c.rms_eps, st));
            float* gate = reinterpret_cast<float*>(ws + L.a);
            float* up = reinterpret_cast<float*>(ws + L.gate2);
            RIFT_TRY(mark(l, 3, 0));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.w_gate), gate, T, c.ffn, d, false, st));
            RIFT_TRY(launch_gemm_f32(hf, static_cast<const float*>(w.w_up), up, T, c.ffn, d, false, st));
            RIFT_TRY(launch_swiglu_f32(gate, up, gate, (long long)T * c.ffn, st));
            RIFT_TRY(mark(l, 3, 1));
            RIFT_TRY(mark(l, 4, 0));
            RIFT_TRY(launch_gemm_f32(gate, static_cast<const float*>(w.w_down), hidden_out, T, d, c.ffn, true, st));
            RIFT_TRY(mark(l, 4, 1));
        }
    }
#undef RIFT_TRY
    return RIFT_OK;
}

namespace {
// decode workspace: RoPE table over max_seqlen + max_new positions, the new
// tokens' positions, h, q, k, v [n_seq][d] and the SwiGLU activation [n_seq][ffn]
struct DecodeLayout {
    size_t rope, pos, h, q, k, v, a, part, total;
};
// the decode GEMMs split K (float32 partials) when every shape allows it
bool decode_skinny(const rift_model_cfg& c) {
    return skinny_supported(3 * c.d, c.d, c.d) && skinny_supported(c.d, c.d, c.d) &&
           skinny_supported(2 * c.ffn, c.d, c.ffn) && skinny_supported(c.d, c.ffn, c.d) && skinny_norm_supported(c.d);
}
size_t decode_part_floats(const rift_model_cfg& c, int64_t n_seq) {
    if (!decode_skinny(c)) return 0;
    const int64_t shapes[4][2] = {{3 * (int64_t)c.d, c.d}, {c.d, c.d}, {2 * (int64_t)c.ffn, c.d}, {c.d, c.ffn}};
    int64_t most = 0;
    for (const auto& nk : shapes) {
        const int64_t f = (int64_t)skinny_splits((int)nk[0], (int)nk[1]) * nk[0];
        most = f > most ? f : most;
    }
    return (size_t)(most * n_seq);
}
DecodeLayout decode_layout(const rift_model_cfg& c, int64_t n_seq, int64_t n_pos) {
    DecodeLayout L{};
    size_t off = 0;
    L.rope = off;
    off += align_up((size_t)n_pos * (size_t)(c.head_dim / 2) * sizeof(float2));
    L.pos = off;
    off += align_up((size_t)n_seq * sizeof(int));
    L.h = off;
    off += align_up((size_t)n_seq * c.d * 2);
    L.q = off;
    off += align_up((size_t)n_seq * c.d * 2);
    L.k = off;
    off += align_up((size_t)n_seq * c.d * 2);
    L.v = off;
    off += align_up((size_t)n_seq * c.d * 2);
    L.a = off;
    off += align_up((size_t)n_seq * c.ffn * 2);
    L.part = off;
    off += align_up(decode_part_floats(c, n_seq) * sizeof(float));
    L.total = off;
    return L;
}
}  // namespace

size_t rift_decode_workspace_size(const rift_model_cfg* cfg, int32_t n_seq, int32_t max_seqlen,
                                  int32_t max_new) {
    if (check_cfg(cfg) != RIFT_OK || n_seq < 0 || max_seqlen < 0 || max_new < 1) return 0;
    return decode_layout(*cfg, n_seq, (int64_t)max_seqlen + max_new).total;
}

rift_status rift_decode_step(const rift_model_cfg* cfg, const rift_layer_weights* layers, const void* x_new,
                             const int32_t* cu_seqlens, int32_t n_seq, int32_t total_tokens,
                             int32_t max_seqlen, int32_t n_prefix, const void* kv_cache, void* kv_new,
                             int32_t max_new, int32_t step, float* hidden_out, void* workspace, size_t ws_bytes,
                             rift_stream stream) {
    rift_status cs = check_cfg(cfg);
    if (cs != RIFT_OK) return cs;
    const rift_model_cfg c = *cfg;
    if (c.dt != RIFT_BF16) return RIFT_ERR_UNSUPPORTED;
    if (n_seq < 0 || total_tokens < 0 || max_seqlen < 0 || max_new < 1 || step < 0 || step >= max_new ||
        (int64_t)max_seqlen + max_new > 16384 || (int64_t)n_seq * c.ffn >= (1ll << 31) ||
        (int64_t)total_tokens * c.d >= (1ll << 31) || n_prefix < 0 || n_prefix > total_tokens ||
        n_prefix > max_seqlen)
        return RIFT_ERR_SHAPE;
    // with a shared prefix the prompts are sequences 1..n_seq of the prefill
    const int32_t* cu_p = cu_seqlens + (n_prefix > 0 ? 1 : 0);
    if (n_seq == 0 || c.n_layers == 0) return RIFT_OK;
    if (x_new == nullptr || cu_seqlens == nullptr || kv_new == nullptr || hidden_out == nullptr ||
        workspace == nullptr || layers == nullptr || (total_tokens > 0 && kv_cache == nullptr))
        return RIFT_ERR_NULL;
    for (int l = 0; l < c.n_layers; ++l) {
        const rift_layer_weights& w = layers[l];
        if (!w.wq || !w.wk || !w.wv || !w.wo || !w.w_gate || !w.w_up || !w.w_down || !w.g_attn ||
            !w.g_ffn)
            return RIFT_ERR_NULL;
    }
    const int n_pos = max_seqlen + max_new;
    const DecodeLayout L = decode_layout(c, n_seq, n_pos);
    if (misaligned(workspace) || ws_bytes < L.total) return RIFT_ERR_WORKSPACE;
    if (init_kernel_attributes() != hipSuccess) return RIFT_ERR_HIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    float2* rope = reinterpret_cast<float2*>(ws + L.rope);
    int* pos = reinterpret_cast<int*>(ws + L.pos);
    uint16_t* h = reinterpret_cast<uint16_t*>(ws + L.h);
    uint16_t* qb = reinterpret_cast<uint16_t*>(ws + L.q);
    uint16_t* kb = reinterpret_cast<uint16_t*>(ws + L.k);
    uint16_t* vb = reinterpret_cast<uint16_t*>(ws + L.v);
    uint16_t* a = reinterpret_cast<uint16_t*>(ws + L.a);
    const int d = c.d;
    const size_t td = (size_t)total_tokens * d;   // one K or V plane of the prefill cache
    const size_t nd = (size_t)n_seq * max_new * d;   // one K or V plane of the decode cache
#define RIFT_TRY(x)                                   \
    do {                                              \
        if ((x) != hipSuccess) return RIFT_ERR_HIP;   \
    } while (0)
    RIFT_TRY(launch_rope_table(rope, n_pos, c.head_dim, c.rope_base, st));
    RIFT_TRY(launch_decode_pos(cu_p, n_seq, n_prefix, step, pos, st));
    if (decode_skinny(c)) {
        // split-K GEMMs; the residual reduce of each layer's last GEMM also
        // applies the next layer's attention RMSNorm
        float* part = reinterpret_cast<float*>(ws + L.part);
        const int F = c.ffn;
        const int s_qkv = skinny_splits(3 * d, d), s_o = skinny_splits(d, d);
        const int s_gu = skinny_splits(2 * F, d), s_dn = skinny_splits(d, F);
        RIFT_TRY(launch_rmsnorm(x_new, true, hidden_out, layers[0].g_attn, true, h, true, n_seq, d, c.rms_eps, st));
        for (int l = 0; l < c.n_layers; ++l) {
            const rift_layer_weights& w = layers[l];
            uint16_t* kn = static_cast<uint16_t*>(kv_new) + (size_t)(2 * l) * nd;
            uint16_t* vn = static_cast<uint16_t*>(kv_new) + (size_t)(2 * l + 1) * nd;
            RIFT_TRY(launch_skinny_gemm(h, static_cast<const uint16_t*>(w.wq), static_cast<const uint16_t*>(w.wk),
                                        static_cast<const uint16_t*>(w.wv), d, n_seq, 3 * d, d, part, st));
            RIFT_TRY(launch_skinny_qkv(part, s_qkv, n_seq, d, c.head_dim, rope, pos, n_pos, qb, kn, vn, max_new,
                                       step, st));
            RIFT_TRY(launch_decode_attention(qb, static_cast<const uint16_t*>(kv_cache) + (size_t)(2 * l) * td,
                                             static_cast<const uint16_t*>(kv_cache) + (size_t)(2 * l + 1) * td, kn,
                                             vn, cu_p, n_seq, total_tokens, n_prefix, c.n_heads, c.head_dim,
                                             n_pos, max_new, step, h, st));
            RIFT_TRY(launch_skinny_gemm(h, static_cast<const uint16_t*>(w.wo), nullptr, nullptr, d, n_seq, d, d,
                                        part, st));
            RIFT_TRY(launch_skinny_resid_norm(part, s_o, n_seq, d, hidden_out, static_cast<const uint16_t*>(w.g_ffn),
                                              h, c.rms_eps, st));
            RIFT_TRY(launch_skinny_gemm(h, static_cast<const uint16_t*>(w.w_gate),
                                        static_cast<const uint16_t*>(w.w_up), nullptr, F, n_seq, 2 * F, d, part, st));
            RIFT_TRY(launch_skinny_swiglu(part, s_gu, n_seq, F, a, st));
            RIFT_TRY(launch_skinny_gemm(a, static_cast<const uint16_t*>(w.w_down), nullptr, nullptr, d, n_seq, d, F,
                                        part, st));
            const bool last = l + 1 == c.n_layers;
            RIFT_TRY(launch_skinny_resid_norm(part, s_dn, n_seq, d, hidden_out,
                                              last ? nullptr : static_cast<const uint16_t*>(layers[l + 1].g_attn),
                                              last ? nullptr : h, c.rms_eps, st));
        }
        return RIFT_OK;
    }
    for (int l = 0; l < c.n_layers; ++l) {
        const rift_layer_weights& w = layers[l];
        const uint16_t* kp = static_cast<const uint16_t*>(kv_cache) + (size_t)(2 * l) * td;
        const uint16_t* vp = static_cast<const uint16_t*>(kv_cache) + (size_t)(2 * l + 1) * td;
        uint16_t* kn = static_cast<uint16_t*>(kv_new) + (size_t)(2 * l) * nd;
        uint16_t* vn = static_cast<uint16_t*>(kv_new) + (size_t)(2 * l + 1) * nd;
        if (l == 0)
            RIFT_TRY(launch_rmsnorm(x_new, true, hidden_out, w.g_attn, true, h, true, n_seq, d, c.rms_eps, st));
        else
            RIFT_TRY(launch_rmsnorm(hidden_out, false, nullptr, w.g_attn, true, h, true, n_seq, d, c.rms_eps, st));
        QkvArgs qa{};
        qa.a = h;
        qa.wq = static_cast<const uint16_t*>(w.wq);
        qa.wk = static_cast<const uint16_t*>(w.wk);
        qa.wv = static_cast<const uint16_t*>(w.wv);
        qa.q = qb;
        qa.k = kb;
        qa.v = vb;
        qa.rope = rope;
        qa.pos = pos;
        qa.n_pos = n_pos;
        qa.M = n_seq;
        qa.d = d;
        qa.hd = c.head_dim;
        RIFT_TRY(launch_gemm_qkv_rope(qa, st));
        RIFT_TRY(launch_kv_append(kb, vb, kn, vn, n_seq, d, max_new, step, st));
        RIFT_TRY(launch_decode_attention(qb, kp, vp, kn, vn, cu_p, n_seq, total_tokens, n_prefix, c.n_heads,
                                         c.head_dim, n_pos, max_new, step, h, st));
        RIFT_TRY(launch_gemm_resid(h, static_cast<const uint16_t*>(w.wo), hidden_out, n_seq, d, d, st));
        RIFT_TRY(launch_rmsnorm(hidden_out, false, nullptr, w.g_ffn, true, h, true, n_seq, d, c.rms_eps, st));
        RIFT_TRY(launch_gemm_swiglu(h, static_cast<const uint16_t*>(w.w_gate), static_cast<const uint16_t*>(w.w_up),
                                    a, n_seq, c.ffn, d, st));
        RIFT_TRY(launch_gemm_resid(a, static_cast<const uint16_t*>(w.w_down), hidden_out, n_seq, d, c.ffn, st));
    }
#undef RIFT_TRY
    return RIFT_OK;
}

}  // extern "C"

// Host-side checks of the C ABI for a build whose host code is instrumented
// with AddressSanitizer and UndefinedBehaviorSanitizer.  Every call here
// either runs entirely on the host (budget assignment, budget split,
// workspace sizes, status strings) or fails argument validation before any
// HIP call, so it needs no GPU.  Exit status 0 when every status code matches;
// the sanitizers abort on the first finding.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/rift.h"

static int g_fail = 0, g_checks = 0;
#define EXPECT(cond)                                                                  \
    do {                                                                              \
        ++g_checks;                                                                   \
        if (!(cond)) {                                                                \
            ++g_fail;                                                                 \
            fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #cond);         \
        }                                                                             \
    } while (0)

static void* const FAKE = reinterpret_cast<void*>(0x1000);   // never dereferenced: validation fails first

int main() {
    EXPECT(rift_abi_version() == RIFT_ABI_VERSION);
    for (int s = -1; s <= 9; ++s) EXPECT(strlen(rift_status_string((rift_status)s)) > 0);
    const int prev = rift_set_debug(1);
    EXPECT(rift_set_debug(prev) == 1);

    // ---- check_finite: validation only
    EXPECT(rift_check_finite(FAKE, RIFT_BF16, 10, nullptr, nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_check_finite(nullptr, RIFT_BF16, 10, (int32_t*)FAKE, nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_check_finite(FAKE, (rift_dtype)5, 10, (int32_t*)FAKE, nullptr) == RIFT_ERR_DTYPE);
    EXPECT(rift_check_finite(FAKE, RIFT_F32, -1, (int32_t*)FAKE, nullptr) == RIFT_ERR_SHAPE);

    // ---- Stage 1: workspace sizes over the whole shape range, validation
    for (int nt : {1, 7, 400, 4096})
        for (int nv : {1, 576, 1024})
            for (int d : {32, 4096, 16384})
                for (int m : {0, 6}) EXPECT(rift_score_workspace_size(nt, nv, d, m) >= (size_t)d * 4);
    EXPECT(rift_score_workspace_size(0, 576, 4096, 0) == 0 && rift_score_workspace_size(4, 576, 4096, -1) == 0);
    double* D = (double*)FAKE;
    float* F = (float*)FAKE;
    int32_t* I = (int32_t*)FAKE;
    void* ws = reinterpret_cast<void*>(0x10000);
    EXPECT(rift_score_tiles(nullptr, RIFT_BF16, 4, 576, 256, FAKE, 15, 2, 0.37, 0, D, nullptr, D, F, I, I, ws, 1 << 20,
                            nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_score_tiles(FAKE, (rift_dtype)7, 4, 576, 256, FAKE, 15, 2, 0.37, 0, D, nullptr, D, F, I, I, ws, 1 << 20,
                            nullptr) == RIFT_ERR_DTYPE);
    EXPECT(rift_score_tiles(FAKE, RIFT_BF16, 4097, 576, 256, FAKE, 15, 2, 0.37, 0, D, nullptr, D, F, I, I, ws, 1 << 20,
                            nullptr) == RIFT_ERR_SHAPE);
    EXPECT(rift_score_tiles(FAKE, RIFT_BF16, 4, 576, 48, FAKE, 15, 2, 0.37, 0, D, nullptr, D, F, I, I, ws, 1 << 20,
                            nullptr) == RIFT_ERR_SHAPE);
    EXPECT(rift_score_tiles(FAKE, RIFT_BF16, 4, 576, 256, FAKE, 15, 2, NAN, 0, D, nullptr, D, F, I, I, ws, 1 << 20,
                            nullptr) == RIFT_ERR_SHAPE);
    EXPECT(rift_score_tiles(FAKE, RIFT_BF16, 4, 576, 256, FAKE, 15, 2, 0.37, 0, D, nullptr, D, F, I, I,
                            reinterpret_cast<void*>(0x10010), 1 << 20, nullptr) == RIFT_ERR_WORKSPACE);
    EXPECT(rift_score_tiles(FAKE, RIFT_BF16, 4, 576, 256, FAKE, 15, 2, 0.37, 6, D, nullptr, D, F, I, I, ws, 64,
                            nullptr) == RIFT_ERR_WORKSPACE);
    EXPECT(rift_score_tiles_noalloc(FAKE, RIFT_BF16, 4096, 1024, 4096, FAKE, 15, 2, 0.37, 6, D, nullptr, D, F, I, I,
                                    nullptr) == RIFT_ERR_WORKSPACE);
    EXPECT(rift_score_tiles_noalloc(FAKE, RIFT_BF16, 4, 576, 256, FAKE, 16, 2, 0.37, 0, D, nullptr, D, F, I, I,
                                    nullptr) == RIFT_ERR_SHAPE);

    // ---- budgets (host only): every kept count up to 4096, default and given tiers
    const int32_t lv[4] = {576, 288, 144, 64}, tn[3] = {1, 3, 4};
    for (int K = 0; K <= 4096; K += (K < 64 ? 1 : 37)) {
        std::vector<int32_t> b((size_t)(K > 0 ? K : 1));
        int64_t tot = -1;
        EXPECT(rift_assign_budgets(K, 576, lv, 4, nullptr, 16, b.data(), &tot) == RIFT_OK);
        int64_t s = 0;
        for (int i = 0; i < K; ++i) s += b[(size_t)i];
        EXPECT(s == tot);
        EXPECT(rift_assign_budgets(K, 576, lv, 4, tn, 16, b.data(), nullptr) == RIFT_OK);
    }
    int32_t out8[8];
    const int32_t bad_lv[2] = {576, 576};
    EXPECT(rift_assign_budgets(8, 576, bad_lv, 2, tn, 2, out8, nullptr) == RIFT_ERR_BUDGET);
    EXPECT(rift_assign_budgets(8, 576, lv, 2, nullptr, 16, out8, nullptr) == RIFT_ERR_BUDGET);
    EXPECT(rift_assign_budgets(-1, 576, lv, 4, nullptr, 16, out8, nullptr) != RIFT_OK);

    // ---- Eq. 2 utility policy (host only)
    const int32_t cl[5] = {576, 432, 288, 144, 72};
    const double ap[5] = {0.92, 0.90, 0.85, 0.74, 0.58}, an[5] = {0.95, 0.95, 0.94, 0.93, 0.91};
    const double en[5] = {1.0, 0.75, 0.5, 0.25, 0.125};
    std::vector<float> p(1000);
    for (size_t i = 0; i < p.size(); ++i) p[i] = (float)i / 999.0f;
    std::vector<int32_t> ub(1000);
    int64_t ut = 0;
    EXPECT(rift_assign_budgets_utility(1000, 576, 5, cl, ap, an, en, 0.1, p.data(), ub.data(), &ut) == RIFT_OK);
    EXPECT(ut > 0);
    p[3] = 1.5f;
    EXPECT(rift_assign_budgets_utility(1000, 576, 5, cl, ap, an, en, 0.1, p.data(), ub.data(), &ut) == RIFT_ERR_BUDGET);
    EXPECT(rift_assign_budgets_utility(10, 576, 65, cl, ap, an, en, 0.1, p.data(), ub.data(), &ut) == RIFT_ERR_SHAPE);

    // ---- budget split (host only)
    std::vector<int32_t> dom(1000), ctx(1000);
    EXPECT(rift_split_budgets(1000, 576, ub.data(), 10, 64, dom.data(), ctx.data()) == RIFT_OK);
    for (int i = 0; i < 1000; ++i) EXPECT(dom[(size_t)i] + ctx[(size_t)i] == ub[(size_t)i]);
    EXPECT(rift_split_budgets(4, 576, ub.data(), 65, 64, dom.data(), ctx.data()) == RIFT_ERR_SHAPE);

    // ---- select / merge / compact: validation only
    EXPECT(rift_select_tokens(D, 4, 1025, I, I, 2, I, I, 10, I, nullptr) == RIFT_ERR_SHAPE);
    EXPECT(rift_select_tokens(D, 4, 576, I, I, 2, nullptr, I, 10, I, nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_select_tokens(D, 1 << 22, 1024, I, I, 2, I, I, 10, I, nullptr) == RIFT_ERR_SHAPE);
    EXPECT(rift_merge_workspace_size(100, 576) > 0);
    EXPECT(rift_merge_context(FAKE, RIFT_BF16, 4, 576, 48, I, I, I, I, 2, FAKE, 10, I, ws, 1 << 20, nullptr) ==
           RIFT_ERR_SHAPE);
    EXPECT(rift_compact(FAKE, RIFT_BF16, 4, 576, 4096, I, nullptr, I, 2, nullptr, nullptr, FAKE, 35, FAKE, 32, 0, FAKE,
                        100, I, I, I, nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_compact(FAKE, RIFT_BF16, 4, 576, 4096, I, I, I, 2, nullptr, nullptr, FAKE, 35, FAKE, 32, 2, FAKE, 100,
                        I, I, I, nullptr) == RIFT_ERR_SHAPE);

    // ---- prefill / decode: workspace sizes and validation only
    rift_model_cfg cfg = {4096, 32, 128, 11008, 32, 1e-6f, 10000.0f, RIFT_BF16};
    EXPECT(rift_prefill_workspace_size(&cfg, 18739, 643) > (size_t)18739 * 4096 * 2);
    EXPECT(rift_prefill_workspace_size(nullptr, 18739, 643) == 0);
    rift_layer_weights lw[32];
    for (auto& l : lw) l = {FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE};
    EXPECT(rift_prefill(&cfg, lw, nullptr, RIFT_BF16, I, I, 100, 18739, 643, 35, F, nullptr, ws, 1 << 20, nullptr,
                        nullptr) == RIFT_ERR_NULL);
    EXPECT(rift_prefill(&cfg, lw, FAKE, RIFT_BF16, I, I, 100, 18739, 643, 35, F, nullptr, ws, 64, nullptr, nullptr) ==
           RIFT_ERR_WORKSPACE);
    rift_model_cfg odd = cfg;
    odd.head_dim = 32;
    odd.n_heads = 128;
    EXPECT(rift_prefill(&odd, lw, FAKE, RIFT_BF16, I, I, 100, 18739, 643, 35, F, nullptr, ws, 1 << 20, nullptr,
                        nullptr) == RIFT_ERR_UNSUPPORTED);
    EXPECT(rift_decode_workspace_size(&cfg, 100, 643, 8) > 0);
    EXPECT(rift_decode_step(&cfg, lw, FAKE, I, 100, 18739, 643, 35, FAKE, FAKE, 8, 8, F, ws, 1 << 20, nullptr) ==
           RIFT_ERR_SHAPE);

    printf("%d checks, %d failed\n", g_checks, g_fail);
    return g_fail == 0 ? 0 : 1;
}

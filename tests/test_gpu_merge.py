"""Contextual-token merge (reading R14) and compaction with contextual rows,
against the oracle: every contextual row bit for bit (its bfloat16 or float32
bits), so every assignment (an arg-max of float64 scores taken in the same
canonical order on both sides) agrees."""
import numpy as np
import pytest

import synth
from oracle import rift_oracle as O
from tests.rift_testlib import shared_layout, download_stored, f64, oracle_stage1, torch_mod, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    torch = torch_mod()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    R.load()
    return R


def run_merge(R, X, dtype, kept, dom_offs, dom_sel, kc, cap=None):
    torch = torch_mod()
    n_keep = len(kept)
    coffs = np.concatenate([[0], np.cumsum(kc)]).astype(np.int32)
    cap = int(coffs[-1]) if cap is None else cap
    Xd = upload(X, dtype)
    ctx = torch.zeros(max(1, cap), X.shape[-1], dtype=Xd.dtype, device="cuda")
    st = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    ws = torch.empty(R.rift_merge_workspace_size(n_keep, X.shape[1]), dtype=torch.uint8, device="cuda")
    R.rift_merge_context(Xd, torch.tensor(list(kept) or [0], dtype=torch.int32, device="cuda"),
                         torch.from_numpy(np.asarray(dom_offs, dtype=np.int32)).cuda(),
                         torch.from_numpy(np.asarray(list(dom_sel) or [0], dtype=np.int32)).cuda(),
                         torch.from_numpy(coffs).cuda(), n_keep, ctx[:cap], st, ws)
    torch.cuda.synchronize()
    return download_stored(ctx[:cap], dtype), coffs, int(st.item())


def oracle_ctx(X, dtype, kept, dom_offs, dom_sel, kc):
    """Contextual rows of the oracle, as stored bits (bf16) or float32 values."""
    X64 = f64(X, dtype)
    rows = []
    for rho, tile in enumerate(kept):
        dom = dom_sel[dom_offs[rho]:dom_offs[rho + 1]]
        vals, _, _ = O.merge_context(X64[int(tile)], dom, int(kc[rho]))
        rows.append(vals)
    v = np.concatenate(rows, axis=0) if rows else np.zeros((0, X.shape[-1]))
    return O.round_f32_to_bf16(v.astype(np.float32)) if dtype == "bf16" else v.astype(np.float32)


@pytest.mark.parametrize("name", ["tiny", "scene8"])
def test_merge_parity_scene(R, name):
    w = synth.get(name)
    sc = synth.make_scene(w)
    ref = oracle_stage1(sc, w.keep_count, w.tau)
    kept = list(ref["order"][: ref["n_keep"]])
    budgets = O.assign_budgets(len(kept), w.levels, w.tier_num, w.tier_den)
    split = [O.split_budget(int(c), w.n_v) for c in budgets]
    dom_b, kc = [s[0] for s in split], [s[1] for s in split]
    offs, sel = O.select_tokens(ref["r"], kept, dom_b)
    got, coffs, st = run_merge(R, sc.tokens, w.dtype, kept, offs, sel, kc)
    exp = oracle_ctx(sc.tokens, w.dtype, kept, offs, sel, kc)
    assert st == 0 and got.shape == exp.shape
    assert np.array_equal(got, exp)


def test_merge_edge_counts(R):
    """k_c = 0 (no rows), 1 (the whole remainder), the whole remainder as
    targets, all-zero tokens (score 0), two identical targets (ties to the
    lower), and a ragged d (three LDS slices, the last partial)."""
    rng = np.random.default_rng(21)
    for dtype, d in (("bf16", 64 * 27), ("f32", 96)):
        n_tiles, n_v = 5, 70
        X = synth.store(rng.standard_normal((n_tiles, n_v, d)).astype(np.float32), dtype)
        if dtype == "bf16":
            X[3, 10:20] = 0                      # zero tokens in tile 3
            X[4, 30] = X[4, 5]                   # identical tokens in tile 4
        else:
            X[3, 10:20] = 0.0
            X[4, 30] = X[4, 5]
        kept = [0, 1, 2, 3, 4]
        dom = [[1, 2, 3], [], list(range(0, 70, 2)), [0, 69], [7, 8]]
        kc = [0, 1, 35, 40, 20]                  # tile 2: the 35 remaining tokens are all targets
        offs = np.concatenate([[0], np.cumsum([len(x) for x in dom])]).astype(np.int32)
        sel = np.concatenate([np.asarray(x, np.int32) for x in dom])
        got, coffs, st = run_merge(R, X, dtype, kept, offs, sel, kc)
        exp = oracle_ctx(X, dtype, kept, offs, sel, kc)
        assert st == 0 and np.array_equal(got, exp), dtype


def test_merge_rejects_bad_input(R):
    rng = np.random.default_rng(2)
    X = synth.store(rng.standard_normal((2, 40, 64)).astype(np.float32), "bf16")
    # a repeated dominant index: status set; the good tile is still merged
    offs = np.array([0, 3, 5], np.int32)
    sel = np.array([1, 1, 4, 0, 9], np.int32)
    got, coffs, st = run_merge(R, X, "bf16", [0, 1], offs, sel, [2, 3])
    assert st == 2
    exp = oracle_ctx(X, "bf16", [1], np.array([0, 2]), np.array([0, 9]), [3])
    assert np.array_equal(got[2:], exp)
    # more contextual tokens than remaining tokens
    got, coffs, st = run_merge(R, X, "bf16", [0], np.array([0, 30], np.int32), np.arange(30, dtype=np.int32), [11])
    assert st == 2
    # contextual rows beyond the capacity
    got, coffs, st = run_merge(R, X, "bf16", [0], np.array([0, 2], np.int32), np.array([0, 1], np.int32), [5],
                               cap=4)
    assert st == 2
    # nothing kept
    got, coffs, st = run_merge(R, X, "bf16", [], np.array([0], np.int32), np.zeros(0, np.int32), [])
    assert st == 0


def test_scene_query_with_merge_packs_the_oracle_batch(R):
    """The pipeline with the merge: dominant selection, contextual rows and
    the packed batch equal the oracle's; the prompt lengths are the budgets."""
    torch = torch_mod()
    from paper_2609_29029_amd.pipeline import PrefillShape, SceneQuery
    w = synth.get("scene8")
    sc = synth.make_scene(w)
    m = w.model
    up = lambda a: upload(a, w.dtype)
    layers = [{k: up(v) for k, v in synth.make_layer(w, 0).items()}]
    q = SceneQuery(up(sc.tokens), up(sc.qbank), up(sc.sys), up(sc.qry), layers,
                   PrefillShape(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base),
                   w.keep_count, w.tau, w.levels, w.tier_num, w.tier_den, merge=(10, 64))
    q.run()
    torch.cuda.synchronize()
    assert q.check_status() == [0, 0, 0]
    ref = oracle_stage1(sc, w.keep_count, w.tau)
    kept = list(ref["order"][: ref["n_keep"]])
    budgets = O.assign_budgets(len(kept), w.levels, w.tier_num, w.tier_den)
    split = [O.split_budget(int(c), w.n_v) for c in budgets]
    offs, sel = O.select_tokens(ref["r"], kept, [s[0] for s in split])
    kc = [s[1] for s in split]
    ctx = oracle_ctx(sc.tokens, w.dtype, kept, offs, sel, kc)
    coffs = np.concatenate([[0], np.cumsum(kc)]).astype(np.int32)
    r_packed, r_cu, r_pos = O.compact(sc.tokens, kept, offs, sel, sc.sys, sc.qry, ctx_rows=ctx, ctx_offsets=coffs)
    assert np.array_equal(download_stored(q.packed, w.dtype), r_packed)
    assert np.array_equal(q.cu_seqlens.cpu().numpy(), r_cu)
    assert np.array_equal(q.position_ids.cpu().numpy(), r_pos)
    assert np.array_equal(np.diff(r_cu), np.asarray(budgets) + w.n_sys + w.n_qry)
    assert bool(torch.isfinite(q.hidden).all())


@pytest.mark.slow
def test_merge_full_size_sampled(R):
    """The 400-tile scene: 100 kept tiles (the first 100 ids) at the rank-tier
    budgets, dominant tokens from the oracle's keys of those tiles; the merge
    runs on all 100 and the contextual rows of one tile per budget tier are
    checked bit for bit."""
    w = synth.get("scene20")
    sc = synth.make_scene(w)
    kept = list(range(100))
    X64 = f64(sc.tokens[:100], w.dtype)
    w32 = O.query_direction(f64(sc.qbank, w.dtype))
    r = O.token_keys(X64.reshape(-1, X64.shape[-1]), w32).reshape(100, w.n_v)
    budgets = O.assign_budgets(100, w.levels, w.tier_num, w.tier_den)
    split = [O.split_budget(int(c), w.n_v) for c in budgets]
    kc = [s[1] for s in split]
    offs, sel = O.select_tokens(r, kept, [s[0] for s in split])
    got, coffs, st = run_merge(R, sc.tokens, w.dtype, kept, offs, sel, kc)
    assert st == 0 and got.shape[0] == sum(kc)
    for rho in (0, 6, 24, 99):   # budgets 576, 288, 144, 64
        exp = oracle_ctx(sc.tokens, w.dtype, [rho], offs[rho:rho + 2] - offs[rho], sel[offs[rho]:offs[rho + 1]],
                         [kc[rho]])
        assert np.array_equal(got[coffs[rho]:coffs[rho + 1]], exp), rho


def test_scene_query_with_merge_and_shared_prefix(R):
    """The merge with the system rows shared: the packed batch is the oracle's
    rearranged (prefix once, then each prompt's dominant, contextual and query
    rows), and the hidden states equal those of the per-prompt packing bit for
    bit."""
    torch = torch_mod()
    from paper_2609_29029_amd.pipeline import PrefillShape, SceneQuery
    w = synth.get("scene8")
    sc = synth.make_scene(w)
    m = w.model
    up = lambda a: upload(a, w.dtype)
    layers = [{k: up(v) for k, v in synth.make_layer(w, 0).items()}]
    qs = []
    for shared in (False, True):
        q = SceneQuery(up(sc.tokens), up(sc.qbank), up(sc.sys), up(sc.qry), layers,
                       PrefillShape(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base),
                       w.keep_count, w.tau, w.levels, w.tier_num, w.tier_den, merge=(10, 64), shared_prefix=shared)
        q.run()
        torch.cuda.synchronize()
        assert q.check_status() == [0, 0, 0]
        qs.append(q)
    qa, qb = qs
    n_sys = sc.sys.shape[0]
    pa, cua, posa = download_stored(qa.packed, w.dtype), qa.cu_seqlens.cpu().numpy(), qa.position_ids.cpu().numpy()
    e_packed, e_cu, e_pos = shared_layout(pa, cua, posa, n_sys)
    assert np.array_equal(download_stored(qb.packed, w.dtype), e_packed)
    assert np.array_equal(qb.cu_seqlens.cpu().numpy(), e_cu) and np.array_equal(qb.position_ids.cpu().numpy(), e_pos)
    ha, hb = qa.hidden.cpu().numpy(), qb.hidden.cpu().numpy()
    cub = qb.cu_seqlens.cpu().numpy()
    for i in range(qa.n_keep):
        a0, a1 = int(cua[i]), int(cua[i + 1])
        assert np.array_equal(ha[a0:a0 + n_sys], hb[:n_sys]), i
        assert np.array_equal(ha[a0 + n_sys:a1], hb[int(cub[i + 1]):int(cub[i + 2])]), i

"""GPU parity of Stage 1 (score), Stage 2 (select) and compaction against the
CPU oracle on the same seeded inputs.  Ranks, keys, token indices and packed
buffers are compared bit for bit; normalised scores and cosines within 1e-3."""
import numpy as np
import pytest

import synth
from oracle import rift_oracle as O
from tests.rift_testlib import shared_layout, f64, oracle_stage1, torch_mod, upload, download_stored

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    torch = torch_mod()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    R.load()
    return R


def run_score(R, tokens, qbank, keep_count, tau, sims=True, knn_m=0):
    torch = torch_mod()
    n_tiles, n_v, d = tokens.shape
    nq = qbank.shape[0]
    out = dict(
        token_key=torch.full((n_tiles * n_v,), float("nan"), dtype=torch.float64, device="cuda"),
        token_sim=torch.full((n_tiles * n_v, nq), float("nan"), dtype=torch.float32, device="cuda") if sims else None,
        tile_score=torch.empty(n_tiles, dtype=torch.float64, device="cuda"),
        tile_u=torch.empty(n_tiles, dtype=torch.float32, device="cuda"),
        tile_order=torch.empty(n_tiles, dtype=torch.int32, device="cuda"),
        n_keep=torch.empty(1, dtype=torch.int32, device="cuda"))
    ws = torch.empty(max(256, R.rift_score_workspace_size(n_tiles, n_v, d, knn_m)), dtype=torch.uint8, device="cuda")
    R.rift_score_tiles(tokens, qbank, keep_count, tau, out["token_key"], out["token_sim"],
                       out["tile_score"], out["tile_u"], out["tile_order"], out["n_keep"], ws, knn_m=knn_m)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def check_stage1(got, ref, X64, Q64, sims=True):
    n_tiles, n_v = ref["r"].shape
    key = got["token_key"].reshape(n_tiles, n_v)
    assert np.array_equal(key, ref["r"]), f"keys differ: max |d| = {np.abs(key - ref['r']).max()}"
    assert not np.any(np.signbit(key) & (key == 0))
    assert np.array_equal(got["tile_score"], ref["s"])
    assert list(got["tile_order"]) == list(ref["order"])
    assert int(got["n_keep"][0]) == ref["n_keep"]
    assert np.abs(got["tile_u"].astype(np.float64) - ref["u"]).max() <= 1e-3
    assert np.array_equal(got["tile_u"], ref["u"].astype(np.float32))
    if sims:
        sim_ref = O.token_sims(X64.reshape(n_tiles * n_v, -1), Q64)
        err = np.abs(got["token_sim"].astype(np.float64) - sim_ref).max()
        assert err <= 1e-3, err


@pytest.mark.parametrize("name", ["tiny", "one_tile", "scene8"])
def test_score_parity(R, name):
    w = synth.get(name)
    sc = synth.make_scene(w)
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), w.keep_count, w.tau)
    ref = oracle_stage1(sc, w.keep_count, w.tau)
    check_stage1(got, ref, f64(sc.tokens, w.dtype), f64(sc.qbank, w.dtype))
    if len(sc.planted):
        # the planted query-aligned tiles rank at the top (sanity, not parity)
        top = set(ref["order"][: len(sc.planted)])
        assert top == set(int(t) for t in sc.planted)


@pytest.mark.parametrize("name,m", [("tiny", 1), ("tiny", 6), ("scene8", 6), ("scene8", 3), ("one_tile", 6)])
def test_score_knn_smoothing_parity(R, name, m):
    """Optional smoothing over the m most similar tiles: smoothed scores, u,
    order and kept count bit for bit (keys as without smoothing)."""
    w = synth.get(name)
    sc = synth.make_scene(w)
    X64, Q64 = f64(sc.tokens, w.dtype), f64(sc.qbank, w.dtype)
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), w.keep_count, w.tau, knn_m=m)
    ref = O.scene_query_stage1(X64, Q64, w.keep_count, w.tau, knn_m=m)
    check_stage1(got, ref, X64, Q64)
    # threshold mode on the smoothed scores
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), 0, 0.37, sims=False, knn_m=m)
    ref = O.scene_query_stage1(X64, Q64, 0, 0.37, knn_m=m)
    check_stage1(got, ref, X64, Q64, sims=False)


def test_score_knn_grouped_tiles(R):
    """Tiles built around three orthogonal directions: each tile's neighbours
    are the rest of its group, so with m = 3 its score is its group's mean."""
    rng = np.random.default_rng(21)
    d, n_v = 64, 64
    base = np.zeros((3, d))
    for g in range(3):
        base[g, 8 * g] = 3.0
    X = np.stack([base[i // 4] + 0.05 * rng.standard_normal((n_v, d)) for i in range(12)])
    X = synth.store(X.astype(np.float32), "f32")
    Q = synth.store(rng.standard_normal((16, d)).astype(np.float32), "f32")
    X64, Q64 = f64(X, "f32"), f64(Q, "f32")
    got = run_score(R, upload(X, "f32"), upload(Q, "f32"), 4, 0.0, sims=False, knn_m=3)
    ref = O.scene_query_stage1(X64, Q64, 4, 0.0, knn_m=3)
    check_stage1(got, ref, X64, Q64, sims=False)
    raw = ref["s_raw"]
    for i in range(12):
        assert abs(got["tile_score"][i] - raw[4 * (i // 4):4 * (i // 4) + 4].mean()) <= 1e-15 * 4


def test_score_threshold_mode(R):
    w = synth.get("scene8")
    sc = synth.make_scene(w)
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), 0, 0.37)
    ref = oracle_stage1(sc, 0, 0.37)
    check_stage1(got, ref, f64(sc.tokens, w.dtype), f64(sc.qbank, w.dtype))
    assert ref["n_keep"] >= 1  # the top tile always has u = 1
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), 0, 1.5, sims=False)
    assert int(got["n_keep"][0]) == 0


@pytest.mark.parametrize("dtype,n_tiles,n_v,d,n_bg", [
    ("f32", 3, 100, 64, 0),      # ragged token count, no background phrases
    ("bf16", 5, 37, 512, 15),    # fewer tokens than one wave, ragged 16-blocks
    ("bf16", 2, 1024, 256, 3),   # maximum tokens per tile
    ("bf16", 9, 70, 96, 1),      # d not a multiple of 64
    ("bf16", 3, 45, 800, 2),     # three whole 256-element row chunks and a 1-step tail
    ("bf16", 2, 33, 4064, 1),    # fifteen whole chunks and a 7-step tail, one token past a 32-token set
    ("f32", 2, 33, 800, 2),      # the float32 path on the same ragged shapes
    ("bf16", 4096, 4, 32, 0),    # the maximum tile count (one sort of 4096 keys), minimum d
    ("bf16", 1024, 8, 32, 1),    # the most tiles ranked by counting
    ("bf16", 1025, 40, 64, 2),   # the fewest ranked by sorting; workgroups straddle tiles
])
def test_score_edge_shapes(R, dtype, n_tiles, n_v, d, n_bg):
    rng = np.random.default_rng(n_tiles * 1000 + n_v)
    x32 = rng.standard_normal((n_tiles, n_v, d)).astype(np.float32)
    x32[0, 3] = 0.0                       # an all-zero token scores +0
    q = rng.standard_normal((1 + n_bg, d))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    X, Q = synth.store(x32, dtype), synth.store(q, dtype)
    got = run_score(R, upload(X, dtype), upload(Q, dtype), 2, 0.37)
    X64, Q64 = f64(X, dtype), f64(Q, dtype)
    ref = O.scene_query_stage1(X64, Q64, 2, 0.37)
    check_stage1(got, ref, X64, Q64)
    assert got["token_key"].reshape(n_tiles, n_v)[0, 3] == 0.0


@pytest.mark.parametrize("n_tiles", [300, 1500])
def test_score_threshold_mode_many_tiles(R, n_tiles):
    """Retention by u >= tau over scenes ranked by counting (300 tiles) and
    by sorting (1,500 tiles): order, u and the kept count against the
    oracle."""
    rng = np.random.default_rng(n_tiles)
    x32 = rng.standard_normal((n_tiles, 20, 64)).astype(np.float32)
    q = rng.standard_normal((3, 64))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    x32[7] += 4.0 * q[0]             # a relevant tile (cosine near 0.45), so u spreads over [0, 1]
    X, Q = synth.store(x32, "bf16"), synth.store(q, "bf16")
    got = run_score(R, upload(X, "bf16"), upload(Q, "bf16"), 0, 0.37)
    X64, Q64 = f64(X, "bf16"), f64(Q, "bf16")
    ref = O.scene_query_stage1(X64, Q64, 0, 0.37)
    check_stage1(got, ref, X64, Q64)
    assert got["tile_order"][0] == 7 and int(got["n_keep"][0]) == ref["n_keep"] >= 1


def test_score_equal_tiles(R):
    """Identical tiles: max == min, so every u is 1 and ids break the ties."""
    rng = np.random.default_rng(5)
    tile = rng.standard_normal((64, 128)).astype(np.float32)
    X = synth.store(np.stack([tile] * 6), "bf16")
    q = rng.standard_normal((4, 128))
    Q = synth.store((q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32), "bf16")
    got = run_score(R, upload(X, "bf16"), upload(Q, "bf16"), 0, 0.99)
    assert list(got["tile_order"]) == list(range(6))
    assert np.all(got["tile_u"] == 1.0) and int(got["n_keep"][0]) == 6
    assert np.all(got["tile_score"] == got["tile_score"][0])


# ----------------------------------------------------------------------------- select
def run_select(R, keys, kept, budgets, cap=None, shift=0):
    """`shift` > 0 places the ids, budgets and offsets `shift` int32 entries
    past a 256-byte boundary (no 16-byte vector access)."""
    torch = torch_mod()
    n_tiles, n_v = keys.shape
    n_keep = len(kept)
    total = int(np.clip(budgets, 0, n_v).sum()) if n_keep else 0
    cap = total if cap is None else cap
    key_d = torch.from_numpy(np.ascontiguousarray(keys.reshape(-1))).cuda()
    pad = [0] * shift
    kept_d = torch.tensor(pad + (list(kept) or [0]), dtype=torch.int32, device="cuda")[shift:]
    bud_d = torch.tensor(pad + (list(budgets) or [0]), dtype=torch.int32, device="cuda")[shift:]
    offs_all = torch.full((shift + n_keep + 1,), -7, dtype=torch.int32, device="cuda")
    offs = offs_all[shift:]
    sel = torch.full((max(1, cap),), -7, dtype=torch.int32, device="cuda")
    status = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    R.rift_select_tokens(key_d, n_tiles, n_v, kept_d, bud_d, n_keep, offs, sel[:cap] if cap else sel[:0], status)
    torch.cuda.synchronize()
    assert np.all(offs_all[:shift].cpu().numpy() == -7)   # nothing written before the offsets
    return offs.cpu().numpy(), sel.cpu().numpy()[:cap], int(status.item())


@pytest.mark.parametrize("ties", [False, True])
def test_select_parity_random_keys(R, ties):
    rng = np.random.default_rng(7 + ties)
    n_tiles, n_v = 12, 576
    keys = (rng.integers(-3, 4, size=(n_tiles, n_v)).astype(np.float64) if ties
            else rng.standard_normal((n_tiles, n_v)))
    kept = list(rng.permutation(n_tiles)[:9])
    budgets = [576, 0, 1, 64, 144, 288, 575, 2, 300]
    offs, sel, st = run_select(R, keys, kept, budgets)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0
    assert np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


def test_select_signed_zeros_and_extremes(R):
    """-0.0 and +0.0 compare equal (ties go to the lower index); negative,
    subnormal and huge keys keep their order."""
    rng = np.random.default_rng(11)
    vals = np.array([-0.0, 0.0, 5e-324, -5e-324, 1e300, -1e300, 1.0, -1.0, 2.0 ** -1074, 0.5])
    keys = rng.choice(vals, size=(6, 300))
    kept = [5, 0, 3, 1]
    budgets = [1, 150, 299, 37]
    offs, sel, st = run_select(R, keys, kept, budgets)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


@pytest.mark.parametrize("n_v", [1, 5, 63, 64, 65, 333, 1024])
def test_select_ragged_sizes(R, n_v):
    rng = np.random.default_rng(n_v)
    keys = rng.integers(0, 3, size=(3, n_v)).astype(np.float64)
    budgets = [n_v, n_v // 2, min(n_v, 1)]
    offs, sel, st = run_select(R, keys, [2, 0, 1], budgets)
    r_offs, r_sel = O.select_tokens(keys, [2, 0, 1], budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


@pytest.mark.parametrize("case", ["dup_in_bucket", "crowded_bucket", "infinities", "two_values", "tiny_range"])
def test_select_narrowing_cases(R, case):
    """Inputs aimed at each way the kernel narrows the candidates: repeated
    values inside the bucket of the budget-th key (ranked by index), one value
    bucket holding most keys (the bit-by-bit fallback), infinite keys (no
    value buckets), two distinct values, and keys a few ulps apart."""
    rng = np.random.default_rng(hash(case) % 2**32)
    n_tiles, n_v = 8, 576
    if case == "dup_in_bucket":
        base = rng.standard_normal((n_tiles, n_v)) * 0.02
        keys = np.where(rng.random((n_tiles, n_v)) < 0.5, np.round(base, 3), base)
    elif case == "crowded_bucket":
        keys = 1.0 + rng.standard_normal((n_tiles, n_v)) * 1e-9
        keys[:, ::97] = rng.standard_normal((n_tiles, 6)) * 100.0
    elif case == "infinities":
        keys = rng.standard_normal((n_tiles, n_v))
        keys[:, 3] = np.inf
        keys[:, 7::50] = -np.inf
    elif case == "two_values":
        keys = rng.choice([0.25, -0.75], size=(n_tiles, n_v))
    else:
        keys = 0.5 + rng.integers(-4, 5, size=(n_tiles, n_v)) * 2.0 ** -52
    kept = list(range(n_tiles))
    budgets = [64, 144, 288, 1, 575, 300, 2, 500]
    offs, sel, st = run_select(R, keys, kept, budgets)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


def test_select_many_tiles(R):
    """More kept tiles than one pass of a workgroup's budget loads (8,192):
    every workgroup's base offset and the whole selection against the oracle."""
    rng = np.random.default_rng(21)
    n_tiles, n_v = 9500, 40
    keys = rng.integers(-20, 21, size=(n_tiles, n_v)).astype(np.float64) * 0.125
    kept = list(rng.permutation(n_tiles)[:9000])
    budgets = list(rng.integers(0, n_v + 1, size=9000))
    offs, sel, st = run_select(R, keys, kept, budgets)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


@pytest.mark.parametrize("n_keep,n_v", [(1024, 48), (1025, 48), (8192, 24), (8193, 24), (8300, 700)])
def test_select_large_call_paths(R, n_keep, n_v):
    """Up to 8,192 kept tiles one launch reads every budget (four tiles a
    workgroup up to 1,024, eight above); above, two launches check the call
    and find the offsets chunk by chunk and the selection reads its offset.
    Both sides of each switch, and keys per lane above 9 (n_v > 576) on the
    chunked path."""
    rng = np.random.default_rng(n_keep + n_v)
    n_tiles = n_keep + 7
    keys = rng.integers(-30, 31, size=(n_tiles, n_v)).astype(np.float64) * 0.25
    kept = list(rng.permutation(n_tiles)[:n_keep])
    budgets = list(rng.integers(0, n_v + 1, size=n_keep))
    offs, sel, st = run_select(R, keys, kept, budgets)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


@pytest.mark.parametrize("n_keep,n_v,shift", [(9216, 576, 0), (8200, 1024, 0), (10241, 576, 1), (8193, 333, 3)])
def test_select_chunked_full_tiles(R, n_keep, n_v, shift):
    """The chunked path on tiles of exactly 9 and 16 keys a lane (no key past
    the tile's end) with normal keys, a whole number of 1,024-tile chunks and
    a one-tile last chunk; ids, budgets and offsets off the 16-byte grid."""
    rng = np.random.default_rng(n_keep * 7 + n_v)
    n_tiles = n_keep + 3
    keys = rng.standard_normal((n_tiles, n_v))
    kept = list(rng.permutation(n_tiles)[:n_keep])
    budgets = list(rng.integers(0, n_v + 1, size=n_keep))
    offs, sel, st = run_select(R, keys, kept, budgets, shift=shift)
    r_offs, r_sel = O.select_tokens(keys, kept, budgets)
    assert st == 0 and np.array_equal(offs, r_offs) and np.array_equal(sel, r_sel)


@pytest.mark.parametrize("flaw", ["budget", "negative", "tile", "capacity", "first", "chunk_start"])
def test_select_large_call_rejects(R, flaw):
    """The chunked path reports a bad call like the one-launch path: status
    RIFT_ERR_BUDGET, every offset 0, nothing written to the selection; flaws
    in a chunk's first entry (whose slot carries the chunk's total) too."""
    rng = np.random.default_rng(5)
    n_tiles, n_v, n_keep = 17000, 20, 16500   # the chunked path, 17 chunks
    keys = rng.standard_normal((n_tiles, n_v))
    kept = list(rng.permutation(n_tiles)[:n_keep])
    budgets = [int(b) for b in rng.integers(0, n_v + 1, size=n_keep)]
    cap = None
    if flaw == "budget":
        budgets[16390] = n_v + 1
    elif flaw == "negative":
        budgets[40] = -3
    elif flaw == "tile":
        kept[16499] = n_tiles
    elif flaw == "first":
        budgets[0] = n_v + 1
    elif flaw == "chunk_start":
        kept[2048] = -1
    else:
        cap = sum(budgets) - 1
    offs, sel, st = run_select(R, keys, kept, budgets, cap=cap)
    assert st == 4 and np.all(offs == 0)
    assert np.all(sel == -7)


def test_select_rejects_bad_budgets(R):
    keys = np.zeros((2, 10))
    for budgets, kept in (([11, 1], [0, 1]), ([-1, 1], [0, 1]), ([1, 1], [0, 2])):
        offs, sel, st = run_select(R, keys, kept, budgets, cap=12)
        assert st == 4 and np.all(offs == 0)              # RIFT_ERR_BUDGET
        assert np.all(sel == -7)                          # nothing written
    offs, sel, st = run_select(R, keys, [0, 1], [5, 5], cap=9)   # total above capacity
    assert st == 4 and np.all(sel == -7)


def test_select_empty(R):
    offs, sel, st = run_select(R, np.zeros((2, 10)), [], [])
    assert st == 0 and list(offs) == [0]


# ----------------------------------------------------------------------------- compact
def run_compact(R, X, dtype, kept, offs, sel, sysr, qry, rows=None, shared=False):
    torch = torch_mod()
    n_keep = len(kept)
    if shared:
        T = sysr.shape[0] + n_keep * qry.shape[0] + int(offs[-1])
    else:
        T = n_keep * (sysr.shape[0] + qry.shape[0]) + int(offs[-1])
    rows = T if rows is None else rows
    Xd = upload(X, dtype)
    packed = torch.zeros(rows, X.shape[-1], dtype=Xd.dtype, device="cuda")
    cu = torch.full((n_keep + (2 if shared else 1),), -7, dtype=torch.int32, device="cuda")
    pos = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    kept_d = torch.tensor(list(kept) or [0], dtype=torch.int32, device="cuda")
    offs_d = torch.tensor(list(offs), dtype=torch.int32, device="cuda")
    sel_d = torch.tensor(list(sel) or [0], dtype=torch.int32, device="cuda")
    R.rift_compact(Xd, kept_d, offs_d, sel_d, n_keep, upload(sysr, dtype), upload(qry, dtype),
                   packed, cu, pos, st, shared_prefix=shared)
    torch.cuda.synchronize()
    return download_stored(packed, dtype), cu.cpu().numpy(), pos.cpu().numpy(), int(st.item())




@pytest.mark.parametrize("name", ["tiny", "scene8"])
def test_compact_parity(R, name):
    w = synth.get(name)
    sc = synth.make_scene(w)
    ref = oracle_stage1(sc, w.keep_count, w.tau)
    kept = list(ref["order"][: ref["n_keep"]])
    budgets = O.assign_budgets(len(kept), w.levels, w.tier_num, w.tier_den)
    offs, sel = O.select_tokens(ref["r"], kept, budgets)
    packed, cu, pos, st = run_compact(R, sc.tokens, w.dtype, kept, offs, sel, sc.sys, sc.qry)
    r_packed, r_cu, r_pos = O.compact(sc.tokens, kept, offs, sel, sc.sys, sc.qry)
    assert st == 0
    assert np.array_equal(packed, r_packed) and np.array_equal(cu, r_cu) and np.array_equal(pos, r_pos)


def test_compact_edges(R):
    rng = np.random.default_rng(3)
    X = synth.store(rng.standard_normal((4, 20, 64)).astype(np.float32), "bf16")
    sysr = synth.store(rng.standard_normal((3, 64)).astype(np.float32), "bf16")
    qry = synth.store(rng.standard_normal((2, 64)).astype(np.float32), "bf16")
    # zero-budget tile, full-budget tile
    kept, offs, sel = [3, 1], np.array([0, 0, 20]), np.arange(20)
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry)
    r = O.compact(X, kept, offs, sel, sysr, qry)
    assert st == 0 and np.array_equal(packed, r[0]) and np.array_equal(cu, r[1]) and np.array_equal(pos, r[2])
    # nothing kept
    packed, cu, pos, st = run_compact(R, X, "bf16", [], np.array([0]), np.zeros(0, int), sysr, qry)
    assert st == 0 and list(cu) == [0]
    # capacity too small: status set, no row beyond capacity written
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry, rows=10)
    assert st == 2
    # token index out of range
    packed, cu, pos, st = run_compact(R, X, "bf16", [0], np.array([0, 2]), np.array([1, 20]), sysr, qry)
    assert st == 2
    # a budget (offset step) larger than n_v
    packed, cu, pos, st = run_compact(R, X, "bf16", [0], np.array([0, 21]), np.arange(21) % 20, sysr, qry)
    assert st == 2
    # offsets that decrease: reported, and no prompt reads past sel_offsets[n_keep] selected indices
    packed, cu, pos, st = run_compact(R, X, "bf16", [0, 1], np.array([0, 15, 5]), np.arange(5), sysr, qry, rows=40)
    assert st == 2
    # a packed buffer longer than the batch: rows past T untouched
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry, rows=40)
    r = O.compact(X, kept, offs, sel, sysr, qry)
    assert st == 0 and np.array_equal(packed[:30], r[0]) and np.all(packed[30:] == 0) and np.all(pos[30:] == -7)


@pytest.mark.parametrize("shared", [False, True])
def test_compact_many_prompts(R, shared):
    """More prompts than the kernel stages in LDS (4096): the prompt of each row
    is then searched in the offsets in global memory (per-prompt and shared
    system rows)."""
    rng = np.random.default_rng(11)
    n_tiles, n_v = 5000, 4
    X = synth.store(rng.standard_normal((n_tiles, n_v, 64)).astype(np.float32), "bf16")
    sysr = synth.store(rng.standard_normal((1, 64)).astype(np.float32), "bf16")
    qry = synth.store(rng.standard_normal((2, 64)).astype(np.float32), "bf16")
    kept = list(rng.permutation(n_tiles)[:4500])
    budgets = rng.integers(0, n_v + 1, size=len(kept))
    offs = np.concatenate([[0], np.cumsum(budgets)])
    sel = np.concatenate([np.sort(rng.permutation(n_v)[:b]) for b in budgets]).astype(np.int64)
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry, shared=shared)
    r_packed, r_cu, r_pos = O.compact(X, kept, offs, sel, sysr, qry)
    if shared:
        r_packed, r_cu, r_pos = shared_layout(r_packed, r_cu, r_pos, sysr.shape[0])
    assert st == 0
    assert np.array_equal(packed, r_packed) and np.array_equal(cu, r_cu) and np.array_equal(pos, r_pos)


@pytest.mark.slow
def test_score_knn_smoothing_full_size(R):
    """The 400-tile scene with 6-neighbour smoothing, every score and rank bit
    for bit."""
    w = synth.get("scene20")
    sc = synth.make_scene(w)
    X64, Q64 = f64(sc.tokens, w.dtype), f64(sc.qbank, w.dtype)
    got = run_score(R, upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype), w.keep_count, w.tau,
                    sims=False, knn_m=6)
    ref = O.scene_query_stage1(X64, Q64, w.keep_count, w.tau, knn_m=6)
    check_stage1(got, ref, X64, Q64, sims=False)


@pytest.mark.parametrize("name", ["tiny", "scene8"])
def test_compact_shared_prefix(R, name):
    """Shared-prefix layout: the system rows once at the front (sequence 0),
    each prompt's own rows after them at positions n_sys onwards; bit for bit
    the oracle's packing rearranged."""
    w = synth.get(name)
    sc = synth.make_scene(w)
    ref = oracle_stage1(sc, w.keep_count, w.tau)
    kept = list(ref["order"][: ref["n_keep"]])
    budgets = O.assign_budgets(len(kept), w.levels, w.tier_num, w.tier_den)
    offs, sel = O.select_tokens(ref["r"], kept, budgets)
    packed, cu, pos, st = run_compact(R, sc.tokens, w.dtype, kept, offs, sel, sc.sys, sc.qry, shared=True)
    e_packed, e_cu, e_pos = shared_layout(*O.compact(sc.tokens, kept, offs, sel, sc.sys, sc.qry), sc.sys.shape[0])
    assert st == 0
    assert np.array_equal(packed, e_packed) and np.array_equal(cu, e_cu) and np.array_equal(pos, e_pos)


def test_compact_shared_prefix_edges(R):
    rng = np.random.default_rng(4)
    X = synth.store(rng.standard_normal((4, 20, 64)).astype(np.float32), "bf16")
    sysr = synth.store(rng.standard_normal((3, 64)).astype(np.float32), "bf16")
    qry = synth.store(rng.standard_normal((2, 64)).astype(np.float32), "bf16")
    kept, offs, sel = [3, 1], np.array([0, 0, 20]), np.arange(20)
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry, shared=True)
    e = shared_layout(*O.compact(X, kept, offs, sel, sysr, qry), 3)
    assert st == 0 and np.array_equal(packed, e[0]) and np.array_equal(cu, e[1]) and np.array_equal(pos, e[2])
    # nothing kept: the prefix alone
    packed, cu, pos, st = run_compact(R, X, "bf16", [], np.array([0]), np.zeros(0, int), sysr, qry, shared=True)
    assert st == 0 and list(cu) == [0, 3] and np.array_equal(packed, sysr) and list(pos) == [0, 1, 2]
    # capacity too small
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr, qry, rows=10, shared=True)
    assert st == 2
    # no system rows: an empty prefix sequence
    packed, cu, pos, st = run_compact(R, X, "bf16", kept, offs, sel, sysr[:0], qry, shared=True)
    e = O.compact(X, kept, offs, sel, sysr[:0], qry)
    assert st == 0 and np.array_equal(packed, e[0]) and list(cu) == [0] + list(e[1]) and np.array_equal(pos, e[2])

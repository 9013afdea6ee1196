"""Non-finite input checks: rift_check_finite on its own, and the debug mode
in which rift_score_tiles, rift_select_tokens and rift_prefill scan their
floating-point inputs first and return RIFT_ERR_NONFINITE, enqueuing nothing
else, when one holds NaN or infinity."""
import numpy as np
import pytest

import synth
from tests.rift_testlib import torch_mod, upload, upload_layer

pytestmark = pytest.mark.gpu

NONFINITE = 7


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    torch = torch_mod()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    R.load()
    return R


@pytest.fixture
def debug(R):
    prev = R.rift_set_debug(True)
    yield
    R.rift_set_debug(prev)


def check(R, x):
    torch = torch_mod()
    st = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    R.rift_check_finite(x, st)
    torch.cuda.synchronize()
    return int(st.item())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_check_finite_planted_values(R, dtype):
    torch = torch_mod()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    n = 100_003   # not a multiple of the 16-byte words
    x = torch.randn(n, device="cuda").to(tdt)
    assert check(R, x) == 0
    assert check(R, x[:0]) == 0
    big = torch.finfo(tdt).max
    x[17] = big
    x[18] = -big
    x[19] = torch.finfo(tdt).tiny / 4   # subnormal: finite
    assert check(R, x) == 0
    for pos in (0, 1, n // 2, n - 1):
        for bad in (float("nan"), float("inf"), float("-inf")):
            y = x.clone()
            y[pos] = bad
            assert check(R, y) == NONFINITE, (pos, bad)
            # a view that starts off a 16-byte boundary takes the element-wise path
            if pos >= 1:
                assert check(R, y[1:]) == NONFINITE, (pos, bad)
    y = x.clone()
    y[0] = float("nan")
    assert check(R, y[1:]) == 0


def score_call(R, tokens, qbank):
    torch = torch_mod()
    n_tiles, n_v, d = tokens.shape
    key = torch.full((n_tiles * n_v,), -5.0, dtype=torch.float64, device="cuda")
    score = torch.empty(n_tiles, dtype=torch.float64, device="cuda")
    u = torch.empty(n_tiles, dtype=torch.float32, device="cuda")
    order = torch.empty(n_tiles, dtype=torch.int32, device="cuda")
    nk = torch.empty(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(R.rift_score_workspace_size(n_tiles, n_v, d), dtype=torch.uint8, device="cuda")
    try:
        R.rift_score_tiles(tokens, qbank, 2, 0.0, key, None, score, u, order, nk, ws)
        status = 0
    except R.RiftError as e:
        status = e.status
    torch.cuda.synchronize()
    return status, key


def test_debug_mode_score(R, debug):
    w = synth.get("tiny")
    sc = synth.make_scene(w)
    tokens, qbank = upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype)
    st, key = score_call(R, tokens, qbank)
    assert st == 0 and bool((key != -5.0).all())
    bad = tokens.clone()
    bad[2, 100, 7] = float("inf")
    st, key = score_call(R, bad, qbank)
    assert st == NONFINITE and bool((key == -5.0).all())      # nothing else ran
    badq = qbank.clone()
    badq[3, 0] = float("nan")
    st, key = score_call(R, tokens, badq)
    assert st == NONFINITE and bool((key == -5.0).all())
    # debug mode off: the call runs (the infinity propagates into the results)
    R.rift_set_debug(False)
    st, key = score_call(R, bad, qbank)
    assert st == 0


def test_nonfinite_token_with_smoothing_keeps_indices_in_range(R):
    """Debug mode off, six-neighbour smoothing, one infinite token: that
    tile's embedding, similarities and score are NaN.  The neighbour search
    still picks a tile in range every round (a NaN similarity ranks last), and
    the NaN score sorts behind every finite one, so the order stays a
    permutation of the tile ids with the bad tile last."""
    torch = torch_mod()
    prev = R.rift_set_debug(False)
    try:
        w = synth.get("scene8")
        sc = synth.make_scene(w)
        tokens, qbank = upload(sc.tokens, w.dtype), upload(sc.qbank, w.dtype)
        bad_tile = 5
        tokens[bad_tile, 100, 7] = float("inf")
        n_tiles, n_v, d = tokens.shape
        key = torch.empty(n_tiles * n_v, dtype=torch.float64, device="cuda")
        score = torch.empty(n_tiles, dtype=torch.float64, device="cuda")
        u = torch.empty(n_tiles, dtype=torch.float32, device="cuda")
        order = torch.empty(n_tiles, dtype=torch.int32, device="cuda")
        nk = torch.empty(1, dtype=torch.int32, device="cuda")
        ws = torch.empty(R.rift_score_workspace_size(n_tiles, n_v, d, 6), dtype=torch.uint8, device="cuda")
        R.rift_score_tiles(tokens, qbank, 16, 0.0, key, None, score, u, order, nk, ws, knn_m=6)
        torch.cuda.synchronize()
        o = order.cpu().numpy()
        s = score.cpu().numpy()
        assert sorted(o.tolist()) == list(range(n_tiles))
        assert o[-1] == bad_tile and int(nk.item()) == 16
        assert not np.isfinite(s[bad_tile])
        assert np.isfinite(np.delete(s, bad_tile)).all()
    finally:
        R.rift_set_debug(prev)


def test_debug_mode_select(R, debug):
    torch = torch_mod()
    rng = np.random.default_rng(1)
    keys = rng.standard_normal((3, 40))
    keys[1, 5] = np.nan
    key_d = torch.from_numpy(keys.reshape(-1)).cuda()
    kept = torch.tensor([0, 2], dtype=torch.int32, device="cuda")
    budgets = torch.tensor([4, 4], dtype=torch.int32, device="cuda")
    offs = torch.full((3,), -7, dtype=torch.int32, device="cuda")
    sel = torch.full((8,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(R.RiftError) as ei:
        R.rift_select_tokens(key_d, 3, 40, kept, budgets, 2, offs, sel, st)
    torch.cuda.synchronize()
    assert ei.value.status == NONFINITE and int(st.item()) == NONFINITE
    assert bool((offs == -7).all()) and bool((sel == -7).all())   # nothing else ran


def test_debug_mode_prefill(R, debug):
    torch = torch_mod()
    w = synth.get("tiny")
    m = w.model
    W = upload_layer(synth.make_layer(w, 0), w.dtype)
    T, L = 40, 40
    x = torch.randn(T, m.d, device="cuda").to(torch.float32 if w.dtype == "f32" else torch.bfloat16)
    cu = torch.tensor([0, T], dtype=torch.int32, device="cuda")
    pos = torch.arange(T, dtype=torch.int32, device="cuda")
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base,
                      R.RIFT_BF16 if w.dtype == "bf16" else R.RIFT_F32)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, L), dtype=torch.uint8, device="cuda")
    out = torch.full((T, m.d), -5.0, dtype=torch.float32, device="cuda")
    R.rift_prefill(cfg, [W], x, cu, pos, 1, L, out, ws)
    torch.cuda.synchronize()
    assert bool((out != -5.0).all())
    Wbad = dict(W)
    Wbad["w_down"] = W["w_down"].clone()
    Wbad["w_down"][3, 5] = float("inf")
    out.fill_(-5.0)
    with pytest.raises(R.RiftError) as ei:
        R.rift_prefill(cfg, [Wbad], x, cu, pos, 1, L, out, ws)
    torch.cuda.synchronize()
    assert ei.value.status == NONFINITE and bool((out == -5.0).all())
    xbad = x.clone()
    xbad[T - 1, m.d - 1] = float("nan")
    with pytest.raises(R.RiftError) as ei:
        R.rift_prefill(cfg, [W], xbad, cu, pos, 1, L, out, ws)
    assert ei.value.status == NONFINITE

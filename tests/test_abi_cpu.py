"""The C-ABI library on the CPU: it loads, exports every symbol include/rift.h
declares, and its host-side logic (argument validation, budget assignment,
workspace sizes) behaves as documented.  No kernel is launched here: every
call below returns before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import rift_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    if not R.lib_available():
        from paper_2609_29029_amd.build import build
        build()
    R.load()
    return R


def declared_symbols():
    with open(os.path.join(ROOT, "include", "rift.h")) as f:
        text = f.read()
    return re.findall(r"RIFT_API\s+[\w\s\*]+?\b(rift_\w+)\s*\(", text)


def test_library_exports_every_declared_symbol(R):
    L = R.load()
    names = declared_symbols()
    assert len(names) == 18
    assert tuple(names) == R.EXPORTS
    for n in names:
        assert hasattr(L, n), n
    assert L.rift_abi_version() == 7
    assert L.rift_status_string(4).decode().startswith("budget")


def test_only_abi_symbols_are_exported(R):
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", R.LIB_PATH], capture_output=True, text=True).stdout
    text_syms = [ln.split()[-1] for ln in out.splitlines() if " T " in ln]
    assert sorted(s for s in text_syms if s.startswith("rift_")) == sorted(R.EXPORTS)


@pytest.mark.parametrize("K", [0, 1, 2, 7, 16, 31, 100, 400])
def test_assign_budgets_matches_oracle(R, K):
    lv, num, den = (576, 288, 144, 64), (1, 3, 4), 16
    got, tot = R.rift_assign_budgets(K, 576, lv, num, den)
    ref = O.assign_budgets(K, lv, num, den)
    assert np.array_equal(got, ref) and tot == int(ref.sum())
    got2, _ = R.rift_assign_budgets(K, 576, lv, None, 16)   # library default tiers
    assert np.array_equal(got2, ref)


def test_assign_budgets_rejects_bad_tables(R):
    from paper_2609_29029_amd import RiftError
    bad = [
        dict(levels=[576, 576], tier_num=[1], tier_den=2),       # not strictly descending
        dict(levels=[700, 64], tier_num=[1], tier_den=2),        # above n_v
        dict(levels=[576, 0], tier_num=[1], tier_den=2),         # below 1
        dict(levels=[576, 64], tier_num=[3], tier_den=2),        # fractions above 1
        dict(levels=[576, 64], tier_num=[-1], tier_den=2),
        dict(levels=[576, 64], tier_num=None, tier_den=16),      # default needs 4 levels
        dict(levels=[576, 64], tier_num=[1], tier_den=0),
    ]
    for b in bad:
        with pytest.raises(RiftError) as e:
            R.rift_assign_budgets(8, 576, b["levels"], b["tier_num"], b["tier_den"])
        assert e.value.status == 4
    with pytest.raises(RiftError):
        R.rift_assign_budgets(-1, 576, [64], [], 16)


FAKE = 0x1000  # a non-NULL value; never dereferenced (validation fails first)


def test_score_validation(R):
    L = R.load()
    args = dict(tokens=FAKE, dt=1, n_tiles=4, n_v=576, d=256, qb=FAKE, n_bg=15, keep=2, tau=0.37, knn=0,
                key=FAKE, sim=None, s=FAKE, u=FAKE, order=FAKE, nk=FAKE, ws=0x10000, wsb=1 << 20)

    def call(**over):
        a = dict(args, **over)
        return L.rift_score_tiles(a["tokens"], a["dt"], a["n_tiles"], a["n_v"], a["d"], a["qb"], a["n_bg"],
                                  a["keep"], a["tau"], a["knn"], a["key"], a["sim"], a["s"], a["u"], a["order"],
                                  a["nk"], a["ws"], a["wsb"], None)
    assert call(tokens=None) == 1
    assert call(key=None) == 1
    assert call(ws=None) == 1
    assert call(dt=7) == 3
    for bad in (dict(n_tiles=0), dict(n_tiles=4097), dict(n_v=0), dict(n_v=1025), dict(d=48),
                dict(d=16416), dict(n_bg=16), dict(n_bg=-1), dict(keep=-1), dict(tau=float("nan")),
                dict(knn=-1)):
        assert call(**bad) == 2, bad
    assert call(ws=0x10010) == 5              # misaligned workspace
    assert call(wsb=16) == 5                  # too small
    assert R.rift_score_workspace_size(4, 576, 4096) >= 4096 * 4
    # smoothing needs inverse norms, embeddings, their dot products and the smoothed scores
    need = R.rift_score_workspace_size(4, 576, 256, 6)
    assert need >= 256 * 4 + 4 * 576 * 8 + 4 * 256 * 4 + 4 * 4 * 8 + 4 * 8
    assert call(knn=6, wsb=need - 1) == 5
    assert R.rift_score_workspace_size(4, 576, 4096, -1) == 0


def test_score_noalloc_validation_and_scratch_limit(R):
    """The workspace-free scoring call validates like rift_score_tiles and
    rejects, before any device work, a call whose workspace would exceed the
    static scratch (16 MiB)."""
    L = R.load()
    args = dict(tokens=FAKE, dt=1, n_tiles=4, n_v=576, d=256, qb=FAKE, n_bg=15, keep=2, tau=0.37, knn=0,
                key=FAKE, sim=None, s=FAKE, u=FAKE, order=FAKE, nk=FAKE)

    def call(**over):
        a = dict(args, **over)
        return L.rift_score_tiles_noalloc(a["tokens"], a["dt"], a["n_tiles"], a["n_v"], a["d"], a["qb"],
                                          a["n_bg"], a["keep"], a["tau"], a["knn"], a["key"], a["sim"], a["s"],
                                          a["u"], a["order"], a["nk"], None)
    assert call(tokens=None) == 1 and call(order=None) == 1
    assert call(dt=7) == 3
    for bad in (dict(n_tiles=0), dict(n_tiles=4097), dict(n_v=1025), dict(d=48), dict(n_bg=16),
                dict(keep=-1), dict(tau=float("nan")), dict(knn=-1)):
        assert call(**bad) == 2, bad
    limit = 16 << 20
    # 4096 tiles of 1024 tokens with smoothing need far more than the scratch
    assert R.rift_score_workspace_size(4096, 1024, 4096, 6) > limit
    assert call(n_tiles=4096, n_v=1024, d=4096, knn=6) == 5
    # the largest scene without smoothing, and 400 x 576 x 4096 with it, fit
    assert R.rift_score_workspace_size(4096, 1024, 16384, 0) <= limit
    assert R.rift_score_workspace_size(400, 576, 4096, 6) <= limit


def test_select_and_compact_validation(R):
    L = R.load()
    # select: NULL outputs, shapes
    assert L.rift_select_tokens(FAKE, 4, 576, FAKE, FAKE, 2, None, FAKE, 10, FAKE, None) == 1
    assert L.rift_select_tokens(FAKE, 4, 576, FAKE, FAKE, 2, FAKE, FAKE, 10, None, None) == 1
    assert L.rift_select_tokens(None, 4, 576, FAKE, FAKE, 2, FAKE, FAKE, 10, FAKE, None) == 1
    assert L.rift_select_tokens(FAKE, 4, 1025, FAKE, FAKE, 2, FAKE, FAKE, 10, FAKE, None) == 2
    assert L.rift_select_tokens(FAKE, 4, 576, FAKE, FAKE, 5, FAKE, FAKE, 10, FAKE, None) == 2
    assert L.rift_select_tokens(FAKE, 4, 576, FAKE, FAKE, 2, FAKE, None, 10, FAKE, None) == 1
    assert L.rift_select_tokens(FAKE, 1 << 22, 1024, FAKE, FAKE, 2, FAKE, FAKE, 10, FAKE, None) == 2
    assert L.rift_select_tokens(FAKE, 4, 576, FAKE, FAKE, 2, FAKE, FAKE, 1 << 31, FAKE, None) == 2
    # compact
    c = L.rift_compact
    assert c(FAKE, 1, 4, 576, 4096, FAKE, None, FAKE, 2, None, None, FAKE, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE, FAKE, None) == 1
    assert c(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, 2, None, None, None, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE, FAKE, None) == 1
    assert c(FAKE, 9, 4, 576, 4096, FAKE, FAKE, FAKE, 2, None, None, FAKE, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE, FAKE, None) == 3
    assert c(FAKE, 1, 4, 576, 4, FAKE, FAKE, FAKE, 2, None, None, FAKE, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE, FAKE, None) == 2
    assert c(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, -1, None, None, FAKE, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE, FAKE, None) == 2
    # two waves per packed row: at most 2^25 rows
    assert c(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, 2, None, None, FAKE, 35, FAKE, 32, 0, FAKE, (1 << 25) + 1, FAKE, FAKE, FAKE,
             None) == 2
    # shared_prefix is 0 or 1
    assert c(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, 2, None, None, FAKE, 35, FAKE, 32, 2, FAKE, 100, FAKE, FAKE, FAKE,
             None) == 2


def test_prefill_validation_and_workspace(R):
    L = R.load()
    cfg = R.model_cfg(4096, 32, 128, 11008, 1, 1e-6, 10000.0, R.RIFT_BF16)
    ws = R.rift_prefill_workspace_size(cfg, 22204, 643)
    # rope table + h, q, k, v [T][d] + a [T][ffn], bf16, + the attention work
    # list: 8-byte entries, (heads / 8) per 128-row block and per sequence
    # (at most T sequences)
    expect = (643 * 64 * 8 + 4 * 22204 * 4096 * 2 + 22204 * 11008 * 2
              + (32 // 8) * ((22204 + 127) // 128 + 22204) * 8)
    assert expect <= ws <= expect + 8 * 256
    # no work list when the head count is not a multiple of 8
    cfg12 = R.model_cfg(768, 12, 64, 2048, 1, 1e-6, 10000.0, R.RIFT_BF16)
    ws12 = R.rift_prefill_workspace_size(cfg12, 1000, 200)
    expect12 = 200 * 32 * 8 + 4 * 1000 * 768 * 2 + 1000 * 2048 * 2
    assert expect12 <= ws12 <= expect12 + 8 * 256
    lw = (R.LayerWeights * 1)(R.LayerWeights(*([FAKE] * 9)))

    def call(c, T=10, n_seq=1, max_len=10, x=FAKE, x_dt=1, wsb=1 << 40, n_prefix=0):
        return L.rift_prefill(ctypes.byref(c), lw, x, x_dt, FAKE, FAKE, n_seq, T, max_len, n_prefix, FAKE, None,
                              0x10000, wsb, None, None)
    assert call(cfg, T=0) == 0                              # nothing to do
    assert call(cfg, x=None) == 1
    assert call(cfg, x_dt=5) == 3
    assert call(cfg, max_len=0) == 2 and call(cfg, n_seq=-1) == 2
    assert call(cfg, wsb=100) == 5
    # a shared prefix: within the batch and max_seqlen, with at least one sequence
    assert call(cfg, n_prefix=-1) == 2 and call(cfg, n_prefix=11) == 2
    assert call(cfg, T=20, max_len=10, n_prefix=11) == 2 and call(cfg, n_seq=0, n_prefix=3) == 2
    for bad in (R.model_cfg(4096, 128, 32, 11008, 1, 1e-6, 1e4, R.RIFT_BF16),   # head_dim 64 or 128 only
                R.model_cfg(4160, 32, 130, 11008, 1, 1e-6, 1e4, R.RIFT_BF16),
                R.model_cfg(1088, 17, 64, 2816, 1, 1e-6, 1e4, R.RIFT_BF16),     # bf16: d % 256
                R.model_cfg(256, 4, 64, 690, 1, 1e-6, 1e4, R.RIFT_F32)):        # ffn % 16
        assert call(bad) == 8   # RIFT_ERR_UNSUPPORTED
    assert call(R.model_cfg(4096, 31, 128, 11008, 1, 1e-6, 1e4, R.RIFT_BF16)) == 2
    assert call(R.model_cfg(4096, 32, 128, 11008, 1, 1e-6, 1e4, 9)) == 3
    assert R.rift_prefill_workspace_size(R.model_cfg(4096, 128, 32, 11008, 1, 1e-6, 1e4, R.RIFT_BF16), 10, 10) == 0
    # bf16 with 64-dimensional heads is a supported shape
    assert R.rift_prefill_workspace_size(R.model_cfg(4096, 64, 64, 11008, 1, 1e-6, 1e4, R.RIFT_BF16), 10, 10) > 0


def test_utility_budgets_match_oracle(R):
    from oracle import rift_oracle as O
    C5 = [576, 432, 288, 144, 72]
    AP = [0.92, 0.90, 0.85, 0.74, 0.58]
    AN = [0.95, 0.95, 0.94, 0.93, 0.91]
    EN = [c / 576 for c in C5]
    rng = np.random.default_rng(31)
    p = np.concatenate([[0.0, 1.0, 0.5], rng.uniform(0, 1, 200)]).astype(np.float32)
    for lam in (0.0, 0.1, 0.37, 100.0):
        b, tot = R.rift_assign_budgets_utility(p, C5, AP, AN, EN, lam, 576)
        ref = O.utility_budgets(p.astype(np.float64), C5, AP, AN, EN, lam)
        assert np.array_equal(b, ref) and tot == int(ref.sum())
    # validation
    L = R.load()
    import ctypes
    with pytest.raises(R.RiftError):
        R.rift_assign_budgets_utility([1.5], C5, AP, AN, EN, 0.1, 576)
    with pytest.raises(R.RiftError):
        R.rift_assign_budgets_utility([0.5], [577] + C5[1:], AP, AN, EN, 0.1, 576)
    with pytest.raises(R.RiftError):
        R.rift_assign_budgets_utility([0.5], C5, AP, AN, EN, float("inf"), 576)
    b, tot = R.rift_assign_budgets_utility([], C5, AP, AN, EN, 0.1, 576)
    assert b.size == 0 and tot == 0


def test_calibration_library_loads_and_rejects_bad_arguments(R):
    """libriftcalib.so (the benchmark's MFMA-ceiling aid, off the Rift path)
    loads and validates its arguments on the host; nothing is launched."""
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2609_29029_amd", "libriftcalib.so"))
    f = L.rift_calib_mfma_bf16
    f.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    p = ctypes.c_void_p(16)
    assert f(3, p, p, 1, 8, None) == -1        # unknown form
    assert f(-1, p, p, 1, 8, None) == -1
    assert f(0, None, p, 1, 8, None) == -1     # null source
    assert f(0, p, p, 0, 8, None) == -1        # no workgroups
    assert f(1, p, p, 1, 12, None) == -1       # iterations not a multiple of 8


def test_check_finite_validation_and_debug_switch(R):
    """rift_check_finite rejects bad arguments on the host (nothing launched);
    rift_set_debug returns the previous setting."""
    L = R.load()
    assert L.rift_check_finite(FAKE, 1, 10, None, None) == 1       # no status word
    assert L.rift_check_finite(None, 1, 10, FAKE, None) == 1       # no input
    assert L.rift_check_finite(FAKE, 5, 10, FAKE, None) == 3       # unknown dtype
    assert L.rift_check_finite(FAKE, 0, -1, FAKE, None) == 2       # negative count
    assert L.rift_status_string(7).decode() == "a floating-point input holds NaN or infinity"
    prev = L.rift_set_debug(1)
    assert L.rift_set_debug(0) == 1
    assert L.rift_set_debug(prev) == 0



def test_split_budgets_and_merge_validation(R):
    """rift_split_budgets against the oracle's split; rift_merge_context
    rejects bad arguments on the host (nothing launched)."""
    b = [0, 1, 64, 128, 144, 288, 575, 576]
    dom, ctx = R.rift_split_budgets(b, 576)
    for c, kd, kc in zip(b, dom, ctx):
        assert (kd, kc) == O.split_budget(c, 576)
    dom, ctx = R.rift_split_budgets(b, 576, 0, 1)          # no merge: everything dominant
    assert list(dom) == b and not ctx.any()
    L = R.load()
    arr = (ctypes.c_int32 * 2)(5, 700)
    out = (ctypes.c_int32 * 2)()
    assert L.rift_split_budgets(2, 576, arr, 10, 64, out, out) == 4      # 700 > n_v
    assert L.rift_split_budgets(2, 576, arr, 65, 64, out, out) == 2      # num > den
    assert L.rift_split_budgets(2, 576, None, 10, 64, out, out) == 1
    assert R.rift_merge_workspace_size(100, 576) >= 100 * 576 * 16
    m = L.rift_merge_context
    ws = R.rift_merge_workspace_size(2, 576)
    assert m(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, None, ws, None) == 1   # no workspace
    assert m(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, None, 2, FAKE, 10, FAKE, 4096, ws, None) == 1  # no ctx_offsets
    assert m(FAKE, 1, 4, 576, 4016, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, 4096, ws, None) == 2  # d % 32
    assert m(FAKE, 1, 4, 2000, 4096, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, 4096, ws, None) == 2  # n_v
    assert m(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, 4096, ws - 1, None) == 5
    assert m(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, 4097, ws, None) == 5  # misaligned
    assert m(FAKE, 7, 4, 576, 4096, FAKE, FAKE, FAKE, FAKE, 2, FAKE, 10, FAKE, 4096, ws, None) == 3
    # compact: contextual rows and offsets go together
    c = L.rift_compact
    assert c(FAKE, 1, 4, 576, 4096, FAKE, FAKE, FAKE, 2, FAKE, None, FAKE, 35, FAKE, 32, 0, FAKE, 100, FAKE, FAKE,
             FAKE, None) == 1



def test_decode_validation(R):
    """rift_decode_step rejects bad arguments on the host (nothing launched)."""
    L = R.load()
    cfg = R.model_cfg(4096, 32, 128, 11008, 1, 1e-6, 10000.0, R.RIFT_BF16)
    f32 = R.model_cfg(256, 4, 64, 688, 1, 1e-6, 10000.0, R.RIFT_F32)
    ws = R.rift_decode_workspace_size(cfg, 4, 643, 8)
    assert ws > 0 and R.rift_decode_workspace_size(cfg, 4, 643, 0) == 0
    lw = (R.LayerWeights * 1)(R.LayerWeights(*([FAKE] * 9)))
    d = L.rift_decode_step
    assert d(ctypes.byref(f32), lw, FAKE, FAKE, 4, 100, 643, 0, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 8
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 643, 0, FAKE, FAKE, 8, 8, FAKE, FAKE, ws, None) == 2  # step
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 16380, 0, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 2
    assert d(ctypes.byref(cfg), lw, None, FAKE, 4, 100, 643, 0, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 1
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 643, 0, None, FAKE, 8, 0, FAKE, FAKE, ws, None) == 1
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 643, 0, FAKE, FAKE, 8, 0, FAKE, FAKE, ws - 1, None) == 5
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 0, 0, 643, 0, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 0  # no prompts
    # shared prefix longer than the prefill batch, or negative
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 643, 101, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 2
    assert d(ctypes.byref(cfg), lw, FAKE, FAKE, 4, 100, 643, -1, FAKE, FAKE, 8, 0, FAKE, FAKE, ws, None) == 2

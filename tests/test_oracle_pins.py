"""Pins for the CPU oracle: each test checks the oracle against something other
than itself -- hand-derived values, closed forms, exact arithmetic, brute force,
or an independent library routine -- so that a dropped term, a wrong sign or a
transposed operand in the oracle fails here.  CPU only."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import rift_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- cdot / csum
def test_cdot_exact_on_small_integers():
    """Small-integer inputs times a power of two: every partial sum is exact,
    so the result must equal the exact integer dot product."""
    rng = np.random.default_rng(11)
    for d in (32, 256, 4096):
        a = rng.integers(-2, 3, size=(5, d)).astype(np.float64) * 2.0 ** -7
        b = rng.integers(-2, 3, size=d).astype(np.float64) * 2.0 ** 3
        exact = [sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(row, b)) for row in a]
        got = O.cdot(a, b)
        assert [Fraction(float(g)) for g in got] == exact


def test_cdot_within_error_bound_of_fsum():
    """Against math.fsum (correctly rounded sum of the exact products): the
    4-accumulator order has error <= (d/4 + 2) eps sum|a_i b_i|.  A missing or
    doubled product (magnitude ~1) would exceed that by orders of magnitude."""
    rng = np.random.default_rng(12)
    d = 4096
    a = synth.bf16_to_f32(synth.round_bf16(rng.standard_normal((8, d)).astype(np.float32))).astype(np.float64)
    b = rng.standard_normal(d).astype(np.float32).astype(np.float64)
    got = O.cdot(a, b)
    for i in range(a.shape[0]):
        ref = math.fsum(a[i] * b)
        bound = (d / 4 + 2) * 2.0 ** -53 * float(np.abs(a[i] * b).sum())
        assert abs(got[i] - ref) <= bound
        assert bound < 1e-9


def test_cdot_order_hand_case():
    """The fixed order, checked on a case where orders disagree (worked by hand):
    granule 0 holds 2^53 and 1, granule 1 holds 1, granule 2 holds -2^53.
    acc0 = 2^53 + 1 -> 2^53 (ties to even), acc1 = 1, acc2 = -2^53, acc3 = 0;
    (acc0 + acc2) + (acc1 + acc3) = 1.  Left-to-right would give 0, exact is 2."""
    a = np.zeros(32)
    a[0], a[1], a[8], a[16] = 2.0 ** 53, 1.0, 1.0, -(2.0 ** 53)
    assert O.cdot(a[None, :], np.ones(32))[0] == 1.0
    # accumulators are fed by granule index mod 4: granule 4 (index 32) joins acc0
    a = np.zeros(64)
    a[0], a[32], a[8] = 2.0 ** 53, 1.0, -(2.0 ** 53)
    # acc0 = 2^53 + 1 -> 2^53; acc1 = -2^53; (acc0 + acc2) + (acc1 + acc3) = 0
    assert O.cdot(a[None, :], np.ones(64))[0] == 0.0


def test_csum64_order_and_value():
    rng = np.random.default_rng(13)
    v = rng.standard_normal(576)
    assert abs(O.csum64(v) - math.fsum(v)) <= 20 * 2.0 ** -53 * np.abs(v).sum()
    # order: lane 0 gets v[0] and v[64]; hand case where it matters
    v = np.zeros(128)
    v[0], v[64], v[1] = 2.0 ** 53, 1.0, 1.0
    # p0 = 2^53 + 1 -> 2^53, p1 = 1; tree: ... p0 += p1 last -> 2^53 + 1 -> 2^53
    assert O.csum64(v) == 2.0 ** 53
    v = np.zeros(128)
    v[0], v[64], v[1], v[65] = 2.0 ** 53, -(2.0 ** 53), 1.0, 1.0
    assert O.csum64(v) == 2.0


# ----------------------------------------------------------------------------- keys
def _unit(v):
    return v / np.sqrt((v * v).sum())


def test_query_direction_matches_eq1_terms():
    """w must make x.w equal Eq. 1's margin x.t - mean_j x.B_j (up to w's
    rounding to float32)."""
    rng = np.random.default_rng(14)
    d, m = 256, 5
    qb = np.stack([_unit(rng.standard_normal(d)) for _ in range(1 + m)]).astype(np.float32).astype(np.float64)
    w = O.query_direction(qb)
    x = rng.standard_normal(d)
    margin = math.fsum(x * qb[0]) - math.fsum(math.fsum(x * qb[j]) for j in range(1, m + 1)) / m
    assert abs(math.fsum(x * w) - margin) <= 2.0 ** -23 * np.abs(x).sum()
    # M = 0 means no background term: w = t
    assert np.array_equal(O.query_direction(qb[:1]), qb[0])


def test_token_key_is_eq1_margin_of_unit_token():
    rng = np.random.default_rng(15)
    d, m = 256, 3
    qb = np.stack([_unit(rng.standard_normal(d)) for _ in range(1 + m)]).astype(np.float32).astype(np.float64)
    w = O.query_direction(qb)
    x = rng.standard_normal((6, d)).astype(np.float32).astype(np.float64)
    r = O.token_keys(x, w)
    for i in range(x.shape[0]):
        xh = x[i] / math.sqrt(math.fsum(x[i] * x[i]))
        cos = [math.fsum(xh * qb[j]) for j in range(1 + m)]
        eq1 = cos[0] - sum(cos[1:]) / m
        assert abs(r[i] - eq1) < 1e-7


def test_token_key_textbook_cosine_without_background():
    rng = np.random.default_rng(16)
    d = 128
    t = _unit(rng.standard_normal(d)).astype(np.float32).astype(np.float64)
    x = rng.standard_normal((4, d))
    r = O.token_keys(x, O.query_direction(t[None, :]))
    for i in range(4):
        ref = math.fsum(x[i] * t) / math.sqrt(math.fsum(x[i] * x[i]))
        assert abs(r[i] - ref) <= 1e-14


def test_token_key_scale_invariance_and_zero():
    rng = np.random.default_rng(17)
    d = 256
    w = rng.standard_normal(d).astype(np.float32).astype(np.float64)
    x = synth.bf16_to_f32(synth.round_bf16(rng.standard_normal((16, d)).astype(np.float32))).astype(np.float64)
    r = O.token_keys(x, w)
    for k in (-3, 1, 5):
        assert np.array_equal(O.token_keys(x * 2.0 ** k, w), r)
    z = O.token_keys(np.zeros((2, d)), w)
    assert np.all(z == 0.0) and not np.any(np.signbit(z))


# ----------------------------------------------------------------------------- token cosines
def test_token_sims_hand_cases():
    """Cosines of Eq. 1's terms (the relevance GEMM's output), worked by hand
    with t = e0 and B_1 = e1: a token along e0 of any length is [1, 0]; along
    e0 + e1 it is [1/sqrt2, 1/sqrt2]; along -e1 it is [0, -1]; an all-zero token
    is [0, 0].  Dividing by |q| instead of |x|, or dropping the 1/|x|, fails the
    first row (3 instead of 1)."""
    d = 32
    e = np.eye(d)
    qb = np.stack([e[0], e[1]])
    x = np.stack([3.0 * e[0], e[0] + e[1], -0.25 * e[1], np.zeros(d)])
    got = O.token_sims(x, qb)
    h = 1.0 / math.sqrt(2.0)
    want = np.array([[1.0, 0.0], [h, h], [0.0, -1.0], [0.0, 0.0]])
    assert got.shape == (4, 2)
    assert np.allclose(got, want, rtol=0, atol=1e-15)
    assert got[3, 0] == 0.0 and got[3, 1] == 0.0


def test_token_sims_against_fsum_cosines():
    """Every element against the correctly rounded dot product over the
    correctly rounded norm, on bfloat16-valued tokens and unit query-bank rows
    rounded to bfloat16 (the stored values of the scenes): the two differ only
    by the rounding of the matrix product and the norm (a few ulps of a value
    below 1).  A transposed or mis-indexed operand gives differences of order
    0.1."""
    rng = np.random.default_rng(19)
    d, m = 256, 15
    rb = lambda a: synth.bf16_to_f32(synth.round_bf16(a.astype(np.float32))).astype(np.float64)
    qb = rb(np.stack([_unit(rng.standard_normal(d)) for _ in range(1 + m)]))
    x = rb(rng.standard_normal((24, d)))
    x[5] += 16.0 * qb[0]         # a planted, strongly aligned token (cosine near 0.7)
    x = rb(x)
    got = O.token_sims(x, qb)
    assert got.shape == (24, 1 + m)
    for i in range(x.shape[0]):
        nrm = math.sqrt(math.fsum(x[i] * x[i]))
        for j in range(1 + m):
            ref = math.fsum(x[i] * qb[j]) / nrm
            assert abs(got[i, j] - ref) <= 1e-15, (i, j, got[i, j], ref)
    assert got[5, 0] > 0.5 > float(np.abs(np.delete(got[:, 0], 5)).max())


def test_token_sims_scale_invariance_and_eq1_margin():
    """Scaling a token by a power of two leaves its cosines bitwise unchanged
    (every product, the norm and the quotient scale exactly).  The Eq. 1 margin
    cos(x, t) - mean_j cos(x, B_j) built from these cosines matches the ranking
    key, which is computed by a different route (one dot product with
    w = t - mean_j B_j rounded to float32) -- to within that rounding."""
    rng = np.random.default_rng(20)
    d, m = 256, 15
    rb = lambda a: synth.bf16_to_f32(synth.round_bf16(a.astype(np.float32))).astype(np.float64)
    qb = rb(np.stack([_unit(rng.standard_normal(d)) for _ in range(1 + m)]))
    x = rb(rng.standard_normal((16, d)))
    s = O.token_sims(x, qb)
    for k in (-4, 3, 9):
        assert np.array_equal(O.token_sims(x * 2.0 ** k, qb), s)
    margin = s[:, 0] - s[:, 1:].mean(axis=1)
    r = O.token_keys(x, O.query_direction(qb))
    assert np.abs(margin - r).max() < 1e-6
    assert np.abs(margin).max() > 1e-2   # the check is not vacuous


# ----------------------------------------------------------------------------- tile scores, u, rank
def test_tile_score_is_eq1_with_mean_unit_embedding():
    """s_i = V_i.t - mean_j V_i.B_j with V_i the mean of unit tokens (reading R1),
    against Eq. 1 evaluated directly with fsum."""
    rng = np.random.default_rng(18)
    d, m, n_tiles, n_v = 64, 4, 3, 70
    qb = np.stack([_unit(rng.standard_normal(d)) for _ in range(1 + m)]).astype(np.float32).astype(np.float64)
    x = rng.standard_normal((n_tiles, n_v, d))
    s = O.tile_scores(np.stack([O.token_keys(x[i], O.query_direction(qb)) for i in range(n_tiles)]))
    for i in range(n_tiles):
        xh = x[i] / np.sqrt((x[i] ** 2).sum(axis=1, keepdims=True))
        V = np.array([math.fsum(xh[:, k]) / n_v for k in range(d)])
        eq1 = math.fsum(V * qb[0]) - sum(math.fsum(V * qb[j]) for j in range(1, m + 1)) / m
        assert abs(s[i] - eq1) < 1e-7


def test_normalise_extremes_and_degenerate():
    rng = np.random.default_rng(19)
    s = rng.standard_normal(400)
    u = O.normalise(s)
    assert u.max() == 1.0 and u.min() == 0.0
    assert u[np.argmax(s)] == 1.0  # App. B Step 3: the top tile has u = 1
    assert np.all(O.normalise(np.full(7, 0.25)) == 1.0)


def test_rank_matches_python_sort_and_permutes():
    rng = np.random.default_rng(20)
    s = rng.integers(0, 5, size=50).astype(np.float64) / 7.0  # many ties
    order, n_keep = O.rank_and_keep(s, O.normalise(s), 10, 0.0)
    ref = sorted(range(50), key=lambda i: (-s[i], i))
    assert list(order) == ref and n_keep == 10
    # threshold mode keeps exactly the u >= tau tiles, as a prefix of the order
    u = O.normalise(s)
    order, n_keep = O.rank_and_keep(s, u, 0, 0.37)
    assert set(order[:n_keep]) == {i for i in range(50) if u[i] >= 0.37}
    # tile scores are independent per tile: permuting tiles permutes s bitwise
    x = rng.standard_normal((6, 64, 32))
    w = rng.standard_normal(32)
    r = np.stack([O.token_keys(x[i], w) for i in range(6)])
    perm = rng.permutation(6)
    assert np.array_equal(O.tile_scores(r[perm]), O.tile_scores(r)[perm])


def test_keep_count_edges():
    s = np.array([0.3, 0.1, 0.2])
    assert O.rank_and_keep(s, O.normalise(s), 10, 0.5)[1] == 3
    assert O.rank_and_keep(s, O.normalise(s), 0, 1.5)[1] == 0   # tau above 1: nothing kept
    assert O.rank_and_keep(s, O.normalise(s), 0, 1.0)[1] == 1   # the top tile always has u = 1


# ----------------------------------------------------------------------------- budgets
def test_budget_tiers_closed_form():
    lv, num, den = (576, 288, 144, 64), (1, 3, 4), 16
    b16 = O.assign_budgets(16, lv, num, den)
    assert [int((b16 == v).sum()) for v in lv] == [1, 3, 4, 8] and int(b16.sum()) == 2528
    b100 = O.assign_budgets(100, lv, num, den)
    assert [int((b100 == v).sum()) for v in lv] == [6, 18, 25, 51] and int(b100.sum()) == 15504
    assert int(b100.sum()) <= int(0.3 * 100 * 576)     # <= 30% of the retained tiles' tokens
    assert list(b100) == sorted(b100, reverse=True)     # higher rank, larger budget
    assert list(O.assign_budgets(1, lv, num, den)) == [64]
    assert len(O.assign_budgets(0, lv, num, den)) == 0
    assert list(O.assign_budgets(2, (64,), (), 16)) == [64, 64]


# ----------------------------------------------------------------------------- selection
def _brute_select(r, k):
    """The unique k-subset S with: for i in S, j not in S, r_i > r_j or
    (r_i == r_j and i < j).  Found by enumerating every subset."""
    n = len(r)
    found = []
    for S in itertools.combinations(range(n), k):
        inside = set(S)
        ok = all((r[i] > r[j]) or (r[i] == r[j] and i < j)
                 for i in inside for j in range(n) if j not in inside)
        if ok:
            found.append(list(S))
    assert len(found) == 1
    return found[0]


def test_select_matches_brute_force_with_ties():
    rng = np.random.default_rng(21)
    for trial in range(40):
        n = int(rng.integers(1, 13))
        r = rng.integers(-2, 3, size=(1, n)).astype(np.float64) if trial % 2 else rng.standard_normal((1, n))
        k = int(rng.integers(0, n + 1))
        offs, sel = O.select_tokens(r, [0], [k])
        assert list(sel) == _brute_select(list(r[0]), k)
        assert list(offs) == [0, k]


def test_select_invariants_full_budget_identity():
    rng = np.random.default_rng(22)
    r = rng.standard_normal((5, 40))
    kept, budgets = [3, 0, 4], [7, 40, 1]
    offs, sel = O.select_tokens(r, kept, budgets)
    for rho, b in enumerate(budgets):
        part = sel[offs[rho]:offs[rho + 1]]
        assert len(part) == b and np.all(np.diff(part) > 0)  # count = budget, sorted, unique
    assert list(sel[offs[1]:offs[2]]) == list(range(40))      # full budget keeps every token in order


# ----------------------------------------------------------------------------- compact
def test_compact_layout_and_full_budget_identity():
    rng = np.random.default_rng(23)
    x = rng.standard_normal((3, 10, 32))
    sysr, qry = rng.standard_normal((2, 32)), rng.standard_normal((3, 32))
    r = rng.standard_normal((3, 10))
    kept = [2, 0]
    offs, sel = O.select_tokens(r, kept, [4, 10])
    packed, cu, pos = O.compact(x, kept, offs, sel, sysr, qry)
    assert list(cu) == [0, 9, 24] and packed.shape == (24, 32)
    assert np.array_equal(pos, np.r_[np.arange(9), np.arange(15)])
    assert np.array_equal(packed[9:11], sysr) and np.array_equal(packed[21:24], qry)
    assert np.array_equal(packed[11:21], x[0])                # full budget: the tile verbatim
    assert np.array_equal(packed[2:6], x[2][sel[:4]])


# ----------------------------------------------------------------------------- golden hand example
def _vec(terms, d):
    v = np.zeros(d)
    for t in terms:
        if t.startswith("3*"):
            v[int(t[3:])] += 3.0
        else:
            v[int(t[1:])] += 1.0
    return v


def test_stage1_hand_example():
    with open(os.path.join(GOLDEN, "stage1_hand_example.json")) as f:
        g = json.load(f)
    d = g["d"]
    x = np.stack([np.stack([_vec(tok, d) for tok in tile]) for tile in g["tiles"]])
    qb = np.stack([_vec([e], d) for e in g["qbank"]])
    st = O.scene_query_stage1(x, qb, 0, g["tau"])
    r2 = math.sqrt(2.0)
    env = {"sqrt": math.sqrt}
    exp_s = [eval(e, env) for e in g["expected"]["s"]]
    exp_u = [eval(e, env) for e in g["expected"]["u"]]
    assert np.allclose(st["s"], exp_s, rtol=0, atol=1e-15), (st["s"], exp_s, r2)
    assert np.allclose(st["u"], exp_u, rtol=0, atol=1e-15)
    assert list(st["order"]) == g["expected"]["order"] and st["n_keep"] == g["expected"]["n_keep"]
    kept = list(st["order"][: st["n_keep"]])
    b = O.assign_budgets(st["n_keep"], g["levels"], g["tier_num"], g["tier_den"])
    assert list(b) == g["expected"]["budgets"]
    offs, sel = O.select_tokens(st["r"], kept, b)
    assert list(offs) == g["expected"]["sel_offsets"] and list(sel) == g["expected"]["sel_idx"]


# ----------------------------------------------------------------------------- prefill pieces
def _naive_attention(q, k, v):
    """Explicit loops: for each query i, softmax over keys 0..i."""
    L, H, hd = q.shape
    out = np.zeros_like(q)
    for h in range(H):
        for i in range(L):
            sc = [sum(q[i, h, c] * k[j, h, c] for c in range(hd)) / math.sqrt(hd) for j in range(i + 1)]
            mx = max(sc)
            e = [math.exp(s - mx) for s in sc]
            z = sum(e)
            for c in range(hd):
                out[i, h, c] = sum(e[j] / z * v[j, h, c] for j in range(i + 1))
    return out


def test_attention_vs_naive_loops():
    rng = np.random.default_rng(24)
    q, k, v = (rng.standard_normal((9, 2, 8)) for _ in range(3))
    assert np.allclose(O.causal_attention(q, k, v), _naive_attention(q, k, v), rtol=0, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(25)
    v = rng.standard_normal((6, 2, 8))
    q = rng.standard_normal((6, 2, 8))
    k = rng.standard_normal((6, 2, 8))
    # length 1: softmax of one score is 1, the output is v
    assert np.allclose(O.causal_attention(q[:1], k[:1], v[:1]), v[:1], atol=1e-15)
    # all-equal scores (zero queries): output i is the mean of v[0..i]
    out = O.causal_attention(np.zeros_like(q), k, v)
    pref = np.cumsum(v, axis=0) / np.arange(1, 7)[:, None, None]
    assert np.allclose(out, pref, atol=1e-14)


def test_rope_identity_norm_and_complex_form():
    rng = np.random.default_rng(26)
    x = rng.standard_normal((5, 3, 16))
    pos = np.array([0, 1, 2, 7, 100])
    y = O.rope(x, pos, 10000.0)
    assert np.allclose(y[0], x[0], atol=0)  # position 0 is the identity
    half = 8
    assert np.allclose(np.sqrt((y ** 2).sum(-1)), np.sqrt((x ** 2).sum(-1)), atol=1e-12)
    # complex form: (x_j + i x_{j+half}) * exp(i pos theta_j)
    for p_i, p in enumerate(pos):
        for j in range(half):
            th = 10000.0 ** (-2 * j / 16)
            z = complex(x[p_i, 0, j], x[p_i, 0, j + half]) * complex(math.cos(p * th), math.sin(p * th))
            assert abs(y[p_i, 0, j] - z.real) < 1e-12 and abs(y[p_i, 0, j + half] - z.imag) < 1e-12


def test_rmsnorm_and_silu_closed_forms():
    x = np.array([[3.0, 4.0]])
    # mean square 12.5 -> x / sqrt(12.5 + eps)
    assert np.allclose(O.rmsnorm(x, np.ones(2), 0.0), x / math.sqrt(12.5), atol=1e-15)
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16


@pytest.mark.slow
def test_decoder_layer_vs_transformers_llama():
    """One layer against transformers' LlamaDecoderLayer in float64 on CPU
    (a library routine, used as is).  The library builds its rotary inverse
    frequencies in float32, so the positions are kept short and the tolerance
    covers that rounding; the angle formula itself is pinned by the complex
    form test above."""
    torch = pytest.importorskip("torch")
    tr = pytest.importorskip("transformers")
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer, LlamaRotaryEmbedding
    w = synth.get("tiny")
    m = w.model
    W = {k: synth.to_f64(v, w.dtype) for k, v in synth.make_layer(w, 0).items()}
    rng = np.random.default_rng(27)
    W["g_attn"] = 1.0 + 0.1 * rng.standard_normal(m.d)   # non-trivial gains exercise the norm weights
    W["g_ffn"] = 1.0 + 0.1 * rng.standard_normal(m.d)
    L = 12
    x = rng.standard_normal((L, m.d))
    cfg = tr.LlamaConfig(hidden_size=m.d, intermediate_size=m.ffn, num_attention_heads=m.n_heads,
                         num_key_value_heads=m.n_heads, head_dim=m.head_dim, rms_norm_eps=m.rms_eps,
                         attention_bias=False, mlp_bias=False, max_position_embeddings=4096,
                         rope_parameters={"rope_type": "default", "rope_theta": m.rope_base})
    cfg._attn_implementation = "eager"
    layer = LlamaDecoderLayer(cfg, 0).double()
    rot = LlamaRotaryEmbedding(cfg).double()
    names = {"self_attn.q_proj.weight": "wq", "self_attn.k_proj.weight": "wk",
             "self_attn.v_proj.weight": "wv", "self_attn.o_proj.weight": "wo",
             "mlp.gate_proj.weight": "w_gate", "mlp.up_proj.weight": "w_up",
             "mlp.down_proj.weight": "w_down", "input_layernorm.weight": "g_attn",
             "post_attention_layernorm.weight": "g_ffn"}
    with torch.no_grad():
        for pn, p in layer.named_parameters():
            p.copy_(torch.from_numpy(W[names[pn]]))
        xt = torch.from_numpy(x)[None]
        pos = torch.arange(L)[None]
        mask = torch.full((L, L), float("-inf"), dtype=torch.float64).triu(1)[None, None]
        ref = layer(xt, attention_mask=mask, position_ids=pos,
                    position_embeddings=rot(xt, pos))[0].numpy()
    got = O.decoder_layer(x, W, m.n_heads, m.head_dim, m.rms_eps, m.rope_base, np.arange(L))
    err = np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)
    assert err.max() < 1e-6, err.max()


# ----------------------------------------------------------------------------- score smoothing (R8)
def _grouped_scene(rng, n_groups=3, per_group=4, n_v=16, d=64):
    """Tiles whose tokens lie close to one of n_groups orthogonal directions."""
    base = np.zeros((n_groups, d))
    for g in range(n_groups):
        base[g, 8 * g] = 3.0
    tiles = []
    for g in range(n_groups):
        for _ in range(per_group):
            tiles.append(base[g] + 0.05 * rng.standard_normal((n_v, d)))
    return np.stack(tiles).astype(np.float32).astype(np.float64)


def test_knn_neighbours_are_the_group_and_score_is_the_group_mean():
    rng = np.random.default_rng(21)
    X = _grouped_scene(rng)
    inv = np.stack([O.token_inv_norms(X[i]) for i in range(X.shape[0])])
    cos = O.tile_similarity(O.tile_embeddings(X, inv))
    s = rng.standard_normal(X.shape[0])
    sm, nbrs = O.knn_smooth(s, cos, 3)
    for i in range(X.shape[0]):
        group = set(range(4 * (i // 4), 4 * (i // 4) + 4)) - {i}
        assert set(nbrs[i]) == group
        assert abs(sm[i] - s[4 * (i // 4):4 * (i // 4) + 4].mean()) <= 1e-15 * 4


def test_knn_off_and_constant_scores():
    rng = np.random.default_rng(22)
    X = rng.standard_normal((5, 64, 32)).astype(np.float32).astype(np.float64)
    Q = rng.standard_normal((16, 32)).astype(np.float32).astype(np.float64)
    a = O.scene_query_stage1(X, Q, 2, 0.0)
    b = O.scene_query_stage1(X, Q, 2, 0.0, knn_m=0)
    assert np.array_equal(a["s"], b["s"]) and np.array_equal(a["s"], a["s_raw"])
    cos = rng.uniform(-1, 1, size=(5, 5))
    sm, _ = O.knn_smooth(np.full(5, 0.375), cos, 3)
    assert np.all(sm == 0.375)


def test_tile_similarity_against_normalised_dot_products():
    rng = np.random.default_rng(23)
    X = rng.standard_normal((7, 20, 64)).astype(np.float32).astype(np.float64)
    inv = np.stack([O.token_inv_norms(X[i]) for i in range(7)])
    E = O.tile_embeddings(X, inv)
    # the embedding is the sum of unit tokens, up to float32 rounding
    unit = X / np.linalg.norm(X, axis=2, keepdims=True)
    assert np.allclose(E, unit.sum(axis=1), rtol=1e-6, atol=1e-6)
    cos = O.tile_similarity(E)
    En = E / np.linalg.norm(E, axis=1, keepdims=True)
    assert np.allclose(cos, En @ En.T, rtol=0, atol=1e-13)
    assert np.array_equal(cos, cos.T)
    assert np.allclose(np.diag(cos), 1.0, atol=1e-15)


def test_knn_ties_go_to_the_lower_tile_and_permutation_equivariance():
    rng = np.random.default_rng(24)
    X = rng.standard_normal((6, 12, 32)).astype(np.float32).astype(np.float64)
    X[4] = X[2]                       # tiles 2 and 4 identical: equal similarity to everyone
    inv = np.stack([O.token_inv_norms(X[i]) for i in range(6)])
    cos = O.tile_similarity(O.tile_embeddings(X, inv))
    s = rng.standard_normal(6)
    _, nbrs = O.knn_smooth(s, cos, 5)
    for i in (0, 1, 3, 5):
        assert nbrs[i].index(2) < nbrs[i].index(4)
    # relabelling tiles relabels the result (random tiles, no ties)
    Y = rng.standard_normal((6, 12, 32)).astype(np.float32).astype(np.float64)
    perm = rng.permutation(6)
    invY = np.stack([O.token_inv_norms(Y[i]) for i in range(6)])
    cY = O.tile_similarity(O.tile_embeddings(Y, invY))
    smY, _ = O.knn_smooth(s, cY, 3)
    Yp = Y[perm]
    invP = np.stack([O.token_inv_norms(Yp[i]) for i in range(6)])
    cP = O.tile_similarity(O.tile_embeddings(Yp, invP))
    smP, _ = O.knn_smooth(s[perm], cP, 3)
    assert np.array_equal(smP, smY[perm])


# ----------------------------------------------------------------------------- utility budgets (R13)
# Stand-in accuracy and energy tables over the paper's budget set for LLaVA-1.5
# (Sec. 2.3 Stage 2): accuracy on object tiles grows with the budget, accuracy
# on empty tiles barely moves, energy is proportional to the budget.
C5 = [576, 432, 288, 144, 72]
AP = [0.92, 0.90, 0.85, 0.74, 0.58]
AN = [0.95, 0.95, 0.94, 0.93, 0.91]
EN = [c / 576 for c in C5]


def test_utility_budgets_hand_worked():
    # p = 1: U = a+ - 0.1 E = 0.82, 0.825, 0.80, 0.715, 0.5675 -> 432
    # p = 0: U = a- - 0.1 E = 0.85, 0.875, 0.89, 0.905, 0.8975 -> 144
    assert list(O.utility_budgets([1.0, 0.0], C5, AP, AN, EN, 0.1)) == [432, 144]
    # no energy cost: the most accurate budget for the object tile, for an empty tile the
    # first of the equal-accuracy 576 / 432 pair by size (the smaller)
    assert list(O.utility_budgets([1.0, 0.0], C5, AP, AN, EN, 0.0)) == [576, 432]
    # energy dominates: the smallest budget for everyone
    assert list(O.utility_budgets([1.0, 0.5, 0.0], C5, AP, AN, EN, 100.0)) == [72, 72, 72]


def test_utility_budgets_ties_and_order_independence():
    # equal utilities everywhere -> the smallest budget, whatever the listing order
    flat = [0.5] * 5
    assert list(O.utility_budgets([0.3], C5, flat, flat, [0.0] * 5, 1.0)) == [72]
    perm = [3, 0, 4, 1, 2]
    a = O.utility_budgets([0.0, 0.25, 0.5, 0.75, 1.0], C5, AP, AN, EN, 0.1)
    b = O.utility_budgets([0.0, 0.25, 0.5, 0.75, 1.0], [C5[i] for i in perm], [AP[i] for i in perm],
                          [AN[i] for i in perm], [EN[i] for i in perm], 0.1)
    assert np.array_equal(a, b)
    # the budget never shrinks as p grows when a+ - a- grows with the budget
    p = np.linspace(0, 1, 101)
    bud = O.utility_budgets(p, C5, AP, AN, EN, 0.1)
    assert np.all(np.diff(bud) >= 0)


# ------------------------------------------------------------------ contextual merge (R14)


def test_split_budget_visionzip_configurations():
    # VisionZip's published splits: 54 + 10 at 64 tokens, 108 + 20 at 128, 162 + 30 at 192
    assert O.split_budget(64, 576) == (54, 10)
    assert O.split_budget(128, 576) == (108, 20)
    assert O.split_budget(192, 576) == (162, 30)
    # nothing left to merge at the full budget; one token left at n_v - 1
    assert O.split_budget(576, 576) == (576, 0)
    assert O.split_budget(575, 576) == (574, 1)
    assert O.split_budget(0, 576) == (0, 0)
    for c in range(0, 577):
        kd, kc = O.split_budget(c, 576)
        assert kd + kc == c and 0 <= kc <= 576 - c


def test_round_f32_to_bf16_against_torch_and_hand_cases():
    torch = pytest.importorskip("torch")
    # hand cases: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> even (1);
    # 1 + 3 * 2^-9 is above halfway -> 1 + 2^-7; -2.5 is exact
    hand = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -9, -2.5, 1.0 + 3 * 2.0 ** -8], np.float32)
    assert list(O.round_f32_to_bf16(hand)) == [0x3F80, 0x3F80, 0x3F81, 0xC020, 0x3F82]
    v = np.random.default_rng(0).standard_normal(100_000).astype(np.float32) * 1e3
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.round_f32_to_bf16(v), ref)


def _int_tokens(rng, n_v, d, lo=-3, hi=4):
    return rng.integers(lo, hi, size=(n_v, d)).astype(np.float64)


def test_merge_all_targets_and_single_target_closed_forms():
    rng = np.random.default_rng(4)
    x = _int_tokens(rng, 20, 64)
    dom = [0, 3, 7]
    R = [t for t in range(20) if t not in dom]
    # as many contextual tokens as remaining tokens: each is its own group
    vals, groups, targets = O.merge_context(x, dom, len(R))
    assert targets == R and groups == [[t] for t in R]
    assert np.array_equal(vals, x[R])
    # one contextual token: the mean of the whole remainder (exact on small integers / 17)
    vals, groups, targets = O.merge_context(x, dom, 1)
    assert targets == [R[0]] and groups == [R]
    assert np.array_equal(vals[0], (x[R].sum(axis=0) / len(R)).astype(np.float32).astype(np.float64))


def test_merge_follows_orthogonal_clusters():
    d = 32
    e0, e1 = np.eye(d)[0], np.eye(d)[1]
    x = np.zeros((12, d))
    x[0] = e0 + e1
    x[1] = e0 - e1                       # dominant tokens: not merged
    for t in range(2, 7):
        x[t] = (t - 1) * e0              # cluster along e0
    for t in range(7, 12):
        x[t] = (t - 6) * 3 * e1          # cluster along e1
    vals, groups, targets = O.merge_context(x, [0, 1], 2)
    assert targets == [2, 7]              # R = 2..11, targets R[0] and R[5]
    assert groups == [[2, 3, 4, 5, 6], [7, 8, 9, 10, 11]]
    assert np.array_equal(vals[0], 3.0 * e0) and np.array_equal(vals[1], 9.0 * e1)


def test_merge_uses_the_cosine_not_the_dot_product():
    d = 32
    x = np.zeros((4, d))
    x[0, 0] = 1.0                        # target 0: short, 0 degrees from the token
    x[1, :2] = [100.0, 100.0]            # target 1: long, 45 degrees from the token
    x[2, 0] = 1.0                        # the token: larger dot product with target 1,
    x[2, 2] = 0.25                       #   larger cosine with target 0
    x[3, 1] = 1.0
    # reordered so that the targets R[0] and R[2] are the two candidate rows
    vals, groups, targets = O.merge_context(x[[0, 2, 1, 3]], [], 2)
    assert targets == [0, 2]              # rows 0 (short target) and 2 (long target)
    assert groups[0] == [0, 1]            # the token (row 1) goes to the short target


def test_merge_ties_scale_invariance_and_invariants():
    rng = np.random.default_rng(9)
    d = 64
    x = rng.standard_normal((30, d)).astype(np.float32).astype(np.float64)
    dom = [1, 5, 6, 20]
    vals, groups, targets = O.merge_context(x, dom, 4)
    R = [t for t in range(30) if t not in dom]
    # every remaining token in exactly one group, each target in its own, groups ascending
    assert sorted(t for g in groups for t in g) == R
    for g, t in zip(groups, targets):
        assert t in g and g == sorted(g)
    # scaling tokens by powers of two changes no assignment (the score scales exactly)
    xs = x.copy()
    xs[R[3]] *= 8.0
    xs[targets[1]] *= 0.25
    _, groups2, _ = O.merge_context(xs, dom, 4)
    assert groups2 == groups
    # brute force with plain normalised dot products agrees when no two cosines are close
    for j, g in enumerate(groups):
        for r in g:
            if r in targets:
                continue
            cos = [float(np.dot(x[r], x[t]) / np.linalg.norm(x[t])) for t in targets]
            best = int(np.argmax(cos))
            srt = sorted(cos, reverse=True)
            if srt[0] - srt[1] > 1e-9:
                assert best == j
    # two identical targets: every token that prefers them goes to the lower one
    xt = x.copy()
    xt[targets[2]] = xt[targets[1]]
    _, g3, _ = O.merge_context(xt, dom, 4)
    assert g3[2] == [targets[2]]


def test_compact_with_contextual_rows_layout():
    x = np.arange(3 * 5 * 2, dtype=np.float64).reshape(3, 5, 2)
    sysr = np.full((2, 2), -1.0)
    qry = np.full((1, 2), -2.0)
    ctx = np.array([[100.0, 100.0], [200.0, 200.0], [300.0, 300.0]])
    packed, cu, pos = O.compact(x, [2, 0], np.array([0, 2, 3]), np.array([1, 4, 0]), sysr, qry,
                                ctx_rows=ctx, ctx_offsets=np.array([0, 2, 3]))
    expect = np.concatenate([sysr, x[2][[1, 4]], ctx[0:2], qry, sysr, x[0][[0]], ctx[2:3], qry])
    assert np.array_equal(packed, expect)
    assert list(cu) == [0, 7, 12] and list(pos) == list(range(7)) + list(range(5))


# ------------------------------------------------------------------ decode (R15)


def _small_layer(rng, d, ffn):
    W = {k: rng.standard_normal(sh) * 0.1 for k, sh in
         (("wq", (d, d)), ("wk", (d, d)), ("wv", (d, d)), ("wo", (d, d)),
          ("w_gate", (ffn, d)), ("w_up", (ffn, d)), ("w_down", (d, ffn)))}
    W["g_attn"] = np.ones(d)
    W["g_ffn"] = np.ones(d)
    return W


def test_decode_is_incremental_prefill_and_causal():
    """Decoding token by token gives what a prefill of the whole extended
    sequence gives on its last rows (causality: appending tokens changes no
    earlier row), and the prompt rows of the extended run equal the prompt's
    own prefill."""
    rng = np.random.default_rng(17)
    d, H, hd, ffn = 32, 4, 8, 48
    layers = [_small_layer(rng, d, ffn) for _ in range(2)]
    prompt = rng.standard_normal((7, d))
    new = rng.standard_normal((3, d))
    out = O.decode_outputs(prompt, new, layers, H, hd, 1e-6, 10000.0)
    full = np.concatenate([prompt, new])
    x = full.copy()
    for W in layers:
        x = O.decoder_layer(x, W, H, hd, 1e-6, 10000.0, np.arange(10))
    assert np.allclose(out, x[7:], rtol=0, atol=1e-12)
    xp = prompt.copy()
    for W in layers:
        xp = O.decoder_layer(xp, W, H, hd, 1e-6, 10000.0, np.arange(7))
    assert np.allclose(x[:7], xp, rtol=0, atol=1e-12)
    # a changed later token leaves the earlier generated outputs unchanged
    new2 = new.copy()
    new2[2] += 1.0
    out2 = O.decode_outputs(prompt, new2, layers, H, hd, 1e-6, 10000.0)
    assert np.array_equal(out2[:2], out[:2]) and not np.allclose(out2[2], out[2])


def test_causal_prefix_states_do_not_depend_on_later_rows():
    """The reading behind the shared system prefix: under causal attention the
    states of a sequence's first P rows, after every layer, are those of the P
    rows alone, whatever follows them (prompts that differ after a common
    prefix agree on it to rounding)."""
    rng = np.random.default_rng(7)
    d, H, hd, F = 64, 4, 16, 96
    mk = lambda *s: rng.standard_normal(s) * 0.2
    layers = [dict(wq=mk(d, d), wk=mk(d, d), wv=mk(d, d), wo=mk(d, d), w_gate=mk(F, d), w_up=mk(F, d),
                   w_down=mk(d, F), g_attn=1 + mk(d), g_ffn=1 + mk(d)) for _ in range(2)]
    P = 5
    prefix = rng.standard_normal((P, d))
    tails = [rng.standard_normal((n, d)) for n in (0, 3, 9)]
    outs = []
    for tail in tails:
        x = np.concatenate([prefix, tail])
        cu = np.array([0, len(x)])
        outs.append(O.prefill(x, cu, np.arange(len(x)), layers, H, hd, 1e-6, 10000.0)[0])
    for o in outs[1:]:
        assert np.allclose(o[:P], outs[0], rtol=1e-12, atol=1e-12)
    # and a change inside the prefix does change what follows
    x2 = np.concatenate([prefix + np.eye(P, d) * 0.5, tails[2]])
    o2 = O.prefill(x2, np.array([0, len(x2)]), np.arange(len(x2)), layers, H, hd, 1e-6, 10000.0)[0]
    assert not np.allclose(o2[P:], outs[2][P:], rtol=1e-6, atol=1e-6)

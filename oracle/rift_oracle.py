"""CPU oracle for the Rift hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the bench's CPU-baseline leg
may import this module.  The GPU library never calls it and shares no code with
it; the only common ground is the seeded input generator (the `synth` package).

Everything here is plain float64 NumPy, written to be checked against the paper
by eye.  Inputs are the generator's stored values widened exactly to float64.

Paper passages followed (Rift, "Exploiting answer-invariant redundancies in
satellite imagery for efficient VLM inference on edge"):
  * Sec. 2.3 Stage 1, Eq. 1 and Listing 1 -- background-margin relevance,
    per-scene min-max normalisation, retention by threshold.
  * App. B Step 3 -- retention is u_i >= tau and the top tile always has u = 1.
  * Sec. 2.3 Stage 2 -- per-tile budgets from a discrete set; VisionZip keeps
    each tile's dominant tokens.
  * Sec. 2.1 and Sec. 2.3 Stage 2 -- each retained tile is an independent
    prompt that the LLaVA-1.5-7B (LLaMA-7B-shaped) decoder prefills.

Readings of points the paper leaves open (numbered as in the design notes):
  R1  V_i is the mean of the tile's unit-normalised vision tokens, so the tile
      score is the mean over tokens of the per-token Eq. 1 margin.
  R2  Eq. 1 is linear in V_i, so the margin is V_i . w with
      w = t - (1/M) sum_j B_j, evaluated in float64 and rounded to float32.
  R3  Ranking keys are float64 results of a fixed summation order (cdot, csum)
      so that the same decisions are reproducible bit for bit.
  R4  Tile order is (score descending, tile id ascending); min-max with
      max == min gives u = 1 for every tile.
  R5  Retention by threshold keeps u >= tau (Listing 1, App. B Step 3).
  R6  Token importance for VisionZip's "dominant tokens" is the per-token
      margin; ties go to the lower token index; kept tokens stay in ascending
      index order.
  R7  Budgets by score rank: tiers of floor(K*num_j/den) kept tiles per level,
      the last level takes the rest.
  R8  Optional score smoothing (Listing 1's note; App. B Step 3): each tile's
      score is averaged with those of its m most visually similar tiles.  The
      tile's embedding for similarity is its summed unit-normalised tokens,
      E_i = fp32(sum over t ascending of x_t * (1/sqrt(n2_t))) with n2_t =
      cdot(x_t, x_t) and the product then the sum each rounded (no fusion);
      similarity is the cosine G_ij / sqrt(G_ii G_jj) of the canonical dot
      products G = cdot(E_i, E_j) (0 when a norm is 0); the neighbours are the
      m largest similarities over j != i, ties to the lower j; the smoothed
      score is (s_i + sum of the neighbours' s in neighbour order) / (1 + m),
      and u and the ranking use it.  Off unless asked for (m = 0).
  R9  Each prompt is [system | kept vision tokens | query text] with positions
      0..L-1.
  R10 RMSNorm gains 1; rotate-half RoPE; attention scale 1/sqrt(hd); the
      output is the residual stream after the last layer, before any final
      norm.
  R13 Optional utility budgets (Eq. 2): U_i(c) = p_i a+_c + (1 - p_i) a-_c
      - lambda E_c evaluated in float64 as ((p a+) + ((1 - p) a-)) - (lambda
      E) with every operation rounded on its own; the budget is the c of
      largest U, ties to the smaller c.  p_i, the trained predictor's
      probability that the tile holds the object, is out of scope: callers
      pass it (the pipeline passes the tile's normalised score u_i).
  R15 Decode after prefill: each generated token's input embedding is
      given; token t of a prompt of length L sits at position L + t and
      attends causally to the prompt and the earlier generated tokens (the
      decoder layers of R10, no vocabulary projection).
  R14 Optional merge of the remainder into contextual tokens (Sec. 2.3
      Stage 2: VisionZip keeps the dominant tokens "and merges the remainder";
      the merge follows VisionZip's published scheme).  A budget c splits into
      k_c = min(floor(c num / den), n_v - c) contextual and k_d = c - k_c
      dominant tokens (num/den = 10/64, VisionZip's 54 + 10 at 64 tokens; at
      the full budget k_c = 0).  The remainder R is the n_v - k_d tokens not
      selected as dominant, ascending; target j is R[floor(j |R| / k_c)].
      Every other token of R joins the target j of largest
      cdot(x_r, x_j) * inv_j (its cosine to the target up to the positive
      factor 1/|x_r|; inv as for R8), ties to the lower j.  Contextual token j
      is the float64 sum of its group in ascending index order divided by the
      group size, rounded to float32 and then to the storage type.  The
      prompt becomes [system | dominant | contextual (j order) | query].
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

# ============================================================================ Stage 1


def query_direction(qbank: np.ndarray) -> np.ndarray:
    """w = t - (1/M) sum_j B_j, per element in float64, then rounded to float32
    (reading R2; Eq. 1 of Sec. 2.3).  qbank row 0 is t, rows 1..M are B_j.
    The background sum runs j = 1..M in order.  Returns float64 holding
    float32-representable values."""
    qb = np.asarray(qbank, dtype=np.float64)
    t = qb[0]
    m = qb.shape[0] - 1
    if m == 0:
        w = t.copy()
    else:
        acc = np.zeros_like(t)
        for j in range(1, m + 1):
            acc = acc + qb[j]
        w = t - acc / m
    return w.astype(np.float32).astype(np.float64)


def cdot(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Float64 dot product of each row of `a` with `b` (a vector, or an array
    shaped like `a`) in the fixed order of
    reading R3.  Elements are grouped in granules of 8 consecutive indices;
    granule g feeds accumulator g mod 4; each accumulator adds its products in
    ascending index order starting from +0; the result is
    (acc0 + acc2) + (acc1 + acc3).  Products of stored inputs (bfloat16 or
    float32 with float32) are exact in float64.  Requires d % 32 == 0."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    d = a.shape[-1]
    if d % 32:
        raise ValueError("cdot needs d % 32 == 0")
    lead = a.shape[:-1]
    a4 = a.reshape(lead + (d // 32, 4, 8))
    b4 = np.broadcast_to(b, a.shape).reshape(lead + (d // 32, 4, 8))
    acc = np.zeros(lead + (4,), dtype=np.float64)
    for s in range(d // 32):          # granule rounds, ascending index
        for j in range(8):            # within a granule, ascending index
            acc = acc + a4[..., s, :, j] * b4[..., s, :, j]
    return (acc[..., 0] + acc[..., 2]) + (acc[..., 1] + acc[..., 3])


def csum64(v: np.ndarray) -> float:
    """Float64 sum of a short vector in the fixed order of reading R3: 64
    partial sums, partial l adds v[l], v[l+64], v[l+128], ... in order from +0;
    then the halving tree p[l] += p[l+s] for s = 32, 16, 8, 4, 2, 1."""
    v = np.asarray(v, dtype=np.float64)
    p = [0.0] * 64
    for i in range(v.shape[0]):
        p[i % 64] = p[i % 64] + float(v[i])
    s = 32
    while s >= 1:
        for lane in range(s):
            p[lane] = p[lane] + p[lane + s]
        s //= 2
    return p[0]


def token_keys(x: np.ndarray, w32: np.ndarray) -> np.ndarray:
    """Per-token Eq. 1 margin of the unit-normalised token (readings R1-R3):
    r = cdot(x, w) / sqrt(cdot(x, x)), float64 with correctly rounded divide
    and square root; r = +0 for an all-zero token; -0 is returned as +0.
    x: [..., d]."""
    n2 = cdot(x, x)
    g = cdot(x, w32)
    with np.errstate(invalid="ignore", divide="ignore"):
        r = g / np.sqrt(n2)
    r = np.where(n2 == 0.0, 0.0, r)
    return r + 0.0


def token_sims(x: np.ndarray, qbank: np.ndarray) -> np.ndarray:
    """Cosine similarity of every token to t and to each B_j (Eq. 1's terms),
    float64 via a plain matrix product.  x: [..., d] -> [..., 1 + M]."""
    x = np.asarray(x, dtype=np.float64)
    q = np.asarray(qbank, dtype=np.float64)
    nrm = np.sqrt((x * x).sum(axis=-1, keepdims=True))
    dots = x @ q.T
    with np.errstate(invalid="ignore", divide="ignore"):
        out = np.where(nrm == 0.0, 0.0, dots / nrm)
    return out


def tile_scores(r: np.ndarray) -> np.ndarray:
    """s_i = mean over the tile's tokens of the per-token margin (reading R1),
    summed with csum64, divided by n_v.  r: [n_tiles][n_v]."""
    r = np.asarray(r, dtype=np.float64)
    n_v = r.shape[1]
    return np.array([csum64(r[i]) / n_v for i in range(r.shape[0])], dtype=np.float64)


def normalise(s: np.ndarray) -> np.ndarray:
    """Per-scene min-max normalisation u = (s - min s) / (max s - min s)
    (Sec. 2.3 Stage 1; Listing 1).  max == min gives u = 1 (reading R4, which
    keeps App. B Step 3's "top tile has u = 1")."""
    s = np.asarray(s, dtype=np.float64)
    lo, hi = s.min(), s.max()
    if hi == lo:
        return np.ones_like(s)
    return (s - lo) / (hi - lo)


def rank_and_keep(s: np.ndarray, u: np.ndarray, keep_count: int, tau: float
                  ) -> Tuple[np.ndarray, int]:
    """Tile order by (s descending, id ascending) (reading R4).  keep_count > 0
    keeps the first min(K, n_tiles) tiles; keep_count == 0 keeps every tile with
    u >= tau (App. B Step 3 and Listing 1 use >=), which is a prefix of the
    order because u is monotone in s."""
    s = np.asarray(s, dtype=np.float64)
    ids = np.arange(s.shape[0])
    order = np.lexsort((ids, -s)).astype(np.int32)
    if keep_count > 0:
        n_keep = min(int(keep_count), s.shape[0])
    else:
        n_keep = int(np.count_nonzero(np.asarray(u, dtype=np.float64) >= tau))
    return order, n_keep


# ============================================================================ Stage 2


def tier_counts(n_keep: int, n_levels: int, tier_num: Sequence[int], tier_den: int
                ) -> List[int]:
    """Kept tiles per budget level (reading R7): level j < last gets
    floor(K * num_j / den), the last level the remainder."""
    counts = [(n_keep * int(tier_num[j])) // int(tier_den) for j in range(n_levels - 1)]
    counts.append(n_keep - sum(counts))
    return counts


def assign_budgets(n_keep: int, levels: Sequence[int], tier_num: Sequence[int],
                   tier_den: int) -> np.ndarray:
    """Budget of kept rank rho (reading R7): higher-ranked tiles get the larger
    levels of the discrete set C (Sec. 2.3 Stage 2)."""
    counts = tier_counts(n_keep, len(levels), tier_num, tier_den)
    out: List[int] = []
    for lvl, c in zip(levels, counts):
        out.extend([int(lvl)] * c)
    return np.array(out, dtype=np.int32)


def utility_budgets(p: Sequence[float], levels: Sequence[int], alpha_pos: Sequence[float],
                    alpha_neg: Sequence[float], energy: Sequence[float], lam: float) -> np.ndarray:
    """Eq. 2 budget per tile (reading R13): the candidate c of largest
    U(c) = p a+_c + (1 - p) a-_c - lambda E_c, ties to the smaller c."""
    out = []
    for pi in p:
        pi = float(pi)
        best_c, best_u = None, None
        for c, ap, an, e in zip(levels, alpha_pos, alpha_neg, energy):
            u = ((pi * float(ap)) + ((1.0 - pi) * float(an))) - (float(lam) * float(e))
            if best_u is None or u > best_u or (u == best_u and int(c) < best_c):
                best_c, best_u = int(c), u
        out.append(best_c)
    return np.array(out, dtype=np.int32)


def select_tokens(r: np.ndarray, kept: Sequence[int], budgets: Sequence[int]
                  ) -> Tuple[np.ndarray, np.ndarray]:
    """For each kept tile, its `budget` most important tokens by (key
    descending, index ascending), emitted in ascending index order (reading R6;
    VisionZip's dominant-token retention, Sec. 2.3 Stage 2).
    Returns (sel_offsets [K+1], sel_idx [sum budgets])."""
    r = np.asarray(r, dtype=np.float64)
    n_v = r.shape[1]
    idx = np.arange(n_v)
    offs = [0]
    parts = []
    for tile, b in zip(kept, budgets):
        order = np.lexsort((idx, -r[int(tile)]))
        parts.append(np.sort(order[: int(b)]))
        offs.append(offs[-1] + int(b))
    sel = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    return np.array(offs, dtype=np.int32), sel


def compact(x: np.ndarray, kept: Sequence[int], sel_offsets: np.ndarray,
            sel_idx: np.ndarray, sys: np.ndarray, qry: np.ndarray,
            ctx_rows: np.ndarray = None, ctx_offsets: np.ndarray = None
            ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Packed varlen batch: sequence rho = [sys | x[kept[rho], sel] | qry]
    (reading R9), or [sys | x[kept[rho], sel] | contextual rows of rho | qry]
    when contextual rows are given (reading R14); cu_seqlens = prefix sums of
    lengths, position ids 0..L-1 per sequence.  Works on any element type (it
    only moves rows)."""
    rows = []
    cu = [0]
    pos = []
    for rho, tile in enumerate(kept):
        sel = sel_idx[sel_offsets[rho]: sel_offsets[rho + 1]]
        parts = [sys, x[int(tile)][sel]]
        if ctx_rows is not None:
            parts.append(ctx_rows[ctx_offsets[rho]: ctx_offsets[rho + 1]])
        seq = np.concatenate(parts + [qry], axis=0)
        rows.append(seq)
        cu.append(cu[-1] + seq.shape[0])
        pos.append(np.arange(seq.shape[0], dtype=np.int32))
    if rows:
        packed = np.concatenate(rows, axis=0)
        position_ids = np.concatenate(pos)
    else:
        packed = np.zeros((0, x.shape[-1]), dtype=x.dtype)
        position_ids = np.zeros(0, dtype=np.int32)
    return packed, np.array(cu, dtype=np.int32), position_ids


# ============================================================================ prefill


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis (LLaMA's RMSNorm)."""
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding (reading R10) on x: [L, H, hd].  Pair
    (j, j + hd/2) turns by angle pos * base^(-2j/hd)."""
    hd = x.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * j / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Softmax attention of one sequence, query i attends keys j <= i, scale
    1/sqrt(hd).  q, k, v: [L, H, hd] -> [L, H, hd]."""
    L, H, hd = q.shape
    out = np.empty_like(q)
    mask = np.tril(np.ones((L, L), dtype=bool))
    for h in range(H):
        sc = (q[:, h, :] @ k[:, h, :].T) / math.sqrt(hd)
        sc = np.where(mask, sc, -np.inf)
        sc = sc - sc.max(axis=1, keepdims=True)
        p = np.exp(sc)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, h, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def decoder_layer(x: np.ndarray, W: Dict[str, np.ndarray], n_heads: int, head_dim: int,
                  eps: float, rope_base: float, positions: np.ndarray) -> np.ndarray:
    """One LLaMA decoder layer on one sequence x: [L, d] (float64).
    W holds wq, wk, wv, wo, w_gate, w_up, w_down in [out][in] layout and the
    RMSNorm gains g_attn, g_ffn."""
    L = x.shape[0]
    h = rmsnorm(x, W["g_attn"], eps)
    q = (h @ W["wq"].T).reshape(L, n_heads, head_dim)
    k = (h @ W["wk"].T).reshape(L, n_heads, head_dim)
    v = (h @ W["wv"].T).reshape(L, n_heads, head_dim)
    q = rope(q, positions, rope_base)
    k = rope(k, positions, rope_base)
    o = causal_attention(q, k, v).reshape(L, n_heads * head_dim)
    x = x + o @ W["wo"].T
    h2 = rmsnorm(x, W["g_ffn"], eps)
    a = silu(h2 @ W["w_gate"].T) * (h2 @ W["w_up"].T)
    return x + a @ W["w_down"].T


def prefill(packed: np.ndarray, cu_seqlens: np.ndarray, position_ids: np.ndarray,
            layers: Sequence[Dict[str, np.ndarray]], n_heads: int, head_dim: int,
            eps: float, rope_base: float, seqs: Sequence[int] | None = None
            ) -> Dict[int, np.ndarray]:
    """Prefill of independent sequences (Sec. 2.1; each retained tile is its
    own VLM call, Sec. 2.3 Stage 2).  Returns {sequence index: hidden [L, d]},
    the residual stream after the last layer, for the requested sequences
    (all by default)."""
    n_seq = len(cu_seqlens) - 1
    seqs = list(range(n_seq)) if seqs is None else list(seqs)
    xs = {i: np.asarray(packed[cu_seqlens[i]:cu_seqlens[i + 1]], dtype=np.float64)
          for i in seqs}
    for W in layers:
        for i in seqs:
            pos = position_ids[cu_seqlens[i]:cu_seqlens[i + 1]]
            xs[i] = decoder_layer(xs[i], W, n_heads, head_dim, eps, rope_base, pos)
    return xs


def decode_outputs(prompt: np.ndarray, new_tokens: np.ndarray,
                   layers: Sequence[Dict[str, np.ndarray]], n_heads: int, head_dim: int,
                   eps: float, rope_base: float) -> np.ndarray:
    """Residual stream after the last layer of each generated token of one
    prompt: token t (input embedding new_tokens[t], position L + t) attends
    causally to the prompt and to the tokens before it, so its output is the
    last row of the decoder stack run on [prompt | new_tokens[:t + 1]] (the
    prompt rows of that run equal the prompt's own prefill).  prompt: [L, d],
    new_tokens: [S, d]; returns [S, d]."""
    prompt = np.asarray(prompt, dtype=np.float64)
    new_tokens = np.asarray(new_tokens, dtype=np.float64)
    out = []
    for t in range(new_tokens.shape[0]):
        x = np.concatenate([prompt, new_tokens[:t + 1]], axis=0)
        pos = np.arange(x.shape[0])
        for W in layers:
            x = decoder_layer(x, W, n_heads, head_dim, eps, rope_base, pos)
        out.append(x[-1])
    return np.stack(out) if out else np.zeros((0, prompt.shape[1]))


# ============================================================================ whole query


def scene_query_stage1(tokens: np.ndarray, qbank: np.ndarray, keep_count: int, tau: float,
                       knn_m: int = 0):
    """Stage 1 of one scene-query on float64 inputs: keys, tile scores, u,
    order, n_keep (Sec. 2.3 Stage 1); with knn_m > 0 the scores are first
    smoothed over each tile's knn_m most similar tiles (reading R8)."""
    w32 = query_direction(qbank)
    r = np.stack([token_keys(tokens[i], w32) for i in range(tokens.shape[0])])
    s_raw = tile_scores(r)
    out = {"w32": w32, "r": r, "s_raw": s_raw}
    s = s_raw
    if knn_m > 0:
        inv = np.stack([token_inv_norms(tokens[i]) for i in range(tokens.shape[0])])
        E = tile_embeddings(tokens, inv)
        cos = tile_similarity(E)
        s, nbrs = knn_smooth(s_raw, cos, knn_m)
        out.update({"inv": inv, "E": E, "cos": cos, "nbrs": nbrs})
    u = normalise(s)
    order, n_keep = rank_and_keep(s, u, keep_count, tau)
    out.update({"s": s, "u": u, "order": order, "n_keep": n_keep})
    return out


# ------------------------------------------------------- optional smoothing (R8)


def token_inv_norms(x: np.ndarray) -> np.ndarray:
    """1/sqrt(n2) per token with n2 = cdot(x, x), correctly rounded square root
    and divide; 0 for an all-zero token.  x: [..., d]."""
    n2 = cdot(x, x)
    with np.errstate(divide="ignore"):
        inv = 1.0 / np.sqrt(n2)
    return np.where(n2 == 0.0, 0.0, inv)


def tile_embeddings(tokens: np.ndarray, inv: np.ndarray) -> np.ndarray:
    """E_i = fp32(sum over tokens t, ascending, of x_t * inv_t), every product
    and every addition rounded to float64 on its own (reading R8).
    tokens: [n_tiles, n_v, d] float64; inv: [n_tiles, n_v].  Returns float64
    holding float32 values."""
    P = np.zeros((tokens.shape[0], tokens.shape[2]), dtype=np.float64)
    for t in range(tokens.shape[1]):
        P = P + tokens[:, t, :] * inv[:, t:t + 1]
    return P.astype(np.float32).astype(np.float64)


def tile_similarity(E: np.ndarray) -> np.ndarray:
    """Cosine of every pair of tile embeddings from the canonical dot
    products: G_ij / sqrt(G_ii * G_jj), 0 where that denominator is 0."""
    n = E.shape[0]
    G = np.empty((n, n), dtype=np.float64)
    for j in range(n):
        G[:, j] = cdot(E, E[j])
    g = np.diag(G).copy()
    den = np.sqrt(g[:, None] * g[None, :])
    with np.errstate(invalid="ignore", divide="ignore"):
        cos = G / den
    return np.where(den == 0.0, 0.0, cos)


def knn_smooth(s: np.ndarray, cos: np.ndarray, m: int):
    """Smoothed scores and neighbour lists: the m (at most n - 1) largest
    cos[i, j] over j != i, ties to the lower j; s'_i = (s_i + s_j1 + ... +
    s_jm) / (1 + m), added in that order (reading R8)."""
    n = s.shape[0]
    m_eff = min(m, n - 1)
    out = np.empty(n, dtype=np.float64)
    nbrs = []
    for i in range(n):
        js = sorted((j for j in range(n) if j != i), key=lambda j: (-cos[i, j], j))[:m_eff]
        acc = float(s[i])
        for j in js:
            acc = acc + float(s[j])
        out[i] = acc / (1 + m_eff)
        nbrs.append(js)
    return out, nbrs


# ------------------------------------------------- optional contextual merge (R14)


def split_budget(c: int, n_v: int, num: int = 10, den: int = 64) -> Tuple[int, int]:
    """(k_d, k_c): dominant and contextual tokens of a budget c (reading R14):
    k_c = min(floor(c num / den), n_v - c), k_d = c - k_c."""
    k_c = min((c * num) // den, n_v - c)
    return c - k_c, k_c


def round_f32_to_bf16(v: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values, round to nearest even
    on the 16 dropped bits (values here are finite)."""
    b = np.asarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def merge_context(x: np.ndarray, dominant: Sequence[int], k_c: int):
    """Contextual tokens of one tile (reading R14).  x: [n_v, d] float64 (the
    stored token values); dominant: the dominant token indices.  Returns
    (values [k_c, d] float64 holding float32 values, groups: list of k_c
    ascending index lists, targets).  Rounding to bfloat16 storage is
    round_f32_to_bf16 of the values."""
    n_v = x.shape[0]
    dom = set(int(t) for t in dominant)
    R = [t for t in range(n_v) if t not in dom]
    if k_c == 0:
        return np.zeros((0, x.shape[1])), [], []
    if k_c > len(R):
        raise ValueError("more contextual tokens than remaining tokens")
    targets = [R[(j * len(R)) // k_c] for j in range(k_c)]
    inv_t = token_inv_norms(x[targets])
    groups = [[t] for t in targets]
    tset = set(targets)
    others = [r for r in R if r not in tset]
    xt = x[targets]
    for i0 in range(0, len(others), 64):       # 64 tokens at a time, every target
        blk = others[i0:i0 + 64]
        a = cdot(np.repeat(x[blk][:, None, :], k_c, axis=1), xt[None, :, :]) * inv_t
        for i, r in enumerate(blk):
            best = 0                            # largest score, ties to the lower j
            for j in range(1, k_c):
                if a[i, j] > a[i, best]:
                    best = j
            groups[best].append(r)
    vals = np.zeros((k_c, x.shape[1]), dtype=np.float64)
    for j, grp in enumerate(groups):
        grp.sort()
        acc = np.zeros(x.shape[1], dtype=np.float64)
        for t in grp:
            acc = acc + x[t]
        vals[j] = (acc / len(grp)).astype(np.float32).astype(np.float64)
    return vals, groups, targets


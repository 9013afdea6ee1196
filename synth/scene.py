"""Seeded synthetic scenes and decoder weights for the Rift hot path.

This is the one module that both the GPU path's tests and the oracle take their
inputs from.  It draws random numbers and rounds them to the storage type; it
contains none of the method's arithmetic (no scores, no selection, no layers).

Stand-ins for what the paper measures on (Sec. 3 Setup, App. A): the xView and
GLH-Bridge imagery, RemoteCLIP and LLaVA-1.5-7B weights are not available, so
tile tokens are Gaussian post-projection embeddings, the query object and the
background phrases are random unit vectors, and decoder weights are N(0, 0.02).

Storage types: "bf16" arrays are numpy uint16 bit patterns (round to nearest
even from float32); "f32" arrays are numpy float32.

Seeds: workload c uses base 0x52494654 + c ("RIFT").  Each tensor draws from
numpy's PCG64 streams keyed by (base, stream_id, ...):

    0  tile tokens (one sub-stream per tile)
    1  caption templates averaged into t
    2  background phrases B_j
    3  which tiles are planted
    4  planted token subsets and fractions
    5  system prompt tokens
    6  query text tokens
    1000 + l   layer l weights: sub-stream (matrix, row-chunk), matrices in the
               order q, k, v, o, gate, up, down
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Dict, List, Tuple

import numpy as np

from .configs import Workload

_ROW_CHUNK = 256


def n_workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _pool() -> ThreadPoolExecutor:
    return ThreadPoolExecutor(max_workers=n_workers())


# ----------------------------------------------------------------------------- rounding
def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.
    Finite inputs only (the generator never produces NaN or Inf)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values to float64."""
    if dtype == "bf16":
        return bf16_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def store(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to the storage type."""
    return round_bf16(x32) if dtype == "bf16" else np.ascontiguousarray(x32, dtype=np.float32)


def _normal(key: Tuple[int, ...], n: int) -> np.ndarray:
    return np.random.default_rng(list(key)).standard_normal(n, dtype=np.float32)


# ----------------------------------------------------------------------------- scene
@dataclass
class Scene:
    w: Workload
    tokens: np.ndarray        # [n_tiles][n_v][d]   storage type
    qbank: np.ndarray         # [1 + n_bg][d]       row 0 = t, rows 1.. = B_j
    sys: np.ndarray           # [n_sys][d]
    qry: np.ndarray           # [n_qry][d]
    planted: np.ndarray       # planted tile ids (sorted)
    planted_mask: np.ndarray  # [n_tiles][n_v] bool: token carries the planted component

    @property
    def dtype(self) -> str:
        return self.w.dtype


def _unit_rows(raw: np.ndarray) -> np.ndarray:
    r = raw.astype(np.float64)
    return r / np.sqrt((r * r).sum(axis=-1, keepdims=True))


def make_query_bank(w: Workload) -> np.ndarray:
    """Row 0: t = unit(mean of n_templates Gaussian template embeddings);
    rows 1..n_bg: unit Gaussian background phrases.  Unit-normalised in float64,
    then rounded to the storage type; the rounded values are the inputs."""
    d, base = w.model.d, w.seed_base
    tmpl = _normal((base, 1), w.n_templates * d).reshape(w.n_templates, d)
    t = _unit_rows(tmpl.astype(np.float64).mean(axis=0, keepdims=True))
    bg = _unit_rows(_normal((base, 2), w.n_bg * d).reshape(w.n_bg, d))
    bank = np.concatenate([t, bg], axis=0).astype(np.float32)
    return store(bank, w.dtype)


def _planted_layout(w: Workload) -> Tuple[np.ndarray, Dict[int, np.ndarray]]:
    if isinstance(w.planted_tiles, int):
        rng = np.random.default_rng([w.seed_base, 3])
        tiles = np.sort(rng.choice(w.n_tiles, size=w.planted_tiles, replace=False))
    else:
        tiles = np.array(sorted(w.planted_tiles), dtype=np.int64)
    rng = np.random.default_rng([w.seed_base, 4])
    rows = {}
    lo, hi = w.planted_frac
    for tid in tiles:
        frac = lo if hi == lo else rng.uniform(lo, hi)
        cnt = int(np.floor(frac * w.n_v))
        rows[int(tid)] = np.sort(rng.choice(w.n_v, size=cnt, replace=False))
    return tiles, rows


def make_scene(w: Workload) -> Scene:
    d, base = w.model.d, w.seed_base
    qbank = make_query_bank(w)
    t32 = bf16_to_f32(qbank[0]) if w.dtype == "bf16" else qbank[0].astype(np.float32)
    tiles, rows = _planted_layout(w)
    mask = np.zeros((w.n_tiles, w.n_v), dtype=bool)
    for tid, rr in rows.items():
        mask[tid, rr] = True

    out_dt = np.uint16 if w.dtype == "bf16" else np.float32
    tokens = np.empty((w.n_tiles, w.n_v, d), dtype=out_dt)

    def one_tile(i: int) -> None:
        x = _normal((base, 0, i), w.n_v * d).reshape(w.n_v, d)
        if i in rows:
            x[rows[i]] += np.float32(w.planted_alpha) * t32
        tokens[i] = store(x, w.dtype)

    with _pool() as ex:
        list(ex.map(one_tile, range(w.n_tiles)))
    sys = store(_normal((base, 5), w.n_sys * d).reshape(w.n_sys, d), w.dtype)
    qry = store(_normal((base, 6), w.n_qry * d).reshape(w.n_qry, d), w.dtype)
    return Scene(w, tokens, qbank, sys, qry, tiles, mask)


# ----------------------------------------------------------------------------- weights
WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def weight_shapes(w: Workload) -> Dict[str, Tuple[int, int]]:
    m = w.model
    d, f = m.d, m.ffn
    return {"wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
            "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f)}


def make_layer(w: Workload, layer: int) -> Dict[str, np.ndarray]:
    """Weights of decoder layer `layer`, nn.Linear layout [out][in], N(0, std)
    rounded to the storage type; RMSNorm gains are 1 (LLaMA's initialisation)."""
    shapes = weight_shapes(w)
    std = np.float32(w.model.weight_std)
    out: Dict[str, np.ndarray] = {}
    jobs: List[Tuple[str, int, int, int]] = []
    for mi, name in enumerate(WEIGHT_NAMES):
        rows, cols = shapes[name]
        out[name] = np.empty((rows, cols), dtype=np.uint16 if w.dtype == "bf16" else np.float32)
        for c0 in range(0, rows, _ROW_CHUNK):
            jobs.append((name, mi, c0, min(rows, c0 + _ROW_CHUNK)))

    def fill(job):
        name, mi, r0, r1 = job
        cols = shapes[name][1]
        x = _normal((w.seed_base, 1000 + layer, mi, r0 // _ROW_CHUNK), (r1 - r0) * cols)
        x *= std
        out[name][r0:r1] = store(x.reshape(r1 - r0, cols), w.dtype)

    with _pool() as ex:
        list(ex.map(fill, jobs))
    one = np.ones(w.model.d, dtype=np.float32)
    out["g_attn"] = store(one, w.dtype)
    out["g_ffn"] = store(one, w.dtype)
    return out

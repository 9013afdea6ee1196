"""ctypes binding of librift.so (include/rift.h).

Argument marshalling only: every function here checks tensor shapes, dtypes
and devices, passes raw pointers and the current HIP stream to the C ABI, and
raises RiftError on a non-OK status.  All computation happens in the HIP
kernels of the library; there is no fallback path.  PyTorch serves as the
device allocator and stream provider.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librift.so")

RIFT_OK = 0
STATUS_NAMES = {0: "RIFT_OK", 1: "RIFT_ERR_NULL", 2: "RIFT_ERR_SHAPE", 3: "RIFT_ERR_DTYPE",
                4: "RIFT_ERR_BUDGET", 5: "RIFT_ERR_WORKSPACE", 6: "RIFT_ERR_HIP",
                7: "RIFT_ERR_NONFINITE", 8: "RIFT_ERR_UNSUPPORTED"}
RIFT_F32 = 0
RIFT_BF16 = 1

# Every symbol include/rift.h declares, in declaration order.
EXPORTS = ("rift_abi_version", "rift_status_string", "rift_set_debug", "rift_check_finite",
           "rift_score_workspace_size",
           "rift_score_tiles", "rift_score_tiles_noalloc", "rift_assign_budgets", "rift_assign_budgets_utility",
           "rift_select_tokens", "rift_split_budgets", "rift_merge_workspace_size", "rift_merge_context",
           "rift_compact",
           "rift_prefill_workspace_size", "rift_prefill", "rift_decode_workspace_size", "rift_decode_step")


class RiftError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({_status_text(status)})")


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "g_attn", "g_ffn")]


class ModelCfg(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ffn", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("dt", ctypes.c_int32)]


_lib: Optional[ctypes.CDLL] = None


def lib_available() -> bool:
    return os.path.exists(LIB_PATH)


def load() -> ctypes.CDLL:
    """Load librift.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_29029_amd.build` (there is no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ, F64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double
    L.rift_abi_version.restype = I32
    L.rift_abi_version.argtypes = []
    L.rift_status_string.restype = ctypes.c_char_p
    L.rift_status_string.argtypes = [I32]
    L.rift_set_debug.restype = I32
    L.rift_set_debug.argtypes = [I32]
    L.rift_check_finite.restype = I32
    L.rift_check_finite.argtypes = [P, I32, I64, P, P]
    L.rift_score_workspace_size.restype = SZ
    L.rift_score_workspace_size.argtypes = [I32, I32, I32, I32]
    L.rift_score_tiles.restype = I32
    L.rift_score_tiles.argtypes = [P, I32, I32, I32, I32, P, I32, I32, F64, I32, P, P, P, P, P, P, P, SZ, P]
    L.rift_score_tiles_noalloc.restype = I32
    L.rift_score_tiles_noalloc.argtypes = [P, I32, I32, I32, I32, P, I32, I32, F64, I32, P, P, P, P, P, P, P]
    L.rift_assign_budgets.restype = I32
    L.rift_assign_budgets.argtypes = [I32, I32, P, I32, P, I32, P, P]
    L.rift_assign_budgets_utility.restype = I32
    L.rift_assign_budgets_utility.argtypes = [I32, I32, I32, P, P, P, P, F64, P, P, P]
    L.rift_select_tokens.restype = I32
    L.rift_select_tokens.argtypes = [P, I32, I32, P, P, I32, P, P, I64, P, P]
    L.rift_split_budgets.restype = I32
    L.rift_split_budgets.argtypes = [I32, I32, P, I32, I32, P, P]
    L.rift_merge_workspace_size.restype = SZ
    L.rift_merge_workspace_size.argtypes = [I32, I32]
    L.rift_merge_context.restype = I32
    L.rift_merge_context.argtypes = [P, I32, I32, I32, I32, P, P, P, P, I32, P, I64, P, P, SZ, P]
    L.rift_compact.restype = I32
    L.rift_compact.argtypes = [P, I32, I32, I32, I32, P, P, P, I32, P, P, P, I32, P, I32, I32, P, I64, P, P, P, P]
    L.rift_prefill_workspace_size.restype = SZ
    L.rift_prefill_workspace_size.argtypes = [ctypes.POINTER(ModelCfg), I32, I32]
    L.rift_decode_workspace_size.restype = SZ
    L.rift_decode_workspace_size.argtypes = [ctypes.POINTER(ModelCfg), I32, I32, I32]
    L.rift_decode_step.restype = I32
    L.rift_decode_step.argtypes = [ctypes.POINTER(ModelCfg), ctypes.POINTER(LayerWeights), P, P, I32, I32, I32,
                                   I32, P, P, I32, I32, P, P, SZ, P]
    L.rift_prefill.restype = I32
    L.rift_prefill.argtypes = [ctypes.POINTER(ModelCfg), ctypes.POINTER(LayerWeights), P, I32, P, P,
                               I32, I32, I32, I32, P, P, P, SZ, P, P]
    _lib = L
    return L


def _status_text(s: int) -> str:
    try:
        return load().rift_status_string(int(s)).decode()
    except Exception:  # pragma: no cover - only for messages
        return "?"


def _check(status: int, where: str) -> None:
    if status != RIFT_OK:
        raise RiftError(status, where)


# ----------------------------------------------------------------------------- helpers
def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _dt_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return RIFT_BF16
    if t.dtype == torch.float32:
        return RIFT_F32
    raise TypeError(f"unsupported storage dtype {t.dtype}")


def _stream(stream) -> Optional[int]:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream) or None


def _need(t, dtype, shape=None, name="tensor"):
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a device tensor")


# ----------------------------------------------------------------------------- checks
def rift_set_debug(on: bool) -> bool:
    """Debug mode of the process on or off; returns the previous setting."""
    return bool(load().rift_set_debug(1 if on else 0))


def rift_check_finite(x, status, stream=None) -> None:
    """status[0] := 0, or RIFT_ERR_NONFINITE if x (bf16 or f32) holds NaN or
    infinity; enqueued on the stream like every call."""
    torch = _torch()
    _need(x, x.dtype, None, "x")
    _need(status, torch.int32, (1,), "status")
    _check(load().rift_check_finite(_ptr(x), _dt_code(x), x.numel(), _ptr(status), _stream(stream)),
           "rift_check_finite")


# ----------------------------------------------------------------------------- Stage 1
def rift_score_workspace_size(n_tiles: int, n_v: int, d: int, knn_m: int = 0) -> int:
    return int(load().rift_score_workspace_size(n_tiles, n_v, d, knn_m))


def rift_score_tiles(tokens, query_bank, keep_count: int, tau: float, token_key, token_sim,
                     tile_score, tile_u, tile_order, n_keep, workspace, stream=None,
                     knn_m: int = 0) -> None:
    torch = _torch()
    n_tiles, n_v, d = tokens.shape
    nq = query_bank.shape[0]
    dt = _dt_code(tokens)
    _need(tokens, tokens.dtype, name="tokens")
    _need(query_bank, tokens.dtype, (nq, d), "query_bank")
    _need(token_key, torch.float64, (n_tiles * n_v,), "token_key")
    if token_sim is not None:
        _need(token_sim, torch.float32, (n_tiles * n_v, nq), "token_sim")
    _need(tile_score, torch.float64, (n_tiles,), "tile_score")
    _need(tile_u, torch.float32, (n_tiles,), "tile_u")
    _need(tile_order, torch.int32, (n_tiles,), "tile_order")
    _need(n_keep, torch.int32, (1,), "n_keep")
    _need(workspace, torch.uint8, None, "workspace")
    st = load().rift_score_tiles(_ptr(tokens), dt, n_tiles, n_v, d, _ptr(query_bank), nq - 1,
                                 int(keep_count), float(tau), int(knn_m), _ptr(token_key), _ptr(token_sim),
                                 _ptr(tile_score), _ptr(tile_u), _ptr(tile_order), _ptr(n_keep),
                                 _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "rift_score_tiles")


def rift_score_tiles_noalloc(tokens, query_bank, keep_count: int, tau: float, token_key, token_sim,
                             tile_score, tile_u, tile_order, n_keep, stream=None, knn_m: int = 0) -> None:
    """rift_score_tiles on the library's static scratch (no workspace)."""
    torch = _torch()
    n_tiles, n_v, d = tokens.shape
    nq = query_bank.shape[0]
    dt = _dt_code(tokens)
    _need(tokens, tokens.dtype, name="tokens")
    _need(query_bank, tokens.dtype, (nq, d), "query_bank")
    _need(token_key, torch.float64, (n_tiles * n_v,), "token_key")
    if token_sim is not None:
        _need(token_sim, torch.float32, (n_tiles * n_v, nq), "token_sim")
    _need(tile_score, torch.float64, (n_tiles,), "tile_score")
    _need(tile_u, torch.float32, (n_tiles,), "tile_u")
    _need(tile_order, torch.int32, (n_tiles,), "tile_order")
    _need(n_keep, torch.int32, (1,), "n_keep")
    st = load().rift_score_tiles_noalloc(_ptr(tokens), dt, n_tiles, n_v, d, _ptr(query_bank), nq - 1,
                                         int(keep_count), float(tau), int(knn_m), _ptr(token_key),
                                         _ptr(token_sim), _ptr(tile_score), _ptr(tile_u), _ptr(tile_order),
                                         _ptr(n_keep), _stream(stream))
    _check(st, "rift_score_tiles_noalloc")


# ----------------------------------------------------------------------------- Stage 2
def rift_assign_budgets(n_keep: int, n_v: int, levels: Sequence[int],
                        tier_num: Optional[Sequence[int]], tier_den: int):
    """Host-only call; returns (budgets as int32 numpy array, total).  tier_num
    None selects the library default ({1, 3, 4}/16 over four levels)."""
    import numpy as np
    lv = np.ascontiguousarray(levels, dtype=np.int32)
    # a valid pointer even when no numerators are needed (a single level)
    tn = None if tier_num is None else np.ascontiguousarray(list(tier_num) + [0], dtype=np.int32)
    out = np.zeros(max(1, n_keep), dtype=np.int32)
    tot = ctypes.c_int64(0)
    st = load().rift_assign_budgets(int(n_keep), int(n_v), lv.ctypes.data, len(lv),
                                    None if tn is None else tn.ctypes.data, int(tier_den),
                                    out.ctypes.data, ctypes.byref(tot))
    _check(st, "rift_assign_budgets")
    return out[:n_keep].copy(), int(tot.value)


def rift_assign_budgets_utility(p, levels: Sequence[int], alpha_pos: Sequence[float],
                                alpha_neg: Sequence[float], energy: Sequence[float], lam: float,
                                n_v: int):
    """Host-only call (Eq. 2); p: per-tile probabilities (float32).  Returns
    (budgets as int32 numpy array, total)."""
    import numpy as np
    pv = np.ascontiguousarray(p, dtype=np.float32)
    lv = np.ascontiguousarray(levels, dtype=np.int32)
    ap = np.ascontiguousarray(alpha_pos, dtype=np.float64)
    an = np.ascontiguousarray(alpha_neg, dtype=np.float64)
    en = np.ascontiguousarray(energy, dtype=np.float64)
    out = np.zeros(max(1, pv.size), dtype=np.int32)
    tot = ctypes.c_int64(0)
    st = load().rift_assign_budgets_utility(int(pv.size), int(n_v), int(lv.size), lv.ctypes.data,
                                            ap.ctypes.data, an.ctypes.data, en.ctypes.data, float(lam),
                                            pv.ctypes.data, out.ctypes.data, ctypes.byref(tot))
    _check(st, "rift_assign_budgets_utility")
    return out[:pv.size].copy(), int(tot.value)


def rift_select_tokens(token_key, n_tiles: int, n_v: int, kept_tiles, budgets, n_keep: int,
                       sel_offsets, sel_idx, status, stream=None) -> None:
    torch = _torch()
    _need(token_key, torch.float64, (n_tiles * n_v,), "token_key")
    _need(sel_offsets, torch.int32, None, "sel_offsets")
    _need(status, torch.int32, (1,), "status")
    if sel_offsets.numel() < n_keep + 1:
        raise ValueError("sel_offsets needs n_keep + 1 entries")
    if n_keep > 0:
        _need(kept_tiles, torch.int32, None, "kept_tiles")
        _need(budgets, torch.int32, None, "budgets")
        if kept_tiles.numel() < n_keep or budgets.numel() < n_keep:
            raise ValueError("kept_tiles and budgets need n_keep entries")
    _need(sel_idx, torch.int32, None, "sel_idx")
    st = load().rift_select_tokens(_ptr(token_key), n_tiles, n_v, _ptr(kept_tiles), _ptr(budgets),
                                   int(n_keep), _ptr(sel_offsets), _ptr(sel_idx), sel_idx.numel(),
                                   _ptr(status), _stream(stream))
    _check(st, "rift_select_tokens")


def rift_split_budgets(budgets, n_v: int, num: int = 10, den: int = 64):
    """Host-only call: (dominant, context) int32 numpy arrays for budgets."""
    import numpy as np
    b = np.ascontiguousarray(budgets, dtype=np.int32)
    dom = np.zeros(max(1, b.size), dtype=np.int32)
    ctx = np.zeros(max(1, b.size), dtype=np.int32)
    st = load().rift_split_budgets(int(b.size), int(n_v), b.ctypes.data if b.size else None, int(num), int(den),
                                   dom.ctypes.data, ctx.ctypes.data)
    _check(st, "rift_split_budgets")
    return dom[:b.size].copy(), ctx[:b.size].copy()


def rift_merge_workspace_size(n_keep: int, n_v: int) -> int:
    return int(load().rift_merge_workspace_size(n_keep, n_v))


def rift_merge_context(tokens, kept_tiles, sel_offsets, sel_idx, ctx_offsets, n_keep: int, ctx_rows,
                       status, workspace, stream=None) -> None:
    torch = _torch()
    n_tiles, n_v, d = tokens.shape
    dt = _dt_code(tokens)
    _need(tokens, tokens.dtype, name="tokens")
    _need(ctx_rows, tokens.dtype, (ctx_rows.shape[0], d), "ctx_rows")
    _need(ctx_offsets, torch.int32, None, "ctx_offsets")
    _need(status, torch.int32, (1,), "status")
    _need(workspace, torch.uint8, None, "workspace")
    if ctx_offsets.numel() < n_keep + 1 or sel_offsets.numel() < n_keep + 1:
        raise ValueError("ctx_offsets and sel_offsets need n_keep + 1 entries")
    st = load().rift_merge_context(_ptr(tokens), dt, n_tiles, n_v, d, _ptr(kept_tiles), _ptr(sel_offsets),
                                   _ptr(sel_idx), _ptr(ctx_offsets), int(n_keep), _ptr(ctx_rows),
                                   ctx_rows.shape[0], _ptr(status), _ptr(workspace), workspace.numel(),
                                   _stream(stream))
    _check(st, "rift_merge_context")


def rift_compact(tokens, kept_tiles, sel_offsets, sel_idx, n_keep: int, sys_emb, qry_emb,
                 packed, cu_seqlens, position_ids, status, stream=None, ctx_rows=None,
                 ctx_offsets=None, shared_prefix: bool = False) -> None:
    """shared_prefix: the system rows once at the front as sequence 0;
    cu_seqlens then needs n_keep + 2 entries."""
    torch = _torch()
    n_tiles, n_v, d = tokens.shape
    dt = _dt_code(tokens)
    _need(tokens, tokens.dtype, name="tokens")
    _need(sys_emb, tokens.dtype, (sys_emb.shape[0], d), "sys_emb")
    _need(qry_emb, tokens.dtype, (qry_emb.shape[0], d), "qry_emb")
    _need(packed, tokens.dtype, (packed.shape[0], d), "packed")
    _need(cu_seqlens, torch.int32, None, "cu_seqlens")
    _need(position_ids, torch.int32, (packed.shape[0],), "position_ids")
    _need(status, torch.int32, (1,), "status")
    if cu_seqlens.numel() < n_keep + 1 + int(bool(shared_prefix)) or sel_offsets.numel() < n_keep + 1:
        raise ValueError("cu_seqlens needs n_keep + 1 entries (+ 1 with a shared prefix), sel_offsets n_keep + 1")
    if (ctx_rows is None) != (ctx_offsets is None):
        raise ValueError("ctx_rows and ctx_offsets go together")
    if ctx_rows is not None:
        _need(ctx_rows, tokens.dtype, (ctx_rows.shape[0], d), "ctx_rows")
        _need(ctx_offsets, torch.int32, None, "ctx_offsets")
        if ctx_offsets.numel() < n_keep + 1:
            raise ValueError("ctx_offsets needs n_keep + 1 entries")
    st = load().rift_compact(_ptr(tokens), dt, n_tiles, n_v, d, _ptr(kept_tiles), _ptr(sel_offsets),
                             _ptr(sel_idx), int(n_keep), _ptr(ctx_rows), _ptr(ctx_offsets),
                             _ptr(sys_emb), sys_emb.shape[0],
                             _ptr(qry_emb), qry_emb.shape[0], int(bool(shared_prefix)), _ptr(packed),
                             packed.shape[0], _ptr(cu_seqlens), _ptr(position_ids), _ptr(status),
                             _stream(stream))
    _check(st, "rift_compact")


# ----------------------------------------------------------------------------- prefill
def model_cfg(d, n_heads, head_dim, ffn, n_layers, rms_eps, rope_base, dt_code) -> ModelCfg:
    return ModelCfg(int(d), int(n_heads), int(head_dim), int(ffn), int(n_layers), float(rms_eps),
                    float(rope_base), int(dt_code))


def rift_prefill_workspace_size(cfg: ModelCfg, total_tokens: int, max_seqlen: int) -> int:
    return int(load().rift_prefill_workspace_size(ctypes.byref(cfg), int(total_tokens), int(max_seqlen)))


def layer_struct(w: dict) -> LayerWeights:
    return LayerWeights(*[_ptr(w[n]) for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
                                                "g_attn", "g_ffn")])


def rift_prefill(cfg: ModelCfg, layers: Sequence[dict], x_in, cu_seqlens, position_ids,
                 n_seq: int, max_seqlen: int, hidden_out, workspace, kv_cache=None,
                 events=None, stream=None, n_prefix: int = 0) -> None:
    """events: optional list of 10 * n_layers torch.cuda.Event(enable_timing=True)
    or None (that mark skipped), recorded around each per-layer stage (see
    include/rift.h).  n_prefix > 0: sequence 0 is a prefix shared by every
    other sequence."""
    torch = _torch()
    T = x_in.shape[0]
    if len(layers) != cfg.n_layers:
        raise ValueError("need one weight set per layer")
    wdt = torch.bfloat16 if cfg.dt == RIFT_BF16 else torch.float32
    for w in layers:
        for n, v in w.items():
            _need(v, wdt, None, n)
    _need(hidden_out, torch.float32, (T, cfg.d), "hidden_out")
    _need(cu_seqlens, torch.int32, (n_seq + 1,), "cu_seqlens")
    _need(position_ids, torch.int32, (T,), "position_ids")
    _need(workspace, torch.uint8, None, "workspace")
    arr = (LayerWeights * max(1, len(layers)))(*[layer_struct(w) for w in layers])
    ev = None
    if events is not None:
        if len(events) != 10 * cfg.n_layers:
            raise ValueError("events needs 10 entries per layer")
        for e in events:          # torch creates the hipEvent on its first record()
            if e is not None and not e.cuda_event:
                e.record()
        ev = (ctypes.c_void_p * len(events))(*[None if e is None else int(e.cuda_event) for e in events])
    st = load().rift_prefill(ctypes.byref(cfg), arr, _ptr(x_in), _dt_code(x_in), _ptr(cu_seqlens),
                             _ptr(position_ids), int(n_seq), int(T), int(max_seqlen), int(n_prefix),
                             _ptr(hidden_out), _ptr(kv_cache), _ptr(workspace), workspace.numel(),
                             ev, _stream(stream))
    _check(st, "rift_prefill")


# ----------------------------------------------------------------------------- decode
def rift_decode_workspace_size(cfg: ModelCfg, n_seq: int, max_seqlen: int, max_new: int) -> int:
    return int(load().rift_decode_workspace_size(ctypes.byref(cfg), int(n_seq), int(max_seqlen), int(max_new)))


def rift_decode_step(cfg: ModelCfg, layers: Sequence[dict], x_new, cu_seqlens, total_tokens: int,
                     max_seqlen: int, kv_cache, kv_new, step: int, hidden_out, workspace,
                     stream=None, n_prefix: int = 0) -> None:
    """One generated token per prompt after rift_prefill (include/rift.h).
    x_new [n_seq][d] bf16; kv_new [n_layers][2][n_seq][max_new][d] bf16;
    n_prefix > 0: the prefill's sequence 0 was a shared prefix (cu_seqlens then
    has n_seq + 2 entries)."""
    torch = _torch()
    n_seq = x_new.shape[0]
    if len(layers) != cfg.n_layers:
        raise ValueError("need one weight set per layer")
    for w in layers:
        for n, v in w.items():
            _need(v, torch.bfloat16, None, n)
    _need(x_new, torch.bfloat16, (n_seq, cfg.d), "x_new")
    _need(cu_seqlens, torch.int32, (n_seq + (2 if n_prefix > 0 else 1),), "cu_seqlens")
    _need(kv_new, torch.bfloat16, None, "kv_new")
    if kv_new.dim() != 5 or tuple(kv_new.shape[:3]) != (cfg.n_layers, 2, n_seq) or kv_new.shape[4] != cfg.d:
        raise ValueError("kv_new must be [n_layers][2][n_seq][max_new][d]")
    if kv_cache is not None:
        _need(kv_cache, torch.bfloat16, (cfg.n_layers, 2, int(total_tokens), cfg.d), "kv_cache")
    _need(hidden_out, torch.float32, (n_seq, cfg.d), "hidden_out")
    _need(workspace, torch.uint8, None, "workspace")
    arr = (LayerWeights * max(1, len(layers)))(*[layer_struct(w) for w in layers])
    st = load().rift_decode_step(ctypes.byref(cfg), arr, _ptr(x_new), _ptr(cu_seqlens), int(n_seq),
                                 int(total_tokens), int(max_seqlen), int(n_prefix), _ptr(kv_cache), _ptr(kv_new),
                                 int(kv_new.shape[3]), int(step), _ptr(hidden_out), _ptr(workspace),
                                 workspace.numel(), _stream(stream))
    _check(st, "rift_decode_step")


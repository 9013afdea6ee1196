"""Shared helpers of the GPU parity tests: upload seeded inputs, run the oracle
on the same stored values, compare."""
from __future__ import annotations

import numpy as np

import synth
from oracle import rift_oracle as O


def torch_mod():
    import torch
    return torch


def upload(a: np.ndarray, dtype: str):
    """Stored synth array -> device tensor of the storage type."""
    torch = torch_mod()
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def download_stored(t, dtype: str) -> np.ndarray:
    """Device tensor of the storage type -> stored numpy representation."""
    torch = torch_mod()
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def upload_layer(W: dict, dtype: str) -> dict:
    return {k: upload(v, dtype) for k, v in W.items()}


def f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return synth.to_f64(a, dtype)


def rowwise_rel_err(y: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of ||y - ref||_inf / ||ref||_inf."""
    num = np.abs(y - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    return float((num / den).max())


def oracle_stage1(scene: synth.Scene, keep_count: int, tau: float):
    return O.scene_query_stage1(f64(scene.tokens, scene.dtype), f64(scene.qbank, scene.dtype),
                                keep_count, tau)


def oracle_layer_weights(W: dict, dtype: str) -> dict:
    return {k: f64(v, dtype) for k, v in W.items()}


def plan_shape(w: synth.Workload):
    from paper_2609_29029_amd.pipeline import PrefillShape
    m = w.model
    return PrefillShape(m.d, m.n_heads, m.head_dim, m.ffn, m.n_layers, m.rms_eps, m.rope_base)


def shared_layout(r_packed, r_cu, r_pos, n_sys):
    """The oracle's per-prompt layout rearranged as a shared prefix: the first
    prompt's n_sys system rows once, then every prompt's rows after them."""
    rows = [r_packed[:n_sys]]
    pos = [np.arange(n_sys)]
    cu = [0, n_sys]
    for i in range(len(r_cu) - 1):
        a, b = int(r_cu[i]) + n_sys, int(r_cu[i + 1])
        rows.append(r_packed[a:b])
        pos.append(r_pos[a:b])
        cu.append(cu[-1] + b - a)
    return np.concatenate(rows), np.array(cu), np.concatenate(pos)

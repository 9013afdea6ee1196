"""One Rift scene-query on the GPU: score -> budgets -> select -> (merge) ->
compact -> prefill, enqueued on one stream through the C ABI.  Buffers are allocated once
per plan (PyTorch as the allocator) and reused across queries.

In keep-top-K mode with rank-tier budgets the number of kept tiles, the
budgets and the packed length are known on the host before the query runs, so
the whole query is enqueued without a device-to-host copy.  Threshold mode
(keep_count == 0) reads n_keep back once after scoring; the Eq. 2 utility
policy reads the kept tiles' normalised scores back once (they stand in for the
object probability p) and assigns budgets on the host.  With `merge`, each
budget is split into dominant and contextual tokens (VisionZip's merge of the
remainder); the prompt length stays the budget.  With `shared_prefix` the
system rows, the same at the head of every prompt, are packed and prefilled
once as sequence 0; the prompts' results are unchanged (causal attention).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

from . import _lib as R


@dataclass
class PrefillShape:
    d: int
    n_heads: int
    head_dim: int
    ffn: int
    n_layers: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0


class SceneQuery:
    """Device buffers and launch sequence of one scene-query shape.

    tokens [n_tiles][n_v][d], qbank [1+M][d], sys [n_sys][d], qry [n_qry][d] and
    every layer weight are device tensors of one storage dtype (bf16 or f32)."""

    def __init__(self, tokens, qbank, sys_emb, qry_emb, layers: Sequence[dict],
                 shape: PrefillShape, keep_count: int, tau: float, levels: Sequence[int],
                 tier_num: Optional[Sequence[int]], tier_den: int, with_sims: bool = True,
                 stream=None, knn_m: int = 0, utility: Optional[dict] = None,
                 merge: Optional[Sequence[int]] = None, shared_prefix: bool = False):
        import torch
        self.torch = torch
        self.dev = tokens.device
        self.tokens, self.qbank, self.sys, self.qry = tokens, qbank, sys_emb, qry_emb
        self.layers = list(layers)
        self.shape = shape
        self.keep_count, self.tau = int(keep_count), float(tau)
        self.levels, self.tier_num, self.tier_den = list(levels), tier_num, int(tier_den)
        self.stream = stream
        self.knn_m = int(knn_m)
        # utility: dict(levels, alpha_pos, alpha_neg, energy, lam) for the Eq. 2 policy
        self.utility = utility
        # merge: (num, den) of the contextual share of each budget, or None
        self.merge = None if merge is None else (int(merge[0]), int(merge[1]))
        self.shared = bool(shared_prefix)
        self.n_prefix = sys_emb.shape[0] if self.shared else 0
        n_tiles, n_v, d = tokens.shape
        self.n_tiles, self.n_v, self.d = n_tiles, n_v, d
        nq = qbank.shape[0]
        dev = self.dev
        f64, f32, i32 = torch.float64, torch.float32, torch.int32
        self.token_key = torch.empty(n_tiles * n_v, dtype=f64, device=dev)
        self.token_sim = torch.empty(n_tiles * n_v, nq, dtype=f32, device=dev) if with_sims else None
        self.tile_score = torch.empty(n_tiles, dtype=f64, device=dev)
        self.tile_u = torch.empty(n_tiles, dtype=f32, device=dev)
        self.tile_order = torch.empty(n_tiles, dtype=i32, device=dev)
        self.n_keep_dev = torch.empty(1, dtype=i32, device=dev)
        self.score_ws = torch.empty(max(256, R.rift_score_workspace_size(n_tiles, n_v, d, self.knn_m)),
                                    dtype=torch.uint8, device=dev)
        self.sel_status = torch.empty(1, dtype=i32, device=dev)
        self.cmp_status = torch.empty(1, dtype=i32, device=dev)
        self.mrg_status = torch.zeros(1, dtype=i32, device=dev)
        self.cfg = R.model_cfg(shape.d, shape.n_heads, shape.head_dim, shape.ffn, shape.n_layers,
                               shape.rms_eps, shape.rope_base,
                               R.RIFT_BF16 if tokens.dtype == torch.bfloat16 else R.RIFT_F32)
        self._planned_keep = None
        self._cap = (0, 0)
        if self.keep_count > 0 and utility is None:
            self._plan(min(self.keep_count, n_tiles))

    # host-side plan for a given number of kept tiles (and budgets, in utility mode)
    def _plan(self, n_keep: int, budgets=None) -> None:
        import numpy as np
        torch = self.torch
        if budgets is None:
            if self._planned_keep == n_keep:
                return
            budgets, total = R.rift_assign_budgets(n_keep, self.n_v, self.levels, self.tier_num,
                                                   self.tier_den)
        else:
            budgets = np.ascontiguousarray(budgets, dtype=np.int32)
            total = int(budgets.sum())
        self.n_keep = n_keep
        self.budgets_host = budgets
        self.n_selected = total      # vision tokens per query (dominant + contextual)
        if self.merge is not None:
            dom, ctx = R.rift_split_budgets(budgets, self.n_v, *self.merge)
        else:
            dom, ctx = budgets, np.zeros(len(budgets), dtype=np.int32)
        self.n_dominant, self.n_context = int(dom.sum()), int(ctx.sum())
        fixed = self.sys.shape[0] + self.qry.shape[0]
        self.max_seqlen = fixed + (int(budgets.max()) if n_keep > 0 else 0)
        if self.shared:
            self.total_tokens = self.n_prefix + n_keep * self.qry.shape[0] + total
        else:
            self.total_tokens = n_keep * fixed + total
        dev = self.dev
        self.budgets = torch.from_numpy(budgets).to(dev) if n_keep > 0 else \
            torch.zeros(1, dtype=torch.int32, device=dev)
        # the budgets select works with: the dominant share when merging
        self.sel_budgets = torch.from_numpy(np.ascontiguousarray(dom, dtype=np.int32)).to(dev) \
            if n_keep > 0 else torch.zeros(1, dtype=torch.int32, device=dev)
        if self.merge is not None:
            coffs = np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32)
            self.ctx_offsets = torch.from_numpy(coffs).to(dev)
            self.ctx_rows = torch.empty(max(1, self.n_context), self.d, dtype=self.tokens.dtype, device=dev)
            mws = max(256, R.rift_merge_workspace_size(n_keep, self.n_v))
            if mws > getattr(self, "_mws_cap", 0):
                self.merge_ws = torch.empty(mws, dtype=torch.uint8, device=dev)
                self._mws_cap = mws
        # buffers grow to the largest plan seen and are reused
        T, P = self.total_tokens, max(1, self.max_seqlen)
        if n_keep + 2 > self._cap[0] or T > self._cap[1] or self._planned_keep is None:
            cap_keep = max(n_keep + 2, self._cap[0])
            cap_T = max(T, self._cap[1], 1)
            self.sel_offsets_all = torch.empty(cap_keep, dtype=torch.int32, device=dev)
            self.cu_seqlens_all = torch.empty(cap_keep, dtype=torch.int32, device=dev)
            self.sel_idx = torch.empty(max(1, cap_T), dtype=torch.int32, device=dev)
            self.packed_all = torch.empty(cap_T, self.d, dtype=self.tokens.dtype, device=dev)
            self.position_all = torch.empty(cap_T, dtype=torch.int32, device=dev)
            self.hidden_all = torch.empty(cap_T, self.d, dtype=torch.float32, device=dev)
            self._cap = (cap_keep, cap_T)
            self._ws_cap = 0
        self.sel_offsets = self.sel_offsets_all[:n_keep + 1]
        self.cu_seqlens = self.cu_seqlens_all[:n_keep + (2 if self.shared else 1)]
        self.n_seq = n_keep + (1 if self.shared else 0)   # sequences of the prefill
        self.packed = self.packed_all[:T]
        self.position_ids = self.position_all[:T]
        self.hidden = self.hidden_all[:T]
        ws = max(256, R.rift_prefill_workspace_size(self.cfg, T, P))
        if ws > getattr(self, "_ws_cap", 0):
            self.prefill_ws = torch.empty(ws, dtype=torch.uint8, device=dev)
            self._ws_cap = ws
        self._planned_keep = n_keep

    def score(self) -> None:
        R.rift_score_tiles(self.tokens, self.qbank, self.keep_count, self.tau, self.token_key,
                           self.token_sim, self.tile_score, self.tile_u, self.tile_order,
                           self.n_keep_dev, self.score_ws, self.stream, knn_m=self.knn_m)

    def select(self) -> None:
        R.rift_select_tokens(self.token_key, self.n_tiles, self.n_v, self.tile_order, self.sel_budgets,
                             self.n_keep, self.sel_offsets, self.sel_idx[:max(1, self.n_dominant)],
                             self.sel_status, self.stream)

    def merge_context(self) -> None:
        if self.merge is None:
            return
        R.rift_merge_context(self.tokens, self.tile_order, self.sel_offsets, self.sel_idx,
                             self.ctx_offsets, self.n_keep, self.ctx_rows[:self.n_context],
                             self.mrg_status, self.merge_ws, self.stream)

    def compact(self) -> None:
        merging = self.merge is not None
        R.rift_compact(self.tokens, self.tile_order, self.sel_offsets, self.sel_idx, self.n_keep,
                       self.sys, self.qry, self.packed, self.cu_seqlens, self.position_ids,
                       self.cmp_status, self.stream,
                       ctx_rows=self.ctx_rows if merging else None,
                       ctx_offsets=self.ctx_offsets if merging else None, shared_prefix=self.shared)

    def prefill(self, events=None) -> None:
        if self.total_tokens == 0:
            return
        R.rift_prefill(self.cfg, self.layers, self.packed, self.cu_seqlens, self.position_ids,
                       self.n_seq, max(1, self.max_seqlen), self.hidden, self.prefill_ws,
                       events=events, stream=self.stream, n_prefix=self.n_prefix)

    def plan_utility(self) -> None:
        """Eq. 2 budgets for the kept tiles, with each tile's normalised score u
        as its object probability p (reads the scores back)."""
        ut = self.utility
        n_keep = int(self.n_keep_dev.item())
        order = self.tile_order[:n_keep].long()
        p = self.tile_u[order].cpu().numpy()
        budgets, _ = R.rift_assign_budgets_utility(p, ut["levels"], ut["alpha_pos"], ut["alpha_neg"],
                                                   ut["energy"], ut["lam"], self.n_v)
        self._plan(n_keep, budgets)

    def run(self) -> None:
        """Enqueue the whole scene-query.  Threshold mode and the utility
        policy synchronise once after scoring."""
        self.score()
        if self.keep_count == 0 or self.utility is not None:
            self.torch.cuda.current_stream().synchronize() if self.stream is None else \
                self.stream.synchronize()
            if self.utility is not None:
                self.plan_utility()
            else:
                self._plan(int(self.n_keep_dev.item()))
        self.select()
        self.merge_context()
        self.compact()
        self.prefill()

    def check_status(self) -> List[int]:
        """Device status words of select and compact, and of the merge when
        it runs (synchronises)."""
        st = [int(self.sel_status.item()), int(self.cmp_status.item())]
        if self.merge is not None:
            st.append(int(self.mrg_status.item()))
        return st

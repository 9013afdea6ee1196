"""Rift hot path on AMD Instinct MI355X: query-conditioned tile scoring and
pruning, elastic per-tile token selection, varlen compaction and LLaMA-7B-shaped
prefill, as hand-written HIP kernels behind the C ABI of include/rift.h."""
from ._lib import (EXPORTS, LIB_PATH, RIFT_BF16, RIFT_F32, LayerWeights, ModelCfg,  # noqa: F401
                   RiftError, lib_available, load, model_cfg, rift_assign_budgets,
                   rift_assign_budgets_utility, rift_check_finite, rift_compact, rift_decode_step,
                   rift_decode_workspace_size,
                   rift_merge_context, rift_merge_workspace_size, rift_prefill,
                   rift_prefill_workspace_size, rift_score_tiles, rift_score_tiles_noalloc,
                   rift_score_workspace_size,
                   rift_select_tokens, rift_set_debug, rift_split_budgets)

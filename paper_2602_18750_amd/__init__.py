"""libhill: HillInfer's per-decode-step token-importance path (arxiv
2602.18750) -- importance scoring, top-k selection and sparse decode
attention -- as hand-written HIP kernels for AMD Instinct MI355X (gfx950)
behind a C ABI (``include/hill.h``).

Importing the package loads nothing; the shared library is loaded on the
first call of a binding function and is required (there is no fallback).
"""
from .hill import (AppParams, AppPlan, BkpCall, BkpDesc, BkpState, HillDesc, HillError, HillStepEvents, Sketch,
                   StepCall, app_balance, bkp_update, budget_k, hill_gather_attn, hill_score, hill_step,
                   hill_step_noalloc, hill_step_tiered, hill_tier_apply, hill_topk, load_library, make_desc,
                   new_importance, new_sketch, new_stream_state, sketch_keys, TierApplyCall, TierDesc, TieredCache, TierStepCall, workspace,
                   workspace_bytes)

__all__ = ["AppParams", "AppPlan", "BkpCall", "BkpDesc", "BkpState", "HillDesc", "HillError", "HillStepEvents",
           "Sketch", "StepCall", "app_balance", "bkp_update", "budget_k", "hill_gather_attn", "hill_score",
           "hill_step", "hill_step_noalloc", "hill_step_tiered", "hill_tier_apply", "hill_topk", "load_library",
           "make_desc", "new_importance", "new_sketch", "new_stream_state", "sketch_keys", "TierApplyCall", "TierDesc", "TieredCache", "TierStepCall",
           "workspace", "workspace_bytes"]

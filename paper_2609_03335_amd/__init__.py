"""MI355X (gfx950) batched scoring of candidate physical execution plans.

The compute path is libwfplan.so (HIP kernels behind the C ABI of
include/wf_plan.h).  PyTorch is used only to hold device memory and to name
the HIP stream.
"""
from __future__ import annotations

from ._lib import (EXPORTS, KEY_DTYPE, SCORE_DTYPE, WF_EHIP, WF_EINVAL, WF_ENOMEM, WF_ENOWINDOW, WF_OK,
                   WF_EUNSUPPORTED, WF_SEARCH_RULES, WF_SEARCH_UNIFORM, WF_ST_CAPACITY, WF_ST_INELIGIBLE,
                   WF_ST_REPLICA, Context, WFError, load, wf_plan_argmin_noalloc, wf_plan_validate_window,
                   wf_plan_version)

__all__ = [
    "Context", "WFError", "wf_plan_argmin_noalloc", "SCORE_DTYPE", "KEY_DTYPE", "EXPORTS", "load", "wf_plan_validate_window",
    "wf_plan_version", "device_plans", "score_batch", "argmin", "scores_to_numpy",
    "keys_to_numpy",
    "WF_OK", "WF_EINVAL", "WF_ENOWINDOW", "WF_ENOMEM", "WF_EHIP", "WF_EUNSUPPORTED",
    "WF_ST_INELIGIBLE", "WF_ST_CAPACITY", "WF_ST_REPLICA", "WF_SEARCH_UNIFORM", "WF_SEARCH_RULES",
]


def device_plans(plans, device="cuda"):
    """Copy a host PlanBatch (workload.PlanBatch) to device tensors."""
    import numpy as np
    import torch
    n = plans.dev.shape[1]
    # the kernels read row-major [P][N] buffers: force C order on both sides
    dev = torch.from_numpy(np.ascontiguousarray(plans.dev)).to(device).contiguous()
    prio = torch.from_numpy(np.ascontiguousarray(plans.prio).view("<i2")).to(device).contiguous()
    flags = torch.from_numpy(np.ascontiguousarray(plans.flags)).to(device).contiguous()
    if n == 0:  # keep a valid (unused) allocation behind empty rows
        dev = torch.zeros((plans.dev.shape[0], 1), dtype=torch.int8, device=device)
        prio = torch.zeros((plans.dev.shape[0], 1), dtype=torch.int16, device=device)
        flags = torch.zeros((plans.dev.shape[0], 1), dtype=torch.uint8, device=device)
    return dev, prio, flags


def score_batch(ctx: Context, dev, prio, flags, n_plans: int, schedule: bool = False,
                n_act: int = 0, n_dev: int = 0, stream=None, reclaims: bool = False):
    """Allocate outputs on the plans' device and enqueue scoring.  Returns
    the raw score buffer (uint8 [P, 32]) and, with ``schedule``, the
    (start, finish, load_start, peak) tensors, followed with ``reclaims`` by
    the [P, N] int64 tensor of reclaimed-model masks (uint64 bits)."""
    import torch
    device = dev.device
    scores = torch.empty((max(1, n_plans), 32), dtype=torch.uint8, device=device)
    sched = None
    if schedule:
        sched = (torch.empty((n_plans, max(1, n_act)), dtype=torch.int64, device=device),
                 torch.empty((n_plans, max(1, n_act)), dtype=torch.int64, device=device),
                 torch.empty((n_plans, max(1, n_act)), dtype=torch.int64, device=device),
                 torch.empty((n_plans, n_dev), dtype=torch.int32, device=device))
        if reclaims:
            sched = sched + (torch.empty((n_plans, max(1, n_act)), dtype=torch.int64, device=device),)
    ctx.wf_plan_score_batch(dev, prio, flags, n_plans, scores, sched, stream)
    return (scores, sched) if schedule else scores


def argmin(ctx: Context, scores, n_plans: int, stream=None):
    import torch
    out = torch.empty(1, dtype=torch.int64, device=scores.device)
    ctx.wf_plan_argmin(scores, n_plans, out, stream)
    return out


def scores_to_numpy(scores, n_plans: int):
    return scores[:n_plans].cpu().numpy().reshape(-1).view(SCORE_DTYPE)[:n_plans]


def keys_to_numpy(keys, n_plans: int):
    """Ranking keys (uint8 [P, 32] device buffer) as a KEY_DTYPE array."""
    return keys[:n_plans].cpu().numpy().reshape(-1).view(KEY_DTYPE)[:n_plans]

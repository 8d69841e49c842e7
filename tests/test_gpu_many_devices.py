"""Pools of 65 to 127 devices (plans carry int8 device ids): each lane of a
wave owns two devices of one plan.  Scores, schedules, reclaimed copies,
ranking keys and generated candidates bytewise against the oracle, under
each reclamation mode (4-bit queue with at most 16 models, the scan with
more, the paper's order, batch limits) and both time arithmetics."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03335_amd as pkg
from paper_2609_03335_amd import workload as W

pytestmark = pytest.mark.gpu
THREADS = max(1, min(16, os.cpu_count() or 1))


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    c = pkg.Context(0)
    yield c
    c.close()


def window(D, seed, M, mode):
    rng = np.random.default_rng(1000 * D + seed)
    kw = dict(n_wf=5, nodes=(3, 14), n_dev=D, n_models=M, same_model_bias=0.5,
              cap_range=(6000, 30000), w_range=(1000, 9000))
    if mode == "fp64":
        kw.update(lat_range=(1, 1 << 30), load_range=(0, 1 << 31))
    win = W.random_window(rng, **kw)
    if mode == "paper":
        win.victim_order = 1
    if mode == "batch":
        win.dev_batch = rng.integers(1, 5, D).astype(np.int32)
    return win, rng


CASES = [(D, seed, M, mode) for D, seed, M, mode in [
    (65, 0, 12, "queue"), (96, 1, 12, "queue"), (127, 2, 16, "queue"),
    (65, 3, 40, "scan"), (127, 4, 64, "scan"),
    (96, 5, 20, "paper"), (127, 6, 12, "paper"),
    (65, 7, 16, "batch"), (127, 8, 30, "batch"),
    (96, 9, 12, "fp64"), (127, 10, 24, "fp64")]]


@pytest.mark.parametrize("D,seed,M,mode", CASES)
def test_scores_and_schedules(ctx, D, seed, M, mode):
    win, rng = window(D, seed, M, mode)
    plans = W.random_plans(win, 300, rng, p_bad_dev=0.002, prio_mode=("any", "perm")[seed % 2])
    P, N = plans.n_plans, win.n_act
    log(f"[many-dev] D={D} M={M} mode={mode} N={N} P={P}")
    ctx.wf_plan_upload_window(win)
    assert ctx.wf_plan_score_kernel() == "score_plans"
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    s = pkg.score_batch(ctx, dev, prio, flags, P)
    s2, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D,
                                reclaims=True)
    torch.cuda.synchronize()
    ref, rs = oracle.score(win, plans, schedule=True, reclaims=True, threads=THREADS)
    assert pkg.scores_to_numpy(s, P).tobytes() == ref.tobytes()
    assert pkg.scores_to_numpy(s2, P).tobytes() == ref.tobytes()
    ok = (ref["status"] & pkg.WF_ST_INELIGIBLE) == 0
    for name, g, r in zip(("start", "finish", "load_start", "peak", "reclaimed"), sched, rs):
        a = g.cpu().numpy()
        if name == "reclaimed":
            a = a.view(np.uint64)
        a = a[:, :r.shape[1]]
        bad = np.nonzero((a[ok] != r[ok]).any(axis=1))[0]
        assert len(bad) == 0, f"{name} differs for plans {np.nonzero(ok)[0][bad[:10]].tolist()}"
    # ranking keys of the same plans
    keys = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(dev, prio, flags, P, keys)
    torch.cuda.synchronize()
    assert pkg.keys_to_numpy(keys, P).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()


@pytest.mark.parametrize("D", [65, 127])
def test_generated_candidates(ctx, D):
    """Device mutations draw among up to 127 eligible devices."""
    win, rng = window(D, 11, 12, "queue")
    plans = W.random_plans(win, 1, rng, prio_mode="perm")
    ctx.wf_plan_upload_window(win)
    inc = (plans.dev[0], plans.prio[0], plans.flags[0])
    td = torch.from_numpy(np.ascontiguousarray(plans.dev[0])).to("cuda:0")
    tp = torch.from_numpy(np.ascontiguousarray(plans.prio[0]).view(np.int16)).to("cuda:0")
    tf = torch.from_numpy(np.ascontiguousarray(plans.flags[0])).to("cuda:0")
    n = 2000
    scores = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(td, tp, tf, 77, 4, 5, n, scores)
    N = win.n_act
    od = torch.empty((n, N), dtype=torch.int8, device="cuda:0")
    op = torch.empty((n, N), dtype=torch.int16, device="cuda:0")
    of = torch.empty((n, (N + 3) // 4), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_rows(td, tp, tf, 77, 4, 5, n, od, op, of)
    torch.cuda.synchronize()
    rd, rp, rf = oracle.search_candidates(win, *inc, 77, 4, 5, n)
    assert od.cpu().numpy().tobytes() == rd.tobytes()
    assert op.cpu().numpy().view(np.uint16).tobytes() == rp.tobytes()
    assert of.cpu().numpy().tobytes() == rf.tobytes()
    assert (rd >= 64).any()  # some mutations reach the second word of the eligibility mask
    cand = W.PlanBatch(rd, rp, rf)
    assert pkg.scores_to_numpy(scores, n).tobytes() == oracle.score(win, cand, threads=THREADS).tobytes()

"""The paper's reclamation order (WF_VICTIM_PAPER) on the GPU against the
oracle: score records and schedules bytewise, ranking keys, generated
candidates."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03335_amd as pkg
from paper_2609_03335_amd import workload as W
from enumerate_plans import best_plan

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


def gpu_score(ctx, win, plans):
    ctx.wf_plan_upload_window(win)
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D)
    best = pkg.argmin(ctx, scores, P)
    torch.cuda.synchronize()
    return (pkg.scores_to_numpy(scores, P), tuple(x.cpu().numpy() for x in sched),
            int(best.item()))


def check(ctx, win, plans, where):
    got, gs, best = gpu_score(ctx, win, plans)
    ref, rs = oracle.score(win, plans, schedule=True, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), where
    ok = ref["status"] & oracle.INELIGIBLE == 0
    N = win.n_act
    for name, a, b in zip(("start", "finish", "load_start", "peak"), gs, rs):
        assert np.array_equal(a[ok][:, :b.shape[1]], b[ok]), (where, name)
    assert best == best_plan(ref)


@pytest.mark.parametrize("cfg,n", [(0, 512), (1, 1024), (2, 128), (3, 24), (4, 4096)])
def test_configs_paper_order(ctx, cfg, n, capfd, monkeypatch):
    win, plans = W.make_config(cfg, n_plans=n)
    win.victim_order = pkg._lib.WF_VICTIM_PAPER
    monkeypatch.setenv("WF_PLAN_VERBOSE", "1")
    log(f"[victim] config {cfg}: {n} plans")
    check(ctx, win, plans, f"config {cfg}")
    assert "reclaim=paper-scan" in capfd.readouterr().err


@pytest.mark.parametrize("seed", range(24))
def test_random_windows_paper_order(ctx, seed):
    rng = np.random.default_rng(95_000 + seed)
    kind = seed % 4
    if kind == 0:  # tight memory: a reclamation on most loads, several devices
        win = W.random_window(rng, n_wf=4, nodes=(2, 9), n_dev=int(rng.integers(2, 5)), n_models=6,
                              cap_range=(8000, 16000), w_range=(2000, 7000), mem_range=(0, 1500))
    elif kind == 1:  # free and costly reloads mixed (infinite and finite ratios)
        win = W.random_window(rng, n_wf=3, nodes=(3, 10), n_dev=3, n_models=5,
                              cap_range=(9000, 15000), w_range=(3000, 6000), load_range=(0, 3))
    elif kind == 2:  # more than 16 models, wide levels
        win = W.random_window(rng, n_wf=int(rng.integers(15, 40)), nodes=(2, 6), n_dev=4,
                              n_models=int(rng.integers(17, 40)), p_edge=0.3,
                              cap_range=(10000, 30000), w_range=(2000, 9000))
    else:  # fused chains
        win = W.random_window(rng, n_wf=4, nodes=(4, 12), n_dev=3, n_models=4, same_model_bias=0.8,
                              cap_range=(8000, 14000), w_range=(3000, 6000))
    win.victim_order = pkg._lib.WF_VICTIM_PAPER
    plans = W.random_plans(win, int(rng.integers(1, 250)), rng,
                           prio_mode=["any", "perm", "globalperm"][seed % 3])
    log(f"[victim] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} P={plans.n_plans}")
    check(ctx, win, plans, f"seed {seed}")


def test_worked_examples_paper_order(ctx):
    from fixtures import load_golden
    for name in ("victim_order", "victim_order_chain", "victim_order_snapshot", "victim_order_ties"):
        win, plans, ix, spec = load_golden(name)
        for order in (pkg._lib.WF_VICTIM_PAPER, pkg._lib.WF_VICTIM_REMAINING_LRU):
            win.victim_order = order
            for pname in spec["plans"]:
                check(ctx, win, plans[pname], (name, pname, order))


def test_keys_and_candidates_paper_order(ctx):
    win, plans = W.make_config(1, n_plans=512)
    win.victim_order = pkg._lib.WF_VICTIM_PAPER
    win.wf_class = (np.arange(win.n_wf) % 3).astype(np.uint8)
    ctx.wf_plan_upload_window(win)
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    keys = torch.empty((512, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(dev, prio, flags, 512, keys)
    torch.cuda.synchronize()
    assert pkg.keys_to_numpy(keys, 512).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    scores = torch.empty((600, 32), dtype=torch.uint8, device="cuda:0")
    inc = (plans.dev[3].copy(), plans.prio[3].copy(), plans.flags[3].copy())
    rows = (torch.from_numpy(inc[0]).cuda(), torch.from_numpy(inc[1].view("<i2")).cuda(),
            torch.from_numpy(inc[2]).cuda())
    ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], 17, 3, 5, 600, scores)
    torch.cuda.synchronize()
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, 17, 3, 5, 600))
    assert pkg.scores_to_numpy(scores, 600).tobytes() == oracle.score(win, cand, threads=THREADS).tobytes()

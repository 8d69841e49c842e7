"""Batch limits (several units per device at once) on the GPU against the
oracle: score records and schedules bytewise, ranking keys, generated
candidates, under both reclamation orders."""
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


def check(ctx, win, plans, where):
    ctx.wf_plan_upload_window(win)
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D)
    best = pkg.argmin(ctx, scores, P)
    torch.cuda.synchronize()
    got = pkg.scores_to_numpy(scores, P)
    ref, rs = oracle.score(win, plans, schedule=True, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), where
    ok = ref["status"] & oracle.INELIGIBLE == 0
    for name, a, b in zip(("start", "finish", "load_start", "peak"), sched, rs):
        a = a.cpu().numpy()
        assert np.array_equal(a[ok][:, :b.shape[1]], b[ok]), (where, name)
    assert int(best.item()) == best_plan(ref)


@pytest.mark.parametrize("cfg,n", [(0, 512), (1, 1024), (2, 96), (4, 4096)])
@pytest.mark.parametrize("order", [0, 1])
def test_configs_with_batch_limits(ctx, cfg, n, order, capfd, monkeypatch):
    win, plans = W.make_config(cfg, n_plans=n)
    rng = np.random.default_rng(cfg)
    win.dev_batch = rng.integers(1, pkg._lib.WF_MAX_BATCH + 1, win.n_dev).astype(np.int32)
    win.dev_batch[0] = 2
    win.victim_order = order
    monkeypatch.setenv("WF_PLAN_VERBOSE", "1")
    log(f"[batch] config {cfg}: {n} plans, order {order}, batch {list(win.dev_batch)}")
    check(ctx, win, plans, f"config {cfg}")
    want = "reclaim=batch-paper-scan" if order else "reclaim=batch-scan"
    assert want in capfd.readouterr().err


@pytest.mark.parametrize("seed", range(24))
def test_random_windows_with_batch_limits(ctx, seed):
    rng = np.random.default_rng(99_000 + seed)
    kind = seed % 4
    D = int(rng.integers(1, 5))
    if kind == 0:  # weightless models: memory of running units decides
        win = W.random_window(rng, n_wf=4, nodes=(2, 9), n_dev=D, n_models=4, w_range=(0, 0),
                              cap_range=(3000, 9000), mem_range=(500, 4000))
    elif kind == 1:  # tight weights: leases block reclamation
        win = W.random_window(rng, n_wf=5, nodes=(2, 8), n_dev=D, n_models=6,
                              cap_range=(8000, 16000), w_range=(2000, 6000), mem_range=(0, 2000))
    elif kind == 2:  # many models (scan), arrivals and busy devices
        win = W.random_window(rng, n_wf=int(rng.integers(4, 20)), nodes=(2, 6), n_dev=D,
                              n_models=int(rng.integers(10, 30)), cap_range=(10000, 30000))
    else:  # fused chains and prefetch
        win = W.random_window(rng, n_wf=4, nodes=(4, 12), n_dev=D, n_models=4, same_model_bias=0.8,
                              cap_range=(9000, 20000), w_range=(2000, 5000))
    win.dev_batch = rng.integers(1, pkg._lib.WF_MAX_BATCH + 1, D).astype(np.int32)
    if (win.dev_batch == 1).all():
        win.dev_batch[0] = 3
    win.victim_order = seed % 2
    plans = W.random_plans(win, int(rng.integers(1, 200)), rng,
                           prio_mode=["any", "perm", "globalperm"][seed % 3])
    log(f"[batch] seed {seed}: N={win.n_act} D={D} M={win.n_models} batch={list(win.dev_batch)} "
        f"P={plans.n_plans}")
    check(ctx, win, plans, f"seed {seed}")


@pytest.mark.parametrize("fit", [8, 9, 16])
def test_sixteen_models_with_batch_limits(ctx, fit):
    """Sixteen equal-weight models, capacity for exactly `fit` of them plus a
    little activation memory, batch limits 2 and 4: the resident set runs
    full and most units reclaim a copy, often with others leased by running
    units."""
    rng = np.random.default_rng(700 + fit)
    win = W.random_window(rng, n_wf=6, nodes=(6, 14), n_dev=2, n_models=16,
                          cap_range=(fit * 1000 + 600, fit * 1000 + 600), w_range=(1000, 1000),
                          mem_range=(0, 200), q_inel=0.0, same_model_bias=0.0)
    win.dev_batch = np.array([2, 4], np.int32)
    plans = W.random_plans(win, 300, rng, prio_mode="perm")
    check(ctx, win, plans, f"fit {fit}")
    if fit < 16:
        assert (oracle.score(win, plans)["n_evicts"] > 0).mean() > 0.5


def test_worked_examples_with_batch_limits(ctx):
    from fixtures import load_golden
    for name in ("batch_memory", "batch_lease"):
        win, plans, ix, spec = load_golden(name)
        for order in (0, 1):
            win.victim_order = order
            for pname in spec["plans"]:
                check(ctx, win, plans[pname], (name, pname, order))


def test_batch_of_one_changes_nothing(ctx):
    win, plans = W.make_config(1, n_plans=512)
    check(ctx, win, plans, "no limits")
    win.dev_batch = np.ones(win.n_dev, np.int32)
    check(ctx, win, plans, "all ones")


def test_keys_and_candidates_with_batch_limits(ctx):
    win, plans = W.make_config(4, n_plans=1024)
    win.dev_batch = np.array([2, 1, 3, 4, 2, 1, 1, 2], np.int32)
    win.wf_class = (np.arange(win.n_wf) % 4).astype(np.uint8)
    ctx.wf_plan_upload_window(win)
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    keys = torch.empty((1024, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(dev, prio, flags, 1024, keys)
    torch.cuda.synchronize()
    assert pkg.keys_to_numpy(keys, 1024).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    scores = torch.empty((700, 32), dtype=torch.uint8, device="cuda:0")
    inc = (plans.dev[5].copy(), plans.prio[5].copy(), plans.flags[5].copy())
    rows = (torch.from_numpy(inc[0]).cuda(), torch.from_numpy(inc[1].view("<i2")).cuda(),
            torch.from_numpy(inc[2]).cuda())
    ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], 23, 2, 0, 700, scores)
    torch.cuda.synchronize()
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, 23, 2, 0, 700))
    assert pkg.scores_to_numpy(scores, 700).tobytes() == oracle.score(win, cand, threads=THREADS).tobytes()

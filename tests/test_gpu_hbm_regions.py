"""Windows too large for LDS: each wave's per-activation arrays live in the
HBM scratch area and its per-(device, model) arrays stay in LDS.  Every
reclamation mode (4-bit queue, scan, the paper's order, batch limits) on
such a window (the scans with the ring layout switched off) against the oracle: score records, schedules, reclaimed copies,
ranking keys and generated candidates, bytewise."""
import os
import re
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


# (models, devices, victim order, batch limit, reclamation mode the host picks)
CASES = {
    "queue": (8, 3, 0, 1, "queue32"),
    "scan": (24, 3, 0, 1, "scan"),
    "paper": (24, 4, 1, 1, "paper-scan"),
    "batch": (24, 3, 0, 3, "batch-scan"),
    "batch_paper": (12, 2, 1, 2, "batch-paper-scan"),
}


def big_window(name):
    M, D, order, batch, _ = CASES[name]
    rng = np.random.default_rng(7_000 + sorted(CASES).index(name))
    win = W.random_window(rng, n_wf=400, nodes=(40, 60), n_dev=D, n_models=M, p_edge=0.1, q_inel=0.0,
                          cap_range=(16000, 40000))
    win.victim_order = order
    if batch > 1:
        win.dev_batch = np.full(D, batch, np.int32)
    assert win.n_act > 16000
    return win, W.random_plans(win, 16, rng, prio_mode="perm")


def layout_line(err):
    m = re.search(r"tables=(\S+)\(\d+ B\) wave=(\d+) B \(lds part (\d+) B\) lds/wg=(\d+) reclaim=(\S+)", err)
    assert m, err
    return m.group(1), int(m.group(2)), int(m.group(3)), int(m.group(4)), m.group(5)


@pytest.mark.parametrize("name", sorted(CASES))
def test_scores_schedules_reclaims(ctx, name, capfd, monkeypatch):
    win, plans = big_window(name)
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    log(f"[hbm] {name}: N={N} D={D} M={win.n_models} P={P}")
    monkeypatch.setenv("WF_PLAN_VERBOSE", "1")
    monkeypatch.setenv("WF_PLAN_RING", "off")  # the scan modes would take the ring layout
    ctx.wf_plan_upload_window(win)
    where, wave, lds_part, lds_wg, mode = layout_line(capfd.readouterr().err)
    assert where == "hbm+scratch" and mode == CASES[name][4], (where, mode)
    assert 0 < lds_part < wave and lds_wg >= lds_part
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D,
                                    reclaims=True)
    best = pkg.argmin(ctx, scores, P)
    torch.cuda.synchronize()
    got = pkg.scores_to_numpy(scores, P)
    ref, rs = oracle.score(win, plans, schedule=True, reclaims=True, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), name
    assert (ref["n_evicts"] > 0).any(), "the case should reclaim"
    ok = ref["status"] & oracle.INELIGIBLE == 0
    for label, a, b in zip(("start", "finish", "load_start", "peak", "reclaimed"), sched, rs):
        a = a.cpu().numpy()
        if b.dtype == np.uint64:
            a = a.view(np.uint64)
        assert np.array_equal(a[ok][:, :b.shape[1]], b[ok]), (name, label)
    assert int(best.item()) == best_plan(ref)


@pytest.mark.parametrize("name", ["scan", "batch_paper"])
def test_keys_and_candidates(ctx, name):
    win, plans = big_window(name)
    P = plans.n_plans
    log(f"[hbm] keys and candidates, {name}: N={win.n_act}")
    ctx.wf_plan_upload_window(win)
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    keys = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(dev, prio, flags, P, keys)
    torch.cuda.synchronize()
    assert pkg.keys_to_numpy(keys, P).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    inc = (plans.dev[0], plans.prio[0], plans.flags[0])
    n = 40
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, 5, 2, 3, n))
    scores = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(dev[0], prio[0], flags[0], 5, 2, 3, n, scores)
    torch.cuda.synchronize()
    assert pkg.scores_to_numpy(scores, n).tobytes() == oracle.score(win, cand, threads=THREADS).tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_random_mid_windows(ctx, seed, capfd, monkeypatch):
    """Windows of 400-3,000 activations with more than 16 models, under the
    three scanning modes: the host picks either layout by the lanes each
    keeps in flight, and both must agree with the oracle bytewise."""
    rng = np.random.default_rng(31_000 + seed)
    D = int(rng.integers(2, 17))
    win = W.random_window(rng, n_wf=int(rng.integers(20, 120)), nodes=(10, 40), n_dev=D,
                          n_models=int(rng.integers(17, 48)), p_edge=0.2, q_inel=0.0,
                          cap_range=(16000, 40000))
    mode = seed % 3
    if mode == 1:
        win.victim_order = 1
    elif mode == 2:
        win.dev_batch = rng.integers(1, 5, size=D).astype(np.int32)
    plans = W.random_plans(win, 40, rng, prio_mode="perm")
    monkeypatch.setenv("WF_PLAN_VERBOSE", "1")
    ctx.wf_plan_upload_window(win)
    where, wave, lds_part, lds_wg, rmode = layout_line(capfd.readouterr().err)
    log(f"[hbm] random {seed}: N={win.n_act} D={D} M={win.n_models} mode={rmode} layout={where}")
    P, N = plans.n_plans, win.n_act
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D)
    torch.cuda.synchronize()
    got = pkg.scores_to_numpy(scores, P)
    ref, rs = oracle.score(win, plans, schedule=True, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), seed
    ok = ref["status"] & oracle.INELIGIBLE == 0
    for label, a, b in zip(("start", "finish", "load_start", "peak"), sched, rs):
        assert np.array_equal(a.cpu().numpy()[ok][:, :b.shape[1]], b[ok]), (seed, label)


def test_two_contexts_two_streams(monkeypatch):
    """Concurrent scoring takes one context per stream: each context owns its
    scratch area, so two HBM-layout launches in flight at once both match
    the oracle."""
    monkeypatch.setenv("WF_PLAN_RING", "off")
    win, plans = big_window("scan")
    P = plans.n_plans
    ref = oracle.score(win, plans, threads=THREADS)
    log(f"[hbm] two contexts on two streams: N={win.n_act} P={P}")
    ctxs = [pkg.Context(0), pkg.Context(0)]
    try:
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        dev, prio, flags = pkg.device_plans(plans, "cuda:0")
        outs = []
        for c in ctxs:
            c.wf_plan_upload_window(win)
        torch.cuda.synchronize()
        for c, s in zip(ctxs, streams):
            sc = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
            c.wf_plan_score_batch(dev, prio, flags, P, sc, None, s)
            outs.append(sc)
        torch.cuda.synchronize()
        for sc in outs:
            assert pkg.scores_to_numpy(sc, P).tobytes() == ref.tobytes()
    finally:
        for c in ctxs:
            c.close()

"""The ring-of-recent-levels layout of the scoring kernel (deep windows in
the scan reclamation modes: the slot entries of the current level and the
finishes of the levels an edge or a fused chain still reaches, in LDS)
against the oracle, bytewise: scores, ranking keys and per-plan schedules.
Each window is also scored with the ring switched off (WF_PLAN_RING=off),
which must give the same bytes, and the layout the library took is read
from its WF_PLAN_VERBOSE report."""
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
RING_LINE = "[wf_plan] ring of recent levels"
TAKEN = []  # whether each random deep window took the ring layout


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    c = pkg.Context(0)
    yield c
    c.close()


def upload(ctx, win, capfd, ring=True):
    """Upload with or without the ring layout; returns whether it was taken."""
    os.environ["WF_PLAN_VERBOSE"] = "1"
    if ring:
        os.environ.pop("WF_PLAN_RING", None)
    else:
        os.environ["WF_PLAN_RING"] = "off"
    try:
        capfd.readouterr()
        ctx.wf_plan_upload_window(win)
        err = capfd.readouterr().err
    finally:
        os.environ.pop("WF_PLAN_VERBOSE", None)
        os.environ.pop("WF_PLAN_RING", None)
    return RING_LINE in err


def gpu_scores(ctx, plans, n):
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_batch(dev, prio, flags, n, scores)
    torch.cuda.synchronize()
    return pkg.scores_to_numpy(scores, n)


def gpu_keys(ctx, plans, n):
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    keys = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(dev, prio, flags, n, keys)
    torch.cuda.synchronize()
    return pkg.keys_to_numpy(keys, n)


def check_schedules(ctx, win, plans, n, tag):
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, n, schedule=True, n_act=win.n_act,
                                    n_dev=win.n_dev, reclaims=True)
    torch.cuda.synchronize()
    ref, rs = oracle.score(win, plans, schedule=True, threads=THREADS, reclaims=True)
    assert pkg.scores_to_numpy(scores, n).tobytes() == ref.tobytes(), tag
    ok = (ref["status"] & pkg.WF_ST_INELIGIBLE) == 0
    for name, g, r in zip(("start", "finish", "load_start", "peak", "reclaimed"), sched, rs):
        a = g.cpu().numpy()
        if name == "reclaimed":
            a = a.view(np.uint64)
        a = a[:, :r.shape[1]]
        bad = np.nonzero((a[ok] != r[ok]).any(axis=1))[0]
        assert len(bad) == 0, f"{tag}: {name} differs for plans {np.nonzero(ok)[0][bad[:10]].tolist()}"


def test_deep_workload(ctx, capfd):
    """The 4,096-activation, 128-level workload: every plan's score, a
    sample of ranking keys and schedules."""
    win, plans = W.make_config(3)
    P = plans.n_plans
    assert upload(ctx, win, capfd), "the ring layout was not taken"
    log(f"[ring] deep workload: {P} plans")
    got = gpu_scores(ctx, plans, P)
    ref = oracle.score(win, plans, threads=THREADS)
    assert got.tobytes() == ref.tobytes()
    sub = plans.take(np.arange(0, P, 16))
    assert gpu_keys(ctx, sub, sub.n_plans).tobytes() == oracle.phi_keys(win, sub, threads=THREADS).tobytes()
    check_schedules(ctx, win, plans.take(np.arange(0, P, 64)), P // 64, "deep workload")
    assert not upload(ctx, win, capfd, ring=False)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes()


def deep_case(seed):
    rng = np.random.default_rng(77_000 + seed)
    D = [4, 8, 16, 6][seed % 4]
    win = W.random_deep_window(rng, n_wf=1 + seed % 3, n_levels=(40, 90), width=(4, 14 + 3 * (seed % 3)),
                               span=1 + seed % 3, p_edge=[0.3, 0.08][seed % 2], n_dev=D,
                               n_models=[20, 24, 40][seed % 3])
    if seed % 4 == 1:
        win.dev_batch = rng.integers(1, 5, D).astype(np.int32)
    if seed % 4 == 2:
        copies = np.array([sum((int(r) >> m) & 1 for r in win.init_resident) for m in range(win.n_models)])
        win.model_replica_cap = np.maximum(copies, rng.integers(max(1, D - 2), D + 1, win.n_models)).astype(np.int32)
    mode = ["perm", "any", "globalperm", "perm"][seed % 4]
    plans = W.random_plans(win, 1500, rng, prio_mode=mode, p_bad_dev=0.02 if seed % 5 == 0 else 0.0)
    return win, plans


@pytest.mark.parametrize("seed", range(12))
def test_random_deep_windows(ctx, capfd, seed):
    """Chains written ahead of their level, edges reaching back up to three
    levels, tied and out-of-range priorities (ranked levels), batch limits,
    replica caps, invalid devices."""
    win, plans = deep_case(seed)
    P = plans.n_plans
    took = upload(ctx, win, capfd)
    log(f"[ring] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} ring={took}")
    # (long fused chains make the ring deep, and small windows fit LDS
    # whole: the host may keep another layout)
    TAKEN.append(took)
    ref = oracle.score(win, plans, threads=THREADS)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes(), f"seed {seed}"
    assert gpu_keys(ctx, plans, P).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    check_schedules(ctx, win, plans.take(np.arange(0, P, 5)), (P + 4) // 5, f"seed {seed}")
    upload(ctx, win, capfd, ring=False)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes()


def test_ring_was_exercised():
    assert len(TAKEN) == 12 and sum(TAKEN) >= 6, TAKEN


@pytest.mark.parametrize("kind", ["fp64", "checked"])
def test_ring_time_modes(ctx, capfd, kind):
    """fp64 times, and uint32 times with the fp64 rescoring pass."""
    rng = np.random.default_rng(5 if kind == "fp64" else 6)
    lat = (1, 1 << 30) if kind == "fp64" else (1 << 22, 1 << 23)
    win = W.random_deep_window(rng, n_levels=(60, 90), width=(6, 16), n_dev=8, n_models=20,
                               lat_range=lat, load_range=(0, 1 << 20))
    plans = W.random_plans(win, 2000, rng, prio_mode="perm")
    assert upload(ctx, win, capfd)
    log(f"[ring] {kind}: N={win.n_act} bits={ctx.wf_plan_time_bits()}")
    ref = oracle.score(win, plans, threads=THREADS)
    assert gpu_scores(ctx, plans, plans.n_plans).tobytes() == ref.tobytes()
    check_schedules(ctx, win, plans.take(np.arange(0, 2000, 10)), 200, kind)


def test_ring_many_devices(ctx, capfd):
    """96 devices: two per lane, one plan per wave."""
    rng = np.random.default_rng(96)
    win = W.random_deep_window(rng, n_levels=(20, 30), width=(4, 20), n_dev=96, n_models=24,
                               cap_range=(6000, 30000), w_range=(1000, 9000))
    plans = W.random_plans(win, 300, rng, prio_mode="perm")
    took = upload(ctx, win, capfd)
    log(f"[ring] 96 devices: N={win.n_act} ring={took}")
    ref = oracle.score(win, plans, threads=THREADS)
    assert gpu_scores(ctx, plans, plans.n_plans).tobytes() == ref.tobytes()
    check_schedules(ctx, win, plans, plans.n_plans, "96 devices")


SEARCH_RING_LINE = "[wf_plan] generated candidates: ring of recent levels"


def gpu_search(ctx, inc, seed, n_mut, first, n, keys=False, mode=0):
    d, p, f = (torch.from_numpy(np.ascontiguousarray(inc[0])).cuda(),
               torch.from_numpy(np.ascontiguousarray(inc[1]).view("<i2")).cuda(),
               torch.from_numpy(np.ascontiguousarray(inc[2])).cuda())
    out = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    if keys:
        ctx.wf_plan_search_keys(d, p, f, seed, n_mut, first, n, out, mode=mode)
    else:
        ctx.wf_plan_search_batch(d, p, f, seed, n_mut, first, n, out, mode=mode)
    torch.cuda.synchronize()
    return pkg.keys_to_numpy(out, n) if keys else pkg.scores_to_numpy(out, n)


def upload_search(ctx, win, capfd, ring=True):
    """Upload; returns whether generated candidates took the ring layout."""
    os.environ["WF_PLAN_VERBOSE"] = "1"
    if ring:
        os.environ.pop("WF_PLAN_RING", None)
    else:
        os.environ["WF_PLAN_RING"] = "off"
    try:
        capfd.readouterr()
        ctx.wf_plan_upload_window(win)
        err = capfd.readouterr().err
    finally:
        os.environ.pop("WF_PLAN_VERBOSE", None)
        os.environ.pop("WF_PLAN_RING", None)
    return SEARCH_RING_LINE in err


@pytest.mark.parametrize("n_mut", [1, 8, 9])
def test_generated_candidates_deep_workload(ctx, capfd, n_mut):
    """Candidates around a plan of the deep workload: kept as the incumbent
    plus their changed sites in the ring layout (at most 8 mutations), or as
    whole rows in the layout without the ring (more mutations), against the
    oracle's candidates scored by the oracle."""
    win, plans = W.make_config(3, n_plans=2)
    inc = (plans.dev[0], plans.prio[0], plans.flags[0])
    took = upload_search(ctx, win, capfd)
    assert took, "generated candidates did not take the ring layout"
    n, seed, first = 1024, 0xC0FFEE + n_mut, 5 * n_mut
    log(f"[ring search] deep workload: {n} candidates, {n_mut} mutations")
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, seed, n_mut, first, n))
    ref = oracle.score(win, cand, threads=THREADS)
    assert gpu_search(ctx, inc, seed, n_mut, first, n).tobytes() == ref.tobytes()
    if n_mut == 8:
        rk = oracle.phi_keys(win, cand, threads=THREADS)
        assert gpu_search(ctx, inc, seed, n_mut, first, n, keys=True).tobytes() == rk.tobytes()
        cr = W.PlanBatch(*oracle.search_candidates(win, *inc, seed, n_mut, first, n,
                                                   mode=oracle.SEARCH_RULES))
        rr = oracle.score(win, cr, threads=THREADS)
        assert gpu_search(ctx, inc, seed, n_mut, first, n, mode=pkg.WF_SEARCH_RULES).tobytes() == rr.tobytes()
    assert not upload_search(ctx, win, capfd, ring=False)
    assert gpu_search(ctx, inc, seed, n_mut, first, n).tobytes() == ref.tobytes()


@pytest.mark.parametrize("seed", range(8))
def test_generated_candidates_random_deep_windows(ctx, capfd, seed):
    """Candidates around a plan of random deep windows (ranked levels, batch
    limits, replica caps, invalid incumbent devices), with and without the
    ring, at mutation counts on both sides of the changed-site limit."""
    win, plans = deep_case(seed)
    inc = (plans.dev[1], plans.prio[1], plans.flags[1])
    took = upload_search(ctx, win, capfd)
    n_mut = [0, 2, 5, 8, 9, 16, 3, 8][seed]
    n, s64, first = 600, 0x9E3779B97F4A7C15 ^ seed, 1000 * seed
    log(f"[ring search] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} ring={took} "
        f"n_mut={n_mut}")
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, s64, n_mut, first, n))
    ref = oracle.score(win, cand, threads=THREADS)
    assert gpu_search(ctx, inc, s64, n_mut, first, n).tobytes() == ref.tobytes(), f"seed {seed}"
    rk = oracle.phi_keys(win, cand, threads=THREADS)
    assert gpu_search(ctx, inc, s64, n_mut, first, n, keys=True).tobytes() == rk.tobytes()
    upload_search(ctx, win, capfd, ring=False)
    assert gpu_search(ctx, inc, s64, n_mut, first, n).tobytes() == ref.tobytes()


FIN_RING_LINE = "[wf_plan] finishes in a ring of recent levels"
PAPER_TAKEN = []  # whether each random deep window's finishes took the ring


def upload_paper(ctx, win, capfd, ring=True):
    """Upload; returns whether the finishes took the ring (the paper's order
    with the order and slot arrays in HBM)."""
    os.environ["WF_PLAN_VERBOSE"] = "1"
    if ring:
        os.environ.pop("WF_PLAN_RING", None)
    else:
        os.environ["WF_PLAN_RING"] = "off"
    try:
        capfd.readouterr()
        ctx.wf_plan_upload_window(win)
        err = capfd.readouterr().err
    finally:
        os.environ.pop("WF_PLAN_VERBOSE", None)
        os.environ.pop("WF_PLAN_RING", None)
    return FIN_RING_LINE in err


@pytest.mark.parametrize("batch", [False, True])
def test_paper_order_deep_workload(ctx, capfd, batch):
    """The paper's reclamation order on the deep workload: the order and the
    next use per slot built before the walk in HBM, the finishes in the ring,
    against the oracle (scores, keys, schedules) and the layout without the
    ring."""
    win, plans = W.make_config(3)
    win.victim_order = 1
    if batch:
        win.dev_batch = np.array([1, 2, 3, 4] * 4, np.int32)
        plans = plans.take(np.arange(0, plans.n_plans, 4))
    P = plans.n_plans
    assert upload_paper(ctx, win, capfd), "the finishes did not take the ring"
    log(f"[ring paper] deep workload: {P} plans, batch limits {batch}")
    ref = oracle.score(win, plans, threads=THREADS)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes()
    sub = plans.take(np.arange(0, P, 16))
    assert gpu_keys(ctx, sub, sub.n_plans).tobytes() == oracle.phi_keys(win, sub, threads=THREADS).tobytes()
    check_schedules(ctx, win, plans.take(np.arange(0, P, 64)), (P + 63) // 64, "paper deep workload")
    assert not upload_paper(ctx, win, capfd, ring=False)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes()


@pytest.mark.parametrize("seed", range(8))
def test_paper_order_random_deep_windows(ctx, capfd, seed):
    """Random deep windows under the paper's order (chains ahead of their
    level, edges up to three levels back, ranked levels, batch limits,
    invalid devices): scores, keys and schedules against the oracle, with
    and without the ring."""
    win, plans = deep_case(seed)
    win.victim_order = 1
    P = plans.n_plans
    took = upload_paper(ctx, win, capfd)
    PAPER_TAKEN.append(took)
    log(f"[ring paper] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} fin ring={took}")
    ref = oracle.score(win, plans, threads=THREADS)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes(), f"seed {seed}"
    assert gpu_keys(ctx, plans, P).tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    check_schedules(ctx, win, plans.take(np.arange(0, P, 5)), (P + 4) // 5, f"paper seed {seed}")
    upload_paper(ctx, win, capfd, ring=False)
    assert gpu_scores(ctx, plans, P).tobytes() == ref.tobytes()


def test_paper_ring_was_exercised():
    """Some of the random deep windows above kept their finishes in the ring
    (the others fit the LDS layout or none of the HBM one's conditions)."""
    assert len(PAPER_TAKEN) == 8 and sum(PAPER_TAKEN) >= 2, PAPER_TAKEN

"""Rule-guided candidates on the GPU (mode WF_SEARCH_RULES of
wf_plan_search_batch, wf_plan_search_rows, wf_plan_search_keys: Algorithm 1's
BestFeasibleBinding and PlanPrefetch, Sec. 3.5) against the oracle's
generator, scorer and ranking keys, element by element, on every workload
configuration and on random windows."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03335_amd as pkg
from paper_2609_03335_amd import workload as W
from enumerate_plans import best_plan
from test_gpu_many_devices import window as many_device_window

pytestmark = pytest.mark.gpu
THREADS = max(1, min(16, os.cpu_count() or 1))
RULES = pkg.WF_SEARCH_RULES


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    c = pkg.Context(0)
    yield c
    c.close()


def rows_on_gpu(d, p, f):
    return (torch.from_numpy(np.ascontiguousarray(d)).cuda(),
            torch.from_numpy(np.ascontiguousarray(p).view("<i2")).cuda(),
            torch.from_numpy(np.ascontiguousarray(f)).cuda())


def with_slack(win, rng):
    """A dispatch slack of the order of the window's load times, so that
    PlanPrefetch both sets and clears bits."""
    load = np.asarray(win.load_us)
    win.prefetch_slack_us = int(rng.integers(0, 2 * int(np.median(load)) + 2))
    return win


def gpu_rows(ctx, win, inc, seed, n_mut, first, n):
    ctx.wf_plan_upload_window(win)
    rows = rows_on_gpu(*inc)
    N, nb = win.n_act, (win.n_act + 3) // 4
    od = torch.empty((n, N), dtype=torch.int8, device="cuda:0")
    op = torch.empty((n, N), dtype=torch.int16, device="cuda:0")
    of = torch.empty((n, nb), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_rows(rows[0], rows[1], rows[2], seed, n_mut, first, n, od, op, of, mode=RULES)
    torch.cuda.synchronize()
    return od.cpu().numpy(), op.cpu().numpy().view("<u2"), of.cpu().numpy()


def gpu_scores(ctx, win, inc, seed, n_mut, first, n):
    ctx.wf_plan_upload_window(win)
    rows = rows_on_gpu(*inc)
    scores = torch.empty((max(n, 1), 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], seed, n_mut, first, n, scores, mode=RULES)
    best = torch.empty(1, dtype=torch.int64, device="cuda:0")
    ctx.wf_plan_argmin(scores, n, best)
    torch.cuda.synchronize()
    return pkg.scores_to_numpy(scores, n), int(best.item())


def check_rows(ctx, win, inc, seed, n_mut, first, n):
    gd, gp, gf = gpu_rows(ctx, win, inc, seed, n_mut, first, n)
    cd, cp, cf = oracle.search_candidates(win, *inc, seed, n_mut, first, n, mode=oracle.SEARCH_RULES)
    assert gd.tobytes() == cd.tobytes()
    assert gp.tobytes() == cp.tobytes()
    assert gf.tobytes() == cf.tobytes()
    return cd, cp, cf


@pytest.mark.parametrize("cfg", range(5))
def test_rule_rows_match_oracle(ctx, cfg):
    win, plans = W.make_config(cfg, n_plans=4)
    with_slack(win, np.random.default_rng(cfg))
    inc = (plans.dev[2].copy(), plans.prio[2].copy(), plans.flags[2].copy())
    log(f"[rules rows] config {cfg}: N={win.n_act} D={win.n_dev} slack={win.prefetch_slack_us}")
    cd, _, cf = check_rows(ctx, win, inc, 0xFEED + cfg, 6, 1000 * cfg, 256)
    # the rules changed something: devices moved and prefetch bits both set and cleared
    assert (cd != inc[0]).any()
    _, pf = W.unpack_flags(cf, win.n_act)
    _, pf0 = W.unpack_flags(inc[2][None, :], win.n_act)
    assert (pf & ~pf0).any() or (~pf & pf0).any()


@pytest.mark.parametrize("cfg,n,n_mut", [(0, 512, 2), (1, 2048, 3), (2, 256, 4), (3, 128, 2),
                                         (4, 8192, 2)])
def test_rule_scores_match_oracle(ctx, cfg, n, n_mut):
    win, plans = W.make_config(cfg, n_plans=4)
    with_slack(win, np.random.default_rng(10 + cfg))
    inc = (plans.dev[cfg % 4].copy(), plans.prio[cfg % 4].copy(), plans.flags[cfg % 4].copy())
    seed, first = 0x5151 ^ cfg, 777 * cfg
    log(f"[rules scores] config {cfg}: {n} candidates, {n_mut} mutations")
    got, best = gpu_scores(ctx, win, inc, seed, n_mut, first, n)
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, seed, n_mut, first, n,
                                                 mode=oracle.SEARCH_RULES))
    ref = oracle.score(win, cand, threads=THREADS)
    assert got.tobytes() == ref.tobytes()
    assert best == best_plan(ref)


@pytest.mark.parametrize("cfg,n,n_mut", [(1, 1024, 3), (4, 2048, 2)])
def test_rule_keys_match_oracle(ctx, cfg, n, n_mut):
    win, plans = W.make_config(cfg, n_plans=2)
    with_slack(win, np.random.default_rng(20 + cfg))
    ctx.wf_plan_upload_window(win)
    inc = (plans.dev[1].copy(), plans.prio[1].copy(), plans.flags[1].copy())
    rows = rows_on_gpu(*inc)
    keys = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_keys(rows[0], rows[1], rows[2], 31, n_mut, 5, n, keys, mode=RULES)
    torch.cuda.synchronize()
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, 31, n_mut, 5, n, mode=oracle.SEARCH_RULES))
    ref = oracle.phi_keys(win, cand, threads=THREADS)
    assert pkg.keys_to_numpy(keys, n).tobytes() == ref.tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_rule_random_windows(ctx, seed):
    """Free loads, resident replicas, late arrivals, invalid incumbent
    devices and odd N."""
    rng = np.random.default_rng(52_000 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 6)), nodes=(1, 12),
                          n_dev=int(rng.integers(1, 7)), n_models=int(rng.integers(1, 7)))
    load = np.asarray(win.load_us).copy()
    load[rng.random(load.size) < 0.15] = 0
    win.load_us = load.astype(np.int32)
    win.prefetch_slack_us = int(rng.integers(0, 3000))
    plans = W.random_plans(win, 1, rng, prio_mode="perm", p_bad_dev=0.1 if seed % 3 == 0 else 0.0)
    inc = (plans.dev[0].copy(), plans.prio[0].copy(), plans.flags[0].copy())
    n_mut, n = int(rng.integers(0, 10)), 500
    s64 = int(rng.integers(0, 1 << 62))
    log(f"[rules random] seed {seed}: N={win.n_act} D={win.n_dev} n_mut={n_mut}")
    check_rows(ctx, win, inc, s64, n_mut, 0, n)
    got, best = gpu_scores(ctx, win, inc, s64, n_mut, 0, n)
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, s64, n_mut, 0, n, mode=oracle.SEARCH_RULES))
    ref = oracle.score(win, cand, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), f"seed {seed}"
    assert best == best_plan(ref)


@pytest.mark.parametrize("D", [96, 127])
def test_rule_many_devices(ctx, D):
    """Best bindings and prefetch masks above device 63."""
    win, rng = many_device_window(D, 21, 12, "queue")
    with_slack(win, rng)
    plans = W.random_plans(win, 1, rng, prio_mode="perm")
    inc = (plans.dev[0].copy(), plans.prio[0].copy(), plans.flags[0].copy())
    log(f"[rules many devices] D={D} N={win.n_act}")
    cd, _, _ = check_rows(ctx, win, inc, 4242, 5, 0, 1500)
    got, _ = gpu_scores(ctx, win, inc, 4242, 5, 0, 1500)
    ref = oracle.score(win, W.PlanBatch(*oracle.search_candidates(
        win, *inc, 4242, 5, 0, 1500, mode=oracle.SEARCH_RULES)), threads=THREADS)
    assert got.tobytes() == ref.tobytes()


def test_rule_mode_errors_and_zero_mutations(ctx):
    win, plans = W.make_config(0, n_plans=1)
    win.prefetch_slack_us = 100
    ctx.wf_plan_upload_window(win)
    inc = (plans.dev[0], plans.prio[0], plans.flags[0])
    rows = rows_on_gpu(*inc)
    scores = torch.zeros((8, 32), dtype=torch.uint8, device="cuda:0")
    for bad in (-1, 2, 7):
        with pytest.raises(pkg.WFError) as e:
            ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], 1, 1, 0, 8, scores, mode=bad)
        assert e.value.status == pkg.WF_EINVAL
    got, _ = gpu_scores(ctx, win, inc, 9, 0, 0, 8)
    assert got.tobytes() == np.repeat(oracle.score(win, plans), 8).tobytes()

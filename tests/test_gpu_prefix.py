"""The reclaimed copies of the schedule output and the prefix commit of
Algorithm 1 (wf_plan_prefix) on the GPU against the oracle, bytewise; the
hand-derived example of tests/golden/prefix_commit.json."""
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


def gpu_schedule(ctx, win, plans):
    ctx.wf_plan_upload_window(win)
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores, sched = pkg.score_batch(ctx, dev, prio, flags, P, schedule=True, n_act=N, n_dev=D,
                                    reclaims=True)
    return dev, scores, sched


def check(ctx, win, plans, where, n_prefix=8):
    dev, scores, sched = gpu_schedule(ctx, win, plans)
    torch.cuda.synchronize()
    P, N = plans.n_plans, win.n_act
    got = pkg.scores_to_numpy(scores, P)
    ref, rs = oracle.score(win, plans, schedule=True, reclaims=True, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), where
    ok = ref["status"] & oracle.INELIGIBLE == 0
    for name, a, b in zip(("start", "finish", "load_start", "peak", "reclaimed"), sched, rs):
        a = a.cpu().numpy()
        if name == "reclaimed":
            a = a.view(np.uint64)
        assert np.array_equal(a[ok][:, :b.shape[1]], b[ok]), (where, name)
    # the prefix of a few feasible plans, each from its own rows of the batch
    commit = torch.empty(max(N, 1), dtype=torch.uint8, device="cuda:0")
    crec = torch.empty(max(N, 1), dtype=torch.int64, device="cuda:0")
    t_next = torch.empty(1, dtype=torch.int64, device="cuda:0")
    for p in np.nonzero(ok)[0][:n_prefix]:
        ctx.wf_plan_prefix(dev[p], sched[0][p], sched[1][p], sched[2][p], sched[4][p],
                           commit, crec, t_next)
        torch.cuda.synchronize()
        c, cr, t = oracle.prefix(win, plans.dev[p], rs[0][p], rs[1][p], rs[2][p], rs[4][p])
        assert int(t_next.item()) == t, (where, p)
        assert np.array_equal(commit.cpu().numpy()[:N], c), (where, p)
        assert np.array_equal(crec.cpu().numpy()[:N].view(np.uint64), cr), (where, p)


def test_worked_example(ctx):
    from fixtures import load_golden
    win, plans, ix, spec = load_golden("prefix_commit")
    models = [m["name"] for m in spec["models"]]
    for pname, pre in spec["expect_prefix"].items():
        check(ctx, win, plans[pname], pname, n_prefix=1)
        dev, scores, sched = gpu_schedule(ctx, win, plans[pname])
        N = win.n_act
        commit = torch.empty(N, dtype=torch.uint8, device="cuda:0")
        crec = torch.empty(N, dtype=torch.int64, device="cuda:0")
        t_next = torch.empty(1, dtype=torch.int64, device="cuda:0")
        ctx.wf_plan_prefix(dev[0], sched[0][0], sched[1][0], sched[2][0], sched[4][0], commit, crec,
                           t_next)
        torch.cuda.synchronize()
        assert int(t_next.item()) == pre["t_next"], pname
        c = commit.cpu().numpy()
        r = crec.cpu().numpy().view(np.uint64)
        for n, i in ix.items():
            assert bool(c[i] & 1) == (n in pre["grant"]), (pname, n)
            assert bool(c[i] & 2) == (n in pre["load"]), (pname, n)
            assert int(r[i]) == sum(1 << models.index(m) for m in pre["reclaimed"].get(n, [])), (pname, n)


@pytest.mark.parametrize("cfg,n", [(0, 256), (1, 256), (2, 64), (4, 1024)])
def test_configs(ctx, cfg, n):
    win, plans = W.make_config(cfg, n_plans=n)
    log(f"[prefix] config {cfg}: {n} plans")
    check(ctx, win, plans, f"config {cfg}")


@pytest.mark.parametrize("seed", range(18))
def test_random_windows(ctx, seed):
    rng = np.random.default_rng(63_000 + seed)
    D = int(rng.integers(1, 5))
    win = W.random_window(rng, n_wf=int(rng.integers(1, 6)), nodes=(2, 9), n_dev=D,
                          n_models=int(rng.integers(2, 20)), cap_range=(8000, 20000),
                          w_range=(2000, 7000))
    if seed % 3 == 1:
        win.victim_order = 1
    if seed % 3 == 2:
        win.dev_batch = rng.integers(1, 5, D).astype(np.int32)
    plans = W.random_plans(win, int(rng.integers(1, 120)), rng,
                           prio_mode=["any", "perm", "globalperm"][seed % 3])
    log(f"[prefix] seed {seed}: N={win.n_act} D={D} M={win.n_models} P={plans.n_plans}")
    check(ctx, win, plans, f"seed {seed}")


def test_prefix_arguments(ctx):
    win, plans = W.make_config(0, n_plans=4)
    dev, scores, sched = gpu_schedule(ctx, win, plans)
    N = win.n_act
    commit = torch.empty(N, dtype=torch.uint8, device="cuda:0")
    crec = torch.empty(N, dtype=torch.int64, device="cuda:0")
    with pytest.raises(pkg.WFError) as e:
        ctx.wf_plan_prefix(dev[0], sched[0][0], sched[1][0], sched[2][0], sched[4][0], commit, crec, None)
    assert e.value.status == pkg.WF_EINVAL
    t_next = torch.empty(1, dtype=torch.int64, device="cuda:0")
    with pytest.raises(pkg.WFError) as e:
        ctx.wf_plan_prefix(dev[0], sched[0][0], None, sched[2][0], sched[4][0], commit, crec, t_next)
    assert e.value.status == pkg.WF_EINVAL
    c2 = pkg.Context(0)
    try:
        with pytest.raises(pkg.WFError) as e:
            c2.wf_plan_prefix(dev[0], sched[0][0], sched[1][0], sched[2][0], sched[4][0], commit, crec,
                              t_next)
        assert e.value.status == pkg.WF_ENOWINDOW
    finally:
        c2.close()


def test_empty_window(ctx):
    """No activations: only the next event is written (none: INT64_MAX), and
    the plan and schedule arrays may be NULL."""
    win = W.Window(n_act=0, n_wf=0, n_models=2, n_dev=3, act_wf=np.zeros(0, np.int32),
                   act_model=np.zeros(0, np.int32), pred_off=np.zeros(1, np.int32),
                   pred_idx=np.zeros(0, np.int32), lat_us=np.zeros(0, np.int32),
                   mem_mib=np.zeros(0, np.int32), wf_arrival_us=np.zeros(0, np.int64),
                   dev_cap_mib=np.array([100, 50, 70], np.int32), model_mib=np.array([30, 20], np.int32),
                   load_us=np.zeros(6, np.int32), init_resident=np.array([3, 0, 2], np.uint64),
                   dev_free0_us=np.zeros(3, np.int64))
    ctx.wf_plan_upload_window(win)
    t_next = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    ctx.wf_plan_prefix(None, None, None, None, None, None, None, t_next)
    torch.cuda.synchronize()
    c, cr, t = oracle.prefix(win, np.zeros(0, np.int8), np.zeros(0, np.int64), np.zeros(0, np.int64),
                             np.zeros(0, np.int64), np.zeros(0, np.uint64))
    assert int(t_next.item()) == t == np.iinfo(np.int64).max

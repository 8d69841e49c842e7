"""The lean scoring kernel (lean.hip) against the oracle and against the
general kernel on the same plans: which windows it serves, and bytewise
equal records on the workloads it serves and on random windows that stress
its paths (tied and out-of-range priorities, invalid devices, fused chains,
initial residency, busy devices, tight memory, saturating uint32 times)."""
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


def score(win, plans, general=False):
    """Records of every plan, and the kernel that scored them."""
    old = os.environ.get("WF_PLAN_KERNEL")
    if general:
        os.environ["WF_PLAN_KERNEL"] = "general"
    try:
        with pkg.Context(0) as ctx:
            ctx.wf_plan_upload_window(win)
            kern = (ctx.wf_plan_score_kernel(), ctx.wf_plan_time_bits())
            P = plans.n_plans
            dev, prio, flags = pkg.device_plans(plans, "cuda:0")
            s = pkg.score_batch(ctx, dev, prio, flags, P)
            torch.cuda.synchronize()
            return pkg.scores_to_numpy(s, P), kern
    finally:
        if general:
            if old is None:
                del os.environ["WF_PLAN_KERNEL"]
            else:
                os.environ["WF_PLAN_KERNEL"] = old


@pytest.mark.parametrize("cfg,n", [(0, 512), (1, 16384), (4, 65536)])
def test_workloads_served_by_the_lean_kernel(cfg, n):
    win, plans = W.make_config(cfg, n_plans=n)
    log(f"[lean] config {cfg}: {n} plans")
    got, kern = score(win, plans)
    assert kern[0] == "score_lean"
    gen, kern_g = score(win, plans, general=True)
    assert kern_g[0] == "score_plans"
    assert got.tobytes() == gen.tobytes()
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()


@pytest.mark.parametrize("cfg", [2, 3])
def test_workloads_outside_the_lean_kernel(cfg):
    win, _ = W.make_config(cfg, n_plans=1)
    with pkg.Context(0) as ctx:
        ctx.wf_plan_upload_window(win)
        assert ctx.wf_plan_score_kernel() == "score_plans"


@pytest.mark.parametrize("seed", range(24))
def test_random_windows(seed):
    rng = np.random.default_rng(9000 + seed)
    kw = dict(n_wf=int(rng.integers(1, 7)), nodes=(1, 12), n_dev=int(rng.integers(1, 13)),
              n_models=int(rng.integers(1, 17)), same_model_bias=0.6)
    if seed % 4 == 1:  # tight memory: frequent reclamation and CAPACITY plans
        kw.update(cap_range=(3000, 12000), w_range=(1000, 9000))
    if seed % 4 == 2:  # long loads and run times: uint32 times checked, some saturate
        kw.update(lat_range=(1, 1 << 29), load_range=(0, 1 << 30))
    win = W.random_window(rng, **kw)
    mode = ("any", "perm", "globalperm")[seed % 3]
    plans = W.random_plans(win, 700, rng, p_bad_dev=0.02 if seed % 5 == 0 else 0.0,
                           prio_mode=mode)
    got, kern = score(win, plans)
    ref = oracle.score(win, plans, threads=THREADS)
    log(f"[lean] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} kernel={kern}")
    if win.n_act <= 512 and win.n_models <= 16 and kern[1] == 32:
        assert kern[0] == "score_lean"
    assert got.tobytes() == ref.tobytes()
    gen, _ = score(win, plans, general=True)
    assert got.tobytes() == gen.tobytes()


def keys(win, plans, general=False):
    old = os.environ.get("WF_PLAN_KERNEL")
    if general:
        os.environ["WF_PLAN_KERNEL"] = "general"
    try:
        with pkg.Context(0) as ctx:
            ctx.wf_plan_upload_window(win)
            P = plans.n_plans
            dev, prio, flags = pkg.device_plans(plans, "cuda:0")
            out = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
            ctx.wf_plan_score_keys(dev, prio, flags, P, out)
            torch.cuda.synchronize()
            return pkg.keys_to_numpy(out, P), ctx.wf_plan_score_kernel()
    finally:
        if general:
            if old is None:
                del os.environ["WF_PLAN_KERNEL"]
            else:
                os.environ["WF_PLAN_KERNEL"] = old


@pytest.mark.parametrize("cfg,n", [(1, 16384), (4, 65536)])
def test_ranking_keys_of_the_lean_kernel(cfg, n):
    """Eq. 12 keys from the lean kernel's key mode, with priority classes."""
    win, plans = W.make_config(cfg, n_plans=n)
    win.wf_class = (np.arange(win.n_wf) % 4).astype(np.uint8)
    log(f"[lean keys] config {cfg}: {n} plans")
    got, kern = keys(win, plans)
    assert kern == "score_lean"
    assert got.tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    gen, _ = keys(win, plans, general=True)
    assert got.tobytes() == gen.tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_ranking_keys_random_windows(seed):
    rng = np.random.default_rng(19_000 + seed)
    kw = dict(n_wf=int(rng.integers(1, 7)), nodes=(1, 12), n_dev=int(rng.integers(1, 13)),
              n_models=int(rng.integers(1, 17)), same_model_bias=0.6)
    if seed % 3 == 1:
        kw.update(cap_range=(3000, 12000), w_range=(1000, 9000))
    if seed % 3 == 2:
        kw.update(lat_range=(1, 1 << 29), load_range=(0, 1 << 30))
    win = W.random_window(rng, **kw)
    win.wf_class = rng.integers(0, 4, win.n_wf).astype(np.uint8)
    # half the workflows arrive at time 0 (ready work)
    win.wf_arrival_us = np.where(rng.random(win.n_wf) < 0.5, 0, win.wf_arrival_us).astype(np.int64)
    plans = W.random_plans(win, 600, rng, prio_mode=("any", "perm", "globalperm")[seed % 3],
                           p_bad_dev=0.02 if seed % 4 == 0 else 0.0)
    got, kern = keys(win, plans)
    log(f"[lean keys] seed {seed}: N={win.n_act} M={win.n_models} kernel={kern}")
    assert got.tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()


@pytest.mark.parametrize("cfg,n,limit", [(0, 512, 2), (1, 16384, 4), (4, 65536, 2), (4, 8192, 3)])
def test_batch_limits_in_the_lean_kernel(cfg, n, limit):
    """Devices with batch limits (several units at once, memory checked
    against the running units, leases on their models): the lean kernel's
    batch mode against the oracle and the general kernel."""
    win, plans = W.make_config(cfg, n_plans=n)
    win.dev_batch = np.full(win.n_dev, limit, np.int32)
    win.dev_batch[0] = 1
    log(f"[lean batch] config {cfg}: {n} plans, limit {limit}")
    got, kern = score(win, plans)
    assert kern[0] == "score_lean"
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()
    gen, kern_g = score(win, plans, general=True)
    assert kern_g[0] == "score_plans"
    assert got.tobytes() == gen.tobytes()


@pytest.mark.parametrize("seed", range(24))
def test_batch_limits_random_windows(seed):
    rng = np.random.default_rng(29_000 + seed)
    kind = seed % 4
    D = int(rng.integers(1, 9))
    if kind == 0:  # weightless models: the running units' memory decides
        win = W.random_window(rng, n_wf=4, nodes=(2, 9), n_dev=D, n_models=4, w_range=(0, 0),
                              cap_range=(3000, 9000), mem_range=(500, 4000))
    elif kind == 1:  # tight weights: leases hold copies back from reclamation
        win = W.random_window(rng, n_wf=5, nodes=(2, 10), n_dev=D, n_models=int(rng.integers(4, 17)),
                              cap_range=(8000, 16000), w_range=(2000, 6000), mem_range=(0, 2000))
    elif kind == 2:  # long run and load times: uint32 times checked, some saturate
        win = W.random_window(rng, n_wf=int(rng.integers(2, 8)), nodes=(2, 10), n_dev=D,
                              n_models=int(rng.integers(2, 17)), lat_range=(1, 1 << 29),
                              load_range=(0, 1 << 30))
    else:  # fused chains, prefetch, busy devices
        win = W.random_window(rng, n_wf=4, nodes=(4, 12), n_dev=D, n_models=6, same_model_bias=0.8,
                              cap_range=(9000, 20000), w_range=(2000, 5000))
    win.dev_batch = rng.integers(1, pkg._lib.WF_MAX_BATCH + 1, D).astype(np.int32)
    if (win.dev_batch == 1).all():
        win.dev_batch[0] = 2
    plans = W.random_plans(win, int(rng.integers(64, 700)), rng,
                           prio_mode=("any", "perm", "globalperm")[seed % 3],
                           p_bad_dev=0.02 if seed % 5 == 0 else 0.0)
    got, kern = score(win, plans)
    log(f"[lean batch] seed {seed}: N={win.n_act} D={D} M={win.n_models} "
        f"batch={list(win.dev_batch)} kernel={kern}")
    if win.n_act <= 512 and kern[1] == 32:
        assert kern[0] == "score_lean"
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()
    gen, _ = score(win, plans, general=True)
    assert got.tobytes() == gen.tobytes()


def test_batch_limits_keys_and_replica_caps():
    """With batch limits the lean kernel scores plans only: ranking keys come
    from the general kernel, and so does everything once replicas are capped
    as well."""
    win, plans = W.make_config(1, n_plans=2048)
    win.dev_batch = np.full(win.n_dev, 2, np.int32)
    win.wf_class = (np.arange(win.n_wf) % 4).astype(np.uint8)
    got, kern = keys(win, plans)
    assert kern == "score_lean"
    assert got.tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()
    win.model_replica_cap = np.full(win.n_models, win.n_dev, np.int32)
    got, kern = score(win, plans)
    assert kern[0] == "score_plans"
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()


@pytest.mark.parametrize("cfg,n", [(0, 512), (1, 16384), (4, 65536)])
def test_paper_order_in_the_lean_kernel(cfg, n):
    """The paper's reclamation order (copies held on another device as the
    level starts, then next-use distance per reload time, then recency) in
    the lean kernel against the oracle and the general kernel."""
    win, plans = W.make_config(cfg, n_plans=n)
    win.victim_order = 1
    log(f"[lean paper] config {cfg}: {n} plans")
    got, kern = score(win, plans)
    assert kern[0] == "score_lean"
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()
    gen, kern_g = score(win, plans, general=True)
    assert kern_g[0] == "score_plans"
    assert got.tobytes() == gen.tobytes()


@pytest.mark.parametrize("seed", range(24))
def test_paper_order_random_windows(seed):
    rng = np.random.default_rng(39_000 + seed)
    kw = dict(n_wf=int(rng.integers(1, 7)), nodes=(1, 12), n_dev=int(rng.integers(1, 13)),
              n_models=int(rng.integers(1, 17)), same_model_bias=0.6)
    if seed % 4 == 1:  # tight memory: frequent reclamation among several copies
        kw.update(cap_range=(3000, 12000), w_range=(1000, 9000))
    if seed % 4 == 2:  # long loads and run times: uint32 times checked, some saturate
        kw.update(lat_range=(1, 1 << 29), load_range=(0, 1 << 30))
    if seed % 4 == 3:  # free reloads (infinite ratios) next to costly ones
        kw.update(load_range=(0, 3), cap_range=(4000, 14000), w_range=(1000, 6000))
    win = W.random_window(rng, **kw)
    win.victim_order = 1
    plans = W.random_plans(win, int(rng.integers(64, 700)), rng,
                           prio_mode=("any", "perm", "globalperm")[seed % 3],
                           p_bad_dev=0.02 if seed % 5 == 0 else 0.0)
    got, kern = score(win, plans)
    log(f"[lean paper] seed {seed}: N={win.n_act} D={win.n_dev} M={win.n_models} kernel={kern}")
    if win.n_act <= 512 and kern[1] == 32:
        assert kern[0] == "score_lean"
    assert got.tobytes() == oracle.score(win, plans, threads=THREADS).tobytes()
    gen, _ = score(win, plans, general=True)
    assert got.tobytes() == gen.tobytes()


def test_paper_order_keys_stay_general():
    """With the paper's order the lean kernel scores plans only: ranking keys
    come from the general kernel."""
    win, plans = W.make_config(1, n_plans=2048)
    win.victim_order = 1
    win.wf_class = (np.arange(win.n_wf) % 4).astype(np.uint8)
    got, kern = keys(win, plans)
    assert kern == "score_lean"
    assert got.tobytes() == oracle.phi_keys(win, plans, threads=THREADS).tobytes()


@pytest.mark.parametrize("n_act", [256, 320])
def test_paper_order_one_device_many_units(n_act):
    """Every unit of most plans on device 0 of eight: next-use indices up to
    n_act - 1 (one-byte entries up to 256 activations, two-byte entries
    beyond)."""
    rng = np.random.default_rng(41_000 + n_act)
    win = W.random_window(rng, n_wf=n_act // 16, nodes=(16, 16), n_dev=8, n_models=5,
                          cap_range=(6000, 9000), w_range=(1000, 4000), mem_range=(0, 1000),
                          q_inel=0.0, same_model_bias=0.2)
    assert win.n_act == n_act
    win.victim_order = 1
    plans = W.random_plans(win, 128, rng, prio_mode="perm")
    plans.dev[:120] = 0
    got, kern = score(win, plans)
    assert kern[0] == "score_lean"
    ref = oracle.score(win, plans, threads=THREADS)
    assert got.tobytes() == ref.tobytes()
    assert (ref["n_evicts"][:120] > 0).all()

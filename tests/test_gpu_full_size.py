"""Every scoring mode at the throughput workload's full size (256
activations, 1,048,576 plans) in the launch configuration the benchmark
times, every record against the oracle: the paper's reclamation order,
batch limits, the ranking keys of Eq. 12, and generated candidates."""
import dataclasses
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


@pytest.fixture(scope="module")
def full():
    win, plans = W.make_config(4)
    assert plans.n_plans == 1 << 20
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    return win, plans, (dev, prio, flags)


def score_all(ctx, win, rows, P):
    ctx.wf_plan_upload_window(win)
    scores = pkg.score_batch(ctx, *rows, P)
    best = pkg.argmin(ctx, scores, P)
    torch.cuda.synchronize()
    return pkg.scores_to_numpy(scores, P), int(best.item())


@pytest.mark.parametrize("mode", ["paper_order", "batch_limit_2", "batch_limit_4"])
def test_window_options_full_size(ctx, full, mode):
    win, plans, rows = full
    if mode == "paper_order":
        w = dataclasses.replace(win, victim_order=1)
    else:
        w = dataclasses.replace(win, dev_batch=np.full(win.n_dev, int(mode[-1]), np.int32))
    log(f"[full] {mode}: P={plans.n_plans}")
    got, best = score_all(ctx, w, rows, plans.n_plans)
    ref = oracle.score(w, plans, threads=THREADS)
    assert got.tobytes() == ref.tobytes(), mode
    assert best == best_plan(ref)


def test_keys_full_size(ctx, full):
    win, plans, rows = full
    P = plans.n_plans
    log(f"[full] keys: P={P}")
    ctx.wf_plan_upload_window(win)
    keys = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_score_keys(*rows, P, keys)
    out = torch.empty(1, dtype=torch.int64, device="cuda:0")
    ctx.wf_plan_argmin_keys(keys, P, out)
    torch.cuda.synchronize()
    got = pkg.keys_to_numpy(keys, P)
    ref = oracle.phi_keys(win, plans, threads=THREADS)
    assert got.tobytes() == ref.tobytes()
    ok = np.nonzero(ref["status"] == 0)[0]
    want = -1
    if len(ok):
        order = np.lexsort(tuple(ref[k][ok] for k in ("h_life_us",)) +
                           (-ref["timely_prefetch"][ok].astype(np.int64), ref["c_ready_us"][ok]) +
                           tuple(-ref["admitted"][ok][:, c].astype(np.int64) for c in range(3, -1, -1)))
        want = int(ok[order[0]])
    assert int(out.item()) == want


def test_generated_candidates_full_size(ctx, full):
    win, plans, rows = full
    n = plans.n_plans
    log(f"[full] candidates: n={n}")
    ctx.wf_plan_upload_window(win)
    inc = (plans.dev[3].copy(), plans.prio[3].copy(), plans.flags[3].copy())
    drows = (torch.from_numpy(inc[0]).cuda(), torch.from_numpy(inc[1].view("<i2")).cuda(),
             torch.from_numpy(inc[2]).cuda())
    scores = torch.empty((n, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(drows[0], drows[1], drows[2], 0x5EED, 2, 0, n, scores)
    best = pkg.argmin(ctx, scores, n)
    torch.cuda.synchronize()
    cand = W.PlanBatch(*oracle.search_candidates(win, *inc, 0x5EED, 2, 0, n))
    ref = oracle.score(win, cand, threads=THREADS)
    assert pkg.scores_to_numpy(scores, n).tobytes() == ref.tobytes()
    assert int(best.item()) == best_plan(ref)

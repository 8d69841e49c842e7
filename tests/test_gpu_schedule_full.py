"""Per-plan schedules of every plan of every benchmark workload against the
oracle: start, finish, load start and reclaimed copies per activation and
peak memory per device, bytewise, through the schedule-writing kernel
instantiation, in chunks that bound host and device memory (the
1,048,576-plan workload in chunks of 65,536 plans)."""
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


def chunk_plans(N):
    # at most 512 MiB of int64 schedule rows per chunk (four [chunk][N] arrays)
    return 65536 if N <= 256 else max(256, (1 << 29) // (N * 8 * 4))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_every_plan_schedule(ctx, cfg):
    win, plans = W.make_config(cfg)
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    ctx.wf_plan_upload_window(win)
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    C = min(P, chunk_plans(N))
    for c0 in range(0, P, C):
        c1 = min(P, c0 + C)
        n = c1 - c0
        log(f"[sched-full] config {cfg}: plans {c0}..{c1 - 1} of {P}")
        scores, sched = pkg.score_batch(ctx, dev[c0:c1], prio[c0:c1], flags[c0:c1], n,
                                        schedule=True, n_act=N, n_dev=D, reclaims=True)
        torch.cuda.synchronize()
        got = pkg.scores_to_numpy(scores, n)
        ref, rs = oracle.score(win, plans, begin=c0, end=c1, schedule=True, threads=THREADS,
                               reclaims=True)
        assert got.tobytes() == ref.tobytes(), f"config {cfg}: score records differ in {c0}..{c1}"
        ok = (ref["status"] & pkg.WF_ST_INELIGIBLE) == 0
        for name, g, r in zip(("start", "finish", "load_start", "peak", "reclaimed"), sched, rs):
            a = g.cpu().numpy()
            if name == "reclaimed":
                a = a.view(np.uint64)
            a = a[:, :r.shape[1]]
            bad = np.nonzero((a[ok] != r[ok]).any(axis=1))[0]
            assert len(bad) == 0, (f"config {cfg}: {name} differs for plans "
                                   f"{(c0 + np.nonzero(ok)[0][bad[:10]]).tolist()}")
        del scores, sched

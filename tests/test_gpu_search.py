"""Candidates generated around an incumbent on the GPU (wf_plan_search_batch,
wf_plan_search_rows) against the oracle's generator and scorer, element by
element: the candidate rows bytewise, the score records bytewise, the argmin
exactly."""
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


def incumbent(plans, k=0):
    return plans.dev[k].copy(), plans.prio[k].copy(), plans.flags[k].copy()


def to_dev(d, p, f, offset=0):
    """Incumbent rows on the GPU; offset > 0 shifts them off 4-byte alignment."""
    if offset == 0:
        return (torch.from_numpy(np.ascontiguousarray(d)).cuda(),
                torch.from_numpy(np.ascontiguousarray(p).view("<i2")).cuda(),
                torch.from_numpy(np.ascontiguousarray(f)).cuda())
    bd = torch.zeros(d.size + offset, dtype=torch.int8, device="cuda:0")
    bp = torch.zeros(p.size + offset, dtype=torch.int16, device="cuda:0")
    bf = torch.zeros(f.size + offset, dtype=torch.uint8, device="cuda:0")
    if d.size:
        bd[offset:] = torch.from_numpy(d).cuda()
        bp[offset:] = torch.from_numpy(p.view("<i2")).cuda()
    if f.size:
        bf[offset:] = torch.from_numpy(f).cuda()
    return (bd.data_ptr() + offset, bp.data_ptr() + 2 * offset, bf.data_ptr() + offset,
            (bd, bp, bf))


def gpu_search(ctx, win, inc, seed, n_mut, first, n, offset=0):
    ctx.wf_plan_upload_window(win)
    rows = to_dev(*inc, offset=offset)
    scores = torch.empty((max(n, 1), 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], seed, n_mut, first, n, scores)
    best = torch.empty(1, dtype=torch.int64, device="cuda:0")
    ctx.wf_plan_argmin(scores, n, best)
    torch.cuda.synchronize()
    return pkg.scores_to_numpy(scores, n), int(best.item())


def oracle_search(win, inc, seed, n_mut, first, n):
    cd, cp, cf = oracle.search_candidates(win, *inc, seed, n_mut, first, n)
    return oracle.score(win, W.PlanBatch(cd, cp, cf), threads=THREADS), (cd, cp, cf)


@pytest.mark.parametrize("cfg,n,n_mut", [(0, 512, 1), (0, 300, 6), (1, 2048, 3), (2, 512, 4),
                                         (3, 128, 2), (4, 20000, 2), (4, 5000, 0)])
def test_search_scores_match_oracle(ctx, cfg, n, n_mut):
    win, plans = W.make_config(cfg, n_plans=4)
    inc = incumbent(plans, cfg % 4)
    seed, first = 0x9E3779B97F4A7C15 ^ cfg, 12345 * cfg
    log(f"[search] config {cfg}: {n} candidates, {n_mut} mutations")
    got, best = gpu_search(ctx, win, inc, seed, n_mut, first, n)
    ref, _ = oracle_search(win, inc, seed, n_mut, first, n)
    assert got.tobytes() == ref.tobytes()
    assert best == best_plan(ref)


@pytest.mark.parametrize("cfg,n_mut", [(0, 5), (1, 2), (4, 9), (4, 64)])
def test_search_rows_match_oracle(ctx, cfg, n_mut):
    win, plans = W.make_config(cfg, n_plans=4)
    inc = incumbent(plans, 1)
    seed, first, n = 77 + cfg, (1 << 32) - 10, 64
    ctx.wf_plan_upload_window(win)
    rows = to_dev(*inc)
    N, nb = win.n_act, (win.n_act + 3) // 4
    od = torch.empty((n, N), dtype=torch.int8, device="cuda:0")
    op = torch.empty((n, N), dtype=torch.int16, device="cuda:0")
    of = torch.empty((n, nb), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_rows(rows[0], rows[1], rows[2], seed, n_mut, first, n, od, op, of)
    torch.cuda.synchronize()
    cd, cp, cf = oracle.search_candidates(win, *inc, seed, n_mut, first, n)
    assert (od.cpu().numpy() == cd).all()
    assert (op.cpu().numpy().view("<u2") == cp).all()
    assert (of.cpu().numpy() == cf).all()


@pytest.mark.parametrize("seed", range(16))
def test_search_random_windows(ctx, seed):
    """Arbitrary windows and incumbents: odd N (byte-wise rows), fused chains,
    tied or out-of-range priorities (the ranked order), invalid devices."""
    rng = np.random.default_rng(40_000 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 5)), nodes=(1, 14),
                          n_dev=int(rng.integers(1, 7)), n_models=int(rng.integers(1, 9)))
    mode = ["any", "perm", "globalperm"][seed % 3]
    plans = W.random_plans(win, 1, rng, prio_mode=mode, p_bad_dev=0.05 if seed % 4 == 0 else 0.0)
    inc = incumbent(plans)
    n_mut, n = int(rng.integers(0, 12)), 700
    s64 = int(rng.integers(0, 1 << 62)) * 3
    first = int(rng.integers(0, 1 << 40))
    got, best = gpu_search(ctx, win, inc, s64, n_mut, first, n)
    ref, _ = oracle_search(win, inc, s64, n_mut, first, n)
    assert got.tobytes() == ref.tobytes(), f"seed {seed}"
    assert best == best_plan(ref)


def test_search_misaligned_incumbent(ctx):
    win, plans = W.make_config(1, n_plans=2)
    inc = incumbent(plans)
    got, _ = gpu_search(ctx, win, inc, 5, 3, 0, 400, offset=1)
    ref, _ = oracle_search(win, inc, 5, 3, 0, 400)
    assert got.tobytes() == ref.tobytes()


def test_search_large_window(ctx):
    """A window whose per-plan state does not fit in LDS (HBM scratch)."""
    rng = np.random.default_rng(5)
    win = W.random_window(rng, n_wf=400, nodes=(40, 60), n_dev=4, n_models=8, p_edge=0.1)
    plans = W.random_plans(win, 1, rng, prio_mode="perm")
    inc = incumbent(plans)
    got, best = gpu_search(ctx, win, inc, 11, 4, 3, 24)
    ref, _ = oracle_search(win, inc, 11, 4, 3, 24)
    assert got.tobytes() == ref.tobytes()


def test_search_edge_cases(ctx):
    win, plans = W.make_config(0, n_plans=2)
    inc = incumbent(plans)
    ctx.wf_plan_upload_window(win)
    rows = to_dev(*inc)
    scores = torch.zeros((4, 32), dtype=torch.uint8, device="cuda:0")
    ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], 1, 2, 0, 0, scores)  # no candidates
    for bad in (dict(n_mut=-1), dict(n_mut=pkg._lib.WF_MAX_MUT + 1), dict(first=-1),
                dict(first=(1 << 62) - 2, n=4)):
        kw = dict(n_mut=1, first=0, n=4)
        kw.update(bad)
        with pytest.raises(pkg.WFError) as e:
            ctx.wf_plan_search_batch(rows[0], rows[1], rows[2], 1, kw["n_mut"], kw["first"], kw["n"],
                                     scores)
        assert e.value.status == pkg.WF_EINVAL
    # the last admissible candidates
    got, _ = gpu_search(ctx, win, inc, 3, 7, (1 << 62) - 40, 40)
    ref, _ = oracle_search(win, inc, 3, 7, (1 << 62) - 40, 40)
    assert got.tobytes() == ref.tobytes()


def test_search_zero_mutations_equal_scoring_the_incumbent(ctx):
    win, plans = W.make_config(4, n_plans=1)
    inc = incumbent(plans)
    got, best = gpu_search(ctx, win, inc, 9, 0, 0, 100)
    ref = oracle.score(win, plans)
    assert (got.tobytes() == np.repeat(ref, 100).tobytes())

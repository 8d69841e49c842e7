"""The argmin that allocates nothing (wf_plan_argmin_noalloc, through the C
ABI) against the context's argmin (wf_plan_argmin) on the same records:
two calls in a row on one GPU, the second with a smaller input, so that a
partial minimum left in the static work area by the first call would show
in the second."""
import sys

import numpy as np
import pytest
import torch

import paper_2609_03335_amd as pkg
from paper_2609_03335_amd import workload as W

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def records(n, seed, feasible_frac=0.5, levels=64):
    """n score records: objectives drawn from few values (many ties), a
    share of them infeasible."""
    rng = np.random.default_rng(seed)
    r = np.zeros(n, dtype=pkg.SCORE_DTYPE)
    r["objective"] = rng.integers(0, levels, n).astype(np.float32) * np.float32(1.5) + np.float32(7)
    r["status"] = np.where(rng.random(n) < feasible_frac, 0, rng.integers(1, 4, n)).astype(np.uint32)
    return r


def expected(r):
    ok = np.flatnonzero(r["status"] == 0)
    if ok.size == 0:
        return -1
    return int(ok[np.argmin(r["objective"][ok])])


def both(ctx, r):
    buf = torch.from_numpy(r.view(np.uint8).reshape(-1, 32).copy()).to("cuda:0")
    n = len(r)
    a = torch.full((1,), -7, dtype=torch.int64, device="cuda:0")
    b = torch.full((1,), -7, dtype=torch.int64, device="cuda:0")
    ctx.wf_plan_argmin(buf, n, a)
    pkg.wf_plan_argmin_noalloc(buf, n, b)
    torch.cuda.synchronize()
    return int(a.item()), int(b.item())


def test_noalloc_argmin_matches_context_argmin_twice():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(0)
    win, _ = W.make_config(0)
    with pkg.Context(0) as ctx:
        ctx.wf_plan_upload_window(win)
        # a large call (every one of the 512 partial minima written), then a
        # smaller one whose minimum is worse than the first call's
        big = records(1_000_003, seed=1)
        big["objective"][999_000] = np.float32(-5.0)
        big["status"][999_000] = 0
        log("[noalloc] call 1: n =", len(big))
        a, b = both(ctx, big)
        assert a == expected(big) == 999_000
        assert b == a
        small = records(5_000, seed=2)
        log("[noalloc] call 2: n =", len(small))
        a, b = both(ctx, small)
        assert a == expected(small)
        assert b == a
        # fewer plans than one block, and none feasible
        none = records(100, seed=3, feasible_frac=0.0)
        log("[noalloc] call 3: n =", len(none))
        a, b = both(ctx, none)
        assert a == b == -1
        # an empty batch writes -1
        out = torch.full((1,), 5, dtype=torch.int64, device="cuda:0")
        pkg.wf_plan_argmin_noalloc(None, 0, out)
        torch.cuda.synchronize()
        assert int(out.item()) == -1


def test_noalloc_argmin_rejects_sizes_beyond_the_limit():
    out = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    with pytest.raises(pkg.WFError) as e:
        pkg.wf_plan_argmin_noalloc(0x1000, 1 << 32, out)
    assert e.value.status == pkg.WF_EINVAL

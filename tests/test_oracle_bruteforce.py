"""Exhaustive enumeration of all plans of tiny windows (N <= 5, D = 2)."""
import numpy as np
import pytest

import oracle
import pins
from enumerate_plans import best_plan, enumerate_plans, tiny_window
from paper_2609_03335_amd import workload as W


@pytest.mark.parametrize("seed", range(6))
def test_exhaustive(seed):
    win = tiny_window(seed)
    plans = enumerate_plans(win)
    assert plans.n_plans > 50
    sc, sched = oracle.score(win, plans, schedule=True)
    # the optimum is unique in value; an optimal plan with every prefetch bit
    # set exists because prefetching never delays anything
    b = best_plan(sc)
    assert b >= 0
    fuse, pf = W.unpack_flags(plans.flags, win.n_act)
    allpf = np.nonzero(pf.all(axis=1) & (sc["status"] == 0))[0]
    assert sc["objective"][allpf].min() == sc["objective"][b]
    # a sample of the enumeration against the second formulation
    rng = np.random.default_rng(seed)
    for p in rng.choice(plans.n_plans, size=min(60, plans.n_plans), replace=False):
        assert not pins.compare_plan(win, plans, int(p), sc, sched)
    # every plan that differs only in a fuse bit on a non-fusible activation
    # scores the same (the bit is ignored)
    nonfus = [v for v in range(win.n_act) if v not in pins.fusible_set(win)]
    if nonfus:
        v = nonfus[0]
        fl = plans.flags.copy()
        fl[:, v // 4] ^= np.uint8(1 << (2 * (v % 4)))
        sc2 = oracle.score(win, W.PlanBatch(plans.dev, plans.prio, fl))
        assert (sc2 == sc).all()

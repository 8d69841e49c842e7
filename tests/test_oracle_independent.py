"""The oracle against an independent second formulation (tests/pins.py) on
random windows with every feature switched on: arrivals, device free times,
initial residency, ineligible entries, fused chains, prefetch bits, priority
ties, and capacities tight enough to force evictions and over-capacity.
Also the copies each unit reclaims (schedule output), from the replayed
resident sets."""
import numpy as np
import pytest

import oracle
from paper_2609_03335_amd import workload as W
import pins


def _check(win, plans):
    sc, sched = oracle.score(win, plans, schedule=True, reclaims=True)
    errs = []
    for p in range(plans.n_plans):
        errs += pins.compare_plan(win, plans, p, sc, sched)
    assert not errs, "\n".join(errs[:20])
    return sc


@pytest.mark.parametrize("seed", range(40))
def test_random_windows(seed):
    rng = np.random.default_rng(1000 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(1, 7),
                          n_dev=int(rng.integers(1, 4)), n_models=int(rng.integers(1, 6)))
    plans = W.random_plans(win, 24, rng, p_bad_dev=0.02 if seed % 3 == 0 else 0.0,
                           prio_mode=["any", "perm", "globalperm"][seed % 3])
    _check(win, plans)


@pytest.mark.parametrize("seed", range(12))
def test_tight_capacity(seed):
    """Small devices and big models: evictions every step, CAPACITY set."""
    rng = np.random.default_rng(2000 + seed)
    win = W.random_window(rng, n_wf=3, nodes=(2, 6), n_dev=2, n_models=5,
                          cap_range=(3000, 12000), w_range=(2000, 9000), mem_range=(100, 3000))
    plans = W.random_plans(win, 24, rng, prio_mode="any")
    sc = _check(win, plans)
    assert (sc["n_evicts"] > 0).any()


def test_capacity_flag_seen():
    seen = 0
    for seed in range(30):
        rng = np.random.default_rng(3000 + seed)
        win = W.random_window(rng, n_wf=2, nodes=(2, 5), n_dev=2, n_models=4,
                              cap_range=(2000, 6000), w_range=(2000, 6000))
        plans = W.random_plans(win, 16, rng)
        sc = _check(win, plans)
        seen += int(((sc["status"] & 2) > 0).sum())
    assert seen > 0


def test_config0_all_plans():
    win, plans = W.make_config(0)
    _check(win, plans.slice(0, 128))


def test_config1_sample():
    win, plans = W.make_config(1, n_plans=3)
    _check(win, plans)

"""Pins of the replica cap (Sec. 3.5: scale-out subject to the replica cap)
in the oracle, under the reading that a plan is over the cap when a model
is held, in some topological level, on more devices than its cap (held as
the level's units start, or loaded for one of them):

* a worked example derived by hand (tests/golden/replica_cap.json): a copy
  spread over two devices in one level, a second copy loaded in a later
  level while the first remains, a copy that moves (reclaimed, then loaded
  elsewhere) and stays within the cap;
* a second formulation (tests/pins.py replica_over) that replays each
  device's units level by level, compared plan by plan;
* the cap is a check only: every other field equals the uncapped run;
* caps of at least the number of devices never flag a plan, and raising a
  cap never adds the flag;
* windows whose caps are below 1 or below the initial copies are refused.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import pins
from fixtures import load_golden
from paper_2609_03335_amd import workload as W


def _uncapped(win):
    return dataclasses.replace(win, model_replica_cap=None)


def _random_capped(seed, n_plans=120):
    rng = np.random.default_rng(700 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(2, 6)), nodes=(2, 7),
                          n_dev=int(rng.integers(2, 6)), n_models=int(rng.integers(1, 6)),
                          cap_range=(6000, 25000), same_model_bias=0.5)
    D, M = win.n_dev, win.n_models
    init = np.array([sum(((int(win.init_resident[d]) >> m) & 1) for d in range(D)) for m in range(M)])
    win.model_replica_cap = np.maximum(init, rng.integers(1, D + 1, M)).astype(np.int32)
    plans = W.random_plans(win, n_plans, rng, prio_mode=("any", "perm")[seed % 2])
    return win, plans


def test_worked_example():
    win, plans, ix, spec = load_golden("replica_cap")
    for name, pl in plans.items():
        sc = oracle.score(win, pl)
        free = oracle.score(_uncapped(win), pl)
        assert int(sc["status"][0]) == spec["expect_status"][name], name
        assert int(sc["n_evicts"][0]) == spec["expect_evicts"][name], name
        assert int(free["status"][0]) == 0, name
        for k in ("makespan_us", "p95_us", "objective", "min_headroom_mib", "n_loads", "n_evicts"):
            assert sc[k][0] == free[k][0], (name, k)


def _check_second_formulation(seed):
    """Plans of one random window whose flag matches; returns how many are
    over the cap."""
    win, plans = _random_capped(seed)
    sc = oracle.score(win, plans)
    flagged = 0
    for p in range(plans.n_plans):
        dev, prio, fuse, pf = pins.plan_rows(win, plans, p)
        units = pins.form_units(win, dev, prio, fuse)
        if units is None:
            assert int(sc["status"][p]) == oracle.INELIGIBLE
            continue
        over = pins.replica_over(win, units)
        assert bool(int(sc["status"][p]) & oracle.REPLICA) == over, (seed, p)
        flagged += over
    return flagged


@pytest.mark.parametrize("seed", range(12))
def test_against_second_formulation(seed):
    _check_second_formulation(seed)


def test_both_outcomes_occur():
    """The random windows flag some plans and pass others."""
    flagged = sum(_check_second_formulation(s) for s in range(12))
    assert 0 < flagged < 12 * 120


@pytest.mark.parametrize("seed", range(6))
def test_cap_is_a_check_only(seed):
    win, plans = _random_capped(seed)
    a, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    b, (st2, fi2, ls2, pk2) = oracle.score(_uncapped(win), plans, schedule=True)
    assert np.array_equal(a["status"] & ~np.uint32(oracle.REPLICA), b["status"])
    for k in ("makespan_us", "p95_us", "objective", "min_headroom_mib", "n_loads", "n_evicts"):
        assert np.array_equal(a[k], b[k]), k
    for x, y in ((st, st2), (fi, fi2), (ls, ls2), (pk, pk2)):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("seed", range(6))
def test_large_caps_never_flag_and_raising_caps_never_adds(seed):
    win, plans = _random_capped(seed)
    big = dataclasses.replace(win, model_replica_cap=np.full(win.n_models, win.n_dev, np.int32))
    assert not (oracle.score(big, plans)["status"] & oracle.REPLICA).any()
    base = oracle.score(win, plans)["status"] & oracle.REPLICA
    rng = np.random.default_rng(seed)
    more = win.model_replica_cap + rng.integers(0, 2, win.n_models).astype(np.int32)
    raised = oracle.score(dataclasses.replace(win, model_replica_cap=more), plans)["status"] & oracle.REPLICA
    assert not (raised & ~base).any()


def test_invalid_caps_refused():
    win, plans = _random_capped(0, n_plans=2)
    zero = dataclasses.replace(win, model_replica_cap=np.zeros(win.n_models, np.int32))
    with pytest.raises(oracle.OracleError):
        oracle.score(zero, plans)
    win2 = dataclasses.replace(win, init_resident=np.full(win.n_dev, 1, np.uint64),
                               dev_cap_mib=np.full(win.n_dev, 1 << 29, np.int32),
                               model_replica_cap=np.ones(win.n_models, np.int32))
    if win2.n_dev > 1:
        with pytest.raises(oracle.OracleError):
            oracle.score(win2, plans)

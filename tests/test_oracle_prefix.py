"""Pins of the oracle's prefix commit (Algorithm 1, Prefix_t) and of the
reclaimed copies it reports per unit.

* A worked example derived by hand (tests/golden/prefix_commit.json): one
  plan whose next event is a load's end, with a committed reclamation; one
  whose next event is a workflow's arrival, with an action that begins
  exactly then (not committed).
* A closed form: one device, every model resident, one workflow arriving at
  0 whose units form a chain: the next event is the first finish after 0
  (a unit of zero length at time 0 ends no earlier than it starts, so it is
  no event), and the units that start before it are committed.
* Invariants on random windows: the next event is an event (a finish, a load
  end or an arrival after 0) and none lies between 0 and it; an action is
  committed exactly when it begins before it; committed reclamations are the
  unit's own; the reclaimed copies of a plan add up to its eviction count.
"""
import numpy as np
import pytest

import oracle
from fixtures import load_golden
from paper_2609_03335_amd import workload as W


def _mask(names, models):
    return sum(1 << models.index(n) for n in names)


def test_worked_example():
    win, plans, ix, spec = load_golden("prefix_commit")
    models = [m["name"] for m in spec["models"]]
    for pname, exp in spec["expect_times"].items():
        sc, (st, fi, ls, pk, rc) = oracle.score(win, plans[pname], schedule=True, reclaims=True)
        for key, arr in (("start", st), ("finish", fi), ("load_start", ls)):
            for n, v in exp[key].items():
                assert int(arr[0, ix[n]]) == v, (pname, key, n)
        for n, v in exp["reclaimed"].items():
            assert int(rc[0, ix[n]]) == _mask(v, models), (pname, "reclaimed", n)
        for k in ("makespan", "min_headroom", "status", "n_loads", "n_evicts"):
            field = {"makespan": "makespan_us", "min_headroom": "min_headroom_mib"}.get(k, k)
            assert int(sc[field][0]) == exp[k], (pname, k)
        pre = spec["expect_prefix"][pname]
        commit, crec, t_next = oracle.prefix(win, plans[pname].dev[0], st[0], fi[0], ls[0], rc[0])
        assert t_next == pre["t_next"], pname
        for n, i in ix.items():
            assert bool(commit[i] & 1) == (n in pre["grant"]), (pname, "grant", n)
            assert bool(commit[i] & 2) == (n in pre["load"]), (pname, "load", n)
            assert int(crec[i]) == _mask(pre["reclaimed"].get(n, []), models), (pname, "reclaimed", n)


def test_device_out_of_range_is_rejected():
    win, plans, ix, spec = load_golden("prefix_commit")
    sc, (st, fi, ls, pk, rc) = oracle.score(win, plans["p"], schedule=True, reclaims=True)
    bad = plans["p"].dev[0].copy()
    bad[0] = win.n_dev
    with pytest.raises(oracle.OracleError):
        oracle.prefix(win, bad, st[0], fi[0], ls[0], rc[0])


@pytest.mark.parametrize("seed", range(8))
def test_single_device_chain(seed):
    rng = np.random.default_rng(61_000 + seed)
    T = int(rng.integers(2, 8))
    lat = rng.integers(1, 1000, T)
    if seed % 2:
        lat[0] = 0  # a zero-length first unit: its finish at 0 is no event
    win = W.Window(
        n_act=T, n_wf=1, n_models=2, n_dev=1, act_wf=np.zeros(T, np.int32),
        act_model=rng.integers(0, 2, T).astype(np.int32),
        pred_off=np.concatenate([[0], np.arange(T)]).astype(np.int32),
        pred_idx=np.arange(max(T - 1, 0), dtype=np.int32), lat_us=lat.astype(np.int32),
        mem_mib=np.zeros(T, np.int32), wf_arrival_us=np.zeros(1, np.int64),
        dev_cap_mib=np.array([100], np.int32), model_mib=np.array([10, 10], np.int32),
        load_us=np.array([50, 70], np.int32), init_resident=np.array([3], np.uint64),
        dev_free0_us=np.zeros(1, np.int64), name="chain")
    plan = W.PlanBatch(np.zeros((1, T), np.int8), np.zeros((1, T), np.uint16),
                       np.zeros((1, (T + 3) // 4), np.uint8))
    sc, (st, fi, ls, pk, rc) = oracle.score(win, plan, schedule=True, reclaims=True)
    commit, crec, t_next = oracle.prefix(win, plan.dev[0], st[0], fi[0], ls[0], rc[0])
    finish = np.cumsum(lat)
    start = finish - lat
    assert np.array_equal(fi[0], finish) and np.array_equal(st[0], start)
    assert t_next == int(finish[finish > 0][0])
    assert commit.tolist() == [int(x < t_next) for x in start]
    assert commit[0] == 1 and commit[1] == (1 if lat[0] == 0 else 0)
    assert not crec.any() and not rc.any()


@pytest.mark.parametrize("seed", range(12))
def test_invariants(seed):
    rng = np.random.default_rng(62_000 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 5)), nodes=(2, 7), n_dev=int(rng.integers(1, 4)),
                          n_models=5, cap_range=(8000, 16000), w_range=(2000, 7000))
    if seed % 3 == 1:
        win.victim_order = oracle.VICTIM_PAPER
    if seed % 3 == 2:
        win.dev_batch = rng.integers(1, oracle.MAX_BATCH + 1, win.n_dev).astype(np.int32)
    plans = W.random_plans(win, 40, rng)
    sc, (st, fi, ls, pk, rc) = oracle.score(win, plans, schedule=True, reclaims=True)
    N, D = win.n_act, win.n_dev
    load = win.load_us.reshape(win.n_models, D)
    for p in range(plans.n_plans):
        if sc["status"][p] & oracle.INELIGIBLE:
            continue
        # reclaimed copies add up to the plan's evictions
        assert sum(bin(int(x)).count("1") for x in rc[p]) == int(sc["n_evicts"][p])
        commit, crec, t = oracle.prefix(win, plans.dev[p], st[p], fi[p], ls[p], rc[p])
        dev = plans.dev[p].astype(int)
        ends = [int(x) for x in fi[p]]
        ends += [int(ls[p, i]) + int(load[win.act_model[i], dev[i]]) for i in range(N) if ls[p, i] >= 0]
        ends += [int(a) for a in win.wf_arrival_us]
        later = [e for e in ends if e > 0]
        assert t == (min(later) if later else np.iinfo(np.int64).max)
        for i in range(N):
            assert bool(commit[i] & 1) == (st[p, i] < t)
            assert bool(commit[i] & 2) == (0 <= ls[p, i] < t)
            assert int(crec[i]) in (0, int(rc[p, i]))
            # a unit's first action is its load when it loads
            first = ls[p, i] if ls[p, i] >= 0 else st[p, i]
            assert (int(crec[i]) == int(rc[p, i])) == (first < t or rc[p, i] == 0)

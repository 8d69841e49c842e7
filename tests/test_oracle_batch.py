"""Pins of the oracle's batch limit (Eq. 11 and the replica batch limit B_q;
continuous batching, Sec. 4): a device runs up to B units at once, memory is
checked at each first action against the units still running, running
units lease their models.

* Worked examples (tests/golden/batch_*.json), derived by hand: a unit that
  waits for memory (and the finish-time boundary), a reclamation blocked by
  leases until a unit completes.
* A closed form: with as many slots as units on every device, every model
  resident and ample memory, a unit waits only for its release and for the
  unit before it in its device's queue to have started:
  start = max(release, previous start on the device), by a separate
  recursion over the resource order.
* Invariants read from the schedule: no more than B units of a device
  overlap; with weightless models the activation memory of overlapping
  units never exceeds the capacity in a feasible plan; no model is loaded
  onto a device while a unit of that model runs there (its lease).
* B = 1 everywhere is the one-unit device: identical to no batch limits.
"""
import numpy as np
import pytest

import oracle
from fixtures import load_golden
from paper_2609_03335_amd import workload as W


@pytest.mark.parametrize("name", ["batch_memory", "batch_lease"])
def test_worked_examples(name):
    win, plans, ix, spec = load_golden(name)
    for pname, exp in spec["expect_times"].items():
        sc, (st, fi, ls, pk) = oracle.score(win, plans[pname], schedule=True)
        for key, arr in (("start", st), ("finish", fi), ("load_start", ls)):
            for n, v in exp[key].items():
                assert int(arr[0, ix[n]]) == v, (name, key, n)
        assert int(sc["makespan_us"][0]) == exp["makespan"]
        assert int(sc["min_headroom_mib"][0]) == exp["min_headroom"]
        assert int(sc["status"][0]) == exp["status"]
        for k in ("n_evicts", "n_loads"):
            if k in exp:
                assert int(sc[k][0]) == exp[k]


def test_batch_outside_range_is_rejected():
    win, plans, ix, spec = load_golden("batch_memory")
    for bad in (0, oracle.MAX_BATCH + 1):
        win.dev_batch = np.array([bad], np.int32)
        with pytest.raises(oracle.OracleError):
            oracle.score(win, plans["shared"])


@pytest.mark.parametrize("seed", range(6))
def test_batch_one_is_the_one_unit_device(seed):
    rng = np.random.default_rng(96_000 + seed)
    win = W.random_window(rng, n_wf=4, nodes=(2, 9), n_dev=3, n_models=5,
                          cap_range=(9000, 20000), w_range=(2000, 7000))
    plans = W.random_plans(win, 80, rng)
    a = oracle.score(win, plans, schedule=True)
    win.dev_batch = np.ones(win.n_dev, np.int32)
    b = oracle.score(win, plans, schedule=True)
    assert a[0].tobytes() == b[0].tobytes()
    for x, y in zip(a[1], b[1]):
        assert np.array_equal(x, y)


def _queue_finish(win, plan_dev, plan_prio):
    """Finish times when every device has a free slot for every unit: units
    in (level, priority, index) order, each starting at the later of its
    release and the previous start on its device."""
    N, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(N, D)
    preds = [win.pred_idx[win.pred_off[i]:win.pred_off[i + 1]] for i in range(N)]
    level = np.zeros(N, np.int64)
    for v in range(N):
        level[v] = 1 + max((level[u] for u in preds[v]), default=-1)
    fin = np.zeros(N, np.int64)
    prev = np.zeros(D, np.int64)
    for v in sorted(range(N), key=lambda v: (level[v], plan_prio[v], v)):
        r = max([int(win.wf_arrival_us[win.act_wf[v]])] + [int(fin[u]) for u in preds[v]])
        s = max(r, int(prev[plan_dev[v]]))
        prev[plan_dev[v]] = s
        fin[v] = s + int(lat[v, plan_dev[v]])
    return fin


@pytest.mark.parametrize("seed", range(10))
def test_contention_free_longest_path(seed):
    rng = np.random.default_rng(97_000 + seed)
    D = int(rng.integers(2, 6))
    win = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(2, 6), n_dev=D, n_models=4,
                          q_inel=0.0, free0=False, resident=False, cap_range=(1 << 29, 1 << 29))
    N = win.n_act
    if N > oracle.MAX_BATCH * D:
        pytest.skip("more units than slots")
    win.init_resident = np.full(D, (1 << win.n_models) - 1, np.uint64)
    win.dev_batch = np.full(D, oracle.MAX_BATCH, np.int32)
    dev = np.array([[i % D for i in range(N)]], np.int8)  # at most MAX_BATCH units per device
    prio = np.array([rng.permutation(N)], np.uint16)
    plans = W.PlanBatch(dev, prio, np.zeros((1, (N + 3) // 4), np.uint8))
    sc, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    assert sc["status"][0] == 0 and sc["n_loads"][0] == 0
    assert np.array_equal(fi[0], _queue_finish(win, dev[0], prio[0]))


def _first_action(ls, st, v):
    return ls[v] if ls[v] >= 0 else st[v]


def _unit_spans(win, plans, p, sched):
    """(device, first action, unit end, model, memory, head) per unit."""
    st, fi, ls = sched[0][p], sched[1][p], sched[2][p]
    N, D = win.n_act, win.n_dev
    preds = [win.pred_idx[win.pred_off[i]:win.pred_off[i + 1]] for i in range(N)]
    succ = [[] for _ in range(N)]
    for v in range(N):
        for u in preds[v]:
            succ[u].append(v)
    fuse, _ = W.unpack_flags(plans.flags[p:p + 1], N)
    member = np.array([fuse[0][v] and len(preds[v]) == 1 and len(succ[preds[v][0]]) == 1
                       and win.act_model[preds[v][0]] == win.act_model[v] for v in range(N)])
    mem = win.mem_mib.reshape(N, D)
    spans = []
    for h in range(N):
        if member[h]:
            continue
        d = int(plans.dev[p, h])
        v, mx = h, int(mem[h, d])
        while len(succ[v]) == 1 and member[succ[v][0]]:
            v = succ[v][0]
            mx = max(mx, int(mem[v, d]))
        spans.append((d, int(_first_action(ls, st, h)), int(fi[v]), int(win.act_model[h]), mx, h))
    return spans


@pytest.mark.parametrize("seed", range(12))
def test_schedule_invariants(seed):
    rng = np.random.default_rng(98_000 + seed)
    D = int(rng.integers(1, 4))
    weightless = seed % 2 == 0
    win = W.random_window(rng, n_wf=int(rng.integers(2, 6)), nodes=(2, 8), n_dev=D, n_models=5,
                          cap_range=(4000, 12000) if weightless else (9000, 18000),
                          w_range=(0, 0) if weightless else (1500, 5000),
                          mem_range=(500, 4000), q_inel=0.0)
    win.dev_batch = rng.integers(1, oracle.MAX_BATCH + 1, D).astype(np.int32)
    plans = W.random_plans(win, 120, rng, prio_mode=["any", "perm"][seed % 2])
    sc, sched = oracle.score(win, plans, schedule=True)
    n_feasible = 0
    for p in range(plans.n_plans):
        if sc["status"][p] & oracle.INELIGIBLE:
            continue
        spans = _unit_spans(win, plans, p, sched)
        for d in range(D):
            on = [s for s in spans if s[0] == d]
            for (_, t0, t1, m, mx, h) in on:
                running = [s for s in on if s[1] <= t0 < s[2]]
                # at most B units run at once on the device
                assert len(running) <= win.dev_batch[d], (p, d, h)
                if weightless and sc["status"][p] == 0:
                    assert sum(s[4] for s in running) <= win.dev_cap_mib[d], (p, d, h)
                # a model is never loaded while a unit of it runs there
                if sched[2][p][h] >= 0:
                    assert not any(s[3] == m and s[1] < t0 < s[2] for s in on if s[5] != h), (p, d, h)
        n_feasible += sc["status"][p] == 0
    assert n_feasible > 0

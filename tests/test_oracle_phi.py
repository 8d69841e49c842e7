"""Pins of the oracle's ranking key (Eq. 12, Sec. 3.5):
Phi = (-A_1, ..., -A_K, C_F, -P_N, H_life).

* Worked examples (tests/golden/phi_*.json): every term derived by hand in
  the fixture, including a reload after reclamation, a prefetch whose load
  ends exactly at the release, a ready unit that is not admitted, a
  workflow that has not arrived by the window time, and priority classes.
* A second formulation: C_F, P_N, H_life and (for feasible plans) A_k
  recomputed from the oracle's schedule output -- start, finish and load
  start of every activation -- with a different characterisation of the
  reload cost: a load of a model that was already present on the device
  earlier (initially resident or loaded before) must follow a reclamation
  of it.
* Invariants that hold whatever the plan.
"""
import numpy as np
import pytest

import oracle
from fixtures import load_golden
from paper_2609_03335_amd import workload as W


def _as_dict(k):
    return {"admitted": [int(x) for x in k["admitted"]], "c_ready_us": int(k["c_ready_us"]),
            "timely_prefetch": int(k["timely_prefetch"]), "h_life_us": int(k["h_life_us"]),
            "status": int(k["status"])}


@pytest.mark.parametrize("name", ["phi_reload", "phi_prefetch", "phi_ready_prefetch"])
def test_worked_examples(name):
    win, plans, ix, spec = load_golden(name)
    for pname, exp in spec["expect_phi"].items():
        assert _as_dict(oracle.phi_keys(win, plans[pname])[0]) == exp, pname
    wf_names = [w["name"] for w in spec["workflows"]]
    for vname, var in spec.get("class_variants", {}).items():
        win.wf_class = np.array([var["classes"][n] for n in wf_names], np.uint8)
        for pname, exp in var["expect_phi"].items():
            assert _as_dict(oracle.phi_keys(win, plans[pname])[0]) == exp, (vname, pname)


def test_class_outside_range_is_rejected():
    win, plans, ix, spec = load_golden("phi_reload")
    win.wf_class = np.array([0, oracle.MAX_CLASSES], np.uint8)
    with pytest.raises(oracle.OracleError):
        oracle.phi_keys(win, plans["reload"])


# ---------------------------------------------------------------------------
# second formulation from the schedule
# ---------------------------------------------------------------------------


def _structure(win):
    """Levels, unique parent/child and the fusion condition (Eq. 3), here in
    Python from the CSR arrays."""
    N = win.n_act
    preds = [list(win.pred_idx[win.pred_off[i]:win.pred_off[i + 1]]) for i in range(N)]
    succ = [[] for _ in range(N)]
    for v in range(N):
        for u in preds[v]:
            succ[u].append(v)
    level = np.zeros(N, np.int64)
    for v in range(N):
        level[v] = 1 + max((level[u] for u in preds[v]), default=-1)
    fusible = np.array([len(preds[v]) == 1 and len(succ[preds[v][0]]) == 1
                        and win.act_model[preds[v][0]] == win.act_model[v] for v in range(N)], bool)
    return preds, succ, level, fusible


def _phi_from_schedule(win, plans, p, sched, status, struct):
    preds, succ, level, fusible = struct
    N, D = win.n_act, win.n_dev
    st, fi, ls = sched[0][p], sched[1][p], sched[2][p]
    fuse, pf = W.unpack_flags(plans.flags[p:p + 1], N)
    fuse, pf = fuse[0], pf[0]
    dev, prio = plans.dev[p].astype(np.int64), plans.prio[p].astype(np.int64)
    load = win.load_us.reshape(win.n_models, D)
    member = fuse & fusible
    heads = [h for h in range(N) if not member[h]]

    def chain_end(h):
        v = h
        while len(succ[v]) == 1 and member[succ[v][0]]:
            v = succ[v][0]
        return v

    cls = win.wf_class if win.wf_class is not None else np.zeros(win.n_wf, np.uint8)
    ready = {h: len(preds[h]) == 0 and win.wf_arrival_us[win.act_wf[h]] <= 0 for h in heads}
    release = {h: max([int(win.wf_arrival_us[win.act_wf[h]])] + [int(fi[u]) for u in preds[h]])
               for h in heads}
    admitted = [0] * oracle.MAX_CLASSES
    c_ready = 0
    if status == 0:
        for h in heads:
            if ready[h]:
                admitted[cls[win.act_wf[h]]] += 1
                c_ready = max(c_ready, int(fi[chain_end(h)]))
    timely = 0
    for h in heads:
        if not ready[h] and pf[h] and ls[h] >= 0 and ls[h] + load[win.act_model[h], dev[h]] <= release[h]:
            timely += 1
    h_life = 0
    free0 = win.dev_free0_us if win.dev_free0_us is not None else np.zeros(D, np.int64)
    for d in range(D):
        seq = sorted((h for h in heads if dev[h] == d), key=lambda h: (level[h], prio[h], h))
        seen = {m for m in range(win.n_models) if (int(win.init_resident[d]) >> m) & 1}
        prev_end = int(free0[d])
        for h in seq:
            m = int(win.act_model[h])
            if ls[h] >= 0:
                if m in seen:  # present before: it was reclaimed in between
                    h_life += int(load[m, d])
                if ready[h]:
                    h_life += int(st[h]) - max(release[h], prev_end)
                seen.add(m)
            prev_end = int(fi[chain_end(h)])
    return admitted, c_ready, timely, h_life


def _random_case(seed):
    rng = np.random.default_rng(70_000 + seed)
    kind = seed % 3
    if kind == 0:
        win = W.random_window(rng, n_wf=int(rng.integers(2, 6)), nodes=(1, 8),
                              n_dev=int(rng.integers(1, 4)), n_models=int(rng.integers(2, 6)))
    elif kind == 1:  # tight memory: reclamation and reloads on most loads
        win = W.random_window(rng, n_wf=4, nodes=(2, 7), n_dev=2, n_models=5,
                              cap_range=(9000, 16000), w_range=(3000, 8000), mem_range=(0, 1500))
    else:  # fused chains, long prefetch windows
        win = W.random_window(rng, n_wf=3, nodes=(3, 9), n_dev=3, n_models=3, same_model_bias=0.8,
                              lat_range=(100, 5000), load_range=(0, 3000), cap_range=(30000, 60000))
    # about half of the workflows arrive at the window time (their sources
    # are ready work), the others later
    arr = win.wf_arrival_us.copy()
    arr[rng.random(win.n_wf) < 0.5] = 0
    win.wf_arrival_us = arr
    win.wf_class = rng.integers(0, oracle.MAX_CLASSES, win.n_wf).astype(np.uint8)
    plans = W.random_plans(win, 150, rng, prio_mode=["any", "perm"][seed % 2])
    return win, plans


@pytest.mark.parametrize("seed", range(12))
def test_phi_from_schedule(seed):
    win, plans = _random_case(seed)
    sc, sched = oracle.score(win, plans, schedule=True)
    keys = oracle.phi_keys(win, plans)
    struct = _structure(win)
    assert (keys["status"] == sc["status"]).all()
    n_feasible = 0
    for p in range(plans.n_plans):
        if sc["status"][p] & oracle.INELIGIBLE:
            assert _as_dict(keys[p]) == {"admitted": [0] * 4, "c_ready_us": 0, "timely_prefetch": 0,
                                         "h_life_us": 0, "status": oracle.INELIGIBLE}
            continue
        A, cf, pn, h = _phi_from_schedule(win, plans, p, sched, int(sc["status"][p]), struct)
        assert int(keys["timely_prefetch"][p]) == pn, p
        assert int(keys["h_life_us"][p]) == h, p
        if sc["status"][p] == 0:
            n_feasible += 1
            assert [int(x) for x in keys["admitted"][p]] == A, p
            assert int(keys["c_ready_us"][p]) == cf, p
    assert n_feasible > 0


@pytest.mark.parametrize("seed", range(6))
def test_phi_invariants(seed):
    win, plans = _random_case(100 + seed)
    sc = oracle.score(win, plans)
    keys = oracle.phi_keys(win, plans)
    preds, succ, level, fusible = _structure(win)
    N = win.n_act
    fuse, pf = W.unpack_flags(plans.flags, N)
    no_pred = np.array([len(preds[i]) == 0 for i in range(N)])
    arrived = win.wf_arrival_us[win.act_wf] <= 0
    for p in range(plans.n_plans):
        if sc["status"][p] & oracle.INELIGIBLE:
            continue
        head = ~(fuse[p] & fusible)
        ready = head & no_pred & arrived
        per_class = np.bincount(win.wf_class[win.act_wf[ready]], minlength=oracle.MAX_CLASSES)
        A = keys["admitted"][p].astype(np.int64)
        assert (A <= per_class).all()
        if sc["status"][p] == 0:
            assert (A == per_class).all()
        assert keys["timely_prefetch"][p] <= int((head & pf[p] & ~ready).sum())
        assert keys["h_life_us"][p] >= 0
        assert keys["c_ready_us"][p] <= sc["makespan_us"][p] + win.wf_arrival_us.min()
        if A.sum() == 0:
            assert keys["c_ready_us"][p] == 0
    # without prefetch bits there is no timely prefetch
    plans0 = W.PlanBatch(plans.dev, plans.prio, plans.flags & np.uint8(0x55))
    assert (oracle.phi_keys(win, plans0)["timely_prefetch"] == 0).all()

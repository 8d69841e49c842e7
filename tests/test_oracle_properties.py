"""Closed forms, lower bounds, invariants and metamorphic relations that the
oracle must satisfy whatever its implementation (no formula is retyped here:
each check is a consequence of the definitions, computed another way)."""
import networkx as nx
import numpy as np
import pytest

import oracle
from paper_2609_03335_amd import workload as W
import pins


def _window(n_wf, parents_per_wf, models, n_dev, lat, mem, cap, weights, load,
            arrivals=None, free0=None, resident=None, w_mk=1.0, w_p95=0.5):
    """Build a window from explicit per-workflow parent lists (local ids)."""
    b = W._Builder()
    k = 0
    for pw in parents_per_wf:
        b.add_workflow(pw, models[k:k + len(pw)])
        k += len(pw)
    act_wf, act_model, off, idx, nw = b.finish()
    assert nw == n_wf
    n = len(act_wf)
    # tables were given in build order; permute rows into the level-sorted numbering
    order = np.lexsort((np.array(b.local), np.array(b.wf_of),
                        W._depths(n, b.parents, range(n))))
    lat = np.asarray(lat, np.int32).reshape(n, n_dev)[order]
    mem = np.asarray(mem, np.int32).reshape(n, n_dev)[order]
    return W.Window(
        n_act=n, n_wf=n_wf, n_models=len(weights), n_dev=n_dev, act_wf=act_wf,
        act_model=act_model, pred_off=off, pred_idx=idx, lat_us=lat.reshape(-1),
        mem_mib=mem.reshape(-1),
        wf_arrival_us=np.zeros(n_wf, np.int64) if arrivals is None else np.asarray(arrivals, np.int64),
        dev_cap_mib=np.asarray(cap, np.int32), model_mib=np.asarray(weights, np.int32),
        load_us=np.asarray(load, np.int32).reshape(-1),
        init_resident=np.zeros(n_dev, np.uint64) if resident is None else np.asarray(resident, np.uint64),
        dev_free0_us=np.zeros(n_dev, np.int64) if free0 is None else np.asarray(free0, np.int64),
        w_makespan=w_mk, w_p95=w_p95), order


# ---------------------------------------------------------------------------
# P1: one device, ample memory: finish of the k-th unit in resource order is
#     free0 + sum_{j<=k} (T_j + [first use of a non-resident model] * L_j)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(15))
def test_single_device_closed_form(seed):
    rng = np.random.default_rng(seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(1, 6), n_dev=1, n_models=4,
                          cap_range=(10 ** 8, 10 ** 8), q_inel=0.0, arrivals=False)
    plans = W.random_plans(win, 16, rng, p_fuse=0.0, prio_mode="perm")
    sc, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    lat = win.lat_us.reshape(win.n_act, 1)[:, 0].astype(np.int64)
    load = win.load_us.astype(np.int64)
    lv = pins.nx_levels(win)
    for p in range(plans.n_plans):
        order = sorted(range(win.n_act), key=lambda i: (lv[i], plans.prio[p, i], i))
        t = int(win.dev_free0_us[0])
        seen = {m for m in range(win.n_models) if (int(win.init_resident[0]) >> m) & 1}
        for i in order:
            m = int(win.act_model[i])
            if m not in seen:
                t += int(load[m])
                seen.add(m)
            t += int(lat[i])
            assert fi[p, i] == t
        assert sc["makespan_us"][p] == t
        assert sc["n_evicts"][p] == 0 and sc["status"][p] == 0


# ---------------------------------------------------------------------------
# P2: no contention (one device per activation, every model resident, ample
#     memory): the timeline is the DAG longest path from the arrivals
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(15))
def test_contention_free_longest_path(seed):
    rng = np.random.default_rng(100 + seed)
    base = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(1, 7), n_dev=1, n_models=3)
    n = base.n_act
    D = n
    lat = rng.integers(1, 1000, size=(n, D)).astype(np.int32)
    win = W.Window(n_act=n, n_wf=base.n_wf, n_models=3, n_dev=D, act_wf=base.act_wf,
                   act_model=base.act_model, pred_off=base.pred_off, pred_idx=base.pred_idx,
                   lat_us=lat.reshape(-1), mem_mib=np.full(n * D, 10, np.int32),
                   wf_arrival_us=rng.integers(0, 5000, size=base.n_wf).astype(np.int64),
                   dev_cap_mib=np.full(D, 10 ** 6, np.int32), model_mib=np.full(3, 100, np.int32),
                   load_us=np.full(3 * D, 777, np.int32), init_resident=np.full(D, 7, np.uint64),
                   dev_free0_us=np.zeros(D, np.int64))
    plans = W.random_plans(win, 4, rng, p_fuse=0.0)
    plans.dev[:] = np.arange(n, dtype=np.int8)[None, :]
    sc, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    g = nx.DiGraph()
    for v in range(n):
        g.add_edge("src", v, weight=int(win.wf_arrival_us[win.act_wf[v]]) + int(lat[v, v]))
        for u in win.preds(v):
            g.add_edge(int(u), v, weight=int(lat[v, v]))
    for p in range(plans.n_plans):
        assert sc["n_loads"][p] == 0
        for v in range(n):
            sub = g.subgraph(nx.ancestors(g, v) | {v})
            assert fi[p, v] == nx.dag_longest_path_length(sub), (p, v)
        assert (ls[p] == -1).all()


# ---------------------------------------------------------------------------
# P5 lower bounds and P6 invariants on random windows
# ---------------------------------------------------------------------------
def _unit_info(win, plans, p):
    dev, prio, fuse, pf = pins.plan_rows(win, plans, p)
    return pins.form_units(win, dev, prio, fuse), pf


@pytest.mark.parametrize("seed", range(25))
def test_bounds_and_invariants(seed):
    rng = np.random.default_rng(200 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(1, 7),
                          n_dev=int(rng.integers(1, 4)), n_models=int(rng.integers(1, 5)),
                          cap_range=(6000, 30000))
    plans = W.random_plans(win, 20, rng, prio_mode=["any", "perm"][seed % 2])
    sc, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    D = win.n_dev
    lat = win.lat_us.reshape(win.n_act, D).astype(np.int64)
    load = win.load_us.reshape(win.n_models, D).astype(np.int64)
    cap = win.dev_cap_mib.astype(np.int64)
    arr = win.wf_arrival_us
    for p in range(plans.n_plans):
        units, pf = _unit_info(win, plans, p)
        if units is None:
            assert sc["status"][p] == 1
            continue
        dev_of = {v: u.device for u in units for v in u.chain}
        # precedence and durations
        for v in range(win.n_act):
            assert fi[p, v] == st[p, v] + lat[v, dev_of[v]]
            assert st[p, v] >= arr[win.act_wf[v]]
            for u in win.preds(v):
                assert st[p, v] >= fi[p, int(u)]
        # device slots never overlap and follow the resource order
        t_dev = {d: int(win.dev_free0_us[d]) for d in range(D)}
        for u in units:
            d = u.device
            slot0 = ls[p, u.head] if ls[p, u.head] >= 0 else st[p, u.head]
            assert slot0 >= t_dev[d]
            if ls[p, u.head] >= 0:
                le = ls[p, u.head] + load[u.model, d]
                assert le <= st[p, u.head]
                if not pf[u.head]:
                    r = max([int(arr[u.wf])] + [int(fi[p, int(q)]) for q in win.preds(u.head)])
                    assert ls[p, u.head] == max(r, t_dev[d])
            for a, b in zip(u.chain, u.chain[1:]):
                assert st[p, b] == fi[p, a]  # members back-to-back
                assert ls[p, b] == -1
            t_dev[d] = fi[p, u.chain[-1]]
        # feasibility and headroom
        st_p = int(sc["status"][p])
        if st_p == 0:
            assert (pk[p] <= cap).all()
        assert bool(st_p & 2) == (sc["min_headroom_mib"][p] < 0)
        assert sc["min_headroom_mib"][p] == (cap - pk[p]).min()
        used_pairs = {(u.device, u.model) for u in units}
        cold = {(d, m) for d, m in used_pairs if not (int(win.init_resident[d]) >> m) & 1}
        assert sc["n_loads"][p] >= len(cold)
        assert sc["n_loads"][p] == int((ls[p] >= 0).sum())
        # P5: critical path and device-busy lower bounds
        mk = int(sc["makespan_us"][p])
        a0 = int(arr.min())
        cp = np.zeros(win.n_act, np.int64)
        for v in range(win.n_act):
            cp[v] = max([int(arr[win.act_wf[v]])] + [int(cp[int(u)]) for u in win.preds(v)]) \
                + lat[v, dev_of[v]]
        assert mk >= cp.max() - a0
        busy = {d: int(win.dev_free0_us[d]) for d in range(D)}
        for u in units:
            busy[u.device] += sum(int(lat[v, u.device]) for v in u.chain)
            if ls[p, u.head] >= 0:
                busy[u.device] += int(load[u.model, u.device])
        assert mk >= max(busy.values()) - a0


# ---------------------------------------------------------------------------
# P7 metamorphic relations
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(20))
def test_prefetch_never_hurts(seed):
    rng = np.random.default_rng(300 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(1, 4)), nodes=(2, 7), n_dev=2, n_models=4,
                          cap_range=(8000, 25000))
    plans = W.random_plans(win, 16, rng, p_prefetch=0.0)
    fuse, pf = W.unpack_flags(plans.flags, win.n_act)
    plans_pf = W.PlanBatch(plans.dev, plans.prio, W.pack_flags(fuse, np.ones_like(pf)))
    a, (sa, fa, _, pa) = oracle.score(win, plans, schedule=True)
    b, (sb, fb, _, pb) = oracle.score(win, plans_pf, schedule=True)
    ok = a["status"] & 1 == 0
    assert (a["status"] == b["status"]).all()
    assert (sb[ok] <= sa[ok]).all() and (fb[ok] <= fa[ok]).all()
    assert (b["makespan_us"][ok] <= a["makespan_us"][ok]).all()
    # lifecycle decisions do not depend on time
    for k in ("n_loads", "n_evicts", "min_headroom_mib"):
        assert (a[k][ok] == b[k][ok]).all()
    assert (pa[ok] == pb[ok]).all()


@pytest.mark.parametrize("seed", range(20))
def test_shorter_costs_never_hurt(seed):
    rng = np.random.default_rng(400 + seed)
    win = W.random_window(rng, n_wf=3, nodes=(2, 6), n_dev=2, n_models=4, cap_range=(8000, 25000))
    plans = W.random_plans(win, 16, rng)
    faster = W.Window(**{**win.arrays()})
    lat = win.lat_us.copy()
    pos = lat >= 0
    lat[pos] = lat[pos] - rng.integers(0, 1, size=pos.sum(), endpoint=True) * (lat[pos] // 2)
    faster.lat_us = lat
    faster.load_us = win.load_us - rng.integers(0, 2, size=win.load_us.shape) * (win.load_us // 3)
    a, (_, fa, _, _) = oracle.score(win, plans, schedule=True)
    b, (_, fb, _, _) = oracle.score(faster, plans, schedule=True)
    ok = a["status"] & 1 == 0
    assert (fb[ok] <= fa[ok]).all()


@pytest.mark.parametrize("seed", range(15))
def test_time_shift_and_relabel(seed):
    rng = np.random.default_rng(500 + seed)
    win = W.random_window(rng, n_wf=3, nodes=(1, 6), n_dev=3, n_models=4)
    plans = W.random_plans(win, 16, rng)
    a, (sa, fa, la, _) = oracle.score(win, plans, schedule=True)
    delta = int(rng.integers(1, 10 ** 9))
    shifted = W.Window(**{**win.arrays()})
    shifted.wf_arrival_us = win.wf_arrival_us + delta
    shifted.dev_free0_us = win.dev_free0_us + delta
    b, (sb, fb, lb, _) = oracle.score(shifted, plans, schedule=True)
    ok = a["status"] & 1 == 0
    assert (sb[ok] == sa[ok] + delta).all() and (fb[ok] == fa[ok] + delta).all()
    assert (np.where(la[ok] >= 0, la[ok] + delta, -1) == lb[ok]).all()
    for k in ("makespan_us", "p95_us", "objective", "status", "n_loads", "n_evicts"):
        assert (a[k] == b[k]).all()
    # relabel workflows with a permutation: nothing changes
    perm = rng.permutation(win.n_wf)
    relab = W.Window(**{**win.arrays()})
    relab.act_wf = perm[win.act_wf].astype(np.int32)
    relab.wf_arrival_us = np.empty_like(win.wf_arrival_us)
    relab.wf_arrival_us[perm] = win.wf_arrival_us
    c, (sc_, fc, _, _) = oracle.score(relab, plans, schedule=True)
    assert (sc_[ok] == sa[ok]).all()
    for k in ("makespan_us", "p95_us", "objective", "status"):
        assert (a[k] == c[k]).all()


def test_objective_is_fp32_of_integer_outputs():
    rng = np.random.default_rng(7)
    win, plans = W.make_config(1, n_plans=64)
    sc = oracle.score(win, plans)
    mk = sc["makespan_us"].astype(np.float32)
    p95 = sc["p95_us"].astype(np.float32)
    want = np.float32(win.w_makespan) * mk + np.float32(win.w_p95) * p95
    assert (want.view(np.uint32) == sc["objective"].view(np.uint32)).all()
    assert (sc["p95_us"] <= sc["makespan_us"]).all()


def test_p95_nearest_rank_against_numpy():
    """p95 equals numpy's inverted-CDF percentile of per-workflow latency."""
    win, plans = W.make_config(2, n_plans=8)
    sc, (st, fi, _, _) = oracle.score(win, plans, schedule=True)
    for p in range(plans.n_plans):
        comp = [fi[p][win.act_wf == w].max() - win.wf_arrival_us[w] for w in range(win.n_wf)]
        assert sc["p95_us"][p] == int(np.percentile(comp, 95, method="inverted_cdf"))
        assert sc["makespan_us"][p] == fi[p].max() - win.wf_arrival_us.min()


def test_empty_window():
    win = W.Window(n_act=0, n_wf=0, n_models=1, n_dev=2, act_wf=np.zeros(0, np.int32),
                   act_model=np.zeros(0, np.int32), pred_off=np.zeros(1, np.int32),
                   pred_idx=np.zeros(0, np.int32), lat_us=np.zeros(0, np.int32),
                   mem_mib=np.zeros(0, np.int32), wf_arrival_us=np.zeros(0, np.int64),
                   dev_cap_mib=np.array([100, 50], np.int32), model_mib=np.array([30], np.int32),
                   load_us=np.zeros(2, np.int32), init_resident=np.array([1, 0], np.uint64),
                   dev_free0_us=np.zeros(2, np.int64))
    plans = W.PlanBatch(np.zeros((3, 0), np.int8), np.zeros((3, 0), np.uint16),
                        np.zeros((3, 0), np.uint8))
    sc = oracle.score(win, plans)
    assert (sc["makespan_us"] == 0).all() and (sc["status"] == 0).all()
    assert (sc["min_headroom_mib"] == 50).all()


@pytest.mark.parametrize("bad", ["pred_order", "not_level_sorted", "wf_range", "empty_wf"])
def test_oracle_rejects_invalid_windows(bad):
    rng = np.random.default_rng(11)
    win = W.random_window(rng, n_wf=2, nodes=(3, 5), n_dev=2, n_models=3, p_edge=1.0)
    w2 = W.Window(**{**win.arrays()})
    if bad == "pred_order":
        w2.pred_idx = win.pred_idx.copy()
        i = int(np.nonzero(np.diff(win.pred_off))[0][-1])
        w2.pred_idx[win.pred_off[i]] = i  # self-loop
    elif bad == "not_level_sorted":
        # move a source (level 0) after a level-1 activation by swapping rows
        w2.pred_off = np.zeros(win.n_act + 1, np.int32)
        w2.pred_off[2:] = 1
        w2.pred_idx = np.array([0], np.int32)  # activation 1 depends on 0, the rest are sources
    elif bad == "wf_range":
        w2.act_wf = win.act_wf.copy()
        w2.act_wf[0] = win.n_wf
    elif bad == "empty_wf":
        w2.n_wf = win.n_wf + 1
        w2.wf_arrival_us = np.concatenate([win.wf_arrival_us, [0]])
    plans = W.random_plans(w2, 2, rng)
    with pytest.raises(oracle.OracleError):
        oracle.score(w2, plans)


def test_p95_nearest_rank_many_workflow_counts():
    """Nearest-rank p95 for every workflow count 1..40 (the rank rule only
    shows on counts where 0.95 W has a small fractional part)."""
    for n_wf in range(1, 41):
        rng = np.random.default_rng(600 + n_wf)
        win = W.random_window(rng, n_wf=n_wf, nodes=(1, 2), n_dev=2, n_models=2)
        plans = W.random_plans(win, 3, rng, p_bad_dev=0.0)
        sc, (st, fi, _, _) = oracle.score(win, plans, schedule=True)
        for p in range(plans.n_plans):
            if sc["status"][p] & 1:
                continue
            comp = [fi[p][win.act_wf == w].max() - win.wf_arrival_us[w] for w in range(n_wf)]
            assert sc["p95_us"][p] == int(np.percentile(comp, 95, method="inverted_cdf")), n_wf


@pytest.mark.parametrize("slack", [-1, 0, 1])
def test_exact_fit_boundary(slack):
    """Eq. 11 admits memory equal to capacity.  One device, model A resident,
    one activation of model B with weights W_B and memory m: it fits beside A
    iff W_A + W_B + m <= cap; otherwise A is reclaimed; if B alone does not
    fit (W_B + m > cap) the plan is over capacity."""
    WA, WB, m = 5000, 7000, 1000
    for case in ("beside", "alone"):
        cap = (WA + WB + m + slack) if case == "beside" else (WB + m + slack)
        win, _ = _window(1, [[[]]], [1], 1, lat=[[100]], mem=[[m]], cap=[cap],
                         weights=[WA, WB], load=[[10], [20]], resident=[1 if WA <= cap else 0])
        plans = W.PlanBatch(np.zeros((1, 1), np.int8), np.zeros((1, 1), np.uint16),
                            np.zeros((1, 1), np.uint8))
        sc = oracle.score(win, plans)[0]
        if case == "beside":
            assert sc["n_evicts"] == (1 if slack < 0 else 0)
            assert sc["status"] == 0
            assert sc["min_headroom_mib"] == (cap - WB - m if slack < 0 else slack)
        else:
            assert sc["status"] == (2 if slack < 0 else 0)
            assert sc["min_headroom_mib"] == slack

"""Pins of the oracle's rule-guided candidate generator (Algorithm 1 and
Sec. 3.5: BestFeasibleBinding and PlanPrefetch as mutation kinds 0 and 3):

* a worked example derived by hand (tests/golden/search_rules.json):
  resident reuse ahead of a faster non-resident device, the fastest of two
  resident replicas, loads ranked by unlocked ready work per load time, a
  free load, equal values broken by run time, earliest releases and the
  prefetch threshold with the dispatch slack;
* a second formulation in Python (exact rational comparisons, the
  earliest release as a longest path over a networkx DAG) and a Python
  replay of whole mutation sequences on random windows;
* kinds 1 and 2 are the uniform mode's, the unknown mode is refused.
"""
from fractions import Fraction

import networkx as nx
import numpy as np
import pytest

import oracle
from fixtures import load_golden
from paper_2609_03335_amd import workload as W
from test_oracle_search import _levels, py_philox

RULES = oracle.SEARCH_RULES
M32 = 0xFFFFFFFF


def second_formulation(win):
    """Best binding, earliest release and readiness of every activation."""
    N, D, M = win.n_act, win.n_dev, win.n_models
    lat = np.asarray(win.lat_us).reshape(N, D)
    load = np.asarray(win.load_us).reshape(M, D)
    arr = np.asarray(win.wf_arrival_us)
    ready = [len(win.preds(i)) == 0 and arr[win.act_wf[i]] <= 0 for i in range(N)]
    unlock = {(m, d): sum(int(lat[i, d]) for i in range(N)
                          if ready[i] and win.act_model[i] == m and lat[i, d] >= 0)
              for m in range(M) for d in range(D)}
    best = []
    for i in range(N):
        m = int(win.act_model[i])
        elig = [d for d in range(D) if lat[i, d] >= 0]
        res = [d for d in elig if (int(win.init_resident[d]) >> m) & 1]
        if not elig:
            best.append(-1)
        elif res:
            best.append(min(res, key=lambda d: (lat[i, d], d)))
        else:
            # a free load outranks every finite value
            def value(d):
                if load[m, d] == 0:
                    return (1, Fraction(0))
                return (0, Fraction(unlock[(m, d)], int(load[m, d])))
            top = max(value(d) for d in elig)
            best.append(min((d for d in elig if value(d) == top), key=lambda d: (lat[i, d], d)))
    # earliest release: the longest path from the origin, an activation's
    # own edge weighing its fastest run
    g = nx.DiGraph()
    for i in range(N):
        g.add_edge("origin", ("start", i), weight=int(arr[win.act_wf[i]]))
        fast = min([int(x) for x in lat[i] if x >= 0], default=0)
        g.add_edge(("start", i), ("end", i), weight=fast)
        for p in win.preds(i):
            g.add_edge(("end", int(p)), ("start", i), weight=0)
    dist = {"origin": 0}
    for v in nx.topological_sort(g):
        for _, w, a in g.out_edges(v, data=True):
            dist[w] = max(dist.get(w, -1), dist[v] + a["weight"])
    rel = [dist[("start", i)] for i in range(N)]
    return best, rel, ready


def replay(win, d, p, f, seed, n_mut, first, count, tables):
    """Whole candidates, mutation after mutation, from the Python Philox."""
    best, rel, ready = tables
    N, D = win.n_act, win.n_dev
    lat = np.asarray(win.lat_us).reshape(N, D)
    load = np.asarray(win.load_us).reshape(win.n_models, D)
    lv = _levels(win)
    out = []
    for k in range(count):
        c = first + k
        ed, ep, ef = d.copy(), p.copy(), f.copy()
        for t in range(n_mut):
            r0, r1, r2, _ = py_philox((c & M32, c >> 32, t, 0), (seed & M32, seed >> 32))
            i, kind = (r1 * N) >> 32, r0 >> 30
            if kind == 0:
                if best[i] >= 0:
                    ed[i] = best[i]
            elif kind == 1:
                same = np.nonzero(lv == lv[i])[0]
                j = int(same[0]) + ((r2 * len(same)) >> 32)
                ep[i], ep[j] = ep[j], ep[i]
            elif kind == 2:
                ef[i // 4] ^= 1 << (2 * (i % 4))
            elif 0 <= ed[i] < D:
                bit = 1 << (2 * (i % 4) + 1)
                on = (not ready[i]) and rel[i] <= int(load[win.act_model[i], ed[i]]) + win.prefetch_slack_us
                ef[i // 4] = (int(ef[i // 4]) | bit) if on else (int(ef[i // 4]) & (0xFF ^ bit))
        out.append((ed, ep, ef))
    return out


def check(win, d, p, f, seed, n_mut, first, count, tables):
    cd, cp, cf = oracle.search_candidates(win, d, p, f, seed, n_mut, first, count, mode=RULES)
    for k, (ed, ep, ef) in enumerate(replay(win, d, p, f, seed, n_mut, first, count, tables)):
        assert (cd[k] == ed).all() and (cp[k] == ep).all() and (cf[k] == ef).all(), k


def test_worked_example():
    win, plans, ix, spec = load_golden("search_rules")
    assert win.prefetch_slack_us == 30
    devs = [x["name"] for x in spec["devices"]]
    names = sorted(ix, key=ix.get)
    best = [devs.index(spec["expect_binding"][nm]) for nm in names]
    inc = plans["incumbent"]
    d, p, f = inc.dev[0], inc.prio[0], inc.flags[0]
    N = win.n_act
    seed, count = 0xC0FFEE, 400
    cd, cp, cf = oracle.search_candidates(win, d, p, f, seed, 1, 0, count, mode=RULES)
    _, pf0 = W.unpack_flags(f[None, :], N)
    kinds = set()
    for c in range(count):
        r0, r1, _, _ = py_philox((c, 0, 0, 0), (seed & M32, seed >> 32))
        i, kind = (r1 * N) >> 32, r0 >> 30
        kinds.add(kind)
        if kind == 0:
            want = d.copy()
            want[i] = best[i]
            assert (cd[c] == want).all() and (cf[c] == f).all(), names[i]
        elif kind == 3:
            _, pf = W.unpack_flags(cf[c:c + 1], N)
            want = pf0[0].copy()
            want[i] = bool(spec["expect_prefetch"][names[i]])
            assert (pf[0] == want).all() and (cd[c] == d).all(), names[i]
    assert kinds == {0, 1, 2, 3}
    # the second formulation agrees with the hand derivation
    b2, rel, ready = second_formulation(win)
    assert b2 == best
    assert [rel[ix[n]] for n in ("W0.d", "W0.e", "W1.f")] == [40, 65, 500]
    assert [ready[ix[n]] for n in names] == [n in ("W0.a", "W0.b", "W0.c") for n in names]


@pytest.mark.parametrize("seed", range(8))
def test_against_second_formulation(seed):
    rng = np.random.default_rng(3100 + seed)
    win = W.random_window(rng, n_wf=int(rng.integers(2, 6)), nodes=(2, 8), n_dev=int(rng.integers(2, 7)),
                          n_models=int(rng.integers(1, 6)))
    # a few free loads, some residency and a slack of either size
    load = np.asarray(win.load_us).copy()
    load[rng.random(load.size) < 0.15] = 0
    win.load_us = load.astype(np.int32)
    win.init_resident = rng.integers(0, 1 << win.n_models, win.n_dev).astype(np.uint64) & np.uint64(
        rng.integers(0, 2) * ((1 << win.n_models) - 1))
    win.prefetch_slack_us = int(rng.integers(0, 2000))
    plans = W.random_plans(win, 1, rng, prio_mode="perm")
    tables = second_formulation(win)
    d, p, f = plans.dev[0], plans.prio[0], plans.flags[0]
    check(win, d, p, f, 0x5EED + seed, 1, 0, 40 * win.n_act, tables)
    check(win, d, p, f, 0xABC + seed, 7, 1 << 33, 200, tables)


def test_config_windows():
    for cfg in (0, 1):
        win, plans = W.make_config(cfg, n_plans=1)
        win.prefetch_slack_us = 500
        tables = second_formulation(win)
        check(win, plans.dev[0], plans.prio[0], plans.flags[0], 77, 5, 10, 50, tables)


def test_uniform_kinds_unchanged_and_zero_mutations():
    win, plans = W.make_config(1, n_plans=1)
    d, p, f = plans.dev[0], plans.prio[0], plans.flags[0]
    cd, cp, cf = oracle.search_candidates(win, d, p, f, 3, 0, 0, 5, mode=RULES)
    assert (cd == d).all() and (cp == p).all() and (cf == f).all()
    rd, rp, rf = oracle.search_candidates(win, d, p, f, 21, 1, 0, 300, mode=RULES)
    ud, up, uf = oracle.search_candidates(win, d, p, f, 21, 1, 0, 300)
    N = win.n_act
    for c in range(300):
        r0, _, _, _ = py_philox((c, 0, 0, 0), (21, 0))
        if (r0 >> 30) in (1, 2):
            assert (rd[c] == ud[c]).all() and (rp[c] == up[c]).all() and (rf[c] == uf[c]).all()
    assert N > 0


def test_unknown_mode_refused():
    win, plans = W.make_config(0, n_plans=1)
    with pytest.raises(oracle.OracleError):
        oracle.search_candidates(win, plans.dev[0], plans.prio[0], plans.flags[0], 1, 1, 0, 1, mode=2)

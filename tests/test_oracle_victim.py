"""Pins of the oracle's paper victim order (Sec. 3.5, reclamation: copies
held on another device first, then the largest ratio of next-use distance to
reload time, then least recently used).

* Worked examples (tests/golden/victim_order*.json), each derived by hand in
  the fixture: a choice decided by redundancy, one decided by the ratio of
  next-use distance to reload cost against the least-recently-used order,
  and one where the level-start snapshot of the pool differs from the live
  residency.
* Belady's theorem: on one device with equal model sizes, equal load times
  and a capacity of k models, preferring the copy whose next use is farthest
  (no next use = infinitely far) minimises the number of loads (Belady,
  IBM Systems Journal 1966).  The oracle's load count under the paper order
  must equal the minimum found by exhaustive search over every eviction
  choice, and never exceed the default order's count.
"""
import functools

import numpy as np
import pytest

import oracle
from fixtures import load_golden
from paper_2609_03335_amd import workload as W


@pytest.mark.parametrize("name", ["victim_order", "victim_order_chain", "victim_order_snapshot",
                                  "victim_order_ties"])
def test_worked_examples(name):
    win, plans, ix, spec = load_golden(name)
    inv = {i: n for n, i in ix.items()}
    for pname, exp in spec["expect_loads"].items():
        for order, key in ((oracle.VICTIM_PAPER, "paper"), (oracle.VICTIM_REMAINING_LRU, "default")):
            win.victim_order = order
            sc, (st, fi, ls, pk) = oracle.score(win, plans[pname], schedule=True)
            loads = sorted(inv[i] for i in range(win.n_act) if ls[0, i] >= 0)
            assert loads == sorted(exp[key]), (name, pname, key)
            assert sc["status"][0] == 0


def test_unknown_victim_order_is_rejected():
    win, plans, ix, spec = load_golden("victim_order")
    win.victim_order = 2
    with pytest.raises(oracle.OracleError):
        oracle.score(win, plans["redundancy"])


def _chain_window(seq, k, n_models, init, load_us=500):
    """One device holding k models of 10 MiB; a single workflow whose
    activations form a chain using models seq[0], seq[1], ... in order."""
    T = len(seq)
    return W.Window(
        n_act=T, n_wf=1, n_models=n_models, n_dev=1,
        act_wf=np.zeros(T, np.int32), act_model=np.asarray(seq, np.int32),
        pred_off=np.concatenate([[0], np.arange(T)]).astype(np.int32),
        pred_idx=np.arange(max(T - 1, 0), dtype=np.int32),
        lat_us=np.full(T, 7, np.int32), mem_mib=np.zeros(T, np.int32),
        wf_arrival_us=np.zeros(1, np.int64), dev_cap_mib=np.array([10 * k], np.int32),
        model_mib=np.full(n_models, 10, np.int32), load_us=np.full(n_models, load_us, np.int32),
        init_resident=np.array([sum(1 << m for m in init)], np.uint64),
        dev_free0_us=np.zeros(1, np.int64), name="chain")


def _min_loads(seq, k, init):
    """Fewest loads over every choice of victim (exhaustive, memoised)."""
    @functools.lru_cache(maxsize=None)
    def go(i, cache):
        if i == len(seq):
            return 0
        m = seq[i]
        if m in cache:
            return go(i + 1, cache)
        if len(cache) < k:
            return 1 + go(i + 1, cache | frozenset([m]))
        return 1 + min(go(i + 1, (cache - frozenset([v])) | frozenset([m])) for v in cache)
    return go(0, frozenset(init))


@pytest.mark.parametrize("seed", range(40))
def test_paper_order_is_belady_optimal_on_one_device(seed):
    rng = np.random.default_rng(90_000 + seed)
    n_models = int(rng.integers(2, 6))
    k = int(rng.integers(1, n_models))
    T = int(rng.integers(2, 13))
    seq = [int(x) for x in rng.integers(0, n_models, T)]
    init = [int(x) for x in rng.choice(n_models, size=int(rng.integers(0, k + 1)), replace=False)]
    win = _chain_window(seq, k, n_models, init)
    plan = W.PlanBatch(np.zeros((1, T), np.int8), np.zeros((1, T), np.uint16),
                       np.zeros((1, (T + 3) // 4), np.uint8))
    win.victim_order = oracle.VICTIM_PAPER
    paper = int(oracle.score(win, plan)["n_loads"][0])
    win.victim_order = oracle.VICTIM_REMAINING_LRU
    default = int(oracle.score(win, plan)["n_loads"][0])
    best = _min_loads(tuple(seq), k, tuple(sorted(init)))
    assert paper == best, (seq, k, init, paper, best)
    assert default >= best


@pytest.mark.parametrize("seed", range(6))
def test_paper_order_keeps_the_timeline_invariants(seed):
    """The victim order changes only which copy goes: every unit still runs
    after its release and after its load, and every reclaimed copy had been
    resident."""
    rng = np.random.default_rng(91_000 + seed)
    win = W.random_window(rng, n_wf=4, nodes=(2, 8), n_dev=3, n_models=6,
                          cap_range=(9000, 16000), w_range=(3000, 8000), mem_range=(0, 1500))
    win.victim_order = oracle.VICTIM_PAPER
    plans = W.random_plans(win, 100, rng, prio_mode="perm")
    sc, (st, fi, ls, pk) = oracle.score(win, plans, schedule=True)
    n_init = sum(bin(int(r)).count("1") for r in win.init_resident)
    load = win.load_us.reshape(win.n_models, win.n_dev)
    for p in range(plans.n_plans):
        if sc["status"][p] & oracle.INELIGIBLE:
            continue
        for v in range(win.n_act):
            for u in win.pred_idx[win.pred_off[v]:win.pred_off[v + 1]]:
                assert st[p, v] >= fi[p, u]
            assert st[p, v] >= win.wf_arrival_us[win.act_wf[v]]
            if ls[p, v] >= 0:
                assert ls[p, v] + load[win.act_model[v], plans.dev[p, v]] <= st[p, v]
        # every reclaimed copy was resident first: loaded, or in the snapshot
        assert sc["n_evicts"][p] <= sc["n_loads"][p] + n_init

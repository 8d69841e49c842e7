"""The paper's two worked examples (tests/golden/*.json, cited there):
shared lifecycle actions across workflows (Fig. 4) and the fused QMSum
aggregation chain (Eq. 3, Eq. 4).  Structural claims come from the paper;
the timelines are derived here in closed form from the fixture's numbers."""
import numpy as np

import oracle
from fixtures import load_golden


def _loads(win, plans, sched, model_names, dev=None):
    st, fi, ls, pk = sched
    counts = {}
    for i in np.nonzero(ls[0] >= 0)[0]:
        if dev is not None and plans.dev[0, i] != dev:
            continue
        m = model_names[win.act_model[i]]
        counts[m] = counts.get(m, 0) + 1
    return counts


def test_fig4_one_load_one_prefetch_shared_by_two_workflows():
    win, plans, ix, spec = load_golden("fig4_shared_lifecycle")
    models = [m["name"] for m in spec["models"]]
    L8, L14 = 5000, 8000            # load_us of Q8 / Q14 in the fixture
    Ta, Tb = 300, 400               # run times of the Q8 / Q14 activations
    for pname, exp in spec["expect"].items():
        sc, sched = oracle.score(win, plans[pname], schedule=True)
        st, fi, ls, pk = sched
        assert _loads(win, plans[pname], sched, models) == exp["loads_per_model"]
        assert int(sc["n_evicts"][0]) == exp["evictions"]
        assert (sc["status"][0] == 0) == exp["feasible"]
        # the Q8 load serves both ready units: W1.q8 loads, W2.q8 reuses it
        assert ls[0, ix["W1.q8"]] == 0 and ls[0, ix["W2.q8"]] == -1
        assert fi[0, ix["W1.q8"]] == L8 + Ta and fi[0, ix["W2.q8"]] == L8 + 2 * Ta
        # the Q14 action serves both near-ready units
        assert ls[0, ix["W2.q14"]] == -1
        if pname == "shared_prefetch":
            # prefetched: the load starts at the window time, overlapping Q8 work
            assert ls[0, ix["W1.q14"]] == 0
            b1 = max(L8 + Ta, L14) + Tb
        else:
            # plain load (alpha_F): waits until the unit is released
            assert ls[0, ix["W1.q14"]] == L8 + Ta
            b1 = L8 + Ta + L14 + Tb
        assert fi[0, ix["W1.q14"]] == b1
        assert fi[0, ix["W2.q14"]] == max(L8 + 2 * Ta, b1) + Tb
        assert sc["makespan_us"][0] == max(L8 + 2 * Ta, b1) + Tb
    a = oracle.score(win, plans["shared_prefetch"])
    b = oracle.score(win, plans["shared_load_only"])
    assert a["makespan_us"][0] < b["makespan_us"][0]


def test_qmsum_fused_chain_one_grant_one_replica():
    win, plans, ix, spec = load_golden("qmsum_fused_chain")
    models = [m["name"] for m in spec["models"]]
    devs = [d["name"] for d in spec["devices"]]
    lat = win.lat_us.reshape(win.n_act, win.n_dev)
    g = [ix["QMSum.g1"], ix["QMSum.g2"], ix["QMSum.g3"]]
    a100 = devs.index("A100-40GB")
    res = {}
    for pname, exp in spec["expect"].items():
        sc, sched = oracle.score(win, plans[pname], schedule=True)
        st, fi, ls, pk = sched
        res[pname] = (sc, st, fi, ls)
        assert (sc["status"][0] == 0) == exp["feasible"]
        for dname, per_model in exp["loads_per_model_on"].items():
            got = _loads(win, plans[pname], sched, models, dev=devs.index(dname))
            for m, k in per_model.items():
                assert got.get(m, 0) == k, (pname, m, got)
    sc, st, fi, ls = res["fused"]
    # one grant: members start exactly when the previous member finishes,
    # so the unit's run time is the sum of the members' (Eq. 4)
    assert st[0, g[1]] == fi[0, g[0]] and st[0, g[2]] == fi[0, g[1]]
    assert fi[0, g[2]] - st[0, g[0]] == int(lat[g, a100].sum())
    assert ls[0, g[1]] == -1 and ls[0, g[2]] == -1
    # the competitor runs after the whole chain on the shared device
    x5 = ix["Other.x5"]
    assert ls[0, x5] >= fi[0, g[2]]
    # unfused: the competitor is placed between g1 and g2 and forces a reload
    usc, ust, ufi, uls = res["unfused"]
    assert uls[0, x5] >= ufi[0, g[0]] and ust[0, g[1]] > ufi[0, x5] - 1
    assert uls[0, g[1]] >= ufi[0, x5]
    assert usc["n_loads"][0] == sc["n_loads"][0] + 1
    assert fi[0, g[2]] < ufi[0, g[2]]

"""Exhaustive plan enumeration on tiny windows: every within-level order (as
priorities), every eligible placement, every subset of fuse bits on fusible
activations and every subset of prefetch bits."""
import itertools

import numpy as np

from paper_2609_03335_amd import workload as W
import pins


def enumerate_plans(win, limit=200000):
    n, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(n, D)
    lv = pins.nx_levels(win)
    levels = [list(np.nonzero(lv == k)[0]) for k in range(int(lv.max()) + 1)] if n else []
    orders = [list(itertools.permutations(range(len(L)))) for L in levels]
    elig = [list(np.nonzero(lat[i] >= 0)[0]) for i in range(n)]
    fus = sorted(pins.fusible_set(win))
    rows_dev, rows_prio, rows_fuse, rows_pf = [], [], [], []
    for perm_choice in itertools.product(*orders):
        prio = np.zeros(n, np.uint16)
        for L, perm in zip(levels, perm_choice):
            for rank, j in enumerate(perm):
                prio[L[j]] = rank
        for devs in itertools.product(*elig):
            for fbits in itertools.product((0, 1), repeat=len(fus)):
                fuse = np.zeros(n, bool)
                fuse[fus] = np.array(fbits, bool) if fus else fuse[fus]
                for pbits in itertools.product((0, 1), repeat=n):
                    rows_dev.append(devs)
                    rows_prio.append(prio)
                    rows_fuse.append(fuse)
                    rows_pf.append(pbits)
                    if len(rows_dev) > limit:
                        raise ValueError("too many plans")
    return W.PlanBatch(np.asarray(rows_dev, np.int8).reshape(-1, n),
                       np.asarray(rows_prio, np.uint16).reshape(-1, n),
                       W.pack_flags(np.asarray(rows_fuse, bool).reshape(-1, n),
                                    np.asarray(rows_pf, bool).reshape(-1, n)))


def best_plan(scores):
    """Feasible plan with the smallest objective, lowest index on ties;
    -1 when no plan is feasible."""
    ok = np.nonzero(scores["status"] == 0)[0]
    if len(ok) == 0:
        return -1
    obj = scores["objective"][ok]
    return int(ok[np.argmin(obj)])  # argmin returns the first minimum


def tiny_window(seed, n_nodes=(4, 5)):
    rng = np.random.default_rng(seed)
    while True:
        win = W.random_window(rng, n_wf=2, nodes=(2, 3), n_dev=2, n_models=3,
                              cap_range=(6000, 20000), same_model_bias=0.7, name=f"tiny{seed}")
        if n_nodes[0] <= win.n_act <= n_nodes[1]:
            return win

"""Pins of the oracle's candidate generator (candidates around an incumbent
plan, drawn with Philox4x32-10).

* The generator itself: the published known-answer vectors of
  Philox4x32-10 (Salmon et al., SC'11), for the oracle's C implementation
  and for a separate Python implementation used below.
* The mapping from draws to mutations: a candidate with one mutation is
  decoded here from the Python Philox and checked site by site.
* Structure every candidate must have whatever the draws: priorities stay a
  permutation of the incumbent's inside each level, re-placed devices are
  eligible, at most one site changes per mutation, n_mut = 0 gives the
  incumbent, candidates do not depend on how a range is split, and the four
  kinds and the activations are drawn about uniformly.
"""
import numpy as np
import pytest

import oracle
from paper_2609_03335_amd import workload as W

KAT = [  # (counter, key, output) of Philox4x32-10
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]
M32 = (1 << 32) - 1


def py_philox(ctr, key):
    """Philox4x32-10 in plain Python integers."""
    x = list(ctr)
    k0, k1 = key
    for _ in range(10):
        a = 0xD2511F53 * x[0]
        b = 0xCD9E8D57 * x[2]
        x = [((b >> 32) ^ x[1] ^ k0) & M32, b & M32, ((a >> 32) ^ x[3] ^ k1) & M32, a & M32]
        k0 = (k0 + 0x9E3779B9) & M32
        k1 = (k1 + 0xBB67AE85) & M32
    return tuple(x)


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    assert tuple(int(v) for v in oracle.philox4x32_10(ctr, key)) == want
    assert py_philox(ctr, key) == want


def _incumbent(cfg=1, seed=0):
    win, plans = W.make_config(cfg, n_plans=4)
    return win, plans.dev[seed], plans.prio[seed], plans.flags[seed]


def _levels(win):
    lv = oracle.levels(win)
    return lv


def test_zero_mutations_give_the_incumbent():
    win, d, p, f = _incumbent()
    cd, cp, cf = oracle.search_candidates(win, d, p, f, seed=7, n_mut=0, first=0, count=20)
    assert (cd == d).all() and (cp == p).all() and (cf == f).all()


def test_ranges_are_independent_of_splitting():
    win, d, p, f = _incumbent()
    seed = (0x1234 << 32) | 0x9876
    whole = oracle.search_candidates(win, d, p, f, seed, 3, first=(1 << 32) - 5, count=40)
    a = oracle.search_candidates(win, d, p, f, seed, 3, first=(1 << 32) - 5, count=13)
    b = oracle.search_candidates(win, d, p, f, seed, 3, first=(1 << 32) + 8, count=27)
    for x, y, z in zip(whole, a, b):
        assert (x == np.concatenate([y, z])).all()


def test_one_mutation_decoded_site_by_site():
    win, d, p, f = _incumbent()
    N, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(N, D)
    lv = _levels(win)
    seed = 0xDEADBEEF12345678
    cd, cp, cf = oracle.search_candidates(win, d, p, f, seed, 1, first=1000, count=400)
    kinds = set()
    for k in range(400):
        c = 1000 + k
        r0, r1, r2, _ = py_philox((c & M32, c >> 32, 0, 0), (seed & M32, seed >> 32))
        i = (r1 * N) >> 32
        kind = r0 >> 30
        kinds.add(kind)
        ed, ep, ef = d.copy(), p.copy(), f.copy()
        if kind == 0:
            elig = np.nonzero(lat[i] >= 0)[0]
            ed[i] = elig[(r2 * len(elig)) >> 32]
        elif kind == 1:
            same = np.nonzero(lv == lv[i])[0]
            lo, w = int(same[0]), len(same)
            j = lo + ((r2 * w) >> 32)
            ep[i], ep[j] = p[j], p[i]
        elif kind == 2:
            ef[i // 4] ^= 1 << (2 * (i % 4))
        else:
            ef[i // 4] ^= 1 << (2 * (i % 4) + 1)
        assert (cd[k] == ed).all() and (cp[k] == ep).all() and (cf[k] == ef).all(), (c, kind, i)
    assert kinds == {0, 1, 2, 3}


@pytest.mark.parametrize("n_mut", [1, 4, 17])
def test_candidate_structure(n_mut):
    rng = np.random.default_rng(n_mut)
    win = W.random_window(rng, n_wf=3, nodes=(4, 12), n_dev=4, n_models=5)
    plans = W.random_plans(win, 1, rng, prio_mode="perm")
    d, p, f = plans.dev[0], plans.prio[0], plans.flags[0]
    N, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(N, D)
    lv = _levels(win)
    cd, cp, cf = oracle.search_candidates(win, d, p, f, 99, n_mut, first=0, count=300)
    fu0, pf0 = W.unpack_flags(f[None, :], N)
    fu, pf = W.unpack_flags(cf, N)
    for k in range(300):
        moved = np.nonzero(cd[k] != d)[0]
        assert (lat[moved, cd[k][moved]] >= 0).all()  # re-placed devices are eligible
        for l in np.unique(lv):  # priorities permuted inside each level only
            idx = lv == l
            assert sorted(cp[k][idx]) == sorted(p[idx])
        flips = int((fu[k] != fu0[0]).sum() + (pf[k] != pf0[0]).sum())
        swapped = int((cp[k] != p).sum())
        # each mutation changes one device, two priorities or one bit
        assert len(moved) + flips + (swapped + 1) // 2 <= n_mut


def test_kinds_and_sites_about_uniform():
    win, d, p, f = _incumbent(cfg=4)
    N = win.n_act
    seed = 5
    counts = np.zeros(4)
    sites = np.zeros(N)
    for c in range(20000):
        r0, r1, _, _ = py_philox((c, 0, 0, 0), (seed, 0))
        counts[r0 >> 30] += 1
        sites[(r1 * N) >> 32] += 1
    assert (np.abs(counts / 20000 - 0.25) < 0.02).all()
    assert sites.min() > 0 and sites.max() < 3 * 20000 / N


def test_empty_window_candidates():
    win = W.random_window(np.random.default_rng(0), n_wf=1, nodes=(1, 1))
    win = W.Window(**{**win.arrays(), "n_act": 0, "n_wf": 0, "act_wf": np.zeros(0, np.int32),
                      "act_model": np.zeros(0, np.int32), "pred_off": np.zeros(1, np.int32),
                      "pred_idx": np.zeros(0, np.int32), "lat_us": np.zeros(0, np.int32),
                      "mem_mib": np.zeros(0, np.int32), "wf_arrival_us": np.zeros(0, np.int64)})
    cd, cp, cf = oracle.search_candidates(win, np.zeros(0, np.int8), np.zeros(0, np.uint16),
                                          np.zeros(0, np.uint8), 3, 5, first=0, count=4)
    assert cd.shape == (4, 0) and cp.shape == (4, 0) and cf.shape == (4, 0)

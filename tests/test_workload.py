"""The seeded input generator: determinism, sizes and input-layout rules."""
import numpy as np
import pytest

from paper_2609_03335_amd import workload as W
import pins

SIZES = {  # N, W, M, D, P
    0: (16, 2, 4, 3, 512),
    1: (400, 30, 16, 8, 16384),
    2: (1024, 64, 32, 12, 65536),
    3: (4096, 1, 24, 16, 8192),
    4: (256, 16, 16, 8, 1048576),
}


@pytest.mark.parametrize("cfg", range(5))
def test_window_shapes_and_layout(cfg):
    win = W.make_window(cfg)
    N, Wf, M, D, P = SIZES[cfg]
    assert (win.n_act, win.n_wf, win.n_models, win.n_dev) == (N, Wf, M, D)
    assert W.CONFIGS[cfg]["n_plans"] == P
    lv = pins.nx_levels(win)
    assert (np.diff(lv) >= 0).all(), "numbering must be level-sorted"
    lat = win.lat_us.reshape(N, D)
    assert ((lat >= 0).sum(axis=1) >= 1).all(), "every activation has an eligible device"
    assert (lat[lat >= 0] >= 1).all()
    mem = win.mem_mib.reshape(N, D)
    assert ((mem >= 1024) & (mem <= 8192)).all()
    assert (mem == mem[:, :1]).all(), "activation memory is broadcast over devices"
    # Eq. 8 first cut: an eligible entry fits weights plus activation memory
    need = win.model_mib[win.act_model][:, None] + mem
    assert (need[lat >= 0] <= np.broadcast_to(win.dev_cap_mib, (N, D))[lat >= 0]).all()
    for d in range(D):
        used = sum(int(win.model_mib[m]) for m in range(M) if (int(win.init_resident[d]) >> m) & 1)
        assert used <= win.dev_cap_mib[d]
    assert (win.wf_arrival_us >= 0).all()
    for w in range(Wf):
        assert (win.act_wf == w).any()
    for i in range(N):
        ps = win.preds(i)
        assert (ps < i).all() and (np.diff(ps) > 0).all()
        if len(ps):
            assert (win.act_wf[ps] == win.act_wf[i]).all(), "edges stay inside a workflow"


def test_config_specific_shapes():
    w1 = W.make_window(1)
    assert sum(bin(int(x)).count("1") for x in w1.init_resident) <= 5
    w2 = W.make_window(2)
    assert w2.wf_arrival_us[0] == 0 and (np.diff(w2.wf_arrival_us) >= 0).all()
    assert 0.5 * 63 * 50000 < w2.wf_arrival_us[-1] < 2 * 63 * 50000
    w3 = W.make_window(3)
    lv = pins.nx_levels(w3)
    assert lv.max() == 127 and (np.bincount(lv) == 32).all()
    w4 = W.make_window(4)
    assert (np.bincount(w4.act_wf) == 16).all()
    for cfg, w in ((1, w1), (2, w2), (3, w3)):
        assert list(w.dev_cap_mib[:3]) == [24576, 49152, 196608]
    assert list(w4.dev_cap_mib[:3]) == [24576, 49152, 81920]


def test_determinism():
    a_w, a_p = W.make_config(1, n_plans=256)
    b_w, b_p = W.make_config(1, n_plans=256)
    for k, v in a_w.arrays().items():
        assert np.array_equal(np.asarray(v), np.asarray(b_w.arrays()[k])), k
    assert np.array_equal(a_p.dev, b_p.dev) and np.array_equal(a_p.prio, b_p.prio)
    assert np.array_equal(a_p.flags, b_p.flags)


@pytest.mark.parametrize("cfg", [0, 1, 2, 4])
def test_plans_follow_the_recipe(cfg):
    win, plans = W.make_config(cfg, n_plans=512)
    N, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(N, D)
    assert plans.dev.shape == (512, N) and plans.flags.shape == (512, (N + 3) // 4)
    rows = np.arange(N)[None, :].repeat(512, 0)
    assert (lat[rows, plans.dev.astype(np.int64)] >= 0).all(), "placement on eligible devices"
    lv = pins.nx_levels(win)
    for lo in np.unique(lv):
        idx = np.nonzero(lv == lo)[0]
        seg = np.sort(plans.prio[:, idx].astype(np.int64), axis=1)
        assert (seg == idx[None, :]).all(), "a level-major permutation of priorities"
    fuse, pf = W.unpack_flags(plans.flags, N)
    assert 0.15 < pf.mean() < 0.25
    for v in np.nonzero(fuse.any(axis=0))[0]:
        (u,) = win.preds(v)
        assert win.act_model[u] == win.act_model[v]
        f = fuse[:, v]
        assert (plans.dev[f, v] == plans.dev[f, u]).all()


def test_flag_packing_roundtrip():
    rng = np.random.default_rng(0)
    for n in (1, 3, 4, 5, 17):
        f = rng.random((7, n)) < 0.5
        p = rng.random((7, n)) < 0.5
        packed = W.pack_flags(f, p)
        assert packed.shape == (7, (n + 3) // 4)
        f2, p2 = W.unpack_flags(packed, n)
        assert (f == f2).all() and (p == p2).all()
        # bit 2*(i%4) of byte i//4 is fuse, the next bit prefetch
        for i in range(n):
            assert ((packed[:, i // 4] >> (2 * (i % 4))) & 1 == f[:, i]).all()
            assert ((packed[:, i // 4] >> (2 * (i % 4) + 1)) & 1 == p[:, i]).all()


def test_npz_roundtrip(tmp_path):
    win, plans = W.make_config(0)
    W.save_npz(str(tmp_path / "c0.npz"), win, plans)
    w2, p2 = W.load_npz(str(tmp_path / "c0.npz"))
    assert w2.n_act == win.n_act and np.array_equal(p2.prio, plans.prio)
    assert np.array_equal(w2.lat_us, win.lat_us) and w2.name == win.name

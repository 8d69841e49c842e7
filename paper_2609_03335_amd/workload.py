"""Seeded synthetic scheduling windows and candidate-plan batches.

This module only *draws inputs*: workflow DAGs, predicted cost tables, pool
state and candidate plans.  It contains none of the scoring arithmetic
(fusion, ordering, lifecycle, timeline, reductions); both the GPU path and the
CPU oracle consume what it produces.

Shapes follow the paper's workloads: concurrent agent workflows sharing a
heterogeneous GPU pool (Sec. 2 and 4), burst or Poisson arrivals (Sec. 4,
arrival processes), model loads that dominate activation run time (Sec. 2,
Fig. 1), a device-specific latency/memory/load table per activation (Eq. 1)
with an eligibility cut (Eq. 8), and plans that pick a device, a priority, a
fusion bit (Eq. 3) and a prefetch bit (Eq. 5) per activation.

Inputs follow the library's window and plan layout:
  * activations are numbered in non-decreasing topological level;
  * tables are row-major: ``lat_us[i * D + d]``, ``load_us[m * D + d]``;
  * plans are row-major: ``dev[P][N]`` int8, ``prio[P][N]`` uint16,
    ``flags[P][ceil(N/4)]`` uint8 where activation ``i`` owns bit
    ``2*(i%4)`` (fuse) and ``2*(i%4)+1`` (prefetch) of byte ``i//4``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Window", "PlanBatch", "CONFIGS", "make_config", "make_window",
    "make_plans", "random_window", "random_deep_window", "random_plans", "pack_flags",
    "unpack_flags", "save_npz", "load_npz",
]

# --------------------------------------------------------------------------
# containers
# --------------------------------------------------------------------------


@dataclasses.dataclass
class Window:
    """A planning window: logical workflows, predicted costs, pool snapshot."""

    n_act: int
    n_wf: int
    n_models: int
    n_dev: int
    act_wf: np.ndarray          # int32[N]
    act_model: np.ndarray       # int32[N]
    pred_off: np.ndarray        # int32[N+1]  CSR of predecessors
    pred_idx: np.ndarray        # int32[nnz]  pred_idx[k] < i for row i
    lat_us: np.ndarray          # int32[N*D]  -1 = ineligible
    mem_mib: np.ndarray         # int32[N*D]
    wf_arrival_us: np.ndarray   # int64[W]
    dev_cap_mib: np.ndarray     # int32[D]
    model_mib: np.ndarray       # int32[M]
    load_us: np.ndarray         # int32[M*D]
    init_resident: np.ndarray   # uint64[D] bitmask over models
    dev_free0_us: np.ndarray    # int64[D]
    w_makespan: float = 1.0
    w_p95: float = 0.5
    name: str = "window"
    # uint8[W] priority class of each workflow for the ranking key of Eq. 12
    # (0 ranked first, below 4); None puts every workflow in class 0
    wf_class: Optional[np.ndarray] = None
    # reclamation victim order: 0 = no remaining use first, then least
    # recently used; 1 = the paper's (copies held on another device, then
    # next-use distance per reload time, then least recently used)
    victim_order: int = 0
    # int32[D] batch limit of each device (units it runs at once, 1..4);
    # None = 1 everywhere
    dev_batch: Optional[np.ndarray] = None
    # int32[M] replica cap of each model (copies held across the pool in one
    # topological level, Sec. 3.5 scale-out), >= 1; None = no cap
    model_replica_cap: Optional[np.ndarray] = None
    # dispatch slack of the rule-guided prefetch alternative (us, >= 0)
    prefetch_slack_us: int = 0

    def arrays(self):
        return {f.name: getattr(self, f.name) for f in dataclasses.fields(self)}

    @property
    def n_edges(self) -> int:
        return int(self.pred_off[-1]) if self.n_act else 0

    def preds(self, i: int) -> np.ndarray:
        return self.pred_idx[self.pred_off[i]:self.pred_off[i + 1]]


@dataclasses.dataclass
class PlanBatch:
    dev: np.ndarray    # int8[P][N]
    prio: np.ndarray   # uint16[P][N]
    flags: np.ndarray  # uint8[P][ceil(N/4)]

    @property
    def n_plans(self) -> int:
        return int(self.dev.shape[0])

    def slice(self, a: int, b: int) -> "PlanBatch":
        return PlanBatch(self.dev[a:b], self.prio[a:b], self.flags[a:b])

    def take(self, idx) -> "PlanBatch":
        idx = np.asarray(idx)
        return PlanBatch(self.dev[idx], self.prio[idx], self.flags[idx])


# --------------------------------------------------------------------------
# flag packing
# --------------------------------------------------------------------------


def pack_flags(fuse: np.ndarray, prefetch: np.ndarray) -> np.ndarray:
    """[P][N] bool x2 -> uint8[P][ceil(N/4)] (2 bits per activation)."""
    fuse = np.asarray(fuse, dtype=bool)
    prefetch = np.asarray(prefetch, dtype=bool)
    p, n = fuse.shape
    nb = (n + 3) // 4
    pad = nb * 4 - n
    if pad:
        z = np.zeros((p, pad), dtype=bool)
        fuse = np.concatenate([fuse, z], axis=1)
        prefetch = np.concatenate([prefetch, z], axis=1)
    out = np.zeros((p, nb), dtype=np.uint8)
    for j in range(4):
        out |= fuse[:, j::4].astype(np.uint8) << (2 * j)
        out |= prefetch[:, j::4].astype(np.uint8) << (2 * j + 1)
    return out


def unpack_flags(flags: np.ndarray, n: int) -> Tuple[np.ndarray, np.ndarray]:
    flags = np.asarray(flags, dtype=np.uint8)
    p = flags.shape[0]
    fuse = np.zeros((p, n), dtype=bool)
    pf = np.zeros((p, n), dtype=bool)
    for j in range(4):
        cols = np.arange(j, n, 4)
        fuse[:, cols] = (flags[:, cols // 4] >> (2 * j)) & 1
        pf[:, cols] = (flags[:, cols // 4] >> (2 * j + 1)) & 1
    return fuse, pf


# --------------------------------------------------------------------------
# helpers (graph construction only)
# --------------------------------------------------------------------------


def _depths(n: int, parents: Sequence[Sequence[int]], topo: Sequence[int]) -> np.ndarray:
    """Topological depth of each node, used only to number activations
    level-sorted as the input layout requires."""
    depth = np.zeros(n, dtype=np.int64)
    for v in topo:
        ps = parents[v]
        if ps:
            depth[v] = 1 + max(depth[u] for u in ps)
    return depth


class _Builder:
    """Accumulates workflows (local node ids, parent lists, models)."""

    def __init__(self):
        self.wf_nodes: List[int] = []     # number of nodes per workflow
        self.parents: List[List[int]] = []  # global ids (build order)
        self.models: List[int] = []
        self.wf_of: List[int] = []
        self.local: List[int] = []

    def add_workflow(self, parents_local: Sequence[Sequence[int]], models: Sequence[int]):
        base = len(self.parents)
        w = len(self.wf_nodes)
        self.wf_nodes.append(len(parents_local))
        for j, ps in enumerate(parents_local):
            self.parents.append([base + u for u in ps])
            self.models.append(int(models[j]))
            self.wf_of.append(w)
            self.local.append(j)

    def finish(self):
        """Renumber level-sorted (stable by level, workflow, local id)."""
        n = len(self.parents)
        # build order is topological inside each workflow (parents first)
        depth = _depths(n, self.parents, range(n))
        key = np.lexsort((np.array(self.local), np.array(self.wf_of), depth))
        new_of_old = np.empty(n, dtype=np.int64)
        new_of_old[key] = np.arange(n)
        pred_lists = []
        for new in range(n):
            old = key[new]
            pred_lists.append(sorted(int(new_of_old[u]) for u in self.parents[old]))
        act_wf = np.array([self.wf_of[k] for k in key], dtype=np.int32)
        act_model = np.array([self.models[k] for k in key], dtype=np.int32)
        off = np.zeros(n + 1, dtype=np.int32)
        off[1:] = np.cumsum([len(p) for p in pred_lists])
        idx = np.array([u for p in pred_lists for u in p], dtype=np.int32)
        return act_wf, act_model, off, idx, len(self.wf_nodes)


def _layered_parents(rng, layer_sizes, p_edge, span=1, force_parent=False):
    """Random layered DAG: each node may take a parent in the previous
    ``span`` layers with probability ``p_edge`` each."""
    starts = np.concatenate([[0], np.cumsum(layer_sizes)]).astype(int)
    parents = []
    for li, sz in enumerate(layer_sizes):
        for _ in range(sz):
            ps = []
            for back in range(1, span + 1):
                if li - back < 0:
                    continue
                lo, hi = starts[li - back], starts[li - back + 1]
                draw = rng.random(hi - lo) < p_edge
                ps.extend(int(lo + k) for k in np.nonzero(draw)[0])
            if force_parent and li > 0 and not any(starts[li - 1] <= u < starts[li] for u in ps):
                lo, hi = starts[li - 1], starts[li]
                ps.append(int(rng.integers(lo, hi)))
            parents.append(sorted(ps))
    return parents


def _even_layers(n, k):
    base, extra = divmod(n, k)
    return [base + (1 if i < extra else 0) for i in range(k)]


# scenario shapes (local parent lists, role of each node)
def _fanout_shape(width=8):
    parents = [[]] + [[0] for _ in range(width)] + [list(range(1, width + 1))]
    roles = [0] + [1] * width + [2]
    return parents, roles, 3


def _chain_shape(n_loops=2, extra_nodes=0):
    # plan, code, test, review, (code, test, review) * n_loops, repair, validate
    roles = [0, 1, 2, 3]
    for _ in range(n_loops):
        roles += [1, 2, 3]
    roles += [1, 2, 3][:extra_nodes]  # partially unrolled last loop
    roles += [4, 5]
    parents = [[]] + [[j - 1] for j in range(1, len(roles))]
    return parents, roles, 6


def _mapreduce_shape(width=16):
    parents = [[]] + [[0] for _ in range(width)] + [list(range(1, width + 1))]
    roles = [0] + [1] * width + [2]
    return parents, roles, 3


def _add_shape(b: _Builder, rng, shape, n_models):
    parents, roles, n_roles = shape
    role_model = rng.integers(0, n_models, size=n_roles)
    b.add_workflow(parents, [role_model[r] for r in roles])


# --------------------------------------------------------------------------
# the five benchmark configurations
# --------------------------------------------------------------------------

TIER_CAP_SMALL = (24576, 49152, 81920)     # MiB, configs 0 and 4
TIER_CAP_LARGE = (24576, 49152, 196608)    # MiB, configs 1-3
TIER_MULT_LARGE = (1.8, 1.3, 1.0)

CONFIGS = {
    0: dict(name="c0-tiny: 2 wf x 8 act, D=3, M=4, P=512", n_plans=512),
    1: dict(name="c1-mixed: 30 wf (fan-out/chain/map-reduce), N=400, D=8, M=16, P=16384", n_plans=16384),
    2: dict(name="c2-burst: 64 wf Poisson 50ms, N=1024, D=12, M=32, P=65536", n_plans=65536),
    3: dict(name="c3-deep: 1 wf 128x32 levels, N=4096, D=16, M=24, P=8192", n_plans=8192),
    4: dict(name="c4-stress: 16 wf x 16 act, N=256, D=8, M=16, P=1048576", n_plans=1048576),
}


def _tables(rng, act_model, n_dev, n_models, caps, mults, q_inel, w_hi):
    """Cost tables (Eq. 1) with the Eq. 8 eligibility cut applied."""
    n = len(act_model)
    raw = rng.lognormal(mean=math.log(2e5), sigma=0.6, size=(n, n_dev))
    raw = raw * np.asarray(mults, dtype=np.float64)[np.arange(n_dev) % 3][None, :]
    lat = np.maximum(np.rint(raw), 1).astype(np.int64)
    mem = rng.integers(1024, 8192, size=n, endpoint=True).astype(np.int64)
    weights = rng.integers(4096, w_hi, size=n_models, endpoint=True).astype(np.int64)
    u = rng.uniform(0.8, 1.2, size=(n_models, n_dev))
    load = np.rint(weights[:, None] * 2.0 ** 20 / (2e9 * u) * 1e6).astype(np.int64)
    cap = np.asarray([caps[d % 3] for d in range(n_dev)], dtype=np.int64)
    drop = rng.random((n, n_dev)) < q_inel
    too_big = (weights[act_model][:, None] + mem[:, None]) > cap[None, :]
    out = np.where(drop | too_big, -1, lat)
    big = int(np.argmax(cap))  # lowest index among the largest capacity
    empty = (out < 0).all(axis=1)
    out[empty, big] = lat[empty, big]
    mem_tab = np.repeat(mem[:, None], n_dev, axis=1)
    return (out.astype(np.int32).reshape(-1), mem_tab.astype(np.int32).reshape(-1),
            weights.astype(np.int32), load.astype(np.int32).reshape(-1), cap.astype(np.int32))


def _residency(rng, n_dev, n_models, weights, cap, frac):
    res = np.zeros(n_dev, dtype=np.uint64)
    if frac <= 0:
        return res
    k = int(round(frac * n_models))
    used = np.zeros(n_dev, dtype=np.int64)
    for m in rng.choice(n_models, size=k, replace=False):
        d = int(rng.integers(0, n_dev))
        if used[d] + weights[m] <= cap[d]:
            used[d] += weights[m]
            res[d] |= np.uint64(1) << np.uint64(int(m))
    return res


def make_window(cfg_id: int) -> Window:
    """The seeded window of one benchmark configuration."""
    root = np.random.SeedSequence(cfg_id)
    win_seed, _ = root.spawn(2)
    rng = np.random.default_rng(win_seed)
    b = _Builder()
    arrivals = None
    if cfg_id == 0:
        D, M, caps, mults, q, w_hi, frac = 3, 4, TIER_CAP_SMALL, (1.0, 1.0, 1.0), 0.10, 40960, 0.0
        for _ in range(2):
            par = _layered_parents(rng, _even_layers(8, 3), 0.4)
            b.add_workflow(par, rng.integers(0, M, size=8))
    elif cfg_id == 1:
        D, M, caps, mults, q, w_hi, frac = 8, 16, TIER_CAP_LARGE, TIER_MULT_LARGE, 0.10, 40960, 0.3
        for shape in (_fanout_shape(), _chain_shape(), _mapreduce_shape()):
            for _ in range(10):
                _add_shape(b, rng, shape, M)
    elif cfg_id == 2:
        D, M, caps, mults, q, w_hi, frac = 12, 32, TIER_CAP_LARGE, TIER_MULT_LARGE, 0.15, 40960, 0.3
        kinds = rng.integers(0, 3, size=64)
        sizes = {0: 10, 1: 12, 2: 18}
        n0 = sum(sizes[int(k)] for k in kinds)
        assert n0 <= 1024
        chains = [i for i, k in enumerate(kinds) if k == 1]
        extra = {i: 0 for i in chains}  # extra activations per chain instance
        need, j = 1024 - n0, 0
        while need > 0:
            add = min(3, need)
            extra[chains[j % len(chains)]] += add
            need -= add
            j += 1
        for i, k in enumerate(kinds):
            if k == 0:
                _add_shape(b, rng, _fanout_shape(), M)
            elif k == 1:
                e = extra[i]
                _add_shape(b, rng, _chain_shape(2 + e // 3, e % 3), M)
            else:
                _add_shape(b, rng, _mapreduce_shape(), M)
        gaps = np.rint(rng.exponential(50000.0, size=63)).astype(np.int64)
        arrivals = np.concatenate([[0], np.cumsum(gaps)]).astype(np.int64)
    elif cfg_id == 3:
        D, M, caps, mults, q, w_hi, frac = 16, 24, TIER_CAP_LARGE, TIER_MULT_LARGE, 0.10, 81920, 0.0
        par = _layered_parents(rng, [32] * 128, 0.15, span=2, force_parent=True)
        b.add_workflow(par, rng.integers(0, M, size=4096))
    elif cfg_id == 4:
        D, M, caps, mults, q, w_hi, frac = 8, 16, TIER_CAP_SMALL, (1.0, 1.0, 1.0), 0.10, 40960, 0.0
        for _ in range(16):
            par = _layered_parents(rng, _even_layers(16, 4), 0.4)
            b.add_workflow(par, rng.integers(0, M, size=16))
    else:
        raise ValueError(f"unknown config {cfg_id}")
    act_wf, act_model, off, idx, W = b.finish()
    lat, mem, weights, load, cap = _tables(rng, act_model, D, M, caps, mults, q, w_hi)
    res = _residency(rng, D, M, weights, cap, frac)
    if arrivals is None:
        arrivals = np.zeros(W, dtype=np.int64)
    return Window(
        n_act=len(act_wf), n_wf=W, n_models=M, n_dev=D, act_wf=act_wf,
        act_model=act_model, pred_off=off, pred_idx=idx, lat_us=lat, mem_mib=mem,
        wf_arrival_us=arrivals, dev_cap_mib=cap, model_mib=weights, load_us=load,
        init_resident=res, dev_free0_us=np.zeros(D, dtype=np.int64),
        w_makespan=1.0, w_p95=0.5, name=CONFIGS[cfg_id]["name"])


# --------------------------------------------------------------------------
# plans
# --------------------------------------------------------------------------


def _levels_for_layout(win: Window) -> np.ndarray:
    """Depth per activation (input numbering is level-sorted, so this is only
    used to find each level's index range for drawing priorities)."""
    n = win.n_act
    parents = [list(win.preds(i)) for i in range(n)]
    return _depths(n, parents, range(n))


def _fuse_candidates(win: Window):
    """Activations whose single parent uses the same model.  Fuse bits are
    drawn only there; the scorer itself decides which bits form chains."""
    out = []
    for v in range(win.n_act):
        ps = win.preds(v)
        if len(ps) == 1 and win.act_model[ps[0]] == win.act_model[v]:
            out.append((v, int(ps[0])))
    return out


def make_plans(win: Window, n_plans: int, rng: np.random.Generator,
               p_fuse: float = 0.3, p_prefetch: float = 0.2,
               chunk: int = 1 << 18) -> PlanBatch:
    """Candidate plans: device uniform over eligible devices, a random
    level-major topological priority, fuse and prefetch bits."""
    n, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(n, D)
    elig = [np.nonzero(lat[i] >= 0)[0].astype(np.int8) for i in range(n)]
    levels = _levels_for_layout(win)
    bounds = np.concatenate([[0], np.nonzero(np.diff(levels))[0] + 1, [n]]) if n else np.array([0])
    cands = _fuse_candidates(win)
    dev = np.empty((n_plans, n), dtype=np.int8)
    prio = np.empty((n_plans, n), dtype=np.uint16)
    flags = np.empty((n_plans, (n + 3) // 4), dtype=np.uint8)
    for a in range(0, n_plans, chunk):
        b = min(n_plans, a + chunk)
        p = b - a
        for i in range(n):
            e = elig[i]
            dev[a:b, i] = e[rng.integers(0, len(e), size=p)] if len(e) else 0
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            w = int(hi - lo)
            base = np.broadcast_to(np.arange(w, dtype=np.uint16), (p, w))
            prio[a:b, lo:hi] = lo + rng.permuted(base, axis=1)
        fuse = np.zeros((p, n), dtype=bool)
        for v, u in cands:
            f = rng.random(p) < p_fuse
            du = dev[a:b, u].astype(np.int64)
            ok = lat[v][du] >= 0
            f &= ok
            fuse[:, v] = f
            dev[a:b, v] = np.where(f, dev[a:b, u], dev[a:b, v])
        pf = rng.random((p, n)) < p_prefetch
        flags[a:b] = pack_flags(fuse, pf)
    return PlanBatch(dev, prio, flags)


def make_config(cfg_id: int, n_plans: Optional[int] = None) -> Tuple[Window, PlanBatch]:
    """Window and plan batch of a benchmark configuration (seeded by id)."""
    win = make_window(cfg_id)
    root = np.random.SeedSequence(cfg_id)
    _, plan_seed = root.spawn(2)
    rng = np.random.default_rng(plan_seed)
    P = CONFIGS[cfg_id]["n_plans"] if n_plans is None else n_plans
    return win, make_plans(win, P, rng)


# --------------------------------------------------------------------------
# random windows and adversarial plans for tests
# --------------------------------------------------------------------------


def random_window(rng: np.random.Generator, n_wf: int = 2, nodes=(1, 6), n_dev: int = 3,
                  n_models: int = 4, p_edge: float = 0.5, q_inel: float = 0.1,
                  cap_range=(8000, 40000), w_range=(1000, 12000), mem_range=(100, 4000),
                  lat_range=(1, 1000), load_range=(0, 5000), arrivals: bool = True,
                  free0: bool = True, resident: bool = True, same_model_bias: float = 0.3,
                  name: str = "random") -> Window:
    """Small random window with every feature switched on (arrivals, free
    times, initial residency, ineligible entries, same-model chains)."""
    b = _Builder()
    for _ in range(n_wf):
        k = int(rng.integers(nodes[0], nodes[1] + 1))
        n_layers = int(rng.integers(1, k + 1))
        par = _layered_parents(rng, _even_layers(k, n_layers), p_edge)
        models = rng.integers(0, n_models, size=k)
        for j, ps in enumerate(par):  # bias towards same-model parent->child
            if len(ps) == 1 and rng.random() < same_model_bias:
                models[j] = models[ps[0]]
        b.add_workflow(par, models)
    return _random_tables(b, rng, n_dev, n_models, q_inel, cap_range, w_range, mem_range, lat_range,
                          load_range, arrivals, free0, resident, name)


def random_deep_window(rng: np.random.Generator, n_wf: int = 1, n_levels=(20, 60), width=(1, 12),
                       span: int = 2, p_edge: float = 0.3, n_dev: int = 8, n_models: int = 20,
                       same_model_bias: float = 0.5, **kw) -> Window:
    """Deep layered workflows (many topological levels, edges reaching back
    up to ``span`` levels, a parent in the previous level for every node
    past the first, same-model parent->child chains), with the tables of
    random_window (its keyword arguments)."""
    b = _Builder()
    for _ in range(n_wf):
        L = int(rng.integers(n_levels[0], n_levels[1] + 1))
        sizes = [int(rng.integers(width[0], width[1] + 1)) for _ in range(L)]
        par = _layered_parents(rng, sizes, p_edge, span=span, force_parent=True)
        k = sum(sizes)
        models = rng.integers(0, n_models, size=k)
        for j, ps in enumerate(par):
            if len(ps) == 1 and rng.random() < same_model_bias:
                models[j] = models[ps[0]]
        b.add_workflow(par, models)
    args = dict(q_inel=0.1, cap_range=(8000, 40000), w_range=(1000, 12000), mem_range=(100, 4000),
                lat_range=(1, 1000), load_range=(0, 5000), arrivals=True, free0=True, resident=True,
                name="random-deep")
    args.update(kw)
    return _random_tables(b, rng, n_dev, n_models, **args)


def _random_tables(b, rng, n_dev, n_models, q_inel, cap_range, w_range, mem_range, lat_range,
                   load_range, arrivals, free0, resident, name) -> Window:
    act_wf, act_model, off, idx, W = b.finish()
    n, D, M = len(act_wf), n_dev, n_models
    cap = rng.integers(cap_range[0], cap_range[1], size=D, endpoint=True).astype(np.int32)
    weights = rng.integers(w_range[0], w_range[1], size=M, endpoint=True).astype(np.int32)
    mem = rng.integers(mem_range[0], mem_range[1], size=(n, D), endpoint=True).astype(np.int32)
    lat = rng.integers(lat_range[0], lat_range[1], size=(n, D), endpoint=True).astype(np.int32)
    lat[rng.random((n, D)) < q_inel] = -1
    for i in np.nonzero((lat < 0).all(axis=1))[0]:  # keep one eligible device per row
        lat[i, rng.integers(0, D)] = rng.integers(lat_range[0], lat_range[1], endpoint=True)
    load = rng.integers(load_range[0], load_range[1], size=(M, D), endpoint=True).astype(np.int32)
    res = np.zeros(D, dtype=np.uint64)
    if resident:
        for d in range(D):
            used = 0
            for m in rng.permutation(M):
                if rng.random() < 0.4 and used + weights[m] <= cap[d]:
                    used += int(weights[m])
                    res[d] |= np.uint64(1) << np.uint64(int(m))
    arr = (rng.integers(0, 3000, size=W) if arrivals else np.zeros(W)).astype(np.int64)
    f0 = (rng.integers(0, 2000, size=D) if free0 else np.zeros(D)).astype(np.int64)
    return Window(n_act=n, n_wf=W, n_models=M, n_dev=D, act_wf=act_wf, act_model=act_model,
                  pred_off=off, pred_idx=idx, lat_us=lat.reshape(-1), mem_mib=mem.reshape(-1),
                  wf_arrival_us=arr, dev_cap_mib=cap, model_mib=weights,
                  load_us=load.reshape(-1), init_resident=res, dev_free0_us=f0,
                  w_makespan=float(rng.choice([1.0, 0.75, 2.0])),
                  w_p95=float(rng.choice([0.5, 0.0, 1.25])), name=name)


def random_plans(win: Window, n_plans: int, rng: np.random.Generator,
                 p_fuse: float = 0.5, p_prefetch: float = 0.3, p_bad_dev: float = 0.0,
                 prio_mode: str = "any") -> PlanBatch:
    """Unconstrained plans: any eligible device (optionally invalid ones),
    priorities with ties ("any"), a level-major permutation ("perm"), or a
    permutation that ignores levels ("globalperm")."""
    n, D = win.n_act, win.n_dev
    lat = win.lat_us.reshape(n, D)
    dev = np.empty((n_plans, n), dtype=np.int8)
    for i in range(n):
        e = np.nonzero(lat[i] >= 0)[0]
        if len(e) == 0:
            e = np.arange(D)
        dev[:, i] = e[rng.integers(0, len(e), size=n_plans)]
    if p_bad_dev > 0:
        bad = rng.random((n_plans, n)) < p_bad_dev
        choices = np.array([-1, D, 127, -128, 0], dtype=np.int8)
        pick = choices[rng.integers(0, len(choices), size=(n_plans, n))]
        lat_bad = rng.integers(0, D, size=(n_plans, n)).astype(np.int8)
        dev = np.where(bad, np.where(rng.random((n_plans, n)) < 0.5, pick, lat_bad), dev)
    if prio_mode == "any":
        prio = rng.integers(0, max(2, n // 2), size=(n_plans, n)).astype(np.uint16)
        wide = rng.random(n_plans) < 0.3
        prio[wide] = rng.integers(0, 65536, size=(int(wide.sum()), n)).astype(np.uint16)
    elif prio_mode == "perm":
        levels = _levels_for_layout(win)
        prio = np.empty((n_plans, n), dtype=np.uint16)
        bounds = np.concatenate([[0], np.nonzero(np.diff(levels))[0] + 1, [n]]) if n else [0]
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            base = np.broadcast_to(np.arange(hi - lo, dtype=np.uint16), (n_plans, hi - lo))
            prio[:, lo:hi] = lo + rng.permuted(base, axis=1)
    elif prio_mode == "globalperm":
        base = np.broadcast_to(np.arange(n, dtype=np.uint16), (n_plans, n))
        prio = rng.permuted(base, axis=1).astype(np.uint16)
    else:
        raise ValueError(prio_mode)
    fuse = rng.random((n_plans, n)) < p_fuse
    pf = rng.random((n_plans, n)) < p_prefetch
    return PlanBatch(np.ascontiguousarray(dev), np.ascontiguousarray(prio, dtype=np.uint16),
                     np.ascontiguousarray(pack_flags(fuse, pf)))


# --------------------------------------------------------------------------
# persistence
# --------------------------------------------------------------------------


def save_npz(path: str, win: Window, plans: Optional[PlanBatch] = None) -> None:
    arrs = {f"w_{k}": np.asarray(v) for k, v in win.arrays().items() if v is not None}
    if plans is not None:
        arrs.update(p_dev=plans.dev, p_prio=plans.prio, p_flags=plans.flags)
    np.savez(path, **arrs)


def load_npz(path: str):
    z = np.load(path, allow_pickle=False)
    kw = {}
    for f in dataclasses.fields(Window):
        if f"w_{f.name}" not in z:  # an optional field that was None
            continue
        v = z[f"w_{f.name}"]
        kw[f.name] = v.item() if v.ndim == 0 else v
    kw["name"] = str(kw["name"])
    for k in ("n_act", "n_wf", "n_models", "n_dev"):
        kw[k] = int(kw[k])
    for k in ("w_makespan", "w_p95"):
        kw[k] = float(kw[k])
    if "victim_order" in kw:
        kw["victim_order"] = int(kw["victim_order"])
    win = Window(**kw)
    plans = PlanBatch(z["p_dev"], z["p_prio"], z["p_flags"]) if "p_dev" in z else None
    return win, plans

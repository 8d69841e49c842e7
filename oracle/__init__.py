"""CPU reference scorer (oracle) -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it.  ``oracle.c`` holds the scoring arithmetic; this module
only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")

INELIGIBLE = 1
CAPACITY = 2
REPLICA = 4
VICTIM_REMAINING_LRU = 0
VICTIM_PAPER = 1
MAX_BATCH = 4

SCORE_DTYPE = np.dtype([
    ("makespan_us", "<i8"), ("p95_us", "<i8"), ("objective", "<f4"),
    ("status", "<u4"), ("min_headroom_mib", "<i4"), ("n_loads", "<u2"),
    ("n_evicts", "<u2"),
])
assert SCORE_DTYPE.itemsize == 32

MAX_CLASSES = 4
PHI_DTYPE = np.dtype([
    ("c_ready_us", "<i8"), ("h_life_us", "<i8"), ("admitted", "<u2", (MAX_CLASSES,)),
    ("timely_prefetch", "<u2"), ("pad", "<u2"), ("status", "<u4"),
])
assert PHI_DTYPE.itemsize == 32


def build(force: bool = True, src: str = SRC_PATH, out: str = LIB_PATH) -> str:
    """Compile liboracle.so with gcc (plain C99, no FMA contraction)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.check_call([
            "gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fPIC", "-shared",
            "-Wall", "-Wextra", "-I", _HERE, "-o", tmp, src])
        os.replace(tmp, out)
    return out


class _Win(ctypes.Structure):
    _fields_ = [
        ("n_act", ctypes.c_int32), ("n_wf", ctypes.c_int32),
        ("n_models", ctypes.c_int32), ("n_dev", ctypes.c_int32),
        ("act_wf", ctypes.c_void_p), ("act_model", ctypes.c_void_p),
        ("pred_off", ctypes.c_void_p), ("pred_idx", ctypes.c_void_p),
        ("lat_us", ctypes.c_void_p), ("mem_mib", ctypes.c_void_p),
        ("wf_arrival_us", ctypes.c_void_p), ("dev_cap_mib", ctypes.c_void_p),
        ("model_mib", ctypes.c_void_p), ("load_us", ctypes.c_void_p),
        ("init_resident", ctypes.c_void_p), ("dev_free0_us", ctypes.c_void_p),
        ("w_makespan", ctypes.c_float), ("w_p95", ctypes.c_float),
        ("victim_order", ctypes.c_int32),
        ("dev_batch", ctypes.c_void_p),
        ("replica_cap", ctypes.c_void_p),
        ("prefetch_slack_us", ctypes.c_int64),
    ]


_libs = {}
_lock = threading.Lock()


def _load(path: Optional[str] = None):
    """Load (building on first use) the oracle library; ``path`` selects an
    alternative build of oracle.c (the mutation tests use this)."""
    path = path or LIB_PATH
    with _lock:
        if path not in _libs:
            if path == LIB_PATH and not os.path.exists(path):
                build(force=True)
            lib = ctypes.CDLL(path)
            lib.orc_score_plans.restype = ctypes.c_int
            lib.orc_score_plans.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_int64] + [ctypes.c_void_p] * 6
            lib.orc_prefix.restype = ctypes.c_int
            lib.orc_prefix.argtypes = [ctypes.c_void_p] * 9
            lib.orc_phi_keys.restype = ctypes.c_int
            lib.orc_phi_keys.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int64, ctypes.c_void_p]
            lib.orc_levels.restype = ctypes.c_int
            lib.orc_levels.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.orc_philox4x32_10.restype = None
            lib.orc_philox4x32_10.argtypes = [ctypes.c_void_p] * 3
            lib.orc_search_candidates.restype = ctypes.c_int
            lib.orc_search_candidates.argtypes = ([ctypes.c_void_p] * 4 + [ctypes.c_uint64, ctypes.c_int32,
                                                  ctypes.c_int64, ctypes.c_int64, ctypes.c_int32]
                                                 + [ctypes.c_void_p] * 3)
            _libs[path] = lib
    return _libs[path]


class OracleError(RuntimeError):
    pass


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


class _WinHolder:
    """Keeps the contiguous arrays alive while the C struct points at them."""

    def __init__(self, win):
        self.keep = {
            "act_wf": _c(win.act_wf, np.int32), "act_model": _c(win.act_model, np.int32),
            "pred_off": _c(win.pred_off, np.int32), "pred_idx": _c(win.pred_idx, np.int32),
            "lat_us": _c(win.lat_us, np.int32), "mem_mib": _c(win.mem_mib, np.int32),
            "wf_arrival_us": _c(win.wf_arrival_us, np.int64),
            "dev_cap_mib": _c(win.dev_cap_mib, np.int32), "model_mib": _c(win.model_mib, np.int32),
            "load_us": _c(win.load_us, np.int32), "init_resident": _c(win.init_resident, np.uint64),
            "dev_free0_us": None if win.dev_free0_us is None else _c(win.dev_free0_us, np.int64),
            "dev_batch": (None if getattr(win, "dev_batch", None) is None
                          else _c(win.dev_batch, np.int32)),
            "replica_cap": (None if getattr(win, "model_replica_cap", None) is None
                            else _c(win.model_replica_cap, np.int32)),
        }
        if self.keep["pred_idx"].size == 0:
            self.keep["pred_idx"] = np.zeros(1, dtype=np.int32)
        s = _Win()
        s.n_act, s.n_wf, s.n_models, s.n_dev = win.n_act, win.n_wf, win.n_models, win.n_dev
        for k, v in self.keep.items():
            setattr(s, k, None if v is None else v.ctypes.data)
        s.w_makespan, s.w_p95 = win.w_makespan, win.w_p95
        s.victim_order = int(getattr(win, "victim_order", 0))
        s.prefetch_slack_us = int(getattr(win, "prefetch_slack_us", 0))
        self.struct = s


def levels(win, lib_path: Optional[str] = None) -> np.ndarray:
    lib = _load(lib_path)
    h = _WinHolder(win)
    out = np.zeros(max(1, win.n_act), dtype=np.int32)
    rc = lib.orc_levels(ctypes.byref(h.struct), out.ctypes.data)
    if rc:
        raise OracleError(f"oracle rejected window (code {rc})")
    return out[:win.n_act]


def _plan_rows(win, plans, begin, end):
    N = win.n_act
    P = end - begin
    if N == 0:
        # zero-width rows: give the C code a valid (unused) pointer
        return np.zeros((P, 1), np.int8), np.zeros((P, 1), np.uint16), np.zeros((P, 1), np.uint8)
    return (np.ascontiguousarray(plans.dev[begin:end], dtype=np.int8),
            np.ascontiguousarray(plans.prio[begin:end], dtype=np.uint16),
            np.ascontiguousarray(plans.flags[begin:end], dtype=np.uint8))


def _run_split(run, P, threads):
    """run(a, b) over [0, P), split into contiguous ranges on threads."""
    if threads <= 1 or P < 2 * threads:
        rc = run(0, P)
        if rc:
            raise OracleError(f"oracle rejected window (code {rc})")
        return
    bounds = np.linspace(0, P, threads + 1).astype(np.int64)
    rcs = [0] * threads

    def worker(t):
        rcs[t] = run(int(bounds[t]), int(bounds[t + 1]))
    ts = [threading.Thread(target=worker, args=(t,)) for t in range(threads)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    if any(rcs):
        raise OracleError(f"oracle rejected window (codes {rcs})")


def score(win, plans, begin: int = 0, end: Optional[int] = None, schedule: bool = False,
          threads: int = 1, lib_path: Optional[str] = None, reclaims: bool = False):
    """Score plans [begin, end) of ``plans``.  Returns a structured score
    array, and with ``schedule=True`` also (start, finish, load_start, peak),
    with ``reclaims=True`` as well followed by the [P][N] uint64 masks of the
    copies reclaimed before each unit."""
    lib = _load(lib_path)
    h = _WinHolder(win)
    end = plans.n_plans if end is None else end
    P = end - begin
    N, D = win.n_act, win.n_dev
    dev, prio, flags = _plan_rows(win, plans, begin, end)
    scores = np.zeros(P, dtype=SCORE_DTYPE)
    sched = None
    if schedule:
        sched = (np.zeros((P, N), np.int64), np.zeros((P, N), np.int64),
                 np.zeros((P, N), np.int64), np.zeros((P, D), np.int32))
        if reclaims:
            sched = sched + (np.zeros((P, N), np.uint64),)

    def run(a, b):
        if b <= a:
            return 0

        def ptr(arr):
            return None if arr is None else arr.ctypes.data + a * arr.strides[0]

        s0, s1, s2, s3 = sched[:4] if sched is not None else (None, None, None, None)
        s4 = sched[4] if sched is not None and len(sched) > 4 else None
        return lib.orc_score_plans(ctypes.byref(h.struct), ptr(dev), ptr(prio), ptr(flags),
                                   b - a, ptr(scores), ptr(s0), ptr(s1), ptr(s2), ptr(s3), ptr(s4))

    _run_split(run, P, threads)
    if schedule:
        return scores, sched
    return scores


def prefix(win, dev_row, start, finish, load_start, reclaimed, lib_path: Optional[str] = None):
    """Prefix commit of Algorithm 1 for one plan (its device row and
    schedule rows): (commit uint8[N], commit_reclaimed uint64[N], t_next)."""
    lib = _load(lib_path)
    h = _WinHolder(win)
    N = win.n_act
    arrs = [np.ascontiguousarray(x, dt) for x, dt in ((dev_row, np.int8), (start, np.int64),
                                                      (finish, np.int64), (load_start, np.int64),
                                                      (reclaimed, np.uint64))]
    for x in arrs:
        assert x.shape == (N,)
    commit = np.zeros(N, np.uint8)
    crec = np.zeros(N, np.uint64)
    t_next = np.zeros(1, np.int64)
    rc = lib.orc_prefix(ctypes.byref(h.struct), *[x.ctypes.data for x in arrs], commit.ctypes.data,
                        crec.ctypes.data, t_next.ctypes.data)
    if rc:
        raise OracleError(rc)
    return commit, crec, int(t_next[0])


def phi_keys(win, plans, begin: int = 0, end: Optional[int] = None, threads: int = 1,
             lib_path: Optional[str] = None) -> np.ndarray:
    """Ranking keys (Eq. 12) of plans [begin, end) as a PHI_DTYPE array; the
    workflow classes come from ``win.wf_class`` (None: all class 0)."""
    lib = _load(lib_path)
    h = _WinHolder(win)
    end = plans.n_plans if end is None else end
    P = end - begin
    dev, prio, flags = _plan_rows(win, plans, begin, end)
    cls = getattr(win, "wf_class", None)
    cls = None if cls is None else np.ascontiguousarray(cls, dtype=np.uint8)
    keys = np.zeros(P, dtype=PHI_DTYPE)

    def run(a, b):
        if b <= a:
            return 0
        return lib.orc_phi_keys(ctypes.byref(h.struct), None if cls is None else cls.ctypes.data,
                                dev.ctypes.data + a * dev.strides[0],
                                prio.ctypes.data + a * prio.strides[0],
                                flags.ctypes.data + a * flags.strides[0], b - a,
                                keys.ctypes.data + a * keys.strides[0])

    _run_split(run, P, threads)
    return keys


def phi_order_key(k) -> tuple:
    """The lexicographic key of Eq. 12 for one PHI_DTYPE record:
    (-A_1, ..., -A_K, C_F, -P_N, H_life)."""
    return tuple(-int(a) for a in k["admitted"]) + (int(k["c_ready_us"]), -int(k["timely_prefetch"]),
                                                    int(k["h_life_us"]))


def philox4x32_10(ctr, key, lib_path: Optional[str] = None) -> np.ndarray:
    """Philox4x32-10 of one 4-word counter under a 2-word key."""
    lib = _load(lib_path)
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib.orc_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


SEARCH_UNIFORM, SEARCH_RULES = 0, 1


def search_candidates(win, dev, prio, flags, seed: int, n_mut: int, first: int, count: int,
                      lib_path: Optional[str] = None, mode: int = SEARCH_UNIFORM):
    """Rows (dev, prio, flags) of candidates first .. first+count-1 around the
    incumbent rows (one plan each); mode SEARCH_RULES takes the device and
    prefetch alternatives from the rules of Algorithm 1 (oracle.h)."""
    lib = _load(lib_path)
    h = _WinHolder(win)
    N = win.n_act
    nb = (N + 3) // 4
    d = np.ascontiguousarray(dev, dtype=np.int8).reshape(-1)
    p = np.ascontiguousarray(prio, dtype=np.uint16).reshape(-1)
    f = np.ascontiguousarray(flags, dtype=np.uint8).reshape(-1)
    assert d.size == N and p.size == N and f.size == nb
    od = np.zeros((count, max(N, 1)), np.int8)
    op = np.zeros((count, max(N, 1)), np.uint16)
    of = np.zeros((count, max(nb, 1)), np.uint8)
    dd = d if N else np.zeros(1, np.int8)
    pp = p if N else np.zeros(1, np.uint16)
    ff = f if nb else np.zeros(1, np.uint8)
    rc = lib.orc_search_candidates(ctypes.byref(h.struct), dd.ctypes.data, pp.ctypes.data,
                                   ff.ctypes.data, int(seed) & ((1 << 64) - 1), int(n_mut),
                                   int(first), int(count), int(mode), od.ctypes.data,
                                   op.ctypes.data, of.ctypes.data)
    if rc:
        raise OracleError(f"oracle rejected window (code {rc})")
    return od[:, :N].copy(), op[:, :N].copy(), of[:, :nb].copy()

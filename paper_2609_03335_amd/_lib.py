"""ctypes binding of libwfplan.so.  Function names follow include/wf_plan.h;
this module only marshals arguments (host arrays for the window, device
pointers and a HIP stream for the plan batch).  Every step of scoring runs in
the gfx950 kernels; there is no CPU fallback: if the library is missing or
no GPU is present, calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libwfplan.so")

WF_OK, WF_EINVAL, WF_ENOWINDOW, WF_ENOMEM, WF_EHIP, WF_EUNSUPPORTED = range(6)
STATUS_NAMES = {0: "WF_OK", 1: "WF_EINVAL", 2: "WF_ENOWINDOW", 3: "WF_ENOMEM", 4: "WF_EHIP",
                5: "WF_EUNSUPPORTED"}
WF_ST_INELIGIBLE = 1
WF_ST_CAPACITY = 2
WF_ST_REPLICA = 4
WF_MAX_ACT, WF_MAX_MODELS, WF_MAX_DEV, WF_MAX_MUT = 65535, 64, 127, 64
WF_MAX_CLASSES = 4
WF_VICTIM_REMAINING_LRU, WF_VICTIM_PAPER = 0, 1
WF_MAX_BATCH = 4
WF_SEARCH_UNIFORM, WF_SEARCH_RULES = 0, 1

SCORE_DTYPE = np.dtype([
    ("makespan_us", "<i8"), ("p95_us", "<i8"), ("objective", "<f4"),
    ("status", "<u4"), ("min_headroom_mib", "<i4"), ("n_loads", "<u2"),
    ("n_evicts", "<u2"),
])
assert SCORE_DTYPE.itemsize == 32

# wf_plan_key: the ranking key of Eq. 12
KEY_DTYPE = np.dtype([
    ("c_ready_us", "<i8"), ("h_life_us", "<i8"), ("admitted", "<u2", (WF_MAX_CLASSES,)),
    ("timely_prefetch", "<u2"), ("pad", "<u2"), ("status", "<u4"),
])
assert KEY_DTYPE.itemsize == 32

# every symbol declared in include/wf_plan.h
EXPORTS = ("wf_plan_ctx_create", "wf_plan_ctx_destroy", "wf_plan_last_error",
           "wf_plan_validate_window", "wf_plan_upload_window", "wf_plan_score_batch",
           "wf_plan_argmin", "wf_plan_argmin_noalloc", "wf_plan_search_batch", "wf_plan_search_rows",
           "wf_plan_score_keys", "wf_plan_search_keys", "wf_plan_argmin_keys",
           "wf_plan_prefix", "wf_plan_time_bits", "wf_plan_score_kernel", "wf_plan_version")


class WFError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class wf_window_desc(ctypes.Structure):
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
        ("wf_class", ctypes.c_void_p),
        ("victim_order", ctypes.c_int32),
        ("dev_batch", ctypes.c_void_p),
        ("model_replica_cap", ctypes.c_void_p),
        ("prefetch_slack_us", ctypes.c_int64),
    ]


class wf_plan_sched(ctypes.Structure):
    _fields_ = [("start_us", ctypes.c_void_p), ("finish_us", ctypes.c_void_p),
                ("load_start_us", ctypes.c_void_p), ("peak_mib", ctypes.c_void_p),
                ("reclaimed_models", ctypes.c_void_p)]


_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libwfplan.so; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build the gfx950 library first "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(p)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.wf_plan_ctx_create.argtypes = [i32, ctypes.POINTER(vp)]
    lib.wf_plan_ctx_create.restype = i32
    lib.wf_plan_ctx_destroy.argtypes = [vp]
    lib.wf_plan_ctx_destroy.restype = None
    lib.wf_plan_last_error.argtypes = [vp]
    lib.wf_plan_last_error.restype = ctypes.c_char_p
    lib.wf_plan_validate_window.argtypes = [vp, ctypes.c_char_p, ctypes.c_size_t]
    lib.wf_plan_validate_window.restype = i32
    lib.wf_plan_upload_window.argtypes = [vp, vp]
    lib.wf_plan_upload_window.restype = i32
    lib.wf_plan_score_batch.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp]
    lib.wf_plan_score_batch.restype = i32
    lib.wf_plan_argmin.argtypes = [vp, vp, i64, vp, vp]
    lib.wf_plan_argmin.restype = i32
    lib.wf_plan_argmin_noalloc.argtypes = [vp, i64, vp, vp]
    lib.wf_plan_argmin_noalloc.restype = i32
    u64 = ctypes.c_uint64
    lib.wf_plan_search_batch.argtypes = [vp, vp, vp, vp, i32, u64, i32, i64, i64, vp, vp]
    lib.wf_plan_search_batch.restype = i32
    lib.wf_plan_search_rows.argtypes = [vp, vp, vp, vp, i32, u64, i32, i64, i64, vp, vp, vp, vp]
    lib.wf_plan_search_rows.restype = i32
    lib.wf_plan_score_keys.argtypes = [vp, vp, vp, vp, i64, vp, vp]
    lib.wf_plan_score_keys.restype = ctypes.c_int
    lib.wf_plan_search_keys.argtypes = [vp, vp, vp, vp, i32, u64, i32, i64, i64, vp, vp]
    lib.wf_plan_search_keys.restype = ctypes.c_int
    lib.wf_plan_argmin_keys.argtypes = [vp, vp, i64, vp, vp]
    lib.wf_plan_argmin_keys.restype = ctypes.c_int
    lib.wf_plan_prefix.argtypes = [vp] * 10
    lib.wf_plan_prefix.restype = i32
    lib.wf_plan_time_bits.argtypes = [vp]
    lib.wf_plan_time_bits.restype = i32
    lib.wf_plan_score_kernel.argtypes = [vp]
    lib.wf_plan_score_kernel.restype = ctypes.c_char_p
    lib.wf_plan_version.argtypes = []
    lib.wf_plan_version.restype = ctypes.c_char_p
    # an entry point without a declared signature would take Python ints as
    # 32-bit C ints and cut device addresses short
    for name in EXPORTS:
        if getattr(lib, name).argtypes is None:
            raise RuntimeError(f"{name}: no ctypes signature declared")
    if path is None:
        _lib = lib
    return lib


class _Desc:
    """A wf_window_desc plus the contiguous host arrays it points at."""

    def __init__(self, win):
        def c(a, dt):
            a = np.ascontiguousarray(a, dtype=dt)
            return a if a.size else np.zeros(1, dtype=dt)
        self.keep = dict(
            act_wf=c(win.act_wf, np.int32), act_model=c(win.act_model, np.int32),
            pred_off=c(win.pred_off, np.int32), pred_idx=c(win.pred_idx, np.int32),
            lat_us=c(win.lat_us, np.int32), mem_mib=c(win.mem_mib, np.int32),
            wf_arrival_us=c(win.wf_arrival_us, np.int64), dev_cap_mib=c(win.dev_cap_mib, np.int32),
            model_mib=c(win.model_mib, np.int32), load_us=c(win.load_us, np.int32),
            init_resident=c(win.init_resident, np.uint64))
        free0 = getattr(win, "dev_free0_us", None)
        self.keep["dev_free0_us"] = None if free0 is None else c(free0, np.int64)
        cls = getattr(win, "wf_class", None)
        self.keep["wf_class"] = None if cls is None else c(cls, np.uint8)
        bat = getattr(win, "dev_batch", None)
        self.keep["dev_batch"] = None if bat is None else c(bat, np.int32)
        rc = getattr(win, "model_replica_cap", None)
        self.keep["model_replica_cap"] = None if rc is None else c(rc, np.int32)
        d = wf_window_desc()
        d.n_act, d.n_wf, d.n_models, d.n_dev = win.n_act, win.n_wf, win.n_models, win.n_dev
        for k, v in self.keep.items():
            setattr(d, k, None if v is None else v.ctypes.data)
        d.w_makespan, d.w_p95 = win.w_makespan, win.w_p95
        d.victim_order = int(getattr(win, "victim_order", 0))
        d.prefetch_slack_us = int(getattr(win, "prefetch_slack_us", 0))
        self.desc = d


def _ptr(x) -> Optional[int]:
    """Device address of a buffer; tensors must be dense row-major (the ABI
    takes flat row-major arrays).  No placement or size check: the Context
    methods check tensors with _buf before calling the library."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "is_contiguous") and not x.is_contiguous():
        raise ValueError("device buffers must be contiguous row-major tensors")
    return int(x.data_ptr())


def _buf(x, need: int, device: int, name: str) -> Optional[int]:
    """Device address of a buffer argument after the checks the library
    cannot make on a bare pointer: a torch tensor must be contiguous, live on
    GPU `device` and hold at least `need` bytes.  A raw int is taken as a
    device address the caller vouches for; None passes through (the library
    rejects a missing required array)."""
    if x is None or isinstance(x, int):
        return x
    if not hasattr(x, "data_ptr"):
        raise TypeError(f"{name}: expected a torch tensor or a device address")
    if not x.is_contiguous():
        raise ValueError(f"{name}: device buffers must be contiguous row-major tensors")
    if not x.is_cuda:
        raise ValueError(f"{name}: a host tensor cannot be passed to the GPU library")
    if x.device.index != device:
        raise ValueError(f"{name}: tensor on cuda:{x.device.index}, context on cuda:{device}")
    nbytes = x.numel() * x.element_size()
    if nbytes < need:
        raise ValueError(f"{name}: {nbytes} bytes, at least {need} needed")
    return int(x.data_ptr())


def wf_plan_version() -> str:
    return load().wf_plan_version().decode()


def wf_plan_validate_window(win) -> tuple:
    """Host-only validation: (status, message)."""
    lib = load()
    d = _Desc(win)
    buf = ctypes.create_string_buffer(512)
    st = lib.wf_plan_validate_window(ctypes.byref(d.desc), buf, len(buf))
    return st, buf.value.decode()


def wf_plan_argmin_noalloc(scores, n_plans: int, out_index, stream=None) -> None:
    """wf_plan_argmin without a context or any allocation, on the current
    HIP device (its work area is the library's static array).  Tensors must
    live on the current device."""
    lib = load()
    n = int(n_plans)
    sized = n if 0 <= n < (1 << 32) else 0
    cur = 0
    if any(x is not None and not isinstance(x, int) for x in (scores, out_index)):
        import torch
        cur = torch.cuda.current_device()
    st = lib.wf_plan_argmin_noalloc(_buf(scores, 32 * sized, cur, "scores"), n,
                                    _buf(out_index, 8, cur, "out_index"), _stream(stream))
    if st != WF_OK:
        raise WFError(st, lib.wf_plan_last_error(None).decode())


class Context:
    """A wf_plan_ctx on one HIP device.  Tensor arguments are checked before
    any call reaches the library (GPU tensor, the context's device, enough
    bytes for the uploaded window's sizes)."""

    def __init__(self, device: int = 0):
        self.lib = load()
        h = ctypes.c_void_p()
        st = self.lib.wf_plan_ctx_create(device, ctypes.byref(h))
        if st != WF_OK:
            raise WFError(st, self.lib.wf_plan_last_error(None).decode())
        self.handle = h
        self.device = device
        self._nd = (0, 0)  # (N, D) of the uploaded window

    def _check(self, st):
        if st != WF_OK:
            raise WFError(st, self.lib.wf_plan_last_error(self.handle).decode())

    @staticmethod
    def _cnt(n, limit=1 << 62) -> int:
        """A plan count for sizing buffers; a count the library will refuse
        (negative or above its limit) sizes nothing, so that the library's
        WF_EINVAL reaches the caller."""
        n = int(n)
        return n if 0 <= n <= limit else 0

    def _b(self, x, need: int, name: str) -> Optional[int]:
        return _buf(x, max(int(need), 0), self.device, name)

    def _rows(self, dev, prio, flags, n: int):
        """Addresses of n plan rows (dev [n][N], prio [n][N], flags [n][ceil(N/4)])."""
        N = self._nd[0]
        return (self._b(dev, n * N, "dev"), self._b(prio, 2 * n * N, "prio"),
                self._b(flags, n * ((N + 3) // 4), "flags"))

    def wf_plan_upload_window(self, win) -> None:
        d = _Desc(win)
        self._check(self.lib.wf_plan_upload_window(self.handle, ctypes.byref(d.desc)))
        self._nd = (int(win.n_act), int(win.n_dev))

    def wf_plan_score_batch(self, dev, prio, flags, n_plans: int, scores, sched=None,
                            stream=None) -> None:
        """dev/prio/flags/scores (and the schedule arrays: start, finish,
        load_start, peak and optionally reclaimed) are device buffers: torch
        tensors or raw device addresses."""
        P = self._cnt(n_plans)
        N, D = self._nd
        s = None
        if sched is not None:
            sched = tuple(sched) + (None,) * (5 - len(sched))
            needs = (8 * P * N, 8 * P * N, 8 * P * N, 4 * P * D, 8 * P * N)
            names = ("start_us", "finish_us", "load_start_us", "peak_mib", "reclaimed_models")
            s = wf_plan_sched(*(self._b(x, k, nm) for x, k, nm in zip(sched, needs, names)))
        self._check(self.lib.wf_plan_score_batch(
            self.handle, *self._rows(dev, prio, flags, P), int(n_plans),
            self._b(scores, 32 * P, "scores"), None if s is None else ctypes.byref(s),
            _stream(stream)))

    def wf_plan_prefix(self, dev, start, finish, load_start, reclaimed, commit,
                       commit_reclaimed, t_next, stream=None) -> None:
        """One plan's device row and schedule rows in; commit flags, committed
        reclamations and the next event time out (all device buffers)."""
        N = self._nd[0]
        self._check(self.lib.wf_plan_prefix(
            self.handle, self._b(dev, N, "dev"), self._b(start, 8 * N, "start_us"),
            self._b(finish, 8 * N, "finish_us"), self._b(load_start, 8 * N, "load_start_us"),
            self._b(reclaimed, 8 * N, "reclaimed"), self._b(commit, N, "commit"),
            self._b(commit_reclaimed, 8 * N, "commit_reclaimed"), self._b(t_next, 8, "t_next_us"),
            _stream(stream)))

    def wf_plan_argmin(self, scores, n_plans: int, out_index, stream=None) -> None:
        self._check(self.lib.wf_plan_argmin(
            self.handle, self._b(scores, 32 * self._cnt(n_plans, (1 << 32) - 1), "scores"), int(n_plans),
            self._b(out_index, 8, "out_index"), _stream(stream)))

    def wf_plan_search_batch(self, dev, prio, flags, seed: int, n_mut: int, first: int,
                             n_candidates: int, scores, stream=None,
                             mode: int = WF_SEARCH_UNIFORM) -> None:
        """Score candidates first .. first+n_candidates-1 generated around the
        incumbent rows dev/prio/flags (device buffers of one plan); mode is
        WF_SEARCH_UNIFORM or WF_SEARCH_RULES."""
        self._check(self.lib.wf_plan_search_batch(
            self.handle, *self._rows(dev, prio, flags, 1), int(mode), int(seed) & ((1 << 64) - 1),
            int(n_mut), int(first), int(n_candidates),
            self._b(scores, 32 * self._cnt(n_candidates), "scores"), _stream(stream)))

    def wf_plan_search_rows(self, dev, prio, flags, seed: int, n_mut: int, first: int,
                            n_candidates: int, out_dev, out_prio, out_flags, stream=None,
                            mode: int = WF_SEARCH_UNIFORM) -> None:
        """Write the rows of candidates first .. first+n_candidates-1."""
        n = self._cnt(n_candidates)
        N = self._nd[0]
        self._check(self.lib.wf_plan_search_rows(
            self.handle, *self._rows(dev, prio, flags, 1), int(mode), int(seed) & ((1 << 64) - 1),
            int(n_mut), int(first), int(n_candidates), self._b(out_dev, n * N, "out_dev"),
            self._b(out_prio, 2 * n * N, "out_prio"),
            self._b(out_flags, n * ((N + 3) // 4), "out_flags"), _stream(stream)))

    def wf_plan_score_keys(self, dev, prio, flags, n_plans: int, keys, stream=None) -> None:
        """Ranking keys (Eq. 12) of plans 0..n_plans-1 into keys (32 B each)."""
        P = self._cnt(n_plans)
        self._check(self.lib.wf_plan_score_keys(
            self.handle, *self._rows(dev, prio, flags, P), int(n_plans),
            self._b(keys, 32 * P, "keys"), _stream(stream)))

    def wf_plan_search_keys(self, dev, prio, flags, seed: int, n_mut: int, first: int,
                            n_candidates: int, keys, stream=None,
                            mode: int = WF_SEARCH_UNIFORM) -> None:
        """Ranking keys of candidates generated around the incumbent rows."""
        self._check(self.lib.wf_plan_search_keys(
            self.handle, *self._rows(dev, prio, flags, 1), int(mode), int(seed) & ((1 << 64) - 1),
            int(n_mut), int(first), int(n_candidates),
            self._b(keys, 32 * self._cnt(n_candidates), "keys"), _stream(stream)))

    def wf_plan_argmin_keys(self, keys, n_plans: int, out_index, stream=None) -> None:
        self._check(self.lib.wf_plan_argmin_keys(
            self.handle, self._b(keys, 32 * self._cnt(n_plans), "keys"), int(n_plans),
            self._b(out_index, 8, "out_index"), _stream(stream)))

    def wf_plan_time_bits(self) -> int:
        return int(self.lib.wf_plan_time_bits(self.handle))

    def wf_plan_score_kernel(self) -> str:
        return self.lib.wf_plan_score_kernel(self.handle).decode()

    def close(self):
        if getattr(self, "handle", None):
            self.lib.wf_plan_ctx_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _stream(stream) -> Optional[int]:
    if stream is None:
        try:
            import torch
            return int(torch.cuda.current_stream().cuda_stream) or None
        except Exception:
            return None
    if isinstance(stream, int):
        return stream or None
    return int(stream.cuda_stream) or None

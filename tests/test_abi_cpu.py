"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every function include/wf_plan.h declares, the score record has the
declared layout, and window validation rejects what it should."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_03335_amd as pkg
from paper_2609_03335_amd import _lib, workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wf_plan.h")


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_03335_amd import build
        build.build()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wf_plan_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    names = declared_functions()
    assert set(names) == set(_lib.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    assert pkg.wf_plan_version().startswith("wf_plan")


def test_every_entry_point_has_a_full_signature():
    """Each binding declares the C signature, with one ctypes type per
    parameter of the header's prototype: an undeclared pointer argument
    would reach the library cut to 32 bits."""
    lib = _lib.load()
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for name in _lib.EXPORTS:
        m = re.search(r"\b" + name + r"\s*\(([^)]*)\)\s*;", text)
        assert m, name
        params = [x for x in m.group(1).split(",") if x.strip() and x.strip() != "void"]
        argtypes = getattr(lib, name).argtypes
        assert argtypes is not None, name
        assert len(argtypes) == len(params), (name, len(argtypes), len(params))
        for ctype, decl in zip(argtypes, params):
            if "*" in decl:  # every pointer travels as a full address
                assert ctype in (ctypes.c_void_p, ctypes.c_char_p) or hasattr(ctype, "contents"), (name, decl)


def test_time_bits_without_window():
    assert _lib.load().wf_plan_time_bits(None) == 0


def test_score_record_layout():
    text = open(HEADER).read()
    assert "int64_t makespan_us;" in text and "uint16_t n_evicts;" in text
    assert pkg.SCORE_DTYPE.itemsize == 32
    assert [pkg.SCORE_DTYPE.fields[k][1] for k in pkg.SCORE_DTYPE.names] == [0, 8, 16, 20, 24, 28, 30]


def test_key_record_layout():
    text = open(HEADER).read()
    assert "uint16_t admitted[WF_MAX_CLASSES];" in text and "} wf_plan_key;" in text
    assert pkg.KEY_DTYPE.itemsize == 32
    assert [pkg.KEY_DTYPE.fields[k][1] for k in pkg.KEY_DTYPE.names] == [0, 8, 16, 24, 26, 28]


def test_classes_in_range_pass():
    w = _ok_window()
    w.wf_class = np.arange(w.n_wf, dtype=np.uint8) % pkg._lib.WF_MAX_CLASSES
    assert pkg.wf_plan_validate_window(w)[0] == pkg.WF_OK


def test_no_gpu_context_fails_cleanly():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(pkg.WFError) as e:
        pkg.Context(0)
    assert e.value.status == pkg.WF_EHIP


def _ok_window():
    return W.make_window(0)


def test_valid_windows_pass():
    for cfg in range(5):
        st, msg = pkg.wf_plan_validate_window(W.make_window(cfg))
        assert st == pkg.WF_OK, msg
    rng = np.random.default_rng(0)
    for _ in range(20):
        st, msg = pkg.wf_plan_validate_window(W.random_window(rng))
        assert st == pkg.WF_OK, msg


def _mutate(fn):
    w = _ok_window()
    w2 = W.Window(**{k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in w.arrays().items()})
    fn(w2)
    return w2


BAD = {
    "n_models_zero": lambda w: setattr(w, "n_models", 0),
    "n_models_65": lambda w: setattr(w, "n_models", 65),
    "n_dev_128": lambda w: setattr(w, "n_dev", 128),
    "n_wf_zero": lambda w: setattr(w, "n_wf", 0),
    "pred_self_loop": lambda w: w.pred_idx.__setitem__(0, int(np.nonzero(np.diff(w.pred_off))[0][0])),
    "pred_off_nonzero_start": lambda w: w.pred_off.__setitem__(0, 1),
    "model_out_of_range": lambda w: w.act_model.__setitem__(0, w.n_models),
    "wf_out_of_range": lambda w: w.act_wf.__setitem__(0, -1),
    "latency_below_minus_one": lambda w: w.lat_us.__setitem__(0, -2),
    "negative_memory": lambda w: w.mem_mib.__setitem__(0, -5),
    "huge_memory": lambda w: w.mem_mib.__setitem__(0, (1 << 28) + 1),
    "negative_arrival": lambda w: w.wf_arrival_us.__setitem__(0, -1),
    "negative_load": lambda w: w.load_us.__setitem__(0, -1),
    "cap_too_big": lambda w: w.dev_cap_mib.__setitem__(0, (1 << 30) + 1),
    "resident_unknown_model": lambda w: w.init_resident.__setitem__(0, np.uint64(1 << 10)),
    "resident_over_capacity": lambda w: (w.model_mib.__setitem__(0, 30000),
                                         w.init_resident.__setitem__(0, np.uint64(1))),
    "negative_weight": lambda w: setattr(w, "w_p95", -0.5),
    "nan_weight": lambda w: setattr(w, "w_makespan", float("nan")),
    "empty_workflow": lambda w: (setattr(w, "n_wf", 3), setattr(w, "wf_arrival_us", np.zeros(3, np.int64))),
    "negative_free0": lambda w: w.dev_free0_us.__setitem__(0, -3),
    "class_out_of_range": lambda w: setattr(w, "wf_class",
                                            np.full(w.n_wf, pkg._lib.WF_MAX_CLASSES, np.uint8)),
    "victim_order_unknown": lambda w: setattr(w, "victim_order", 2),
    "batch_zero": lambda w: setattr(w, "dev_batch", np.zeros(w.n_dev, np.int32)),
    "batch_too_big": lambda w: setattr(w, "dev_batch", np.full(w.n_dev, pkg._lib.WF_MAX_BATCH + 1, np.int32)),
    "replica_cap_zero": lambda w: setattr(w, "model_replica_cap", np.zeros(w.n_models, np.int32)),
    "replica_cap_below_initial_copies": lambda w: (
        w.init_resident.__setitem__(slice(None), np.uint64(1)),
        w.dev_cap_mib.__setitem__(slice(None), 1 << 29),
        setattr(w, "model_replica_cap", np.ones(w.n_models, np.int32))),
    "prefetch_slack_negative": lambda w: setattr(w, "prefetch_slack_us", -1),
    "prefetch_slack_too_big": lambda w: setattr(w, "prefetch_slack_us", (1 << 52) + 1),
}


@pytest.mark.parametrize("name", sorted(BAD))
def test_invalid_windows_rejected(name):
    w = _mutate(BAD[name])
    st, msg = pkg.wf_plan_validate_window(w)
    assert st == pkg.WF_EINVAL and msg, (name, st, msg)


def test_prefetch_slack_limits_accepted():
    for slack in (0, 1, 1 << 52):
        w = _mutate(lambda w: setattr(w, "prefetch_slack_us", slack))
        assert pkg.wf_plan_validate_window(w)[0] == pkg.WF_OK


def test_not_level_sorted_rejected():
    # activation 1 depends on 0 (level 1); activation 2 is a source (level 0)
    w = W.Window(n_act=3, n_wf=1, n_models=1, n_dev=1, act_wf=np.zeros(3, np.int32),
                 act_model=np.zeros(3, np.int32), pred_off=np.array([0, 0, 1, 1], np.int32),
                 pred_idx=np.array([0], np.int32), lat_us=np.ones(3, np.int32),
                 mem_mib=np.ones(3, np.int32), wf_arrival_us=np.zeros(1, np.int64),
                 dev_cap_mib=np.array([100], np.int32), model_mib=np.array([10], np.int32),
                 load_us=np.array([5], np.int32), init_resident=np.zeros(1, np.uint64),
                 dev_free0_us=np.zeros(1, np.int64))
    st, msg = pkg.wf_plan_validate_window(w)
    assert st == pkg.WF_EINVAL and "level" in msg
    w.pred_off = np.array([0, 0, 0, 1], np.int32)  # 2 depends on 0: sorted
    assert pkg.wf_plan_validate_window(w)[0] == pkg.WF_OK


def test_duplicate_predecessor_rejected():
    w = W.make_window(1)
    row = int(np.nonzero(np.diff(w.pred_off) >= 2)[0][0])
    w.pred_idx = w.pred_idx.copy()
    w.pred_idx[w.pred_off[row] + 1] = w.pred_idx[w.pred_off[row]]
    st, msg = pkg.wf_plan_validate_window(w)
    assert st == pkg.WF_EINVAL and "increasing" in msg


def test_empty_window_is_valid():
    w = W.Window(n_act=0, n_wf=0, n_models=1, n_dev=1, act_wf=np.zeros(0, np.int32),
                 act_model=np.zeros(0, np.int32), pred_off=np.zeros(1, np.int32),
                 pred_idx=np.zeros(0, np.int32), lat_us=np.zeros(0, np.int32),
                 mem_mib=np.zeros(0, np.int32), wf_arrival_us=np.zeros(0, np.int64),
                 dev_cap_mib=np.array([10], np.int32), model_mib=np.array([1], np.int32),
                 load_us=np.zeros(1, np.int32), init_resident=np.zeros(1, np.uint64),
                 dev_free0_us=np.zeros(1, np.int64))
    assert pkg.wf_plan_validate_window(w)[0] == pkg.WF_OK


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError):
        _lib.load(str(tmp_path / "missing.so"))


def test_device_buffers_are_row_major():
    """Plan buffers handed to the library are dense row-major even when the
    host arrays are not (a Fortran-ordered priority array once reached the
    kernel transposed)."""
    import torch
    rng = np.random.default_rng(3)
    win = W.random_window(rng)
    plans = W.random_plans(win, 7, rng, prio_mode="globalperm")
    fortran = W.PlanBatch(np.asfortranarray(plans.dev), np.asfortranarray(plans.prio),
                          np.asfortranarray(plans.flags))
    dev, prio, flags = pkg.device_plans(fortran, "cpu")
    for t, a in ((dev, plans.dev), (prio, plans.prio.view(np.int16)), (flags, plans.flags)):
        assert t.is_contiguous()
        assert t.numpy().tobytes() == np.ascontiguousarray(a).tobytes()
    with pytest.raises(ValueError):
        _lib._ptr(torch.zeros((4, 3), dtype=torch.int16).t())


def _struct_fields(name):
    """Member names of `typedef struct { ... } name;` in the header, in order."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    m = re.search(r"typedef struct\s*\{([^}]*)\}\s*" + name + r"\s*;", text)
    assert m, name
    out = []
    for decl in m.group(1).split(";"):
        decl = decl.strip()
        if not decl:
            continue
        # "const int32_t *a, *b" or "float w_makespan, w_p95" or "uint16_t admitted[4]"
        head, *rest = decl.split(",")
        names = [head.split()[-1]] + [r.strip() for r in rest]
        out += [re.sub(r"[\*\s]|\[.*\]", "", n) for n in names]
    return out


@pytest.mark.parametrize("name", ["wf_window_desc", "wf_plan_sched"])
def test_binding_structs_follow_the_header(name):
    """The ctypes mirrors list the header's members in the header's order."""
    py = [f[0] for f in getattr(_lib, name)._fields_]
    assert py == _struct_fields(name)


class _FakeGpuTensor:
    """Stands in for a torch CUDA tensor on a machine without a GPU: the
    binding's checks read only these attributes."""

    class _Dev:
        def __init__(self, index):
            self.index = index

    def __init__(self, nbytes, index=0, cuda=True, contiguous=True):
        self._n, self.is_cuda, self._c = nbytes, cuda, contiguous
        self.device = self._Dev(index)

    def is_contiguous(self):
        return self._c

    def numel(self):
        return self._n

    def element_size(self):
        return 1

    def data_ptr(self):
        return 0x7f0000000000


def test_buffer_checks_before_the_library():
    """A host tensor, a tensor on another GPU, a strided tensor or one too
    small for the call never reach the kernels as an address."""
    import torch
    with pytest.raises(ValueError, match="host tensor"):
        _lib._buf(torch.zeros(64, dtype=torch.uint8), 32, 0, "scores")
    with pytest.raises(ValueError, match="cuda:1"):
        _lib._buf(_FakeGpuTensor(64, index=1), 32, 0, "scores")
    with pytest.raises(ValueError, match="contiguous"):
        _lib._buf(_FakeGpuTensor(64, contiguous=False), 32, 0, "scores")
    with pytest.raises(ValueError, match="at least 64"):
        _lib._buf(_FakeGpuTensor(63), 64, 0, "scores")
    assert _lib._buf(_FakeGpuTensor(64), 64, 0, "scores") == 0x7f0000000000
    assert _lib._buf(None, 64, 0, "scores") is None
    assert _lib._buf(0x1000, 64, 0, "scores") == 0x1000  # a raw address is the caller's


def test_context_methods_size_buffers_from_the_window(monkeypatch):
    """Each Context method asks for the bytes the uploaded window implies:
    a [P][N] schedule array one row short is refused before the call."""
    class _NoLib:  # any call reaching the library fails the test
        def __getattr__(self, name):
            def call(*a):
                raise AssertionError(f"{name} reached the library")
            return call
    ctx = _lib.Context.__new__(_lib.Context)
    ctx.lib, ctx.handle, ctx.device, ctx._nd = _NoLib(), None, 0, (10, 3)
    P = 4
    rows = (_FakeGpuTensor(P * 10), _FakeGpuTensor(2 * P * 10), _FakeGpuTensor(P * 3))
    ok_sched = [_FakeGpuTensor(8 * P * 10)] * 3 + [_FakeGpuTensor(4 * P * 3)]
    short = list(ok_sched)
    short[1] = _FakeGpuTensor(8 * (P - 1) * 10)
    with pytest.raises(ValueError, match="finish_us"):
        ctx.wf_plan_score_batch(*rows, P, _FakeGpuTensor(32 * P), short)
    with pytest.raises(ValueError, match="scores"):
        ctx.wf_plan_score_batch(*rows, P, _FakeGpuTensor(32 * P - 1))
    with pytest.raises(ValueError, match="prio"):
        ctx.wf_plan_score_keys(rows[0], _FakeGpuTensor(2 * P * 10 - 2), rows[2], P,
                               _FakeGpuTensor(32 * P))
    with pytest.raises(ValueError, match="peak_mib"):
        ctx.wf_plan_score_batch(*rows, P, _FakeGpuTensor(32 * P),
                                ok_sched[:3] + [_FakeGpuTensor(4 * P * 3 - 4)])
    with pytest.raises(ValueError, match="out_dev"):
        ctx.wf_plan_search_rows(_FakeGpuTensor(10), _FakeGpuTensor(20), _FakeGpuTensor(3), 1, 1, 0,
                                5, _FakeGpuTensor(49), _FakeGpuTensor(100), _FakeGpuTensor(15))


def test_noalloc_argmin_argument_errors_without_gpu():
    """Argument errors of the allocation-free argmin are found on the host,
    before any HIP call."""
    lib = _lib.load()
    assert lib.wf_plan_argmin_noalloc(None, -1, 0x1000, None) == _lib.WF_EINVAL
    assert lib.wf_plan_argmin_noalloc(0x1000, 1 << 32, 0x1000, None) == _lib.WF_EINVAL
    assert b"2^32" in lib.wf_plan_last_error(None)
    assert lib.wf_plan_argmin_noalloc(0x1000, 5, None, None) == _lib.WF_EINVAL
    assert lib.wf_plan_argmin_noalloc(None, 5, 0x1000, None) == _lib.WF_EINVAL


def test_score_kernel_without_window():
    assert _lib.load().wf_plan_score_kernel(None) == b""


@pytest.mark.parametrize("D", [65, 96, 127])
def test_pools_up_to_127_devices_validate(D):
    """Plans carry int8 device ids: pools of up to 127 devices are valid."""
    rng = np.random.default_rng(D)
    st, msg = pkg.wf_plan_validate_window(W.random_window(rng, n_dev=D, n_models=20))
    assert st == pkg.WF_OK, msg

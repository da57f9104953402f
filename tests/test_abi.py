"""Host-side checks of libckm that need no GPU: the library loads, exports
every function include/ckm.h declares, and rejects malformed graphs and
arguments before touching the device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from paper_1910_02653_amd import ckm

HEADER = os.path.join(ROOT, "include", "ckm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ckm_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert set(names) == set(ckm.EXPORTS)
    L = ckm.lib()
    for name in names:
        assert hasattr(L, name), name


def test_no_torch_types_in_header():
    text = open(HEADER).read()
    assert "torch" not in re.sub(r"/\*.*?\*/", "", text, flags=re.S)


def create(n, deps, cost=None, size=None, m_input=0, m_param=0, users=None):
    ptr = np.zeros(n + 1, np.int32)
    flat = []
    for j, d in enumerate(deps):
        flat.extend(d)
        ptr[j + 1] = len(flat)
    idx = np.asarray(flat if flat else [0], np.int32)
    cost = np.ones(n, np.int64) if cost is None else np.asarray(cost, np.int64)
    size = np.ones(n, np.int64) if size is None else np.asarray(size, np.int64)
    h = C.c_void_p()
    up = ui = None
    if users is not None:
        up = np.zeros(n + 1, np.int32)
        uf = []
        for i, u in enumerate(users):
            uf.extend(u)
            up[i + 1] = len(uf)
        ui = np.asarray(uf if uf else [0], np.int32)
    st = ckm.lib().ckm_graph_create(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p),
                                    None if up is None else up.ctypes.data_as(C.c_void_p),
                                    None if ui is None else ui.ctypes.data_as(C.c_void_p),
                                    cost.ctypes.data_as(C.c_void_p), size.ctypes.data_as(C.c_void_p),
                                    m_input, m_param, C.byref(h))
    return st, h


@pytest.mark.parametrize("case,status", [
    (dict(n=0, deps=[]), ckm.E_INVALID_ARG),
    (dict(n=4097, deps=[[]] * 4097), ckm.E_UNSUPPORTED),
    (dict(n=3, deps=[[], [1], []]), ckm.E_GRAPH),             # self edge
    (dict(n=3, deps=[[], [2], []]), ckm.E_GRAPH),             # forward in numbering
    (dict(n=3, deps=[[], [0], [1, 1]]), ckm.E_GRAPH),         # duplicate
    (dict(n=3, deps=[[], [0], [-1]]), ckm.E_GRAPH),           # out of range
    (dict(n=3, deps=[[], [0], [1]], users=[[1], [], [2]]), ckm.E_GRAPH),   # users != transpose
    (dict(n=3, deps=[[], [0], [1]], users=[[2], [1], []]), ckm.E_GRAPH),
    (dict(n=2, deps=[[], [0]], cost=[1, -1]), ckm.E_INVALID_ARG),
    (dict(n=2, deps=[[], [0]], size=[-5, 1]), ckm.E_INVALID_ARG),
    (dict(n=2, deps=[[], [0]], m_param=-1), ckm.E_INVALID_ARG),
    (dict(n=2, deps=[[], [0]], size=[2 ** 62, 2 ** 62]), ckm.E_OVERFLOW),      # sum M past INT64_MAX
    (dict(n=2, deps=[[], [0]], size=[2 ** 62 - 1, 2 ** 62 - 1], m_input=2), ckm.E_OVERFLOW),
    (dict(n=2, deps=[[], [0]], size=[1, 1], m_param=2 ** 62), ckm.E_OVERFLOW),  # 2 M_param
    (dict(n=2, deps=[[], [0]], cost=[2 ** 63 - 1, 1]), ckm.E_OVERFLOW),        # sum C
    (dict(n=4096, deps=[[]] * 4096, cost=[2 ** 52] + [0] * 4095), ckm.E_OVERFLOW),  # n * sum C
    (dict(n=7, deps=[[]] * 7, cost=[(2 ** 63 - 1) // 7 + 1] + [0] * 6), ckm.E_OVERFLOW),
])
def test_graph_validation_errors(case, status):
    st, h = create(**case)
    assert st == status, ckm.last_error()
    assert not h.value
    assert ckm.last_error()


@pytest.mark.parametrize("case", [
    dict(n=2, deps=[[], [0]], size=[2 ** 62 - 1, 2 ** 62 - 1], m_input=1),    # M_in + sum M = INT64_MAX
    dict(n=2, deps=[[], [0]], size=[1, 2 ** 62], m_param=2 ** 61 - 1),       # 2 M_param counted twice
    dict(n=1, deps=[[]], cost=[2 ** 63 - 1]),                                # n sum C = INT64_MAX
    dict(n=7, deps=[[]] * 7, cost=[(2 ** 63 - 1) // 7] + [0] * 6),
    dict(n=3, deps=[[], [0], [1]], size=[2 ** 55, 3, 2 ** 53 + 1], cost=[2 ** 58, 1, 2 ** 53]),
])
def test_graph_totals_up_to_int64_max_accepted(case):
    """Only totals beyond INT64_MAX are refused: a graph at the limit passes
    validation (here it then needs a device, which a CPU-only host lacks)."""
    st, h = create(**case)
    assert st != ckm.E_OVERFLOW, ckm.last_error()
    assert st in (ckm.OK, ckm.E_DEVICE), ckm.last_error()
    if h.value:
        ckm.lib().ckm_graph_destroy(h)


def test_edge_count_checked_before_the_edges_are_read():
    """dep_ptr[n] above n(n-1)/2 is rejected before dep_idx (one entry here)
    is read or anything is sized by it."""
    n = 3
    ptr = np.array([0, 0, 0, 2 ** 31 - 1], np.int32)
    idx = np.zeros(1, np.int32)
    ones = np.ones(n, np.int64)
    h = C.c_void_p()
    st = ckm.lib().ckm_graph_create(n, ptr.ctypes.data_as(C.c_void_p), idx.ctypes.data_as(C.c_void_p), None, None,
                                    ones.ctypes.data_as(C.c_void_p), ones.ctypes.data_as(C.c_void_p), 0, 0,
                                    C.byref(h))
    assert st == ckm.E_GRAPH and not h.value
    assert "edges" in ckm.last_error()


def test_null_arguments_rejected():
    L = ckm.lib()
    h = C.c_void_p()
    assert L.ckm_graph_create(2, None, None, None, None, None, None, 0, 0, C.byref(h)) == ckm.E_INVALID_ARG
    assert L.ckm_graph_create(2, None, None, None, None, None, None, 0, 0, None) == ckm.E_INVALID_ARG
    sz = C.c_size_t()
    assert L.ckm_workspace_size(None, 4, C.byref(sz)) == ckm.E_INVALID_ARG
    assert L.ckm_workspace_size_min(None, 4, C.byref(sz)) == ckm.E_INVALID_ARG
    assert L.ckm_round_eval(None, None, 0, 4, 0, 0, 0, None, None, None, None, None, None) == ckm.E_INVALID_ARG
    assert L.ckm_evaluate_async(None, 4, 0, 0, 0, None, 0, None) == ckm.E_INVALID_ARG
    assert L.ckm_select_async(None, 4, 0, 0, 0, None, None, None, None, None, None, None, None, 0,
                              None) == ckm.E_INVALID_ARG
    assert L.ckm_quantize_async(None, None, 0, None, 0, None) == ckm.E_INVALID_ARG
    assert L.ckm_round_eval_async(None, None, 0, 4, 0, 0, 0, None, None, None, None, None, None, None, None,
                                  0, None) == ckm.E_INVALID_ARG
    assert L.ckm_eval_schedules(None, None, 4, 0, None, None, None, None, None) == ckm.E_INVALID_ARG
    assert L.ckm_eval_schedules_async(None, None, 4, 0, None, None, None, None, None, None, None, 0,
                                      None) == ckm.E_INVALID_ARG
    assert L.ckm_threshold_eval(None, None, 4, None, 4, 0, None, None, None, None, None, None) == ckm.E_INVALID_ARG
    assert L.ckm_threshold_eval_async(None, None, 4, None, 4, 0, None, None, None, None, None, None, None, None, 0,
                                      None) == ckm.E_INVALID_ARG
    assert L.ckm_plan(None, None, None, 0, None, 0, None, None) == ckm.E_INVALID_ARG
    assert L.ckm_plan_async(None, None, None, 0, None, 0, None, None, None, None, 0, None) == ckm.E_INVALID_ARG
    assert L.ckm_max_batch(None, None, 4, 4, 0, 0, 0, 0, None, None, None) == ckm.E_INVALID_ARG
    assert L.ckm_max_batch_async(None, 4, 0, 0, None, None, None, None, None, 0, None) == ckm.E_INVALID_ARG
    assert L.ckm_round_async(None, 4, 0, 0, None, 0, None) == ckm.E_INVALID_ARG
    assert L.ckm_graph_num_nodes(None) == -1
    L.ckm_graph_destroy(None)


def test_binding_checks_arrays_before_the_library_reads_them():
    """The binding passes bare pointers, so it checks shapes, dtypes and
    devices itself: an S* with fewer than n rows or columns, host tensors
    where device tensors belong, and short result tensors are refused."""
    import torch
    with pytest.raises(ValueError):
        ckm._host_s(np.zeros((4, 5)), 5)          # 4 rows, n = 5
    with pytest.raises(ValueError):
        ckm._host_s(np.zeros(25), 5)              # not 2-D
    assert ckm._host_s(np.zeros((5, 7), np.float32), 5).dtype == np.float64
    with pytest.raises(ValueError):
        ckm._dev_s(torch.zeros((5, 5), dtype=torch.float64), 5)   # host tensor
    with pytest.raises(ValueError):
        ckm._dev(torch.zeros(8, dtype=torch.int64), "peak", torch.int64, 8)
    with pytest.raises(ValueError):
        ckm._work(torch.zeros(64, dtype=torch.uint8))

"""Thin ctypes binding of libckm (include/ckm.h): argument marshalling only.

Every step of the path runs in the library's HIP kernels; this module only
converts numpy / torch arguments to pointers. It never falls back to another
implementation: if libckm.so is missing, loading raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libckm.so")

OK, E_INVALID_ARG, E_GRAPH, E_OVERFLOW, E_UNSUPPORTED, E_NOMEM, E_DEVICE = range(7)
F_DET0 = 1
F_ROUNDED = 2
MAX_NODES = 4096
MAX_CANDIDATES = 1 << 24
MAX_THRESHOLDS = 1 << 16

# every extern "C" symbol declared in include/ckm.h
EXPORTS = (
    "ckm_graph_create", "ckm_graph_destroy", "ckm_graph_num_nodes", "ckm_round_eval",
    "ckm_workspace_size", "ckm_workspace_size_min", "ckm_quantize_async", "ckm_round_async",
    "ckm_evaluate_async", "ckm_select_async", "ckm_round_eval_async", "ckm_eval_schedules", "ckm_eval_schedules_async", "ckm_threshold_eval",
    "ckm_threshold_eval_async", "ckm_plan", "ckm_plan_async", "ckm_max_batch",
    "ckm_max_batch_async", "ckm_round_eval_noalloc", "ckm_last_error",
)
NOALLOC_SCRATCH_BYTES = 256 << 20
PLAN_EARLY_FREE = 1
OP_COMPUTE, OP_DEALLOCATE = 0, 1


class CkmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("ckm status %d: %s" % (status, msg))
        self.status = status


_lib = None


def lib():
    """Load libckm.so (built by __graft_entry__.build() / build.py)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libckm.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        # torch ships its own HIP runtime with the same soname (libamdhip64.so.7).
        # Loading torch first makes libckm bind to that runtime, so the process
        # has one HIP runtime and torch's streams and allocations are valid in
        # libckm's calls. Loaded the other way round, two runtimes would coexist.
        import torch  # noqa: F401
        L = C.CDLL(LIB_PATH)
        p, i32, i64, u32, u64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_size_t
        L.ckm_graph_create.argtypes = [i32, p, p, p, p, p, p, i64, i64, C.POINTER(p)]
        L.ckm_graph_create.restype = C.c_int
        L.ckm_graph_destroy.argtypes = [p]
        L.ckm_graph_destroy.restype = None
        L.ckm_graph_num_nodes.argtypes = [p]
        L.ckm_graph_num_nodes.restype = i32
        L.ckm_round_eval.argtypes = [p, p, i64, i32, u64, i64, u32, p, p, p, p, p, p]
        L.ckm_round_eval.restype = C.c_int
        L.ckm_workspace_size.argtypes = [p, i32, C.POINTER(sz)]
        L.ckm_workspace_size.restype = C.c_int
        L.ckm_workspace_size_min.argtypes = [p, i32, C.POINTER(sz)]
        L.ckm_workspace_size_min.restype = C.c_int
        L.ckm_quantize_async.argtypes = [p, p, i64, p, sz, p]
        L.ckm_quantize_async.restype = C.c_int
        L.ckm_round_async.argtypes = [p, i32, u64, u32, p, sz, p]
        L.ckm_round_async.restype = C.c_int
        L.ckm_evaluate_async.argtypes = [p, i32, u64, u32, i32, p, sz, p]
        L.ckm_evaluate_async.restype = C.c_int
        L.ckm_select_async.argtypes = [p, i32, u64, i64, u32, p, p, p, p, p, p, p, p, sz, p]
        L.ckm_select_async.restype = C.c_int
        L.ckm_round_eval_async.argtypes = [p, p, i64, i32, u64, i64, u32, p, p, p, p, p, p, p, p, sz, p]
        L.ckm_round_eval_async.restype = C.c_int
        L.ckm_round_eval_noalloc.argtypes = [p, p, i64, i32, u64, i64, u32, p, p, p, p, p, p, p, p]
        L.ckm_round_eval_noalloc.restype = C.c_int
        L.ckm_eval_schedules.argtypes = [p, p, i32, i64, p, p, p, p, p]
        L.ckm_eval_schedules.restype = C.c_int
        L.ckm_eval_schedules_async.argtypes = [p, p, i32, i64, p, p, p, p, p, p, p, sz, p]
        L.ckm_eval_schedules_async.restype = C.c_int
        L.ckm_threshold_eval.argtypes = [p, p, i64, p, i32, i64, p, p, p, p, p, p]
        L.ckm_threshold_eval.restype = C.c_int
        L.ckm_threshold_eval_async.argtypes = [p, p, i64, p, i32, i64, p, p, p, p, p, p, p, p, sz, p]
        L.ckm_threshold_eval_async.restype = C.c_int
        L.ckm_plan.argtypes = [p, p, p, u32, p, i64, p, p]
        L.ckm_plan.restype = C.c_int
        L.ckm_plan_async.argtypes = [p, p, p, u32, p, i64, p, p, p, p, sz, p]
        L.ckm_plan_async.restype = C.c_int
        L.ckm_max_batch.argtypes = [p, p, i64, i32, u64, u32, i64, i64, p, p, p]
        L.ckm_max_batch.restype = C.c_int
        L.ckm_max_batch_async.argtypes = [p, i32, i64, i64, p, p, p, p, p, sz, p]
        L.ckm_max_batch_async.restype = C.c_int
        L.ckm_last_error.argtypes = []
        L.ckm_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().ckm_last_error().decode()


def _check(status: int):
    if status != OK:
        raise CkmError(status, last_error())


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)



def _host_s(s_frac, n: int) -> np.ndarray:
    """S* as a C-contiguous float64 array with at least n rows and n columns
    (the library reads n rows of stride shape[1])."""
    s = np.ascontiguousarray(s_frac, dtype=np.float64)
    if s.ndim != 2 or s.shape[0] < n or s.shape[1] < n:
        raise ValueError("S* must be a 2-D array of at least [%d][%d], got shape %s" % (n, n, s.shape))
    return s


def _dev(t, name: str, dtype, numel: int = 0):
    """Pointer of a contiguous device tensor of the given dtype holding at
    least numel elements (the library cannot check sizes behind a pointer)."""
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.numel() < numel:
        raise ValueError("%s holds %d elements, %d needed" % (name, t.numel(), numel))
    return C.c_void_p(t.data_ptr())


def _dev_s(t, n: int):
    """(pointer, row stride) of a float64 device S* with at least n x n
    entries and unit column stride."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float64 or t.dim() != 2:
        raise ValueError("S* must be a 2-D float64 device tensor")
    if t.shape[0] < n or t.shape[1] < n or (n > 1 and t.stride(1) != 1) or t.stride(0) < n:
        raise ValueError("S* must hold at least [%d][%d] entries in rows of unit column stride, got shape %s, "
                         "strides %s" % (n, n, tuple(t.shape), t.stride()))
    return C.c_void_p(t.data_ptr()), t.stride(0)


def _work(work):
    import torch
    if not isinstance(work, torch.Tensor) or not work.is_cuda or not work.is_contiguous():
        raise ValueError("work must be a contiguous device tensor")
    return C.c_void_p(work.data_ptr()), work.numel() * work.element_size()


def _stream_ptr(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


class Graph:
    """A graph uploaded to the current HIP device (ckm_graph_create)."""

    def __init__(self, n, dep_ptr, dep_idx, cost, size, m_input, m_param, user_ptr=None, user_idx=None):
        dp = np.ascontiguousarray(dep_ptr, dtype=np.int32)
        di = np.ascontiguousarray(dep_idx, dtype=np.int32)
        up = None if user_ptr is None else np.ascontiguousarray(user_ptr, dtype=np.int32)
        ui = None if user_idx is None else np.ascontiguousarray(user_idx, dtype=np.int32)
        c = np.ascontiguousarray(cost, dtype=np.int64)
        s = np.ascontiguousarray(size, dtype=np.int64)
        h = C.c_void_p()
        self._h = None
        _check(lib().ckm_graph_create(int(n), _np_ptr(dp), _np_ptr(di) if di.size else None, _np_ptr(up),
                                      _np_ptr(ui) if (ui is not None and ui.size) else None, _np_ptr(c),
                                      _np_ptr(s), int(m_input), int(m_param), C.byref(h)))
        self._h = h
        self.n = int(n)
        self.W = (self.n + 63) // 64

    @classmethod
    def from_workload(cls, w) -> "Graph":
        return cls(w.n, w.dep_ptr, w.dep_idx, w.cost, w.size, w.m_input, w.m_param)

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h is not None and self._h.value:
            lib().ckm_graph_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_size(self, K: int, rows: bool = True) -> int:
        """Work-buffer bytes for K candidates; rows=False: the smallest
        accepted size, without the row array."""
        out = C.c_size_t()
        fn = lib().ckm_workspace_size if rows else lib().ckm_workspace_size_min
        _check(fn(self._h, int(K), C.byref(out)))
        return int(out.value)

    # -- synchronous, host arrays -----------------------------------------
    def round_eval(self, s_frac, K: int, seed: int, budget: int, flags: int = 0, want_rows: bool = True):
        s = _host_s(s_frac, self.n)
        peak = np.zeros(K, np.int64)
        cost = np.zeros(K, np.int64)
        feas = np.zeros(K, np.uint8)
        bk = np.zeros(1, np.int32)
        bS = np.zeros((self.n, self.W), np.uint64) if want_rows else None
        bR = np.zeros((self.n, self.W), np.uint64) if want_rows else None
        _check(lib().ckm_round_eval(self._h, _np_ptr(s), s.shape[1], int(K), int(seed), int(budget), int(flags),
                                    _np_ptr(peak), _np_ptr(cost), _np_ptr(feas), _np_ptr(bk), _np_ptr(bS),
                                    _np_ptr(bR)))
        return dict(peak=peak, cost=cost, feasible=feas, best_k=int(bk[0]), best_S=bS, best_R=bR)

    def threshold_eval(self, s_frac, p, budget: int, want_rows: bool = True):
        """One deterministic candidate per threshold p_k (ckm_threshold_eval)."""
        s = _host_s(s_frac, self.n)
        pk = np.ascontiguousarray(p, dtype=np.float64).reshape(-1)
        K = pk.size
        peak = np.zeros(K, np.int64)
        cost = np.zeros(K, np.int64)
        feas = np.zeros(K, np.uint8)
        bk = np.zeros(1, np.int32)
        bS = np.zeros((self.n, self.W), np.uint64) if want_rows else None
        bR = np.zeros((self.n, self.W), np.uint64) if want_rows else None
        _check(lib().ckm_threshold_eval(self._h, _np_ptr(s), s.shape[1], _np_ptr(pk), int(K), int(budget),
                                        _np_ptr(peak), _np_ptr(cost), _np_ptr(feas), _np_ptr(bk), _np_ptr(bS),
                                        _np_ptr(bR)))
        return dict(peak=peak, cost=cost, feasible=feas, best_k=int(bk[0]), best_S=bS, best_R=bR)

    def max_batch(self, s_frac, K: int, seed: int, budget: int, cost_cap: int, flags: int = 0):
        """Largest batch multiplier of each rounded candidate (ckm_max_batch)."""
        s = _host_s(s_frac, self.n)
        batch = np.zeros(K, np.int64)
        bk = np.zeros(1, np.int32)
        bb = np.zeros(1, np.int64)
        _check(lib().ckm_max_batch(self._h, _np_ptr(s), s.shape[1], int(K), int(seed), int(flags), int(budget),
                                   int(cost_cap), _np_ptr(batch), _np_ptr(bk), _np_ptr(bb)))
        return dict(batch=batch, best_k=int(bk[0]), best_batch=int(bb[0]))

    def max_batch_async(self, K, budget, cost_cap, d_batch, d_best_k, d_best_batch, d_status, work, stream=None):
        import torch
        wp, wb = _work(work)
        _check(lib().ckm_max_batch_async(self._h, int(K), int(budget), int(cost_cap),
                                         _dev(d_batch, "batch", torch.int64, K), _dev(d_best_k, "best_k", torch.int32, 1),
                                         _dev(d_best_batch, "best_batch", torch.int64, 1),
                                         _dev(d_status, "status", torch.int32, 1), wp, wb, _stream_ptr(stream)))

    def plan(self, S_rows, R_rows, early: bool = False, capacity=None, want_mem: bool = True):
        """Algorithm 1's execution plan of (S, R) bit rows (ckm_plan): statements
        [count][4] int32 (op, node, register, stage) and the memory after each.
        capacity None: ask for the count first."""
        S = np.ascontiguousarray(S_rows, dtype=np.uint64)
        R = np.ascontiguousarray(R_rows, dtype=np.uint64)
        if S.shape != (self.n, self.W) or R.shape != (self.n, self.W):
            raise ValueError("S and R must have shape [%d][%d]" % (self.n, self.W))
        flags = PLAN_EARLY_FREE if early else 0
        cnt = np.zeros(1, np.int64)
        if capacity is None:
            _check(lib().ckm_plan(self._h, _np_ptr(S), _np_ptr(R), flags, None, 0, _np_ptr(cnt), None))
            capacity = int(cnt[0])
        P = np.zeros((max(int(capacity), 1), 4), np.int32)
        mem = np.zeros(max(int(capacity), 1), np.int64) if want_mem else None
        _check(lib().ckm_plan(self._h, _np_ptr(S), _np_ptr(R), flags, _np_ptr(P), int(capacity), _np_ptr(cnt),
                              _np_ptr(mem)))
        c = int(cnt[0])
        return P[:c].copy(), (mem[:c].copy() if want_mem else None)

    def plan_async(self, d_S, d_R, early, d_P, capacity, d_count, d_mem, d_status, work, stream=None):
        """Device tensors: d_S, d_R int64 [n][W]; d_P int32 [capacity][4] or None."""
        import torch
        rows = self.n * self.W
        cap = int(capacity) if d_P is not None else 0
        wp, wb = _work(work)
        _check(lib().ckm_plan_async(self._h, _dev(d_S, "S", torch.int64, rows), _dev(d_R, "R", torch.int64, rows),
                                    PLAN_EARLY_FREE if early else 0, _dev(d_P, "P", torch.int32, 4 * cap),
                                    int(capacity), _dev(d_count, "count", torch.int64, 1),
                                    _dev(d_mem, "mem", torch.int64, cap), _dev(d_status, "status", torch.int32, 1),
                                    wp, wb, _stream_ptr(stream)))

    def eval_schedules(self, S_rows, budget: int, want_rows: bool = True):
        """K given checkpoint matrices as uint64 bit rows [K][n][W] (ckm_eval_schedules)."""
        S = np.ascontiguousarray(S_rows, dtype=np.uint64)
        if S.ndim != 3 or S.shape[1:] != (self.n, self.W):
            raise ValueError("S_rows must have shape [K][%d][%d]" % (self.n, self.W))
        K = S.shape[0]
        peak = np.zeros(K, np.int64)
        cost = np.zeros(K, np.int64)
        feas = np.zeros(K, np.uint8)
        bk = np.zeros(1, np.int32)
        bR = np.zeros((self.n, self.W), np.uint64) if want_rows else None
        _check(lib().ckm_eval_schedules(self._h, _np_ptr(S), int(K), int(budget), _np_ptr(peak), _np_ptr(cost),
                                        _np_ptr(feas), _np_ptr(bk), _np_ptr(bR)))
        return dict(peak=peak, cost=cost, feasible=feas, best_k=int(bk[0]), best_R=bR)

    # -- asynchronous, torch device tensors ---------------------------------
    def _out(self, out: dict, K: int):
        """Pointers of the result tensors (see alloc_outputs) for K candidates."""
        import torch
        rows = self.n * self.W
        return (_dev(out["peak"], "peak", torch.int64, K), _dev(out["cost"], "cost", torch.int64, K),
                _dev(out["feasible"], "feasible", torch.uint8, K), _dev(out["best_k"], "best_k", torch.int32, 1),
                _dev(out.get("best_S"), "best_S", torch.int64, rows), _dev(out.get("best_R"), "best_R", torch.int64, rows),
                _dev(out.get("status"), "status", torch.int32, 1))

    def quantize_async(self, d_s_frac, work, stream=None):
        sp, ld = _dev_s(d_s_frac, self.n)
        wp, wb = _work(work)
        _check(lib().ckm_quantize_async(self._h, sp, ld, wp, wb, _stream_ptr(stream)))

    def round_async(self, K, seed, flags, work, stream=None):
        wp, wb = _work(work)
        _check(lib().ckm_round_async(self._h, int(K), int(seed), int(flags), wp, wb, _stream_ptr(stream)))

    def evaluate_async(self, K, seed, flags, work, stage_splits: int = 0, stream=None):
        wp, wb = _work(work)
        _check(lib().ckm_evaluate_async(self._h, int(K), int(seed), int(flags), int(stage_splits), wp, wb,
                                        _stream_ptr(stream)))

    def select_async(self, K, seed, budget, flags, out: dict, work, stream=None):
        peak, cost, feas, bk, bS, bR, st = self._out(out, K)
        wp, wb = _work(work)
        _check(lib().ckm_select_async(self._h, int(K), int(seed), int(budget), int(flags), peak, cost, feas, bk,
                                      bS, bR, st, wp, wb, _stream_ptr(stream)))

    def round_eval_async(self, d_s_frac, K, seed, budget, flags, out: dict, work, stream=None):
        sp, ld = _dev_s(d_s_frac, self.n)
        peak, cost, feas, bk, bS, bR, st = self._out(out, K)
        wp, wb = _work(work)
        _check(lib().ckm_round_eval_async(self._h, sp, ld, int(K), int(seed), int(budget), int(flags), peak, cost,
                                          feas, bk, bS, bR, st, wp, wb, _stream_ptr(stream)))

    def round_eval_noalloc(self, d_s_frac, K, seed, budget, flags, out: dict, stream=None):
        """ckm_round_eval_async on the library's static per-device work area."""
        sp, ld = _dev_s(d_s_frac, self.n)
        peak, cost, feas, bk, bS, bR, st = self._out(out, K)
        _check(lib().ckm_round_eval_noalloc(self._h, sp, ld, int(K), int(seed), int(budget), int(flags), peak, cost,
                                            feas, bk, bS, bR, st, _stream_ptr(stream)))

    def eval_schedules_async(self, d_S, K, budget, out: dict, work, stream=None):
        """d_S: int64 device tensor holding K x n x W bit-row words."""
        import torch
        peak, cost, feas, bk, _, bR, st = self._out(out, K)
        wp, wb = _work(work)
        _check(lib().ckm_eval_schedules_async(self._h, _dev(d_S, "S", torch.int64, int(K) * self.n * self.W),
                                              int(K), int(budget), peak, cost, feas, bk, bR, st, wp, wb,
                                              _stream_ptr(stream)))

    def threshold_eval_async(self, d_s_frac, d_p, budget, out: dict, work, stream=None):
        """d_p: float64 device tensor of K thresholds."""
        import torch
        sp, ld = _dev_s(d_s_frac, self.n)
        K = int(d_p.numel())
        pp = _dev(d_p, "thresholds", torch.float64, K)
        peak, cost, feas, bk, bS, bR, st = self._out(out, K)
        wp, wb = _work(work)
        _check(lib().ckm_threshold_eval_async(self._h, sp, ld, pp, K, int(budget), peak, cost, feas, bk, bS, bR, st,
                                              wp, wb, _stream_ptr(stream)))

    def alloc_outputs(self, K: int, device="cuda", rows: bool = True) -> dict:
        """Device tensors for the async calls (torch: memory only)."""
        import torch
        W = self.W
        out = dict(peak=torch.empty(K, dtype=torch.int64, device=device),
                   cost=torch.empty(K, dtype=torch.int64, device=device),
                   feasible=torch.empty(K, dtype=torch.uint8, device=device),
                   best_k=torch.empty(1, dtype=torch.int32, device=device),
                   status=torch.empty(1, dtype=torch.int32, device=device))
        if rows:
            out["best_S"] = torch.empty((self.n, W), dtype=torch.int64, device=device)
            out["best_R"] = torch.empty((self.n, W), dtype=torch.int64, device=device)
        return out

    def alloc_work(self, K: int, device="cuda", rows: bool = True):
        import torch
        return torch.empty(self.workspace_size(K, rows), dtype=torch.uint8, device=device)


def rows_to_numpy(t) -> np.ndarray:
    """int64 device rows -> uint64 numpy bit rows."""
    return t.cpu().numpy().view(np.uint64)

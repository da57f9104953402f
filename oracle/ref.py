"""ctypes binding of the CPU oracle (test infrastructure only).

Only the test suite, the smoke entry point and the benchmark's CPU-baseline
leg may import this module. It loads oracle/libckm_ref.so, building it with
gcc when it is missing.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libckm_ref.so")
SOURCES = [os.path.join(HERE, "ckm_ref.c")]

OK, E_INVALID_ARG, E_GRAPH, E_OVERFLOW = 0, 1, 2, 3
F_DET0 = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C99, -O2)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared", "-o", tmp] + SOURCES + ["-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = C.CDLL(LIB_PATH)
        p = C.c_void_p
        L.ckm_ref_philox4x32_10.argtypes = [p, p, p]
        L.ckm_ref_philox4x32_10.restype = None
        L.ckm_ref_draw.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32]
        L.ckm_ref_draw.restype = C.c_uint32
        L.ckm_ref_validate_graph.argtypes = [C.c_int32, p, p, p, p, C.c_int64, C.c_int64]
        L.ckm_ref_validate_graph.restype = C.c_int
        L.ckm_ref_quantize.argtypes = [C.c_int32, p, C.c_int64, p]
        L.ckm_ref_quantize.restype = C.c_int
        L.ckm_ref_round_random.argtypes = [C.c_int32, p, C.c_uint64, C.c_uint32, p]
        L.ckm_ref_round_random.restype = None
        L.ckm_ref_round_det.argtypes = [C.c_int32, p, C.c_int64, p]
        L.ckm_ref_round_det.restype = None
        L.ckm_ref_round_threshold.argtypes = [C.c_int32, p, C.c_int64, C.c_double, p]
        L.ckm_ref_round_threshold.restype = C.c_int
        L.ckm_ref_check_schedule.argtypes = [C.c_int32, p, p, p, p]
        L.ckm_ref_check_schedule.restype = C.c_int
        L.ckm_ref_plan.argtypes = [C.c_int32, p, p, p, C.c_int64, C.c_int64, p, p, C.c_int, p, p, C.c_int64, p]
        L.ckm_ref_plan.restype = C.c_int
        L.ckm_ref_max_batch.argtypes = [C.c_int32, p, p, p, p, C.c_int64, C.c_int64, p, p, C.c_int64, C.c_int64,
                                        C.c_int64]
        L.ckm_ref_max_batch.restype = C.c_int64
        L.ckm_ref_solve_R.argtypes = [C.c_int32, p, p, p, p]
        L.ckm_ref_solve_R.restype = None
        L.ckm_ref_simulate.argtypes = [C.c_int32, p, p, p, p, C.c_int64, C.c_int64, p, p, p, p, p, p, p]
        L.ckm_ref_simulate.restype = None
        L.ckm_ref_eval_candidate.argtypes = [C.c_int32, p, p, p, p, C.c_int64, C.c_int64, p, C.c_int64, p,
                                             C.c_uint64, C.c_uint32, C.c_uint32, p, p, p, p]
        L.ckm_ref_eval_candidate.restype = C.c_int
        L.ckm_ref_round_eval.argtypes = [C.c_int32, p, p, p, p, C.c_int64, C.c_int64, p, C.c_int64, C.c_int32,
                                         C.c_uint64, C.c_int64, C.c_uint32, p, p, p, p, p, p]
        L.ckm_ref_round_eval.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _graph(w):
    ptr = np.ascontiguousarray(w.dep_ptr, dtype=np.int32)
    idx = np.ascontiguousarray(w.dep_idx, dtype=np.int32)
    if idx.size == 0:
        idx = np.zeros(1, dtype=np.int32)
    return ptr, idx, np.ascontiguousarray(w.cost, np.int64), np.ascontiguousarray(w.size, np.int64)


def philox4x32_10(key, ctr):
    k = np.asarray(key, dtype=np.uint32)
    c = np.asarray(ctr, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().ckm_ref_philox4x32_10(_ptr(k), _ptr(c), _ptr(out))
    return out


def draw(seed: int, k: int, t: int, i: int) -> int:
    return int(lib().ckm_ref_draw(seed, k, t, i))


def validate_graph(n, dep_ptr, dep_idx, cost, size, m_input, m_param) -> int:
    dp = np.ascontiguousarray(dep_ptr, np.int32)
    di = np.ascontiguousarray(dep_idx, np.int32) if len(dep_idx) else np.zeros(1, np.int32)
    return int(lib().ckm_ref_validate_graph(n, _ptr(dp), _ptr(di), _ptr(np.ascontiguousarray(cost, np.int64)),
                                            _ptr(np.ascontiguousarray(size, np.int64)), m_input, m_param))


def quantize(s_frac):
    s = np.ascontiguousarray(s_frac, dtype=np.float64)
    n = s.shape[0]
    q = np.zeros((n, n), dtype=np.uint32)
    st = lib().ckm_ref_quantize(n, _ptr(s), s.shape[1], _ptr(q))
    if st != OK:
        raise ValueError("quantize: status %d" % st)
    return q


def round_random(q, seed: int, k: int):
    q = np.ascontiguousarray(q, dtype=np.uint32)
    n = q.shape[0]
    S = np.zeros((n, n), dtype=np.uint8)
    lib().ckm_ref_round_random(n, _ptr(q), seed, k, _ptr(S))
    return S


def round_det(s_frac):
    s = np.ascontiguousarray(s_frac, dtype=np.float64)
    n = s.shape[0]
    S = np.zeros((n, n), dtype=np.uint8)
    lib().ckm_ref_round_det(n, _ptr(s), s.shape[1], _ptr(S))
    return S


def solve_R(w, S):
    ptr, idx, _, _ = _graph(w)
    S = np.ascontiguousarray(S, dtype=np.uint8)
    R = np.zeros_like(S)
    lib().ckm_ref_solve_R(w.n, _ptr(ptr), _ptr(idx), _ptr(S), _ptr(R))
    return R


def simulate(w, S, R):
    """-> dict(peak, cost, stage_peak[n], max_frees, U_end[n])."""
    ptr, idx, cost, size = _graph(w)
    S = np.ascontiguousarray(S, dtype=np.uint8)
    R = np.ascontiguousarray(R, dtype=np.uint8)
    peak = np.zeros(1, np.int64)
    tc = np.zeros(1, np.int64)
    sp = np.zeros(w.n, np.int64)
    ue = np.zeros(w.n, np.int64)
    mf = np.zeros(1, np.int32)
    lib().ckm_ref_simulate(w.n, _ptr(ptr), _ptr(idx), _ptr(cost), _ptr(size), w.m_input, w.m_param,
                           _ptr(S), _ptr(R), _ptr(peak), _ptr(tc), _ptr(sp), _ptr(mf), _ptr(ue))
    return dict(peak=int(peak[0]), cost=int(tc[0]), stage_peak=sp, max_frees=int(mf[0]), U_end=ue)


def eval_candidate(w, k: int, flags: int = 0, q=None, want_rows: bool = False):
    """-> (peak, cost[, S, R]) for candidate k of workload w."""
    ptr, idx, cost, size = _graph(w)
    s = np.ascontiguousarray(w.s_frac, np.float64)
    if q is None:
        q = quantize(s)
    q = np.ascontiguousarray(q, np.uint32)
    peak = np.zeros(1, np.int64)
    tc = np.zeros(1, np.int64)
    S = np.zeros((w.n, w.n), np.uint8) if want_rows else None
    R = np.zeros((w.n, w.n), np.uint8) if want_rows else None
    st = lib().ckm_ref_eval_candidate(w.n, _ptr(ptr), _ptr(idx), _ptr(cost), _ptr(size), w.m_input, w.m_param,
                                      _ptr(s), s.shape[1], _ptr(q), w.seed, k, flags, _ptr(peak), _ptr(tc),
                                      _ptr(S), _ptr(R))
    if st != OK:
        raise ValueError("eval_candidate: status %d" % st)
    if want_rows:
        return int(peak[0]), int(tc[0]), S, R
    return int(peak[0]), int(tc[0])


def round_threshold(s_frac, p: float):
    """S[t][i] = [clamp(S*[t][i], 0, 1) > p] for i < t (Section 5.1 at threshold p)."""
    s = np.ascontiguousarray(s_frac, dtype=np.float64)
    n = s.shape[0]
    S = np.zeros((n, n), dtype=np.uint8)
    st = lib().ckm_ref_round_threshold(n, _ptr(s), s.shape[1], float(p), _ptr(S))
    if st != OK:
        raise ValueError("round_threshold: status %d" % st)
    return S


def threshold_eval(w, p, budget=None):
    """One candidate per threshold p_k: deterministic rounding at p_k, then
    Algorithm 2, the simulation and the feasible argmin, as for supplied
    schedules. Adds the best candidate's S rows."""
    budget = w.budget if budget is None else budget
    Ss = [round_threshold(w.s_frac, pk) for pk in np.asarray(p, np.float64)]
    r = eval_schedules(w, Ss, budget)
    W = (w.n + 63) // 64
    r["best_S"] = pack_rows(Ss[r["best_k"]]) if r["best_k"] >= 0 else np.zeros((w.n, W), np.uint64)
    return r


def round_eval(w, K=None, seed=None, budget=None, flags: int = 0, want_rows: bool = True):
    """The whole batched path on the CPU. Returns a dict of numpy results."""
    K = w.K if K is None else K
    seed = w.seed if seed is None else seed
    budget = w.budget if budget is None else budget
    ptr, idx, cost, size = _graph(w)
    s = np.ascontiguousarray(w.s_frac, np.float64)
    W = (w.n + 63) // 64
    peak = np.zeros(K, np.int64)
    tc = np.zeros(K, np.int64)
    feas = np.zeros(K, np.uint8)
    bk = np.zeros(1, np.int32)
    bS = np.zeros((w.n, W), np.uint64) if want_rows else None
    bR = np.zeros((w.n, W), np.uint64) if want_rows else None
    st = lib().ckm_ref_round_eval(w.n, _ptr(ptr), _ptr(idx), _ptr(cost), _ptr(size), w.m_input, w.m_param,
                                  _ptr(s), s.shape[1], K, seed, budget, flags, _ptr(peak), _ptr(tc), _ptr(feas),
                                  _ptr(bk), _ptr(bS), _ptr(bR))
    if st != OK:
        raise ValueError("round_eval: status %d" % st)
    return dict(peak=peak, cost=tc, feasible=feas, best_k=int(bk[0]), best_S=bS, best_R=bR)


def eval_schedules(w, S_mats, budget: int):
    """Given checkpoint matrices (each n x n 0/1; only the strict lower
    triangle is used): Algorithm 2's R (Section 5.2), the U/FREE simulation
    (Section 4.4) and cost (Section 4.3) of each, feasibility peak <= budget,
    and the lexicographic minimum of (cost, peak, k) over feasible k (-1 if
    none) with its R rows."""
    peaks, costs, Rs = [], [], []
    for S in S_mats:
        S = np.tril(np.asarray(S, dtype=np.uint8), -1)
        R = solve_R(w, S)
        sim = simulate(w, S, R)
        peaks.append(sim["peak"])
        costs.append(sim["cost"])
        Rs.append(R)
    feas = [p <= budget for p in peaks]
    best = -1
    for k in range(len(peaks)):
        if feas[k] and (best < 0 or (costs[k], peaks[k], k) < (costs[best], peaks[best], best)):
            best = k
    W = (w.n + 63) // 64
    best_R = pack_rows(Rs[best]) if best >= 0 else np.zeros((w.n, W), np.uint64)
    return dict(peak=np.array(peaks, np.int64), cost=np.array(costs, np.int64),
                feasible=np.array(feas, np.uint8), best_k=best, best_R=best_R)


def check_schedule(w, S, R) -> int:
    ptr, idx, _, _ = _graph(w)
    S = np.ascontiguousarray(S, dtype=np.uint8)
    R = np.ascontiguousarray(R, dtype=np.uint8)
    return lib().ckm_ref_check_schedule(w.n, _ptr(ptr), _ptr(idx), _ptr(S), _ptr(R))


def plan(w, S, R, early: bool = False):
    """Algorithm 1's execution plan of (S, R): (stmts [count][4] int32 as
    (op, node, register, stage), mem [count] int64)."""
    ptr, idx, _, size = _graph(w)
    S = np.ascontiguousarray(S, dtype=np.uint8)
    R = np.ascontiguousarray(R, dtype=np.uint8)
    cap = int(2 * R.astype(np.int64).sum()) + 1
    stmts = np.zeros((cap, 4), np.int32)
    mem = np.zeros(cap, np.int64)
    cnt = np.zeros(1, np.int64)
    st = lib().ckm_ref_plan(w.n, _ptr(ptr), _ptr(idx), _ptr(size), w.m_input, w.m_param, _ptr(S), _ptr(R),
                            1 if early else 0, _ptr(stmts), _ptr(mem), cap, _ptr(cnt))
    if st != OK:
        raise ValueError("plan: status %d" % st)
    c = int(cnt[0])
    assert c <= cap
    return stmts[:c].copy(), mem[:c].copy()


def max_batch(w, S, R, budget: int, cost_cap: int, limit: int = 1 << 40) -> int:
    """Largest B with peak(B * M) <= budget and cost <= cost_cap, by search
    over the simulator (sizes scaled, M_input and M_param not)."""
    ptr, idx, cost, size = _graph(w)
    S = np.ascontiguousarray(S, dtype=np.uint8)
    R = np.ascontiguousarray(R, dtype=np.uint8)
    return int(lib().ckm_ref_max_batch(w.n, _ptr(ptr), _ptr(idx), _ptr(cost), _ptr(size), w.m_input, w.m_param,
                                       _ptr(S), _ptr(R), int(budget), int(cost_cap), int(limit)))


def pack_rows(X) -> np.ndarray:
    """n x n 0/1 matrix -> n x W uint64 bit rows (bit i%64 of word i/64)."""
    X = np.asarray(X, dtype=np.uint8)
    n = X.shape[0]
    W = (n + 63) // 64
    pad = np.zeros((n, W * 64), dtype=np.uint8)
    pad[:, :X.shape[1]] = X
    bits = np.packbits(pad.reshape(n, W, 64), axis=2, bitorder="little")
    return bits.view(np.uint64).reshape(n, W).copy()

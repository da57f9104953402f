"""Graph input forms the C ABI accepts: Deps rows in any order and an
explicit Users CSR (which must be the transpose of Deps, in any order).

Each graph is created twice, once from sorted rows with Users derived, once
with every Deps row reversed and an explicit Users CSR whose rows are
shuffled. Both must give the same bits on every entry point (rounding,
supplied schedules, threshold family, execution plan), and the unsorted
graph's results must equal the oracle's on that same unsorted graph.
"""
import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def unsorted_forms(w, seed):
    """(dep_idx with every row reversed, user_ptr, user_idx with rows shuffled)."""
    rng = np.random.default_rng(seed)
    n = w.n
    di = w.dep_idx.copy()
    for j in range(n):
        a, b = int(w.dep_ptr[j]), int(w.dep_ptr[j + 1])
        di[a:b] = di[a:b][::-1].copy()
    users = [[] for _ in range(n)]
    for j in range(n):
        for i in w.deps(j):
            users[int(i)].append(j)
    up, ui = [0], []
    for i in range(n):
        u = list(users[i])
        rng.shuffle(u)
        ui += u
        up.append(len(ui))
    return di, np.array(up, np.int32), np.array(ui, np.int32)


def graphs(w, seed):
    di, up, ui = unsorted_forms(w, seed)
    assert any(not np.all(np.diff(di[w.dep_ptr[j]:w.dep_ptr[j + 1]]) > 0) for j in range(w.n))
    g_sorted = ckm.Graph.from_workload(w)
    g_unsorted = ckm.Graph(w.n, w.dep_ptr, di, w.cost, w.size, w.m_input, w.m_param, user_ptr=up, user_idx=ui)
    return g_sorted, g_unsorted, w.replace(dep_idx=di)


def same(a, b):
    for key in a:
        if a[key] is None:
            assert b[key] is None
        elif isinstance(a[key], np.ndarray):
            assert np.array_equal(a[key], b[key]), key
        else:
            assert a[key] == b[key], key


WORKLOADS = [
    ("unet n=337", lambda: wl.config(3).replace(K=128)),
    ("wide random dag", lambda: wl.random_dag(150, seed=12, K=96, max_deg=12, window=150, max_size=1000,
                                              max_cost=1000, s_kind="uniform", budget_pct=60.0)),
]


@pytest.mark.parametrize("name,make", WORKLOADS, ids=[x[0] for x in WORKLOADS])
def test_unsorted_deps_and_explicit_users(name, make):
    w = make()
    g_s, g_u, wu = graphs(w, seed=w.n)
    try:
        # rounding path, at a budget where some candidates are feasible
        probe = g_s.round_eval(w.s_frac, w.K, w.seed, 2 ** 62)
        budget = int(np.median(probe["peak"]))
        log("%s: round_eval K=%d" % (name, w.K))
        a = g_s.round_eval(w.s_frac, w.K, w.seed, budget)
        b = g_u.round_eval(w.s_frac, w.K, w.seed, budget)
        same(a, b)
        orc = ref.round_eval(wu, budget=budget)
        for key in ("peak", "cost", "feasible", "best_S", "best_R"):
            assert np.array_equal(b[key], orc[key]), key
        assert b["best_k"] == orc["best_k"] >= 0
        # supplied schedules
        sched = wl.random_schedules(w.n, 40, seed=7, density=0.3, kind="intervals", junk=True)
        log("%s: eval_schedules" % name)
        a = g_s.eval_schedules(sched, budget)
        b = g_u.eval_schedules(sched, budget)
        same(a, b)
        o = ref.eval_schedules(wu, list(np.tril(wl.unpack_schedules(sched, w.n), -1)), budget)
        for key in ("peak", "cost", "feasible", "best_R"):
            assert np.array_equal(b[key], o[key]), key
        assert b["best_k"] == o["best_k"]
        # threshold family
        p = np.linspace(0.0, 1.0, 33)
        log("%s: threshold_eval" % name)
        a = g_s.threshold_eval(w.s_frac, p, budget)
        b = g_u.threshold_eval(w.s_frac, p, budget)
        same(a, b)
        o = ref.threshold_eval(wu, p, budget)
        for key in ("peak", "cost", "feasible", "best_S", "best_R"):
            assert np.array_equal(b[key], o[key]), key
        # execution plan of the rounding path's best candidate, late and early
        bk = orc["best_k"]
        _, _, S, R = ref.eval_candidate(wu, bk, want_rows=True)
        for early in (False, True):
            log("%s: plan early=%d" % (name, early))
            st_s, mem_s = g_s.plan(ref.pack_rows(S), ref.pack_rows(R), early=early)
            st_u, mem_u = g_u.plan(ref.pack_rows(S), ref.pack_rows(R), early=early)
            assert np.array_equal(st_s, st_u) and np.array_equal(mem_s, mem_u)
            st_o, mem_o = ref.plan(wu, S, R, early=early)
            assert np.array_equal(st_u, st_o) and np.array_equal(mem_u, mem_o)
    finally:
        g_s.close()
        g_u.close()

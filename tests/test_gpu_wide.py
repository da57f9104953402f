"""Graphs whose sums reach 2^53 (sizes or costs the evaluate kernels cannot
sum exactly in binary64): the library switches to int64 sums. Every value
here is odd and above 2^53 in places, so a binary64 sum would round.

Each graph is checked against the oracle (int64 throughout): every candidate
of the rounding path at two budgets with the best S and R rows, supplied
schedules, the threshold family, the execution plan of the best candidate
(memory after every statement), and the largest batch multiplier.
"""
import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

from test_gpu_parity import check_full, gpu_round_eval

pytestmark = pytest.mark.gpu

INT64_MAX = 2 ** 63 - 1


def log(msg):
    print(msg, flush=True)


def widen(w, m_shift, c_shift, seed):
    """Sizes and costs scaled by 2^shift plus an odd term: integers far above
    2^53 that binary64 cannot hold exactly."""
    rng = np.random.default_rng(seed)
    size = (w.size.astype(np.int64) << m_shift) + (rng.integers(1, 1 << 20, w.n) | 1)
    cost = (w.cost.astype(np.int64) << c_shift) + (rng.integers(1, 1 << 20, w.n) | 1)
    m_in, m_par = (1 << 40) + 3, (1 << 41) + 5
    total_m = m_in + 2 * m_par + sum(int(x) for x in size)
    total_c = sum(int(x) for x in cost)
    assert total_m <= INT64_MAX and w.n * total_c <= INT64_MAX
    assert total_m >= 2 ** 53 or total_c >= 2 ** 53
    budget = (total_m * 3) // 10
    return w.replace(size=size, cost=cost, m_input=m_in, m_param=m_par, budget=budget), total_m, total_c


CASES = [
    # linear chain, n = 17: sum M about 2^55, sum C about 2^58
    ("chain", lambda: wl.config(1), 29, 47),
    # ResNet-like, n = 129: sum M about 2^56, sum C about 2^55
    ("resnet", lambda: wl.config(2).replace(K=128), 25, 33),
    # random DAG, n = 150, fan-in up to 12
    ("random", lambda: wl.random_dag(150, seed=5, K=96, max_deg=12, window=150, max_size=1000, max_cost=1000,
                                     s_kind="uniform", budget_pct=60.0), 40, 39),
]


@pytest.mark.parametrize("name,make,m_shift,c_shift", CASES, ids=[c[0] for c in CASES])
def test_wide_graph_parity(name, make, m_shift, c_shift):
    w, total_m, total_c = widen(make(), m_shift, c_shift, seed=len(name))
    log("%s: n=%d K=%d sum M = 2^%.1f, sum C = 2^%.1f" % (name, w.n, w.K, np.log2(total_m), np.log2(total_c)))
    got = gpu_round_eval(w)
    peak, cost = check_full(w, got)
    assert int(peak.max()) >= 2 ** 53 or int(cost.max()) >= 2 ** 53
    med = int(np.median(peak))
    got2 = gpu_round_eval(w, budget=med)
    check_full(w, got2, budget=med)
    assert got2["best_k"] >= 0
    g = ckm.Graph.from_workload(w)
    try:
        # supplied schedules
        sched = wl.random_schedules(w.n, 24, seed=3, density=0.3, kind="intervals", junk=True)
        log("%s: eval_schedules" % name)
        a = g.eval_schedules(sched, med)
        o = ref.eval_schedules(w, list(np.tril(wl.unpack_schedules(sched, w.n), -1)), med)
        for key in ("peak", "cost", "feasible", "best_R"):
            assert np.array_equal(a[key], o[key]), key
        assert a["best_k"] == o["best_k"]
        # threshold family
        p = np.linspace(0.0, 1.0, 21)
        log("%s: threshold_eval" % name)
        a = g.threshold_eval(w.s_frac, p, med)
        o = ref.threshold_eval(w, p, med)
        for key in ("peak", "cost", "feasible", "best_S", "best_R"):
            assert np.array_equal(a[key], o[key]), key
        # execution plan of the best candidate, late and early
        bk = got2["best_k"]
        _, _, S, R = ref.eval_candidate(w, bk, want_rows=True)
        for early in (False, True):
            log("%s: plan early=%d" % (name, early))
            st, mem = g.plan(ref.pack_rows(S), ref.pack_rows(R), early=early)
            st_o, mem_o = ref.plan(w, S, R, early=early)
            assert np.array_equal(st, st_o) and np.array_equal(mem, mem_o)
        # largest batch multiplier, sampled against the oracle's search
        base = w.m_input + 2 * w.m_param
        budget = int(base + 3 * (med - base))
        cap = int(np.median(cost))
        log("%s: max_batch" % name)
        mb = g.max_batch(w.s_frac, w.K, w.seed, budget, cap)
        q = ref.quantize(w.s_frac)
        for k in (0, 1, w.K // 2, w.K - 1):
            _, _, S, R = ref.eval_candidate(w, k, q=q, want_rows=True)
            assert mb["batch"][k] == ref.max_batch(w, S, R, budget, cap), k
    finally:
        g.close()

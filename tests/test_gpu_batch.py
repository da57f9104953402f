"""Bit-exact parity of the largest batch multiplier (ckm_max_batch, through
the C ABI) with the CPU oracle, which finds B by searching over its
simulator with every node size scaled. Expected values come from the oracle
only.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

pytestmark = pytest.mark.gpu

THREADS = min(16, os.cpu_count() or 4)
INT64_MAX = (1 << 63) - 1


def log(msg):
    print(msg, flush=True)


def oracle_batches(w, ks, budget, cost_cap):
    """{k: (B, peak, cost)} for rounded candidates k."""
    q = ref.quantize(w.s_frac)

    def one(k):
        S = ref.round_random(q, w.seed, k)
        R = ref.solve_R(w, S)
        sim = ref.simulate(w, S, R)
        return ref.max_batch(w, S, R, budget, cost_cap), sim["peak"], sim["cost"]

    with ThreadPoolExecutor(THREADS) as ex:
        res = list(ex.map(one, [int(k) for k in ks]))
    return dict(zip([int(k) for k in ks], res))


def best_of(orc):
    cands = [(-B, c, p, k) for k, (B, p, c) in orc.items() if B > 0]
    return min(cands)[3] if cands else -1


def gpu_max_batch(w, K, budget, cost_cap):
    g = ckm.Graph.from_workload(w)
    try:
        return g.max_batch(w.s_frac, K, w.seed, budget, cost_cap)
    finally:
        g.close()


def peaks_costs(w, K):
    g = ckm.Graph.from_workload(w)
    try:
        r = g.round_eval(w.s_frac, K, w.seed, 2 ** 62, 0, want_rows=False)
    finally:
        g.close()
    return r["peak"], r["cost"]


@pytest.mark.parametrize("cfg,K", [(1, 64), (2, 96), (3, 64)])
def test_configs(cfg, K):
    w = wl.config(cfg)
    peak, cost = peaks_costs(w, K)
    base = w.m_input + 2 * w.m_param
    for budget_mult, cap_q in ((3.0, 0.5), (1.5, 1.0), (20.0, 0.2)):
        budget = int(base + budget_mult * (np.median(peak) - base))
        cap = int(np.quantile(cost, cap_q))
        log("config %d K=%d budget x%.1f cap q%.1f" % (cfg, K, budget_mult, cap_q))
        got = gpu_max_batch(w, K, budget, cap)
        orc = oracle_batches(w, range(K), budget, cap)
        want = np.array([orc[k][0] for k in range(K)], np.int64)
        bad = np.nonzero(got["batch"] != want)[0]
        assert bad.size == 0, "k=%s gpu=%s oracle=%s" % (bad[:5], got["batch"][bad[:5]], want[bad[:5]])
        bk = best_of(orc)
        assert got["best_k"] == bk
        assert got["best_batch"] == (orc[bk][0] if bk >= 0 else 0)


def test_config4_transformer_sampled():
    """All K = 1024 candidates of the transformer workload: a spread of 24
    against the oracle's search over its simulator, and the whole array
    against the linear form of the GPU's own peaks and costs (which the
    rounding-path tests check against the oracle for every candidate)."""
    w = wl.config(4)
    K = w.K
    peak, cost = peaks_costs(w, K)
    base = w.m_input + 2 * w.m_param
    budget = int(base + 2.5 * (np.median(peak) - base))
    cap = int(np.median(cost))
    log("config 4 K=%d" % K)
    got = gpu_max_batch(w, K, budget, cap)
    rng = np.random.default_rng(44)
    ks = sorted(set([0, 1, 63, 64, 127, 200, 255, 511, 1023] + [int(k) for k in rng.integers(0, K, 15)]))
    orc = oracle_batches(w, ks, budget, cap)
    for k in ks:
        assert got["batch"][k] == orc[k][0], k
    assert len({int(got["batch"][k]) for k in ks}) > 1      # the sample spans several multipliers
    lin = np.where((cost <= cap) & (peak <= budget), (budget - base) // np.maximum(peak - base, 1), 0)
    assert np.array_equal(got["batch"], lin)
    bk = int(got["best_k"])
    assert bk >= 0 and got["batch"][bk] == oracle_batches(w, [bk], budget, cap)[bk][0]


@pytest.mark.parametrize("n,K", [(1, 1), (2, 5), (33, 64), (65, 70), (129, 33)])
def test_random_dag_sweep(n, K):
    w = wl.random_dag(n, seed=n + K, K=K, window=min(n, 16), max_deg=3, max_size=1000, max_cost=100,
                      m_input=11, m_param=3)
    peak, cost = peaks_costs(w, K)
    base = w.m_input + 2 * w.m_param
    budget = int(base + 4 * (np.median(peak) - base)) if n > 1 else int(3 * peak[0])
    cap = int(np.quantile(cost, 0.7))
    log("random dag n=%d K=%d" % (n, K))
    got = gpu_max_batch(w, K, budget, cap)
    orc = oracle_batches(w, range(K), budget, cap)
    assert np.array_equal(got["batch"], np.array([orc[k][0] for k in range(K)], np.int64))
    bk = best_of(orc)
    assert got["best_k"] == bk


def test_edge_cases():
    w = wl.config(2)
    K = 32
    base = w.m_input + 2 * w.m_param
    got = gpu_max_batch(w, K, base - 1, 2 ** 62)       # nothing fits even at B = 1
    assert not got["batch"].any() and got["best_k"] == -1 and got["best_batch"] == 0
    got = gpu_max_batch(w, K, 2 ** 50, 0)             # every cost is over the cap
    assert not got["batch"].any() and got["best_k"] == -1
    # no activation bytes: every B is unbounded; ties go to the cheapest
    w0 = w.replace(size=np.zeros(w.n, np.int64), K=K)
    got = gpu_max_batch(w0, K, base, 2 ** 62)
    assert np.all(got["batch"] == INT64_MAX)
    _, cost = peaks_costs(w0, K)
    assert got["best_k"] == int(np.lexsort((np.arange(K), cost))[0])


def test_async_beside_select():
    """max_batch_async after evaluate, on the same work buffer as select."""
    import torch
    w = wl.config(3)
    K = 200
    g = ckm.Graph.from_workload(w)
    try:
        peak, cost = peaks_costs(w, K)
        base = w.m_input + 2 * w.m_param
        budget = int(base + 3 * (np.median(peak) - base))
        cap = int(np.median(cost))
        sync = g.max_batch(w.s_frac, K, w.seed, budget, cap)
        work = g.alloc_work(K)
        out = g.alloc_outputs(K)
        d_s = torch.from_numpy(w.s_frac).cuda()
        g.quantize_async(d_s, work)
        g.evaluate_async(K, w.seed, 0, work)
        g.select_async(K, w.seed, budget, 0, out, work)
        d_b = torch.empty(K, dtype=torch.int64, device="cuda")
        d_bk = torch.empty(1, dtype=torch.int32, device="cuda")
        d_bb = torch.empty(1, dtype=torch.int64, device="cuda")
        d_st = torch.full((1,), -3, dtype=torch.int32, device="cuda")
        g.max_batch_async(K, budget, cap, d_b, d_bk, d_bb, d_st, work)
        torch.cuda.synchronize()
        assert int(d_st.item()) == ckm.OK
        assert np.array_equal(d_b.cpu().numpy(), sync["batch"])
        assert int(d_bk.item()) == sync["best_k"] and int(d_bb.item()) == sync["best_batch"]
        assert np.array_equal(out["peak"].cpu().numpy(), peak)
        # a NaN in S* reaches d_status
        s2 = w.s_frac.copy()
        s2[40, 2] = np.nan
        g.quantize_async(torch.from_numpy(s2).cuda(), work)
        g.evaluate_async(K, w.seed, 0, work)
        g.max_batch_async(K, budget, cap, d_b, d_bk, d_bb, d_st, work)
        torch.cuda.synchronize()
        assert int(d_st.item()) == ckm.E_INVALID_ARG
        with pytest.raises(ckm.CkmError) as e:
            g.max_batch(s2, K, w.seed, budget, cap)
        assert e.value.status == ckm.E_INVALID_ARG
    finally:
        g.close()

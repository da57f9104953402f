"""Bit-exact parity of the threshold family (ckm_threshold_eval, through the
C ABI) with the CPU oracle: candidate k is S* rounded at threshold p_k.

Inputs are the seeded synthetic workloads with threshold grids that are
unsorted, hold duplicates, lie partly outside [0, 1], and hit S* values
exactly. Expected values come from the oracle only.
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


def log(msg):
    print(msg, flush=True)


def oracle_thresholds(w, p, ks=None):
    """{k: (peak, cost)} for threshold candidates from the oracle."""
    ks = range(len(p)) if ks is None else ks

    def one(k):
        S = ref.round_threshold(w.s_frac, float(p[k]))
        sim = ref.simulate(w, S, ref.solve_R(w, S))
        return sim["peak"], sim["cost"]

    with ThreadPoolExecutor(THREADS) as ex:
        res = list(ex.map(one, [int(k) for k in ks]))
    return dict(zip([int(k) for k in ks], res))


def lexi_best(peak, cost, budget):
    cands = [(int(cost[k]), int(peak[k]), k) for k in range(len(peak)) if peak[k] <= budget]
    return min(cands)[2] if cands else -1


def gpu_eval(w, p, budget, s=None):
    g = ckm.Graph.from_workload(w)
    try:
        return g.threshold_eval(w.s_frac if s is None else s, p, budget)
    finally:
        g.close()


def check_rows(w, got, p, bk):
    if bk < 0:
        assert not got["best_S"].any() and not got["best_R"].any()
        return
    S = ref.round_threshold(w.s_frac, float(p[bk]))
    assert np.array_equal(got["best_S"], ref.pack_rows(S)), "best_S differs"
    assert np.array_equal(got["best_R"], ref.pack_rows(ref.solve_R(w, S))), "best_R differs"


def check(w, p, got, budget):
    orc = oracle_thresholds(w, p)
    K = len(p)
    peak = np.array([orc[k][0] for k in range(K)], np.int64)
    cost = np.array([orc[k][1] for k in range(K)], np.int64)
    bad = np.nonzero((got["peak"] != peak) | (got["cost"] != cost))[0]
    assert bad.size == 0, "mismatch at k=%s p=%s gpu=%s oracle=%s" % (
        bad[:5], p[bad[:5]], [(int(got["peak"][k]), int(got["cost"][k])) for k in bad[:5]],
        [orc[int(k)] for k in bad[:5]])
    assert np.array_equal(got["feasible"], (peak <= budget).astype(np.uint8))
    bk = lexi_best(peak, cost, budget)
    assert got["best_k"] == bk
    check_rows(w, got, p, bk)
    return peak, cost


def grid(K, seed):
    """K thresholds: an even grid over [-0.05, 1.05], shuffled, with a few
    duplicates and the exact values 0, 0.5 and 1."""
    rng = np.random.default_rng(seed)
    p = np.linspace(-0.05, 1.05, K)
    if K >= 8:
        p[:3] = [0.0, 0.5, 1.0]
        p[3:6] = p[6:9] if K >= 9 else p[3:6]
    rng.shuffle(p)
    return p


@pytest.mark.parametrize("cfg,K", [(1, 64), (2, 100), (3, 130)])
def test_configs_threshold_grid(cfg, K):
    w = wl.config(cfg)
    p = grid(K, cfg)
    log("config %d n=%d K=%d" % (cfg, w.n, K))
    got = gpu_eval(w, p, w.budget)
    peak, _ = check(w, p, got, w.budget)
    med = int(np.median(peak))
    log("config %d median budget %d" % (cfg, med))
    got2 = gpu_eval(w, p, med)
    check(w, p, got2, med)
    assert got2["best_k"] >= 0


def test_config4_transformer_grid():
    w = wl.config(4)
    p = grid(128, 4)
    log("config 4 n=%d K=128" % w.n)
    got = gpu_eval(w, p, w.budget)
    peak, _ = check(w, p, got, w.budget)
    med = int(np.median(peak))
    check(w, p, gpu_eval(w, p, med), med)


def test_config5_sampled():
    """n = 4001 (128-word register row): sampled thresholds against the oracle."""
    w = wl.config(5)
    p = grid(96, 5)
    log("config 5 n=%d K=96" % w.n)
    got = gpu_eval(w, p, w.budget)
    ks = [0, 1, 31, 63, 64, 95]
    orc = oracle_thresholds(w, p, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k
    budget = int(np.quantile(got["peak"], 0.5))
    got2 = gpu_eval(w, p, budget)
    bk = lexi_best(got2["peak"], got2["cost"], budget)
    assert got2["best_k"] == bk >= 0
    assert (int(got2["peak"][bk]), int(got2["cost"][bk])) == oracle_thresholds(w, p, [bk])[bk]
    check_rows(w, got2, p, bk)


def test_max_nodes_sampled():
    """n = 4096, the largest graph (both rows in LDS): sampled thresholds
    against the oracle, best S and R included."""
    n = 4096
    w = wl.random_dag(n, seed=4098, K=80, window=40, max_deg=3, max_size=1000, max_cost=1000, s_kind="uniform",
                      budget_pct=55.0)
    p = grid(80, 6)
    log("n=%d K=80" % n)
    got = gpu_eval(w, p, 2 ** 62)
    ks = [0, 1, 63, 64, 79]
    orc = oracle_thresholds(w, p, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k
    budget = int(np.quantile(got["peak"], 0.5))
    got2 = gpu_eval(w, p, budget)
    bk = lexi_best(got2["peak"], got2["cost"], budget)
    assert got2["best_k"] == bk >= 0
    assert (int(got2["peak"][bk]), int(got2["cost"][bk])) == oracle_thresholds(w, p, [bk])[bk]
    check_rows(w, got2, p, bk)


def test_exact_ties_and_clamping():
    """S* on a 1/16 lattice (with values outside [0, 1]) and thresholds on
    the same lattice: every comparison at a tie must come out 'not greater'."""
    w = wl.config(2)
    rng = np.random.default_rng(9)
    s = np.tril(rng.integers(-3, 20, size=(w.n, w.n)) / 16.0, -1)
    w2 = w.replace(s_frac=s)
    p = rng.permutation(np.arange(-2, 19) / 16.0)
    log("lattice ties K=%d" % len(p))
    got = gpu_eval(w2, p, w.budget)
    peak, _ = check(w2, p, got, w.budget)
    med = int(np.median(peak))
    check(w2, p, gpu_eval(w2, p, med), med)


def test_half_threshold_is_det0_candidate():
    """p = 0.5 is Algorithm 2's deterministic rounding: the same peak, cost
    and rows as candidate 0 of the rounding path under CKM_F_DET0."""
    w = wl.config(3)
    g = ckm.Graph.from_workload(w)
    try:
        big = 2 ** 62
        a = g.round_eval(w.s_frac, 1, w.seed, big, ckm.F_DET0)
        b = g.threshold_eval(w.s_frac, [0.5], big)
    finally:
        g.close()
    for key in ("peak", "cost", "feasible", "best_S", "best_R"):
        assert np.array_equal(a[key], b[key]), key
    assert a["best_k"] == b["best_k"] == 0


@pytest.mark.parametrize("n,K", [(1, 1), (2, 3), (33, 65), (64, 64), (65, 7), (129, 200), (257, 33)])
def test_random_dag_sweep(n, K):
    w = wl.random_dag(n, seed=5 * n + K, K=K, window=min(n, 24), max_deg=3, max_size=1000, max_cost=1000,
                      s_kind="beta", budget_pct=55.0)
    p = grid(K, n)
    log("random dag n=%d K=%d" % (n, K))
    got = gpu_eval(w, p, w.budget)
    peak, _ = check(w, p, got, w.budget)
    med = int(np.median(peak))
    check(w, p, gpu_eval(w, p, med), med)


def test_many_thresholds_sampled():
    """K = 5000 (a dense grid with many duplicates): sampled candidates."""
    w = wl.config(2)
    rng = np.random.default_rng(3)
    p = np.round(rng.random(5000), 3)
    log("K=5000")
    got = gpu_eval(w, p, w.budget)
    ks = [0, 1, 63, 64, 4095, 4999] + list(rng.integers(0, 5000, 10))
    orc = oracle_thresholds(w, p, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[int(k)], k
    # candidates with equal thresholds are identical
    _, first = np.unique(p, return_index=True)
    for k in ks:
        j = first[np.searchsorted(np.unique(p), p[k])]
        assert got["peak"][k] == got["peak"][j] and got["cost"][k] == got["cost"][j]
    assert got["best_k"] == lexi_best(got["peak"], got["cost"], w.budget)


def test_async_matches_sync_strided_and_nan():
    import torch
    w = wl.config(3)
    p = grid(150, 33)
    g = ckm.Graph.from_workload(w)
    try:
        budget = int(w.budget * 2.5)
        sync = g.threshold_eval(w.s_frac, p, budget)
        K = len(p)
        work = g.alloc_work(K)
        big = torch.zeros((w.n, w.n + 3), dtype=torch.float64, device="cuda")
        big[:, :w.n] = torch.from_numpy(w.s_frac)
        d_p = torch.from_numpy(p).cuda()
        out = g.alloc_outputs(K)
        out["status"].fill_(-123)
        g.threshold_eval_async(big, d_p, budget, out, work)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.OK
        for key in ("peak", "cost", "feasible"):
            assert np.array_equal(out[key].cpu().numpy(), sync[key]), key
        assert int(out["best_k"].item()) == sync["best_k"]
        assert np.array_equal(ckm.rows_to_numpy(out["best_S"]), sync["best_S"])
        assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), sync["best_R"])
        check(w, p, sync, budget)
        # a NaN threshold, then a NaN in S*, reach d_status; a NaN above the
        # diagonal is never read
        p_bad = p.copy()
        p_bad[7] = np.nan
        g.threshold_eval_async(big, torch.from_numpy(p_bad).cuda(), budget, out, work)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.E_INVALID_ARG
        big[40, 3] = float("nan")
        g.threshold_eval_async(big, d_p, budget, out, work)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.E_INVALID_ARG
        big[40, 3] = 0.25
        big[3, 40] = float("nan")
        g.threshold_eval_async(big, d_p, budget, out, work)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.OK
        with pytest.raises(ckm.CkmError) as e:
            g.threshold_eval(w.s_frac, p_bad, budget)
        assert e.value.status == ckm.E_INVALID_ARG
        with pytest.raises(ckm.CkmError) as e:
            g.threshold_eval(w.s_frac, np.zeros(ckm.MAX_THRESHOLDS + 1), budget)
        assert e.value.status == ckm.E_UNSUPPORTED
    finally:
        g.close()


@pytest.mark.parametrize("cfg,K", [(2, 100), (3, 130), (4, 200)])
def test_row_array_and_in_kernel_rows_agree(cfg, K):
    """With the row array (threshold rows made once) and without it (made in
    the evaluate kernel): the same results as the synchronous call, checked
    against the oracle."""
    import torch
    w = wl.config(cfg)
    p = grid(K, 20 + cfg)
    g = ckm.Graph.from_workload(w)
    try:
        assert g.workspace_size(K, rows=False) < g.workspace_size(K)
        budget = int(np.median(g.threshold_eval(w.s_frac, p, 2 ** 62)["peak"]))
        sync = g.threshold_eval(w.s_frac, p, budget)
        d_s = torch.from_numpy(w.s_frac).cuda()
        d_p = torch.from_numpy(p).cuda()
        for with_rows in (True, False):
            log("config %d K=%d row array %s" % (cfg, K, with_rows))
            work = g.alloc_work(K, rows=with_rows)
            out = g.alloc_outputs(K)
            g.threshold_eval_async(d_s, d_p, budget, out, work)
            torch.cuda.synchronize()
            assert int(out["status"].item()) == ckm.OK
            for key in ("peak", "cost", "feasible"):
                assert np.array_equal(out[key].cpu().numpy(), sync[key]), key
            assert int(out["best_k"].item()) == sync["best_k"] >= 0
            assert np.array_equal(ckm.rows_to_numpy(out["best_S"]), sync["best_S"])
            assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), sync["best_R"])
    finally:
        g.close()
    if cfg < 4:
        check(w, p, sync, budget)
    else:
        orc = oracle_thresholds(w, p, [0, 63, 64, 199, sync["best_k"]])
        for k, pc in orc.items():
            assert (int(sync["peak"][k]), int(sync["cost"][k])) == pc, k

"""Bit-exact parity of batch evaluation of supplied checkpoint matrices
(ckm_eval_schedules, through the C ABI) with the CPU oracle.

The inputs are seeded synthetic schedules (paper_1910_02653_amd.workloads
random_schedules) on the standard workloads and random DAGs, with random bits
on and above the diagonal and in the row padding that the evaluation must
ignore. Expected values come from the oracle only.
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


def oracle_schedules(w, rows, ks=None):
    """{k: (peak, cost)} of the supplied schedules from the oracle."""
    ks = range(rows.shape[0]) if ks is None else ks

    def one(k):
        S = np.tril(wl.unpack_schedules(rows[k:k + 1], w.n)[0], -1)
        sim = ref.simulate(w, S, ref.solve_R(w, S))
        return sim["peak"], sim["cost"]

    with ThreadPoolExecutor(THREADS) as ex:
        res = list(ex.map(one, [int(k) for k in ks]))
    return dict(zip([int(k) for k in ks], res))


def lexi_best(peak, cost, budget):
    cands = [(int(cost[k]), int(peak[k]), k) for k in range(len(peak)) if peak[k] <= budget]
    return min(cands)[2] if cands else -1


def gpu_eval(w, rows, budget):
    g = ckm.Graph.from_workload(w)
    try:
        return g.eval_schedules(rows, budget)
    finally:
        g.close()


def check(w, rows, got, budget):
    K = rows.shape[0]
    orc = oracle_schedules(w, rows)
    peak = np.array([orc[k][0] for k in range(K)], np.int64)
    cost = np.array([orc[k][1] for k in range(K)], np.int64)
    bad = np.nonzero((got["peak"] != peak) | (got["cost"] != cost))[0]
    assert bad.size == 0, "mismatch at k=%s gpu=%s oracle=%s" % (
        bad[:5], [(int(got["peak"][k]), int(got["cost"][k])) for k in bad[:5]], [orc[int(k)] for k in bad[:5]])
    assert np.array_equal(got["feasible"], (peak <= budget).astype(np.uint8))
    bk = lexi_best(peak, cost, budget)
    assert got["best_k"] == bk
    if bk < 0:
        assert not got["best_R"].any()
    else:
        S = np.tril(wl.unpack_schedules(rows[bk:bk + 1], w.n)[0], -1)
        assert np.array_equal(got["best_R"], ref.pack_rows(ref.solve_R(w, S))), "best_R differs"
    return peak, cost


CASES = [(1, 64, 0.3, "bernoulli"), (2, 100, 0.1, "intervals"), (3, 130, 0.5, "bernoulli"),
         (3, 64, 0.3, "intervals")]


@pytest.mark.parametrize("cfg,K,density,kind", CASES)
def test_configs_random_schedules(cfg, K, density, kind):
    w = wl.config(cfg)
    rows = wl.random_schedules(w.n, K, seed=cfg * 100 + K, density=density, kind=kind)
    log("config %d n=%d K=%d %s %.2f" % (cfg, w.n, K, kind, density))
    got = gpu_eval(w, rows, w.budget)
    peak, _ = check(w, rows, got, w.budget)
    med = int(np.median(peak))
    log("config %d median budget %d" % (cfg, med))
    got2 = gpu_eval(w, rows, med)
    check(w, rows, got2, med)
    assert got2["best_k"] >= 0


def test_config4_transformer_schedules():
    w = wl.config(4)
    K = 96
    rows = wl.random_schedules(w.n, K, seed=404, density=0.2, kind="intervals")
    log("config 4 n=%d K=%d" % (w.n, K))
    got = gpu_eval(w, rows, w.budget)
    peak, _ = check(w, rows, got, w.budget)
    med = int(np.median(peak))
    check(w, rows, gpu_eval(w, rows, med), med)


def test_config5_sampled():
    """n = 4001 (128-word register row): sampled candidates against the oracle."""
    w = wl.config(5)
    K = 70
    rows = wl.random_schedules(w.n, K, seed=505, density=0.1, kind="intervals")
    log("config 5 n=%d K=%d" % (w.n, K))
    got = gpu_eval(w, rows, w.budget)
    ks = [0, 1, 33, 63, 64, 69]
    orc = oracle_schedules(w, rows, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k
    budget = int(np.quantile(got["peak"], 0.5))
    got2 = gpu_eval(w, rows, budget)
    bk = lexi_best(got2["peak"], got2["cost"], budget)
    assert got2["best_k"] == bk >= 0
    assert (int(got2["peak"][bk]), int(got2["cost"][bk])) == oracle_schedules(w, rows, [bk])[bk]
    S = np.tril(wl.unpack_schedules(rows[bk:bk + 1], w.n)[0], -1)
    assert np.array_equal(got2["best_R"], ref.pack_rows(ref.solve_R(w, S)))


def test_max_nodes_sampled():
    """n = 4096, the largest graph (both rows in LDS, 128-word rows in the
    transpose kernel): sampled candidates against the oracle."""
    n, K = 4096, 70
    w = wl.random_dag(n, seed=4096, K=K, window=40, max_deg=3, max_size=1000, max_cost=1000, s_kind="uniform",
                      budget_pct=55.0)
    rows = wl.random_schedules(n, K, seed=4097, density=0.2, kind="intervals")
    log("n=%d K=%d" % (n, K))
    got = gpu_eval(w, rows, 2 ** 62)
    ks = [0, 1, 63, 64, 69]
    orc = oracle_schedules(w, rows, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k
    budget = int(np.quantile(got["peak"], 0.5))
    got2 = gpu_eval(w, rows, budget)
    bk = lexi_best(got2["peak"], got2["cost"], budget)
    assert got2["best_k"] == bk >= 0
    assert (int(got2["peak"][bk]), int(got2["cost"][bk])) == oracle_schedules(w, rows, [bk])[bk]
    S = np.tril(wl.unpack_schedules(rows[bk:bk + 1], w.n)[0], -1)
    assert np.array_equal(got2["best_R"], ref.pack_rows(ref.solve_R(w, S)))


def test_closed_forms_checkpoint_all_and_none():
    """Checkpoint-all (cost sum C, peak M_in + 2 M_param + sum M, R = I) next
    to the all-zero schedule, on a transformer-sized graph."""
    w = wl.config(3)
    n, W = w.n, (w.n + 63) // 64
    full = ref.pack_rows(np.tri(n, n, -1, dtype=np.uint8))
    rows = np.stack([np.zeros((n, W), np.uint64), full, full])
    got = gpu_eval(w, rows, 2 ** 62)
    assert int(got["cost"][1]) == int(w.cost.sum())
    assert int(got["peak"][1]) == w.m_input + 2 * w.m_param + int(w.size.sum())
    assert got["peak"][2] == got["peak"][1] and got["cost"][2] == got["cost"][1]
    check(w, rows, got, 2 ** 62)
    if got["best_k"] == 1:
        assert np.array_equal(got["best_R"], ref.pack_rows(np.eye(n, dtype=np.uint8)))


SWEEP = [(1, 1), (2, 3), (31, 63), (32, 64), (33, 65), (63, 7), (64, 128), (65, 129), (127, 40),
         (129, 64), (200, 33), (257, 20)]


@pytest.mark.parametrize("n,K", SWEEP)
def test_random_dag_sweep(n, K):
    w = wl.random_dag(n, seed=3 * n + K, K=K, window=min(n, 24), max_deg=3, max_size=1000, max_cost=1000,
                      budget_pct=55.0)
    rows = wl.random_schedules(n, K, seed=n + 7 * K, density=0.25, kind="bernoulli" if n % 2 else "intervals")
    log("random dag n=%d K=%d" % (n, K))
    got = gpu_eval(w, rows, w.budget)
    peak, _ = check(w, rows, got, w.budget)
    med = int(np.median(peak))
    check(w, rows, gpu_eval(w, rows, med), med)


def test_rounded_candidates_round_trip():
    """The oracle's rounded S of each candidate, supplied back as schedules,
    reproduces the rounding path's peaks, costs, argmin and R."""
    w = wl.config(2).replace(K=96)
    Ss = np.stack([ref.pack_rows(ref.eval_candidate(w, k, want_rows=True)[2]) for k in range(w.K)])
    log("round trip K=%d" % w.K)
    g = ckm.Graph.from_workload(w)
    try:
        a = g.round_eval(w.s_frac, w.K, w.seed, w.budget, 0)
        b = g.eval_schedules(Ss, w.budget)
    finally:
        g.close()
    for key in ("peak", "cost", "feasible", "best_R"):
        assert np.array_equal(a[key], b[key]), key
    assert a["best_k"] == b["best_k"]


def test_async_matches_sync_and_reuses_work():
    """The async form on device tensors, after a rounding-path call on the
    same work buffer, and a second call with fewer schedules."""
    import torch
    w = wl.config(3)
    K = 200
    rows = wl.random_schedules(w.n, K, seed=77, density=0.3, kind="intervals")
    g = ckm.Graph.from_workload(w)
    try:
        sync = g.eval_schedules(rows, w.budget * 2)
        work = g.alloc_work(K)
        out = g.alloc_outputs(K)
        g.round_eval_async(torch.from_numpy(w.s_frac).cuda(), K, w.seed, w.budget, 0, out, work)
        d_S = torch.from_numpy(rows.view(np.int64)).cuda()
        for kk in (K, 37):
            log("async K=%d" % kk)
            out = g.alloc_outputs(kk)
            out["status"].fill_(-123)
            g.eval_schedules_async(d_S[:kk], kk, w.budget * 2, out, work)
            torch.cuda.synchronize()
            assert int(out["status"].item()) == ckm.OK
            peak = out["peak"].cpu().numpy()
            cost = out["cost"].cpu().numpy()
            assert np.array_equal(peak, sync["peak"][:kk]) and np.array_equal(cost, sync["cost"][:kk])
            assert np.array_equal(out["feasible"].cpu().numpy(), sync["feasible"][:kk])
            bk = lexi_best(peak, cost, w.budget * 2)
            assert int(out["best_k"].item()) == bk
            if kk == K:
                assert bk == sync["best_k"]
                assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), sync["best_R"])
        check(w, rows, sync, w.budget * 2)
    finally:
        g.close()


def test_nothing_feasible_and_bad_args():
    w = wl.config(2)
    rows = wl.random_schedules(w.n, 5, seed=1, density=0.5)
    got = gpu_eval(w, rows, 0)
    assert got["best_k"] == -1 and not got["feasible"].any() and not got["best_R"].any()
    g = ckm.Graph.from_workload(w)
    try:
        with pytest.raises(ckm.CkmError) as e:
            g.eval_schedules(rows, -1)
        assert e.value.status == ckm.E_INVALID_ARG
        with pytest.raises(ValueError):
            g.eval_schedules(rows[:, :-1], 0)
    finally:
        g.close()


@pytest.mark.parametrize("cfg,K", [(2, 100), (3, 130), (4, 200)])
def test_row_array_and_in_kernel_rows_agree(cfg, K):
    """With the row array (the caller's matrices transposed into it once) and
    without it (each lane reads its own matrix in the evaluate kernel): the
    same results as the synchronous call, checked against the oracle."""
    import torch
    w = wl.config(cfg)
    rows = wl.random_schedules(w.n, K, seed=10 + cfg, density=0.3, kind="bernoulli", junk=True)
    g = ckm.Graph.from_workload(w)
    try:
        assert g.workspace_size(K, rows=False) < g.workspace_size(K)
        budget = int(np.median(g.eval_schedules(rows, 2 ** 62)["peak"]))
        sync = g.eval_schedules(rows, budget)
        d_S = torch.from_numpy(rows.view(np.int64)).cuda()
        for with_rows in (True, False):
            log("config %d K=%d row array %s" % (cfg, K, with_rows))
            work = g.alloc_work(K, rows=with_rows)
            out = g.alloc_outputs(K)
            g.eval_schedules_async(d_S, K, budget, out, work)
            torch.cuda.synchronize()
            for key in ("peak", "cost", "feasible"):
                assert np.array_equal(out[key].cpu().numpy(), sync[key]), key
            assert int(out["best_k"].item()) == sync["best_k"] >= 0
            assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), sync["best_R"])
    finally:
        g.close()
    if cfg < 4:
        check(w, rows, sync, budget)
    else:
        orc = oracle_schedules(w, rows, [0, 63, 64, 199, sync["best_k"]])
        for k, pc in orc.items():
            assert (int(sync["peak"][k]), int(sync["cost"][k])) == pc, k

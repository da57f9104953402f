"""Bit-exact parity of the HIP path (through the C ABI) with the CPU oracle.

Every result is integer (peak bytes, cost, feasible flags, best index, S and
R bit rows), so the bar is equality. Inputs are the seeded synthetic
workloads (paper_1910_02653_amd.workloads); expected values come from the
oracle only.
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


def oracle_candidates(w, ks, flags=0, seed=None):
    """{k: (peak, cost)} from the oracle, candidates evaluated on a thread pool."""
    ww = w if seed is None else w.replace(seed=seed)
    q = ref.quantize(ww.s_frac)
    with ThreadPoolExecutor(THREADS) as ex:
        res = list(ex.map(lambda k: ref.eval_candidate(ww, int(k), flags=flags, q=q), ks))
    return dict(zip([int(k) for k in ks], res))


def lexi_best(peak, cost, budget):
    cands = [(int(cost[k]), int(peak[k]), k) for k in range(len(peak)) if peak[k] <= budget]
    return min(cands)[2] if cands else -1


def check_full(w, got, flags=0, budget=None, seed=None):
    """Compare a GPU result over all K candidates with the oracle."""
    budget = w.budget if budget is None else budget
    orc = oracle_candidates(w, range(w.K), flags=flags, seed=seed)
    peak = np.array([orc[k][0] for k in range(w.K)], np.int64)
    cost = np.array([orc[k][1] for k in range(w.K)], np.int64)
    bad = np.nonzero((got["peak"] != peak) | (got["cost"] != cost))[0]
    assert bad.size == 0, "mismatch at k=%s gpu=%s oracle=%s" % (
        bad[:5], [(int(got["peak"][k]), int(got["cost"][k])) for k in bad[:5]],
        [orc[int(k)] for k in bad[:5]])
    assert np.array_equal(got["feasible"], (peak <= budget).astype(np.uint8))
    bk = lexi_best(peak, cost, budget)
    assert got["best_k"] == bk
    check_rows(w, got, bk, flags, seed)
    return peak, cost


def check_rows(w, got, bk, flags=0, seed=None):
    if got.get("best_S") is None:
        return
    if bk < 0:
        assert not got["best_S"].any() and not got["best_R"].any()
        return
    ww = w if seed is None else w.replace(seed=seed)
    _, _, S, R = ref.eval_candidate(ww, bk, flags=flags, want_rows=True)
    assert np.array_equal(got["best_S"], ref.pack_rows(S)), "best_S differs"
    assert np.array_equal(got["best_R"], ref.pack_rows(R)), "best_R differs"


def gpu_round_eval(w, K=None, seed=None, budget=None, flags=0):
    g = ckm.Graph.from_workload(w)
    try:
        return g.round_eval(w.s_frac, w.K if K is None else K, w.seed if seed is None else seed,
                            w.budget if budget is None else budget, flags)
    finally:
        g.close()


def test_single_hip_runtime_in_process():
    """libckm and torch share one HIP runtime (no second libamdhip64 mapped)."""
    import torch
    ckm.lib()
    torch.zeros(1, device="cuda")
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            if "libamdhip64" in line:
                paths.add(line.split()[-1])
    assert len(paths) == 1, paths


# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_small_configs_full_parity(cfg):
    w = wl.config(cfg)
    log("config %d n=%d K=%d" % (cfg, w.n, w.K))
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)
    # feasible-rich: budget at the median candidate peak exercises the argmin
    med = int(np.median(peak))
    log("config %d median budget %d" % (cfg, med))
    got2 = gpu_round_eval(w, budget=med)
    check_full(w, got2, budget=med)
    assert got2["best_k"] >= 0


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_small_configs_sparse_checkpoints(cfg):
    """S* scaled by 0.2: few checkpoints, long recomputation closures."""
    w = wl.config(cfg)
    w = w.replace(s_frac=0.2 * w.s_frac, K=min(w.K, 128))
    log("config %d sparse K=%d" % (cfg, w.K))
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)
    med = int(np.median(peak))
    check_full(w, gpu_round_eval(w, budget=med), budget=med)


@pytest.mark.parametrize("cfg", [1, 2])
def test_det0_candidate(cfg):
    w = wl.config(cfg)
    log("config %d DET0" % cfg)
    got = gpu_round_eval(w, flags=ckm.F_DET0)
    check_full(w, got, flags=ckm.F_DET0)
    big = int(got["peak"].max())
    got2 = gpu_round_eval(w, flags=ckm.F_DET0, budget=big)
    check_full(w, got2, flags=ckm.F_DET0, budget=big)


def test_many_candidates_two_stage_select():
    """K = 70,001 (more than one select block handles: reduction in blocks,
    then the argmin) on workload 1, every candidate against the oracle at a
    budget about half of them meet."""
    w = wl.config(1).replace(K=70001)
    peak0 = gpu_round_eval(w, budget=2 ** 62)["peak"]
    budget = int(np.median(peak0))
    log("K=%d budget %d" % (w.K, budget))
    got = gpu_round_eval(w, budget=budget)
    check_full(w, got, budget=budget)
    assert got["best_k"] >= 0


def test_config4_transformer_full_parity():
    w = wl.config(4)
    log("config 4 n=%d K=%d" % (w.n, w.K))
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)
    med = int(np.median(peak))
    log("config 4 median budget")
    check_full(w, gpu_round_eval(w, budget=med), budget=med)


def test_config4_sparse_sampled():
    w = wl.config(4)
    w = w.replace(s_frac=0.2 * w.s_frac, K=96)
    log("config 4 sparse K=96")
    got = gpu_round_eval(w)
    check_full(w, got)


FIXTURE5 = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "workload5_oracle.npz")


def test_config5_random_dag_all_candidates():
    """n = 4001, K = 4096: every candidate's peak and cost against the
    oracle's, stored by tests/golden/make_workload5_fixture.py (which calls
    only the oracle); the argmin and the best candidate's S and R rows at two
    budgets where some candidates are feasible, against the oracle run here."""
    w = wl.config(5)
    fx = np.load(FIXTURE5)
    assert int(fx["n"]) == w.n and int(fx["K"]) == w.K and int(fx["seed"]) == w.seed
    peak, cost = fx["peak"], fx["cost"]
    log("config 5 n=%d K=%d" % (w.n, w.K))
    got = gpu_round_eval(w)
    bad = np.nonzero((got["peak"] != peak) | (got["cost"] != cost))[0]
    assert bad.size == 0, "mismatch at k=%s" % bad[:8]
    assert np.array_equal(got["feasible"], (peak <= w.budget).astype(np.uint8))
    assert got["best_k"] == lexi_best(peak, cost, w.budget)
    for q in (0.3, 0.5):
        budget = int(np.quantile(peak, q))
        log("config 5 budget at the %.1f peak quantile" % q)
        got2 = gpu_round_eval(w, budget=budget)
        assert np.array_equal(got2["peak"], peak) and np.array_equal(got2["cost"], cost)
        bk = lexi_best(peak, cost, budget)
        assert got2["best_k"] == bk >= 0
        check_rows(w, got2, bk)


SEED64 = 0x89ABCDEF01234567       # both 32-bit halves of the Philox key nonzero


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_seed_with_high_word(cfg):
    """A seed whose high 32 bits are nonzero (the second Philox key word):
    every candidate, with and without the deterministic candidate 0."""
    w = wl.config(cfg)
    for flags in (0, ckm.F_DET0):
        log("config %d seed 0x%x flags %d" % (cfg, SEED64, flags))
        got = gpu_round_eval(w, seed=SEED64, flags=flags)
        peak, _ = check_full(w, got, flags=flags, seed=SEED64)
        med = int(np.median(peak))
        got2 = gpu_round_eval(w, seed=SEED64, flags=flags, budget=med)
        check_full(w, got2, flags=flags, budget=med, seed=SEED64)
    # the high word changes the draws
    assert not np.array_equal(gpu_round_eval(w, seed=SEED64)["peak"],
                              gpu_round_eval(w, seed=SEED64 & 0xFFFFFFFF)["peak"])


SWEEP = [(1, 3, "uniform"), (2, 5, "uniform"), (3, 4, "beta"), (5, 9, "binary"), (17, 64, "sparse"),
         (31, 63, "uniform"), (32, 65, "beta"), (33, 1, "sparse"), (63, 64, "uniform"), (64, 130, "beta"),
         (65, 7, "sparse"), (100, 33, "binary"), (127, 64, "uniform"), (128, 65, "sparse"), (129, 40, "beta"),
         (200, 70, "uniform"), (257, 20, "sparse"), (300, 64, "beta")]


@pytest.mark.parametrize("n,K,kind", SWEEP)
def test_random_dag_sweep(n, K, kind):
    w = wl.random_dag(n, seed=n * 7 + K, K=K, s_kind=kind, window=min(n, 24), max_deg=3,
                      max_size=1000, max_cost=1000, budget_pct=55.0)
    log("random dag n=%d K=%d %s" % (n, K, kind))
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)
    med = int(np.median(peak))
    check_full(w, gpu_round_eval(w, budget=med), budget=med)


@pytest.mark.parametrize("n", [1023, 1024, 1500, 2047, 2048, 3000, 4095])
def test_register_row_widths(n):
    """Rows of 32, 64 and 128 words in registers (n < 1024, < 2048, < 4096;
    n = 4095 fills all 128 words):
    graphs on both sides of each boundary, sampled candidates against the
    oracle, the rest through the argmin and the best rows."""
    w = wl.random_dag(n, seed=n, K=70, window=40, max_deg=3, max_size=1000, max_cost=1000, s_kind="uniform",
                      budget_pct=55.0)
    log("register rows n=%d" % n)
    got = gpu_round_eval(w)
    ks = [0, 1, 63, 64, 69]
    orc = oracle_candidates(w, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k
    budget = int(np.median(got["peak"]))
    got2 = gpu_round_eval(w, budget=budget)
    assert np.array_equal(got2["peak"], got["peak"]) and np.array_equal(got2["cost"], got["cost"])
    bk = lexi_best(got2["peak"], got2["cost"], budget)
    assert got2["best_k"] == bk >= 0
    assert (int(got2["peak"][bk]), int(got2["cost"][bk])) == oracle_candidates(w, [bk])[bk]
    check_rows(w, got2, bk)


def test_dense_wide_graph():
    """Many deps and users per node (fan-in / fan-out up to 40)."""
    w = wl.random_dag(150, seed=11, K=70, max_deg=40, window=150, s_kind="uniform", budget_pct=60.0)
    log("dense wide graph")
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)


def boundary_graph():
    """A 200-node graph whose slow nodes sit at the limits of the record's
    second form (14 far users, 6 deps, 4 far later users per dep) and one
    past each, next to a chain that keeps every node reachable."""
    n = 200
    deps = [set() if v == 0 else {v - 1} for v in range(n)]
    deps[150] |= {0, 10, 20, 30, 40}            # 6 deps: second form
    deps[160] |= {1, 11, 21, 31, 41, 51}        # 7 deps: CSR lists
    for k in range(14):                         # node 5: 14 users beyond 5 + 32
        deps[40 + 5 * k].add(5)
    for k in range(15):                         # node 6: 15 of them
        deps[41 + 5 * k].add(6)
    deps[60].add(7)                             # dep 7 of node 60: 4 users beyond 60 + 32
    for u in (100, 110, 120, 130):
        deps[u].add(7)
    deps[61].add(8)                             # dep 8 of node 61: 5 of them
    for u in (101, 111, 121, 131, 141):
        deps[u].add(8)
    ptr, idx = wl.csr_from_deps([sorted(d) for d in deps])
    rng = np.random.default_rng(200)
    size = rng.integers(1, 1000, n).astype(np.int64)
    cost = rng.integers(1, 1000, n).astype(np.int64)
    return wl.Workload("form_limits", n, ptr, idx, cost, size, 7, 3, wl.s_frac_uniform(n, 21), 130, 21, 1 << 40)


def test_slow_node_form_limits():
    """Slow nodes at and one past each limit of the record's second form:
    every candidate against the oracle, and the best rows at a budget where
    some are feasible."""
    w = boundary_graph()
    log("form limits n=%d K=%d" % (w.n, w.K))
    got = gpu_round_eval(w)
    peak, _ = check_full(w, got)
    med = int(np.median(peak))
    check_full(w, gpu_round_eval(w, budget=med), budget=med)


def test_max_nodes_chain():
    """n = 4096 (the largest graph): a chain with a mirrored backward pass."""
    F = 2047
    fwd = [[]] + [[v - 1] for v in range(1, F)]
    deps, size, cost, _ = wl.mirror_training_graph(fwd, np.full(F, 3 << 20), np.full(F, 50), 4, 7)
    deps.append([len(deps) - 1])           # one extra node: n = 4096
    size = np.append(size, 1 << 20)
    cost = np.append(cost, 9)
    ptr, idx = wl.csr_from_deps(deps)
    n = len(deps)
    assert n == 4096
    w = wl.Workload("chain4096", n, ptr, idx, cost, size, 1 << 20, 1 << 20, wl.s_frac_uniform(n, 9), 64, 9,
                    1 << 40)
    log("max nodes chain")
    got = gpu_round_eval(w)
    orc = oracle_candidates(w, [0, 37, 63])
    for k, v in orc.items():
        assert (int(got["peak"][k]), int(got["cost"][k])) == v
    assert got["best_k"] == lexi_best(got["peak"], got["cost"], w.budget)
    check_rows(w, got, got["best_k"])


@pytest.mark.parametrize("n", [337, 1500, 2047, 4095])
def test_in_kernel_rows_without_row_arrays(n):
    """The rounding path on a work buffer without the row arrays: rows
    rounded in the evaluate kernel (register rows of 32, 64 and 128 words) and the
    best R recomputed by Algorithm 2 in the closure kernel. Every output
    equals the row-array path's, whose results the oracle checks; the best
    candidate's rows are checked against the oracle here too."""
    import torch
    w = wl.config(3) if n == 337 else wl.random_dag(n, seed=n + 1, K=200, window=40, max_deg=3, max_size=1000,
                                                    max_cost=1000, s_kind="uniform", budget_pct=55.0)
    g = ckm.Graph.from_workload(w)
    try:
        K = w.K if n == 337 else 200
        full = g.round_eval(w.s_frac, K, w.seed, 2 ** 62)
        budget = int(np.median(full["peak"]))
        want = g.round_eval(w.s_frac, K, w.seed, budget)
        small = g.alloc_work(K, rows=False)
        assert small.numel() < g.workspace_size(K)
        out = g.alloc_outputs(K)
        log("n=%d K=%d in-kernel rows" % (n, K))
        g.round_eval_async(torch.from_numpy(w.s_frac).cuda(), K, w.seed, budget, 0, out, small)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.OK
        for key in ("peak", "cost", "feasible"):
            assert np.array_equal(out[key].cpu().numpy(), want[key]), key
        assert int(out["best_k"].item()) == want["best_k"] >= 0
        assert np.array_equal(ckm.rows_to_numpy(out["best_S"]), want["best_S"])
        assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), want["best_R"])
        direct = out["peak"].cpu().numpy(), out["cost"].cpu().numpy()
    finally:
        g.close()
    check_rows(w.replace(K=K), want, want["best_k"])
    # the in-kernel path's own outputs against the oracle, candidate by candidate
    ks = [0, 1, 63, 64, 65, 127, 128, K - 1]
    orc = oracle_candidates(w, ks)
    for k in ks:
        assert (int(direct[0][k]), int(direct[1][k])) == orc[k], k


def test_async_stages_and_split_invariance():
    """The staged async calls give the same bits for any stage split (a race
    or a split-boundary error would change them)."""
    import torch
    w = wl.config(3)
    w = w.replace(K=200)
    g = ckm.Graph.from_workload(w)
    d_s = torch.from_numpy(w.s_frac).cuda()
    work = g.alloc_work(w.K)
    ref_out = None
    budget = w.budget * 3
    for splits in (1, 2, 7, 64, 10 ** 6, 0):
        log("splits %d" % splits)
        out = g.alloc_outputs(w.K)
        g.quantize_async(d_s, work)
        g.evaluate_async(w.K, w.seed, 0, work, stage_splits=splits)
        g.select_async(w.K, w.seed, budget, 0, out, work)
        torch.cuda.synchronize()
        res = dict(peak=out["peak"].cpu().numpy(), cost=out["cost"].cpu().numpy(),
                   feasible=out["feasible"].cpu().numpy(), best_k=int(out["best_k"].item()),
                   best_S=ckm.rows_to_numpy(out["best_S"]), best_R=ckm.rows_to_numpy(out["best_R"]))
        assert int(out["status"].item()) == ckm.OK
        if ref_out is None:
            check_full(w, res, budget=budget)
            ref_out = res
        else:
            for key in ("peak", "cost", "feasible", "best_S", "best_R"):
                assert np.array_equal(res[key], ref_out[key]), (splits, key)
            assert res["best_k"] == ref_out["best_k"]
    # the staged form with rounding on its own (ckm_round_async + CKM_F_ROUNDED)
    out = g.alloc_outputs(w.K)
    g.quantize_async(d_s, work)
    g.round_async(w.K, w.seed, 0, work)
    g.evaluate_async(w.K, w.seed, ckm.F_ROUNDED, work)
    g.select_async(w.K, w.seed, budget, ckm.F_ROUNDED, out, work)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    assert np.array_equal(out["peak"].cpu().numpy(), ref_out["peak"])
    assert np.array_equal(ckm.rows_to_numpy(out["best_R"]), ref_out["best_R"])
    # the one-call async form agrees too, on a strided S*
    big = torch.zeros((w.n, w.n + 5), dtype=torch.float64, device="cuda")
    big[:, :w.n] = d_s
    out = g.alloc_outputs(w.K)
    g.round_eval_async(big, w.K, w.seed, budget, 0, out, work)
    torch.cuda.synchronize()
    assert np.array_equal(out["peak"].cpu().numpy(), ref_out["peak"])
    assert int(out["best_k"].item()) == ref_out["best_k"]
    g.close()


def test_rounded_flag_without_row_array():
    """n = 4001, K = 4096 on a work buffer without the row arrays:
    ckm_round_async does nothing and evaluate with CKM_F_ROUNDED rounds
    inside, with the same results for every candidate as the one-call form
    on a buffer with the row arrays (4.1 GB of S rows, streamed)."""
    import torch
    w = wl.config(5)
    g = ckm.Graph.from_workload(w)
    try:
        work = g.alloc_work(w.K)
        small = g.alloc_work(w.K, rows=False)
        assert small.numel() < work.numel()
        d_s = torch.from_numpy(w.s_frac).cuda()
        budget = int(w.budget * 2)
        a = g.alloc_outputs(w.K)
        g.round_eval_async(d_s, w.K, w.seed, budget, 0, a, work)
        torch.cuda.synchronize()
        del work
        b = g.alloc_outputs(w.K)
        g.quantize_async(d_s, small)
        g.round_async(w.K, w.seed, 0, small)
        g.evaluate_async(w.K, w.seed, ckm.F_ROUNDED, small)
        g.select_async(w.K, w.seed, budget, 0, b, small)
        torch.cuda.synchronize()
        log("config 5 rounded flag")
        for key in ("peak", "cost", "feasible", "best_k"):
            assert torch.equal(a[key], b[key]), key
    finally:
        g.close()


def test_nan_reported():
    import torch
    w = wl.config(2).replace(K=8)
    s = w.s_frac.copy()
    s[50, 3] = np.nan
    with pytest.raises(ckm.CkmError) as e:
        gpu_round_eval(w.replace(s_frac=s))
    assert e.value.status == ckm.E_INVALID_ARG
    g = ckm.Graph.from_workload(w)
    work = g.alloc_work(w.K)
    out = g.alloc_outputs(w.K)
    g.round_eval_async(torch.from_numpy(s).cuda(), w.K, w.seed, w.budget, 0, out, work)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.E_INVALID_ARG
    s2 = w.s_frac.copy()
    s2[3, 50] = np.nan                      # above the diagonal: never read
    g.round_eval_async(torch.from_numpy(s2).cuda(), w.K, w.seed, w.budget, 0, out, work)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    g.close()


def test_out_of_range_s_values_clamped():
    w = wl.config(2).replace(K=64)
    s = w.s_frac * 3.0 - 1.0               # values in [-1, 2], clamped to [0, 1]
    s = np.tril(s, -1)
    w2 = w.replace(s_frac=s)
    got = gpu_round_eval(w2)
    check_full(w2, got)

"""ckm_round_eval_noalloc: the rounding path on the library's static work area.

Two calls in a row on one device, the second on a smaller problem, each
compared output by output with ckm_round_eval_async on a work buffer of its
own (and the second also with the oracle): the area keeps the first call's
contents, so a stage that read something it did not write would show here.
A problem larger than the area is refused before any launch.
"""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def run_both(g, w, K, seed, budget, flags):
    d_s = torch.from_numpy(w.s_frac).to("cuda")
    out_a = g.alloc_outputs(K)
    g.round_eval_async(d_s, K, seed, budget, flags, out_a, g.alloc_work(K))
    out_b = g.alloc_outputs(K)
    g.round_eval_noalloc(d_s, K, seed, budget, flags, out_b)
    torch.cuda.synchronize()
    a = {k: v.cpu().numpy() for k, v in out_a.items()}
    b = {k: v.cpu().numpy() for k, v in out_b.items()}
    assert int(b["status"][0]) == ckm.OK
    for key in a:
        assert np.array_equal(a[key], b[key]), key
    return b


def test_noalloc_two_calls_match_async():
    torch.cuda.set_device(0)
    # call 1: the transformer stack, n = 1009, K = 1024 (row arrays fit the area)
    w4 = wl.config(4)
    g4 = ckm.Graph.from_workload(w4)
    try:
        probe = g4.alloc_outputs(w4.K)
        g4.round_eval_async(torch.from_numpy(w4.s_frac).to("cuda"), w4.K, w4.seed, w4.budget, 0, probe,
                            g4.alloc_work(w4.K))
        torch.cuda.synchronize()
        budget4 = int(np.median(probe["peak"].cpu().numpy()))
        log("noalloc call 1: n=%d K=%d budget=%d" % (w4.n, w4.K, budget4))
        b = run_both(g4, w4, w4.K, w4.seed, budget4, 0)
        assert int(b["best_k"][0]) >= 0
    finally:
        g4.close()
    # call 2: smaller graph and K on the same area, a seed with both key words
    w3 = wl.config(3)
    K, seed = 200, (0x89ABCDEF << 32) | 0x01234567
    g3 = ckm.Graph.from_workload(w3)
    try:
        probe = g3.alloc_outputs(K)
        g3.round_eval_async(torch.from_numpy(w3.s_frac).to("cuda"), K, seed, w3.budget, ckm.F_DET0, probe,
                            g3.alloc_work(K))
        torch.cuda.synchronize()
        budget3 = int(np.median(probe["peak"].cpu().numpy()))
        log("noalloc call 2: n=%d K=%d budget=%d" % (w3.n, K, budget3))
        b = run_both(g3, w3, K, seed, budget3, ckm.F_DET0)
        orc = ref.round_eval(w3, K=K, seed=seed, budget=budget3, flags=ref.F_DET0)
        assert np.array_equal(b["peak"], orc["peak"])
        assert np.array_equal(b["cost"], orc["cost"])
        assert np.array_equal(b["feasible"], orc["feasible"])
        assert int(b["best_k"][0]) == orc["best_k"] >= 0
        assert np.array_equal(b["best_S"].view(np.uint64), orc["best_S"])
        assert np.array_equal(b["best_R"].view(np.uint64), orc["best_R"])
    finally:
        g3.close()


def test_noalloc_refuses_problem_larger_than_area():
    torch.cuda.set_device(0)
    w = wl.random_dag(4096, 1)
    g = ckm.Graph.from_workload(w)
    try:
        K = ckm.MAX_CANDIDATES
        assert g.workspace_size(K, rows=False) > ckm.NOALLOC_SCRATCH_BYTES
        d_s = torch.zeros((w.n, w.n), dtype=torch.float64, device="cuda")
        out = {"peak": torch.empty(K, dtype=torch.int64, device="cuda"),
               "cost": torch.empty(K, dtype=torch.int64, device="cuda"),
               "feasible": torch.empty(K, dtype=torch.uint8, device="cuda"),
               "best_k": torch.empty(1, dtype=torch.int32, device="cuda"),
               "best_S": None, "best_R": None,
               "status": torch.empty(1, dtype=torch.int32, device="cuda")}
        with pytest.raises(ckm.CkmError) as e:
            g.round_eval_noalloc(d_s, K, 1, 0, 0, out)
        assert e.value.status == ckm.E_UNSUPPORTED
    finally:
        g.close()

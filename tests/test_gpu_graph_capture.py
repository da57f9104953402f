"""The asynchronous entry points under HIP graph capture.

ckm_round_eval_async (quantize, rounding, Algorithm 2 repair and simulation,
select) enqueues kernel launches only, plus, on seen-path graphs with eight
or more candidate groups, an event fork to the graph's second stream and a
join back. A graph captured from one call is replayed several times, with
the program's own eager work (the same call on other buffers, outputs
overwritten) and synchronizations between the replays, and every replay must
equal the eager call bit for bit, which the oracle checks in turn.
"""
import numpy as np
import pytest
import torch

from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl
from test_gpu_parity import check_full, log, oracle_candidates

pytestmark = pytest.mark.gpu

KEYS = ("peak", "cost", "feasible", "best_k", "best_S", "best_R", "status")


def host(out):
    return {k: out[k].cpu().numpy().copy() for k in KEYS}


def as_result(h):
    return dict(peak=h["peak"], cost=h["cost"], feasible=h["feasible"], best_k=int(h["best_k"][0]),
                best_S=h["best_S"].view(np.uint64), best_R=h["best_R"].view(np.uint64))


def replay_matches_eager(w, budget, replays=4):
    g = ckm.Graph.from_workload(w)
    try:
        K = w.K
        d_s = torch.from_numpy(w.s_frac).cuda()
        work_e, out_e = g.alloc_work(K), g.alloc_outputs(K)
        g.round_eval_async(d_s, K, w.seed, budget, 0, out_e, work_e)
        torch.cuda.synchronize()
        eager = host(out_e)
        assert int(eager["status"][0]) == ckm.OK

        work_c, out_c = g.alloc_work(K), g.alloc_outputs(K)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):   # one warm call on the capture buffers
            g.round_eval_async(d_s, K, w.seed, budget, 0, out_c, work_c)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        cg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(cg):
            g.round_eval_async(d_s, K, w.seed, budget, 0, out_c, work_c)
        torch.cuda.synchronize()
        for r in range(replays):
            # eager work between replays, and outputs overwritten first
            for key in ("peak", "cost"):
                out_c[key].fill_(-7)
            out_c["feasible"].fill_(3)
            out_c["best_k"].fill_(-9)
            out_c["best_S"].fill_(5)
            g.round_eval_async(d_s, K, w.seed + 1 + r, budget, 0, out_e, work_e)
            torch.cuda.synchronize()
            cg.replay()
            torch.cuda.synchronize()
            got = host(out_c)
            for key in KEYS:
                assert np.array_equal(got[key], eager[key]), (r, key)
        return as_result(eager)
    finally:
        g.close()


def replay_peaks(w):
    g = ckm.Graph.from_workload(w)
    try:
        return g.round_eval(w.s_frac, w.K, w.seed, w.budget)["peak"]
    finally:
        g.close()


def test_capture_mask_path_full_parity():
    """Workload 2 (n = 129, K = 256): the mask path, every candidate."""
    w = wl.config(2)
    log("graph capture: config 2 n=%d K=%d" % (w.n, w.K))
    got = replay_matches_eager(w, w.budget)
    check_full(w, got)


def test_capture_transformer_sampled():
    """Workload 4 (n = 1009, K = 1024) at its own budget: sampled candidates
    and the best rows against the oracle."""
    w = wl.config(4)
    log("graph capture: config 4 n=%d K=%d" % (w.n, w.K))
    got = replay_matches_eager(w, w.budget, replays=3)
    ks = [0, 1, 63, 64, 511, 1023]
    orc = oracle_candidates(w, ks)
    for k in ks:
        assert (int(got["peak"][k]), int(got["cost"][k])) == orc[k], k


def test_capture_seen_path_overlapped():
    """A seen-path graph whose seen bits hold the evaluate to 14 waves per
    CU, K = 520 (nine groups): the captured call forks to the graph's second
    stream and joins back; every candidate."""
    from test_gpu_seen import lds_bound_graph
    w = lds_bound_graph(520)
    w = w.replace(budget=int(np.median(replay_peaks(w))))
    log("graph capture: seen path n=%d K=%d" % (w.n, w.K))
    got = replay_matches_eager(w, w.budget)
    check_full(w, got)

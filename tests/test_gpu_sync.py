"""The synchronous entry points reuse a stream and device / pinned buffers
kept on the graph. These tests check that reuse changes no result: calls of
growing and shrinking size, different entry points in turn on one graph, a
failed call followed by a good one, and concurrent calls from several
threads (some of which then run on private buffers). Each result is compared
with the same call on a graph of its own (nothing reused), whose results the
parity tests check against the oracle; a few are checked against the oracle
here as well.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def same(a, b):
    assert a.keys() == b.keys()
    for key in a:
        if isinstance(a[key], np.ndarray) or a[key] is None:
            assert (a[key] is None and b[key] is None) or np.array_equal(a[key], b[key]), key
        else:
            assert a[key] == b[key], key


def fresh(w, fn):
    g = ckm.Graph.from_workload(w)
    try:
        return fn(g)
    finally:
        g.close()


def test_grow_shrink_and_mixed_calls():
    w = wl.config(3)
    big = int(w.budget * 2.5)
    p = np.linspace(0.0, 1.0, 40)
    sched = wl.random_schedules(w.n, 24, seed=3, density=0.3, kind="intervals", junk=False)
    S0, R0 = ref.eval_candidate(w, 0, want_rows=True)[2:]
    calls = [
        ("round K=64", lambda g: g.round_eval(w.s_frac, 64, w.seed, big)),
        ("round K=600", lambda g: g.round_eval(w.s_frac, 600, w.seed + 1, big)),
        ("threshold K=40", lambda g: g.threshold_eval(w.s_frac, p, big)),
        ("round K=3", lambda g: g.round_eval(w.s_frac, 3, w.seed, big, want_rows=False)),
        ("schedules K=24", lambda g: g.eval_schedules(sched, big)),
        ("plan", lambda g: dict(zip(("st", "mem"), g.plan(ref.pack_rows(S0), ref.pack_rows(R0))))),
        ("max batch K=100", lambda g: g.max_batch(w.s_frac, 100, w.seed, big, 2 ** 62)),
        ("round K=64 again", lambda g: g.round_eval(w.s_frac, 64, w.seed, big)),
    ]
    g = ckm.Graph.from_workload(w)
    try:
        for name, fn in calls:
            log(name)
            same(fn(g), fresh(w, fn))
    finally:
        g.close()
    # the first call against the oracle
    got = fresh(w, calls[0][1])
    for k in (0, 17, 63):
        assert (int(got["peak"][k]), int(got["cost"][k])) == ref.eval_candidate(w, k)


def test_error_then_good_call():
    w = wl.config(2)
    g = ckm.Graph.from_workload(w)
    try:
        want = g.round_eval(w.s_frac, 50, w.seed, w.budget)
        s = w.s_frac.copy()
        s[100, 7] = np.nan
        with pytest.raises(ckm.CkmError) as e:
            g.round_eval(s, 50, w.seed, w.budget)
        assert e.value.status == ckm.E_INVALID_ARG and "NaN" in str(e.value)
        with pytest.raises(ckm.CkmError):
            g.max_batch(s, 50, w.seed, w.budget, 2 ** 62)
        s[7, 100] = np.nan                  # above the diagonal: never read
        s[100, 7] = 0.5
        got = g.round_eval(s, 50, w.seed, w.budget)
        ref_s = w.s_frac.copy()
        ref_s[100, 7] = 0.5
        same(got, fresh(w, lambda h: h.round_eval(ref_s, 50, w.seed, w.budget)))
        same(g.round_eval(w.s_frac, 50, w.seed, w.budget), want)
        # a strided S* (ld > n) through the staging copy
        wide = np.zeros((w.n, w.n + 5))
        wide[:, :w.n] = w.s_frac
        wide[:, w.n:] = np.nan
        same(g.round_eval(wide, 50, w.seed, w.budget), want)
    finally:
        g.close()


def test_concurrent_threads_one_graph():
    w = wl.config(3)
    big = int(w.budget * 2.5)
    jobs = [(K, seed) for K in (32, 200, 64, 129) for seed in (1, 2, 3)]
    want = {job: fresh(w, lambda g, job=job: g.round_eval(w.s_frac, job[0], job[1], big)) for job in jobs}
    g = ckm.Graph.from_workload(w)
    try:
        log("%d calls on 6 threads" % len(jobs))
        with ThreadPoolExecutor(6) as ex:
            for _ in range(2):
                res = list(ex.map(lambda job: g.round_eval(w.s_frac, job[0], job[1], big), jobs))
                for job, r in zip(jobs, res):
                    same(r, want[job])
    finally:
        g.close()


def test_binding_refuses_wrong_device_tensors():
    """Wrong dtype, layout or size of a device argument is a ValueError from
    the binding, raised before any launch."""
    import torch
    w = wl.config(2)
    K = 64
    g = ckm.Graph.from_workload(w)
    try:
        work = g.alloc_work(K)
        out = g.alloc_outputs(K)
        d_s = torch.from_numpy(w.s_frac).cuda()
        with pytest.raises(ValueError):
            g.quantize_async(d_s.float(), work)                  # float32 S*
        with pytest.raises(ValueError):
            g.quantize_async(d_s[:-1], work)                     # n - 1 rows
        with pytest.raises(ValueError):
            g.quantize_async(d_s.t(), work)                      # column stride n
        short = dict(out, peak=out["peak"][:K - 1])
        with pytest.raises(ValueError):
            g.round_eval_async(d_s, K, w.seed, w.budget, 0, short, work)
        bad = dict(out, best_k=out["best_k"].to(torch.int64))
        with pytest.raises(ValueError):
            g.round_eval_async(d_s, K, w.seed, w.budget, 0, bad, work)
        # the correct call still runs
        g.round_eval_async(d_s, K, w.seed, w.budget, 0, out, work)
        torch.cuda.synchronize()
        assert int(out["status"].item()) == ckm.OK
        want = g.round_eval(w.s_frac, K, w.seed, w.budget)
        assert np.array_equal(out["peak"].cpu().numpy(), want["peak"])
    finally:
        g.close()


def test_async_calls_from_threads_on_own_streams():
    """Async calls on one graph from 4 threads, each with its own stream and
    work buffer (calls only enqueue; the graph is shared read-only), give the
    synchronous call's results."""
    import torch
    w = wl.config(3)
    big = int(w.budget * 2.5)
    jobs = [(K, seed) for K in (64, 300) for seed in (5, 6)]
    want = {job: fresh(w, lambda g, job=job: g.round_eval(w.s_frac, job[0], job[1], big)) for job in jobs}
    g = ckm.Graph.from_workload(w)
    d_s = torch.from_numpy(w.s_frac).cuda()
    torch.cuda.synchronize()

    def run(job):
        K, seed = job
        stream = torch.cuda.Stream()
        with torch.cuda.stream(stream):
            work = g.alloc_work(K)
            out = g.alloc_outputs(K)
        g.round_eval_async(d_s, K, seed, big, 0, out, work, stream)
        stream.synchronize()
        return {k: v.cpu().numpy() for k, v in out.items()}

    try:
        log("%d async jobs on 4 threads" % len(jobs))
        with ThreadPoolExecutor(4) as ex:
            for _ in range(2):
                for job, got in zip(jobs, ex.map(run, jobs)):
                    assert int(got["status"][0]) == ckm.OK
                    for key in ("peak", "cost", "feasible"):
                        assert np.array_equal(got[key], want[job][key]), (job, key)
                    assert int(got["best_k"][0]) == want[job]["best_k"]
                    assert np.array_equal(got["best_S"].view(np.uint64), want[job]["best_S"])
                    assert np.array_equal(got["best_R"].view(np.uint64), want[job]["best_R"])
    finally:
        g.close()


def test_async_threads_on_one_overlapped_graph():
    """The same from 4 threads on a graph whose evaluate takes the overlapped
    launch (the graph's second stream, shared by the calls, and its two
    events): every result equals the call that stays on one stream (the
    entry point that allocates nothing), and sampled candidates the oracle."""
    import torch
    from test_gpu_seen import lds_bound_graph
    w = lds_bound_graph(520)
    big = 1 << 40
    jobs = [(K, seed) for K in (520, 600) for seed in (5, 6)]

    def single_stream(g, K, seed):
        d = torch.from_numpy(w.s_frac).cuda()
        out = g.alloc_outputs(K)
        g.round_eval_noalloc(d, K, seed, big, 0, out)
        torch.cuda.synchronize()
        return {k: v.cpu().numpy() for k, v in out.items()}

    want = {job: fresh(w, lambda g, job=job: single_stream(g, *job)) for job in jobs}
    for (K, seed), res in want.items():
        ks = [0, 63, 64, K - 1]
        orc = {k: ref.eval_candidate(w.replace(seed=seed), k) for k in ks}
        for k in ks:
            assert (int(res["peak"][k]), int(res["cost"][k])) == orc[k], (K, seed, k)
    g = ckm.Graph.from_workload(w)
    d_s = torch.from_numpy(w.s_frac).cuda()
    torch.cuda.synchronize()

    def run(job):
        K, seed = job
        stream = torch.cuda.Stream()
        with torch.cuda.stream(stream):
            work = g.alloc_work(K)
            out = g.alloc_outputs(K)
        g.round_eval_async(d_s, K, seed, big, 0, out, work, stream)
        stream.synchronize()
        return {k: v.cpu().numpy() for k, v in out.items()}

    try:
        log("%d overlapped async jobs on 4 threads" % len(jobs))
        with ThreadPoolExecutor(4) as ex:
            for _ in range(2):
                for job, got in zip(jobs, ex.map(run, jobs)):
                    for key in ("status", "peak", "cost", "feasible", "best_k", "best_S", "best_R"):
                        assert np.array_equal(got[key], want[job][key]), (job, key)
    finally:
        g.close()

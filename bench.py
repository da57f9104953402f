"""Throughput of batched candidate-schedule evaluation on one MI355X.

A step is one pass of the whole path over the transformer-stack workload
(n = 1009 nodes, K = 1024 candidates, 25 % budget): thresholds from S*,
rounding of every candidate's S rows, Algorithm 2 repair + memory/cost
simulation of every candidate (both in one ckm_evaluate_async call; the
evaluate kernel is the dominant one, and split steps, with the rounding
launched on its own by ckm_round_async, time it alone with HIP events on its
stream), per-candidate reduction, argmin, and the best candidate's S and R
rows.
The graph and S* are resident in HBM before timing starts.

Prints one JSON line. `value` is candidate schedules evaluated per second.
`roofline` prices the dominant kernel (the evaluate kernel) against HBM
bandwidth with the algorithmic bytes of bit-packed S and R rows, each
written once and read once: 4 * n * ceil(n/64) * 8 bytes per candidate.
`roofline_alu` prices the same launch against the vector ALU issue rate:
VALU instructions per launch (committed rocprofv3 counters of the current
kernel source, else null) x 64 lanes / the launch time, against 256 CUs x 4
SIMDs x 16 lanes x 2.4 GHz. (The kernel's own limit is its scalar issue and
the round trip of each node's loads; the vector unit is about 70 % busy.)
`roofline_step` prices the whole timed step with the same bytes.
`cpu_baseline` times the CPU oracle on a bounded sample of the same
workload (about 15 s of wall time, whole passes over the candidates), on the host threads a one-GPU job is
granted (16, or fewer when the affinity set is smaller; candidates split
across them) and on one thread, with the CPU model, the machine's logical
CPU count and the affinity set recorded.
`hbm_copy` is the bandwidth a plain device copy reaches on the same GPU, the
achievable line beside the 8 TB/s peak. `host_round_trip` times the
synchronous call that takes S* from host memory and returns host results
(PCIe transfers and the call's own copies included; its buffers stay on
the graph between calls). `supplied_schedules` times the batch evaluation of K given integral
checkpoint matrices (banded, 30 % of values kept) on the same graph: Algorithm
2 repair, simulation, argmin and the best R, with the matrices resident in HBM.
`threshold_family` times K deterministic candidates [clamp(S*) > p_k] on an
even threshold grid over [0, 1] for the same graph and S*: keys, evaluation,
argmin and the best S and R.
`max_batch` times quantize + evaluate + the largest batch multiplier of
every candidate (budget 3x the median activation peak, cost cap at the
median cost) on the same workload.
`pipelined` times the same steps over two work buffers, a step's thresholds
and rounding on a second stream beside the previous step's evaluation (whose
tail, and the small kernels, leave room for it), timed by events around the
whole loop only:
per-step timing events on the main stream stop the two from overlapping.
`feasible_budget` times the same step at the median-peak budget, where
select also writes the best candidate's S and R rows.
`execution_plan` times Algorithm 1's plan (with the memory after each
statement) for the step's best candidate, or candidate 0's rows when none
is feasible, read from HBM where the step left them.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidate schedules evaluated/sec at n=1000,K=1024; % HBM roofline"
HBM_PEAK_GBS = 8000.0
# int32 VALU lane-operations per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
ALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_eval_transformer_n1009_K1024.json")
KERNEL_SRC = os.path.join(ROOT, "paper_1910_02653_amd", "csrc", "ckm_kernels.hip")


def kernel_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_counters():
    """Counters of one evaluate launch from committed rocprofv3 runs (HBM
    bytes, VALU instructions), if they were taken on the current kernel
    source; else {}."""
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return {}
    if d.get("kernel_sha256_16") != kernel_hash():
        return {}
    return d


# Host threads a one-GPU job is granted on the machines it runs on.
HOST_THREADS_PER_GPU = 16


def host_info():
    """CPU model, logical CPUs of the machine, CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": os.cpu_count() or 1, "affinity_cpus": affinity}


def host_threads() -> int:
    """Oracle threads: the CPUs of this process's affinity set, at most the
    16 host threads a one-GPU job is granted (more would contend with other
    jobs on the same host, whatever the affinity set shows)."""
    return max(1, min(HOST_THREADS_PER_GPU, host_info()["affinity_cpus"]))


def progress(msg):
    """One line on stderr as each part of the run ends (the JSON line alone
    goes to stdout)."""
    print("[bench] " + msg, file=sys.stderr, flush=True)


def cpu_baseline(w, sample: int, single: int, target_s: float = 15.0):
    """The oracle on candidates 0 .. sample-1 of the workload, split by
    candidate over the oracle threads (each thread runs the unmodified oracle
    on its own candidates; candidates are independent), and on candidates
    0 .. single-1 in one thread. Each run takes whole passes over its
    candidates until about target_s seconds (the multi-thread run) or a third
    of that (the single thread) have passed, at least one pass."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import ref
    q = ref.quantize(w.s_frac)
    threads = host_threads()

    def passes(ks, seconds):
        """Whole passes over ks until `seconds` have passed: candidates done."""
        done = 0
        end = time.perf_counter() + seconds
        while True:
            for k in ks:
                ref.eval_candidate(w, k, q=q)
            done += len(ks)
            if time.perf_counter() >= end:
                return done

    t = time.perf_counter()
    ref.eval_candidate(w, 0, q=q)
    one = time.perf_counter() - t
    # fewer candidates where one pass over them would take much longer
    single = max(1, min(single, int(target_s / 3 / one)))
    sample = max(threads, min(sample, int(target_s * threads / one)))
    t = time.perf_counter()
    n1 = passes(range(single), target_s / 3)
    dt1 = time.perf_counter() - t
    chunks = [range(i, sample, threads) for i in range(threads)]
    t = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        done = sum(ex.map(lambda ks: passes(ks, target_s), chunks))
    dt = time.perf_counter() - t
    info = host_info()
    return {"value": done / dt, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "stage_evals_per_s": done * w.n / dt,
            "sample": "%d candidate evaluations over candidates 0-%d of the same %d-candidate workload "
                      "(%s, n=%d): rounding + Algorithm 2 repair + literal U/FREE simulation per candidate, "
                      "%d threads (candidates split across them), %.1f s wall"
                      % (done, sample - 1, w.K, w.name, w.n, threads, dt),
            "host": dict(info, threads_used=threads,
                         thread_cap="at most %d: the host threads a one-GPU job is granted" % HOST_THREADS_PER_GPU),
            "single_thread": {"value": n1 / dt1, "unit": "candidates/s", "cores": 1,
                              "sample": "%d candidate evaluations over candidates 0-%d, %.1f s"
                                        % (n1, single - 1, dt1)}}


def copy_bandwidth(stream, nbytes: int = 1 << 30, reps: int = 10):
    """Achievable HBM bandwidth of a plain device copy (read + write bytes per
    second), timed with events on the bench stream."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    with torch.cuda.stream(stream):
        for _ in range(2):
            b.copy_(a)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            b.copy_(a)
        t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del a, b
    torch.cuda.empty_cache()
    return 2 * nbytes / (ms * 1e-3) / 1e9


def time_host_round_trip(g, w, K, steps):
    """The synchronous ckm_round_eval: S* from host memory, results back to
    host memory, work buffer allocated inside the call (PCIe included)."""
    for _ in range(2):
        g.round_eval(w.s_frac, K, w.seed, w.budget)
    ts = []
    for _ in range(steps):
        t = time.perf_counter()
        g.round_eval(w.s_frac, K, w.seed, w.budget)
        ts.append(time.perf_counter() - t)
    ms = 1e3 * sorted(ts)[len(ts) // 2]
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_call_median": ms, "steps": steps,
            "input": "host S* (%.1f MB fp64) in, host peak/cost/feasible and best S/R out, "
                     "synchronous C-ABI call" % (w.s_frac.nbytes / 1e6)}


def time_schedules(g, w, K, steps, stream):
    """Throughput of ckm_eval_schedules_async on K banded integral S matrices."""
    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm
    from paper_1910_02653_amd import workloads as wl

    rows = wl.random_schedules(w.n, K, seed=w.seed + 1, density=0.3, kind="intervals", junk=False)
    d_S = torch.from_numpy(rows.view(np.int64)).cuda()
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)
    for _ in range(3):
        g.eval_schedules_async(d_S, K, w.budget, out, work, stream)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        g.eval_schedules_async(d_S, K, w.budget, out, work, stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_call": ms, "steps": steps,
            "input": "K=%d banded S matrices (each value kept with p=0.3 over a random stage range), "
                     "%.1f MB of bit rows in HBM" % (K, rows.nbytes / 1e6)}


def time_thresholds(g, w, K, steps, stream, d_s):
    """Throughput of ckm_threshold_eval_async on an even grid of K thresholds."""
    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm

    d_p = torch.from_numpy(np.linspace(0.0, 1.0, K)).cuda()
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)
    for _ in range(3):
        g.threshold_eval_async(d_s, d_p, w.budget, out, work, stream)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        g.threshold_eval_async(d_s, d_p, w.budget, out, work, stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_call": ms, "steps": steps,
            "input": "K=%d thresholds evenly spaced over [0, 1] on the workload's S*" % K}


def time_max_batch(g, w, steps, stream, d_s):
    """Throughput of quantize + evaluate + ckm_max_batch_async."""
    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm

    K = w.K
    work = g.alloc_work(K)
    out = g.alloc_outputs(K, rows=False)
    g.round_eval_async(d_s, K, w.seed, 2 ** 62, 0, out, work, stream)
    torch.cuda.synchronize()
    peak, cost = out["peak"].cpu().numpy(), out["cost"].cpu().numpy()
    base = w.m_input + 2 * w.m_param
    budget = int(base + 3 * (np.median(peak) - base))
    cap = int(np.median(cost))
    d_b = torch.empty(K, dtype=torch.int64, device="cuda")
    d_bk = torch.empty(1, dtype=torch.int32, device="cuda")
    d_bb = torch.empty(1, dtype=torch.int64, device="cuda")
    d_st = torch.empty(1, dtype=torch.int32, device="cuda")

    def call():
        g.quantize_async(d_s, work, stream)
        g.evaluate_async(K, w.seed, 0, work, stream=stream)
        g.max_batch_async(K, budget, cap, d_b, d_bk, d_bb, d_st, work, stream)

    for _ in range(3):
        call()
    torch.cuda.synchronize()
    assert int(d_st.item()) == ckm.OK
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        call()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_call": ms, "steps": steps,
            "best_k": int(d_bk.item()), "best_batch": int(d_bb.item()),
            "input": "K=%d rounded candidates, budget %d B (3x the median activation peak), cost cap %d "
                     "(median cost)" % (K, budget, cap)}


def time_feasible(g, w, steps, stream, d_s):
    """The bench step at a budget half the candidates meet (the median
    peak), so select also writes the best candidate's S and R rows."""
    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm

    K = w.K
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)
    g.round_eval_async(d_s, K, w.seed, 2 ** 62, 0, out, work, stream)
    torch.cuda.synchronize()
    budget = int(np.median(out["peak"].cpu().numpy()))

    def call():
        g.quantize_async(d_s, work, stream)
        g.round_async(K, w.seed, 0, work, stream)
        g.evaluate_async(K, w.seed, ckm.F_ROUNDED, work, stream=stream)
        g.select_async(K, w.seed, budget, ckm.F_ROUNDED, out, work, stream)

    for _ in range(3):
        call()
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK and int(out["best_k"].item()) >= 0
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        call()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_step": ms, "steps": steps,
            "best_k": int(out["best_k"].item()),
            "input": "the bench step at the median-peak budget %d B (best S and R rows written)" % budget}


def time_pipelined(g, w, steps, stream, d_s):
    """Consecutive steps overlapped: thresholds and rounding of step i+1 (on
    a second stream, into the other of two work buffers) beside the
    evaluation and selection of step i. Events order each buffer's reuse."""
    import torch

    from paper_1910_02653_amd import ckm

    K = w.K
    works = [g.alloc_work(K), g.alloc_work(K)]
    out = g.alloc_outputs(K)
    side = torch.cuda.Stream()              # default priority, like the main stream
    rounded = [torch.cuda.Event(), torch.cuda.Event()]
    released = [torch.cuda.Event(), torch.cuda.Event()]
    for e in released:
        e.record(stream)

    def step(i):
        b = i & 1
        side.wait_event(released[b])        # the step two back is done with this buffer
        g.quantize_async(d_s, works[b], side)
        g.round_async(K, w.seed, 0, works[b], side)
        rounded[b].record(side)
        stream.wait_event(rounded[b])
        g.evaluate_async(K, w.seed, ckm.F_ROUNDED, works[b], stream=stream)
        g.select_async(K, w.seed, w.budget, 0, out, works[b], stream)
        released[b].record(stream)

    for i in range(10):
        step(i)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(steps):
        step(i)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_step": ms, "steps": steps,
            "input": "the bench step, consecutive steps overlapped on two streams and two work buffers"}


def time_graph(g, w, steps, d_s):
    """The bench step captured once into a HIP graph (torch.cuda.CUDAGraph
    over the library's launches) and replayed: the same kernels without the
    host's per-launch work. Every replay repeats the whole step."""
    import torch

    from paper_1910_02653_amd import ckm

    K = w.K
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)

    def step():
        g.quantize_async(d_s, work)
        g.evaluate_async(K, w.seed, 0, work)
        g.select_async(K, w.seed, w.budget, 0, out, work)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    cg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(cg):
        step()
    torch.cuda.synchronize()
    for _ in range(10):
        cg.replay()
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        cg.replay()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"value": K / (ms * 1e-3), "unit": "candidates/s", "ms_per_step": ms, "steps": steps,
            "input": "the bench step captured once into a HIP graph, replayed"}


def time_plan(g, w, steps, stream, d_s):
    """Throughput of ckm_plan_async on one schedule of the workload: the best
    candidate at the median-peak budget (a budget some candidates meet)."""
    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm

    K = w.K
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)
    g.round_eval_async(d_s, K, w.seed, 2 ** 62, 0, out, work, stream)
    torch.cuda.synchronize()
    budget = int(np.median(out["peak"].cpu().numpy()))
    g.round_eval_async(d_s, K, w.seed, budget, 0, out, work, stream)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK and int(out["best_k"].item()) >= 0
    cap = w.n * (w.n + 1)
    d_P = torch.empty((cap, 4), dtype=torch.int32, device="cuda")
    d_mem = torch.empty(cap, dtype=torch.int64, device="cuda")
    d_cnt = torch.empty(1, dtype=torch.int64, device="cuda")
    d_st = torch.empty(1, dtype=torch.int32, device="cuda")
    for _ in range(3):
        g.plan_async(out["best_S"], out["best_R"], False, d_P, cap, d_cnt, d_mem, d_st, work, stream)
    torch.cuda.synchronize()
    assert int(d_st.item()) == ckm.OK
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        g.plan_async(out["best_S"], out["best_R"], False, d_P, cap, d_cnt, d_mem, d_st, work, stream)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    cnt = int(d_cnt.item())
    return {"ms_per_call": ms, "statements": cnt, "statements_per_s": cnt / (ms * 1e-3), "steps": steps,
            "input": "candidate %d of %d (best at the median-peak budget %d B), n=%d"
                     % (int(out["best_k"].item()), K, budget, w.n)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4, help="workload 1..5 (4 = transformer stack)")
    ap.add_argument("--splits", type=int, default=0, help="stage splits per 64 candidates (0 = auto)")
    ap.add_argument("--cpu-sample", type=int, default=1024,
                    help="oracle candidates to time on all host threads (0 = skip)")
    ap.add_argument("--cpu-single", type=int, default=128, help="oracle candidates to time on one thread")
    ap.add_argument("--host-steps", type=int, default=10,
                    help="timed synchronous calls with host buffers (0 = skip)")
    ap.add_argument("--sched-steps", type=int, default=20,
                    help="timed calls of the supplied-schedule evaluation (0 = skip)")
    ap.add_argument("--thr-steps", type=int, default=20,
                    help="timed calls of the threshold-family evaluation (0 = skip)")
    ap.add_argument("--plan-steps", type=int, default=20,
                    help="timed calls of the execution-plan generation (0 = skip)")
    ap.add_argument("--graph-steps", type=int, default=100,
                    help="replays of the step captured into a HIP graph (0 = skip)")
    ap.add_argument("--pipe-steps", type=int, default=100,
                    help="timed steps with consecutive steps overlapped (0 = skip)")
    ap.add_argument("--feasible-steps", type=int, default=20,
                    help="timed steps at the median-peak budget (0 = skip)")
    ap.add_argument("--batch-steps", type=int, default=20,
                    help="timed calls of the largest-batch search (0 = skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(candidates would shard across GPUs with one small all-gather; not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1910_02653_amd import ckm
    from paper_1910_02653_amd import workloads as wl

    torch.cuda.set_device(0)
    w = wl.config(args.config)
    n, K = w.n, w.K
    W = (n + 63) // 64
    g = ckm.Graph.from_workload(w)
    d_s = torch.from_numpy(w.s_frac).cuda()
    work = g.alloc_work(K)
    out = g.alloc_outputs(K)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        # quantize, round + evaluate (one call: the library overlaps the
        # rounding of later candidate groups with the evaluate of earlier
        # ones), select
        if ev is not None:
            ev[0].record(stream)
        g.quantize_async(d_s, work, stream)
        g.evaluate_async(K, w.seed, 0, work, stage_splits=args.splits, stream=stream)
        g.select_async(K, w.seed, w.budget, 0, out, work, stream)
        if ev is not None:
            ev[1].record(stream)

    def split_step(ev):
        # the same step with the rounding as a launch of its own, so that
        # events around the evaluate kernel time it alone
        g.quantize_async(d_s, work, stream)
        g.round_async(K, w.seed, 0, work, stream)
        ev[0].record(stream)
        g.evaluate_async(K, w.seed, ckm.F_ROUNDED, work, stage_splits=args.splits, stream=stream)
        ev[1].record(stream)
        g.select_async(K, w.seed, w.budget, 0, out, work, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert int(out["status"].item()) == ckm.OK

    # the timed steps: nothing but the steps between the two events
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for i in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps
    # the same number of steps again with events around each step, for the
    # per-step median, and split steps with events around the evaluate
    # kernel, for its time (events in the stream add a little time of their
    # own, so these steps are not the timed ones)
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(2)) for _ in range(args.steps)]
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    step_ms = [e[0].elapsed_time(e[1]) for e in evs]
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(2)) for _ in range(args.steps)]
    for i in range(args.steps):
        split_step(evs[i])
    torch.cuda.synchronize()
    eval_ms = [e[0].elapsed_time(e[1]) for e in evs]
    eval_avg_ms = float(np.mean(eval_ms))
    copy_gbs = copy_bandwidth(stream)

    b_cand = 4 * n * W * 8
    achieved = K * b_cand / (eval_avg_ms * 1e-3) / 1e9
    # the committed counters are those of the transformer workload's launch
    counters = measured_counters() if args.config == 4 else {}
    traffic = counters.get("hbm_bytes_per_launch")
    valu = counters.get("valu_insts_per_launch")
    result = {
        "metric": METRIC,
        "value": K / (ms_step * 1e-3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": "%s n=%d K=%d budget %.0f%% of checkpoint-all (seq 2048, hidden 2048, "
                               "24 blocks, mirrored backward)" % (w.name, n, K, w.budget_pct)
                   if args.config == 4 else "%s n=%d K=%d" % (w.name, n, K),
                   "n": n, "K": K, "budget": int(w.budget), "stage_splits": args.splits},
        "ms_per_step_median": float(np.median(step_ms)),
        "stage_evals_per_s": K * n / (ms_step * 1e-3),
        "evaluate_kernel_ms": eval_avg_ms,
        "evaluate_kernel_ms_median": float(np.median(eval_ms)),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic},
        "roofline_step": {"bound": "hbm", "achieved": K * b_cand / (ms_step * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                          "unit": "GB/s", "frac": K * b_cand / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          "note": "the same algorithmic bytes over the whole timed step"},
        "roofline_alu": ({"bound": "alu", "achieved": valu * 64 / (eval_avg_ms * 1e-3) / 1e12,
                          "peak": ALU_PEAK_TOPS, "unit": "T lane-ops/s",
                          "frac": valu * 64 / (eval_avg_ms * 1e-3) / 1e12 / ALU_PEAK_TOPS,
                          "valu_insts_per_launch": valu} if valu else None),
        "hbm_copy": {"achieved": copy_gbs, "unit": "GB/s", "kernel": "device copy of 1 GiB (read + write)",
                     "evaluate_frac": achieved / copy_gbs},
        "wall_s": wall,
    }
    progress("timed steps: %.4f ms per step" % ms_step)
    legs = [
        ("host_round_trip", args.host_steps, lambda: time_host_round_trip(g, w, K, args.host_steps)),
        ("graph_replay", args.graph_steps, lambda: time_graph(g, w, args.graph_steps, d_s)),
        ("pipelined", args.pipe_steps, lambda: time_pipelined(g, w, args.pipe_steps, stream, d_s)),
        ("feasible_budget", args.feasible_steps, lambda: time_feasible(g, w, args.feasible_steps, stream, d_s)),
        ("supplied_schedules", args.sched_steps, lambda: time_schedules(g, w, K, args.sched_steps, stream)),
        ("max_batch", args.batch_steps, lambda: time_max_batch(g, w, args.batch_steps, stream, d_s)),
        ("execution_plan", args.plan_steps, lambda: time_plan(g, w, args.plan_steps, stream, d_s)),
        ("threshold_family", args.thr_steps, lambda: time_thresholds(g, w, K, args.thr_steps, stream, d_s)),
        ("cpu_baseline", args.cpu_sample,
         lambda: cpu_baseline(w, min(args.cpu_sample, K), min(args.cpu_single, K))),
    ]
    for name, count, run in legs:
        if count > 0:
            result[name] = run()
            progress("%s done" % name)
    print(json.dumps(result), flush=True)
    g.close()


if __name__ == "__main__":
    main()

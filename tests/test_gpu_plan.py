"""Bit-exact parity of execution-plan generation (ckm_plan, Section 4.9
Algorithm 1, through the C ABI) with the CPU oracle: every statement (op,
node, register, stage) and the memory after it, late and early
deallocation of unused checkpoints, and the checks of (S, R).

Schedules are Algorithm 2's output on seeded synthetic workloads (the
oracle's rounding and repair), plus the GPU's own best candidate. Expected
values come from the oracle only.
"""
import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import ckm
from paper_1910_02653_amd import workloads as wl

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def junk_above(rows, n, seed, strict):
    """Random bits on / above the diagonal (strict: i >= t, else i > t) and
    in the padding: the plan must ignore them."""
    rng = np.random.default_rng(seed)
    W = rows.shape[1]
    bits = (rng.random((n, W * 64)) < 0.5)
    t = np.arange(n)[:, None]
    i = np.arange(W * 64)[None, :]
    keep_out = (i >= t) if strict else (i > t)
    bits &= keep_out
    packed = np.packbits(bits.astype(np.uint8).reshape(n, W, 64), axis=2, bitorder="little")
    return rows | packed.view(np.uint64).reshape(n, W)


def check_plan(w, S, R, g=None, junk=False, seed=0):
    """GPU plan of (S, R) (n x n 0/1) against the oracle, late and early."""
    own = g is None
    g = ckm.Graph.from_workload(w) if own else g
    try:
        Sr, Rr = ref.pack_rows(S), ref.pack_rows(R)
        if junk:
            Sr = junk_above(Sr, w.n, seed, strict=True)
            Rr = junk_above(Rr, w.n, seed + 1, strict=False)
        for early in (False, True):
            want_st, want_mem = ref.plan(w, S, R, early=early)
            got_st, got_mem = g.plan(Sr, Rr, early=early)
            assert got_st.shape == want_st.shape, (early, got_st.shape, want_st.shape)
            bad = np.nonzero(np.any(got_st != want_st, axis=1))[0]
            assert bad.size == 0, "statement %d: gpu %s oracle %s" % (bad[0], got_st[bad[0]], want_st[bad[0]])
            assert np.array_equal(got_mem, want_mem), "memory differs (early=%s)" % early
        return len(want_st)
    finally:
        if own:
            g.close()


def oracle_schedule(w, k):
    _, _, S, R = ref.eval_candidate(w, k, want_rows=True)
    return S, R


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_configs_candidates(cfg):
    w = wl.config(cfg)
    for k in (0, 1, 5):
        S, R = oracle_schedule(w, k)
        log("config %d candidate %d" % (cfg, k))
        check_plan(w, S, R, junk=(k == 1), seed=k)


def test_config3_sparse_long_closures():
    w = wl.config(3)
    w = w.replace(s_frac=0.2 * w.s_frac)
    S, R = oracle_schedule(w, 3)
    log("config 3 sparse")
    check_plan(w, S, R)


def test_config4_transformer():
    w = wl.config(4)
    S, R = oracle_schedule(w, 7)
    log("config 4 n=%d" % w.n)
    cnt = check_plan(w, S, R)
    assert cnt == 2 * int(R.sum())


def test_config5_random_dag():
    """n = 4001: every statement of one candidate's plan."""
    w = wl.config(5)
    S, R = oracle_schedule(w, 2)
    log("config 5 n=%d" % w.n)
    check_plan(w, S, R)


def test_max_nodes():
    """n = 4096, the largest graph: 128-word columns in the R transpose."""
    w = wl.random_dag(4096, seed=4099, K=4, window=40, max_deg=3, max_size=1000, max_cost=1000,
                      s_kind="uniform", m_input=5, m_param=3)
    S, R = oracle_schedule(w, 1)
    log("n=%d" % w.n)
    check_plan(w, S, R, junk=True, seed=4)


SWEEP = [(1, 0), (2, 1), (3, 2), (31, 3), (32, 4), (33, 5), (63, 6), (64, 7), (65, 8), (127, 9), (129, 10),
         (200, 11), (300, 12)]


@pytest.mark.parametrize("n,seed", SWEEP)
def test_random_dag_sweep(n, seed):
    for kind in ("uniform", "sparse", "binary"):
        w = wl.random_dag(n, seed, max_deg=4, window=min(n, 20), max_size=1000, s_kind=kind, m_input=5,
                          m_param=3)
        S, R = oracle_schedule(w, seed % 4)
        log("random dag n=%d %s" % (n, kind))
        check_plan(w, S, R, junk=(kind == "binary"), seed=seed)


def test_checkpoint_all_and_none():
    w = wl.config(2)
    n = w.n
    full = np.tri(n, n, -1, dtype=np.uint8)
    for S in (full, np.zeros((n, n), np.uint8)):
        R = ref.solve_R(w, S)
        check_plan(w, S, R)


def test_best_candidate_from_round_eval_async():
    """The plan of the rounding path's best candidate, chained on one stream
    with no host round trip."""
    import torch
    w = wl.config(3)
    g = ckm.Graph.from_workload(w)
    try:
        K = 256
        budget = int(w.budget * 2.5)
        work = g.alloc_work(K)
        out = g.alloc_outputs(K)
        g.round_eval_async(torch.from_numpy(w.s_frac).cuda(), K, w.seed, budget, 0, out, work)
        cap = ckm.MAX_NODES * 0 + w.n * (w.n + 1)
        d_P = torch.empty((cap, 4), dtype=torch.int32, device="cuda")
        d_mem = torch.empty(cap, dtype=torch.int64, device="cuda")
        d_cnt = torch.empty(1, dtype=torch.int64, device="cuda")
        d_st = torch.full((1,), -5, dtype=torch.int32, device="cuda")
        g.plan_async(out["best_S"], out["best_R"], False, d_P, cap, d_cnt, d_mem, d_st, work)
        torch.cuda.synchronize()
        bk = int(out["best_k"].item())
        assert bk >= 0
        assert int(d_st.item()) == ckm.OK
        c = int(d_cnt.item())
        _, _, S, R = ref.eval_candidate(w, bk, want_rows=True)
        want_st, want_mem = ref.plan(w, S, R)
        assert c == len(want_st)
        assert np.array_equal(d_P[:c].cpu().numpy(), want_st)
        assert np.array_equal(d_mem[:c].cpu().numpy(), want_mem)
        # peak of the plan = the candidate's peak
        assert int(want_mem.max()) == int(out["peak"][bk].item())
        # count only, then too small a capacity
        g.plan_async(out["best_S"], out["best_R"], True, None, 0, d_cnt, None, d_st, work)
        torch.cuda.synchronize()
        assert int(d_cnt.item()) == c and int(d_st.item()) == ckm.OK
        d_st.fill_(-5)
        g.plan_async(out["best_S"], out["best_R"], False, d_P, c - 1, d_cnt, d_mem, d_st, work)
        torch.cuda.synchronize()
        assert int(d_cnt.item()) == c and int(d_st.item()) == ckm.E_INVALID_ARG
    finally:
        g.close()


def test_invalid_schedules_rejected():
    """(4a), (1b), (1c) and a kept-and-recomputed value are checked."""
    w = wl.config(2)
    S, R = oracle_schedule(w, 0)
    g = ckm.Graph.from_workload(w)
    try:
        ts, is_ = np.nonzero(np.tril(R, -1))
        cases = []
        R1 = R.copy()
        R1[40, 40] = 0
        cases.append(("4a", S, R1))
        R2 = R.copy()
        R2[ts[0], is_[0]] = 0               # Algorithm 2's R is least: this breaks (1b) or (1c)
        cases.append(("dropped", S, R2))
        st_, si_ = np.nonzero(S)
        R3 = R.copy()
        R3[st_[0], si_[0]] = 1
        cases.append(("kept and recomputed", S, R3))
        S4 = S.copy()
        S4[w.n - 1, :w.n - 1] = 1           # (1c): values kept that were not resident
        cases.append(("1c", S4, R))
        for name, Sx, Rx in cases:
            assert ref.check_schedule(w, Sx, Rx) == ref.E_INVALID_ARG, name
            log("invalid: %s" % name)
            with pytest.raises(ckm.CkmError) as e:
                g.plan(ref.pack_rows(Sx), ref.pack_rows(Rx))
            assert e.value.status == ckm.E_INVALID_ARG, name
        # too small a capacity: an error, and the count is reported
        c = len(ref.plan(w, S, R)[0])
        with pytest.raises(ckm.CkmError) as e:
            g.plan(ref.pack_rows(S), ref.pack_rows(R), capacity=c - 1)
        assert e.value.status == ckm.E_INVALID_ARG
        st, _ = g.plan(ref.pack_rows(S), ref.pack_rows(R), capacity=c + 10)
        assert len(st) == c
    finally:
        g.close()

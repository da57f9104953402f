"""Pins of the oracle's execution-plan generator (Section 4.9, Algorithm 1)
and of its schedule check, on the CPU.

- Hand-worked plans in tests/golden/ (the diamond of the Algorithm 2 worked
  example, and a chain with an unused checkpoint, late and early).
- An independent replay of every plan: registers are defined once and freed
  once, every computed node finds its deps live, the values live at the end
  of stage t are exactly S[t+1], nothing is live at the end, and the memory
  after each statement equals the U recurrence of the simulator (stage peaks
  and end-of-stage memory), which is pinned on its own.
- The check: Algorithm 2's R passes; removing any single entry of that R
  (its least feasible R) or overlapping it with S fails.
"""
import os

import numpy as np
import pytest

from oracle import ref
from paper_1910_02653_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
OPS = {"compute": 0, "deallocate": 1}


def read_plan_fixture(name):
    """Lines '[label] op node register stage memory' -> {label: (stmts, mem)}."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            label = tok.pop(0) if tok[0] not in OPS else ""
            st, mem = out.setdefault(label, ([], []))
            st.append([OPS[tok[0]], int(tok[1]), int(tok[2]), int(tok[3])])
            mem.append(int(tok[4]))
    return {k: (np.array(v[0], np.int32), np.array(v[1], np.int64)) for k, v in out.items()}


def graph(deps, size, m_input=0, m_param=0):
    ptr, idx = wl.csr_from_deps(deps)
    n = len(deps)
    return wl.Workload("g", n, ptr, idx, np.ones(n, np.int64), np.asarray(size, np.int64), m_input, m_param,
                       np.zeros((n, n)), 1, 0, 0)


def test_diamond_plan_golden():
    w = graph([[], [0], [0], [1, 2]], [1, 2, 4, 8])
    S = np.zeros((4, 4), np.uint8)
    S[2, 0] = S[3, 2] = 1
    R = ref.solve_R(w, S)
    want_st, want_mem = read_plan_fixture("plan_diamond.txt")[""]
    st, mem = ref.plan(w, S, R)
    assert st.tolist() == want_st.tolist()
    assert mem.tolist() == want_mem.tolist()


def test_descending_csr_plan_golden():
    """Releases after one compute come in increasing node order, also when
    the graph's CSR row lists the dependencies in another order."""
    n = 4
    ptr = np.array([0, 0, 0, 0, 3], np.int32)
    idx = np.array([2, 0, 1], np.int32)          # node 3's row, unsorted
    w = wl.Workload("g", n, ptr, idx, np.ones(n, np.int64), np.array([1, 2, 4, 8], np.int64), 0, 0,
                    np.zeros((n, n)), 1, 0, 0)
    S = np.zeros((n, n), np.uint8)
    R = ref.solve_R(w, S)
    want_R = np.eye(n, dtype=np.uint8)
    want_R[3, :3] = 1
    assert np.array_equal(R, want_R)
    want_st, want_mem = read_plan_fixture("plan_descending_deps.txt")[""]
    for early in (False, True):                  # no unused checkpoints: same plan
        st, mem = ref.plan(w, S, R, early=early)
        assert st.tolist() == want_st.tolist()
        assert mem.tolist() == want_mem.tolist()
    # the same graph with its rows sorted gives the same plan
    ws = w.replace(dep_idx=np.array([0, 1, 2], np.int32))
    st, mem = ref.plan(ws, S, R)
    assert st.tolist() == want_st.tolist()


def test_unused_checkpoint_plans_golden():
    w = graph([[], [0], [1]], [1, 2, 4])
    S = np.zeros((3, 3), np.uint8)
    S[1, 0] = S[2, 0] = S[2, 1] = 1
    R = ref.solve_R(w, S)
    assert np.array_equal(R, np.eye(3, dtype=np.uint8))
    fx = read_plan_fixture("plan_unused_checkpoint.txt")
    for label, early in (("late", False), ("early", True)):
        st, mem = ref.plan(w, S, R, early=early)
        assert st.tolist() == fx[label][0].tolist(), label
        assert mem.tolist() == fx[label][1].tolist(), label
    sim = ref.simulate(w, S, R)
    assert list(sim["stage_peak"]) == [1, 3, 7]


def replay(w, S, R, st, mem):
    """Interpret the plan; check it against (S, R) and the simulator."""
    n = w.n
    deps = [w.dep_idx[w.dep_ptr[j]:w.dep_ptr[j + 1]].tolist() for j in range(n)]
    base = w.m_input + 2 * w.m_param
    live = {}                      # register -> node
    seen = set()
    computes = 0
    stage_max = np.full(n, np.iinfo(np.int64).min, np.int64)
    end_mem = np.zeros(n, np.int64)
    last_stage = -1
    used_bytes = base
    for s, (op, node, reg, t) in enumerate(st.tolist()):
        assert t >= last_stage, "stages out of order"
        if t != last_stage:
            if last_stage >= 0:
                # end of stage last_stage: the live values are S[last_stage + 1]
                nodes = sorted(live.values())
                want = np.nonzero(S[last_stage + 1, :last_stage + 1])[0].tolist() if last_stage + 1 < n else []
                assert nodes == want, "live set at the end of stage %d" % last_stage
                end_mem[last_stage] = used_bytes
            last_stage = t
        if op == 0:
            assert reg not in seen, "register defined twice"
            assert R[t, node] == 1
            seen.add(reg)
            for i in deps[node]:
                assert i in live.values(), "v%d computed without its dep v%d live" % (node, i)
            live[reg] = node
            used_bytes += int(w.size[node])
            computes += 1
        else:
            assert live.get(reg) == node, "deallocating a dead or wrong register"
            del live[reg]
            used_bytes -= int(w.size[node])
        assert mem[s] == used_bytes
        stage_max[t] = max(stage_max[t], used_bytes)
    assert not live, "values live after the last stage"
    end_mem[last_stage] = used_bytes
    assert computes == int(R.sum())
    assert sorted(seen) == list(range(computes)), "registers are not numbered in order"
    return stage_max, end_mem


@pytest.mark.parametrize("n,seed,kind", [(8, 0, "uniform"), (17, 1, "sparse"), (30, 2, "beta"),
                                         (45, 3, "uniform"), (64, 4, "binary")])
def test_plan_replay_matches_simulation(n, seed, kind):
    w = wl.random_dag(n, seed, max_deg=3, window=10, max_size=50, s_kind=kind, m_input=3, m_param=2)
    q = ref.quantize(w.s_frac)
    for k in range(4):
        S = ref.round_random(q, seed, k)
        R = ref.solve_R(w, S)
        assert ref.check_schedule(w, S, R) == ref.OK
        sim = ref.simulate(w, S, R)
        st, mem = ref.plan(w, S, R)
        stage_max, end_mem = replay(w, S, R, st, mem)
        # the late plan's memory is the U recurrence: same stage peaks. At a
        # stage's end the plan holds base + the kept values; the recurrence
        # still counts the unused checkpoints that the plan deallocates there
        assert np.array_equal(stage_max, sim["stage_peak"])
        base = w.m_input + 2 * w.m_param
        users = [[] for _ in range(n)]
        for j in range(n):
            for i in w.dep_idx[w.dep_ptr[j]:w.dep_ptr[j + 1]]:
                users[int(i)].append(j)
        for t in range(n):
            kept = S[t + 1] if t + 1 < n else np.zeros(n, np.uint8)
            assert end_mem[t] == base + int((w.size * kept).sum())
            unused = sum(int(w.size[i]) for i in range(t)
                         if S[t, i] and not kept[i] and not any(j <= t and R[t, j] for j in users[i]))
            assert sim["U_end"][t] == end_mem[t] + unused
        # early: the same statements with unused checkpoints moved to the
        # start of their stage; never more memory
        st2, mem2 = ref.plan(w, S, R, early=True)
        stage_max2, _ = replay(w, S, R, st2, mem2)
        assert np.all(stage_max2 <= stage_max)
        assert sorted(map(tuple, st2.tolist())) == sorted(map(tuple, st.tolist()))


def test_check_schedule_minimality():
    """Algorithm 2's R is the least feasible R (pinned by brute force in
    test_oracle): dropping any off-diagonal entry breaks (1b) or (1c),
    dropping a diagonal one breaks (4a), and recomputing a kept value is
    rejected."""
    w = wl.random_dag(12, 7, max_deg=3, window=6)
    rng = np.random.default_rng(1)
    for _ in range(5):
        S = np.tril((rng.random((12, 12)) < 0.3).astype(np.uint8), -1)
        R = ref.solve_R(w, S)
        assert ref.check_schedule(w, S, R) == ref.OK
        for t, i in zip(*np.nonzero(R)):
            R2 = R.copy()
            R2[t, i] = 0
            assert ref.check_schedule(w, S, R2) == ref.E_INVALID_ARG, (t, i)
        ts, is_ = np.nonzero(S)
        if ts.size:
            R3 = R.copy()
            R3[ts[0], is_[0]] = 1
            assert ref.check_schedule(w, S, R3) == ref.E_INVALID_ARG
    with pytest.raises(ValueError):
        ref.plan(w, S, np.zeros_like(R))

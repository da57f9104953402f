"""Seeded synthetic inputs: training data-flow graphs and fractional checkpoint matrices.

This module only builds inputs. It performs none of the method's arithmetic
(no rounding, no recomputation solve, no memory simulation); the GPU library
and the CPU oracle both consume what it produces.

A graph follows the problem statement of Section 4.1: nodes numbered in a
topological order (a node depends only on lower-numbered nodes), each with an
output size M_v and a compute cost C_v, both int64. A fractional checkpoint
matrix S* stands in for the LP relaxation of Section 5.1: an n x n float64
matrix whose strict lower triangle holds values in [0, 1] and whose diagonal
and upper triangle are zero (frontier-advancing stages, Section 4.6).

Training graphs are built from a forward graph by a mirror rule: the gradient
node g_v of forward node f_v depends on f_v and on the gradient nodes of every
forward user of v; a loss node depends on every forward sink and is its own
mirror. Nodes are numbered forward nodes first, then the loss, then gradient
nodes in reverse forward order, so g_v = 2F - v for F forward nodes.

The five standard workloads (`config(1)` .. `config(5)`) are a linear chain,
a ResNet-like residual graph, a U-Net-like encoder/decoder, a transformer
stack and a deep random DAG. Each uses numpy's default_rng: S* from `seed`,
graph sizes, costs and edges from `seed + 100`.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

MIB = 1 << 20
KIB = 1 << 10


@dataclasses.dataclass
class Workload:
    """One evaluation problem: graph + fractional S* + candidate count + budget."""

    name: str
    n: int
    dep_ptr: np.ndarray   # int32 [n+1], CSR row pointers of Deps
    dep_idx: np.ndarray   # int32 [E], sorted ascending within each row
    cost: np.ndarray      # int64 [n]
    size: np.ndarray      # int64 [n]  (M_v, bytes)
    m_input: int
    m_param: int
    s_frac: np.ndarray    # float64 [n, n]
    K: int
    seed: int
    budget: int
    budget_pct: Optional[float] = None

    @property
    def num_edges(self) -> int:
        return int(self.dep_idx.shape[0])

    def deps(self, j: int) -> np.ndarray:
        return self.dep_idx[self.dep_ptr[j]:self.dep_ptr[j + 1]]

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# ---------------------------------------------------------------------------
# graph construction helpers
# ---------------------------------------------------------------------------

def csr_from_deps(deps: Sequence[Sequence[int]]) -> tuple[np.ndarray, np.ndarray]:
    ptr = np.zeros(len(deps) + 1, dtype=np.int32)
    flat: List[int] = []
    for j, d in enumerate(deps):
        ds = sorted(set(int(x) for x in d))
        flat.extend(ds)
        ptr[j + 1] = len(flat)
    return ptr, np.asarray(flat, dtype=np.int32)


def mirror_training_graph(fwd_deps: Sequence[Sequence[int]],
                          fwd_size: Sequence[int], fwd_cost: Sequence[int],
                          loss_size: int, loss_cost: int,
                          bwd_cost: Optional[Sequence[int]] = None):
    """Forward graph -> forward + loss + backward graph (mirror rule above).

    Returns (deps list, size int64[n], cost int64[n]) with n = 2F + 1.
    Gradient node sizes equal their forward node's size; gradient costs are
    `bwd_cost` if given, else twice the forward cost.
    """
    F = len(fwd_deps)
    users_fwd: List[List[int]] = [[] for _ in range(F)]
    for j, d in enumerate(fwd_deps):
        for i in d:
            if not (0 <= i < j):
                raise ValueError("forward edge %d->%d not topological" % (i, j))
            users_fwd[i].append(j)
    loss = F
    sinks = [v for v in range(F) if not users_fwd[v]]
    n = 2 * F + 1
    deps: List[List[int]] = [list(d) for d in fwd_deps] + [sinks] + [[] for _ in range(F)]

    def mirror(u: int) -> int:
        return loss if u == loss else 2 * F - u

    for v in range(F):
        g = 2 * F - v
        us = list(users_fwd[v]) + ([loss] if v in sinks else [])
        deps[g] = [v] + [mirror(u) for u in us]
    size = np.zeros(n, dtype=np.int64)
    cost = np.zeros(n, dtype=np.int64)
    size[:F] = np.asarray(fwd_size, dtype=np.int64)
    cost[:F] = np.asarray(fwd_cost, dtype=np.int64)
    size[loss] = int(loss_size)
    cost[loss] = int(loss_cost)
    bc = np.asarray(bwd_cost if bwd_cost is not None else 2 * np.asarray(fwd_cost, dtype=np.int64),
                    dtype=np.int64)
    for v in range(F):
        size[2 * F - v] = size[v]
        cost[2 * F - v] = bc[v]
    return deps, size, cost, sinks


def _lognormal_int(rng: np.random.Generator, mu: float, sigma: float, count: int) -> np.ndarray:
    x = rng.lognormal(mean=mu, sigma=sigma, size=count)
    return np.maximum(1, np.rint(x)).astype(np.int64)


def lower_triangle(n: int, values: np.ndarray) -> np.ndarray:
    """Place `values` (length n(n-1)/2) into the strict lower triangle, row-major."""
    s = np.zeros((n, n), dtype=np.float64)
    r, c = np.tril_indices(n, -1)
    s[r, c] = values
    return s


def s_frac_uniform(n: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return lower_triangle(n, rng.random(n * (n - 1) // 2))


def s_frac_beta(n: int, a: float, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return lower_triangle(n, rng.beta(a, a, size=n * (n - 1) // 2))


def checkpoint_all_budget(size: np.ndarray, m_input: int, m_param: int, pct: float) -> int:
    """The workloads' budget rule: pct percent of (M_in + 2 M_param + sum M), floored.

    Every workload states its budget as a percentage of the memory needed
    when every value is kept (constant overhead plus all outputs).
    """
    total = int(m_input) + 2 * int(m_param) + int(np.sum(size, dtype=np.int64))
    return (total * int(round(pct * 1000))) // 100000


def _assemble(name, deps, size, cost, s_frac, K, seed, pct, m_input=MIB, m_param=MIB) -> Workload:
    ptr, idx = csr_from_deps(deps)
    n = len(deps)
    return Workload(name=name, n=n, dep_ptr=ptr, dep_idx=idx, cost=np.asarray(cost, np.int64),
                    size=np.asarray(size, np.int64), m_input=int(m_input), m_param=int(m_param),
                    s_frac=s_frac, K=int(K), seed=int(seed),
                    budget=checkpoint_all_budget(np.asarray(size, np.int64), m_input, m_param, pct),
                    budget_pct=pct)


# ---------------------------------------------------------------------------
# the five standard workloads
# ---------------------------------------------------------------------------

def linear_chain(seed: int = 0, K: int = 64, pct: float = 50.0, layers: int = 8) -> Workload:
    """8 forward ops, 1 loss, 8 backward ops (n = 17); C = 100, M = 4 MiB everywhere."""
    fwd = [[]] + [[v - 1] for v in range(1, layers)]
    deps, size, cost, _ = mirror_training_graph(
        fwd, [4 * MIB] * layers, [100] * layers, 4 * MIB, 100, bwd_cost=[100] * layers)
    n = len(deps)
    return _assemble("linear_chain", deps, size, cost, s_frac_uniform(n, seed), K, seed, pct)


def resnet_like(seed: int = 1, K: int = 256, pct: float = 40.0, blocks: int = 32) -> Workload:
    """32 blocks of 2 ops; chain edges plus a skip (2b-1) -> (2b+1); mirrored (n = 129)."""
    F = 2 * blocks
    fwd: List[List[int]] = [[]]
    for v in range(1, F):
        d = [v - 1]
        if v % 2 == 1 and v >= 3:
            d.append(v - 2)
        fwd.append(d)
    grng = np.random.default_rng(seed + 100)
    size = _lognormal_int(grng, math.log(8 * MIB), 0.7, F)
    cost = _lognormal_int(grng, math.log(1e4), 1.0, F)
    deps, sz, cs, sinks = mirror_training_graph(fwd, size, cost, 4, max(1, int(size[-1]) // 4))
    n = len(deps)
    return _assemble("resnet_like", deps, sz, cs, s_frac_beta(n, 0.5, seed), K, seed, pct)


def unet_like(seed: int = 2, K: int = 512, pct: float = 30.0, levels: int = 5,
              ops_per_level: int = 8) -> Workload:
    """5-level encoder/decoder, 8 conv+activation ops per level, long skips (n = 337).

    Order: enc0, down0, enc1, down1, ..., enc4, dec4, up3, dec3, ..., up0, dec0.
    Activations are 64 MiB / 2^level. The last node of encoder level l feeds
    the first node of decoder level l (for the deepest level that edge is the
    chain edge itself).
    """
    grng = np.random.default_rng(seed + 100)
    sizes: List[int] = []
    fwd: List[List[int]] = []
    enc_last = {}
    dec_first = {}

    def add(sz: int, extra: Sequence[int] = ()):
        v = len(fwd)
        d = ([v - 1] if v > 0 else []) + [x for x in extra if x != v - 1]
        fwd.append(d)
        sizes.append(sz)
        return v

    per_level = 2 * ops_per_level
    for lvl in range(levels):
        for _ in range(per_level):
            last = add((64 * MIB) >> lvl)
        enc_last[lvl] = last
        if lvl < levels - 1:
            add((64 * MIB) >> (lvl + 1))          # downsample
    for lvl in range(levels - 1, -1, -1):
        if lvl < levels - 1:
            add((64 * MIB) >> lvl)                # upsample
        first = add((64 * MIB) >> lvl, extra=[enc_last[lvl]])
        dec_first[lvl] = first
        for _ in range(per_level - 1):
            add((64 * MIB) >> lvl)
    F = len(fwd)
    size = np.asarray(sizes, dtype=np.int64)
    noise = grng.uniform(0.5, 2.0, size=F)
    cost = np.maximum(1, np.rint(size / 1024.0 * noise)).astype(np.int64)
    deps, sz, cs, _ = mirror_training_graph(fwd, size, cost, 4, max(1, int(size[-1]) // 4))
    n = len(deps)
    return _assemble("unet_like", deps, sz, cs, s_frac_beta(n, 0.5, seed), K, seed, pct)


# per-block forward ops of the transformer workload: (name, deps by name, size, flops)
def _transformer_block_ops(s: int, h: int, heads: int, ffn: int, elt: int):
    sh = s * h * elt
    sc = heads * s * s * elt
    mm = 2 * s * h * h
    att = 2 * s * s * h
    stats = 2 * s * 4
    return [
        ("ln1_stats", ["x"], stats, 4 * s * h),
        ("ln1_norm", ["x", "ln1_stats"], sh, 4 * s * h),
        ("q", ["ln1_norm"], sh, mm),
        ("k", ["ln1_norm"], sh, mm),
        ("v", ["ln1_norm"], sh, mm),
        ("scores", ["q", "k"], sc, att),
        ("scale", ["scores"], sc, heads * s * s),
        ("mask", ["scale"], sc, heads * s * s),
        ("softmax", ["mask"], sc, 5 * heads * s * s),
        ("attn_dropout", ["softmax"], sc, 2 * heads * s * s),
        ("context", ["attn_dropout", "v"], sh, att),
        ("head_merge", ["context"], sh, s * h),
        ("out_proj", ["head_merge"], sh, mm),
        ("out_dropout", ["out_proj"], sh, 2 * s * h),
        ("res1", ["out_dropout", "x"], sh, s * h),
        ("ln2_stats", ["res1"], stats, 4 * s * h),
        ("ln2_norm", ["res1", "ln2_stats"], sh, 4 * s * h),
        ("mlp_up", ["ln2_norm"], s * ffn * elt, 2 * s * h * ffn),
        ("gelu", ["mlp_up"], s * ffn * elt, 8 * s * ffn),
        ("mlp_down", ["gelu"], sh, 2 * s * h * ffn),
        ("res2", ["mlp_down", "res1"], sh, s * h),
    ]


def transformer_stack(seed: int = 3, K: int = 1024, pct: float = 25.0, blocks: int = 24,
                      seq: int = 2048, hidden: int = 2048, heads: int = 16) -> Workload:
    """24 blocks x 21 forward nodes, fp16 tensors, FLOP costs, mirrored (n = 1009).

    Sizes: [seq, hidden] fp16 = 8 MiB; score-shaped tensors heads*seq^2 fp16 =
    128 MiB; MLP hidden 4*hidden; layer-norm statistics 2 fp32 per token.
    Costs are forward FLOPs (matmul 2mkn, elementwise a few per element);
    backward costs are twice the forward ones. The block input of block 0 is
    the network input (held in M_in), so it adds no edge.
    """
    ops = _transformer_block_ops(seq, hidden, heads, 4 * hidden, 2)
    fwd: List[List[int]] = []
    size: List[int] = []
    cost: List[int] = []
    x = None
    for _ in range(blocks):
        ids = {"x": x}
        for name, dnames, sz, fl in ops:
            d = [ids[dn] for dn in dnames if ids[dn] is not None]
            ids[name] = len(fwd)
            fwd.append(d)
            size.append(sz)
            cost.append(fl)
        x = ids["res2"]
    deps, sz, cs, _ = mirror_training_graph(fwd, size, cost, 4, max(1, size[-1] // 2))
    n = len(deps)
    return _assemble("transformer_stack", deps, sz, cs, s_frac_beta(n, 0.3, seed), K, seed, pct)


def random_dag_stress(seed: int = 4, K: int = 4096, pct: float = 20.0, F: int = 2000,
                      window: int = 16) -> Workload:
    """2000 forward nodes with 1-3 predecessors in a window of 16; mirrored (n = 4001)."""
    grng = np.random.default_rng(seed + 100)
    fwd: List[List[int]] = [[]]
    for j in range(1, F):
        d = min(int(grng.integers(1, 4)), j)
        lo = max(0, j - window)
        preds = grng.choice(np.arange(lo, j), size=d, replace=False)
        fwd.append(sorted(int(p) for p in preds))
    size = _lognormal_int(grng, math.log(16 * MIB), 1.0, F)
    cost = _lognormal_int(grng, math.log(5e3), 1.2, F)
    sinks = [v for v in range(F) if all(v not in d for d in fwd[v + 1:v + window + 1])]
    loss_cost = max(1, int(sum(int(size[v]) for v in sinks)) // 4)
    deps, sz, cs, _ = mirror_training_graph(fwd, size, cost, 4, loss_cost)
    n = len(deps)
    return _assemble("random_dag_stress", deps, sz, cs, s_frac_uniform(n, seed), K, seed, pct)


CONFIG_BUILDERS = {1: linear_chain, 2: resnet_like, 3: unet_like, 4: transformer_stack,
                   5: random_dag_stress}


def config(i: int, **kw) -> Workload:
    """Standard workload i in 1..5 (linear chain .. random DAG)."""
    return CONFIG_BUILDERS[i](**kw)


# ---------------------------------------------------------------------------
# small random problems for tests
# ---------------------------------------------------------------------------

def random_dag(n: int, seed: int, max_deg: int = 3, window: int = 8, max_size: int = 9,
               max_cost: int = 9, s_kind: str = "uniform", K: int = 8,
               budget_pct: float = 60.0, m_input: int = 1, m_param: int = 1) -> Workload:
    """An arbitrary topologically numbered DAG with small integer sizes and costs."""
    rng = np.random.default_rng(seed)
    deps: List[List[int]] = [[]]
    for j in range(1, n):
        lo = max(0, j - window)
        d = int(rng.integers(0, max_deg + 1))
        d = min(d, j - lo)
        preds = rng.choice(np.arange(lo, j), size=d, replace=False) if d else []
        deps.append(sorted(int(p) for p in preds))
    size = rng.integers(1, max_size + 1, size=n).astype(np.int64)
    cost = rng.integers(1, max_cost + 1, size=n).astype(np.int64)
    cnt = n * (n - 1) // 2
    if s_kind == "uniform":
        vals = rng.random(cnt)
    elif s_kind == "beta":
        vals = rng.beta(0.3, 0.3, size=cnt)
    elif s_kind == "binary":
        vals = (rng.random(cnt) < 0.5).astype(np.float64)
    elif s_kind == "sparse":
        vals = 0.2 * rng.random(cnt)
    else:
        raise ValueError(s_kind)
    ptr, idx = csr_from_deps(deps)
    return Workload(name="random_dag_%d_%d" % (n, seed), n=n, dep_ptr=ptr, dep_idx=idx, cost=cost,
                    size=size, m_input=m_input, m_param=m_param, s_frac=lower_triangle(n, vals),
                    K=K, seed=seed,
                    budget=checkpoint_all_budget(size, m_input, m_param, budget_pct),
                    budget_pct=budget_pct)


# ---------------------------------------------------------------------------
# supplied checkpoint matrices (integral S) for batch evaluation
# ---------------------------------------------------------------------------

def random_schedules(n: int, K: int, seed: int, density: float = 0.3, kind: str = "bernoulli",
                     junk: bool = True) -> np.ndarray:
    """K checkpoint matrices as bit rows [K][n][ceil(n/64)] uint64 (bit i % 64
    of word i / 64 of row t is S[t][i]).

    kind "bernoulli": each strict-lower entry is 1 with probability density.
    kind "intervals": each value i is kept with probability density, from
    stage i + 1 up to a uniformly drawn last stage (the banded shape of
    checkpoint schedules, where a stored value stays resident for a while).
    junk: also set random bits on and above the diagonal and in the padding
    past node n - 1; the evaluation must ignore them."""
    rng = np.random.default_rng(seed)
    W = (n + 63) // 64
    out = np.zeros((K, n, W), np.uint64)
    tri = np.tri(n, W * 64, -1, dtype=bool)
    for k in range(K):
        if kind == "bernoulli":
            bits = rng.random((n, W * 64)) < density
        elif kind == "intervals":
            keep = rng.random(n) < density
            first = np.arange(1, n + 1)
            end = first + np.floor(rng.random(n) * (n + 1 - first)).astype(np.int64)
            t = np.arange(n)[:, None]
            i = np.arange(W * 64)[None, :]
            i_c = np.minimum(i, n - 1)
            bits = (i < n) & keep[i_c] & (t > i) & (t < end[i_c])
        else:
            raise ValueError(kind)
        bits = bits & tri
        if junk:
            bits = bits | ((rng.random((n, W * 64)) < 0.5) & ~tri)
        packed = np.packbits(bits.astype(np.uint8).reshape(n, W, 64), axis=2, bitorder="little")
        out[k] = packed.view(np.uint64).reshape(n, W)
    return out


def unpack_schedules(rows: np.ndarray, n: int) -> np.ndarray:
    """[K][n][W] uint64 bit rows -> [K][n][n] uint8 0/1 (the inverse layout)."""
    rows = np.ascontiguousarray(rows, np.uint64)
    K = rows.shape[0]
    bits = np.unpackbits(rows.view(np.uint8).reshape(K, n, -1), axis=2, bitorder="little")
    return bits[:, :, :n].copy()

"""Seeded synthetic workloads: graphs, features, weights and update streams.

This module only draws random inputs. It holds none of the incremental method's
arithmetic, and it is the one piece of Python that both the CPU oracle (under
``oracle/``) and the HIP path (through the C ABI) consume.

The graphs stand in for the datasets of the paper's evaluation (Sec. VII-A.2,
Table "Graph datasets used in experiments"), which are not available here:

* ``tiny``            directed Erdos-Renyi G(n, m), n=2000, m=16000.
* ``sparse_mid``      directed Chung-Lu power law (exponent 2.1) shaped like
                      ogbn-arxiv: 169,343 vertices, 1,166,243 arcs, 128 features.
* ``sparse_mid_mean`` the same graph with a 3-layer GraphSAGE-mean model.
* ``sparse_mid_gc_sum``, ``sparse_mid_gc_mean``, ``sparse_mid_gin``,
  ``sparse_mid_gc_wsum``  the same graph with the evaluation's GraphConv-sum,
                      GraphConv-mean, GIN-sum and GraphConv-weighted-sum workloads
                      (2 layers, 128-256-40; the last on arcs weighted uniformly in
                      [0.5, 1.5), inserts carrying their weights).
* ``dense_large``     undirected Chung-Lu (exponent 2.1) shaped like
                      ogbn-products: 2,449,029 vertices, 61,859,140 edges, 100 features.
* ``dense_large_2l``  the same graph with a 2-layer model (the paper's 2-layer
                      Products numbers are quoted on 2-layer workloads).
* ``stress``          RMAT(0.57, 0.19, 0.19, 0.05), 2^23 vertices, 200M arcs, GCN.

Update streams follow the paper's recipe (Sec. VII-A.2): inserts are edges held
out of the generated graph, deletes are random snapshot edges, feature updates
replace a random vertex's row with fresh N(0,1) values.

Op records are int32 rows ``(kind, u, v, feat_row)`` with kind 1 = edge insert,
2 = edge delete, 3 = feature replacement (``feat_row`` indexes the batch's
feature-row block; ``v`` is -1 for feature ops and ``feat_row`` -1 for edge ops).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Tuple

import numpy as np

OP_INSERT = 1
OP_DELETE = 2
OP_FEATURE = 3

AGG_SUM = "sum"
AGG_MEAN = "mean"
AGG_GCN = "gcn"
AGG_GC_SUM = "gc_sum"    # GraphConv, sum aggregator (no self term)
AGG_GC_MEAN = "gc_mean"  # GraphConv, mean aggregator (no self term)
AGG_GIN = "gin"          # GINConv, sum aggregator, two-layer MLP
AGG_GC_WSUM = "gc_wsum"  # GraphConv, sum weighted by stored arc weights (no self term)


@dataclasses.dataclass(frozen=True)
class GraphSpec:
    kind: str                 # "er" | "chung_lu" | "rmat"
    n: int
    m: int                    # edges in the snapshot (undirected: unordered pairs)
    undirected: bool = False
    gamma: float = 2.1        # power-law exponent (chung_lu)
    rmat: Tuple[float, float, float, float] = (0.57, 0.19, 0.19, 0.05)
    holdout: float = 0.10     # extra edges drawn and held out as the insert pool
    weighted: bool = False    # arcs carry weights, uniform in [0.5, 1.5) (inserts too)


@dataclasses.dataclass(frozen=True)
class ModelSpec:
    agg: str                  # "sum" | "mean" | "gcn" | "gc_sum" | "gc_mean" | "gin"
    dims: Tuple[int, ...]     # d_0 .. d_L
    gin_eps: float = 0.0      # GIN: weight 1 + eps of the own embedding


@dataclasses.dataclass(frozen=True)
class StreamSpec:
    batch_sizes: Tuple[int, ...]
    # op mix: either exact per-batch counts ("exact") or per-op probabilities
    mix: Tuple[float, float, float]   # insert, delete, feature
    exact: bool = False
    hub_biased: bool = False


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    name: str
    graph: GraphSpec
    model: ModelSpec
    stream: StreamSpec
    seed: int = 0


CONFIGS: Dict[str, WorkloadSpec] = {
    "tiny": WorkloadSpec(
        "tiny",
        GraphSpec("er", 2000, 16000),
        ModelSpec(AGG_SUM, (16, 16, 8)),
        StreamSpec((100,), (45, 45, 10), exact=True)),
    "sparse_mid": WorkloadSpec(
        "sparse_mid",
        GraphSpec("chung_lu", 169_343, 1_166_243),
        ModelSpec(AGG_SUM, (128, 256, 40)),
        StreamSpec((1, 10, 100, 1000), (1 / 3, 1 / 3, 1 / 3))),
    "sparse_mid_mean": WorkloadSpec(
        "sparse_mid_mean",
        GraphSpec("chung_lu", 169_343, 1_166_243),
        ModelSpec(AGG_MEAN, (128, 256, 256, 40)),
        StreamSpec((100,), (1 / 3, 1 / 3, 1 / 3))),
    # the evaluation's other workloads (Sec. VII-A: GC-S, GC-M, GI-S) on the
    # Arxiv-shaped graph, 2 layers like sparse_mid (which is GS-S)
    "sparse_mid_gc_sum": WorkloadSpec(
        "sparse_mid_gc_sum",
        GraphSpec("chung_lu", 169_343, 1_166_243),
        ModelSpec(AGG_GC_SUM, (128, 256, 40)),
        StreamSpec((1, 10, 100, 1000), (1 / 3, 1 / 3, 1 / 3))),
    "sparse_mid_gc_mean": WorkloadSpec(
        "sparse_mid_gc_mean",
        GraphSpec("chung_lu", 169_343, 1_166_243),
        ModelSpec(AGG_GC_MEAN, (128, 256, 40)),
        StreamSpec((1, 10, 100, 1000), (1 / 3, 1 / 3, 1 / 3))),
    "sparse_mid_gc_wsum": WorkloadSpec(
        "sparse_mid_gc_wsum",
        GraphSpec("chung_lu", 169_343, 1_166_243, weighted=True),
        ModelSpec(AGG_GC_WSUM, (128, 256, 40)),
        StreamSpec((1, 10, 100, 1000), (1 / 3, 1 / 3, 1 / 3))),
    "sparse_mid_gin": WorkloadSpec(
        "sparse_mid_gin",
        GraphSpec("chung_lu", 169_343, 1_166_243),
        ModelSpec(AGG_GIN, (128, 256, 40), gin_eps=0.1),
        StreamSpec((1, 10, 100, 1000), (1 / 3, 1 / 3, 1 / 3))),
    "dense_large": WorkloadSpec(
        "dense_large",
        GraphSpec("chung_lu", 2_449_029, 61_859_140, undirected=True),
        ModelSpec(AGG_SUM, (100, 256, 256, 47)),
        StreamSpec((10, 100, 1000), (0.4, 0.4, 0.2))),
    "dense_large_2l": WorkloadSpec(
        "dense_large_2l",
        GraphSpec("chung_lu", 2_449_029, 61_859_140, undirected=True),
        ModelSpec(AGG_SUM, (100, 256, 47)),
        StreamSpec((10, 100, 1000), (0.4, 0.4, 0.2))),
    "stress": WorkloadSpec(
        "stress",
        GraphSpec("rmat", 1 << 23, 200_000_000),
        ModelSpec(AGG_GCN, (64, 256, 64)),
        StreamSpec((10_000,), (1 / 3, 1 / 3, 1 / 3), hub_biased=True)),
}


def seeds(seed: int) -> List[np.random.Generator]:
    """Four independent generators: graph, features, weights, stream."""
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(4)]


def edge_weights_rng(seed: int) -> np.random.Generator:
    """A fifth independent generator, for arc weights (the first four of the same
    spawn are those of seeds(), so unweighted workloads are unchanged)."""
    return np.random.default_rng(np.random.SeedSequence(seed).spawn(5)[4])


def arc_weights(rng: np.random.Generator, count: int) -> np.ndarray:
    return rng.uniform(0.5, 1.5, count).astype(np.float32)


def weight_bits(w) -> np.ndarray:
    """Float32 weights as the int32 bit patterns an insert op carries in its fourth field."""
    return np.ascontiguousarray(np.asarray(w, np.float32)).view(np.int32)


# ----------------------------------------------------------------------------
# graphs
# ----------------------------------------------------------------------------

def chung_lu_weights(n: int, total: float, gamma: float) -> np.ndarray:
    """Expected-degree weights w_i = c (i + i0)^(-1/(gamma-1)), sum = total, with
    i0 chosen so that the largest weight equals sqrt(total) (the admissibility cap
    of the Chung-Lu model)."""
    beta = 1.0 / (gamma - 1.0)
    idx = np.arange(n, dtype=np.float64)
    cap = np.sqrt(total)

    def w0(i0: float) -> float:
        base = (idx + i0) ** (-beta)
        return total * base[0] / base.sum()

    lo, hi = 1e-9, float(n)
    if w0(hi) > cap:          # cannot reach the cap: take the flattest admissible curve
        i0 = hi
    else:
        for _ in range(80):
            mid = np.sqrt(lo * hi)
            if w0(mid) > cap:
                lo = mid
            else:
                hi = mid
        i0 = hi
    base = (idx + i0) ** (-beta)
    return total * base / base.sum()


def _draw(rng: np.random.Generator, cdf: np.ndarray, count: int) -> np.ndarray:
    """`count` independent indices with P(i) proportional to cdf[i] - cdf[i-1]."""
    r = rng.random(count) * cdf[-1]
    return np.minimum(np.searchsorted(cdf, r, side="right"), len(cdf) - 1).astype(np.int64)


def _draw_many(rng: np.random.Generator, p: np.ndarray, count: int, shuffle: bool = True) -> np.ndarray:
    """`count` i.i.d. indices with probabilities p: multinomial counts per index,
    laid out in a uniformly random order (same law as independent draws, without
    a search per draw). With shuffle=False they come sorted; pairing a sorted
    sample with a shuffled independent one still gives i.i.d. pairs."""
    counts = rng.multinomial(count, p)
    idx = np.repeat(np.arange(p.size, dtype=np.int64), counts)
    if shuffle:
        rng.shuffle(idx)
    return idx


_THREADS = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))


def _unique_sorted_chunk(x: np.ndarray) -> np.ndarray:
    x = np.sort(x)
    if x.size == 0:
        return x
    keep = np.empty(x.size, bool)
    keep[0] = True
    np.not_equal(x[1:], x[:-1], out=keep[1:])
    return x[keep]


def _sorted_unique(x: np.ndarray) -> np.ndarray:
    """Sorted distinct values (introsort; NumPy's stable sort of int64 is a much
    slower merge sort)."""
    return _unique_sorted_chunk(x)


def _distinct(rng, n, target, sampler, undirected):
    """Draw arcs (or unordered pairs) until `target` distinct non-loop keys exist."""
    keys = np.empty(0, np.int64)
    first = True
    while keys.size < target:
        need = target - keys.size
        u, v = sampler(int(need * (1.15 if first else 1.5)) + 1024)
        ok = u != v
        u, v = u[ok], v[ok]
        if undirected:
            u, v = np.minimum(u, v), np.maximum(u, v)
        cand = _sorted_unique(u * n + v)
        if first:
            keys, first = cand, False
            continue
        pos = np.searchsorted(keys, cand)
        hit = (pos < keys.size) & (keys[np.minimum(pos, keys.size - 1)] == cand)
        new = cand[~hit]
        keys = np.insert(keys, np.searchsorted(keys, new), new)
    if keys.size > target:
        drop = np.zeros(keys.size, bool)
        drop[rng.choice(keys.size, keys.size - target, replace=False)] = True
        keys = keys[~drop]
    return keys


def generate_graph(spec: GraphSpec, rng: np.random.Generator):
    """Returns (snapshot_src, snapshot_dst, pool_src, pool_dst) as int32 arrays.

    Undirected graphs list each edge once with src < dst. The pool holds extra
    edges from the same distribution, absent from the snapshot, streamed later
    as inserts."""
    n = spec.n
    total = spec.m + int(np.ceil(spec.m * spec.holdout))
    if spec.kind == "er":
        def sampler(c):
            return rng.integers(0, n, c, dtype=np.int64), rng.integers(0, n, c, dtype=np.int64)
    elif spec.kind == "chung_lu":
        if spec.undirected:
            w = chung_lu_weights(n, 2.0 * total, spec.gamma)
            p = w[np.argsort(rng.permutation(n))]
            p = p / p.sum()

            def sampler(c):
                return _draw_many(rng, p, c, shuffle=False), _draw_many(rng, p, c)
        else:
            w = chung_lu_weights(n, float(total), spec.gamma)
            p_out = w[np.argsort(rng.permutation(n))]
            p_in = w[np.argsort(rng.permutation(n))]
            p_out, p_in = p_out / p_out.sum(), p_in / p_in.sum()

            def sampler(c):
                return _draw_many(rng, p_out, c, shuffle=False), _draw_many(rng, p_in, c)
    elif spec.kind == "rmat":
        scale = int(np.log2(n))
        assert (1 << scale) == n
        a, b, c_, _d = spec.rmat
        relabel = rng.permutation(n).astype(np.int64)

        t1, t2, t3 = np.float32(a), np.float32(a + b), np.float32(a + b + c_)

        def rmat_chunk(seed, k):
            # quadrant per level from one uniform: a -> (0,0), b -> (0,1), c -> (1,0), d -> (1,1)
            g = np.random.default_rng(seed)
            u = np.zeros(k, np.int32)
            v = np.zeros(k, np.int32)
            r = np.empty(k, np.float32)
            hi_half = np.empty(k, np.bool_)
            vbit = np.empty(k, np.bool_)
            dq = np.empty(k, np.bool_)
            for _ in range(scale):
                g.random(out=r, dtype=np.float32)
                np.greater_equal(r, t2, out=hi_half)          # c or d: source bit set
                np.left_shift(u, 1, out=u)
                np.bitwise_or(u, hi_half, out=u)
                np.greater_equal(r, t1, out=vbit)
                np.logical_xor(vbit, hi_half, out=vbit)       # b
                np.greater_equal(r, t3, out=dq)               # d
                np.logical_or(vbit, dq, out=vbit)             # b or d: sink bit set
                np.left_shift(v, 1, out=v)
                np.bitwise_or(v, vbit, out=v)
            return relabel[u], relabel[v]

        def sampler(c):
            # fixed-size chunks, each with its own generator seeded from rng, so the
            # result does not depend on the thread count or scheduling
            sizes = [min(1 << 22, c - lo) for lo in range(0, c, 1 << 22)]
            chunk_seeds = rng.integers(0, 2**63 - 1, size=len(sizes))
            with ThreadPoolExecutor(_THREADS) as ex:
                parts = list(ex.map(rmat_chunk, chunk_seeds, sizes))
            return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])
    else:
        raise ValueError(spec.kind)
    keys = _distinct(rng, n, total, sampler, spec.undirected)
    in_pool = np.zeros(keys.size, bool)
    in_pool[rng.choice(keys.size, keys.size - spec.m, replace=False)] = True
    snap, pool = keys[~in_pool], keys[in_pool]
    rng.shuffle(pool)
    return ((snap // n).astype(np.int32), (snap % n).astype(np.int32),
            (pool // n).astype(np.int32), (pool % n).astype(np.int32))


def erdos_renyi(n: int, m: int, rng: np.random.Generator, undirected: bool = False):
    """Small helper for tests: m distinct non-loop arcs (or edges) on n vertices."""
    keys = _distinct(rng, n, m, lambda c: (rng.integers(0, n, c), rng.integers(0, n, c)),
                     undirected)
    return (keys // n).astype(np.int32), (keys % n).astype(np.int32)


# ----------------------------------------------------------------------------
# features and weights
# ----------------------------------------------------------------------------

def features(n: int, d: int, rng: np.random.Generator) -> np.ndarray:
    return rng.standard_normal((n, d), dtype=np.float32)


@dataclasses.dataclass
class ModelWeights:
    agg: str
    dims: Tuple[int, ...]
    w_self: List[Optional[np.ndarray]]   # [d_l, d_{l-1}] float32, None for GCN / GraphConv / GIN
    w_neigh: List[np.ndarray]            # [d_l, d_{l-1}] float32 (GCN, GraphConv: the single W;
                                         # GIN: the MLP's first layer, [d_l, d_{l-1}])
    bias: List[np.ndarray]               # [d_l] float32 (GIN: the MLP's first bias)
    relu: List[bool]                     # activation after each layer
    w_out: List[np.ndarray] = dataclasses.field(default_factory=list)  # GIN: MLP second layer [d_l, d_l]
    b_out: List[np.ndarray] = dataclasses.field(default_factory=list)  # GIN: its bias [d_l]
    gin_eps: float = 0.0

    @property
    def num_layers(self) -> int:
        return len(self.dims) - 1


def glorot(rng: np.random.Generator, fan_out: int, fan_in: int) -> np.ndarray:
    lim = np.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-lim, lim, (fan_out, fan_in)).astype(np.float32)


def model_weights(spec: ModelSpec, rng: np.random.Generator, bias_std: float = 0.0,
                  last_relu: bool = False) -> ModelWeights:
    """Glorot-uniform weights (gain 1), drawn separately for the self and neighbour
    matrices; ReLU after every layer but the last; bias zero unless bias_std > 0."""
    L = len(spec.dims) - 1
    ws, wn, bs, act, wo, bo = [], [], [], [], [], []

    def bias(d):
        if bias_std > 0:
            return (rng.standard_normal(d) * bias_std).astype(np.float32)
        return np.zeros(d, np.float32)

    for l in range(1, L + 1):
        din, dout = spec.dims[l - 1], spec.dims[l]
        if spec.agg in (AGG_GCN, AGG_GC_SUM, AGG_GC_MEAN, AGG_GC_WSUM, AGG_GIN):
            ws.append(None)
        else:
            ws.append(glorot(rng, dout, din))
        wn.append(glorot(rng, dout, din))
        bs.append(bias(dout))
        if spec.agg == AGG_GIN:  # the MLP's second layer (hidden width d_l)
            wo.append(glorot(rng, dout, dout))
            bo.append(bias(dout))
        act.append(l < L or last_relu)
    return ModelWeights(spec.agg, tuple(spec.dims), ws, wn, bs, act, wo, bo, spec.gin_eps)


# ----------------------------------------------------------------------------
# update streams
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Batch:
    ops: np.ndarray          # [B, 4] int32 (kind, u, v, feat_row)
    feat_rows: np.ndarray    # [k, d0] float32

    @property
    def size(self) -> int:
        return int(self.ops.shape[0])


class UpdateStream:
    """Conflict-free benchmark stream (Sec. VII-A.2 recipe): inserts come from the
    held-out pool, deletes from a random permutation of snapshot edges, feature
    updates pick uniform vertices with fresh N(0,1) rows. Every op is effective."""

    def __init__(self, n: int, d0: int, snap_src, snap_dst, pool_src, pool_dst,
                 spec: StreamSpec, rng: np.random.Generator, out_deg=None, in_deg=None, pool_w=None):
        self.n, self.d0, self.spec, self.rng = n, d0, spec, rng
        self.pool_w = pool_w  # weighted graphs: each pool edge's weight
        self.snap_src, self.snap_dst = snap_src, snap_dst
        self.pool_src, self.pool_dst = pool_src, pool_dst
        self._del_order = rng.permutation(snap_src.size)
        self._del_next = 0
        self._ins_next = 0
        if spec.hub_biased:
            assert out_deg is not None and in_deg is not None
            self._cdf_out = np.cumsum(out_deg.astype(np.float64) + 1.0)
            self._cdf_in = np.cumsum(in_deg.astype(np.float64) + 1.0)
            keys = snap_src.astype(np.int64) * n + snap_dst
            if keys.size > 1 and not np.all(keys[1:] > keys[:-1]):
                keys = np.sort(keys)     # generate_graph already returns the snapshot sorted
            self._keys = keys
            self._inserted = set()

    def _kinds(self, bs: int) -> np.ndarray:
        if self.spec.exact:
            cnt = np.array(self.spec.mix, np.int64)
            assert cnt.sum() == bs, "exact op mix must add up to the batch size"
            kinds = np.repeat(np.array([OP_INSERT, OP_DELETE, OP_FEATURE]), cnt)
            return kinds[self.rng.permutation(bs)]
        p = np.array(self.spec.mix, np.float64)
        return self.rng.choice(np.array([OP_INSERT, OP_DELETE, OP_FEATURE]), bs, p=p / p.sum())

    def _hub_insert(self) -> Tuple[int, int]:
        while True:
            u = int(_draw(self.rng, self._cdf_out, 1)[0])
            v = int(_draw(self.rng, self._cdf_in, 1)[0])
            if u == v:
                continue
            key = u * self.n + v
            j = np.searchsorted(self._keys, key)
            if (j < self._keys.size and self._keys[j] == key) or key in self._inserted:
                continue
            self._inserted.add(key)
            return u, v

    def next_batch(self, bs: int) -> Batch:
        kinds = self._kinds(bs)
        ops = np.full((bs, 4), -1, np.int32)
        ops[:, 0] = kinds
        nfeat = int((kinds == OP_FEATURE).sum())
        feat_rows = self.rng.standard_normal((nfeat, self.d0), dtype=np.float32)
        f = 0
        for i, k in enumerate(kinds):
            if k == OP_INSERT:
                if self.spec.hub_biased:
                    ops[i, 1], ops[i, 2] = self._hub_insert()
                else:
                    if self._ins_next >= self.pool_src.size:
                        raise RuntimeError("insert pool exhausted")
                    j = self._ins_next
                    self._ins_next += 1
                    ops[i, 1], ops[i, 2] = self.pool_src[j], self.pool_dst[j]
                    if self.pool_w is not None:
                        ops[i, 3] = weight_bits(self.pool_w[j : j + 1])[0]
            elif k == OP_DELETE:
                if self._del_next >= self._del_order.size:
                    raise RuntimeError("delete pool exhausted")
                j = self._del_order[self._del_next]
                self._del_next += 1
                ops[i, 1], ops[i, 2] = self.snap_src[j], self.snap_dst[j]
            else:
                if self.spec.hub_biased:
                    ops[i, 1] = int(_draw(self.rng, self._cdf_out, 1)[0])
                else:
                    ops[i, 1] = self.rng.integers(0, self.n)
                ops[i, 3] = f
                f += 1
        return Batch(ops, feat_rows)


def adversarial_batch(rng: np.random.Generator, n: int, d0: int, bs: int,
                      hot: int = 12, existing: Optional[Tuple[np.ndarray, np.ndarray]] = None,
                      p_selfloop: float = 0.05, weighted: bool = False) -> Batch:
    """A batch designed to collide: ops mostly touch a small hot vertex set, so it
    holds repeated inserts/deletes of one edge, insert-then-delete, deletes of
    absent edges, self-loops and repeated feature writes. Sequential semantics
    decide the outcome. weighted: inserts carry weights from a few values, so
    inserts of present arcs sometimes keep and sometimes change their weight."""
    hot_set = rng.choice(n, size=min(hot, n), replace=False)
    ops = np.full((bs, 4), -1, np.int32)
    nfeat = 0
    for i in range(bs):
        r = rng.random()
        if r < 0.4:
            kind = OP_INSERT
        elif r < 0.8:
            kind = OP_DELETE
        else:
            kind = OP_FEATURE
        ops[i, 0] = kind
        if kind == OP_FEATURE:
            ops[i, 1] = rng.choice(hot_set) if rng.random() < 0.7 else rng.integers(0, n)
            ops[i, 3] = nfeat
            nfeat += 1
            continue
        if kind == OP_DELETE and existing is not None and existing[0].size and rng.random() < 0.5:
            j = rng.integers(0, existing[0].size)
            u, v = int(existing[0][j]), int(existing[1][j])
        elif rng.random() < p_selfloop:
            u = v = int(rng.choice(hot_set))
        else:
            u, v = int(rng.choice(hot_set)), int(rng.choice(hot_set))
            if rng.random() < 0.3:
                v = int(rng.integers(0, n))
        if kind == OP_INSERT and existing is not None and existing[0].size and rng.random() < 0.25:
            j = rng.integers(0, existing[0].size)  # an arc that may be present: a weight update
            u, v = int(existing[0][j]), int(existing[1][j])
        ops[i, 1], ops[i, 2] = u, v
        if weighted and kind == OP_INSERT:
            ops[i, 3] = weight_bits([rng.choice([0.5, 1.0, 1.25])])[0]
    feat_rows = rng.standard_normal((nfeat, d0), dtype=np.float32)
    return Batch(ops, feat_rows)


# ----------------------------------------------------------------------------
# one-call workload construction
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    src: np.ndarray
    dst: np.ndarray
    pool_src: np.ndarray
    pool_dst: np.ndarray
    x: np.ndarray
    weights: ModelWeights
    stream: UpdateStream
    edge_w: Optional[np.ndarray] = None   # weighted graphs: float32 weight per snapshot edge

    @property
    def n(self) -> int:
        return self.spec.graph.n


def build_workload(name_or_spec, seed: Optional[int] = None, bias_std: float = 0.0,
                   graph_override: Optional[GraphSpec] = None) -> Workload:
    spec = CONFIGS[name_or_spec] if isinstance(name_or_spec, str) else name_or_spec
    if seed is not None:
        spec = dataclasses.replace(spec, seed=seed)
    if graph_override is not None:
        spec = dataclasses.replace(spec, graph=graph_override)
    g_rng, f_rng, w_rng, s_rng = seeds(spec.seed)
    src, dst, psrc, pdst = generate_graph(spec.graph, g_rng)
    x = features(spec.graph.n, spec.model.dims[0], f_rng)
    w = model_weights(spec.model, w_rng, bias_std=bias_std)
    out_deg = in_deg = None
    if spec.stream.hub_biased:
        out_deg = np.bincount(src, minlength=spec.graph.n)
        in_deg = np.bincount(dst, minlength=spec.graph.n)
        if spec.graph.undirected:
            out_deg = in_deg = out_deg + in_deg
    edge_w = pool_w = None
    if spec.graph.weighted:
        e_rng = edge_weights_rng(spec.seed)
        edge_w = arc_weights(e_rng, src.size)
        pool_w = arc_weights(e_rng, psrc.size)
    stream = UpdateStream(spec.graph.n, spec.model.dims[0], src, dst, psrc, pdst,
                          spec.stream, s_rng, out_deg, in_deg, pool_w)
    return Workload(spec, src, dst, psrc, pdst, x, w, stream, edge_w)

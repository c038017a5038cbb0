"""CPU oracle for exact incremental GNN embedding propagation (Ripple, arXiv 2505.12112).

TEST INFRASTRUCTURE. Only the test-suite, the package smoke check and the
benchmark's CPU-baseline timing may import this module. The HIP library never
calls it, and it shares no code with the library: it does not know about
cached aggregates, deltas, frontiers or bitmaps. It recomputes every layer of
the GNN from scratch on the post-batch graph and derives the affected vertex
sets from the graph structure alone.

Passages followed:

* GNN layer: Sec. II-A, Eq. (1)-(2): x^l_u = Aggregate^l({h^{l-1}_v : v in N(u)}),
  h^l_u = sigma(Update^l(h^{l-1}_u, x^l_u)).
* Linear aggregators sum, mean and weighted sum: Sec. II-C, table "Popular Linear
  Aggregation functions in GNNs".
* N(u) is the set of in-neighbours; updates flow from source to sink along
  out-edges: Sec. IV-B (inserting C->A first changes h^1 of the sink A, whose
  recompute pulls the h^0 of all of A's in-neighbours).
* Update types (edge insert, edge delete, vertex-feature change; no vertex
  insert/delete) and fixed-size batches: Sec. IV-A.
* Affected vertices: an edge update touches the sink at every hop, and a vertex
  touched at hop l touches its out-neighbours at hop l+1; a feature update of u
  touches u's out-neighbours at hop 1: Sec. II-B and Sec. IV-B. No pruning:
  every reached vertex counts as affected: Sec. IV-C.
* Combined updates give the same result as applying them one by one: Sec.
  IV-C.1 ("Combining multiple updates at a vertex").
* Exact within floating-point precision: Sec. VI.

Readings where the paper is silent (each is listed with its reason in the
design notes of the repository):

* simple directed graph: inserting a present arc, deleting an absent arc and
  inserting or deleting a self-loop change nothing;
* a batch has sequential semantics: the net effect is what applying its ops in
  order would leave (last feature write wins);
* on an undirected graph an edge op acts on both arcs;
* GraphSAGE: h = sigma(W_self h_self + W_neigh agg + b) with agg the sum, or the
  mean (0 when the in-degree is 0);
* GCN with symmetric normalisation: implicit self-loop,
  alpha_uv = 1/sqrt((d_out(u)+1)(d_in(v)+1));
* GraphConv with sum or mean (the evaluation's GC-S and GC-M workloads, Sec.
  VII-A): h = sigma(W agg + b), no self term and no self-loop, so a vertex whose
  own embedding changed is not affected at the next hop unless a neighbour is;
* GINConv with sum (GI-S): h = sigma(MLP((1 + eps) h_self + sum)), the MLP a
  linear layer, a ReLU and a second linear layer;
* GraphConv with weighted sum (GC-W): the arcs carry stored weights alpha_uv
  and agg = sum_u alpha_uv h_u (Sec. II-C table; Sec. IV-C.1: each message is
  scaled by the weight of its arc); an insert carries the new arc's weight and
  an insert of a present arc sets its weight;
* ReLU after every layer but the last.

Arithmetic is float64 by default; the aggregation uses a scipy sparse product
and the transform a dense matrix product.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import scipy.sparse as sp

OP_INSERT = 1
OP_DELETE = 2
OP_FEATURE = 3


# ----------------------------------------------------------------------------
# model
# ----------------------------------------------------------------------------

# GraphSAGE (self weight + neighbour weight): "sum", "mean"; GCN: "gcn";
# GraphConv (neighbour weight only, no self term): "gc_sum", "gc_mean", and
# "gc_wsum" (the sum weighted by the arcs' stored weights);
# GINConv: "gin" (sum, (1 + eps) self term, two-layer MLP).
AGGREGATORS = ("sum", "mean", "gcn", "gc_sum", "gc_mean", "gin", "gc_wsum")


def has_self_term(agg: str) -> bool:
    """Whether a vertex's own previous embedding enters its update."""
    return agg not in ("gc_sum", "gc_mean", "gc_wsum")


@dataclasses.dataclass
class OracleModel:
    """Weights are [out, in] (y = W x). SAGE: w_self, w_neigh [d_l, d_{l-1}];
    GCN / GraphConv: w_neigh only. GIN: w_neigh [hidden, d_{l-1}] and bias [hidden]
    are the MLP's first layer, w_out [d_l, hidden] and b_out [d_l] its second."""
    agg: str
    w_self: List[Optional[np.ndarray]]
    w_neigh: List[np.ndarray]
    bias: List[np.ndarray]
    relu: List[bool]
    w_out: List[np.ndarray] = dataclasses.field(default_factory=list)
    b_out: List[np.ndarray] = dataclasses.field(default_factory=list)
    gin_eps: float = 0.0

    @property
    def num_layers(self) -> int:
        return len(self.w_neigh)

    @staticmethod
    def from_weights(mw, dtype=np.float64) -> "OracleModel":
        """Accepts any object with agg / w_self / w_neigh / bias / relu attributes
        (and w_out / b_out / gin_eps for GIN)."""
        return OracleModel(
            mw.agg,
            [None if w is None else np.asarray(w, dtype) for w in mw.w_self],
            [np.asarray(w, dtype) for w in mw.w_neigh],
            [np.asarray(b, dtype) for b in mw.bias],
            list(mw.relu),
            [np.asarray(w, dtype) for w in (getattr(mw, "w_out", None) or [])],
            [np.asarray(b, dtype) for b in (getattr(mw, "b_out", None) or [])],
            float(getattr(mw, "gin_eps", 0.0)))


# ----------------------------------------------------------------------------
# graph: a set of arcs kept as sorted int64 keys u*n + v
# ----------------------------------------------------------------------------

class OracleGraph:
    """Arcs as sorted keys u * n + v; on a weighted graph `w` holds each arc's
    weight (float64, aligned with `keys`), else None."""

    def __init__(self, n: int, src, dst, undirected: bool = False, weights=None):
        self.n = int(n)
        self.undirected = bool(undirected)
        src = np.asarray(src, np.int64)
        dst = np.asarray(dst, np.int64)
        w = None if weights is None else np.asarray(weights, np.float64)
        if undirected:
            src, dst = np.concatenate([src, dst]), np.concatenate([dst, src])
            w = None if w is None else np.concatenate([w, w])
        keys = src * self.n + dst
        ok = src != dst
        keys = keys[ok]
        self.keys, first = np.unique(keys, return_index=True)
        self.w = None if w is None else w[ok][first]

    def copy(self) -> "OracleGraph":
        g = OracleGraph.__new__(OracleGraph)
        g.n, g.undirected, g.keys = self.n, self.undirected, self.keys.copy()
        g.w = None if self.w is None else self.w.copy()
        return g

    def in_sorted(self) -> Tuple[np.ndarray, np.ndarray]:
        """(sources, sinks) of all arcs ordered by sink, then source (cached)."""
        s, d, _ = self.in_sorted_weighted()
        return s, d

    def in_sorted_weighted(self):
        """(sources, sinks, weights or None) ordered by sink, then source (cached)."""
        cached = getattr(self, "_in_sorted", None)
        if cached is None or cached[0] is not self.keys:
            ik = (self.keys % self.n) * self.n + self.keys // self.n
            order = np.argsort(ik, kind="stable")
            ik = ik[order]
            cached = (self.keys, ik % self.n, ik // self.n, None if self.w is None else self.w[order])
            self._in_sorted = cached
        return cached[1], cached[2], cached[3]

    @property
    def num_arcs(self) -> int:
        return int(self.keys.size)

    def arcs(self) -> Tuple[np.ndarray, np.ndarray]:
        return self.keys // self.n, self.keys % self.n

    def has_arcs(self, keys: np.ndarray) -> np.ndarray:
        keys = np.asarray(keys, np.int64)
        j = np.searchsorted(self.keys, keys)
        jj = np.minimum(j, max(self.keys.size - 1, 0))
        return (j < self.keys.size) & (self.keys[jj] == keys) if self.keys.size else \
            np.zeros(keys.shape, bool)

    def out_degree(self) -> np.ndarray:
        return np.bincount(self.keys // self.n, minlength=self.n)

    def in_degree(self) -> np.ndarray:
        return np.bincount(self.keys % self.n, minlength=self.n)

    def out_neighbours(self, verts: np.ndarray) -> np.ndarray:
        """All v with (u, v) an arc for some u in verts (with repeats)."""
        verts = np.asarray(verts, np.int64)
        if verts.size == 0:
            return np.empty(0, np.int64)
        lo = np.searchsorted(self.keys, verts * self.n)
        hi = np.searchsorted(self.keys, (verts + 1) * self.n)
        cnt = hi - lo
        total = int(cnt.sum())
        if total == 0:
            return np.empty(0, np.int64)
        starts = np.repeat(lo - (np.cumsum(cnt) - cnt), cnt)
        return self.keys[starts + np.arange(total)] % self.n

    def weight_of(self, keys: np.ndarray) -> np.ndarray:
        """Weights of present arcs given by key (1 on an unweighted graph)."""
        if self.w is None:
            return np.ones(np.asarray(keys).shape)
        return self.w[np.searchsorted(self.keys, keys)]

    def in_adjacency(self, weights: Optional[np.ndarray] = None, dtype=np.float64) -> sp.csr_matrix:
        """Sparse A with A[v, u] = weight of arc u->v (1 by default): row v lists
        v's in-neighbours, so A @ H sums in-neighbour rows (Eq. (1))."""
        u, v = self.arcs()
        w = np.ones(u.size, dtype) if weights is None else np.asarray(weights, dtype)
        return sp.csr_matrix((w, (v, u)), shape=(self.n, self.n))


# ----------------------------------------------------------------------------
# applying a batch (sequential semantics) and its net effect
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class NetEffect:
    ins_src: np.ndarray
    ins_dst: np.ndarray
    del_src: np.ndarray
    del_dst: np.ndarray
    features: np.ndarray       # F: sorted distinct vertices with a feature write
    heads: np.ndarray          # sorted distinct sinks of net-changed arcs
    tails: np.ndarray          # sorted distinct sources of net-changed arcs
    out_deg_changed: np.ndarray  # sorted vertices whose out-degree changed
    edge_keys: int             # distinct non-loop edge keys the batch touched
    noop_edge_ops: int         # self-loop edge ops + touched keys with no net change
    rew_src: np.ndarray = dataclasses.field(default_factory=lambda: np.empty(0, np.int64))
    rew_dst: np.ndarray = dataclasses.field(default_factory=lambda: np.empty(0, np.int64))
    # arcs present before and after whose weight changed (weighted graphs)


def apply_batch(graph: OracleGraph, x: np.ndarray, ops: np.ndarray,
                feat_rows: np.ndarray, inplace: bool = False) -> Tuple[OracleGraph, np.ndarray, NetEffect]:
    """Applies `ops` in order to (graph, x) and returns (graph', x', net effect);
    with inplace=True the feature matrix x itself is updated and returned.

    An insert sets an arc present and a delete sets it absent, so the final
    state of an arc is fixed by the last op naming it; comparing with the
    pre-batch state gives the net inserts and deletes. Undirected graphs apply
    each edge op to both arcs and count the unordered edge once. On a weighted
    graph an insert carries the arc's weight (the op's fourth field, as float32
    bits) and also sets the weight of an arc already present, so the last op
    fixes the weight too; an arc present before and after with another weight is
    reweighted (its sink's neighbourhood changed)."""
    n = graph.n
    ops = np.asarray(ops, np.int32).reshape(-1, 4)
    op_w = ops[:, 3].copy().view(np.float32).astype(np.float64)
    weighted = graph.w is not None
    x_new = x if inplace else np.array(x, copy=True)
    final: Dict[Tuple[int, int], Tuple[bool, float]] = {}
    feat_vertices = set()
    selfloops = 0
    for (kind, u, v, f), wt in zip(ops.tolist(), op_w.tolist()):
        if kind == OP_FEATURE:
            x_new[u] = feat_rows[f]
            feat_vertices.add(u)
            continue
        if kind not in (OP_INSERT, OP_DELETE):
            raise ValueError(f"bad op kind {kind}")
        if u == v:
            selfloops += 1
            continue
        key = (min(u, v), max(u, v)) if graph.undirected else (u, v)
        final[key] = (kind == OP_INSERT, wt if weighted else 1.0)
    keys_touched = list(final.keys())
    ins, dels, rew, ins_w, rew_w = [], [], [], [], []
    noop_keys = 0
    if keys_touched:
        arr = np.array(keys_touched, np.int64)
        karr = arr[:, 0] * n + arr[:, 1]
        present = graph.has_arcs(karr)
        old_w = np.ones(karr.size)
        if weighted and present.any():
            old_w[present] = graph.weight_of(karr[present])
        for (a, b), was, ow in zip(keys_touched, present.tolist(), old_w.tolist()):
            now, nw = final[(a, b)]
            pairs = [(a, b), (b, a)] if graph.undirected else [(a, b)]
            if now and was:
                if weighted and nw != ow:
                    rew.extend(pairs)
                    rew_w.extend([nw] * len(pairs))
                else:
                    noop_keys += 1
                continue
            if now == was:
                noop_keys += 1
                continue
            (ins if now else dels).extend(pairs)
            if now:
                ins_w.extend([nw] * len(pairs))
    ins = np.array(ins, np.int64).reshape(-1, 2)
    dels = np.array(dels, np.int64).reshape(-1, 2)
    rew = np.array(rew, np.int64).reshape(-1, 2)
    g2 = graph.copy()
    keep, kw = g2.keys, g2.w
    if dels.size:
        at = np.searchsorted(keep, dels[:, 0] * n + dels[:, 1])
        keep = np.delete(keep, at)
        kw = None if kw is None else np.delete(kw, at)
    if rew.size:
        kw[np.searchsorted(keep, rew[:, 0] * n + rew[:, 1])] = rew_w
    if ins.size:
        nk = ins[:, 0] * n + ins[:, 1]
        order = np.argsort(nk)
        at = np.searchsorted(keep, nk[order])
        keep = np.insert(keep, at, nk[order])
        kw = None if kw is None else np.insert(kw, at, np.asarray(ins_w)[order])
    g2.keys, g2.w = keep, kw
    ch = np.concatenate([ins, dels, rew]) if (ins.size or dels.size or rew.size) else np.empty((0, 2), np.int64)
    od_change = np.zeros(n, np.int64)
    np.add.at(od_change, ins[:, 0], 1)
    np.add.at(od_change, dels[:, 0], -1)
    net = NetEffect(
        ins[:, 0], ins[:, 1], dels[:, 0], dels[:, 1],
        np.array(sorted(feat_vertices), np.int64),
        np.unique(ch[:, 1]), np.unique(ch[:, 0]),
        np.nonzero(od_change)[0].astype(np.int64),
        len(keys_touched), noop_keys + selfloops, rew[:, 0], rew[:, 1])
    return g2, x_new, net


# ----------------------------------------------------------------------------
# full layer-wise recompute (the definition, Eq. (1)-(2))
# ----------------------------------------------------------------------------

def aggregate(graph: OracleGraph, h: np.ndarray, agg: str) -> np.ndarray:
    """x_v = Aggregate({h_u : u in N_in(v)}) for every v (table of linear
    aggregators). GCN's weighted sum includes v itself (implicit self-loop)."""
    h = np.asarray(h)
    if agg in ("sum", "gc_sum", "gin"):
        return graph.in_adjacency(dtype=h.dtype) @ h
    if agg == "gc_wsum":
        return graph.in_adjacency(graph.w, dtype=h.dtype) @ h
    if agg in ("mean", "gc_mean"):
        s = graph.in_adjacency(dtype=h.dtype) @ h
        deg = graph.in_degree()
        out = np.zeros_like(s)
        nz = deg > 0
        out[nz] = s[nz] / deg[nz, None]
        return out
    if agg == "gcn":
        dout = graph.out_degree().astype(h.dtype)
        din = graph.in_degree().astype(h.dtype)
        u, v = graph.arcs()
        alpha = 1.0 / np.sqrt((dout[u] + 1.0) * (din[v] + 1.0))
        a = graph.in_adjacency(alpha, dtype=h.dtype)
        a_self = 1.0 / np.sqrt((dout + 1.0) * (din + 1.0))
        return a @ h + a_self[:, None] * h
    raise ValueError(agg)


def update(model: OracleModel, l: int, h_self: np.ndarray, agg: np.ndarray) -> np.ndarray:
    """Update^l then sigma (Eq. (2)) for rows with own embedding h_self and
    aggregate agg."""
    wn, b = model.w_neigh[l - 1], model.bias[l - 1]
    if model.agg in ("gcn", "gc_sum", "gc_mean", "gc_wsum"):
        out = agg @ wn.T + b
    elif model.agg == "gin":
        hidden = np.maximum(((1.0 + model.gin_eps) * h_self + agg) @ wn.T + b, 0.0)
        out = hidden @ model.w_out[l - 1].T + model.b_out[l - 1]
    else:
        out = h_self @ model.w_self[l - 1].T + agg @ wn.T + b
    if model.relu[l - 1]:
        out = np.maximum(out, 0.0)
    return out


def layer(graph: OracleGraph, h_prev: np.ndarray, model: OracleModel, l: int) -> np.ndarray:
    """One layer l (1-based) for every vertex (Eq. (1)-(2))."""
    return update(model, l, h_prev, aggregate(graph, h_prev, model.agg))


def full_recompute(graph: OracleGraph, x: np.ndarray, model: OracleModel,
                   dtype=np.float64) -> List[np.ndarray]:
    """[H^0 = X, H^1, ..., H^L] for all vertices, layer by layer."""
    hs = [np.asarray(x, dtype)]
    m = model if dtype == np.float64 else OracleModel.from_weights(model, dtype)
    for l in range(1, model.num_layers + 1):
        hs.append(layer(graph, hs[-1], m, l))
    return hs


# ----------------------------------------------------------------------------
# structural affected sets
# ----------------------------------------------------------------------------

def affected_sets(graph_post: OracleGraph, net: NetEffect, agg: str,
                  num_layers: int) -> List[np.ndarray]:
    """A^0 .. A^L as sorted int64 arrays.

    A^0 = F (vertices whose features were written). At hop l the vertices whose
    layer-(l-1) contribution changed are D^l = A^{l-1}, plus, under GCN, every
    vertex whose out-degree changed (its normalisation scales all its outgoing
    contributions and its own self-loop). A^l holds D^l's post-batch
    out-neighbours, every sink of a net-changed arc (its neighbourhood changed),
    and, for models with a self term, D^l itself (its own previous embedding
    enters its update; GraphConv has none)."""
    sets = [np.unique(net.features)]
    for _ in range(num_layers):
        d = sets[-1]
        if agg == "gcn":
            d = np.union1d(d, net.out_deg_changed)
        a = np.union1d(graph_post.out_neighbours(d), net.heads)
        if has_self_term(agg):
            a = np.union1d(a, d)
        sets.append(a.astype(np.int64))
    return sets


# ----------------------------------------------------------------------------
# sampled vertex-wise evaluation (for graphs too large to recompute often)
# ----------------------------------------------------------------------------

def sampled_embeddings(graph: OracleGraph, x: np.ndarray, model: OracleModel,
                       vertices: Sequence[int], upto_layer: Optional[int] = None,
                       dtype=np.float64) -> Tuple[np.ndarray, np.ndarray]:
    """h^l_v at layer l = upto_layer (default L) for the given vertices, computed
    only on the in-neighbourhood Eq. (1)-(2) reach (vertex-wise inference).
    Returns (sorted distinct vertices, their rows)."""
    L = model.num_layers if upto_layer is None else int(upto_layer)
    verts = np.unique(np.asarray(vertices, np.int64))
    s_sorted, d_sorted, w_sorted = graph.in_sorted_weighted()
    dout = graph.out_degree().astype(dtype)
    din = graph.in_degree().astype(dtype)

    def in_arcs(rows):
        lo = np.searchsorted(d_sorted, rows)
        hi = np.searchsorted(d_sorted, rows, side="right")
        cnt = hi - lo
        row_of = np.repeat(np.arange(rows.size), cnt)
        start = np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt)
        idx = start + np.arange(int(cnt.sum()))
        return row_of, s_sorted[idx], (None if w_sorted is None else w_sorted[idx])

    m = model if dtype == np.float64 else OracleModel.from_weights(model, dtype)
    need = [None] * (L + 1)
    need[L] = verts
    for l in range(L, 0, -1):
        _, us, _ = in_arcs(need[l])
        need[l - 1] = np.union1d(need[l], us)
    h = np.asarray(x, dtype)[need[0]]
    for l in range(1, L + 1):
        rows, prev = need[l], need[l - 1]
        row_of, us, ws = in_arcs(rows)
        col = np.searchsorted(prev, us)
        if model.agg == "gc_wsum":
            w = ws.astype(dtype)
        elif model.agg == "gcn":
            w = 1.0 / np.sqrt((dout[us] + 1.0) * (din[rows][row_of] + 1.0))
        elif model.agg in ("mean", "gc_mean"):
            w = 1.0 / din[rows][row_of]
        else:
            w = np.ones(us.size, dtype)
        agg = sp.csr_matrix((w, (row_of, col)), shape=(rows.size, prev.size)) @ h
        self_rows = h[np.searchsorted(prev, rows)]
        if model.agg == "gcn":
            agg = agg + (1.0 / np.sqrt((dout[rows] + 1.0) * (din[rows] + 1.0)))[:, None] * self_rows
        h = update(m, l, self_rows, agg)
    return verts, h


# ----------------------------------------------------------------------------
# a stateful driver and the error measure
# ----------------------------------------------------------------------------

class OracleState:
    """Graph + features + model; applies batches and recomputes on demand."""

    def __init__(self, n, src, dst, x, model: OracleModel, undirected=False, weights=None):
        self.graph = OracleGraph(n, src, dst, undirected, weights)
        self.x = np.asarray(x, np.float64).copy()
        self.model = model

    def apply(self, ops, feat_rows, with_sets: bool = True):
        g2, x2, net = apply_batch(self.graph, self.x, ops, np.asarray(feat_rows, np.float64), inplace=True)
        self.graph, self.x = g2, x2
        sets = affected_sets(g2, net, self.model.agg, self.model.num_layers) if with_sets else None
        return net, sets

    def embeddings(self, dtype=np.float64) -> List[np.ndarray]:
        return full_recompute(self.graph, self.x, self.model, dtype)


def row_relative_error(h: np.ndarray, h_ref: np.ndarray) -> float:
    """max_v ||h_v - h*_v||_inf / max(||h*_v||_inf, eps), eps = 1e-3 * RMS(H*):
    the per-vertex relative error, with a floor so that rows the ReLU zeroed do
    not divide by zero."""
    h = np.asarray(h, np.float64)
    h_ref = np.asarray(h_ref, np.float64)
    if h_ref.size == 0:
        return 0.0
    eps = 1e-3 * math.sqrt(float(np.mean(h_ref * h_ref))) + 1e-30
    num = np.max(np.abs(h - h_ref), axis=1)
    den = np.maximum(np.max(np.abs(h_ref), axis=1), eps)
    return float(np.max(num / den))

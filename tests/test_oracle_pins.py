"""Pins of the CPU oracle against facts that do not come from the oracle itself:
hand-derived closed forms, textbook special cases, the paper's worked examples,
brute force on tiny inputs and invariants the paper states."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import ripple_oracle as O
from paper_2505_12112_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _model(agg, w_self, w_neigh, bias, relu, w_out=(), b_out=(), gin_eps=0.0):
    return O.OracleModel(
        agg,
        [None if w is None else np.array(w, np.float64) for w in w_self],
        [np.array(w, np.float64) for w in w_neigh],
        [np.array(b, np.float64) for b in bias],
        list(relu),
        [np.array(w, np.float64) for w in w_out],
        [np.array(b, np.float64) for b in b_out],
        float(gin_eps))


def _random_model(rng, agg, dims, relu_all=False, relu_none=False, gin_eps=0.3):
    ws, wn, bs, act, wo, bo = [], [], [], [], [], []
    L = len(dims) - 1
    for l in range(1, L + 1):
        ws.append(rng.standard_normal((dims[l], dims[l - 1])) if agg in ("sum", "mean") else None)
        wn.append(rng.standard_normal((dims[l], dims[l - 1])))
        bs.append(rng.standard_normal(dims[l]) * 0.1)
        if agg == "gin":
            wo.append(rng.standard_normal((dims[l], dims[l])))
            bo.append(rng.standard_normal(dims[l]) * 0.1)
        act.append(False if relu_none else (True if relu_all else l < L))
    return O.OracleModel(agg, ws, wn, bs, act, wo, bo, gin_eps if agg == "gin" else 0.0)


def _eval_expr(s):
    return float(eval(s, {"__builtins__": {}}, {"sqrt": math.sqrt}))


# ---------------------------------------------------------------------------
# hand-derived closed forms
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case", ["sage_sum_2layer", "sage_mean_1layer", "gcn_directed_1layer", "gc_sum_2layer",
                                  "gc_mean_1layer", "gin_1layer", "gc_wsum_1layer"])
def test_hand_derived_values(case):
    fx = json.load(open(os.path.join(GOLDEN, "hand_small_graph.json")))
    arcs = np.array(fx["arcs"])
    c = fx["cases"][case]
    g = O.OracleGraph(fx["n"], arcs[:, 0], arcs[:, 1], weights=c.get("arc_weights"))
    m = _model(c["agg"], c["w_self"], c["w_neigh"], c["bias"], c["relu"], c.get("w_out", ()),
               c.get("b_out", ()), c.get("gin_eps", 0.0))
    hs = O.full_recompute(g, np.array(fx["x"], np.float64), m)
    for layer, rows in c["expected"].items():
        want = np.array([[_eval_expr(e) for e in r] for r in rows])
        np.testing.assert_allclose(hs[int(layer)], want, rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------
# textbook special cases
# ---------------------------------------------------------------------------

def test_sum_aggregation_is_brute_force_in_neighbour_sum():
    """W_self=0, W_neigh=I, no bias, no activation: H^1 = plain in-neighbour sum,
    computed here by a loop over the arc list (no sparse algebra)."""
    rng = np.random.default_rng(1)
    n, d = 40, 5
    src, dst = synth.erdos_renyi(n, 150, rng)
    x = rng.standard_normal((n, d))
    m = O.OracleModel("sum", [np.zeros((d, d))], [np.eye(d)], [np.zeros(d)], [False])
    h1 = O.full_recompute(O.OracleGraph(n, src, dst), x, m)[1]
    want = np.zeros((n, d))
    for u, v in zip(src.tolist(), dst.tolist()):
        want[v] += x[u]
    np.testing.assert_allclose(h1, want, rtol=0, atol=1e-12)


def test_gcn_matches_kipf_closed_form_on_undirected_graphs():
    """On an undirected graph GCN's layer is D^-1/2 (A+I) D^-1/2 H W^T + b (Kipf &
    Welling), built here with dense matrices."""
    rng = np.random.default_rng(2)
    n, d0, d1 = 30, 4, 3
    src, dst = synth.erdos_renyi(n, 60, rng, undirected=True)
    a = np.zeros((n, n))
    a[src, dst] = 1
    a[dst, src] = 1
    ahat = a + np.eye(n)
    dinv = np.diag(1.0 / np.sqrt(ahat.sum(1)))
    x = rng.standard_normal((n, d0))
    w = rng.standard_normal((d1, d0))
    b = rng.standard_normal(d1)
    m = O.OracleModel("gcn", [None], [w], [b], [False])
    h1 = O.full_recompute(O.OracleGraph(n, src, dst, undirected=True), x, m)[1]
    want = dinv @ ahat @ dinv @ x @ w.T + b
    np.testing.assert_allclose(h1, want, rtol=0, atol=1e-12)


def test_mean_equals_scaled_sum_on_in_regular_graph():
    """Every vertex has in-degree k (out-degrees vary): SAGE-mean with W_neigh
    equals SAGE-sum with W_neigh / k. Dividing by the out-degree would fail."""
    rng = np.random.default_rng(3)
    n, k, d = 25, 3, 4
    src, dst = [], []
    for v in range(n):
        for u in rng.choice([w for w in range(n) if w != v], k, replace=False):
            src.append(u)
            dst.append(v)
    g = O.OracleGraph(n, src, dst)
    assert len(set(g.out_degree().tolist())) > 1
    x = rng.standard_normal((n, d))
    ws, wn, b = rng.standard_normal((d, d)), rng.standard_normal((d, d)), rng.standard_normal(d)
    hm = O.full_recompute(g, x, O.OracleModel("mean", [ws], [wn], [b], [True]))[1]
    hs = O.full_recompute(g, x, O.OracleModel("sum", [ws], [wn / k], [b], [True]))[1]
    np.testing.assert_allclose(hm, hs, rtol=1e-13, atol=1e-13)


def test_mean_with_no_in_neighbours_is_zero_aggregate():
    g = O.OracleGraph(3, [0], [1])
    x = np.array([[1.0], [2.0], [3.0]])
    m = O.OracleModel("mean", [np.zeros((1, 1))], [np.eye(1)], [np.zeros(1)], [False])
    np.testing.assert_array_equal(O.full_recompute(g, x, m)[1], [[0.0], [1.0], [0.0]])


# ---------------------------------------------------------------------------
# the paper's worked examples (affected sets)
# ---------------------------------------------------------------------------

def _paper_examples():
    return json.load(open(os.path.join(GOLDEN, "paper_examples.json")))["examples"]


@pytest.mark.parametrize("ex", _paper_examples(), ids=lambda e: e["name"])
def test_paper_worked_examples(ex):
    names = ex["vertices"]
    ix = {v: i for i, v in enumerate(names)}
    arcs = np.array([[ix[a], ix[b]] for a, b in ex["arcs"]])
    g = O.OracleGraph(len(names), arcs[:, 0], arcs[:, 1])
    ops, rows = [], []
    for op in ex["batch"]:
        if op[0] == "feature":
            ops.append([O.OP_FEATURE, ix[op[1]], -1, len(rows)])
            rows.append([7.0])
        else:
            kind = O.OP_INSERT if op[0] == "insert" else O.OP_DELETE
            ops.append([kind, ix[op[1]], ix[op[2]], -1])
    x = np.zeros((len(names), 1))
    g2, _, net = O.apply_batch(g, x, np.array(ops), np.array(rows).reshape(-1, 1))
    sets = O.affected_sets(g2, net, ex["agg"], ex["num_layers"])
    for layer, want in ex["affected"].items():
        got = sorted(names[i] for i in sets[int(layer)])
        assert got == sorted(want), (ex["name"], layer, got, want)


# ---------------------------------------------------------------------------
# brute force: structural affected sets vs numerically changed rows
# ---------------------------------------------------------------------------

def _changed_rows(h_pre, h_post):
    return np.nonzero(np.any(h_pre != h_post, axis=1))[0]


def _weights_for(agg, rng, m):
    return rng.uniform(0.5, 1.5, m).astype(np.float32) if agg == "gc_wsum" else None


@pytest.mark.parametrize("agg", ["sum", "mean", "gcn", "gc_sum", "gc_mean", "gc_wsum"])
@pytest.mark.parametrize("undirected", [False, True])
def test_affected_sets_equal_changed_rows_without_activation(agg, undirected):
    """With no activation and generic values, a vertex's embedding changes iff it
    is structurally affected (Sec. IV-C: no pruning, and nothing else changes).
    For GraphConv this includes that a vertex whose own embedding changed, with no
    changed in-neighbour and no changed arc, keeps its next-layer embedding."""
    rng = np.random.default_rng(10 + O.AGGREGATORS.index(agg) + 7 * undirected)
    n, L = 30, 3
    dims = (3, 4, 3, 2)
    for trial in range(12):
        src, dst = synth.erdos_renyi(n, 45 if undirected else 70, rng, undirected=undirected)
        st = O.OracleState(n, src, dst, rng.standard_normal((n, dims[0])),
                           _random_model(rng, agg, dims, relu_none=True), undirected,
                           _weights_for(agg, rng, src.size))
        pre = st.embeddings()
        a, b = st.graph.arcs()
        batch = synth.adversarial_batch(rng, n, dims[0], bs=int(rng.integers(1, 10)),
                                        hot=6, existing=(a, b), weighted=agg == "gc_wsum")
        net, sets = st.apply(batch.ops, batch.feat_rows)
        post = st.embeddings()
        for l in range(1, L + 1):
            np.testing.assert_array_equal(_changed_rows(pre[l], post[l]), sets[l],
                                          err_msg=f"trial {trial} layer {l}")


@pytest.mark.parametrize("agg", ["sum", "mean", "gcn", "gc_sum", "gc_mean", "gin", "gc_wsum"])
def test_changed_rows_within_affected_sets_with_relu(agg):
    rng = np.random.default_rng(30)
    n, dims = 40, (4, 5, 3)
    for _ in range(8):
        src, dst = synth.erdos_renyi(n, 90, rng)
        st = O.OracleState(n, src, dst, rng.standard_normal((n, dims[0])),
                           _random_model(rng, agg, dims, relu_all=True), weights=_weights_for(agg, rng, src.size))
        pre = st.embeddings()
        a, b = st.graph.arcs()
        batch = synth.adversarial_batch(rng, n, dims[0], bs=8, hot=8, existing=(a, b), weighted=agg == "gc_wsum")
        _, sets = st.apply(batch.ops, batch.feat_rows)
        post = st.embeddings()
        for l in range(1, 3):
            assert set(_changed_rows(pre[l], post[l]).tolist()) <= set(sets[l].tolist())


def test_gcn_tail_with_unchanged_out_degree_does_not_dirty_its_out_arcs():
    """u loses one out-arc and gains another in the same batch: d_out(u) is
    unchanged, so only the two sinks are affected at hop 1 (plus nothing else)."""
    g = O.OracleGraph(5, [0, 0, 1], [1, 2, 3])
    ops = np.array([[O.OP_DELETE, 0, 1, -1], [O.OP_INSERT, 0, 4, -1]])
    g2, _, net = O.apply_batch(g, np.zeros((5, 1)), ops, np.zeros((0, 1)))
    assert net.out_deg_changed.size == 0
    sets = O.affected_sets(g2, net, "gcn", 1)
    np.testing.assert_array_equal(sets[1], [1, 4])


# ---------------------------------------------------------------------------
# sequential semantics and invariants
# ---------------------------------------------------------------------------

def _brute_apply(n, arcs_set, x, ops, rows, undirected):
    """Op-by-op application on a Python set (the plain meaning of a batch)."""
    arcs_set = set(arcs_set)
    x = x.copy()
    for kind, u, v, f in ops.tolist():
        if kind == O.OP_FEATURE:
            x[u] = rows[f]
            continue
        if u == v:
            continue
        pairs = [(u, v), (v, u)] if undirected else [(u, v)]
        for p in pairs:
            if kind == O.OP_INSERT:
                arcs_set.add(p)
            else:
                arcs_set.discard(p)
    return arcs_set, x


@pytest.mark.parametrize("undirected", [False, True])
def test_batch_equals_op_by_op_application(undirected):
    """Sec. IV-C.1: combined updates equal the updates applied one at a time."""
    rng = np.random.default_rng(40 + undirected)
    n, d = 25, 3
    for _ in range(20):
        src, dst = synth.erdos_renyi(n, 40, rng, undirected=undirected)
        g = O.OracleGraph(n, src, dst, undirected)
        x = rng.standard_normal((n, d))
        a, b = g.arcs()
        batch = synth.adversarial_batch(rng, n, d, bs=15, hot=5, existing=(a, b))
        g2, x2, net = O.apply_batch(g, x, batch.ops, batch.feat_rows)
        want_set, want_x = _brute_apply(n, zip(a.tolist(), b.tolist()), x, batch.ops,
                                        batch.feat_rows, undirected)
        got = set(zip(*[t.tolist() for t in g2.arcs()]))
        assert got == want_set
        np.testing.assert_array_equal(x2, want_x)
        # one op per batch reaches the same state
        g3, x3 = g, x
        for i in range(batch.size):
            g3, x3, _ = O.apply_batch(g3, x3, batch.ops[i:i + 1], batch.feat_rows)
        np.testing.assert_array_equal(g3.keys, g2.keys)
        np.testing.assert_array_equal(x3, x2)
        # net sets are consistent with the two snapshots
        pre = set(zip(a.tolist(), b.tolist()))
        assert set(zip(net.ins_src.tolist(), net.ins_dst.tolist())) == got - pre
        assert set(zip(net.del_src.tolist(), net.del_dst.tolist())) == pre - got


def test_insert_then_delete_restores_embeddings():
    rng = np.random.default_rng(50)
    n, dims = 30, (3, 4, 2)
    src, dst = synth.erdos_renyi(n, 60, rng)
    st = O.OracleState(n, src, dst, rng.standard_normal((n, 3)), _random_model(rng, "mean", dims))
    before = st.embeddings()
    new = [(u, v) for u, v in itertools.product(range(n), range(n))
           if u != v and not st.graph.has_arcs(np.array([u * n + v]))[0]][:10]
    ins = np.array([[O.OP_INSERT, u, v, -1] for u, v in new])
    dels = np.array([[O.OP_DELETE, u, v, -1] for u, v in new])
    st.apply(ins, np.zeros((0, 3)))
    st.apply(dels, np.zeros((0, 3)))
    after = st.embeddings()
    for l in range(3):
        np.testing.assert_array_equal(before[l], after[l])


def test_noop_accounting():
    g = O.OracleGraph(4, [0, 1], [1, 2])
    ops = np.array([
        [O.OP_INSERT, 0, 1, -1],   # present already: no net change
        [O.OP_DELETE, 2, 3, -1],   # absent: no net change
        [O.OP_INSERT, 3, 3, -1],   # self-loop
        [O.OP_INSERT, 2, 3, -1],   # net insert (last op on key (2,3))
        [O.OP_DELETE, 1, 2, -1],   # net delete
        [O.OP_FEATURE, 1, -1, 0],
        [O.OP_FEATURE, 1, -1, 1],  # last write wins
    ])
    rows = np.array([[1.0, 1.0], [2.0, 2.0]])
    g2, x2, net = O.apply_batch(g, np.zeros((4, 2)), ops, rows)
    assert net.edge_keys == 3 and net.noop_edge_ops == 2
    np.testing.assert_array_equal(net.ins_src, [2])
    np.testing.assert_array_equal(net.del_src, [1])
    np.testing.assert_array_equal(x2[1], [2.0, 2.0])
    np.testing.assert_array_equal(net.heads, [2, 3])
    np.testing.assert_array_equal(net.tails, [1, 2])


def test_permutation_equivariance():
    """Relabelling vertices permutes the embeddings (catches index mix-ups)."""
    rng = np.random.default_rng(60)
    n, dims = 35, (3, 5, 2)
    src, dst = synth.erdos_renyi(n, 80, rng)
    x = rng.standard_normal((n, 3))
    perm = rng.permutation(n)
    for agg in ("sum", "mean", "gcn"):
        m = _random_model(rng, agg, dims)
        h = O.full_recompute(O.OracleGraph(n, src, dst), x, m)
        xp = np.empty_like(x)
        xp[perm] = x
        hp = O.full_recompute(O.OracleGraph(n, perm[src], perm[dst]), xp, m)
        for l in range(3):
            np.testing.assert_allclose(hp[l][perm], h[l], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("agg", ["sum", "mean", "gcn", "gc_sum", "gc_mean", "gin", "gc_wsum"])
def test_sampled_embeddings_match_full_recompute(agg):
    rng = np.random.default_rng(70)
    n, dims = 200, (4, 6, 5, 3)
    src, dst = synth.erdos_renyi(n, 900, rng)
    g = O.OracleGraph(n, src, dst, weights=_weights_for(agg, rng, src.size))
    x = rng.standard_normal((n, 4))
    m = _random_model(rng, agg, dims)
    full = O.full_recompute(g, x, m)
    verts = rng.choice(n, 7, replace=False)
    for layer in (1, 2, 3):
        vs, hv = O.sampled_embeddings(g, x, m, verts, upto_layer=layer)
        np.testing.assert_allclose(hv, full[layer][vs], rtol=1e-12, atol=1e-12)


def test_row_relative_error_definition():
    ref = np.array([[1.0, -2.0], [0.0, 0.0], [4.0, 0.5]])
    got = ref + np.array([[0.0, 2e-4], [0.0, 0.0], [-4e-4, 0.0]])
    # row 0: 2e-4 / 2 = 1e-4; row 2: 4e-4 / 4 = 1e-4
    assert math.isclose(O.row_relative_error(got, ref), 1e-4, rel_tol=1e-9)
    eps = 1e-3 * math.sqrt(np.mean(ref * ref))
    got2 = ref.copy()
    got2[1, 0] = 1e-6
    assert math.isclose(O.row_relative_error(got2, ref), 1e-6 / eps, rel_tol=1e-9)


# ---------------------------------------------------------------------------
# GraphConv and GIN against other definitions
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("agg,sage", [("gc_sum", "sum"), ("gc_mean", "mean")])
def test_graphconv_is_graphsage_without_self_weight(agg, sage):
    """GraphConv's update is GraphSAGE's with the self weight set to zero."""
    rng = np.random.default_rng(80)
    n, dims = 60, (5, 7, 3)
    src, dst = synth.erdos_renyi(n, 200, rng)
    g = O.OracleGraph(n, src, dst)
    x = rng.standard_normal((n, dims[0]))
    gc = _random_model(rng, agg, dims)
    sg = O.OracleModel(sage, [np.zeros((dims[l], dims[l - 1])) for l in (1, 2)], gc.w_neigh, gc.bias, gc.relu)
    for a, b in zip(O.full_recompute(g, x, gc), O.full_recompute(g, x, sg)):
        np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)


def test_gin_matches_a_per_vertex_loop():
    """GIN by brute force: for each vertex, (1 + eps) times its row plus a Python
    loop over its in-neighbours, then the two-layer MLP written out per vertex."""
    rng = np.random.default_rng(81)
    n, dims, eps = 25, (3, 4, 2), 0.25
    src, dst = synth.erdos_renyi(n, 70, rng)
    g = O.OracleGraph(n, src, dst)
    x = rng.standard_normal((n, dims[0]))
    m = _random_model(rng, "gin", dims, gin_eps=eps)
    hs = O.full_recompute(g, x, m)
    a, b = g.arcs()
    h = x
    for l in (1, 2):
        out = np.zeros((n, dims[l]))
        for v in range(n):
            z = (1.0 + eps) * h[v]
            for u in a[b == v]:
                z = z + h[u]
            hid = [max(sum(m.w_neigh[l - 1][i, k] * z[k] for k in range(z.size)) + m.bias[l - 1][i], 0.0)
                   for i in range(dims[l])]
            for j in range(dims[l]):
                y = sum(m.w_out[l - 1][j, i] * hid[i] for i in range(dims[l])) + m.b_out[l - 1][j]
                out[v, j] = max(y, 0.0) if m.relu[l - 1] else y
        np.testing.assert_allclose(hs[l], out, rtol=1e-12, atol=1e-12)
        h = out


# ---------------------------------------------------------------------------
# weighted graphs (GC-W)
# ---------------------------------------------------------------------------

def _brute_apply_weighted(n, arcs, x, ops, rows, undirected):
    """Op-by-op on a dict arc -> weight: an insert sets the arc present with the
    op's weight (also when present), a delete removes it."""
    arcs = dict(arcs)
    x = x.copy()
    wts = np.asarray(ops, np.int32)[:, 3].copy().view(np.float32)
    for (kind, u, v, f), w in zip(np.asarray(ops).tolist(), wts.tolist()):
        if kind == O.OP_FEATURE:
            x[u] = rows[f]
            continue
        if u == v:
            continue
        for p in ([(u, v), (v, u)] if undirected else [(u, v)]):
            if kind == O.OP_INSERT:
                arcs[p] = w
            else:
                arcs.pop(p, None)
    return arcs, x


@pytest.mark.parametrize("undirected", [False, True])
def test_weighted_batch_equals_op_by_op_application(undirected):
    """Weights follow the same sequential semantics: the last insert of an arc
    sets its weight; the net effect splits into inserts, deletes and reweights."""
    rng = np.random.default_rng(90 + undirected)
    n, d = 25, 3
    for _ in range(20):
        src, dst = synth.erdos_renyi(n, 40, rng, undirected=undirected)
        w = rng.uniform(0.5, 1.5, src.size).astype(np.float32)
        g = O.OracleGraph(n, src, dst, undirected, w)
        x = rng.standard_normal((n, d))
        a, b = g.arcs()
        batch = synth.adversarial_batch(rng, n, d, bs=15, hot=5, existing=(a, b), weighted=True)
        g2, x2, net = O.apply_batch(g, x, batch.ops, batch.feat_rows)
        pre = {(u, v): float(wt) for u, v, wt in zip(a.tolist(), b.tolist(), g.w.tolist())}
        want, want_x = _brute_apply_weighted(n, pre, x, batch.ops, batch.feat_rows, undirected)
        u2, v2 = g2.arcs()
        got = {(u, v): float(wt) for u, v, wt in zip(u2.tolist(), v2.tolist(), g2.w.tolist())}
        assert got == want
        np.testing.assert_array_equal(x2, want_x)
        rew = set(zip(net.rew_src.tolist(), net.rew_dst.tolist()))
        assert rew == {k for k in set(pre) & set(got) if pre[k] != got[k]}
        assert set(zip(net.ins_src.tolist(), net.ins_dst.tolist())) == set(got) - set(pre)
        assert set(zip(net.del_src.tolist(), net.del_dst.tolist())) == set(pre) - set(got)
        for u, v in rew:
            assert v in net.heads


def test_weighted_sum_with_unit_weights_is_graphconv_sum():
    rng = np.random.default_rng(91)
    n, dims = 50, (4, 6, 3)
    src, dst = synth.erdos_renyi(n, 180, rng)
    x = rng.standard_normal((n, dims[0]))
    m = _random_model(rng, "gc_wsum", dims)
    unit = O.full_recompute(O.OracleGraph(n, src, dst, weights=np.ones(src.size)), x, m)
    m.agg = "gc_sum"
    plain = O.full_recompute(O.OracleGraph(n, src, dst), x, m)
    for a, b in zip(unit, plain):
        np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)


def test_weighted_sum_matches_a_per_vertex_loop():
    rng = np.random.default_rng(92)
    n, dims = 20, (3, 2)
    src, dst = synth.erdos_renyi(n, 60, rng)
    w = rng.uniform(0.5, 1.5, src.size)
    g = O.OracleGraph(n, src, dst, weights=w)
    x = rng.standard_normal((n, dims[0]))
    m = _random_model(rng, "gc_wsum", dims)
    h1 = O.full_recompute(g, x, m)[1]
    for v in range(n):
        agg = np.zeros(dims[0])
        for u, t, wt in zip(src.tolist(), dst.tolist(), w.tolist()):
            if t == v:
                agg = agg + wt * x[u]
        np.testing.assert_allclose(h1[v], m.w_neigh[0] @ agg + m.bias[0], rtol=1e-12, atol=1e-12)


def test_reinserting_a_present_arc_with_its_own_weight_is_a_noop():
    g = O.OracleGraph(3, [0, 1], [1, 2], weights=[0.75, 1.25])
    ops = np.array([[O.OP_INSERT, 0, 1, 0], [O.OP_INSERT, 1, 2, 0]], np.int32)
    ops[:, 3] = synth.weight_bits([0.75, 2.0])
    g2, _, net = O.apply_batch(g, np.zeros((3, 1)), ops, np.zeros((0, 1)))
    assert net.noop_edge_ops == 1 and net.edge_keys == 2
    np.testing.assert_array_equal(net.rew_src, [1])
    np.testing.assert_array_equal(net.heads, [2])
    np.testing.assert_array_equal(g2.w, [0.75, 2.0])


def test_row_relative_floor_asks_more_than_fp32_on_cancelling_rows():
    """The error measure (row-relative, floor 1e-3 RMS of the layer) against what
    fp32 arithmetic can deliver: on rows whose pre-activation cancels to a small
    fraction of the magnitude of its terms, the float64 definition evaluated in
    float32 from the same fp32 inputs misses 1e-4, yet stays within the fp32
    forward error bound that the GPU hub test allows such rows. Fifty vertices with
    300 in-neighbours each get a self row solved so that W_self h_v nearly cancels
    W_neigh S_v + b."""
    from tests.harness import fp32_forward_bound
    rng = np.random.default_rng(5)
    n, d0, d1 = 600, 8, 6
    src = [rng.choice(np.arange(100, n), 300, replace=False) for _ in range(50)]
    dst = [np.full(300, v) for v in range(50)]
    es, ed = synth.erdos_renyi(n - 100, 3000, rng)
    src = np.concatenate(src + [es + 100]).astype(np.int32)
    dst = np.concatenate(dst + [ed + 100]).astype(np.int32)
    w = synth.model_weights(synth.ModelSpec("sum", (d0, d1)), rng, bias_std=0.1)
    model = O.OracleModel.from_weights(w)
    graph = O.OracleGraph(n, src, dst)
    x = rng.standard_normal((n, d0)).astype(np.float32)
    s = O.aggregate(graph, x.astype(np.float64), "sum")
    target = np.abs(rng.standard_normal((50, d1))) * 1e-3  # small positive pre-activations
    rhs = target - s[:50] @ model.w_neigh[0].T - model.bias[0]
    x[:50] = (rhs @ np.linalg.pinv(model.w_self[0]).T).astype(np.float32)
    ref = O.full_recompute(graph, x, model)
    got = O.full_recompute(graph, x, model, dtype=np.float32)[1].astype(np.float64)
    diff = np.max(np.abs(got - ref[1]), axis=1)
    floor = 1e-3 * np.sqrt(np.mean(ref[1] ** 2))
    r16 = diff / np.maximum(np.max(np.abs(ref[1]), axis=1), floor)
    st = O.OracleState(n, src, dst, x, model)
    bound = fp32_forward_bound(st, ref, 1)
    assert r16[:50].max() > 1e-4, r16[:50].max()  # fp32 cannot resolve R16 on these rows
    assert r16[50:].max() <= 1e-4                   # the other rows meet it
    assert np.all(diff <= bound), (diff / bound).max()

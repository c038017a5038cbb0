"""Parity at the benchmark workloads' full sizes, in the launch configuration
bench.py times (library stream, batch sizes of the workload)."""
import sys
import time

import numpy as np
import pytest

from oracle import ripple_oracle as O
from paper_2505_12112_amd import synth
from tests.harness import BF16_UNIT, FP32_TOL_BF16, Pair, check_embeddings_conditioned

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("bs", [1, 10, 100, 1000])
def test_sparse_mid_full_size(bs):
    """169,343 vertices / 1,166,243 arcs, GraphSAGE-sum 128-256-40, at each of the
    workload's batch sizes: affected sets every batch, all embeddings against a
    float64 full recompute at the end."""
    wl = synth.build_workload("sparse_mid")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights)
    try:
        p.check_embeddings()
        t0 = time.time()
        nb = {1: 50, 10: 30, 100: 20, 1000: 5}[bs]
        for b in range(nb):
            st, _, sets = p.step(wl.stream.next_batch(bs))
        _say(f"sparse_mid bs={bs}: {nb} batches in {time.time() - t0:.1f}s, last |A| = {[s.size for s in sets]}")
        errs = p.check_embeddings()
        _say("  row-relative errors", errs)
        p.check_arcs()
    finally:
        p.close()


def test_sparse_mid_bf16_full_size():
    """The headline workload with bf16 transform operands: 20 batches of 100 with
    affected sets every batch, then every row against a float64 full recompute at
    2e-2 (R16, or the bf16 forward error bound where R16 asks for more than bf16
    resolves)."""
    wl = synth.build_workload("sparse_mid")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights, gemm="bf16")
    try:
        for b in range(20):
            p.step(wl.stream.next_batch(100))
        res = check_embeddings_conditioned(p, FP32_TOL_BF16, BF16_UNIT)
        _say(f"sparse_mid bf16: per layer (max R16 error, rows within the bf16 bound) {res}")
        p.check_arcs()
    finally:
        p.close()


@pytest.mark.parametrize("bs", [100, 1000])
@pytest.mark.parametrize("config", ["sparse_mid_gc_sum", "sparse_mid_gc_mean", "sparse_mid_gin", "sparse_mid_gc_wsum",
                                    "sparse_mid_mean"])
def test_evaluation_workloads_on_the_arxiv_shaped_graph(config, bs):
    """GraphConv-sum, GraphConv-mean, GIN-sum and GraphConv-weighted-sum (2 layers,
    128-256-40) and the 3-layer GraphSAGE-mean at full size, at the batch sizes
    bench.py reports for them: 20 batches of 100 or 5 of 1000 with affected sets
    every batch, then all embeddings against a float64 full recompute."""
    wl = synth.build_workload(config)
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights, edge_w=wl.edge_w)
    nb = 20 if bs == 100 else 5
    try:
        p.check_embeddings()
        t0 = time.time()
        for b in range(nb):
            st, _, sets = p.step(wl.stream.next_batch(bs))
        errs = p.check_embeddings()
        _say(f"{config} bs={bs}: {nb} batches in {time.time() - t0:.1f}s, last |A| = {[s.size for s in sets]}, "
             f"row-relative errors {errs}")
        p.check_arcs()
    finally:
        p.close()


def test_sparse_mid_mean_thousand_batches():
    """The 3-layer mean workload: 1000 consecutive batches of 100, affected sets
    checked every 10th batch, embeddings against full recompute after 500 and 1000."""
    wl = synth.build_workload("sparse_mid_mean")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights)
    try:
        t0 = time.time()
        worst = 0.0
        for b in range(1000):
            batch = wl.stream.next_batch(100)
            if b % 10 == 9:
                p.step(batch)
            else:
                p.lib.apply_updates(batch.ops, batch.feat_rows)
                p.orc.apply(batch.ops, batch.feat_rows, with_sets=False)
            if (b + 1) % 500 == 0:
                errs = p.check_embeddings()
                worst = max(worst, max(errs))
                _say(f"  batch {b + 1} ({time.time() - t0:.0f}s): row-relative errors {['%.2e' % e for e in errs]}")
        p.check_arcs()
        p.check_aggregates()
    finally:
        p.close()


def _sample_vertices(rng, orc, affected, k, max_reach, hubs=16):
    """Up to k affected and k other vertices whose two-hop in-neighbourhood (in arcs)
    stays below max_reach, so the oracle can evaluate them one by one, plus the
    `hubs` vertices of highest in-degree whatever their reach (the rows that receive
    the most messages, and so the most rounding)."""
    src_s, dst_s = orc.graph.in_sorted()
    indeg = np.bincount(dst_s, minlength=orc.graph.n)
    picked = []
    for pool in (affected, rng.integers(0, orc.graph.n, 50 * k)):
        pool = np.asarray(pool)
        got = 0
        for v in rng.permutation(pool)[:50 * k]:
            lo, hi = np.searchsorted(dst_s, [v, v + 1])
            reach = int(indeg[src_s[lo:hi]].sum()) + (hi - lo)
            if reach <= max_reach:
                picked.append(int(v))
                got += 1
                if got == k:
                    break
    top = np.argsort(indeg, kind="stable")[-hubs:] if hubs else np.zeros(0, np.int64)
    return np.unique(np.concatenate([np.array(picked, np.int64), top.astype(np.int64)])), top


def _check_sampled(p, verts, layers, tol=1e-4):
    errs = []
    for l in layers:
        vs, ref = O.sampled_embeddings(p.orc.graph, p.orc.x, p.orc.model, verts, upto_layer=l)
        got = p.lib.get_embeddings(l, vs.astype(np.int32))
        # row-relative error with the floor taken from the sampled reference rows
        err = O.row_relative_error(got, ref)
        errs.append(err)
        assert err <= tol, (l, err)
    return errs


@pytest.mark.parametrize("config,schedule", [("dense_large", ((10, 5), (100, 3), (1000, 2))),
                                             ("dense_large_2l", ((100, 3), (1000, 2)))])
def test_dense_large_full_size(config, schedule):
    """Products-shaped undirected graph at full size (2,449,029 vertices, 61,859,140
    edges), GraphSAGE-sum 100-256-256-47 or 100-256-47, message forms chosen by the
    library as bench.py runs it, on one context: batches of each of the workload's
    sizes in turn (10, 100, 1000) with affected sets compared bit for bit every
    batch, then embeddings of sampled vertices (the 16 highest in-degrees among
    them) at every layer. A cached aggregate that went wrong at any batch size stays
    wrong (messages only add to it), so the final check covers every phase."""
    t0 = time.time()
    wl = synth.build_workload(config)
    _say(f"{config} generated in {time.time() - t0:.0f}s")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights, undirected=True)
    L = len(wl.weights.dims) - 1
    try:
        _say(f"  loaded + bootstrapped, oracle built ({time.time() - t0:.0f}s)")
        rng = np.random.default_rng(5 + sum(bs for bs, _ in schedule))
        seen = {}
        for bs, nb in schedule:
            forms = 0
            for b in range(nb):
                st, _, sets = p.step(wl.stream.next_batch(bs))
                forms |= st["pull_layers"] | st["dense_layers"]
                _say(f"  bs={bs} batch {b}: |A| = {[s.size for s in sets]}, pull layers {st['pull_layers']:b}, "
                     f"dense layers {st['dense_layers']:b}, bucket layers {st['bucket_layers']:b} "
                     f"({time.time() - t0:.0f}s)")
            seen[bs] = forms
        if config == "dense_large":
            assert seen[100] & 0b1000, "the third layer should switch to a pull form at batch 100"
        verts, hubs = _sample_vertices(rng, p.orc, sets[L], 24, 400_000)
        errs = _check_sampled(p, verts, range(1, L + 1))
        _say(f"  {verts.size} sampled vertices (hub in-degrees {np.bincount(p.orc.graph.in_sorted()[1], minlength=wl.n)[hubs][-3:]}), "
             f"row-relative errors {errs} ({time.time() - t0:.0f}s)")
    finally:
        p.close()


def test_dense_large_bf16_full_size():
    """The 3-layer Products-shaped model with bf16 transform operands, as bench.py
    runs its bf16 line: two batches of 1000 with affected sets bit for bit, then the
    sampled vertices (the 16 highest in-degrees among them) at every layer within
    R16's 2e-2 of the float64 oracle."""
    t0 = time.time()
    wl = synth.build_workload("dense_large")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights, undirected=True, gemm="bf16")
    try:
        _say(f"dense_large bf16: loaded + bootstrapped, oracle built ({time.time() - t0:.0f}s)")
        for b in range(2):
            st, _, sets = p.step(wl.stream.next_batch(1000))
            _say(f"  batch {b}: |A| = {[s.size for s in sets]}, dense layers {st['dense_layers']:b}, "
                 f"bucket layers {st['bucket_layers']:b} ({time.time() - t0:.0f}s)")
        verts, _ = _sample_vertices(np.random.default_rng(7), p.orc, sets[3], 24, 400_000)
        errs = _check_sampled(p, verts, (1, 2, 3), tol=FP32_TOL_BF16)
        _say(f"  {verts.size} sampled vertices, row-relative errors {errs} ({time.time() - t0:.0f}s)")
    finally:
        p.close()


@pytest.mark.parametrize("mode", ["auto", "pull", "dense"])
def test_stress_full_size(mode):
    """RMAT graph at full size (2^23 vertices, 200M arcs, GCN 64-256-64), one
    hub-biased batch of 10,000 ops, with the message forms the library chooses
    (as bench.py runs it) or forced: affected sets bit for bit, embeddings of
    sampled vertices (the 16 highest in-degrees among them) at both layers."""
    t0 = time.time()
    wl = synth.build_workload("stress")
    _say(f"stress generated in {time.time() - t0:.0f}s ({mode})")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights, mode=mode)
    try:
        _say(f"  loaded + bootstrapped, oracle built ({time.time() - t0:.0f}s)")
        st, _, sets = p.step(wl.stream.next_batch(10_000))
        if mode != "auto":
            assert st["pull_layers" if mode == "pull" else "dense_layers"] == 0b110
        _say(f"  batch: |A| = {[s.size for s in sets]}, pushed {st['pushed_arcs']}, pull {st['pull_layers']:b}, "
             f"dense {st['dense_layers']:b} ({time.time() - t0:.0f}s)")
        rng = np.random.default_rng(6)
        verts, _ = _sample_vertices(rng, p.orc, sets[2], 24, 2_000_000)
        errs = _check_sampled(p, verts, (1, 2))
        _say(f"  {verts.size} sampled vertices, row-relative errors {errs} ({time.time() - t0:.0f}s)")
    finally:
        p.close()

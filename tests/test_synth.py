"""The seeded input generators: reproducible, the shapes the workloads state,
and benchmark streams whose every op is effective."""
import numpy as np

from oracle import ripple_oracle as O
from paper_2505_12112_amd import synth


def test_same_seed_same_workload():
    a = synth.build_workload("tiny")
    b = synth.build_workload("tiny")
    np.testing.assert_array_equal(a.src, b.src)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.stream.next_batch(100).ops, b.stream.next_batch(100).ops)
    c = synth.build_workload("tiny", seed=1)
    assert not np.array_equal(a.src, c.src)


def test_tiny_shape_and_op_mix():
    w = synth.build_workload("tiny")
    assert w.src.size == 16000 and w.n == 2000 and w.x.shape == (2000, 16)
    assert np.all(w.src != w.dst)
    keys = w.src.astype(np.int64) * w.n + w.dst
    assert np.unique(keys).size == keys.size
    b = w.stream.next_batch(100)
    kinds = np.bincount(b.ops[:, 0], minlength=4)
    assert tuple(kinds[1:]) == (45, 45, 10)
    assert b.feat_rows.shape == (10, 16)
    assert w.weights.dims == (16, 16, 8) and w.weights.relu == [True, False]


def test_chung_lu_weights_cap_and_sum():
    w = synth.chung_lu_weights(10000, 80000.0, 2.1)
    assert abs(w.sum() - 80000.0) < 1e-6 * 80000
    assert abs(w.max() - np.sqrt(80000.0)) < 1e-6 * np.sqrt(80000.0)
    assert np.all(np.diff(w) <= 0)


def test_undirected_generation_lists_each_edge_once():
    spec = synth.GraphSpec("chung_lu", 3000, 20000, undirected=True)
    s, d, ps, pd = synth.generate_graph(spec, np.random.default_rng(0))
    assert s.size == 20000 and np.all(s < d)
    assert np.all(ps < pd)
    k = np.concatenate([s.astype(np.int64) * 3000 + d, ps.astype(np.int64) * 3000 + pd])
    assert np.unique(k).size == k.size


def test_benchmark_stream_ops_are_all_effective():
    spec = synth.dataclasses.replace(
        synth.CONFIGS["sparse_mid"], graph=synth.GraphSpec("chung_lu", 3000, 20000))
    w = synth.build_workload(spec)
    st = O.OracleState(w.n, w.src, w.dst, w.x, O.OracleModel.from_weights(w.weights))
    for _ in range(5):
        b = w.stream.next_batch(100)
        net, _ = st.apply(b.ops, b.feat_rows)
        kinds = np.bincount(b.ops[:, 0], minlength=4)
        assert net.ins_src.size == kinds[1] and net.del_src.size == kinds[2]
        assert net.noop_edge_ops == 0


def test_rmat_generator_small():
    spec = synth.GraphSpec("rmat", 1 << 10, 5000)
    s, d, _, _ = synth.generate_graph(spec, np.random.default_rng(0))
    assert s.size == 5000 and s.max() < 1024 and np.all(s != d)
    deg = np.bincount(s, minlength=1024)
    assert deg.max() > 8 * deg.mean()   # skewed

"""Test helpers: run the HIP library and the CPU oracle side by side on the same
seeded inputs and compare what they produce."""
from __future__ import annotations

import ctypes as C

import numpy as np

from oracle import ripple_oracle as O
from paper_2505_12112_amd import synth
from paper_2505_12112_amd.ripple import Ripple

FP32_TOL = 1e-4   # max row-relative error for the fp32 path


class DeviceCopy:
    """A host array copied into device memory (hipMalloc + hipMemcpy) through the
    HIP runtime the library itself runs on, so that tests need no other GPU
    framework; freed on exit. ptr is 0 for None or an empty array."""

    def __init__(self, arr):
        self.arr = arr
        self.ptr = 0

    def __enter__(self):
        if self.arr is not None and self.arr.nbytes:
            hip = _hip()
            p = C.c_void_p()
            if hip.hipMalloc(C.byref(p), C.c_size_t(self.arr.nbytes)) != 0:
                raise RuntimeError("hipMalloc failed")
            self.ptr = p.value
            if hip.hipMemcpy(C.c_void_p(self.ptr), self.arr.ctypes.data_as(C.c_void_p),
                             C.c_size_t(self.arr.nbytes), 1) != 0:  # host to device
                raise RuntimeError("hipMemcpy failed")
        return self

    def __exit__(self, *exc):
        if self.ptr:
            _hip().hipFree(C.c_void_p(self.ptr))
            self.ptr = 0
        return False


_HIP = None


def _hip():
    global _HIP
    if _HIP is None:
        _HIP = C.CDLL("libamdhip64.so.7")  # the runtime libripple.so is linked against
        _HIP.hipMalloc.argtypes = [C.POINTER(C.c_void_p), C.c_size_t]
        _HIP.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
        _HIP.hipFree.argtypes = [C.c_void_p]
        _HIP.hipStreamCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
        _HIP.hipStreamDestroy.argtypes = [C.c_void_p]
        _HIP.hipMemGetInfo.argtypes = [C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]
    return _HIP


def device_free_bytes() -> int:
    """Free device memory on the current device (hipMemGetInfo)."""
    free, total = C.c_size_t(), C.c_size_t()
    if _hip().hipMemGetInfo(C.byref(free), C.byref(total)) != 0:
        raise RuntimeError("hipMemGetInfo failed")
    return free.value


class CallerStream:
    """A stream the caller owns (hipStreamCreateWithFlags, default priority), for
    contexts that run on a stream they did not create; destroyed on exit."""

    def __enter__(self):
        p = C.c_void_p()
        if _hip().hipStreamCreateWithFlags(C.byref(p), 1) != 0:  # non-blocking
            raise RuntimeError("hipStreamCreateWithFlags failed")
        self.handle = p.value
        return self

    def __exit__(self, *exc):
        _hip().hipStreamDestroy(C.c_void_p(self.handle))
        return False


FP32_TOL_BF16 = 2e-2   # max row-relative error with bf16 transform operands
BF16_UNIT = 2.0 ** -8  # unit roundoff of bf16 (8 significand bits), rounded up


class Pair:
    def __init__(self, n, src, dst, x, weights, undirected=False, transform_first=-1, mode="auto", inputs="host",
                 edge_w=None, graphs=False, gemm="fp32", **lib_kw):
        self.lib = Ripple(n, src, dst, undirected=undirected, weights=edge_w, **lib_kw)
        self.lib.init_embeddings(x, weights, transform_first=transform_first, gemm=gemm)
        self.lib.set_scatter_mode(mode)
        self.lib.set_graphs(graphs)
        self.graphs = graphs  # batches replay captured HIP graphs, else kernels are queued one by one
        self.inputs = inputs  # "host": ripple_apply_updates; "device": the batch staged in HBM first
        self.orc = O.OracleState(n, src, dst, x, O.OracleModel.from_weights(weights), undirected, edge_w)
        self.L = len(weights.dims) - 1
        self.n = n

    def close(self):
        self.lib.close()

    def apply(self, ops, feat_rows):
        """The batch through the library, from host memory or staged in device memory."""
        if self.inputs == "host":
            return self.lib.apply_updates(ops, feat_rows)
        o = np.ascontiguousarray(np.asarray(ops, np.int32).reshape(-1, 4))
        f = None if feat_rows is None or len(feat_rows) == 0 else np.ascontiguousarray(feat_rows, np.float32)
        with DeviceCopy(o) as do, DeviceCopy(f) as df:
            return self.lib.apply_updates_device(do.ptr, o.shape[0], df.ptr, 0 if f is None else f.shape[0])

    def step(self, batch, check_sets=True, check_stats=True):
        st = self.apply(batch.ops, batch.feat_rows)
        net, sets = self.orc.apply(batch.ops, batch.feat_rows)
        if check_sets:
            for l in range(self.L + 1):
                got = self.lib.get_affected(l)
                np.testing.assert_array_equal(got, sets[l].astype(np.int32), err_msg=f"A^{l}")
        if check_stats:
            assert st["ins_arcs"] == net.ins_src.size
            assert st["del_arcs"] == net.del_src.size
            assert st["reweighted_arcs"] == net.rew_src.size
            assert st["graph_replay"] == int(self.graphs), "the batch did not run the way the test asked"
            assert st["features"] == net.features.size
            assert st["edge_keys"] == net.edge_keys
            assert st["noop_edge_ops"] == net.noop_edge_ops
            for l in range(self.L + 1):
                assert st["affected"][l] == sets[l].size
        return st, net, sets

    def embedding_errors(self):
        ref = self.orc.embeddings()
        return [O.row_relative_error(self.lib.get_embeddings(l), ref[l]) for l in range(self.L + 1)]

    def check_embeddings(self, tol=FP32_TOL):
        errs = self.embedding_errors()
        assert max(errs) <= tol, errs
        return errs

    def check_arcs(self):
        """The arc set in both directions, and on a weighted graph every arc's weight."""
        want = self.orc.graph.keys
        for direction in (0, 1):
            s, d = self.lib.get_arcs(direction)
            keys = s.astype(np.int64) * self.n + d
            order = np.argsort(keys)
            np.testing.assert_array_equal(keys[order], want, err_msg=f"direction {direction}")
            if self.orc.graph.w is not None:
                w = self.lib.get_arc_weights(direction)[order]
                np.testing.assert_array_equal(w.astype(np.float64), self.orc.graph.w, err_msg=f"weights {direction}")

    def check_aggregates(self, tol=FP32_TOL, drift_units=1024.0):
        """The library's cached aggregates against their definition on oracle values:
        S^l_v = sum over in-neighbours u of c_u h^{l-1}_u (c_u = 1, or 1/sqrt(dout+1) for GCN).

        S is a running sum of deltas, so a row whose true value cancels to ~0 keeps
        rounding residue of the order of the contributions that cancelled. Two
        measures: the error of each row against max(|S*_v|_inf, RMS(S*)) within tol,
        and, row by row without any floor, against the magnitude of the row's terms,
        max_k sum_u |c_u h_uk| (through |W_neigh| for rows cached transformed), within
        drift_units units of 2^-24: a row summed afresh is within about its in-degree
        of these units and each message added to it since can add about two, so this
        bounds the accumulated rounding of every row, cancelling ones included. (The
        magnitude is floored at a tenth of its RMS over the rows: a row that lost most
        of its in-arcs keeps the rounding of terms larger than its present ones.)"""
        ref = self.orc.embeddings()
        g = self.orc.graph
        c = np.ones(self.n)
        if self.orc.model.agg == "gcn":
            c = 1.0 / np.sqrt(g.out_degree() + 1.0)
        u, _ = g.arcs()
        a = g.in_adjacency(weights=c[u] * (g.w if self.orc.model.agg == "gc_wsum" else 1.0))
        errs = []
        for l in range(1, self.L + 1):
            want = a @ ref[l - 1]
            got = self.lib.get_aggregates(l).astype(np.float64)
            if got.shape[1] != want.shape[1]:   # cached transformed: W_neigh S
                want = want @ self.orc.model.w_neigh[l - 1].T
            rms = float(np.sqrt(np.mean(want * want))) + 1e-30
            num = np.max(np.abs(got - want), axis=1)
            den = np.maximum(np.max(np.abs(want), axis=1), rms)
            r = num / den
            worst = int(np.argmax(r))
            errs.append(float(r[worst]))
            assert r[worst] <= tol, (l, worst, float(num[worst]), float(np.max(np.abs(want[worst]))), rms)
            mag = abs(a) @ np.abs(ref[l - 1])
            if got.shape[1] != mag.shape[1]:
                mag = mag @ np.abs(self.orc.model.w_neigh[l - 1]).T
            m = np.max(mag, axis=1)
            scale = np.maximum(m, 0.1 * float(np.sqrt(np.mean(m * m)))) * 2.0 ** -24
            units = np.where(scale > 0, num / np.where(scale > 0, scale, 1.0), np.where(num > 0, np.inf, 0.0))
            w = int(np.argmax(units))
            assert units[w] <= drift_units, (l, w, float(units[w]), float(num[w]), float(scale[w]))
        return errs


def random_valid_batch(rng, orc: O.OracleState, bs: int, d0: int, mix=(1 / 3, 1 / 3, 1 / 3)) -> synth.Batch:
    """Effective ops against the oracle's current graph: inserts of absent arcs,
    deletes of present arcs, feature replacements (no two ops on one edge)."""
    g = orc.graph
    n = g.n
    kinds = rng.choice([1, 2, 3], bs, p=np.array(mix) / np.sum(mix))
    ops = np.full((bs, 4), -1, np.int32)
    used = set()
    nfeat = 0
    keys = g.keys
    for i, k in enumerate(kinds):
        ops[i, 0] = k
        if k == 3:
            ops[i, 1] = rng.integers(0, n)
            ops[i, 3] = nfeat
            nfeat += 1
            continue
        placed = False
        for _ in range(100):
            if k == 1:
                u, v = int(rng.integers(0, n)), int(rng.integers(0, n))
                if u == v:
                    continue
            else:
                if keys.size == 0:
                    break
                key = int(keys[rng.integers(0, keys.size)])
                u, v = key // n, key % n
            e = (min(u, v), max(u, v)) if g.undirected else (u, v)
            present = bool(g.has_arcs(np.array([u * n + v]))[0])
            if e in used or present != (k == 2):
                continue
            used.add(e)
            ops[i, 1], ops[i, 2] = u, v
            if k == 1 and g.w is not None:  # weighted graph: the new arc's weight
                ops[i, 3] = synth.weight_bits([rng.uniform(0.5, 1.5)])[0]
            placed = True
            break
        if not placed:
            ops[i] = (3, int(rng.integers(0, n)), -1, nfeat)
            nfeat += 1
    feats = rng.standard_normal((nfeat, d0), dtype=np.float32)
    return synth.Batch(ops, feats)


def fp32_forward_bound(orc: O.OracleState, ref, l: int, unit: float = 2.0 ** -24) -> np.ndarray:
    """Per row v of layer l: the forward error bound of evaluating the layer from
    exact inputs in arithmetic of unit roundoff `unit` (fp32 by default),
    2 (K + 16) unit max_k B_vk, where B_vk sums the magnitudes of every term of
    output k's pre-activation (|W_self| |h_v| + |W_neigh| sum_u |c_uv h_u| + |b|;
    GIN: through both layers of its MLP) and K is the length of the row's dot
    products."""
    m = orc.model
    habs = np.abs(ref[l - 1])
    aabs = O.aggregate(orc.graph, habs, m.agg)  # the coefficients are non-negative
    k = m.w_neigh[l - 1].shape[1]
    if m.agg == "gin":
        hidden = ((1.0 + m.gin_eps) * habs + aabs) @ np.abs(m.w_neigh[l - 1]).T + np.abs(m.bias[l - 1])
        b = hidden @ np.abs(m.w_out[l - 1]).T + np.abs(m.b_out[l - 1])
        k += m.w_out[l - 1].shape[1]
    else:
        b = aabs @ np.abs(m.w_neigh[l - 1]).T + np.abs(m.bias[l - 1])
        if m.w_self[l - 1] is not None:
            b = b + habs @ np.abs(m.w_self[l - 1]).T
            k *= 2
    return 2.0 * (k + 16) * unit * np.max(b, axis=1)


def check_embeddings_conditioned(pair: "Pair", tol=FP32_TOL, unit: float = 2.0 ** -24):
    """Every row of every layer meets R16 (max row-relative error tol, floor 1e-3
    RMS), or, where R16 asks for more than the arithmetic resolves (a row whose
    pre-activation cancels to far below the magnitude of its terms), lies within
    the forward error bound of its layer (fp32_forward_bound with that unit
    roundoff). Returns per layer (max R16 error, rows that needed the bound)."""
    ref = pair.orc.embeddings()
    out = []
    for l in range(1, pair.L + 1):
        got = pair.lib.get_embeddings(l).astype(np.float64)
        diff = np.max(np.abs(got - ref[l]), axis=1)
        floor = 1e-3 * float(np.sqrt(np.mean(ref[l] * ref[l])))
        r16 = diff / np.maximum(np.max(np.abs(ref[l]), axis=1), floor)
        bound = fp32_forward_bound(pair.orc, ref, l, unit)
        over = np.flatnonzero(r16 > tol)
        bad = over[diff[over] > bound[over]]
        assert bad.size == 0, (l, bad[:5], r16[bad[:5]], diff[bad[:5]], bound[bad[:5]])
        out.append((float(r16.max()), int(over.size)))
    return out


def aggregate_drift_ulps(pair: "Pair", rows) -> list:
    """How far the cached aggregate rows S^l_v of `rows` are from their definition
    sum_u c_u h*_u (float64, on the oracle's embeddings), in units of 2^-24 times the
    magnitude of the sum's terms, max_k sum_u |c_u h*_uk|: a fresh fp32 sum of the
    row is within about its in-degree of these units, and every message added since
    the row was last summed afresh can add half a unit. Per layer, the worst row."""
    ref = pair.orc.embeddings()
    g = pair.orc.graph
    c = np.ones(pair.n)
    if pair.orc.model.agg == "gcn":
        c = 1.0 / np.sqrt(g.out_degree() + 1.0)
    u, _ = g.arcs()
    a = g.in_adjacency(weights=c[u] * (g.w if pair.orc.model.agg == "gc_wsum" else 1.0))
    rows = np.asarray(rows, np.int64)
    out = []
    for l in range(1, pair.L + 1):
        want = (a @ ref[l - 1])[rows]
        mag = np.max((abs(a) @ np.abs(ref[l - 1]))[rows], axis=1)
        got = pair.lib.get_aggregates(l, rows.astype(np.int32)).astype(np.float64)
        err = np.max(np.abs(got - want), axis=1)
        out.append(float(np.max(err / (np.maximum(mag, 1e-300) * 2.0 ** -24))))
    return out

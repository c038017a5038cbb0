"""ctypes binding of libripple (the C ABI declared in include/ripple.h).

Argument marshalling only: every step of the incremental propagation runs in the
HIP library. Arrays are NumPy host arrays; the library copies them during each
call. If the library is not built, importing this module works but creating a
context raises ``RippleUnavailable`` (there is no fallback path).
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libripple.so")

MAX_LAYERS = 8
NUM_PHASES = 8

OK, E_INVALID, E_STATE, E_OOM, E_DEVICE = 0, 1, 2, 3, 4
AGG = {"sum": 0, "mean": 1, "gcn": 2, "gc_sum": 3, "gc_mean": 4, "gin": 5, "gc_wsum": 6}
GEMM = {"fp32": 0, "bf16": 1}
OP_INSERT, OP_DELETE, OP_FEATURE = 1, 2, 3
PHASES = ["net", "topo", "layer0", "scatter", "compact", "gemm", "other", "total"]

EXPORTED = [
    "ripple_load_graph", "ripple_init_embeddings", "ripple_apply_updates", "ripple_get_embeddings",
    "ripple_get_affected", "ripple_get_aggregates", "ripple_get_arcs", "ripple_device_bytes",
    "ripple_set_profiling", "ripple_get_phase_stats", "ripple_phase_name", "ripple_last_error",
    "ripple_destroy", "ripple_set_scatter_mode", "ripple_apply_updates_device", "ripple_get_arc_weights",
    "ripple_set_graphs", "ripple_set_reanchor", "ripple_get_embeddings_static",
]
SCATTER = {"auto": 0, "push": 1, "pull": 2, "dense": 3, "recompute": 4, "bucket": 5}


class RippleUnavailable(RuntimeError):
    pass


class RippleError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"[status {status}] {msg}")
        self.status = status


class GraphDesc(C.Structure):
    _fields_ = [
        ("num_vertices", C.c_int64), ("num_edges", C.c_int64),
        ("src", C.POINTER(C.c_int32)), ("dst", C.POINTER(C.c_int32)),
        ("undirected", C.c_int32), ("slack", C.c_float), ("min_slack", C.c_int32),
        ("device", C.c_int32), ("stream", C.c_void_p), ("max_device_bytes", C.c_int64),
        ("arena_slots", C.c_int64), ("weight", C.POINTER(C.c_float)),
    ]


class ModelDesc(C.Structure):
    _fields_ = [
        ("num_layers", C.c_int32), ("agg", C.c_int32), ("dims", C.POINTER(C.c_int32)),
        ("w_self", C.POINTER(C.POINTER(C.c_float))), ("w_neigh", C.POINTER(C.POINTER(C.c_float))),
        ("bias", C.POINTER(C.POINTER(C.c_float))), ("relu", C.POINTER(C.c_int32)),
        ("gemm_prec", C.c_int32), ("transform_first", C.c_int32),
        ("w_out", C.POINTER(C.POINTER(C.c_float))), ("b_out", C.POINTER(C.POINTER(C.c_float))),
        ("gin_eps", C.c_float), ("reserved", C.c_int32),
    ]


class BatchStats(C.Structure):
    _fields_ = [
        ("num_ops", C.c_int64), ("edge_keys", C.c_int64), ("noop_edge_ops", C.c_int64),
        ("ins_arcs", C.c_int64), ("del_arcs", C.c_int64), ("features", C.c_int64),
        ("dirty", C.c_int64 * (MAX_LAYERS + 1)), ("affected", C.c_int64 * (MAX_LAYERS + 1)),
        ("pushed_arcs", C.c_int64 * (MAX_LAYERS + 1)), ("dest_rows", C.c_int64 * (MAX_LAYERS + 1)),
        ("relocated_rows", C.c_int64), ("repacks", C.c_int64),
        ("in_arcs", C.c_int64 * (MAX_LAYERS + 1)), ("pull_layers", C.c_int32), ("dense_layers", C.c_int32),
        ("reweighted_arcs", C.c_int64), ("graph_replay", C.c_int64), ("long_rows", C.c_int64),
        ("recompute_layers", C.c_int32), ("bucket_layers", C.c_int32),
    ]


class PhaseStats(C.Structure):
    _fields_ = [("ms", C.c_double), ("launches", C.c_int64), ("bytes", C.c_double), ("flops", C.c_double),
                ("bytes_no_reuse", C.c_double)]


_lib = None


def load_library(path: str = LIB_PATH) -> C.CDLL:
    """Loads libripple.so once; raises RippleUnavailable if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RippleUnavailable(f"{path} is not built (run __graft_entry__.build())")
    lib = C.CDLL(path)
    P = C.POINTER
    vp = C.c_void_p
    lib.ripple_load_graph.argtypes = [P(GraphDesc), P(vp)]
    lib.ripple_init_embeddings.argtypes = [vp, P(C.c_float), P(ModelDesc)]
    lib.ripple_apply_updates.argtypes = [vp, P(C.c_int32), C.c_int64, P(C.c_float), C.c_int64, P(BatchStats)]
    lib.ripple_apply_updates_device.argtypes = [vp, vp, C.c_int64, vp, C.c_int64, P(BatchStats)]
    lib.ripple_get_embeddings.argtypes = [vp, C.c_int32, P(C.c_int32), C.c_int64, P(C.c_float)]
    lib.ripple_get_embeddings_static.argtypes = [vp, C.c_int32, P(C.c_int32), C.c_int64, P(C.c_float)]
    lib.ripple_get_aggregates.argtypes = [vp, C.c_int32, P(C.c_int32), C.c_int64, P(C.c_float), P(C.c_int32)]
    lib.ripple_get_affected.argtypes = [vp, C.c_int32, P(C.c_int32), C.c_int64, P(C.c_int64)]
    lib.ripple_get_arcs.argtypes = [vp, C.c_int32, P(C.c_int32), P(C.c_int32), C.c_int64, P(C.c_int64)]
    lib.ripple_get_arc_weights.argtypes = [vp, C.c_int32, P(C.c_float), C.c_int64, P(C.c_int64)]
    lib.ripple_device_bytes.argtypes = [vp, P(C.c_int64)]
    lib.ripple_set_profiling.argtypes = [vp, C.c_int32]
    lib.ripple_set_scatter_mode.argtypes = [vp, C.c_int32]
    lib.ripple_set_graphs.argtypes = [vp, C.c_int32]
    lib.ripple_set_reanchor.argtypes = [vp, C.c_int64]
    lib.ripple_get_phase_stats.argtypes = [vp, P(PhaseStats), C.c_int32]
    lib.ripple_phase_name.argtypes = [C.c_int32]
    lib.ripple_phase_name.restype = C.c_char_p
    lib.ripple_last_error.argtypes = [vp]
    lib.ripple_last_error.restype = C.c_char_p
    lib.ripple_destroy.argtypes = [vp]
    lib.ripple_destroy.restype = None
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray], ctype):
    if a is None:
        return None
    return a.ctypes.data_as(C.POINTER(ctype))


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


class Ripple:
    """One library context: graph + model state on one GPU."""

    def __init__(self, n: int, src, dst, undirected: bool = False, slack: float = 0.25,
                 min_slack: int = 4, device: int = 0, stream: Optional[int] = None,
                 max_device_bytes: int = 0, arena_slots: int = 0, weights=None):
        """weights: one float per edge for a weighted graph (RIPPLE_AGG_GC_WSUM), else None."""
        self._lib = load_library()
        self._ctx = C.c_void_p()
        src, dst = _i32(src), _i32(dst)
        if src.shape != dst.shape:
            raise ValueError("src and dst differ in length")
        w = None if weights is None else _f32(weights)
        if w is not None and w.shape != src.shape:
            raise ValueError("one weight per edge")
        desc = GraphDesc(int(n), int(src.size), _ptr(src, C.c_int32), _ptr(dst, C.c_int32),
                         int(bool(undirected)), float(slack), int(min_slack), int(device),
                         C.c_void_p(stream) if stream else None, int(max_device_bytes), int(arena_slots),
                         _ptr(w, C.c_float))
        st = self._lib.ripple_load_graph(C.byref(desc), C.byref(self._ctx))
        if st != OK:
            raise RippleError(st, self._lib.ripple_last_error(None).decode())
        self.n = int(n)
        self.undirected = bool(undirected)
        self.dims: List[int] = []
        self.num_layers = 0

    # -- helpers --
    def _check(self, st: int):
        if st != OK:
            raise RippleError(st, self._lib.ripple_last_error(self._ctx).decode())

    def close(self):
        if getattr(self, "_ctx", None) is not None and self._ctx.value:
            self._lib.ripple_destroy(self._ctx)
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- calls --
    def init_embeddings(self, x, weights, gemm: str = "fp32", transform_first: int = -1):
        """weights: object with agg, dims, w_self, w_neigh, bias, relu (and for GIN
        w_out, b_out, gin_eps), e.g. synth.ModelWeights. transform_first: -1 for
        layers that narrow (d_l < d_{l-1}), 0 never, 1 always (GraphSAGE and GCN)."""
        x = _f32(x)
        dims = _i32(weights.dims)
        L = len(dims) - 1
        keep = [x, dims]
        ws = (C.POINTER(C.c_float) * L)()
        wn = (C.POINTER(C.c_float) * L)()
        bs = (C.POINTER(C.c_float) * L)()
        for l in range(L):
            if weights.w_self[l] is not None:
                a = _f32(weights.w_self[l])
                keep.append(a)
                ws[l] = _ptr(a, C.c_float)
            a = _f32(weights.w_neigh[l])
            keep.append(a)
            wn[l] = _ptr(a, C.c_float)
            if weights.bias[l] is not None:
                b = _f32(weights.bias[l])
                keep.append(b)
                bs[l] = _ptr(b, C.c_float)
        relu = _i32([1 if r else 0 for r in weights.relu])
        keep.append(relu)
        wo = bo = None
        if getattr(weights, "w_out", None):  # GIN: the MLP's second layer
            wo = (C.POINTER(C.c_float) * L)()
            bo = (C.POINTER(C.c_float) * L)()
            for l in range(L):
                a = _f32(weights.w_out[l])
                keep.append(a)
                wo[l] = _ptr(a, C.c_float)
                if weights.b_out and weights.b_out[l] is not None:
                    b = _f32(weights.b_out[l])
                    keep.append(b)
                    bo[l] = _ptr(b, C.c_float)
        md = ModelDesc(L, AGG[weights.agg], _ptr(dims, C.c_int32), ws, wn, bs, _ptr(relu, C.c_int32),
                       GEMM[gemm], int(transform_first), wo, bo, float(getattr(weights, "gin_eps", 0.0)), 0)
        self._check(self._lib.ripple_init_embeddings(self._ctx, _ptr(x, C.c_float), C.byref(md)))
        self.dims = [int(d) for d in dims]
        self.num_layers = L

    def apply_updates(self, ops, feat_rows=None) -> Dict[str, object]:
        ops = _i32(ops).reshape(-1, 4)
        fr = None if feat_rows is None or len(feat_rows) == 0 else _f32(feat_rows)
        st = BatchStats()
        self._check(self._lib.ripple_apply_updates(
            self._ctx, _ptr(ops, C.c_int32), int(ops.shape[0]), _ptr(fr, C.c_float),
            0 if fr is None else int(fr.shape[0]), C.byref(st)))
        return self._stats_dict(st)

    def apply_updates_device(self, ops_ptr: int, num_ops: int, feat_ptr: int, num_feat_rows: int,
                             stats: Optional[BatchStats] = None) -> Dict[str, object]:
        """The batch already in device memory: ops_ptr -> int32 [num_ops, 4] and
        feat_ptr -> float32 [num_feat_rows, d_0] on the context's device (raw
        addresses, e.g. a torch tensor's data_ptr(); 0 for none)."""
        st = BatchStats() if stats is None else stats
        self._check(self._lib.ripple_apply_updates_device(
            self._ctx, C.c_void_p(ops_ptr or None), int(num_ops), C.c_void_p(feat_ptr or None),
            int(num_feat_rows), C.byref(st)))
        return st if stats is not None else self._stats_dict(st)

    def _stats_dict(self, st: BatchStats) -> Dict[str, object]:
        L = self.num_layers
        return {
            "num_ops": st.num_ops, "edge_keys": st.edge_keys, "noop_edge_ops": st.noop_edge_ops,
            "ins_arcs": st.ins_arcs, "del_arcs": st.del_arcs, "features": st.features,
            "dirty": list(st.dirty[:L + 1]), "affected": list(st.affected[:L + 1]),
            "pushed_arcs": list(st.pushed_arcs[:L + 1]), "dest_rows": list(st.dest_rows[:L + 1]),
            "relocated_rows": st.relocated_rows, "repacks": st.repacks,
            "in_arcs": list(st.in_arcs[:L + 1]), "pull_layers": st.pull_layers, "dense_layers": st.dense_layers,
            "reweighted_arcs": st.reweighted_arcs, "graph_replay": st.graph_replay, "long_rows": st.long_rows,
            "recompute_layers": st.recompute_layers,
            "bucket_layers": st.bucket_layers,
        }

    def apply_updates_raw(self, ops: np.ndarray, feat_rows: Optional[np.ndarray], stats: BatchStats) -> None:
        """Lowest-overhead form for timing loops: contiguous int32 [B,4] ops and
        float32 rows prepared by the caller; fills `stats` in place."""
        self._check(self._lib.ripple_apply_updates(
            self._ctx, ops.ctypes.data_as(C.POINTER(C.c_int32)), ops.shape[0],
            None if feat_rows is None else feat_rows.ctypes.data_as(C.POINTER(C.c_float)),
            0 if feat_rows is None else feat_rows.shape[0], C.byref(stats)))

    def get_embeddings(self, layer: int, ids: Optional[Sequence[int]] = None) -> np.ndarray:
        d = self.dims[layer]
        if ids is None:
            out = np.empty((self.n, d), np.float32)
            self._check(self._lib.ripple_get_embeddings(self._ctx, layer, None, self.n, _ptr(out, C.c_float)))
        else:
            ids = _i32(ids)
            out = np.empty((ids.size, d), np.float32)
            self._check(self._lib.ripple_get_embeddings(self._ctx, layer, _ptr(ids, C.c_int32), ids.size,
                                                        _ptr(out, C.c_float)))
        return out

    def get_embeddings_static(self, layer: int, ids: Optional[Sequence[int]] = None) -> np.ndarray:
        """As get_embeddings, through the library's fixed staging array (no device
        allocation); at most 32 MiB of ids and rows per call."""
        d = self.dims[layer]
        if ids is None:
            out = np.empty((self.n, d), np.float32)
            self._check(self._lib.ripple_get_embeddings_static(self._ctx, layer, None, self.n,
                                                               _ptr(out, C.c_float)))
        else:
            ids = _i32(ids)
            out = np.empty((ids.size, d), np.float32)
            self._check(self._lib.ripple_get_embeddings_static(self._ctx, layer, _ptr(ids, C.c_int32), ids.size,
                                                               _ptr(out, C.c_float)))
        return out

    def aggregate_width(self, layer: int) -> int:
        w = C.c_int32()
        self._check(self._lib.ripple_get_aggregates(self._ctx, layer, None, 0, None, C.byref(w)))
        return w.value

    def get_aggregates(self, layer: int, ids: Optional[Sequence[int]] = None) -> np.ndarray:
        """The cached aggregate rows of a layer: S (width d_{l-1}) or, for a
        transform-first layer, W_neigh S (width d_l)."""
        d = self.aggregate_width(layer)
        if ids is None:
            out = np.empty((self.n, d), np.float32)
            self._check(self._lib.ripple_get_aggregates(self._ctx, layer, None, self.n, _ptr(out, C.c_float), None))
        else:
            ids = _i32(ids)
            out = np.empty((ids.size, d), np.float32)
            self._check(self._lib.ripple_get_aggregates(self._ctx, layer, _ptr(ids, C.c_int32), ids.size,
                                                        _ptr(out, C.c_float), None))
        return out

    def get_affected(self, layer: int) -> np.ndarray:
        cnt = C.c_int64()
        self._check(self._lib.ripple_get_affected(self._ctx, layer, None, 0, C.byref(cnt)))
        out = np.empty(cnt.value, np.int32)
        if cnt.value:
            self._check(self._lib.ripple_get_affected(self._ctx, layer, _ptr(out, C.c_int32), out.size,
                                                      C.byref(cnt)))
        return out

    def get_arcs(self, direction: int = 0):
        cnt = C.c_int64()
        self._check(self._lib.ripple_get_arcs(self._ctx, direction, None, None, 0, C.byref(cnt)))
        s = np.empty(cnt.value, np.int32)
        d = np.empty(cnt.value, np.int32)
        if cnt.value:
            self._check(self._lib.ripple_get_arcs(self._ctx, direction, _ptr(s, C.c_int32), _ptr(d, C.c_int32),
                                                  s.size, C.byref(cnt)))
        return s, d

    def get_arc_weights(self, direction: int = 0) -> np.ndarray:
        """Weighted graphs: the arcs' weights in get_arcs order."""
        cnt = C.c_int64()
        self._check(self._lib.ripple_get_arc_weights(self._ctx, direction, None, 0, C.byref(cnt)))
        w = np.empty(cnt.value, np.float32)
        if cnt.value:
            self._check(self._lib.ripple_get_arc_weights(self._ctx, direction, _ptr(w, C.c_float), w.size,
                                                         C.byref(cnt)))
        return w

    def set_scatter_mode(self, mode: str):
        """"auto" (default), "push", "pull", "dense" or "recompute": how layers update
        their cached aggregates."""
        self._check(self._lib.ripple_set_scatter_mode(self._ctx, SCATTER[mode]))

    def set_reanchor(self, every: int):
        """Every `every`-th batch recomputes the affected aggregate rows afresh (0: never)."""
        self._check(self._lib.ripple_set_reanchor(self._ctx, int(every)))

    def set_graphs(self, enable: bool):
        """True: batches replay captured HIP graphs; False (default): kernels are queued one by one."""
        self._check(self._lib.ripple_set_graphs(self._ctx, 1 if enable else 0))

    def device_bytes(self) -> int:
        b = C.c_int64()
        self._check(self._lib.ripple_device_bytes(self._ctx, C.byref(b)))
        return b.value

    def set_profiling(self, phases=()):
        """Records HIP events around the named phases (see PHASES); () turns it off."""
        mask = 0
        for p in phases:
            mask |= 1 << PHASES.index(p)
        self._check(self._lib.ripple_set_profiling(self._ctx, mask))

    def phase_stats(self) -> Dict[str, Dict[str, float]]:
        arr = (PhaseStats * NUM_PHASES)()
        self._check(self._lib.ripple_get_phase_stats(self._ctx, arr, NUM_PHASES))
        return {PHASES[p]: {"ms": arr[p].ms, "launches": arr[p].launches, "bytes": arr[p].bytes,
                            "flops": arr[p].flops, "bytes_no_reuse": arr[p].bytes_no_reuse}
                for p in range(NUM_PHASES)}


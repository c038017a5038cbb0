#!/usr/bin/env python
"""Benchmark of the incremental propagation path on one MI355X.

One step = one ripple_apply_updates_device call: a batch of graph updates,
staged in HBM before the timed region, goes in, and the call returns when every
affected vertex's embeddings are updated. Default workload: ``sparse_mid``
(directed Chung-Lu power-law graph, 169,343 vertices, 1,166,243 arcs, 128
features, 2-layer GraphSAGE-sum 128-256-40), batches of 100 ops (each uniformly
an insert, a delete or a feature replacement).

Prints one JSON line: updates/sec over the timed steps (sum of ops / sum of the
host-timed call durations), the per-batch latency percentiles, the same rate for
batches handed over in host memory (PCIe-inclusive, beside the value), the
roofline of the dominant kernel phase (HIP events on the library's stream,
algorithmic bytes or flops per launch, HBM traffic from the committed counters),
and the CPU oracle timed on a bounded sample of the same stream on this host.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--batch B]
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
EVENT_EVERY = 10               # timed batches per batch with HIP events (roofline sample)
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="sparse_mid")
    ap.add_argument("--batch", type=int, default=100)
    ap.add_argument("--cpu-batches", type=int, default=5, help="oracle batches timed for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-events", action="store_true",
                    help="no HIP events in the timed region (the roofline then comes from the profiled pass)")
    ap.add_argument("--graphs", action="store_true",
                    help="replay captured HIP graphs instead of queueing every kernel on its own")
    ap.add_argument("--scatter-mode", default="auto", choices=["auto", "push", "pull", "dense"],
                    help="how every layer adds its messages (default: chosen per layer by the library)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-mebibyte device buffer into another (torch copy kernel), ten times: "
                         "the reference reading for the HBM byte counters")
    return ap.parse_args()


def percentile(xs, q):
    s = sorted(xs)
    if not s:
        return float("nan")
    k = (len(s) - 1) * q
    lo = int(k)
    hi = min(lo + 1, len(s) - 1)
    return s[lo] + (s[hi] - s[lo]) * (k - lo)


def cpu_baseline(wl_name, seed, batches, bs):
    """The oracle as it stands, in its float32 mode, on the first batches of the
    stream: apply the batch (with the affected sets), then recompute every layer
    over the whole graph. On graphs of more than 20M arcs one batch is timed and
    only its first layer is recomputed; the other layers are scaled from it by
    their share of the work (2 m d_{l-1} aggregation flops + 2 n K_l d_l GEMM
    flops per layer), which keeps the sample to tens of seconds."""
    import numpy as np
    from oracle import ripple_oracle as O
    from paper_2505_12112_amd import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    wl = synth.build_workload(wl_name, seed=seed)
    model = O.OracleModel.from_weights(wl.weights)
    st = O.OracleState(wl.n, wl.src, wl.dst, wl.x, model, wl.spec.graph.undirected, wl.edge_w)
    big = wl.src.size * (2 if wl.spec.graph.undirected else 1) > 20_000_000
    dims = list(wl.weights.dims)
    m = st.graph.num_arcs
    gcn = wl.spec.model.agg == "gcn"
    work = [2.0 * m * dims[l - 1] + 2.0 * wl.n * (1 if gcn else 2) * dims[l - 1] * dims[l]
            for l in range(1, len(dims))]
    times = []
    for b in batches[:1] if big else batches:
        t0 = time.perf_counter()
        st.apply(b.ops, b.feat_rows)
        if big:
            t1 = time.perf_counter()
            O.layer(st.graph, st.x.astype(np.float32), O.OracleModel.from_weights(model, np.float32), 1)
            t2 = time.perf_counter()
            times.append((t1 - t0) + (t2 - t1) * sum(work) / work[0])
        else:
            st.embeddings(np.float32)
            times.append(time.perf_counter() - t0)
    med = statistics.median(times)
    how = ("apply + first-layer float32 recompute over all vertices, scaled by the layers' work "
           f"({sum(work) / work[0]:.2f}x)" if big else "apply + full float32 layer-wise recompute")
    return {
        "value": bs / med,
        "unit": "updates/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "sample": (f"first {1 if big else len(batches)} batch(es) of {bs} ops of the {wl_name} stream; per batch: "
                   f"{how} (scipy sparse product, single thread; numpy BLAS, {blas_threads} threads), affected "
                   f"sets; median {med:.3f} s/batch; host has {len(os.sched_getaffinity(0))} cores available"),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU; --gpus must be 1 "
                          "(sharding over several GPUs is not implemented)"}))
        sys.exit(2)
    import numpy as np
    import torch
    if args.copy_calibration:
        n = args.copy_calibration * 2**20 // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(10):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": 4 * n, "copies": 10}))
        return
    from paper_2505_12112_amd import synth
    from paper_2505_12112_amd.ripple import Ripple, BatchStats
    from paper_2505_12112_amd.profiling import read_traffic

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    wl = synth.build_workload(args.config, seed=args.seed)
    spec = wl.spec
    log(f"[bench] generated {args.config}: n={wl.n} edges={wl.src.size} in {time.perf_counter() - t0:.1f}s")
    stream = torch.cuda.current_stream().cuda_stream
    lib = Ripple(wl.n, wl.src, wl.dst, undirected=spec.graph.undirected, device=0, stream=stream or None,
                 weights=wl.edge_w)
    lib.set_scatter_mode(args.scatter_mode)
    lib.set_graphs(args.graphs)
    t0 = time.perf_counter()
    lib.init_embeddings(wl.x, wl.weights)
    torch.cuda.synchronize()
    init_s = time.perf_counter() - t0
    log(f"[bench] bootstrap (all layers, all vertices) {init_s:.3f}s, device bytes {lib.device_bytes() / 2**30:.2f} GiB")

    K, W, bs = args.steps, args.warmup, args.batch
    batches = [wl.stream.next_batch(bs) for _ in range(W + K)]
    # every batch is staged in HBM before the timed region (ripple_apply_updates_device)
    staged = []
    for b in batches:
        o = torch.from_numpy(np.ascontiguousarray(b.ops, np.int32)).cuda()
        f = torch.from_numpy(np.ascontiguousarray(b.feat_rows, np.float32)).cuda() if b.feat_rows.shape[0] else None
        staged.append((o, f, o.data_ptr(), o.shape[0], 0 if f is None else f.data_ptr(),
                       0 if f is None else f.shape[0]))
    torch.cuda.synchronize()
    st = BatchStats()
    for _, _, op, no, fp, nf in staged[:W]:
        lib.apply_updates_device(op, no, fp, nf, st)
    torch.cuda.synchronize()
    log(f"[bench] {W} warm-up batches done")

    # timed region: HIP events around the two rooflined kernel phases on every
    # EVENT_EVERY-th batch (each batch with events pays a few microseconds for them)
    lib.set_profiling(())
    lib.phase_stats()  # reset sums
    L = len(wl.weights.dims) - 1
    lat = []
    aff = np.zeros(L + 1)
    pushed = np.zeros(L + 1)
    in_arcs = np.zeros(L + 1)
    pull_layers = dense_layers = 0
    repacks = relocated = 0
    replays = 0
    # the Python collector stays out of the timed region (a full collection with
    # torch loaded takes tens of milliseconds and is not the library's work)
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t_region = time.perf_counter()
    for i, (_, _, op, no, fp, nf) in enumerate(staged[W:]):
        sample = not args.no_events and i % EVENT_EVERY == 0
        if sample:
            lib.set_profiling(("scatter", "gemm"))
        t1 = time.perf_counter()
        lib.apply_updates_device(op, no, fp, nf, st)
        lat.append(time.perf_counter() - t1)
        if sample:
            lib.set_profiling(())
        aff += np.array(st.affected[:L + 1], dtype=np.float64)
        pushed += np.array(st.pushed_arcs[:L + 1], dtype=np.float64)
        in_arcs += np.array(st.in_arcs[:L + 1], dtype=np.float64)
        pull_layers |= st.pull_layers
        dense_layers |= st.dense_layers
        repacks += st.repacks
        relocated += st.relocated_rows
        replays += st.graph_replay
    torch.cuda.synchronize()
    region_s = time.perf_counter() - t_region
    gc.enable()
    ph = lib.phase_stats()
    log(f"[bench] {K} timed batches in {region_s:.3f}s")

    # the same number of further batches handed over from host memory (the
    # kernels then read ops and feature rows over PCIe): reported beside the value
    host_batches = [wl.stream.next_batch(bs) for _ in range(K)]
    host_prepared = [(np.ascontiguousarray(b.ops, np.int32),
                      np.ascontiguousarray(b.feat_rows, np.float32) if b.feat_rows.shape[0] else None)
                     for b in host_batches]
    host_lat = []
    gc.collect()
    gc.disable()
    for ops, fr in host_prepared:
        t1 = time.perf_counter()
        lib.apply_updates_raw(ops, fr, st)
        host_lat.append(time.perf_counter() - t1)
    gc.enable()

    # a second, untimed pass with every phase recorded, for the breakdown
    extra = [wl.stream.next_batch(bs) for _ in range(min(K, 50))]
    lib.set_profiling(tuple(["net", "topo", "layer0", "scatter", "compact", "gemm", "other", "total"]))
    lib.phase_stats()
    for b in extra:
        lib.apply_updates(b.ops, b.feat_rows)
    breakdown = lib.phase_stats()
    lib.set_profiling(())
    nb = len(extra)
    if args.no_events:
        ph = breakdown

    value = K * bs / sum(lat)
    ms_per_step = 1000.0 * sum(lat) / K

    workload_key = f"{args.config}_b{bs}"

    def roof(name):
        p = ph[name]
        if p["launches"] == 0 or p["ms"] <= 0:
            return None
        # HBM bytes per launch from the committed rocprofv3 counters (null when the
        # kernels changed since they were taken)
        traffic = read_traffic(workload_key, name)
        common = {"traffic": traffic, "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, "
                  "calibrated on a plain copy)", "launches": p["launches"],
                  "avg_launch_us": 1000.0 * p["ms"] / p["launches"]}
        if name == "gemm":
            ach = p["flops"] / (p["ms"] * 1e-3) / 1e12
            return {"kernel": "k_gemm (gather + fp32 MFMA + epilogue)", "bound": "mfma", "achieved": ach,
                    "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": ach / FP32_MFMA_PEAK_TFLOPS,
                    "algorithmic_per_launch": p["flops"] / p["launches"], **common}
        ach = p["bytes"] / (p["ms"] * 1e-3) / 1e9
        return {"kernel": "k_scatter / k_pull_msgs (message step)", "bound": "hbm", "achieved": ach,
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
                "algorithmic_per_launch": p["bytes"] / p["launches"],
                "no_reuse_per_launch": p["bytes_no_reuse"] / p["launches"],
                "bytes_note": "algorithmic: each message row read once, each sink row of S read and written once; "
                              "no_reuse: a message row read per arc that carries it (and, pushed, a row of atomics "
                              "per arc); the counters' traffic falls between the two by the L2 / MALL reuse",
                **common}

    r_scatter, r_gemm = roof("scatter"), roof("gemm")
    dominant = "gemm" if ph["gemm"]["ms"] >= ph["scatter"]["ms"] else "scatter"
    roofline = r_gemm if dominant == "gemm" else r_scatter
    other = r_scatter if dominant == "gemm" else r_gemm

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the CPU oracle on {args.cpu_batches} batches")
        cpu = cpu_baseline(args.config, args.seed, batches[:args.cpu_batches], bs)
        log(f"[bench] oracle {cpu['value']:.1f} updates/s")

    g = spec.graph
    out = {
        "metric": "updates/sec at batch 100 + p50 batch latency; % HBM peak in scatter",
        "value": value,
        "unit": "updates/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": args.config,
            "graph": f"{g.kind}{' undirected' if g.undirected else ''}, n={g.n}, edges={g.m}",
            "layers": list(spec.model.dims),
            "aggregator": spec.model.agg,
            "batch": bs,
            "op_mix": list(spec.stream.mix),
        },
        "latency_ms": {"p50": 1000 * percentile(lat, 0.5), "p90": 1000 * percentile(lat, 0.9),
                       "p99": 1000 * percentile(lat, 0.99), "mean": 1000 * statistics.mean(lat)},
        "inputs": "ops and feature rows resident in HBM before each timed call (ripple_apply_updates_device)",
        "host_inputs": {"value": K * bs / sum(host_lat), "p50_ms": 1000 * percentile(host_lat, 0.5),
                        "note": "further batches handed over in host memory (ripple_apply_updates; the kernels "
                                "read them over PCIe): the PCIe-inclusive rate, not the value"},
        "roofline": roofline,
        "roofline_other": other,
        "cpu_baseline": cpu,
        "frontier_mean": {"affected": (aff / K).tolist(), "pushed_arcs": (pushed / K).tolist(),
                          "in_arcs_of_affected": (in_arcs / K).tolist(),
                          "affected_frac": (aff / K / wl.n).tolist()},
        "message_form": {"mode": args.scatter_mode, "pull_layers_seen": pull_layers,
                         "dense_layers_seen": dense_layers},
        "adjacency": {"rows_moved": int(relocated), "relayouts": int(repacks)},
        "launch": {"graph_replays": int(replays), "direct": K - int(replays),
                   "note": "graph replays (--graphs): one captured HIP graph per launch plan; the "
                           "event-sampled batches queue their kernels one by one"},
        "max_latency_ms": 1000 * max(lat),
        "max_latency_batch": int(np.argmax(lat)),
        "phase_ms_per_batch": {k: v["ms"] / nb for k, v in breakdown.items()},
        "bootstrap_s": init_s,
        "device_gib": lib.device_bytes() / 2**30,
        "paper_context": "Ripple (CPU, 16-core Xeon Gold, real ogbn-arxiv, best over 5 workloads and "
                         "batch sizes 1..1000): about 28,000 updates/s",
    }
    lib.close()
    print(json.dumps(out))


if __name__ == "__main__":
    main()

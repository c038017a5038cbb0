#!/usr/bin/env python
"""Benchmark of the incremental propagation path on one MI355X.

One step = one ripple_apply_updates_device call: a batch of graph updates,
staged in HBM before the timed region, goes in, and the call returns when every
affected vertex's embeddings are updated. Default workload: ``sparse_mid``
(directed Chung-Lu power-law graph, 169,343 vertices, 1,166,243 arcs, 128
features, 2-layer GraphSAGE-sum 128-256-40), batches of 100 ops (each uniformly
an insert, a delete or a feature replacement).

Prints one JSON line:
* value: updates/sec over the timed steps (sum of ops / sum of the host-timed
  call durations; nothing else runs in the timed region), p50/p90/p99 latency;
* host_inputs: the same rate for batches handed over in host memory (the
  PCIe-inclusive rate, beside the value, never the value);
* roofline: the dominant kernel phase of the same workload, from an untimed
  profiled pass in which every kernel of the message and transform phases is
  launched with kernel-only start / stop events (hipExtLaunchKernelGGL), as a
  profiler's kernel trace measures it: algorithmic bytes (or flops) per launch
  over the average kernel duration, against the MI355X peak;
* scatter_large: the message step on the Products-shaped dense_large workload at
  batch 100 (where the scatter moves more than 1 GB per batch), measured the same
  way;
* cpu_baseline: the CPU oracle timed on a bounded sample of the same stream on
  this host.

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
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix
PROFILED_BATCHES = 60          # untimed batches whose kernels are timed for the roofline


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="sparse_mid")
    ap.add_argument("--batch", type=int, default=100)
    ap.add_argument("--gemm", default="fp32", choices=["fp32", "bf16"],
                    help="precision of the transform's operands (bf16: 2e-2 tolerance path)")
    ap.add_argument("--cpu-batches", type=int, default=5, help="oracle batches timed for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--large-config", default="dense_large",
                    help="workload of the scatter_large measurement ('none' to skip)")
    ap.add_argument("--large-batch", type=int, default=100)
    ap.add_argument("--large-batches", type=int, default=30, help="profiled batches of the scatter_large workload")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--graphs", action="store_true",
                    help="replay captured HIP graphs instead of queueing every kernel on its own")
    ap.add_argument("--scatter-mode", default="auto", choices=["auto", "push", "pull", "dense", "recompute", "bucket"],
                    help="how every layer updates its cached aggregates (default: chosen per layer by the library)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-mebibyte device buffer into another (torch copy kernel), ten times: "
                         "the reference reading for the HBM byte counters")
    ap.add_argument("--gather-calibration", type=int, default=0, metavar="MIB",
                    help="only gather every 192-byte row of a MIB-mebibyte table once, in random order (torch "
                         "index_select), ten times: checks the byte counters' scale on random row reads")
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


def stage(batches, torch, np):
    """Each batch's ops and feature rows copied into HBM (before any timed region)."""
    staged = []
    for b in batches:
        o = torch.from_numpy(np.ascontiguousarray(b.ops, np.int32)).cuda()
        f = torch.from_numpy(np.ascontiguousarray(b.feat_rows, np.float32)).cuda() if b.feat_rows.shape[0] else None
        staged.append((o, f, o.data_ptr(), o.shape[0], 0 if f is None else f.data_ptr(),
                       0 if f is None else f.shape[0]))
    return staged


def open_workload(name, seed, torch, scatter_mode, graphs, gemm):
    from paper_2505_12112_amd import synth
    from paper_2505_12112_amd.ripple import Ripple
    t0 = time.perf_counter()
    wl = synth.build_workload(name, seed=seed)
    log(f"[bench] generated {name}: n={wl.n} edges={wl.src.size} in {time.perf_counter() - t0:.1f}s")
    stream = torch.cuda.current_stream().cuda_stream
    lib = Ripple(wl.n, wl.src, wl.dst, undirected=wl.spec.graph.undirected, device=0, stream=stream or None,
                 weights=wl.edge_w)
    lib.set_scatter_mode(scatter_mode)
    lib.set_graphs(graphs)
    t0 = time.perf_counter()
    lib.init_embeddings(wl.x, wl.weights, gemm=gemm)
    torch.cuda.synchronize()
    init_s = time.perf_counter() - t0
    log(f"[bench] {name}: bootstrap (all layers, all vertices) {init_s:.3f}s, "
        f"device bytes {lib.device_bytes() / 2**30:.2f} GiB")
    return wl, lib, init_s


def profiled(lib, staged, phases):
    """Runs the staged batches with kernel timing of `phases` (untimed pass);
    returns the phase sums and the batches' stats."""
    from paper_2505_12112_amd.ripple import BatchStats
    lib.set_profiling(phases)
    lib.phase_stats()  # reset the sums
    st = BatchStats()
    modes = {"pull": 0, "dense": 0, "recompute": 0, "bucket": 0}
    for _, _, op, no, fp, nf in staged:
        lib.apply_updates_device(op, no, fp, nf, st)
        modes["pull"] |= st.pull_layers
        modes["dense"] |= st.dense_layers
        modes["recompute"] |= st.recompute_layers
        modes["bucket"] |= st.bucket_layers
    ph = lib.phase_stats()
    lib.set_profiling(())
    return ph, modes


def roof(p, name, traffic, peak_tflops, gemm_label):
    """Roofline of a phase from its kernel-timed sums: algorithmic work per launch
    over the average kernel duration."""
    if p["launches"] == 0 or p["ms"] <= 0:
        return None
    avg_s = p["ms"] * 1e-3 / p["launches"]
    common = {"launches": p["launches"], "avg_launch_us": 1e6 * avg_s,
              "timing": "kernel-only durations (hipExtLaunchKernelGGL start / stop events) of every launch of the "
                        "phase over an untimed profiled pass",
              "traffic": traffic,
              "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE in separate runs, "
                              "calibrated on a plain copy); null when the kernels changed since they were taken"}
    if name == "gemm":
        per = p["flops"] / p["launches"]
        ach = per / avg_s / 1e12
        return {"kernel": gemm_label, "bound": "mfma", "achieved": ach, "peak": peak_tflops, "unit": "TFLOP/s",
                "frac": ach / peak_tflops, "algorithmic_per_launch": per, **common}
    per = p["bytes"] / p["launches"]
    ach = per / avg_s / 1e9
    return {"kernel": "k_scatter / k_pull_msgs / k_recompute / k_bin_arcs / k_bin_sort / k_bucket_sum (message step)", "bound": "hbm", "achieved": ach,
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS, "algorithmic_per_launch": per,
            "no_reuse_per_launch": p["bytes_no_reuse"] / p["launches"],
            "bytes_note": "algorithmic: each message row read once, each sink row of S read and written once (each "
                          "source row once under recompute); no_reuse: a message row read per arc that carries it "
                          "(and, pushed, a row of atomics per arc)",
            **common}


def scatter_large(args, torch, np):
    """The message step on the large workload at its batch size: warm-up batches,
    then profiled batches with every scatter and transform kernel timed."""
    from paper_2505_12112_amd.profiling import read_traffic
    wl, lib, _ = open_workload(args.large_config, args.seed, torch, "auto", False, args.gemm)
    try:
        bs = args.large_batch
        warm = stage([wl.stream.next_batch(bs) for _ in range(10)], torch, np)
        for _, _, op, no, fp, nf in warm:
            lib.apply_updates_device(op, no, fp, nf)
        meas = stage([wl.stream.next_batch(bs) for _ in range(args.large_batches)], torch, np)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ph, modes = profiled(lib, meas, ("scatter", "gemm", "total"))
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        key = f"{args.large_config}_b{bs}"
        r = roof(ph["scatter"], "scatter", read_traffic(key, "scatter"), None, None)
        g = roof(ph["gemm"], "gemm", read_traffic(key, "gemm"),
                 BF16_MFMA_PEAK_TFLOPS if args.gemm == "bf16" else FP32_MFMA_PEAK_TFLOPS,
                 f"k_gemm (gather + {args.gemm} MFMA + epilogue)")
        if r is None:
            return None
        r.update({"workload": args.large_config, "batch": bs, "batches": args.large_batches,
                  "message_forms_seen": modes, "gemm": g,
                  "batch_ms_mean": ph["total"]["ms"] / max(1, ph["total"]["launches"]),
                  "updates_per_s_profiled": args.large_batches * bs / wall,
                  "note": "profiled batches (kernels timed one by one); context, not the value"})
        return r
    finally:
        lib.close()


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
    if args.gather_calibration:
        rows = args.gather_calibration * 2**20 // 192
        table = torch.ones(rows, 48, dtype=torch.float32, device="cuda")
        perm = torch.randperm(rows, device="cuda")
        out = torch.empty_like(table)
        for _ in range(10):
            torch.index_select(table, 0, perm, out=out)
        torch.cuda.synchronize()
        print(json.dumps({"gather_calibration_rows": rows, "row_bytes": 192, "index_bytes": 8, "gathers": 10}))
        return
    from paper_2505_12112_amd.ripple import BatchStats
    from paper_2505_12112_amd.profiling import read_traffic

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl, lib, init_s = open_workload(args.config, args.seed, torch, args.scatter_mode, args.graphs, args.gemm)
    spec = wl.spec
    K, W, bs = args.steps, args.warmup, args.batch
    batches = [wl.stream.next_batch(bs) for _ in range(W + K)]
    staged = stage(batches, torch, np)  # every batch staged in HBM before the timed region
    torch.cuda.synchronize()
    st = BatchStats()
    for _, _, op, no, fp, nf in staged[:W]:
        lib.apply_updates_device(op, no, fp, nf, st)
    torch.cuda.synchronize()
    log(f"[bench] {W} warm-up batches done")

    # timed region: the calls and nothing else (the stats are read after it)
    L = len(wl.weights.dims) - 1
    stats = [BatchStats() for _ in range(K)]
    lat = []
    gc.collect()
    gc.disable()  # a full collection with torch loaded takes tens of milliseconds
    torch.cuda.synchronize()
    t_region = time.perf_counter()
    for i, (_, _, op, no, fp, nf) in enumerate(staged[W:]):
        t1 = time.perf_counter()
        lib.apply_updates_device(op, no, fp, nf, stats[i])
        lat.append(time.perf_counter() - t1)
    torch.cuda.synchronize()
    region_s = time.perf_counter() - t_region
    gc.enable()
    log(f"[bench] {K} timed batches in {region_s:.3f}s")
    aff = np.array([s.affected[:L + 1] for s in stats], np.float64).mean(0)
    pushed = np.array([s.pushed_arcs[:L + 1] for s in stats], np.float64).mean(0)
    in_arcs = np.array([s.in_arcs[:L + 1] for s in stats], np.float64).mean(0)
    forms = {"pull": 0, "dense": 0, "recompute": 0, "bucket": 0}
    for s in stats:
        forms["pull"] |= s.pull_layers
        forms["dense"] |= s.dense_layers
        forms["recompute"] |= s.recompute_layers
        forms["bucket"] |= s.bucket_layers
    replays = sum(s.graph_replay for s in stats)
    relocated = sum(s.relocated_rows for s in stats)
    repacks = sum(s.repacks for s in stats)

    # the same number of further batches handed over from host memory (the
    # kernels then read ops and feature rows over PCIe): reported beside the value
    host_prepared = [(np.ascontiguousarray(b.ops, np.int32),
                      np.ascontiguousarray(b.feat_rows, np.float32) if b.feat_rows.shape[0] else None)
                     for b in (wl.stream.next_batch(bs) for _ in range(K))]
    host_lat = []
    gc.collect()
    gc.disable()
    for ops, fr in host_prepared:
        t1 = time.perf_counter()
        lib.apply_updates_raw(ops, fr, st)
        host_lat.append(time.perf_counter() - t1)
    gc.enable()

    # untimed profiled pass: every kernel of every phase timed on its own
    prof_staged = stage([wl.stream.next_batch(bs) for _ in range(PROFILED_BATCHES)], torch, np)
    ph, _ = profiled(lib, prof_staged, ("net", "topo", "layer0", "scatter", "compact", "gemm", "other", "total"))
    nb = len(prof_staged)
    key = f"{args.config}_b{bs}"
    gemm_peak = BF16_MFMA_PEAK_TFLOPS if args.gemm == "bf16" else FP32_MFMA_PEAK_TFLOPS
    r_scatter = roof(ph["scatter"], "scatter", read_traffic(key, "scatter"), None, None)
    r_gemm = roof(ph["gemm"], "gemm", read_traffic(key, "gemm"), gemm_peak,
                  f"k_gemm_rows / k_gemm (gather + {args.gemm} MFMA + epilogue)")
    dominant = "gemm" if ph["gemm"]["ms"] >= ph["scatter"]["ms"] else "scatter"
    roofline = r_gemm if dominant == "gemm" else r_scatter
    other = r_scatter if dominant == "gemm" else r_gemm
    device_gib = lib.device_bytes() / 2**30
    lib.close()
    del staged, prof_staged
    torch.cuda.synchronize()

    large = None
    if args.large_config != "none":
        log(f"[bench] scatter_large on {args.large_config} at batch {args.large_batch}")
        large = scatter_large(args, torch, np)

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the CPU oracle on {args.cpu_batches} batches")
        cpu = cpu_baseline(args.config, args.seed, batches[:args.cpu_batches], bs)
        log(f"[bench] oracle {cpu['value']:.1f} updates/s")

    value = K * bs / sum(lat)
    g = spec.graph
    out = {
        "metric": "updates/sec at batch 100 + p50 batch latency; % HBM peak in scatter",
        "value": value,
        "unit": "updates/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": 1000.0 * sum(lat) / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.gemm == "fp32" else "f32 (bf16 transform operands)",
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
                       "p99": 1000 * percentile(lat, 0.99), "mean": 1000 * statistics.mean(lat),
                       "max": 1000 * max(lat)},
        "inputs": "value: ops and feature rows resident in HBM before each timed call (ripple_apply_updates_device)",
        "host_inputs": {"value": K * bs / sum(host_lat), "p50_ms": 1000 * percentile(host_lat, 0.5),
                        "note": "further batches handed over in host memory (ripple_apply_updates; the kernels "
                                "read them over PCIe): the PCIe-inclusive rate, not the value"},
        "roofline": roofline,
        "roofline_other": other,
        "scatter_large": large,
        "cpu_baseline": cpu,
        "frontier_mean": {"affected": aff.tolist(), "pushed_arcs": pushed.tolist(),
                          "in_arcs_of_affected": in_arcs.tolist(), "affected_frac": (aff / wl.n).tolist()},
        "message_form": {"mode": args.scatter_mode, "layers_seen": forms},
        "adjacency": {"rows_moved": int(relocated), "relayouts": int(repacks)},
        "launch": {"graph_replays": int(replays), "direct": K - int(replays)},
        "phase_kernel_ms_per_batch": {k: v["ms"] / nb for k, v in ph.items()},
        "bootstrap_s": init_s,
        "device_gib": device_gib,
        "paper_context": "Ripple (CPU, 16-core Xeon Gold, real ogbn-arxiv, best over 5 workloads and "
                         "batch sizes 1..1000): about 28,000 updates/s",
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()

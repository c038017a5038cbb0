"""Summaries of rocprofv3 output for the committed profiles, and the HBM traffic
figures bench.py reports beside its roofline.

Inputs, all CSV as rocprofv3 writes them with --output-format csv:

* a kernel-trace statistics file (``*_kernel_stats.csv``) and trace
  (``*_kernel_trace.csv``): calls and durations per kernel, per-batch kernel time;
* counter-collection files (``*_counter_collection.csv``): the L2-to-fabric read
  requests by size (TCC_EA0_RDREQ_32B / _64B / _128B) in one run and the write
  requests (TCC_EA0_WRREQ, _64B) in another, each request counted at its size; the
  MFMA counters; and, for the calibration note, FETCH_SIZE and WRITE_SIZE.

The derived FETCH_SIZE counts 128-byte read requests as 64 bytes on this chip (its
formula takes them from TCC_BUBBLE); counting requests at their sizes reads a plain
copy exactly, which the traffic table checks (``bench.py --copy-calibration MIB``).

The traffic table carries a hash of the HIP sources it was measured on; bench.py
reports the figures only while the sources still hash the same (a changed kernel
makes them stale, and then the field is null).

    python -m paper_2505_12112_amd.profiling stats TRACE_DIR TITLE COMMAND > profiles/x.txt
    python -m paper_2505_12112_amd.profiling traffic-sized OUT.md COPY_MIB COPY_RD COPY_WR WORKLOAD=RD,WR,BATCHES,CMD ...
    python -m paper_2505_12112_amd.profiling mfma OUT.md TITLE NAME=DIR,DTYPE,CMD ...
    python -m paper_2505_12112_amd.profiling calibration OUT.md COPY_MIB GATHER_MIB KEY=DIR ... COMMANDS
    python -m paper_2505_12112_amd.profiling traffic OUT.md COPY_MIB COPY_F COPY_W WORKLOAD=F_DIR,W_DIR,BATCHES,CMD ...
      (the FETCH_SIZE / WRITE_SIZE form, scaled by what they read for a copy)
"""
from __future__ import annotations

import csv
import glob
import hashlib
import os
import re
import sys
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TRAFFIC_MD = os.path.join(ROOT, "profiles", "hbm_traffic_counters.md")

# kernels whose launches make up each rooflined phase of bench.py
PHASE_KERNELS = {"scatter": ("k_scatter", "k_pull_msgs", "k_recompute", "k_bin_arcs", "k_bin_sort", "k_bucket_sum"),
                 "gemm": ("k_gemm",)}


def code_only(text: str) -> str:
    """C/C++ source without its comments, whitespace runs collapsed to one space
    (string and character literals kept as written)."""
    parts = []  # code runs (whitespace collapsed) and literals (kept)
    code = []
    i, n = 0, len(text)
    while i < n:
        c = text[i]
        if c == "/" and text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
            continue
        if c == "/" and text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            code.append(" ")
            continue
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            parts.append(" ".join("".join(code).split()))
            parts.append(text[i:j + 1])
            code = []
            i = j + 1
            continue
        code.append(c)
        i += 1
    parts.append(" ".join("".join(code).split()))
    return " ".join(p for p in parts if p)


def source_hash() -> str:
    """sha256 over the code of the HIP sources and headers the library is built from
    (comments and layout do not change it)."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")) + glob.glob(os.path.join(HERE, "csrc", "*.h"))
                   + [os.path.join(ROOT, "include", "ripple.h")])
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8") as fh:
            h.update(code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def kernel_name(full: str) -> str:
    m = re.search(r"(k_\w+(<[^>]*>)?)", full)
    return m.group(1) if m else full.split("(")[0][:48]


def _one(dirpath: str, pattern: str) -> str:
    hits = sorted(glob.glob(os.path.join(dirpath, "**", pattern), recursive=True))
    if not hits:
        raise FileNotFoundError(f"no {pattern} under {dirpath}")
    return hits[0]


NETTING = ("k_net_hash", "k_net_direct", "k_net_decide")


def workload_segments(trace_dir: str):
    """Splits a kernel trace into the workloads one process ran: a segment starts at
    a bootstrap (k_pull) dispatch that follows update batches. Returns, per segment,
    the per-batch kernel time (netting kernel to netting kernel, the netting
    kernels of one batch counted together) and each phase's dispatch durations
    over the segment's batches."""
    rows = list(csv.DictReader(open(_one(trace_dir, "*kernel_trace.csv"))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    segs, cur, seen_batch, prev = [], None, False, ""
    for r in rows:
        k = kernel_name(r["Kernel_Name"])
        ns = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        if k.startswith("k_pull<") and (cur is None or seen_batch):
            cur = {"batches": [], "phases": defaultdict(list)}
            segs.append(cur)
            seen_batch = False
        last, prev = prev, k
        if cur is None:
            continue
        if k in NETTING and last not in NETTING:  # a batch's netting kernels run back to back
            cur["batches"].append([0, k])
            seen_batch = True
        if not cur["batches"]:
            continue
        cur["batches"][-1][0] += ns
        for ph, prefixes in PHASE_KERNELS.items():
            if k.startswith(prefixes):
                cur["phases"][ph].append(ns)
    return segs


def stats_table(trace_dir: str, title: str, command: str, top: int = 24) -> str:
    rows = list(csv.DictReader(open(_one(trace_dir, "*kernel_stats.csv"))))
    out = [f"# {title}", "", f"command: {command}", "",
           " calls     avg_us     min_us     max_us   total_ms    pct  kernel"]
    for r in rows[:top]:
        out.append(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.2f} {int(r['MinNs']) / 1e3:10.2f} "
                   f"{int(r['MaxNs']) / 1e3:10.2f} {float(r['TotalDurationNs']) / 1e6:10.3f} "
                   f"{float(r['Percentage']):6.2f}  {kernel_name(r['Name'])}")
    segs = workload_segments(trace_dir)
    if segs:
        out += ["", "Per workload the process ran (in order), over its update batches (bootstrap left out):",
                "kernel time per batch (first batch, median of the rest) and the average dispatch of each "
                "rooflined phase (gemm: k_gemm*; scatter: k_scatter*, k_pull_msgs*, k_recompute*, k_bin_arcs*, "
                "k_bin_sort, k_bucket_sum*)."]
        for i, sg in enumerate(segs):
            b = [ns for ns, _ in sg["batches"]]
            if not b:
                continue
            rest = sorted(b[1:]) or b
            med = rest[len(rest) // 2]
            ph = "; ".join(f"{p} {len(v)} dispatches avg {sum(v) / len(v) / 1e3:.2f} us"
                           for p, v in sg["phases"].items() if v)
            out.append(f"  workload {i}: {len(b)} batches, first {b[0] / 1e6:.3f} ms, median of the rest "
                       f"{med / 1e6:.3f} ms; {ph}")
    return "\n".join(out) + "\n"


def _counter(dirpath: str, batches_only: bool = False):
    """kernel -> list of (value KiB, duration ns) per dispatch; batches_only keeps
    the dispatches from the first batch on (its netting kernel), leaving out the
    bootstrap."""
    rows = list(csv.DictReader(open(_one(dirpath, "*counter_collection.csv"))))
    t0 = 0
    if batches_only:
        starts = [int(r["Start_Timestamp"]) for r in rows
                  if kernel_name(r["Kernel_Name"]) in ("k_net_hash", "k_net_direct")]
        t0 = min(starts) if starts else 0
    d = defaultdict(list)
    for r in rows:
        if int(r["Start_Timestamp"]) < t0:
            continue
        d[kernel_name(r["Kernel_Name"])].append(
            (float(r["Counter_Value"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    return d


def _copy_factor(copy_dir: str, size_kib: float) -> float:
    vals = [v for k, lst in _counter(copy_dir).items() if "copyBuffer" in k for v, _ in lst]
    if not vals:
        raise ValueError(f"no copy kernel in {copy_dir}")
    return size_kib / (sum(vals) / len(vals))


def calibration_md(copy_mib: int, gather_mib: int, dirs: dict, commands: str) -> str:
    """How the byte counters read on a streaming copy and on random row reads (a
    gather of every 192-byte row of a table once in random order, index_select): the
    derived FETCH_SIZE and WRITE_SIZE, and the request counters by size. dirs: copy /
    gather x fetch / write / rd / wr run directories."""
    rows = gather_mib * 2**20 // 192

    def top(d, multi=False):
        c = _counters_multi(d, False) if multi else _counter(d)
        ks = [k for k in c if "copyBuffer" not in k and "fill" not in k.lower() and not k.startswith("k_state")]
        if multi:
            return max(ks, key=lambda k: sum(c[k].get("TCC_EA0_RDREQ_sum", c[k].get("TCC_EA0_WRREQ_sum", [0])))), c
        return max(ks, key=lambda k: sum(v for v, _ in c[k]) / len(c[k])), c

    copy_bytes = copy_mib * 2**20
    ff = _copy_factor(dirs["copy_fetch"], copy_bytes / 1024.0)
    fw = _copy_factor(dirs["copy_write"], copy_bytes / 1024.0)
    kf, cf = top(dirs["gather_fetch"])
    kw, cw = top(dirs["gather_write"])
    gf = sum(v for v, _ in cf[kf]) / len(cf[kf]) * 1024.0
    gw = sum(v for v, _ in cw[kw]) / len(cw[kw]) * 1024.0
    crd, cwr = _counters_multi(dirs["copy_rd"], False), _counters_multi(dirs["copy_wr"], False)
    kc = next(k for k in crd if "copyBuffer" in k)
    _, cshare, crb, cwb = _sized_bytes(crd[kc], cwr.get(kc, {}))
    kg, grd = top(dirs["gather_rd"], True)
    gwr = _counters_multi(dirs["gather_wr"], False)
    greq, gshare, grb, gwb = _sized_bytes(grd[kg], gwr.get(kg, {}))
    useful = rows * (192 + 8)
    return "\n".join([
        "# How the HBM byte counters read (rocprofv3 --pmc; one run per counter set)", "",
        f"commands: {commands}", "",
        f"Streaming copy of {copy_mib} MiB (bench.py --copy-calibration {copy_mib}): FETCH_SIZE reads "
        f"1/{ff:.3f} of the bytes read and WRITE_SIZE 1/{fw:.3f} of those written. Its reads are "
        f"{100 * cshare:.1f}% 128-byte requests, and counted at their sizes they come to {crb / 2**20:.1f} MiB read and "
        f"{cwb / 2**20:.1f} MiB written: exact. FETCH_SIZE's formula counts 128-byte requests from TCC_BUBBLE, which "
        f"does not count them on this chip, so it takes them as 64 bytes.", "",
        f"Random-order gather of {rows} rows of 192 bytes, each read once, with 8-byte indices "
        f"(bench.py --gather-calibration {gather_mib}; kernel {kg}): {useful / 2**20:.0f} MiB of useful reads; "
        f"FETCH_SIZE reads {gf / 2**20:.0f} MiB; the requests counted at their sizes come to {grb / 2**20:.0f} MiB "
        f"({100 * gshare:.1f}% of {greq:.0f} requests are 128-byte, the rest 64-byte: each row costs two 128-byte "
        f"requests and one 64-byte request, 320 bytes for 192), written {gwb / 2**20:.0f} MiB. So the FETCH_SIZE x 2 "
        f"rule holds only for kernels whose reads are all 128-byte requests; the traffic table counts every "
        f"request at its own size instead (the library's large kernels issue 99-100% 128-byte reads).", ""]) + "\n"


def traffic_md(copy_fetch: str, copy_write: str, copy_mib: int, workloads) -> str:
    """workloads: list of (name, fetch_dir, write_dir, batches, command)."""
    kib = copy_mib * 1024.0
    ff, fw = _copy_factor(copy_fetch, kib), _copy_factor(copy_write, kib)
    out = ["# HBM traffic per dispatch (rocprofv3 FETCH_SIZE and WRITE_SIZE, separate runs)", "",
           f"source-hash: {source_hash()}", "",
           f"Calibration: a {copy_mib} MiB device-to-device copy (bench.py --copy-calibration {copy_mib}) reads "
           f"FETCH_SIZE x {ff:.4f} and WRITE_SIZE x {fw:.4f} of the bytes it moves; the calibrated columns "
           f"below apply these factors.", ""]
    for name, fdir, wdir, batches, cmd in workloads:
        f, w = _counter(fdir, True), _counter(wdir, True)
        out += [f"## {name}", "", f"command (one run per counter): {cmd.replace('COUNTER', 'FETCH_SIZE')} ; "
                f"{cmd.replace('COUNTER', 'WRITE_SIZE')}", "",
                f"Dispatches from the first of {batches} update batches on (the bootstrap is left out).", "",
                "| kernel | dispatches | FETCH KiB/disp | WRITE KiB/disp | HBM MB/disp (calibrated) |",
                "|---|---|---|---|---|"]
        for k in sorted(f, key=lambda k: -sum(v for v, _ in f[k])):
            fv = [v for v, _ in f[k]]
            wv = [v for v, _ in w.get(k, [])]
            fa = sum(fv) / len(fv)
            wa = sum(wv) / len(wv) if wv else 0.0
            out.append(f"| {k} | {len(fv)} | {fa:.1f} | {wa:.1f} | {(ff * fa + fw * wa) * 1024 / 1e6:.3f} |")
        out.append("")
        # per-launch traffic of each rooflined phase over the timed batches' kernels
        for phase, prefixes in PHASE_KERNELS.items():
            tot = n = 0.0
            for k in f:
                if k.startswith(prefixes):
                    fv = [v for v, _ in f[k]]
                    wv = [v for v, _ in w.get(k, [])]
                    tot += ff * sum(fv) + (fw * sum(wv) if wv else 0.0)
                    n += len(fv)
            if n:
                out.append(f"traffic {name} {phase} {tot * 1024 / n:.0f}")
        out.append("")
    return "\n".join(out) + "\n"


def _counters_multi(dirpath: str, batches_only: bool = True):
    """kernel -> {counter -> list of per-dispatch values} from a counter-collection
    CSV holding several counters (one row per dispatch and counter)."""
    rows = list(csv.DictReader(open(_one(dirpath, "*counter_collection.csv"))))
    t0 = 0
    if batches_only:
        starts = [int(r["Start_Timestamp"]) for r in rows
                  if kernel_name(r["Kernel_Name"]) in ("k_net_hash", "k_net_direct")]
        t0 = min(starts) if starts else 0
    d = defaultdict(lambda: defaultdict(list))
    seen = set()
    for r in rows:
        if int(r["Start_Timestamp"]) < t0:
            continue
        k = kernel_name(r["Kernel_Name"])
        d[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
        key = (r.get("Dispatch_Id"), k)
        if key not in seen:  # one duration per dispatch, whatever the number of counters
            seen.add(key)
            d[k]["_ns"].append(float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    return d


MFMA_PEAK_TFLOPS = {"F32": 157.3, "BF16": 2500.0}  # dense MFMA peaks of MI355X


def mfma_md(title: str, runs, simds: int = 1024, clock_ghz: float = 2.4) -> str:
    """MFMA use of the transform kernels from runs of --pmc SQ_INSTS_VALU_MFMA_MOPS_<T>
    SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE: runs = list of (name, dir, command, dtype).
    Per kernel: MFMA flops per dispatch (MOPS x 512), their rate over the
    dispatch's duration (counter-run timestamps) against the dtype's dense peak, and
    the busy fraction of the MFMA units, busy cycles (summed over SIMDs) over the
    duration's cycles at the nominal clock times the SIMD count. GRBM_GUI_ACTIVE
    over the duration's cycles is listed as a check: about 8 (it is summed over the
    XCDs) for long dispatches, more for short ones, whose counting window outlasts
    the kernel."""
    out = [f"# {title}", "",
           f"MFMA flops = SQ_INSTS_VALU_MFMA_MOPS_<T> x 512; rate = flops / dispatch duration; MfmaUtil = "
           f"SQ_VALU_MFMA_BUSY_CYCLES / (duration x {clock_ghz} GHz x {simds} SIMDs); GUI/dur = GRBM_GUI_ACTIVE / "
           f"(duration x {clock_ghz} GHz). Dispatches from the first update batch on; durations are those of the "
           f"counter run (dispatches serialised by the profiler).", ""]
    for name, d, cmd, dtype in runs:
        c = _counters_multi(d)
        mops = f"SQ_INSTS_VALU_MFMA_MOPS_{dtype}"
        peak = MFMA_PEAK_TFLOPS[dtype]
        out += [f"## {name}", "", f"command: {cmd}", "",
                f"| kernel | dispatches | MFMA MFLOP/disp | avg us | TFLOP/s | % of {peak:g} TFLOP/s | "
                "MFMA busy cycles/disp | MfmaUtil % | GUI/dur |", "|---|---|---|---|---|---|---|---|---|"]
        for k in sorted(c, key=lambda k: -sum(c[k].get(mops, [0.0]))):
            m, b, g, ns = (c[k].get(x, []) for x in (mops, "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "_ns"))
            if not k.startswith("k_gemm") or not m or not ns:
                continue
            n = len(m)
            fl = 512.0 * sum(m) / n
            dur = sum(ns) / len(ns)
            cyc = dur * clock_ghz
            busy = sum(b) / len(b) if b else 0.0
            gui = (sum(g) / len(g)) / cyc if g and cyc else 0.0
            rate = fl / dur / 1e3
            out.append(f"| {k} | {n} | {fl / 1e6:.2f} | {dur / 1e3:.2f} | {rate:.2f} | {100 * rate / peak:.2f} | "
                       f"{busy:.0f} | {100 * busy / (cyc * simds):.2f} | {gui:.2f} |")
        out.append("")
    return "\n".join(out) + "\n"


RD_COUNTERS = ("TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum")
WR_COUNTERS = ("TCC_EA0_WRREQ_sum", "TCC_EA0_WRREQ_64B_sum")


def _sized_bytes(rd: dict, wr: dict):
    """Per-dispatch averages: (requests, share of 128-byte reads, read bytes, write bytes)
    from the L2-to-fabric request counters, each request counted at its own size."""
    def avg(d, name):
        v = d.get(name, [])
        return sum(v) / len(v) if v else 0.0
    req = avg(rd, "TCC_EA0_RDREQ_sum")
    c32, c64, c128 = (avg(rd, n) for n in RD_COUNTERS[1:])
    wt, w64 = avg(wr, "TCC_EA0_WRREQ_sum"), avg(wr, "TCC_EA0_WRREQ_64B_sum")
    return req, (c128 / req if req else 0.0), 32 * c32 + 64 * c64 + 128 * c128, 32 * (wt - w64) + 64 * w64


def traffic_sized_md(copy_rd: str, copy_wr: str, copy_mib: int, workloads) -> str:
    """HBM traffic per dispatch from two runs per workload: --pmc of the read request
    counters by size (32, 64, 128 bytes) and of the write request counters, each
    request counted at its size. workloads: list of (name, rd_dir, wr_dir, batches,
    command). The copy run checks the method: its reads and writes must come out at
    the bytes the copy moves."""
    crd, cwr = _counters_multi(copy_rd, False), _counters_multi(copy_wr, False)
    k = next(k for k in crd if "copyBuffer" in k)
    _, _, cr, cw = _sized_bytes(crd[k], cwr.get(k, {}))
    out = ["# HBM traffic per dispatch (L2-to-fabric requests counted at their sizes; reads and writes in separate runs)",
           "", f"source-hash: {source_hash()}", "",
           f"Check: a {copy_mib} MiB device-to-device copy (bench.py --copy-calibration {copy_mib}) comes out at "
           f"{cr / 2**20:.1f} MiB read and {cw / 2**20:.1f} MiB written. Bytes = 32 x TCC_EA0_RDREQ_32B + 64 x "
           f"TCC_EA0_RDREQ_64B + 128 x TCC_EA0_RDREQ_128B (reads), 64 x TCC_EA0_WRREQ_64B + 32 x the other write "
           f"requests (writes); MALL hits count as traffic.", ""]
    for name, rdd, wrd, batches, cmd in workloads:
        rd, wr = _counters_multi(rdd), _counters_multi(wrd)
        out += [f"## {name}", "",
                f"commands (one run per counter set): {cmd.replace('COUNTERS', ' '.join(RD_COUNTERS)).replace('SET', 'rd')} ; "
                f"{cmd.replace('COUNTERS', ' '.join(WR_COUNTERS)).replace('SET', 'wr')}", "",
                f"Dispatches from the first of {batches} update batches on (the bootstrap is left out).", "",
                "| kernel | dispatches | read requests/disp | 128-byte share | read MB/disp | write MB/disp |",
                "|---|---|---|---|---|---|"]
        rows = []
        for kname in rd:
            req, share, rb, wb = _sized_bytes(rd[kname], wr.get(kname, {}))
            rows.append((rb + wb, kname, len(rd[kname].get("_ns", [])), req, share, rb, wb))
        for _, kname, n, req, share, rb, wb in sorted(rows, reverse=True):
            out.append(f"| {kname} | {n} | {req:.0f} | {share:.3f} | {rb / 1e6:.3f} | {wb / 1e6:.3f} |")
        out.append("")
        for phase, prefixes in PHASE_KERNELS.items():
            tot = cnt = 0.0
            for _, kname, n, req, share, rb, wb in rows:
                if kname.startswith(prefixes):
                    tot += (rb + wb) * n
                    cnt += n
            if cnt:
                out.append(f"traffic {name} {phase} {tot / cnt:.0f}")
        out.append("")
    return "\n".join(out) + "\n"


def read_traffic(workload: str, phase: str):
    """Calibrated HBM bytes per launch of `phase` on `workload` from the committed
    table, or None when there is none or it predates the current sources."""
    try:
        text = open(TRAFFIC_MD).read()
    except OSError:
        return None
    m = re.search(r"source-hash: (\w+)", text)
    if not m or m.group(1) != source_hash():
        return None
    m = re.search(rf"^traffic {re.escape(workload)} {phase} (\d+)$", text, re.M)
    return float(m.group(1)) if m else None


def main(argv):
    if argv[:1] == ["stats"]:
        sys.stdout.write(stats_table(argv[1], argv[2], argv[3]))
    elif argv[:1] == ["mfma"]:
        # mfma OUT TITLE NAME=DIR,DTYPE,CMD ...
        runs = []
        for spec in argv[3:]:
            name, rest = spec.split("=", 1)
            d, dtype, cmd = rest.split(",", 2)
            runs.append((name, d, cmd, dtype))
        with open(argv[1], "w") as fh:
            fh.write(mfma_md(argv[2], runs))
    elif argv[:1] == ["traffic-sized"]:
        # traffic-sized OUT COPY_MIB COPY_RD COPY_WR WORKLOAD=RD_DIR,WR_DIR,BATCHES,CMD ...
        wls = []
        for spec in argv[5:]:
            name, rest = spec.split("=", 1)
            rdd, wrd, batches, cmd = rest.split(",", 3)
            wls.append((name, rdd, wrd, int(batches), cmd))
        with open(argv[1], "w") as fh:
            fh.write(traffic_sized_md(argv[3], argv[4], int(argv[2]), wls))
    elif argv[:1] == ["calibration"]:
        # calibration OUT COPY_MIB GATHER_MIB KEY=DIR ... COMMANDS (keys copy_fetch copy_write gather_fetch
        # gather_write copy_rd copy_wr gather_rd gather_wr)
        dirs = dict(a.split("=", 1) for a in argv[4:-1])
        with open(argv[1], "w") as fh:
            fh.write(calibration_md(int(argv[2]), int(argv[3]), dirs, argv[-1]))
    elif argv[:1] == ["traffic"]:
        out, copy_mib, cf, cw = argv[1], int(argv[2]), argv[3], argv[4]
        wls = []
        for spec in argv[5:]:
            name, rest = spec.split("=", 1)
            fdir, wdir, batches, cmd = rest.split(",", 3)
            wls.append((name, fdir, wdir, int(batches), cmd))
        with open(out, "w") as fh:
            fh.write(traffic_md(cf, cw, copy_mib, wls))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))

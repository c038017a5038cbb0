"""The C ABI from a plain C99 program (tests/c_client/ripple_client.c): built with
gcc against include/ripple.h and libripple.so alone, it loads a graph, runs a
model's bootstrap and a stream of batches, and reads the affected sets and
embeddings back; the test checks them against the CPU oracle (sets bit for bit,
embeddings within 1e-4 row-relative error) and checks the statuses of calls
that must be rejected."""
import os
import struct
import subprocess
import sys

import numpy as np
import pytest

from oracle import ripple_oracle as O
from paper_2505_12112_amd import ripple as R
from paper_2505_12112_amd import synth
from tests.harness import FP32_TOL, random_valid_batch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT_SRC = os.path.join(ROOT, "tests", "c_client", "ripple_client.c")


def _build_client(tmp_path):
    if not os.path.exists(R.LIB_PATH):
        pytest.skip("libripple.so not built")
    exe = tmp_path / "ripple_client"
    libdir = os.path.dirname(R.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                    CLIENT_SRC, "-L", libdir, "-lripple", f"-Wl,-rpath,{libdir}", "-o", str(exe)], check=True)
    return exe


def test_client_builds_against_the_header_alone(tmp_path):
    exe = _build_client(tmp_path)
    # without arguments it prints its usage and exits with status 2 (no device call)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 2 and "usage" in r.stderr


@pytest.mark.gpu
@pytest.mark.parametrize("agg", ["sum", "mean", "gcn", "gc_sum"])
def test_c_client_matches_the_oracle(tmp_path, agg):
    print("c client", agg, file=sys.stderr, flush=True)
    exe = _build_client(tmp_path)
    rng = np.random.default_rng(31 + ["sum", "mean", "gcn", "gc_sum"].index(agg))
    n, m, dims = 300, 1500, (12, 40, 7)
    src, dst = synth.erdos_renyi(n, m, rng)
    x = rng.standard_normal((n, dims[0])).astype(np.float32)
    w = synth.model_weights(synth.ModelSpec(agg, dims), rng, bias_std=0.1)
    orc = O.OracleState(n, src, dst, x, O.OracleModel.from_weights(w))
    L = len(dims) - 1
    batches = []
    expect_sets = []
    for b in range(8):
        batch = random_valid_batch(rng, orc, int(rng.integers(1, 50)), dims[0])
        _, sets = orc.apply(batch.ops, batch.feat_rows)
        batches.append(batch)
        expect_sets.append(sets)
    buf = bytearray()
    buf += struct.pack("<5q", n, src.size, L, R.AGG[agg], len(batches))
    buf += np.asarray(dims, "<i4").tobytes() + np.asarray([1 if r else 0 for r in w.relu], "<i4").tobytes()
    buf += np.asarray(src, "<i4").tobytes() + np.asarray(dst, "<i4").tobytes() + x.astype("<f4").tobytes()
    for l in range(L):
        buf += struct.pack("<q", 0 if w.w_self[l] is None else 1)
        if w.w_self[l] is not None:
            buf += np.ascontiguousarray(w.w_self[l], "<f4").tobytes()
        buf += np.ascontiguousarray(w.w_neigh[l], "<f4").tobytes()
        buf += np.ascontiguousarray(w.bias[l], "<f4").tobytes()
    for batch in batches:
        ops = np.ascontiguousarray(np.asarray(batch.ops, np.int32).reshape(-1, 4), "<i4")
        feat = np.ascontiguousarray(batch.feat_rows, "<f4").reshape(-1, dims[0])
        buf += struct.pack("<2q", ops.shape[0], feat.shape[0]) + ops.tobytes() + feat.tobytes()
    fin, fout = tmp_path / "in.bin", tmp_path / "out.bin"
    fin.write_bytes(bytes(buf))
    r = subprocess.run([str(exe), str(fin), str(fout)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = memoryview(fout.read_bytes())
    pos = 0

    def take(dtype, count):
        nonlocal pos
        a = np.frombuffer(out, dtype, count, pos)
        pos += a.nbytes
        return a

    for b, sets in enumerate(expect_sets):
        for l in range(L + 1):
            cnt = int(take("<i8", 1)[0])
            np.testing.assert_array_equal(take("<i4", cnt), sets[l].astype(np.int32), err_msg=f"batch {b} A^{l}")
    ref = orc.embeddings()
    for l in range(L + 1):
        h = take("<f4", n * dims[l]).reshape(n, dims[l])
        assert O.row_relative_error(h, ref[l]) <= FP32_TOL, f"H^{l}"
    bad = take("<i4", 4)
    assert list(bad) == [R.E_INVALID] * 4
    assert pos == len(out)

"""The C ABI without a GPU: the library loads, exports every function the header
declares, its structs have the layout the binding assumes, and argument checks
that run before any device call reject bad input."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2505_12112_amd import ripple as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ripple.h")


def _lib():
    try:
        return R.load_library()
    except R.RippleUnavailable:
        pytest.skip("libripple.so not built")


def test_header_declarations_are_exported():
    lib = _lib()
    text = open(HEADER).read()
    declared = set(re.findall(r"RIPPLE_API\s+[\w\s\*]+?\b(ripple_\w+)\s*\(", text))
    assert declared == set(R.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", R.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (ripple_\w+)", out))
    assert declared <= exported
    for name in declared:
        assert hasattr(lib, name)


def test_struct_layouts_match_the_header(tmp_path):
    src = tmp_path / "sizes.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "ripple.h"\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(ripple_graph_desc),'
                   ' sizeof(ripple_model_desc), sizeof(ripple_batch_stats), sizeof(ripple_phase_stats),'
                   ' sizeof(ripple_op), offsetof(ripple_graph_desc, stream),'
                   ' offsetof(ripple_batch_stats, relocated_rows)); return 0;}\n')
    exe = tmp_path / "sizes"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    got = [int(t) for t in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()]
    assert got == [C.sizeof(R.GraphDesc), C.sizeof(R.ModelDesc), C.sizeof(R.BatchStats), C.sizeof(R.PhaseStats),
                   16, R.GraphDesc.stream.offset, R.BatchStats.relocated_rows.offset]


def _load(n, src, dst, **kw):
    lib = _lib()
    src = np.ascontiguousarray(src, np.int32)
    dst = np.ascontiguousarray(dst, np.int32)
    desc = R.GraphDesc(n, src.size, src.ctypes.data_as(C.POINTER(C.c_int32)),
                       dst.ctypes.data_as(C.POINTER(C.c_int32)), kw.get("undirected", 0), 0.25, 4, 0, None, 0, 0)
    ctx = C.c_void_p(123)
    st = lib.ripple_load_graph(C.byref(desc), C.byref(ctx))
    return st, ctx, lib.ripple_last_error(None).decode()


@pytest.mark.parametrize("case,src,dst,n,msg", [
    ("n_zero", [], [], 0, "num_vertices"),
    ("id_out_of_range", [0, 5], [1, 2], 4, "out of range"),
    ("negative_id", [0, -1], [1, 2], 4, "out of range"),
    ("self_loop", [0, 2], [1, 2], 4, "self-loop"),
    ("repeated_arc", [0, 0], [1, 1], 4, "repeated arc"),
])
def test_load_graph_rejects_bad_snapshots_before_touching_the_device(case, src, dst, n, msg):
    st, ctx, err = _load(n, src, dst)
    assert st == R.E_INVALID
    assert ctx.value is None
    assert msg in err


def test_undirected_pair_listed_twice_is_a_repeated_arc():
    st, _, err = _load(3, [0, 1], [1, 0], undirected=1)
    assert st == R.E_INVALID and "repeated arc" in err


def test_null_context_calls():
    lib = _lib()
    assert lib.ripple_apply_updates(None, None, 0, None, 0, None) == R.E_INVALID
    assert lib.ripple_get_embeddings(None, 0, None, 0, None) == R.E_INVALID
    lib.ripple_destroy(None)
    assert lib.ripple_phase_name(3) == b"scatter"
    assert lib.ripple_phase_name(99) == b""

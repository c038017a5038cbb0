"""Parity at the benchmark workloads' full sizes, in the launch configuration
bench.py times (library stream, batch sizes of the workload)."""
import sys
import time

import numpy as np
import pytest

from oracle import ripple_oracle as O
from paper_2505_12112_amd import synth
from tests.harness import Pair

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("bs", [100, 1000])
def test_sparse_mid_full_size(bs):
    """169,343 vertices / 1,166,243 arcs, GraphSAGE-sum 128-256-40: affected sets
    every batch, all embeddings against a float64 full recompute at the end."""
    wl = synth.build_workload("sparse_mid")
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights)
    try:
        p.check_embeddings()
        t0 = time.time()
        nb = 20 if bs == 100 else 5
        for b in range(nb):
            st, _, sets = p.step(wl.stream.next_batch(bs))
        _say(f"sparse_mid bs={bs}: {nb} batches in {time.time() - t0:.1f}s, last |A| = {[s.size for s in sets]}")
        errs = p.check_embeddings()
        _say("  row-relative errors", errs)
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

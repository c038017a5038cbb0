"""ripple_get_embeddings_static (the entry point that allocates nothing) against
ripple_get_embeddings, through the C ABI: two calls in a row, the second with fewer
rows, must return the same rows bit for bit; a call over the staging array's limit
is rejected; neither the context's device bytes nor the device's free memory move."""
import numpy as np
import pytest

from paper_2505_12112_amd import synth
from paper_2505_12112_amd.ripple import E_INVALID, RippleError
from tests.harness import Pair, device_free_bytes, random_valid_batch

pytestmark = pytest.mark.gpu


def test_static_staging_matches_get_embeddings():
    rng = np.random.default_rng(91)
    wl = synth.build_workload("tiny", bias_std=0.1)
    p = Pair(wl.n, wl.src, wl.dst, wl.x, wl.weights)
    try:
        for _ in range(3):
            p.step(wl.stream.next_batch(100))
        # a first call on this device finds the array's address, and the runtime sets up
        # its copy path (it may reserve memory of its own once); the baseline is taken after
        p.lib.get_embeddings_static(2, np.arange(1500, dtype=np.int32))
        held = p.lib.device_bytes()
        for layer, count in ((2, 1500), (1, 37)):  # the second call is smaller
            ids = rng.integers(0, wl.n, count).astype(np.int32)
            free0 = device_free_bytes()
            got = p.lib.get_embeddings_static(layer, ids)
            assert device_free_bytes() == free0 and p.lib.device_bytes() == held
            want = p.lib.get_embeddings(layer, ids)  # (allocates and frees its staging buffers)
            np.testing.assert_array_equal(got, want)
        # all rows (no staging needed), after another batch
        p.step(random_valid_batch(rng, p.orc, 50, wl.weights.dims[0]))
        for layer in range(3):
            np.testing.assert_array_equal(p.lib.get_embeddings_static(layer), p.lib.get_embeddings(layer))
        # over the limit: 2^21 ids of 16 floats need 8 MiB + 128 MiB
        big = np.zeros(1 << 21, np.int32)
        with pytest.raises(RippleError) as e:
            p.lib.get_embeddings_static(1, big)
        assert e.value.status == E_INVALID and "32 MiB" in str(e.value), str(e.value)
        assert p.lib.device_bytes() == held
    finally:
        p.close()

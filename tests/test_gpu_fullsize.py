"""GPU parity at the full sizes of the sequence-length sweep (batch 1, 8 heads,
d 64, N = 2^10 .. 2^15, fp32 and bf16, C 100, L 10, k 32, both variants) and of
the long-context case (batch 1, 8 heads, N 65536, d 64, bf16, C 200, L 15,
k 64, improved variant).  These sizes take the several-chunk attention path
(partial tiles, merge, sparse kernel) and the several-workgroup K-means path.

The oracle computes every output of these workloads (a few seconds each on
the host cores), so the comparison is element by element, to the same bars as
the smaller cases: codes, assignments and sizes exact, top-k sets up to near
ties, outputs within 2e-5 (fp32) or 2e-2 (bf16).
"""
import numpy as np
import pytest

import gen
import gpu_util
from gpu_util import check_end_to_end

pytestmark = pytest.mark.gpu

_W = {}


def workload(key):
    if key not in _W:
        _W.clear()  # one full-size workload (and its oracle results) resident at a time
        gpu_util.clear_oracle_cache()
        if key[0] == "long":
            _W[key] = gen.make_config(5)
        else:
            _W[key] = gen.make_config(3, N=key[1], dtype=key[2])
    return _W[key]


@pytest.fixture(autouse=True)
def _announce(request):
    print("\n[gpu test] %s" % request.node.name, flush=True)
    yield


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("log2n", [10, 11, 12, 13, 14, 15])
def test_sweep_full_size(log2n, dtype, variant):
    w = workload(("sweep", 1 << log2n, dtype))
    check_end_to_end(w, w.topk if variant == "iclustered" else 0)


def test_long_context_full_size():
    w = workload(("long",))
    check_end_to_end(w, w.topk)


@pytest.mark.parametrize("key", [("long",), ("sweep", 32768, "f32")])
def test_stage_isolated_full_size(key):
    """The oracle's partition and top-k sets injected at the full sizes: every
    mass, rest part and output row comparable, with no near-tie exemption."""
    w = workload(key)
    ref = gpu_util.run_oracle(w, w.topk)
    N = w.q.shape[2]
    assign_in = np.where(ref["assign"] < 0, 0, ref["assign"]).reshape(-1, N)
    topk_in = ref["topk"].reshape(-1, w.C, w.topk)
    got = gpu_util.run_gpu(w, w.topk, assign_in=assign_in, topk_in=topk_in)
    vm = gpu_util.valid_mask(w)
    assert np.array_equal(got["topk"], ref["topk"])
    np.testing.assert_allclose(got["mass"], ref["mass"], rtol=0, atol=1e-5)
    np.testing.assert_allclose(got["values"], ref["vcb"], rtol=0, atol=gpu_util.tol(w))
    err = np.abs(got["out"] - ref["out"])[vm].max()
    print("max abs error: %.3g" % err)
    assert err <= gpu_util.tol(w)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
@pytest.mark.parametrize("log2n", [9, 12])
def test_time_benchmark_protocol_full_size(log2n, variant):
    """The shapes of the time and memory benchmark (6 heads x 64, 2^17 tokens
    per call: batch 256 at N = 512, 32 at N = 4096), which run the one-
    workgroup K-means for many units, up to its largest n."""
    N = 1 << log2n
    key = ("fig4", N)
    if key not in _W:
        _W.clear()
        gpu_util.clear_oracle_cache()
        _W[key] = gen.config_sweep(N, dtype="f32", B=(1 << 17) // N, H=6, d=64)
    w = _W[key]
    check_end_to_end(w, w.topk if variant == "iclustered" else 0)

"""GPU parity on seeded random shapes: batch, heads, length (from 1 to 3000,
chunk edges included), d, dtype, C, n_bits, L, k and ragged lengths (zero
included) drawn per seed; both variants end to end and oracle-top, each
against the fp64 oracle to the same bars as the fixed workloads (codes,
assignments and sizes exact, top-k sets up to near ties, outputs within 2e-5
in fp32 or 2e-2 in bf16)."""
import pytest

import gen
from gpu_util import check_end_to_end, clear_oracle_cache
from test_gpu_otop import check as check_oracle_top

pytestmark = pytest.mark.gpu

SEEDS = list(range(32))


@pytest.mark.parametrize("seed", SEEDS)
def test_random_shapes(seed):
    w = gen.config_random(seed)
    print("\n[gpu case] %s C %d n_bits %d L %d k %d lengths %s" % (
        w.name, w.C, w.n_bits, w.L, w.topk, w.lengths.tolist()), flush=True)
    clear_oracle_cache()
    check_end_to_end(w, 0)
    check_end_to_end(w, w.topk)
    check_oracle_top(w, w.topk)


@pytest.mark.parametrize("seed", SEEDS)
def test_random_shapes_backward(seed):
    """The backward pass of both variants on the same random shapes, against
    the oracle's gradients for the GPU forward's partition and top-k sets."""
    from test_gpu_backward import run_case
    w = gen.config_random(seed)
    print("\n[gpu case] backward %s C %d k %d lengths %s" % (w.name, w.C, w.topk, w.lengths.tolist()),
          flush=True)
    run_case(w, 0)
    run_case(w, w.topk)


@pytest.mark.parametrize("seed", SEEDS[:12])
def test_random_shapes_cooperative_kmeans(seed):
    """The same shapes with the cooperative K-means forced (every length from 0
    up), its centroid sums formed by the K-means kernel for even seeds and by
    the separate kernel for odd ones."""
    import paper_2007_04825_amd as ca
    w = gen.config_random(seed)
    print("\n[gpu case] cooperative %s C %d n_bits %d L %d k %d lengths %s" % (
        w.name, w.C, w.n_bits, w.L, w.topk, w.lengths.tolist()), flush=True)
    clear_oracle_cache()
    try:
        ca.set_kmeans_path(4 if seed % 2 == 0 else 5)
        check_end_to_end(w, 0)
        check_end_to_end(w, w.topk)
    finally:
        ca.set_kmeans_path(0)

"""GPU parity: the HIP library, called through its C ABI, against the fp64
oracle on the same seeded inputs.

Bars (stated by the project's targets):
  * hash codes bit-exact, except bits whose oracle projection lies within
    1e-6 of zero (counted and reported; none are expected, since both sides
    evaluate the projection in fp64 with exact products);
  * cluster assignments and sizes bit-exact given identical codes;
  * top-k sets identical, a difference being accepted only as a near tie
    (every key in the symmetric difference within 1e-5*max(1,|s_k|) of the
    oracle's k-th logit: the fp32 logits of the kernel carry about 1e-6 of
    rounding error);
  * outputs within 2e-5 max-abs for fp32 inputs and 2e-2 for bf16 inputs.
"""
import os

import numpy as np
import pytest

import gen
import oracle
from gpu_util import (check_end_to_end, compare_outputs, run_gpu, run_oracle, tol,
                      topk_mismatches, valid_mask)

pytestmark = pytest.mark.gpu

WORKLOADS = {
    "tiny": lambda: gen.make_config(1),
    "speech": lambda: gen.make_config(2),
    "encoder": lambda: gen.make_config(4),
    "sweep2048_f32": lambda: gen.make_config(3, N=2048, dtype="f32"),
    "sweep4096_bf16": lambda: gen.make_config(3, N=4096, dtype="bf16"),
}
_W = {}


def workload(name):
    if name not in _W:
        _W[name] = WORKLOADS[name]()
    return _W[name]


@pytest.fixture(autouse=True)
def _announce(request):
    print("\n[gpu test] %s" % request.node.name, flush=True)
    yield


@pytest.mark.parametrize("name", list(WORKLOADS))
@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_end_to_end_parity(name, variant):
    w = workload(name)
    check_end_to_end(w, w.topk if variant == "iclustered" else 0)


@pytest.mark.parametrize("name", ["speech", "encoder", "sweep4096_bf16"])
def test_stage_isolated_improved(name):
    """Oracle's partition and top-k sets injected: every row comparable."""
    w = workload(name)
    ref = run_oracle(w, w.topk)
    assign_in = np.where(ref["assign"] < 0, 0, ref["assign"]).reshape(-1, w.q.shape[2])
    topk_in = ref["topk"].reshape(-1, w.C, w.topk)
    got = run_gpu(w, w.topk, assign_in=assign_in, topk_in=topk_in)
    vm = valid_mask(w)
    assert np.array_equal(got["topk"], ref["topk"])
    np.testing.assert_allclose(got["mass"], ref["mass"], rtol=0, atol=1e-5)
    np.testing.assert_allclose(got["values"], ref["vcb"], rtol=0, atol=tol(w))
    err = np.abs(got["out"] - ref["out"])[vm].max()
    print("max abs error: %.3g" % err)
    assert err <= tol(w)


@pytest.mark.parametrize("name", ["tiny", "speech"])
def test_injected_codes_give_oracle_assignment(name):
    w = workload(name)
    ref = run_oracle(w, 0)
    codes = ref["codes"].reshape(-1, w.q.shape[2])
    got = run_gpu(w, 0, codes_in=codes)
    assert np.array_equal(got["assign"], ref["assign"])


@pytest.mark.parametrize("name", ["tiny", "sweep2048_f32", "sweep4096_bf16"])
def test_every_kmeans_driver_agrees(name):
    import paper_2007_04825_amd as ca
    w = workload(name)
    res = []
    try:
        for path in (1, 2, 4, 5):
            ca.set_kmeans_path(path)
            res.append(run_gpu(w, w.topk))
    finally:
        ca.set_kmeans_path(0)
    for r in res[1:]:
        for key in ("codes", "assign", "sizes", "topk"):
            assert np.array_equal(res[0][key], r[key]), key
        np.testing.assert_allclose(r["centroids"], res[0]["centroids"], rtol=0, atol=2e-6)
        assert np.abs(r["out"] - res[0]["out"]).max() <= tol(w)


def test_deterministic_bitwise():
    w = workload("speech")
    a = run_gpu(w, w.topk)
    b = run_gpu(w, w.topk)
    for key in a:
        assert np.array_equal(a[key], b[key]), key


# --------------------------------------------------------------------------
# Invariants that hold at any size (Section 3.2 / 3.3 special cases).
# --------------------------------------------------------------------------

def _exact_attention(q, k, v):
    q, k, v = (np.asarray(x, np.float64) for x in (q, k, v))
    s = q @ k.T / np.sqrt(q.shape[1])
    s = s - s.max(1, keepdims=True)
    a = np.exp(s)
    a /= a.sum(1, keepdims=True)
    return a @ v


@pytest.mark.parametrize("d", [32, 64])
def test_singleton_clusters_reduce_to_exact_attention(d):
    n = 200
    w = gen.config_sweep(N=n, B=1, H=2, d=d, C=n, topk=16)
    assign = np.tile(np.arange(n, dtype=np.int32), (2, 1))
    for topk in (0, 16):
        got = run_gpu(w, topk, assign_in=assign)
        for h in range(2):
            ref = _exact_attention(w.q[0, h], w.k[0, h], w.v[0, h])
            assert np.abs(got["out"][0, h] - ref).max() <= 2e-5


def test_topk_equal_n_reduces_to_exact_attention():
    n = 100
    w = gen.config_sweep(N=n, B=1, H=3, d=64, C=10, topk=n)
    got = run_gpu(w, n)
    for h in range(3):
        ref = _exact_attention(w.q[0, h], w.k[0, h], w.v[0, h])
        assert np.abs(got["out"][0, h] - ref).max() <= 2e-5
    assert np.allclose(got["mass"][got["sizes"] > 0], 1.0, atol=1e-6)


def test_rows_of_attention_sum_to_one():
    """With V = 1 every output row is the sum of its attention row (A^c or A^t)."""
    w = gen.make_config(2)
    w.v = np.where(np.isnan(w.v), w.v, 1.0).astype(np.float32)
    vm = valid_mask(w)
    for topk in (0, w.topk):
        got = run_gpu(w, topk)
        assert np.abs(got["out"][vm] - 1.0).max() <= 2e-6


def test_members_share_clustered_rows():
    w = workload("tiny")
    got = run_gpu(w, 0)
    for h in range(w.q.shape[1]):
        a = got["assign"][0, h]
        for j in np.unique(a):
            rows = got["out"][0, h][a == j]
            assert np.all(rows == rows[0])


# --------------------------------------------------------------------------
# Edge cases: ragged and empty lengths, n below C and k, odd parameters.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_ragged_lengths_nan_padding(variant):
    lens = [0, 1, 2, 15, 16, 17, 31, 33, 64, 99, 100, 101, 255, 256, 257, 300]
    w = gen.config_speech(B=len(lens), H=2, N=300, d=32, C=100, L=4, topk=32, lengths=lens,
                          pad_value=np.nan)
    topk = w.topk if variant == "iclustered" else 0
    ref = run_oracle(w, topk)
    got = run_gpu(w, topk)
    assert np.array_equal(got["assign"], ref["assign"])
    assert not np.isnan(got["out"]).any()
    compare_outputs(w, ref, got, topk)


@pytest.mark.parametrize("C,n_bits,L,topk", [(1, 63, 3, 1), (16, 8, 1, 5), (17, 33, 2, 128),
                                             (256, 63, 3, 64), (5, 1, 2, 7)])
def test_parameter_corners(C, n_bits, L, topk):
    w = gen.config_tiny(B=2, H=2, N=700, d=64, C=C, n_bits=n_bits, L=L, topk=topk)
    w.lengths = np.array([700, 517], np.int32)
    ref = run_oracle(w, topk, key="corner%d_%d_%d_%d" % (C, n_bits, L, topk))
    got = run_gpu(w, topk)
    assert np.array_equal(got["codes"], ref["codes"])
    assert np.array_equal(got["assign"], ref["assign"])
    compare_outputs(w, ref, got, topk)


# Every K-means driver that applies to the length: 1 one workgroup per unit
# (n <= 4096), 2 one launch pair per round, 3 cooperative (all rounds in one
# launch); C = 256 with n above one key chunk (several-chunk attention and
# merge) and above one cooperative block (4096 queries).
BIG_C = [(2100, "f32", 128), (3000, "bf16", 100), (4500, "f32", 64), (9000, "bf16", 128)]


@pytest.mark.parametrize("N,dtype,topk", BIG_C)
@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_many_clusters_every_driver(N, dtype, topk, variant):
    import paper_2007_04825_amd as ca
    w = gen.config_tiny(B=2, H=1, N=N, d=64, C=256, L=4, topk=topk)
    w = gen.with_dtype(w, dtype)
    w.lengths = np.array([N, N - 777], np.int32)
    t = topk if variant == "iclustered" else 0
    ref = run_oracle(w, t, key="bigc%d_%s_%d" % (N, dtype, topk))
    paths = (1, 2, 4, 5) if N <= 4096 else (2, 4, 5)
    results = []
    try:
        for path in paths:
            ca.set_kmeans_path(path)
            got = run_gpu(w, t)
            print("driver %d" % path)
            assert np.array_equal(got["codes"], ref["codes"])
            assert np.array_equal(got["assign"], ref["assign"]), "driver %d" % path
            assert np.array_equal(got["sizes"], ref["sizes"])
            np.testing.assert_allclose(got["centroids"], ref["qc"], rtol=0, atol=2e-6)
            compare_outputs(w, ref, got, t)
            results.append(got)
    finally:
        ca.set_kmeans_path(0)
    for r in results[1:]:
        assert np.array_equal(r["assign"], results[0]["assign"])


def test_coop_kmeans_unit_of_65536_queries():
    """Units of exactly 65536 queries, where one cluster may hold every query
    and a bit count reach 65536: the one-launch K-means' table of 16-bit
    counts leaves the unit's first query out and adds it back on reading.
    Head 0 holds mixture queries, head 1 one row repeated 65536 times (one
    cluster of every query, each set bit counted 65536 times).  Codes,
    assignments, sizes and centroids against the oracle on both one-launch
    forms and the per-round kernels."""
    import paper_2007_04825_amd as ca
    w = gen.config_tiny(B=1, H=2, N=65536, d=32, C=16, L=4, topk=32)
    q = w.q.copy()
    q[0, 1] = q[0, 1, :1]
    w.q = q
    ref = run_oracle(w, 0, key="unit65536")
    assert ref["sizes"][0, 1, 0] == 65536
    try:
        for path in (2, 4, 5):
            ca.set_kmeans_path(path)
            got = run_gpu(w, 0)
            print("driver %d" % path)
            assert np.array_equal(got["codes"], ref["codes"])
            assert np.array_equal(got["assign"], ref["assign"]), "driver %d" % path
            assert np.array_equal(got["sizes"], ref["sizes"]), "driver %d" % path
            np.testing.assert_allclose(got["centroids"], ref["qc"], rtol=0, atol=2e-6)
    finally:
        ca.set_kmeans_path(0)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_full_width_codes_every_driver(variant):
    """64-bit hash codes (every bit of the word a plane) on every K-means
    driver: codes, assignments, sizes and outputs against the oracle."""
    import paper_2007_04825_amd as ca
    w = gen.config_tiny(B=2, H=2, N=3000, d=64, C=100, n_bits=64, L=5, topk=32)
    w.lengths = np.array([3000, 1999], np.int32)
    t = w.topk if variant == "iclustered" else 0
    ref = run_oracle(w, t, key="fullwidth64")
    assert np.any(ref["codes"] >> np.uint64(63))      # bit 63 is in use
    try:
        for path in (1, 2, 4, 5):
            ca.set_kmeans_path(path)
            print("driver %d" % path, flush=True)
            got = run_gpu(w, t)
            assert np.array_equal(got["codes"], ref["codes"])
            assert np.array_equal(got["assign"], ref["assign"]), "driver %d" % path
            assert np.array_equal(got["sizes"], ref["sizes"])
            compare_outputs(w, ref, got, t)
    finally:
        ca.set_kmeans_path(0)


SEEDED = {
    "tiny": lambda: gen.config_tiny(B=1, H=4, N=1024, d=64, C=100, L=10, topk=32),
    "bits64-d32-bf16": lambda: gen.with_dtype(
        gen.config_tiny(B=2, H=3, N=3000, d=32, C=60, n_bits=64, L=5, topk=16), "bf16"),
}


@pytest.mark.parametrize("case", list(SEEDED))
@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_planes_drawn_from_seed(case, variant):
    """No planes given: the library draws them from a seed (Section 3.2.2
    draws them at random).  The drawn planes equal the oracle's draw from
    the same seed (the two sides' fp64 log, cos and sin may differ in the
    last place, so one fp32 ulp is allowed, and nearly every entry must match
    exactly); they are the same on every call and differ for another seed;
    the forward with them is bitwise the forward given those planes, which
    matches the oracle."""
    w = SEEDED[case]()
    H, nb, D = w.planes.shape
    seed = 0x2007048250
    want = oracle.planes_from_seed(seed, H, nb, D).astype(np.float32)
    t = w.topk if variant == "iclustered" else 0
    got = run_gpu(w, t, seed=seed)
    gp = got["planes"]
    ulps = np.abs(gp.view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
    print("plane entries one ulp off the oracle's: %d of %d" % (int((ulps != 0).sum()), ulps.size))
    assert ulps.max() <= 1 and (ulps == 0).mean() >= 0.999
    again = run_gpu(w, t, seed=seed)
    assert np.array_equal(again["planes"], gp) and np.array_equal(again["out"], got["out"])
    other = run_gpu(w, t, seed=seed + 1)
    assert np.mean(other["planes"] == gp) < 0.01
    w.planes = gp
    w.name = "%s-seeded-%s" % (w.name, case)
    given = run_gpu(w, t)
    for key in ("codes", "assign", "out", "values"):
        assert np.array_equal(given[key], got[key]), key
    check_end_to_end(w, t)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_block_kmeans_ragged_and_empty(variant):
    """The several-block K-means drivers with empty, one-row, one-block and
    block-edge sequences in one batch (every block of an empty sequence must
    still describe empty member ranges, or empty centroid sums when the
    K-means kernel forms them)."""
    import paper_2007_04825_amd as ca
    w = gen.config_tiny(B=5, H=1, N=5000, d=32, C=100, L=4, topk=32)
    w.lengths = np.array([5000, 0, 1, 2049, 4097], np.int32)
    t = w.topk if variant == "iclustered" else 0
    ref = run_oracle(w, t, key="blockragged")
    try:
        for path in (2, 4, 5):
            ca.set_kmeans_path(path)
            print("driver %d" % path, flush=True)
            got = run_gpu(w, t)
            assert np.array_equal(got["assign"], ref["assign"]), "driver %d" % path
            assert np.array_equal(got["sizes"], ref["sizes"])
            np.testing.assert_allclose(got["centroids"], ref["qc"], rtol=0, atol=2e-6)
            compare_outputs(w, ref, got, t)
    finally:
        ca.set_kmeans_path(0)


def test_invalid_arguments_enqueue_nothing():
    """A rejected call (through the C ABI) returns its error code and leaves
    the output untouched: nothing was enqueued, also seen after the stream has
    drained."""
    import paper_2007_04825_amd as ca
    torch = pytest.importorskip("torch")
    stream = torch.cuda.current_stream().cuda_stream
    q = torch.zeros((1, 1, 64, 48), device="cuda")             # d = 48: unsupported
    planes = torch.zeros((1, 63, 48), device="cuda")
    out = torch.full((1, 1, 64, 48), 7.25, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    rc = ca.clustered_attention_fwd(q.data_ptr(), q.data_ptr(), q.data_ptr(), None, planes.data_ptr(),
                                    1, 1, 64, 48, ca.CA_F32, 10, 63, 3, 0, out.data_ptr(), ws.data_ptr(),
                                    1 << 20, None, stream)
    assert rc == ca.CA_ERR_UNSUPPORTED
    q32 = torch.zeros((1, 1, 64, 32), device="cuda")
    p32 = torch.zeros((1, 63, 32), device="cuda")
    out32 = torch.full((1, 1, 64, 32), 7.25, device="cuda")
    rc = ca.iclustered_attention_fwd(q32.data_ptr(), q32.data_ptr(), q32.data_ptr(), None,
                                     p32.data_ptr(), 1, 1, 64, 32, ca.CA_F32, 10, 63, 3, 0, 4,
                                     out32.data_ptr(), ws.data_ptr(), 16, None, stream)
    assert rc == ca.CA_ERR_WORKSPACE                        # 16 bytes: far too small
    rc = ca.iclustered_attention_fwd(q32.data_ptr(), q32.data_ptr(), q32.data_ptr(), None,
                                     p32.data_ptr(), 1, 1, 64, 32, ca.CA_F32, 0, 63, 3, 0, 4,
                                     out32.data_ptr(), ws.data_ptr(), 1 << 20, None, stream)
    assert rc == ca.CA_ERR_INVALID_ARG                      # no clusters
    torch.cuda.synchronize()
    assert bool((out == 7.25).all()) and bool((out32 == 7.25).all())


def near_orthogonal_queries(w, seed=0):
    """Every second query of each (sequence, head) is projected off one plane
    (in fp64, then stored in the workload dtype), so that its projection on
    that plane is a rounding-level number: the cases where the matrix-core
    estimate cannot decide the sign and the exact fp64 chain must."""
    q = w.q.astype(np.float64).copy()
    B, H, N, _ = q.shape
    for b in range(B):
        for h in range(H):
            p = w.planes[h].astype(np.float64)
            rows = np.arange(1, N, 2)
            pl = p[rows % w.n_bits]
            coef = np.sum(q[b, h, rows] * pl, axis=1) / np.sum(pl * pl, axis=1)
            q[b, h, rows] -= coef[:, None] * pl
    q = q.astype(np.float32)
    return gen.round_bf16(q) if w.dtype == "bf16" else q


def in_band_count(w):
    """Projections the kernels must recompute in fp64: |p| <= 2^-14 |q| |P|
    for fp32 queries, 2^-16 |q| |P| for bf16 ones (a single exact product per
    dimension leaves a narrower rounding band)."""
    band = 2.0 ** -14 if w.dtype == "f32" else 2.0 ** -16
    cnt = 0
    B, H = w.q.shape[:2]
    for b in range(B):
        n = int(w.lengths[b])
        for h in range(H):
            qq = w.q[b, h, :n].astype(np.float64)
            pp = w.planes[h].astype(np.float64)
            pr = qq @ pp.T
            lim = band * np.linalg.norm(qq, axis=1)[:, None] * np.linalg.norm(pp, axis=1)[None]
            cnt += int(np.sum(np.abs(pr) <= lim))
    return cnt


def oracle_codes(w):
    B, H, N, _ = w.q.shape
    codes = np.zeros((B, H, N), np.uint64)
    for b in range(B):
        n = int(w.lengths[b])
        for h in range(H):
            codes[b, h, :n] = oracle.hash_codes(w.q[b, h, :n], w.planes[h])
    return codes


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64])
def test_hash_exact_inside_rounding_band(path, dtype, d):
    """Hash codes equal the oracle's in every bit, including projections too
    close to zero for the bf16 matrix-core estimate (recomputed in fp64), on
    both the one-workgroup clustering kernel and the standalone hash kernel."""
    import dataclasses
    import paper_2007_04825_amd as ca
    base = gen.config_sweep(N=1000, B=2, H=2, d=d, dtype=dtype, C=20, L=2, topk=8)
    w = dataclasses.replace(base, q=near_orthogonal_queries(base), name=base.name + "_orth")
    nb = in_band_count(w)
    print("projections inside the band: %d" % nb)
    assert nb > 50
    ref = oracle_codes(w)
    try:
        ca.set_kmeans_path(path)
        got = run_gpu(w, 0)
    finally:
        ca.set_kmeans_path(0)
    assert np.array_equal(got["codes"], ref), "codes differ in %d rows" % int(np.sum(got["codes"] != ref))


@pytest.mark.parametrize("path", [1, 2])
def test_hash_planes_not_bf16(path):
    """Planes that are not bf16 values take the exact fp64 path for every
    projection; the codes still equal the oracle's."""
    import dataclasses
    import paper_2007_04825_amd as ca
    base = gen.config_tiny(B=1, H=2, N=700, d=64, C=16, L=2, topk=8)
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence([gen.SEED_ROOT, 1, 70, 0])))
    planes = g.standard_normal(base.planes.shape).astype(np.float32)
    assert np.any(planes.view(np.uint32) & 0xFFFF)
    w = dataclasses.replace(base, planes=planes, name=base.name + "_fp32planes")
    ref = oracle_codes(w)
    try:
        ca.set_kmeans_path(path)
        got = run_gpu(w, 0)
    finally:
        ca.set_kmeans_path(0)
    assert np.array_equal(got["codes"], ref)

"""Pins for the fp64 oracle: each test checks it against something other than
itself -- exact rational arithmetic, brute force on tiny inputs, closed forms,
textbook softmax attention, and the two propositions of the paper.

Which plausible mistakes each group catches is noted in its docstring."""
from fractions import Fraction

import numpy as np
import pytest

import gen
import oracle


def softmax_rows(x):
    x = x - x.max(axis=-1, keepdims=True)
    e = np.exp(x)
    return e / e.sum(axis=-1, keepdims=True)


def exact_attention(q, k, v):
    """Textbook softmax attention, Eq. (1)-(2), written with numpy."""
    q, k, v = (np.asarray(a, np.float64) for a in (q, k, v))
    a = softmax_rows(q @ k.T / np.sqrt(q.shape[1]))
    return a @ v, a


# --------------------------------------------------------------------------
# Hashing (Section 3.2.2).  Exact rational sign of every projection catches a
# wrong sign, a wrong plane index, a transposed operand or a wrong bit order.
# --------------------------------------------------------------------------

def exact_code(qi, planes):
    code = 0
    for b, p in enumerate(planes):
        s = sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(qi, p))
        if s > 0:
            code |= 1 << b
    return code


@pytest.mark.parametrize("seed,n,d,nb", [(0, 9, 4, 7), (1, 5, 16, 63), (2, 3, 32, 64), (3, 4, 8, 1)])
def test_hash_matches_exact_rational_sign(seed, n, d, nb):
    q, _, _ = gen.random_unit(seed, n, d)
    planes = gen.round_bf16(np.random.default_rng(seed).standard_normal((nb, d)).astype(np.float32))
    codes = oracle.hash_codes(q, planes)
    for i in range(n):
        assert int(codes[i]) == exact_code(q[i], planes)
    if nb < 64:
        assert np.all(codes >> np.uint64(nb) == 0)


def test_hash_exact_zero_projection_gives_zero_bit():
    q = np.array([[1.0, 1.0, 0.0, 0.0], [0.0, 0.0, 0.0, 0.0]], np.float32)
    planes = np.array([[1.0, -1.0, 0.0, 0.0], [1.0, 1.0, 0.0, 0.0], [-1.0, 0.0, 0.0, 0.0]], np.float32)
    codes = oracle.hash_codes(q, planes)
    assert int(codes[0]) == 0b010       # plane 0 gives exactly 0, plane 1 > 0, plane 2 < 0
    assert int(codes[1]) == 0           # the zero query hashes to 0


def test_hash_scale_and_negation_invariances():
    q, _, _ = gen.random_unit(5, 64, 64)
    planes = gen.hyperplanes(11, 1, 63, 64)[0]
    c = oracle.hash_codes(q, planes)
    assert np.array_equal(c, oracle.hash_codes(q * np.float32(8.0), planes))
    assert np.array_equal(c, oracle.hash_codes(q * np.float32(0.25), planes))
    proj = oracle.projections(q, planes)
    assert np.all(proj != 0)
    mask = np.uint64((1 << 63) - 1)
    assert np.array_equal(oracle.hash_codes(-q, planes), (~c) & mask)


def test_hash_collision_rate_is_angle_over_pi():
    """Sign random projections: P[bit differs] = angle / pi (Charikar 2002)."""
    g = np.random.default_rng(3)
    d, nb, pairs = 32, 63, 400
    planes = g.standard_normal((nb, d))
    x = g.standard_normal((pairs, d))
    y = g.standard_normal((pairs, d))
    y = 0.6 * x + 0.8 * y
    cx, cy = oracle.hash_codes(x, planes), oracle.hash_codes(y, planes)
    diff = np.array([bin(int(a) ^ int(b)).count("1") for a, b in zip(cx, cy)]) / nb
    cos = (x * y).sum(1) / np.linalg.norm(x, axis=1) / np.linalg.norm(y, axis=1)
    theta = np.arccos(np.clip(cos, -1, 1)) / np.pi
    assert abs(diff.mean() - theta.mean()) < 0.02


# --------------------------------------------------------------------------
# Hamming K-means (Section 3.2.2).  A naive bit-by-bit re-implementation on
# tiny inputs catches a wrong tie rule (assign or majority), an off-by-one in
# the number of rounds, a wrong initialisation or a wrong empty-cluster rule.
# --------------------------------------------------------------------------

def naive_kmeans(codes, C, L):
    codes = [int(c) for c in codes]
    n = len(codes)
    ce = min(C, n)
    cent = [codes[(j * n) // ce] for j in range(ce)]

    def ham(x, y):
        return sum(((x >> b) & 1) != ((y >> b) & 1) for b in range(64))

    assign = [0] * n
    for _ in range(L):
        for i in range(n):
            dists = [ham(codes[i], c) for c in cent]
            assign[i] = dists.index(min(dists))          # first minimum = smallest index
        for j in range(ce):
            members = [codes[i] for i in range(n) if assign[i] == j]
            if not members:
                continue
            new = 0
            for b in range(64):
                ones = sum((m >> b) & 1 for m in members)
                if ones > len(members) - ones:           # strict majority; tie -> 0
                    new |= 1 << b
            cent[j] = new
    return assign, cent


@pytest.mark.parametrize("seed", range(12))
def test_kmeans_equals_naive_on_tiny_inputs(seed):
    g = np.random.default_rng(seed)
    n = int(g.integers(1, 17))
    C = int(g.integers(1, 6))
    L = int(g.integers(1, 5))
    nbits = int(g.choice([4, 8, 63]))
    # few distinct bits so that distance ties and majority ties are frequent
    codes = g.integers(0, 2, size=(n, nbits))
    codes = np.array([sum(int(b) << i for i, b in enumerate(row)) for row in codes], np.uint64)
    a, cent, _ = oracle.kmeans(codes, C, L)
    na, nc = naive_kmeans(codes, C, L)
    assert list(a) == na
    assert [int(c) for c in cent[: len(nc)]] == nc


def test_kmeans_objective_non_increasing_and_final_argmin():
    w = gen.make_config(1)
    codes = oracle.hash_codes(w.q[0, 0], w.planes[0])
    L = 6
    a, cent, obj = oracle.kmeans(codes, 100, L)
    assert np.all(np.diff(obj) <= 0)
    # The last assignment is an argmin (smallest index on ties) for the
    # centroids produced by round L-1.
    _, cent_prev, _ = oracle.kmeans(codes, 100, L - 1)
    d = np.array([[bin(int(h) ^ int(c)).count("1") for c in cent_prev] for h in codes])
    assert np.array_equal(a, d.argmin(axis=1))


def test_kmeans_special_cases():
    g = np.random.default_rng(7)
    codes = np.unique(g.integers(0, 2**63, size=40, dtype=np.uint64))
    n = len(codes)
    a, _, _ = oracle.kmeans(codes, 1, 3)
    assert np.all(a == 0)
    a, cent, _ = oracle.kmeans(codes, n, 3)            # C = n with distinct codes
    assert np.array_equal(a, np.arange(n))
    assert np.array_equal(cent, codes)
    a, _, _ = oracle.kmeans(codes[:5], 50, 2)           # C > n: only n clusters in use
    assert np.array_equal(a, np.arange(5))


def test_kmeans_recovers_well_separated_mixture():
    g = np.random.default_rng(1)
    d, comps, n = 64, 20, 2000
    means = 3 * g.standard_normal((comps, d))
    z = g.integers(0, comps, n)
    q = means[z] + 0.3 * g.standard_normal((n, d))
    planes = g.standard_normal((63, d))
    a, _, _ = oracle.kmeans(oracle.hash_codes(q, planes), comps, 10)
    # purity: most queries share a cluster with the majority of their component
    purity = sum(np.bincount(a[z == c]).max() for c in range(comps) if np.any(z == c)) / n
    assert purity > 0.8


# --------------------------------------------------------------------------
# Centroids, Eq. (3): textbook mean of the members.
# --------------------------------------------------------------------------

def test_centroids_are_member_means():
    q, _, _ = gen.random_unit(4, 50, 16)
    a = np.random.default_rng(4).integers(0, 7, 50).astype(np.int32)
    a[a == 3] = 4                                      # cluster 3 empty
    qc, sizes = oracle.centroids(q, a, 7)
    for j in range(7):
        assert sizes[j] == np.sum(a == j)
        if sizes[j]:
            np.testing.assert_allclose(qc[j], q[a == j].astype(np.float64).mean(0), rtol=0, atol=1e-14)
            assert np.all(qc[j] >= q[a == j].min(0) - 1e-12) and np.all(qc[j] <= q[a == j].max(0) + 1e-12)
        else:
            assert np.all(qc[j] == 0)


# --------------------------------------------------------------------------
# Clustered attention, Eq. (4)-(6).  Singleton clusters reduce it to textbook
# attention (catches a dropped 1/sqrt(d), a transposed product, a wrong
# softmax axis); dense rows summing to 1 and equal member rows catch a wrong
# normalisation or broadcast index.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n,d", [(1, 8), (7, 32), (64, 64)])
def test_clustered_singletons_equal_exact_attention(n, d):
    q, k, v = gen.random_unit(n, n, d)
    out, _, _ = oracle.clustered_from_assign(q, k, v, np.arange(n), n)
    ref, _ = exact_attention(q, k, v)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_clustered_rows_sum_to_one_and_members_share_output():
    q, k, v = gen.random_unit(9, 80, 16)
    a = np.random.default_rng(9).integers(0, 6, 80).astype(np.int32)
    out, qc, vc = oracle.clustered_from_assign(q, k, v, a, 6)
    ac, _ = oracle.dense_rows(q, k, a, 6, 4)
    np.testing.assert_allclose(ac.sum(1), 1.0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out, ac @ v.astype(np.float64), rtol=0, atol=1e-12)
    for j in range(6):
        rows = out[a == j]
        assert np.all(rows == rows[0])
        ref, _ = exact_attention(qc[j:j + 1], k, v)   # the centroid attends like a query
        np.testing.assert_allclose(rows[0], ref[0], rtol=0, atol=1e-12)


def test_proposition_1_bound():
    """||softmax(Q_i K^T/sqrt d) - softmax(Q^c_j K^T/sqrt d)||_2 <=
    ||Q_i - Q^c_j||_2 ||K||_2 / sqrt d  (softmax is 1-Lipschitz)."""
    w = gen.make_config(1)
    q, k = w.q[0, 1][:256].astype(np.float64), w.k[0, 1][:256].astype(np.float64)
    a, _, _ = oracle.kmeans(oracle.hash_codes(q, w.planes[1]), 10, 5)
    qc, _ = oracle.centroids(q, a, 10)
    ac, _ = oracle.dense_rows(q, k, a, 10, 4)
    _, full = exact_attention(q, k, k)
    knorm = np.linalg.norm(k, 2)
    lhs = np.linalg.norm(full - ac, axis=1)
    rhs = np.linalg.norm(q - qc[a], axis=1) * knorm / np.sqrt(q.shape[1])
    assert np.all(lhs <= rhs + 1e-12)


# --------------------------------------------------------------------------
# Top-k selection (Section 3.3): brute force by a stable sort.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_topk_equals_stable_sort(seed):
    g = np.random.default_rng(seed)
    n = int(g.integers(1, 300))
    s = g.integers(-5, 6, n).astype(np.float64)          # many ties
    if seed % 2:
        s = g.standard_normal(n)
    for k in (1, 3, 32, 500):
        top = oracle.topk(s, k)
        order = np.lexsort((np.arange(n), -s))           # logit desc, index asc
        assert np.array_equal(top, np.sort(order[: min(k, n)]))


# --------------------------------------------------------------------------
# Improved clustered attention, Eq. (11) and the supplementary decomposition.
# k = n and singleton clusters reduce it to exact attention; the decomposed
# form must equal the dense A^t V; A^t rows sum to 1 (catches a dropped m_j or
# a rest part that still includes the top-k keys); Proposition 2 holds.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n,d,C", [(5, 8, 2), (40, 32, 4), (96, 64, 7)])
def test_iclustered_k_equals_n_is_exact(n, d, C):
    q, k, v = gen.random_unit(100 + n, n, d)
    a = np.random.default_rng(n).integers(0, C, n).astype(np.int32)
    out, T, mass, vb = oracle.iclustered_from_assign(q, k, v, a, C, n)
    ref, _ = exact_attention(q, k, v)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    used = np.unique(a)
    np.testing.assert_allclose(mass[used], 1.0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(vb[used], 0.0, rtol=0, atol=1e-12)


def test_iclustered_singletons_exact_for_any_k():
    q, k, v = gen.random_unit(77, 50, 16)
    ref, _ = exact_attention(q, k, v)
    for kk in (1, 5, 32):
        out, _, _, _ = oracle.iclustered_from_assign(q, k, v, np.arange(50), 50, kk)
        np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_iclustered_dense_form_rowsums_and_proposition_2(seed):
    w = gen.make_config(1)
    n = 128
    q, k, v = (x[0, seed][:n].astype(np.float64) for x in (w.q, w.k, w.v))
    C, kk = 8, 6
    a, _, _ = oracle.kmeans(oracle.hash_codes(q, w.planes[seed]), C, 5)
    out, T, mass, vb = oracle.iclustered_from_assign(q, k, v, a, C, kk)
    ac, at = oracle.dense_rows(q, k, a, C, kk)
    np.testing.assert_allclose(at.sum(1), 1.0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out, at @ v, rtol=0, atol=1e-12)
    _, full = exact_attention(q, k, v)
    lhs = np.abs(at - full).sum(1)
    rhs = np.abs(ac - full).sum(1)
    assert np.all(lhs <= rhs + 1e-12)
    for j in np.unique(a):
        assert 0 < mass[j] <= 1 + 1e-15
        row = ac[np.argmax(a == j)]
        np.testing.assert_allclose(mass[j], row[T[j][T[j] >= 0]].sum(), rtol=0, atol=1e-13)
        # the selected keys are the k largest entries of the centroid row
        order = np.lexsort((np.arange(n), -row))
        assert np.array_equal(T[j][: kk], np.sort(order[:kk]))


def test_zero_keys_closed_form():
    """K = 0: every logit is 0, so A^c is uniform, T_j is the first k keys
    (ties go to the smaller index), m = k/n, and both variants return mean(V)."""
    n, d, C, kk = 12, 4, 3, 5
    q, _, v = gen.random_unit(5, n, d)
    k = np.zeros((n, d), np.float32)
    a = (np.arange(n) % C).astype(np.int32)
    mean_v = v.astype(np.float64).mean(0)
    out, _, _ = oracle.clustered_from_assign(q, k, v, a, C)
    np.testing.assert_allclose(out, np.broadcast_to(mean_v, (n, d)), rtol=0, atol=1e-14)
    out, T, mass, vb = oracle.iclustered_from_assign(q, k, v, a, C, kk)
    assert np.all(T == np.arange(kk))
    np.testing.assert_allclose(mass, kk / n, rtol=0, atol=1e-15)
    np.testing.assert_allclose(vb, np.broadcast_to(v[kk:].astype(np.float64).sum(0) / n, (C, d)),
                               rtol=0, atol=1e-14)
    np.testing.assert_allclose(out, np.broadcast_to(mean_v, (n, d)), rtol=0, atol=1e-14)


# --------------------------------------------------------------------------
# Batched driver: padding, lengths, exports.
# --------------------------------------------------------------------------

def test_forward_masks_padding_and_matches_per_unit_path():
    w = gen.config_speech(B=3, H=2, N=60, d=8, C=7, L=4, topk=5, lengths=[0, 1, 37],
                          pad_value=np.nan)
    q = np.nan_to_num(w.q, nan=0.0)
    for topk in (0, 5):
        res = oracle.forward(w.q, w.k, w.v, w.lengths, w.planes, w.C, w.n_bits, w.L, topk)
        assert not np.isnan(res["out"]).any()
        for b in range(3):
            n = int(w.lengths[b])
            for h in range(2):
                assert np.all(res["out"][b, h, n:] == 0)
                assert np.all(res["assign"][b, h, n:] == -1)
                if n == 0:
                    continue
                codes = oracle.hash_codes(q[b, h, :n], w.planes[h])
                assert np.array_equal(res["codes"][b, h, :n], codes)
                a, _, _ = oracle.kmeans(codes, w.C, w.L)
                assert np.array_equal(res["assign"][b, h, :n], a)
                if topk:
                    out, T, _, _ = oracle.iclustered_from_assign(q[b, h, :n], w.k[b, h, :n],
                                                                 w.v[b, h, :n], a, w.C, topk)
                else:
                    out, _, _ = oracle.clustered_from_assign(q[b, h, :n], w.k[b, h, :n],
                                                             w.v[b, h, :n], a, w.C)
                np.testing.assert_array_equal(res["out"][b, h, :n], out)


# --------------------------------------------------------------------------
# Projection values (Section 3.2.2) and exact attention (Section 3.1, Eq. 1-2).
# The projections are pinned to exact rational dot products within the error
# bound of recursive fp64 summation (each product of two fp32 values is exact
# in fp64), and their packed signs must be the hash codes; a wrong plane
# index, a transposed operand or a wrong output layout fails.  Exact attention
# is pinned to numpy's softmax attention, to closed forms (zero keys give the
# mean value row, one key gives its value row) and to the permutation
# symmetries of the definition.
# --------------------------------------------------------------------------

def gamma(m):
    u = 2.0 ** -53
    return m * u / (1 - m * u)


@pytest.mark.parametrize("seed,n,d,nb,bf16_planes", [(0, 9, 4, 7, True), (1, 6, 32, 63, True),
                                                     (2, 5, 64, 64, False), (3, 3, 8, 1, False)])
def test_projections_match_exact_rational_dot_products(seed, n, d, nb, bf16_planes):
    q, _, _ = gen.random_unit(20 + seed, n, d)
    planes = np.random.default_rng(seed).standard_normal((nb, d)).astype(np.float32)
    if bf16_planes:
        planes = gen.round_bf16(planes)
    proj = oracle.projections(q, planes)
    assert proj.shape == (n, nb)
    for i in range(n):
        for b in range(nb):
            terms = [Fraction(float(x)) * Fraction(float(y)) for x, y in zip(q[i], planes[b])]
            exact = sum(terms)
            bound = gamma(d - 1) * float(sum(abs(t) for t in terms))
            assert abs(float(Fraction(float(proj[i, b])) - exact)) <= bound
    packed = np.zeros(n, np.uint64)
    for b in range(nb):
        packed |= (proj[:, b] > 0).astype(np.uint64) << np.uint64(b)
    assert np.array_equal(packed, oracle.hash_codes(q, planes))


@pytest.mark.parametrize("n,d", [(1, 4), (13, 8), (70, 32), (33, 64)])
def test_full_attention_equals_numpy_softmax_attention(n, d):
    q, k, v = gen.random_unit(300 + n, n, d, scale=1.5)
    out = oracle.full_attention(q, k, v)
    ref, _ = exact_attention(q, k, v)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    if n == 1:
        np.testing.assert_array_equal(out, v.astype(np.float64))     # one key: its value row


def test_full_attention_closed_forms_and_symmetries():
    n, d = 24, 16
    q, k, v = gen.random_unit(41, n, d)
    # zero keys: uniform weights, every row is the mean value row
    out0 = oracle.full_attention(q, np.zeros_like(k), v)
    np.testing.assert_allclose(out0, np.broadcast_to(v.astype(np.float64).mean(0), (n, d)),
                               rtol=0, atol=1e-14)
    out = oracle.full_attention(q, k, v)
    perm = np.random.default_rng(41).permutation(n)
    # a joint permutation of keys and values leaves every row unchanged ...
    np.testing.assert_allclose(oracle.full_attention(q, k[perm], v[perm]), out, rtol=0, atol=1e-13)
    # ... and a permutation of the queries permutes the rows
    np.testing.assert_allclose(oracle.full_attention(q[perm], k, v), out[perm], rtol=0, atol=1e-13)
    # the 1/sqrt(d) scale: doubling q and halving k changes nothing
    np.testing.assert_allclose(oracle.full_attention(2 * q, k / 2, v), out, rtol=0, atol=1e-13)
    # singleton clusters of the clustered oracle are exact attention
    sing, _, _ = oracle.clustered_from_assign(q, k, v, np.arange(n), n)
    np.testing.assert_allclose(sing, out, rtol=0, atol=1e-12)


def test_centroid_row_logits_and_softmax():
    """Eq. (4) for one row: logits Q^c_j . K_l / sqrt(d) and their softmax."""
    q, k, _ = gen.random_unit(51, 40, 32)
    qc = q[:7].astype(np.float64).mean(0)
    s, a = oracle.centroid_row(qc, k)
    np.testing.assert_allclose(s, k.astype(np.float64) @ qc / np.sqrt(32), rtol=0, atol=1e-13)
    np.testing.assert_allclose(a, softmax_rows(s[None])[0], rtol=0, atol=1e-15)
    assert abs(a.sum() - 1.0) < 1e-14

"""Pins of the oracle-top oracle (the comparison variant of Sec. 4.2 that keeps
each query's k keys of highest attention) against what the definition fixes:
exact softmax attention when k >= n, hard attention when k = 1, a brute-force
search over key subsets, the tie rule, invariance under a joint permutation of
the keys and values, and the masking of a padded batch."""
import itertools

import numpy as np
import pytest
from scipy.special import softmax

import oracle


def rand(n, d, seed):
    r = np.random.default_rng(seed)
    return (r.standard_normal((n, d)) for _ in range(3))


@pytest.mark.parametrize("n,d,k", [(1, 4, 1), (5, 8, 5), (9, 16, 32), (40, 32, 40)])
def test_k_at_least_n_is_exact_attention(n, d, k):
    q, kk, v = rand(n, d, 1)
    out, t = oracle.oracle_top_unit(q, kk, v, k)
    ref = softmax(q @ kk.T / np.sqrt(d), axis=1) @ v
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)
    ke = min(k, n)
    assert np.array_equal(t[:, :ke], np.broadcast_to(np.arange(ke), (n, ke)))
    assert np.all(t[:, ke:] == -1)


def test_k_one_is_hard_attention():
    q, kk, v = rand(30, 8, 2)
    out, t = oracle.oracle_top_unit(q, kk, v, 1)
    best = np.argmax(q @ kk.T, axis=1)
    np.testing.assert_array_equal(t[:, 0], best)
    np.testing.assert_allclose(out, v[best], rtol=0, atol=0)


@pytest.mark.parametrize("n,k", [(6, 2), (7, 3), (8, 4)])
def test_brute_force_subsets(n, k):
    """The top-k set is the k-subset with the largest sum of logits (logits are
    distinct here), and the output is the softmax over that subset alone."""
    d = 4
    q, kk, v = rand(n, d, 10 + n)
    out, t = oracle.oracle_top_unit(q, kk, v, k)
    s = q @ kk.T / np.sqrt(d)
    for i in range(n):
        best = max(itertools.combinations(range(n), k), key=lambda c: s[i, list(c)].sum())
        assert list(t[i]) == list(best)
        w = softmax(s[i, list(best)])
        np.testing.assert_allclose(out[i], w @ v[list(best)], rtol=0, atol=1e-14)


def test_ties_go_to_the_smaller_key_index():
    q, kk, v = rand(8, 4, 3)
    kk[5] = kk[2]  # keys 2 and 5 give every query the same logit
    v[5] = v[2] + 10.0
    s = q @ kk.T
    for i in range(8):
        order = np.argsort(-s[i], kind="stable")
        rank = int(np.where(order == 2)[0][0])  # key 2 comes first among the tied pair
        k_cut = rank + 1  # exactly one of the pair fits
        out, t = oracle.oracle_top_unit(q, kk, v, k_cut)
        assert 2 in t[i] and 5 not in t[i]


def test_joint_permutation_of_keys_and_values():
    q, kk, v = rand(24, 8, 4)
    out, t = oracle.oracle_top_unit(q, kk, v, 5)
    perm = np.random.default_rng(5).permutation(24)
    out_p, t_p = oracle.oracle_top_unit(q, kk[perm], v[perm], 5)
    np.testing.assert_allclose(out_p, out, rtol=0, atol=1e-14)
    for i in range(24):
        assert sorted(perm[t_p[i]].tolist()) == t[i].tolist()


def test_padded_batch():
    r = np.random.default_rng(6)
    B, H, N, d, k = 3, 2, 20, 8, 4
    q, kk, v = (r.standard_normal((B, H, N, d)) for _ in range(3))
    lengths = np.array([20, 7, 1], np.int32)
    out, t = oracle.oracle_top(q, kk, v, lengths, k, num_threads=2)
    for b in range(B):
        n = lengths[b]
        for h in range(H):
            o1, t1 = oracle.oracle_top_unit(q[b, h, :n], kk[b, h, :n], v[b, h, :n], k)
            np.testing.assert_array_equal(out[b, h, :n], o1)
            np.testing.assert_array_equal(t[b, h, :n], t1)
            assert np.all(out[b, h, n:] == 0) and np.all(t[b, h, n:] == -1)
            assert np.all(t[b, h, :n] < n)


def test_rejects_bad_lengths():
    q = np.zeros((1, 1, 4, 4))
    with pytest.raises(ValueError):
        oracle.oracle_top(q, q, q, np.array([5], np.int32), 2)

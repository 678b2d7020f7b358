"""Pins for the oracle's backward pass (gradients with the partition and the
top-k sets held constant).

* Central finite differences of the oracle's own forward pass: a dropped
  term, a wrong sign, a missing 1/sqrt(d) or 1/|S_j| factor, or a transposed
  operand anywhere in the chain shows up as a disagreement of order 1.
* Exact softmax attention differentiated by torch autograd in fp64: singleton
  clusters (both variants) and k = n (improved) reduce the method to exact
  attention as a function of (Q, K, V), so the gradients must agree.
* Translation invariance: adding one vector to every key leaves every
  softmax unchanged, so the key gradients sum to zero."""
import numpy as np
import pytest
import torch

import gen
import oracle


def _inputs(seed, n, d, C):
    rng = np.random.default_rng(1000 + seed)
    q, k, v, g = (rng.standard_normal((n, d)) for _ in range(4))
    assign = rng.integers(0, C, n).astype(np.int32)
    assign[:C] = np.arange(C)  # no empty cluster
    rng.shuffle(assign)
    return q, k, v, g, assign


def _loss(fwd, q, k, v, g):
    return float((fwd(q, k, v) * g).sum())


def _fd_grads(fwd, q, k, v, g, h=1e-6):
    """Central differences of L = sum(out * g) in every input coordinate."""
    grads = []
    for which in range(3):
        base = [q.copy(), k.copy(), v.copy()]
        x = base[which]
        gx = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + h
            lp = _loss(fwd, *base, g)
            x[idx] = old - h
            lm = _loss(fwd, *base, g)
            x[idx] = old
            gx[idx] = (lp - lm) / (2 * h)
        grads.append(gx)
    return grads


def _exact_grads(q, k, v, g):
    """Gradients of sum(softmax(q k^T / sqrt(d)) v * g) by torch autograd, fp64."""
    tq, tk, tv = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v))
    a = torch.softmax(tq @ tk.T / np.sqrt(q.shape[1]), dim=-1)
    ((a @ tv) * torch.tensor(g, dtype=torch.float64)).sum().backward()
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("seed,n,d,C", [(0, 9, 4, 3), (1, 12, 3, 5), (2, 7, 5, 1)])
def test_clustered_backward_matches_finite_differences(seed, n, d, C):
    q, k, v, g, assign = _inputs(seed, n, d, C)
    fwd = lambda q_, k_, v_: oracle.clustered_from_assign(q_, k_, v_, assign, C)[0]
    want = _fd_grads(fwd, q, k, v, g)
    got = oracle.clustered_backward(q, k, v, assign, C, g)
    for w, x in zip(want, got):
        np.testing.assert_allclose(x, w, atol=2e-7, rtol=0)


@pytest.mark.parametrize("seed,n,d,C,topk", [(0, 10, 4, 3, 3), (1, 12, 3, 4, 5), (2, 9, 5, 2, 1),
                                             (3, 8, 4, 3, 8)])
def test_iclustered_backward_matches_finite_differences(seed, n, d, C, topk):
    q, k, v, g, assign = _inputs(seed, n, d, C)
    _, T, _, _ = oracle.iclustered_from_assign(q, k, v, assign, C, topk)
    fwd = lambda q_, k_, v_: oracle.iclustered_from_assign(q_, k_, v_, assign, C, topk, topk_in=T)[0]
    want = _fd_grads(fwd, q, k, v, g)
    got = oracle.iclustered_backward(q, k, v, assign, C, topk, g, topk_in=T)
    for w, x in zip(want, got):
        np.testing.assert_allclose(x, w, atol=2e-7, rtol=0)
    # selecting T inside the backward gives the same sets, hence the same gradients
    got2 = oracle.iclustered_backward(q, k, v, assign, C, topk, g)
    for a, b in zip(got, got2):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("n,d", [(6, 4), (17, 8)])
def test_singleton_clusters_give_exact_attention_gradients(n, d):
    q, k, v, g, _ = _inputs(5, n, d, n)
    ident = np.arange(n, dtype=np.int32)
    want = _exact_grads(q, k, v, g)
    for got in (oracle.clustered_backward(q, k, v, ident, n, g),
                oracle.iclustered_backward(q, k, v, ident, n, 3, g),
                oracle.iclustered_backward(q, k, v, ident, n, 1, g)):
        for w, x in zip(want, got):
            np.testing.assert_allclose(x, w, atol=1e-12, rtol=1e-10)


@pytest.mark.parametrize("n,d,C", [(10, 4, 3), (16, 8, 5)])
def test_iclustered_k_equals_n_gives_exact_attention_gradients(n, d, C):
    q, k, v, g, assign = _inputs(6, n, d, C)
    want = _exact_grads(q, k, v, g)
    got = oracle.iclustered_backward(q, k, v, assign, C, n, g)
    for w, x in zip(want, got):
        np.testing.assert_allclose(x, w, atol=1e-12, rtol=1e-10)


@pytest.mark.parametrize("topk", [0, 3])
def test_key_gradients_sum_to_zero_and_members_share_centroid_gradient(topk):
    q, k, v, g, assign = _inputs(7, 20, 6, 4)
    if topk:
        dq, dk, dv = oracle.iclustered_backward(q, k, v, assign, 4, topk, g)
    else:
        dq, dk, dv = oracle.clustered_backward(q, k, v, assign, 4, g)
        for j in range(4):  # Eq. (3): every member receives dQ^c_j / |S_j|
            rows = dq[assign == j]
            np.testing.assert_array_equal(rows, np.broadcast_to(rows[0], rows.shape))
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, atol=1e-12)


def test_batch_backward_masks_padding_and_matches_per_unit_path():
    w = gen.config_speech(B=3, H=2, N=40, d=8, C=6, L=3, topk=4, lengths=[40, 23, 0])
    rng = np.random.default_rng(9)
    dout = rng.standard_normal(w.q.shape)
    for topk in (0, w.topk):
        fw = oracle.forward(w.q, w.k, w.v, w.lengths, w.planes, w.C, w.n_bits, w.L, topk)
        dq, dk, dv = oracle.backward(w.q, w.k, w.v, w.lengths, w.C, topk, fw["assign"],
                                     fw["topk"] if topk else None, dout)
        for b in range(3):
            n = int(w.lengths[b])
            for h in range(2):
                for x in (dq, dk, dv):
                    assert np.all(x[b, h, n:] == 0)
                if n == 0:
                    continue
                args = (w.q[b, h, :n], w.k[b, h, :n], w.v[b, h, :n], fw["assign"][b, h, :n], w.C)
                if topk:
                    ref = oracle.iclustered_backward(*args, topk, dout[b, h, :n],
                                                     topk_in=fw["topk"][b, h])
                else:
                    ref = oracle.clustered_backward(*args, dout[b, h, :n])
                for x, r in zip((dq, dk, dv), ref):
                    np.testing.assert_array_equal(x[b, h, :n], r)

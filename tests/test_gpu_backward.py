"""GPU parity of the backward pass (clustered and improved), through the C ABI,
against the fp64 oracle's gradients for the same partition and top-k sets.

Tolerance (derived in the design notes from the fp32 arithmetic): every
gradient component must satisfy |gpu - oracle| <= 2e-5 * max(1, max |oracle|)
over its tensor, for fp32 and for bf16 inputs alike (bf16 inputs are exact
bf16 values that the oracle widens without rounding, so the only error is the
kernels' fp32 arithmetic).  Padded rows must be exactly 0."""
import numpy as np
import pytest

import gen
from gpu_util import oracle_backward_for, run_gpu_backward, valid_mask

pytestmark = pytest.mark.gpu

REL = 2e-5


def check_grads(w, topk, got, ref, vm, label=""):
    for name, x, r in zip(("dq", "dk", "dv"), got, ref):
        scale = max(1.0, float(np.abs(r[vm]).max()))
        err = float(np.abs(x - r)[vm].max())
        print("%s %s: max abs err %.3g, scale %.3g, rel %.3g" % (label, name, err, scale, err / scale))
        assert np.all(x[~vm] == 0), "%s padded rows must be 0" % name
        assert err <= REL * scale, "%s: %.3g > %.3g" % (name, err, REL * scale)


def run_case(w, topk, extra=0, pad_value=0.0):
    dout = gen.output_gradient(w, extra=extra, pad_value=pad_value)
    grads, fwd = run_gpu_backward(w, topk, dout)
    ref = oracle_backward_for(w, topk, dout, fwd)
    check_grads(w, topk, grads[0], ref, valid_mask(w), label="%s k=%d" % (w.name, topk))
    return grads, fwd


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_backward_tiny(variant):
    w = gen.config_tiny()
    run_case(w, w.topk if variant == "iclustered" else 0)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_backward_speech_full_size(variant):
    w = gen.config_speech()
    run_case(w, w.topk if variant == "iclustered" else 0)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_backward_encoder_bf16(variant):
    w = gen.config_encoder()
    run_case(w, w.topk if variant == "iclustered" else 0)


@pytest.mark.parametrize("N,dtype", [(2048, "f32"), (4096, "bf16")])
@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_backward_several_key_chunks(N, dtype, variant):
    w = gen.config_sweep(N, dtype=dtype, H=4)
    run_case(w, w.topk if variant == "iclustered" else 0)


@pytest.mark.parametrize("variant", ["clustered", "iclustered"])
def test_backward_ragged_nan_padding(variant):
    lens = [0, 1, 2, 15, 16, 17, 31, 33, 64, 99, 100, 101, 127, 128, 129, 300]
    w = gen.config_speech(B=len(lens), H=2, N=300, d=32, C=100, L=4, topk=32, lengths=lens,
                          pad_value=np.nan)
    run_case(w, w.topk if variant == "iclustered" else 0, pad_value=np.nan)


@pytest.mark.parametrize("C,topk", [(1, 1), (17, 128), (256, 64), (5, 7)])
def test_backward_parameter_corners(C, topk):
    w = gen.config_tiny(B=2, H=2, N=700, d=64, C=C, L=3, topk=topk)
    w.lengths = np.array([700, 517], np.int32)
    run_case(w, topk)


def test_backward_is_deterministic():
    w = gen.config_speech(B=4, H=2)
    for topk in (0, w.topk):
        dout = gen.output_gradient(w, extra=3)
        grads, _ = run_gpu_backward(w, topk, dout, repeat=2)
        for a, b in zip(grads[0], grads[1]):
            assert np.array_equal(a, b)


@pytest.mark.parametrize("topk", [0, 5])
def test_backward_singletons_equal_exact_attention_gradient(topk):
    """C = n with the identity partition: both variants are exact softmax
    attention, so the GPU gradients must equal torch autograd's (fp64, CPU)."""
    import torch
    n = 200
    w = gen.config_tiny(B=1, H=2, N=n, d=32, C=n, L=1, topk=max(topk, 1))
    ident = np.broadcast_to(np.arange(n, dtype=np.int32), (2, n)).copy()
    dout = gen.output_gradient(w, extra=5)
    grads, _ = run_gpu_backward(w, topk, dout, assign_in=ident)
    for h in range(2):
        tq, tk, tv = (torch.tensor(x[0, h], dtype=torch.float64, requires_grad=True)
                      for x in (w.q, w.k, w.v))
        a = torch.softmax(tq @ tk.T / np.sqrt(32), dim=-1)
        ((a @ tv) * torch.tensor(dout[0, h], dtype=torch.float64)).sum().backward()
        for x, r in zip(grads[0], (tq.grad, tk.grad, tv.grad)):
            r = r.numpy()
            assert np.abs(x[0, h] - r).max() <= REL * max(1.0, np.abs(r).max())


def test_backward_flags_terms_beyond_the_fixed_point_range():
    """The top-k parts of dK and dV are summed as 64-bit fixed-point integers
    that hold terms up to 2^22 in magnitude.  An output gradient scaled far
    beyond that must mark the affected entries as NaN (not clamp them), and
    only entries of keys that some top-k set holds; dQ stays finite."""
    w = gen.config_tiny(B=1, H=2, N=512, d=32, C=20, L=4, topk=8)
    dout = gen.output_gradient(w) * np.float32(1e9)
    grads, fwd = run_gpu_backward(w, w.topk, dout)
    dq, dk, dv = grads[0]
    assert np.isfinite(dq).all()
    B, H, N, _ = w.q.shape
    held = np.zeros((B, H, N), bool)
    for b in range(B):
        for h in range(H):
            t = fwd["topk"][b, h].reshape(-1)
            held[b, h, t[t >= 0]] = True
    flagged = np.isnan(dk).any(axis=-1) | np.isnan(dv).any(axis=-1)
    print("flagged keys: %d of %d held by a top-k set" % (int(flagged.sum()), int(held.sum())))
    assert flagged.any()
    assert not (flagged & ~held).any()
    assert np.isfinite(dk[~held]).all() and np.isfinite(dv[~held]).all()

"""Seeded synthetic workloads for clustered / improved-clustered attention.

This module only draws inputs: it holds none of the method's arithmetic and is
the one piece shared by the tests, the benchmark and the oracle driver.

Every array is drawn in fp64 from numpy's Philox counter-based generator,
seeded by ``SeedSequence([200704825, config, stream, extra])``, rounded to
fp32 (round-to-nearest-even), and, where the workload is bf16, rounded again to
the nearest bf16 value (ties to even) while being stored in a float32 array.
The stream ids are: 0 query noise, 1 keys, 2 values, 3 mixture means,
4 query labels, 5 lengths, 6 drift phases, 7 hyperplanes, 8 key labels,
9 output gradients (backward-pass tests and benchmark).

The paper's workloads (speech encoders on WSJ / Switchboard, a RoBERTa encoder
on GLUE / SQuAD, and the synthetic length sweep of its time benchmark) are
represented only by their shapes, lengths and value statistics: no dataset
content is reproduced.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_ROOT = 200704825


def rng(config: int, stream: int, extra: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence(
        [SEED_ROOT, int(config), int(stream), int(extra)])))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 value (ties to even); fp32 storage."""
    u = np.array(x, dtype=np.float32).view(np.uint32)  # a copy
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)  # wraps modulo 2^32, like the 64-bit form truncated
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


def hyperplanes(config: int, heads: int, n_bits: int, d: int, extra: int = 0) -> np.ndarray:
    """Hash planes [heads, n_bits, d]: iid N(0, 1), rounded to bf16 values."""
    p = rng(config, 7, extra).standard_normal((heads, n_bits, d))
    return round_bf16(p.astype(np.float32))


@dataclass
class Workload:
    name: str
    q: np.ndarray            # [B, H, N, d] float32 (bf16-representable when dtype == 'bf16')
    k: np.ndarray
    v: np.ndarray
    lengths: np.ndarray      # [B] int32
    planes: np.ndarray       # [H, n_bits, d] float32, bf16-representable
    C: int
    n_bits: int
    L: int
    topk: int
    dtype: str               # 'f32' or 'bf16'
    variants: tuple = ("clustered", "iclustered")
    meta: dict = field(default_factory=dict)

    @property
    def shape(self):
        return self.q.shape

    def queries(self) -> int:
        return int(self.lengths.astype(np.int64).sum()) * self.q.shape[1]


def _mixture(config, B, H, N, d, n_comp, sigma, stream_means=3, stream_labels=4,
             stream_noise=0, scale=1.0, extra=0):
    means = rng(config, stream_means, extra).standard_normal((B, H, n_comp, d))
    labels = rng(config, stream_labels, extra).integers(0, n_comp, size=(B, H, N))
    noise = rng(config, stream_noise, extra).standard_normal((B, H, N, d))
    x = scale * np.take_along_axis(means, labels[..., None], axis=2)
    return x + sigma * noise


def _finish(x, dtype):
    x = x.astype(np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def config_tiny(B=1, H=4, N=1024, d=64, C=100, n_bits=63, L=10, topk=32, seed_cfg=1):
    """Tiny case: queries from a 100-component Gaussian mixture (means N(0,1),
    sigma 0.3), keys and values iid N(0, 1); fp32."""
    q = _mixture(seed_cfg, B, H, N, d, 100, 0.3)
    k = rng(seed_cfg, 1).standard_normal((B, H, N, d))
    v = rng(seed_cfg, 2).standard_normal((B, H, N, d))
    return Workload("tiny_b%dh%dn%dd%d_f32" % (B, H, N, d), _finish(q, "f32"), _finish(k, "f32"),
                    _finish(v, "f32"), np.full(B, N, np.int32),
                    hyperplanes(seed_cfg, H, n_bits, d), C, n_bits, L, topk, "f32")


def config_speech(B=32, H=6, N=800, d=32, C=100, n_bits=63, L=10, topk=32, seed_cfg=2,
                  min_len=400, pad_value=0.0, lengths=None):
    """Speech-encoder-shaped layer: lengths uniform in [min_len, N], Q/K/V iid
    N(0,1) plus a sinusoid of period 100 steps along time with a random phase
    per (head, channel), drawn separately for Q, K and V; fp32.  Rows past a
    sample's length hold pad_value.  ``lengths`` overrides the drawn lengths."""
    if lengths is None:
        lengths = rng(seed_cfg, 5).integers(min_len, N + 1, size=B)
    lengths = np.asarray(lengths, dtype=np.int32)
    t = np.arange(N, dtype=np.float64)[None, None, :, None]
    phases = rng(seed_cfg, 6).uniform(0.0, 2 * np.pi, size=(3, 1, H, 1, d))
    out = []
    for which, stream in enumerate((0, 1, 2)):
        x = rng(seed_cfg, stream).standard_normal((B, H, N, d))
        x = x + np.sin(2 * np.pi * t / 100.0 + phases[which])
        x = x.astype(np.float32)
        mask = np.arange(N)[None, None, :, None] >= lengths[:, None, None, None]
        x = np.where(mask, np.float32(pad_value), x)
        out.append(x.astype(np.float32))
    return Workload("speech_b%dh%dn%dd%d_f32" % (B, H, N, d), out[0], out[1], out[2], lengths,
                    hyperplanes(seed_cfg, H, n_bits, d), C, n_bits, L, topk, "f32")


def config_sweep(N, dtype="f32", B=1, H=8, d=64, C=100, n_bits=63, L=10, topk=32, seed_cfg=3):
    """Length sweep: Q, K, V iid N(0, 1); the bf16 variant rounds the same fp32
    draw."""
    q = rng(seed_cfg, 0, N).standard_normal((B, H, N, d))
    k = rng(seed_cfg, 1, N).standard_normal((B, H, N, d))
    v = rng(seed_cfg, 2, N).standard_normal((B, H, N, d))
    return Workload("sweep_b%dh%dn%dd%d_%s" % (B, H, N, d, dtype), _finish(q, dtype),
                    _finish(k, dtype), _finish(v, dtype), np.full(B, N, np.int32),
                    hyperplanes(seed_cfg, H, n_bits, d, N), C, n_bits, L, topk, dtype)


def config_encoder(B=8, H=12, N=512, d=64, C=25, n_bits=63, L=10, topk=32, seed_cfg=4):
    """Pretrained-encoder-shaped approximation: 25 mixture means N(0, I);
    Q = mu[zq] + 0.3 eps, K = 1.5 mu[zk] + 0.3 eps' with independent labels,
    V iid N(0,1); bf16 storage.  Matching query/key pairs give logits near 12,
    others spread about N(0, 1.5^2): peaked, heavy-tailed attention rows."""
    means = rng(seed_cfg, 3).standard_normal((B, H, 25, d))
    zq = rng(seed_cfg, 4).integers(0, 25, size=(B, H, N))
    zk = rng(seed_cfg, 8).integers(0, 25, size=(B, H, N))
    eq = rng(seed_cfg, 0).standard_normal((B, H, N, d))
    ek = rng(seed_cfg, 1).standard_normal((B, H, N, d))
    q = np.take_along_axis(means, zq[..., None].repeat(d, -1), axis=2) + 0.3 * eq
    k = 1.5 * np.take_along_axis(means, zk[..., None].repeat(d, -1), axis=2) + 0.3 * ek
    v = rng(seed_cfg, 2).standard_normal((B, H, N, d))
    return Workload("encoder_b%dh%dn%dd%d_bf16" % (B, H, N, d), _finish(q, "bf16"),
                    _finish(k, "bf16"), _finish(v, "bf16"), np.full(B, N, np.int32),
                    hyperplanes(seed_cfg, H, n_bits, d), C, n_bits, L, topk, "bf16")


def config_long(B=1, H=8, N=65536, d=64, C=200, n_bits=63, L=15, topk=64, seed_cfg=5):
    """Long-context stress: queries from a 200-component mixture (sigma 0.3),
    K, V iid N(0, 1); bf16 storage; improved clustered attention only."""
    q = _mixture(seed_cfg, B, H, N, d, 200, 0.3)
    k = rng(seed_cfg, 1).standard_normal((B, H, N, d))
    v = rng(seed_cfg, 2).standard_normal((B, H, N, d))
    return Workload("long_b%dh%dn%dd%d_bf16" % (B, H, N, d), _finish(q, "bf16"),
                    _finish(k, "bf16"), _finish(v, "bf16"), np.full(B, N, np.int32),
                    hyperplanes(seed_cfg, H, n_bits, d), C, n_bits, L, topk, "bf16",
                    variants=("iclustered",))


def config_random(seed: int) -> Workload:
    """Seeded random shapes for broad parity checks: batch 1-3, heads 1-3,
    N from 1 to 3000 (small and chunk-edge sizes favoured), d 32 or 64, fp32
    or bf16, C 1-256, n_bits 1-63, L 1-12, k 1-128, ragged lengths (the first
    sequence full, the others uniform in [0, N]); queries from a Gaussian
    mixture of about C / 2 components (sigma 0.3), keys and values iid N(0, 1),
    padded rows 0."""
    r = np.random.default_rng([seed, 77])
    B = int(r.integers(1, 4))
    H = int(r.integers(1, 4))
    N = int(r.choice([1, 2, 5, 16, 17, 63, 100, 257, 600, 1024, 1025, 2100, 3000]))
    d = int(r.choice([32, 64]))
    dtype = str(r.choice(["f32", "bf16"]))
    C = int(r.choice([1, 3, 16, 17, 100, 256]))
    n_bits = int(r.choice([1, 8, 31, 63]))
    L = int(r.integers(1, 13))
    topk = int(r.choice([1, 2, 16, 32, 33, 64, 128]))
    lengths = r.integers(0, N + 1, size=B).astype(np.int32)
    lengths[0] = N
    q = _mixture(10, B, H, N, d, max(1, C // 2), 0.3, extra=seed)
    k = rng(10, 1, seed).standard_normal((B, H, N, d))
    v = rng(10, 2, seed).standard_normal((B, H, N, d))
    mask = np.arange(N)[None, None, :, None] >= lengths[:, None, None, None]
    q, k, v = (np.where(mask, 0.0, x) for x in (q, k, v))
    return Workload("random%d_b%dh%dn%dd%d_%s" % (seed, B, H, N, d, dtype), _finish(q, dtype),
                    _finish(k, dtype), _finish(v, dtype), lengths, hyperplanes(10, H, n_bits, d, seed),
                    C, n_bits, L, topk, dtype)


def with_dtype(w: Workload, dtype: str) -> Workload:
    """The same workload stored as dtype: 'bf16' rounds Q, K and V to the
    nearest bf16 values, 'f32' leaves them."""
    import dataclasses
    if dtype == w.dtype:
        return w
    if dtype != "bf16" or w.dtype != "f32":
        raise ValueError("only fp32 -> bf16 is supported")
    return dataclasses.replace(w, q=round_bf16(w.q), k=round_bf16(w.k), v=round_bf16(w.v),
                               dtype="bf16", name=w.name.replace("_f32", "") + "_bf16")


def make_config(cfg: int, **kw) -> Workload:
    """The five workloads: 1 tiny, 2 speech, 3 sweep (pass N=, dtype=), 4 encoder,
    5 long."""
    if cfg == 1:
        return config_tiny(**kw)
    if cfg == 2:
        return config_speech(**kw)
    if cfg == 3:
        return config_sweep(**kw)
    if cfg == 4:
        return config_encoder(**kw)
    if cfg == 5:
        return config_long(**kw)
    raise ValueError("unknown workload %r" % cfg)


def random_unit(seed, n, d, scale=1.0, dtype="f32"):
    """Small iid-normal (q, k, v) of one (batch, head), for property tests."""
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence([SEED_ROOT, 99, int(seed)])))
    x = (scale * g.standard_normal((3, n, d))).astype(np.float32)
    if dtype == "bf16":
        x = round_bf16(x)
    return x[0], x[1], x[2]


def output_gradient(w: Workload, extra: int = 0, pad_value: float = 0.0) -> np.ndarray:
    """An upstream gradient for the attention output of workload w: iid N(0, 1)
    of the output's shape, rounded like the inputs (fp32, then bf16 for bf16
    workloads); rows past each sequence's length hold pad_value."""
    cfg = {"tiny": 1, "speech": 2, "sweep": 3, "encoder": 4, "long": 5}.get(w.name.split("_")[0], 0)
    g = rng(cfg, 9, extra).standard_normal(w.q.shape).astype(np.float32)
    if w.dtype == "bf16":
        g = round_bf16(g)
    N = w.q.shape[2]
    pad = np.arange(N)[None, None, :, None] >= w.lengths[:, None, None, None]
    return np.where(pad, np.float32(pad_value), g).astype(np.float32)

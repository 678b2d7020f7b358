"""fp64 CPU oracle for clustered / improved-clustered attention.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never calls it and shares no code with it.

The arithmetic lives in ``oracle.c`` (plain C, fp64); this module compiles it
with gcc when needed and wraps it with numpy through ctypes.  Every input is
widened to float64 exactly (fp32 and bf16 values are representable in fp64).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_HDR = os.path.join(_HERE, "oracle.h")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (fp64, OpenMP over (batch, head) units)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= max(
        os.path.getmtime(_SRC), os.path.getmtime(_HDR)
    ):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O3", "-std=c11", "-fno-fast-math", "-fopenmp", "-fPIC",
           "-shared", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    lib = ctypes.CDLL(_LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    u64p = ctypes.POINTER(ctypes.c_uint64)
    i32p = ctypes.POINTER(ctypes.c_int32)
    i64p = ctypes.POINTER(ctypes.c_int64)
    i64, i32 = ctypes.c_int64, ctypes.c_int
    lib.orc_full_attention.argtypes = [dp, dp, dp, i64, i32, dp]
    lib.orc_hash.argtypes = [dp, i64, i32, dp, i32, u64p]
    lib.orc_philox4x64_10.argtypes = [u64p, u64p, u64p]
    lib.orc_planes.argtypes = [ctypes.c_uint64, i32, i32, i32, dp]
    lib.orc_projections.argtypes = [dp, i64, i32, dp, i32, dp]
    lib.orc_kmeans.argtypes = [u64p, i64, i32, i32, i32p, u64p, i64p]
    lib.orc_centroids.argtypes = [dp, i64, i32, i32p, i32, dp, i64p]
    lib.orc_centroid_row.argtypes = [dp, dp, i64, i32, dp, dp]
    lib.orc_topk.argtypes = [dp, i64, i32, i32p]
    lib.orc_topk.restype = i32
    lib.orc_clustered_from_assign.argtypes = [dp, dp, dp, i64, i32, i32p, i32, dp, dp, dp]
    lib.orc_iclustered_from_assign.argtypes = [dp, dp, dp, i64, i32, i32p, i32, i32,
                                               i32p, dp, i32p, dp, dp]
    lib.orc_dense_rows.argtypes = [dp, dp, i64, i32, i32p, i32, i32, dp, dp]
    lib.orc_forward.argtypes = [dp, dp, dp, i32p, i32, i32, i64, i32, dp, i32, i32,
                                i32, i32, i32, dp, u64p, i32p, i32p, dp, i32p, dp, dp]
    lib.orc_forward.restype = i32
    lib.orc_clustered_backward.argtypes = [dp, dp, dp, i64, i32, i32p, i32, dp, dp, dp, dp]
    lib.orc_iclustered_backward.argtypes = [dp, dp, dp, i64, i32, i32p, i32, i32, i32p, dp,
                                            dp, dp, dp]
    lib.orc_backward.argtypes = [dp, dp, dp, i32p, i32, i32, i64, i32, i32, i32, i32p, i32p,
                                 dp, i32, dp, dp, dp]
    lib.orc_backward.restype = i32
    lib.orc_oracle_top.argtypes = [dp, dp, dp, i64, i32, i32, dp, i32p]
    lib.orc_oracle_top_forward.argtypes = [dp, dp, dp, i32p, i32, i32, i64, i32, i32, i32, dp,
                                           i32p]
    lib.orc_oracle_top_forward.restype = i32
    _lib = lib
    return lib


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def full_attention(q, k, v):
    """Exact softmax attention of one (batch, head): q, k, v are [n, d]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, d = q.shape
    out = np.zeros((n, d), np.float64)
    _load().orc_full_attention(_ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double),
                               _ptr(v, ctypes.c_double), n, d, _ptr(out, ctypes.c_double))
    return out


def philox4x64_10(counter, key):
    """The generator's four output words for a 4-word counter and a 2-word key."""
    ctr = np.ascontiguousarray(np.asarray(counter, dtype=np.uint64).reshape(4))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint64).reshape(2))
    out = np.zeros(4, np.uint64)
    _load().orc_philox4x64_10(_ptr(ctr, ctypes.c_uint64), _ptr(k, ctypes.c_uint64),
                              _ptr(out, ctypes.c_uint64))
    return out


def planes_from_seed(seed, heads, n_bits, d):
    """Hash planes [heads, n_bits, d] drawn from a seed (fp32 values held in fp64)."""
    out = np.zeros((heads, n_bits, d), np.float64)
    _load().orc_planes(int(seed) & 0xffffffffffffffff, heads, n_bits, d,
                       _ptr(out, ctypes.c_double))
    return out


def hash_codes(q, planes):
    """Sign-of-random-projection codes of [n, d] queries with [n_bits, d] planes."""
    q, planes = _f64(q), _f64(planes)
    n, d = q.shape
    codes = np.zeros(n, np.uint64)
    _load().orc_hash(_ptr(q, ctypes.c_double), n, d, _ptr(planes, ctypes.c_double),
                     planes.shape[0], _ptr(codes, ctypes.c_uint64))
    return codes


def projections(q, planes):
    q, planes = _f64(q), _f64(planes)
    n, d = q.shape
    out = np.zeros((n, planes.shape[0]), np.float64)
    _load().orc_projections(_ptr(q, ctypes.c_double), n, d, _ptr(planes, ctypes.c_double),
                            planes.shape[0], _ptr(out, ctypes.c_double))
    return out


def kmeans(codes, C, L):
    """Hamming K-means on uint64 codes.  Returns (assign, centroids, objective)."""
    codes = np.ascontiguousarray(codes, dtype=np.uint64)
    n = codes.shape[0]
    assign = np.full(n, -1, np.int32)
    cent = np.zeros(C, np.uint64)
    obj = np.zeros(2 * L, np.int64)
    _load().orc_kmeans(_ptr(codes, ctypes.c_uint64), n, C, L, _ptr(assign, ctypes.c_int32),
                       _ptr(cent, ctypes.c_uint64), _ptr(obj, ctypes.c_int64))
    return assign, cent, obj


def centroids(q, assign, C):
    q = _f64(q)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    qc = np.zeros((C, d), np.float64)
    sizes = np.zeros(C, np.int64)
    _load().orc_centroids(_ptr(q, ctypes.c_double), n, d, _ptr(assign, ctypes.c_int32), C,
                          _ptr(qc, ctypes.c_double), _ptr(sizes, ctypes.c_int64))
    return qc, sizes


def centroid_row(qcj, k):
    qcj, k = _f64(qcj), _f64(k)
    n, d = k.shape
    s = np.zeros(n, np.float64)
    a = np.zeros(n, np.float64)
    _load().orc_centroid_row(_ptr(qcj, ctypes.c_double), _ptr(k, ctypes.c_double), n, d,
                             _ptr(s, ctypes.c_double), _ptr(a, ctypes.c_double))
    return s, a


def topk(s, k):
    s = _f64(s)
    n = s.shape[0]
    top = np.full(max(min(k, n), 1), -1, np.int32)
    ke = _load().orc_topk(_ptr(s, ctypes.c_double), n, k, _ptr(top, ctypes.c_int32))
    return top[:ke]


def clustered_from_assign(q, k, v, assign, C):
    """Clustered attention of one (batch, head) for a given partition."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    out = np.zeros((n, d), np.float64)
    qc = np.zeros((C, d), np.float64)
    vc = np.zeros((C, d), np.float64)
    _load().orc_clustered_from_assign(
        _ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double), _ptr(v, ctypes.c_double), n, d,
        _ptr(assign, ctypes.c_int32), C, _ptr(out, ctypes.c_double),
        _ptr(qc, ctypes.c_double), _ptr(vc, ctypes.c_double))
    return out, qc, vc


def iclustered_from_assign(q, k, v, assign, C, topk_, topk_in=None):
    """Improved clustered attention of one (batch, head) for a given partition.

    Returns (out, T, mass, Vb) with T as [C, topk] ascending, -1 padded."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    out = np.zeros((n, d), np.float64)
    tk = np.full((C, topk_), -1, np.int32)
    mass = np.zeros(C, np.float64)
    vb = np.zeros((C, d), np.float64)
    tin = None if topk_in is None else np.ascontiguousarray(topk_in, dtype=np.int32)
    _load().orc_iclustered_from_assign(
        _ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double), _ptr(v, ctypes.c_double), n, d,
        _ptr(assign, ctypes.c_int32), C, topk_, _ptr(tin, ctypes.c_int32),
        _ptr(out, ctypes.c_double), _ptr(tk, ctypes.c_int32), _ptr(mass, ctypes.c_double),
        _ptr(vb, ctypes.c_double))
    return out, tk, mass, vb


def dense_rows(q, k, assign, C, topk_):
    """Dense [n, n] matrices (A^c row of each query's cluster, A^t of Eq. 11)."""
    q, k = _f64(q), _f64(k)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    ac = np.zeros((n, n), np.float64)
    at = np.zeros((n, n), np.float64)
    _load().orc_dense_rows(_ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double), n, d,
                           _ptr(assign, ctypes.c_int32), C, topk_,
                           _ptr(ac, ctypes.c_double), _ptr(at, ctypes.c_double))
    return ac, at


def forward(q, k, v, lengths, planes, C, n_bits, L, topk_=0, num_threads=None,
            exports=True):
    """Whole forward pass over [B, H, N, d] inputs.

    topk_ <= 0 runs clustered attention, topk_ >= 1 improved clustered attention.
    Returns a dict with 'out' and, if exports, the intermediate results."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, d = q.shape
    planes = _f64(planes)
    assert planes.shape == (H, n_bits, d)
    lens = None if lengths is None else np.ascontiguousarray(lengths, dtype=np.int32)
    out = np.zeros((B, H, N, d), np.float64)
    res = {"out": out}
    if exports:
        res["codes"] = np.zeros((B, H, N), np.uint64)
        res["assign"] = np.zeros((B, H, N), np.int32)
        res["sizes"] = np.zeros((B, H, C), np.int32)
        res["qc"] = np.zeros((B, H, C, d), np.float64)
        res["topk"] = np.zeros((B, H, C, max(topk_, 1)), np.int32)
        res["mass"] = np.zeros((B, H, C), np.float64)
        res["vcb"] = np.zeros((B, H, C, d), np.float64)
    g = res.get
    if num_threads is None:
        num_threads = os.cpu_count() or 1
    rc = _load().orc_forward(
        _ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double), _ptr(v, ctypes.c_double),
        _ptr(lens, ctypes.c_int32), B, H, N, d, _ptr(planes, ctypes.c_double), n_bits, C, L,
        topk_, int(num_threads), _ptr(out, ctypes.c_double),
        _ptr(g("codes"), ctypes.c_uint64), _ptr(g("assign"), ctypes.c_int32),
        _ptr(g("sizes"), ctypes.c_int32), _ptr(g("qc"), ctypes.c_double),
        _ptr(g("topk"), ctypes.c_int32) if topk_ > 0 else None,
        _ptr(g("mass"), ctypes.c_double), _ptr(g("vcb"), ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return res


def clustered_backward(q, k, v, assign, C, dout):
    """Gradients (dq, dk, dv) of clustered attention of one (batch, head) for a
    fixed partition, given the output gradient dout [n, d]."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    dq, dk, dv = (np.zeros((n, d), np.float64) for _ in range(3))
    P = ctypes.c_double
    _load().orc_clustered_backward(_ptr(q, P), _ptr(k, P), _ptr(v, P), n, d,
                                   _ptr(assign, ctypes.c_int32), C, _ptr(dout, P),
                                   _ptr(dq, P), _ptr(dk, P), _ptr(dv, P))
    return dq, dk, dv


def iclustered_backward(q, k, v, assign, C, topk_, dout, topk_in=None):
    """Gradients (dq, dk, dv) of improved clustered attention of one (batch,
    head) for a fixed partition and fixed top-k sets (selected as in the
    forward pass when topk_in is None)."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    n, d = q.shape
    dq, dk, dv = (np.zeros((n, d), np.float64) for _ in range(3))
    tin = None if topk_in is None else np.ascontiguousarray(topk_in, dtype=np.int32)
    P = ctypes.c_double
    _load().orc_iclustered_backward(_ptr(q, P), _ptr(k, P), _ptr(v, P), n, d,
                                    _ptr(assign, ctypes.c_int32), C, topk_,
                                    _ptr(tin, ctypes.c_int32), _ptr(dout, P),
                                    _ptr(dq, P), _ptr(dk, P), _ptr(dv, P))
    return dq, dk, dv


def backward(q, k, v, lengths, C, topk_, assign, topk_sets, dout, num_threads=None):
    """Gradients over [B, H, N, d] inputs for the partition (assign [B, H, N])
    and, for topk_ >= 1, the top-k sets (topk_sets [B, H, C, topk_]) of a
    forward pass.  Returns (dq, dk, dv); padded rows get zero gradients."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, N, d = q.shape
    lens = None if lengths is None else np.ascontiguousarray(lengths, dtype=np.int32)
    assign = np.ascontiguousarray(assign, dtype=np.int32)
    ts = None
    if topk_ > 0 and topk_sets is not None:
        ts = np.ascontiguousarray(topk_sets, dtype=np.int32)
        assert ts.shape == (B, H, C, topk_)
    dq, dk, dv = (np.zeros((B, H, N, d), np.float64) for _ in range(3))
    if num_threads is None:
        num_threads = os.cpu_count() or 1
    P = ctypes.c_double
    rc = _load().orc_backward(_ptr(q, P), _ptr(k, P), _ptr(v, P), _ptr(lens, ctypes.c_int32),
                              B, H, N, d, C, topk_, _ptr(assign, ctypes.c_int32),
                              _ptr(ts, ctypes.c_int32), _ptr(dout, P), int(num_threads),
                              _ptr(dq, P), _ptr(dk, P), _ptr(dv, P))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return dq, dk, dv


def oracle_top_unit(q, k, v, topk_):
    """Oracle-top for one (sequence, head) of n queries and keys: each query
    attends to its topk_ keys of highest logit only, with the softmax
    renormalised over them.  Returns (out [n, d], T [n, topk_], -1 padded)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, d = q.shape
    out = np.zeros((n, d), np.float64)
    t = np.full((n, topk_), -1, np.int32)
    P = ctypes.c_double
    _load().orc_oracle_top(_ptr(q, P), _ptr(k, P), _ptr(v, P), n, d, topk_, _ptr(out, P),
                           _ptr(t, ctypes.c_int32))
    return out, t


def oracle_top(q, k, v, lengths, topk_, num_threads=None):
    """Oracle-top over [B, H, N, d] inputs with per-sequence lengths (None: all
    N).  Returns (out [B, H, N, d], T [B, H, N, topk_]); padded rows give 0 and
    -1."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, N, d = q.shape
    lens = None if lengths is None else np.ascontiguousarray(lengths, dtype=np.int32)
    out = np.zeros((B, H, N, d), np.float64)
    t = np.full((B, H, N, topk_), -1, np.int32)
    if num_threads is None:
        num_threads = os.cpu_count() or 1
    P = ctypes.c_double
    rc = _load().orc_oracle_top_forward(_ptr(q, P), _ptr(k, P), _ptr(v, P),
                                        _ptr(lens, ctypes.c_int32), B, H, N, d, topk_,
                                        int(num_threads), _ptr(out, P), _ptr(t, ctypes.c_int32))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return out, t

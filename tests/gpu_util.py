"""Shared helpers of the GPU tests: run the HIP library through the C ABI on a
generated workload and fetch every exported stage result as numpy arrays."""
from __future__ import annotations

import numpy as np

import oracle


def torch_mod():
    import torch
    return torch


def to_dev(x, dtype):
    """float32 numpy array -> device tensor of the workload dtype (exact for
    bf16-representable values)."""
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def run_gpu(w, topk, codes_in=None, assign_in=None, topk_in=None, lengths=True, C=None, L=None,
            q=None):
    """Runs the library on workload w.  topk = 0 -> clustered variant.
    Returns a dict of numpy arrays (out as float64)."""
    import paper_2007_04825_amd as ca
    torch = torch_mod()
    C = w.C if C is None else C
    L = w.L if L is None else L
    qn = w.q if q is None else q
    B, H, N, D = qn.shape
    qd, kd, vd = to_dev(qn, w.dtype), to_dev(w.k, w.dtype), to_dev(w.v, w.dtype)
    planes = torch.from_numpy(np.ascontiguousarray(w.planes)).cuda()
    lens = torch.from_numpy(w.lengths.astype(np.int32)).cuda() if lengths else None
    U = B * H
    kk = max(topk, 1)
    ex = dict(
        codes_out=torch.zeros((U, N), dtype=torch.int64, device="cuda"),
        assign_out=torch.zeros((U, N), dtype=torch.int32, device="cuda"),
        sizes_out=torch.zeros((U, C), dtype=torch.int32, device="cuda"),
        centroids_out=torch.zeros((U, C, D), dtype=torch.float32, device="cuda"),
        values_out=torch.zeros((U, C, D), dtype=torch.float32, device="cuda"),
        topk_out=torch.zeros((U, C, kk), dtype=torch.int32, device="cuda"),
        mass_out=torch.zeros((U, C), dtype=torch.float32, device="cuda"),
    )
    inj = {}
    if codes_in is not None:
        inj["codes_in"] = torch.from_numpy(np.ascontiguousarray(codes_in).view(np.int64)).cuda()
    if assign_in is not None:
        inj["assign_in"] = torch.from_numpy(np.ascontiguousarray(assign_in, dtype=np.int32)).cuda()
    if topk_in is not None:
        inj["topk_in"] = torch.from_numpy(np.ascontiguousarray(topk_in, dtype=np.int32)).cuda()
    aux = ca.make_aux(**ex, **inj)
    if topk > 0:
        out = ca.iclustered_attention(qd, kd, vd, planes, C, w.n_bits, L, topk, lengths=lens, aux=aux)
    else:
        out = ca.clustered_attention(qd, kd, vd, planes, C, w.n_bits, L, lengths=lens, aux=aux)
    torch.cuda.synchronize()
    res = {k.replace("_out", ""): v.cpu().numpy() for k, v in ex.items()}
    res["codes"] = res["codes"].view(np.uint64).reshape(B, H, N)
    res["assign"] = res["assign"].reshape(B, H, N)
    res["sizes"] = res["sizes"].reshape(B, H, C)
    res["centroids"] = res["centroids"].reshape(B, H, C, D)
    res["values"] = res["values"].reshape(B, H, C, D)
    res["topk"] = res["topk"].reshape(B, H, C, kk)
    res["mass"] = res["mass"].reshape(B, H, C)
    res["out"] = out.float().cpu().numpy().astype(np.float64)
    return res


_ORACLE_CACHE = {}


def run_oracle(w, topk, C=None, L=None, key=None):
    C = w.C if C is None else C
    L = w.L if L is None else L
    ck = (key or w.name, topk, C, L)
    if ck not in _ORACLE_CACHE:
        q = np.nan_to_num(w.q, nan=0.0)
        _ORACLE_CACHE[ck] = oracle.forward(q, w.k, w.v, w.lengths, w.planes, C, w.n_bits, L, topk)
    return _ORACLE_CACHE[ck]


def topk_mismatches(w, ref, got, topk, rel_delta=1e-5):
    """Clusters whose GPU top-k set differs from the oracle's.  Returns
    (list of (b, h, j), list of violations).  A difference is accepted only as a
    near tie: every key in the symmetric difference must have an oracle logit
    within rel_delta * max(1, |s_k|) of the oracle's k-th largest logit."""
    B, H, C = ref["sizes"].shape
    diff, bad = [], []
    for b in range(B):
        n = int(w.lengths[b])
        kk = min(topk, n)
        for h in range(H):
            for j in range(C):
                if ref["sizes"][b, h, j] == 0:
                    continue
                t_ref = ref["topk"][b, h, j, :kk]
                t_got = got["topk"][b, h, j, :kk]
                if np.array_equal(t_ref, t_got):
                    continue
                diff.append((b, h, j))
                s, _ = oracle.centroid_row(ref["qc"][b, h, j], w.k[b, h, :n])
                kth = np.sort(s)[::-1][kk - 1]
                delta = rel_delta * max(1.0, abs(kth))
                sym = np.setxor1d(t_ref, t_got)
                if np.any(sym < 0) or np.any(np.abs(s[sym[sym >= 0]] - kth) > delta):
                    bad.append((b, h, j, sym.tolist()))
    return diff, bad

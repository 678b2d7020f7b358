"""Clustered and improved-clustered attention forward pass on MI355X (gfx950).

A thin ctypes binding over the C ABI declared in ``include/clustered_attn.h``
(``libclustered_attn.so`` in this directory).  It only marshals arguments:
torch tensors supply device memory and the current HIP stream; every step of
the method runs in the library's HIP kernels.  There is no CPU fallback: if
the library is missing or no GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = [
    "CA_OK", "CA_ERR_INVALID_ARG", "CA_ERR_UNSUPPORTED", "CA_ERR_WORKSPACE", "CA_ERR_HIP",
    "CA_F32", "CA_BF16", "Aux", "ClusteredAttnError", "library", "lib_path",
    "workspace_bytes", "clustered_attention_fwd", "iclustered_attention_fwd",
    "clustered_attention", "iclustered_attention", "set_kmeans_path", "EXPORTED_SYMBOLS",
    "backward_workspace_bytes", "clustered_attention_bwd", "iclustered_attention_bwd",
    "clustered_attention_backward", "iclustered_attention_backward",
    "oracle_top_workspace_bytes", "oracle_top_attention_fwd", "oracle_top_attention",
    "iclustered_attention_fwd_noalloc", "NOALLOC_SCRATCH_BYTES",
]

CA_OK = 0
CA_ERR_INVALID_ARG = -1
CA_ERR_UNSUPPORTED = -2
CA_ERR_WORKSPACE = -3
CA_ERR_HIP = -4
CA_F32 = 0
CA_BF16 = 1

EXPORTED_SYMBOLS = ("ca_workspace_bytes", "clustered_attention_fwd", "iclustered_attention_fwd",
                    "ca_last_error", "ca_version", "ca_set_kmeans_path", "ca_time_next_stage",
                    "ca_backward_workspace_bytes", "clustered_attention_bwd",
                    "iclustered_attention_bwd", "ca_oracle_top_workspace_bytes",
                    "oracle_top_attention_fwd", "iclustered_attention_fwd_noalloc")
# bytes of the allocation-free entry point's device scratch (the header's
# CA_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024
CA_KERNEL_HASH, CA_KERNEL_KMEANS, CA_KERNEL_CENTROIDS, CA_KERNEL_CENTROID_ATTN, CA_KERNEL_OUTPUT = \
    1, 2, 3, 4, 5
CA_KERNEL_BWD_CENTROID = 6
CA_KERNEL_ATTN_TILE = 7
STAGES = {"hash": 1, "kmeans": 2, "centroids": 3, "centroid_attn": 4, "output": 5}

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libclustered_attn.so")
_lib = None


class ClusteredAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("clustered_attn error %d: %s" % (code, msg))
        self.code = code


class Aux(ctypes.Structure):
    """Mirror of ``ca_aux`` (all device pointers, 0 = unused)."""
    _fields_ = [(name, ctypes.c_void_p) for name in (
        "codes_in", "assign_in", "topk_in", "codes_out", "assign_out", "sizes_out",
        "centroids_out", "topk_out", "mass_out", "values_out", "planes_out")]


def library():
    """Loads the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(lib_path):
        raise RuntimeError("libclustered_attn.so is not built; run "
                           "`python -c 'import __graft_entry__ as g; g.build()'`")
    # torch ships its own HIP runtime: importing it first makes the library
    # bind to the runtime that owns the caller's device memory and streams,
    # whichever of the two the caller touches first
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(lib_path)
    vp, i32, sz, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_uint64
    lib.ca_workspace_bytes.argtypes = [i32] * 8
    lib.ca_workspace_bytes.restype = sz
    common = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32]
    lib.clustered_attention_fwd.argtypes = common + [u64, vp, vp, sz, ctypes.POINTER(Aux), vp]
    lib.clustered_attention_fwd.restype = i32
    lib.iclustered_attention_fwd.argtypes = common + [u64, i32, vp, vp, sz, ctypes.POINTER(Aux), vp]
    lib.iclustered_attention_fwd.restype = i32
    lib.iclustered_attention_fwd_noalloc.argtypes = common + [u64, i32, vp, ctypes.POINTER(Aux), vp]
    lib.iclustered_attention_fwd_noalloc.restype = i32
    lib.ca_last_error.argtypes = []
    lib.ca_last_error.restype = ctypes.c_char_p
    lib.ca_version.restype = i32
    lib.ca_set_kmeans_path.argtypes = [i32]
    lib.ca_set_kmeans_path.restype = i32
    lib.ca_time_next_stage.argtypes = [i32, vp, vp]
    lib.ca_time_next_stage.restype = i32
    lib.ca_backward_workspace_bytes.argtypes = [i32] * 7
    lib.ca_backward_workspace_bytes.restype = sz
    bcommon = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32]
    btail = [vp, vp, vp, vp, vp, sz, vp, sz, vp]
    lib.clustered_attention_bwd.argtypes = bcommon + btail
    lib.clustered_attention_bwd.restype = i32
    lib.iclustered_attention_bwd.argtypes = bcommon + [i32] + btail
    lib.iclustered_attention_bwd.restype = i32
    lib.ca_oracle_top_workspace_bytes.argtypes = [i32] * 6
    lib.ca_oracle_top_workspace_bytes.restype = sz
    lib.oracle_top_attention_fwd.argtypes = [vp, vp, vp, vp] + [i32] * 6 + [vp, vp, vp, sz, vp]
    lib.oracle_top_attention_fwd.restype = i32
    _lib = lib
    return lib


def _check(rc: int):
    if rc != CA_OK:
        raise ClusteredAttnError(rc, library().ca_last_error().decode())


def workspace_bytes(batch, heads, n, d, dtype, n_clusters, n_bits, topk=0) -> int:
    return int(library().ca_workspace_bytes(batch, heads, n, d, dtype, n_clusters, n_bits, topk))


def backward_workspace_bytes(batch, heads, n, d, dtype, n_clusters, topk=0) -> int:
    return int(library().ca_backward_workspace_bytes(batch, heads, n, d, dtype, n_clusters, topk))


def clustered_attention_bwd(q, k, v, lengths, batch, heads, n, d, dtype, n_clusters, dout, dq, dk,
                            dv, workspace, workspace_nbytes, bwd_workspace, bwd_workspace_nbytes,
                            stream=None):
    """Raw call with integer device addresses; returns the status code."""
    return library().clustered_attention_bwd(q, k, v, lengths, batch, heads, n, d, dtype,
                                             n_clusters, dout, dq, dk, dv, workspace,
                                             workspace_nbytes, bwd_workspace,
                                             bwd_workspace_nbytes, stream)


def iclustered_attention_bwd(q, k, v, lengths, batch, heads, n, d, dtype, n_clusters, topk, dout,
                             dq, dk, dv, workspace, workspace_nbytes, bwd_workspace,
                             bwd_workspace_nbytes, stream=None):
    """Raw call with integer device addresses; returns the status code."""
    return library().iclustered_attention_bwd(q, k, v, lengths, batch, heads, n, d, dtype,
                                              n_clusters, topk, dout, dq, dk, dv, workspace,
                                              workspace_nbytes, bwd_workspace,
                                              bwd_workspace_nbytes, stream)


def oracle_top_workspace_bytes(batch, heads, n, d, dtype, topk) -> int:
    return int(library().ca_oracle_top_workspace_bytes(batch, heads, n, d, dtype, topk))


def oracle_top_attention_fwd(q, k, v, lengths, batch, heads, n, d, dtype, topk, out, topk_out,
                             workspace, workspace_nbytes, stream=None):
    """Raw call with integer device addresses; returns the status code."""
    return library().oracle_top_attention_fwd(q, k, v, lengths, batch, heads, n, d, dtype, topk,
                                              out, topk_out, workspace, workspace_nbytes, stream)


def time_next_stage(stage: int, start_event, stop_event):
    """Arms the one-shot event pair (torch.cuda.Event objects) around a stage
    of the next forward call on this thread."""
    _check(library().ca_time_next_stage(int(stage), start_event.cuda_event, stop_event.cuda_event))


def set_kmeans_path(path: int):
    """0 automatic, 1 one workgroup per unit, 2 one kernel pair per Lloyd round,
    3 one cooperative launch for all rounds; 4 and 5 as 3 with the centroid
    sums formed by the K-means kernel (4) or by a separate kernel (5)."""
    _check(library().ca_set_kmeans_path(int(path)))


def _seed(seed) -> int:
    return int(seed) & 0xFFFFFFFFFFFFFFFF


def clustered_attention_fwd(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters,
                            n_bits, lloyd_iters, seed, out, workspace, workspace_nbytes, aux=None,
                            stream=None):
    """Raw call with integer device addresses (planes None: drawn from seed);
    returns the status code."""
    return library().clustered_attention_fwd(
        q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters, n_bits, lloyd_iters,
        _seed(seed), out, workspace, workspace_nbytes,
        ctypes.byref(aux) if aux is not None else None, stream)


def iclustered_attention_fwd(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters,
                             n_bits, lloyd_iters, seed, topk, out, workspace, workspace_nbytes,
                             aux=None, stream=None):
    """Raw call with integer device addresses (planes None: drawn from seed);
    returns the status code."""
    return library().iclustered_attention_fwd(
        q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters, n_bits, lloyd_iters,
        _seed(seed), topk, out, workspace, workspace_nbytes,
        ctypes.byref(aux) if aux is not None else None, stream)


def iclustered_attention_fwd_noalloc(q, k, v, lengths, planes, batch, heads, n, d, dtype,
                                     n_clusters, n_bits, lloyd_iters, seed, topk, out, aux=None,
                                     stream=None):
    """Raw call of the allocation-free entry point (the library's own device
    scratch instead of a workspace) with integer device addresses; returns the
    status code."""
    return library().iclustered_attention_fwd_noalloc(
        q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters, n_bits, lloyd_iters,
        _seed(seed), topk, out, ctypes.byref(aux) if aux is not None else None, stream)


# ---------------------------------------------------------------------------
# torch convenience layer (device memory and stream plumbing only)
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return CA_F32
    if t.dtype == torch.bfloat16:
        return CA_BF16
    raise TypeError("q, k, v must be float32 or bfloat16, got %s" % t.dtype)


def _ptr(t):
    return None if t is None else t.data_ptr()


def make_aux(**tensors) -> Aux:
    """Builds an Aux from keyword tensors (e.g. codes_out=t); others stay 0."""
    aux = Aux()
    for name, t in tensors.items():
        if t is not None:
            setattr(aux, name, t.data_ptr())
    return aux


def _prepare(q, k, v, planes, lengths):
    torch = _torch()
    if not (q.is_cuda and k.is_cuda and v.is_cuda):
        raise ValueError("q, k, v must be device tensors")
    if q.dim() != 4 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share the shape [batch, heads, n, d]")
    if not (q.dtype == k.dtype == v.dtype):
        raise ValueError("q, k, v must share a dtype")
    for t in (q, k, v):
        if not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous")
    if planes is not None and (planes.dtype != torch.float32 or not planes.is_cuda
                               or not planes.is_contiguous()):
        raise ValueError("planes must be a contiguous float32 device tensor [heads, n_bits, d]")
    if lengths is not None and (lengths.dtype != torch.int32 or not lengths.is_cuda):
        raise ValueError("lengths must be an int32 device tensor [batch]")
    return q.shape


def _workspace(nbytes, device, workspace):
    torch = _torch()
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError("workspace too small: need %d bytes" % nbytes)
        return workspace
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def clustered_attention(q, k, v, planes=None, n_clusters=100, n_bits=63, lloyd_iters=10,
                        lengths=None, out=None, workspace=None, aux: Optional[Aux] = None,
                        seed=0):
    """Clustered attention forward (Section 3.2) on torch device tensors;
    planes None: the library draws them from seed."""
    torch = _torch()
    B, H, N, D = _prepare(q, k, v, planes, lengths)
    dt = _dtype_code(q)
    need = workspace_bytes(B, H, N, D, dt, n_clusters, n_bits, 0)
    if need == 0:
        _check(library().clustered_attention_fwd(None, None, None, None, None, B, H, N, D, dt,
                                                 n_clusters, n_bits, lloyd_iters, 0, None, None,
                                                 0, None, None))
    ws = _workspace(need, q.device, workspace)
    if out is None:
        out = torch.empty_like(q)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(clustered_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), _ptr(lengths),
                                   _ptr(planes), B, H, N, D, dt, n_clusters, n_bits, lloyd_iters,
                                   seed, out.data_ptr(), ws.data_ptr(), need, aux, stream))
    return out


def iclustered_attention(q, k, v, planes=None, n_clusters=100, n_bits=63, lloyd_iters=10, topk=32,
                         lengths=None, out=None, workspace=None, aux: Optional[Aux] = None,
                         seed=0):
    """Improved clustered attention forward (Section 3.3) on torch device
    tensors; planes None: the library draws them from seed."""
    torch = _torch()
    B, H, N, D = _prepare(q, k, v, planes, lengths)
    dt = _dtype_code(q)
    need = workspace_bytes(B, H, N, D, dt, n_clusters, n_bits, topk)
    if need == 0:
        _check(library().iclustered_attention_fwd(None, None, None, None, None, B, H, N, D, dt,
                                                  n_clusters, n_bits, lloyd_iters, 0, topk, None,
                                                  None, 0, None, None))
    ws = _workspace(need, q.device, workspace)
    if out is None:
        out = torch.empty_like(q)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(iclustered_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), _ptr(lengths),
                                    _ptr(planes), B, H, N, D, dt, n_clusters, n_bits, lloyd_iters,
                                    seed, topk, out.data_ptr(), ws.data_ptr(), need, aux, stream))
    return out


def oracle_top_attention(q, k, v, topk=32, lengths=None, out=None, topk_out=None,
                         workspace=None):
    """Oracle-top attention (each query attends to its topk keys of highest
    logit only, softmax renormalised over them) on torch device tensors.
    topk_out: optional int32 device tensor [batch, heads, n, topk] that
    receives the sets.  Pass k=q for the shared-QK input mode."""
    torch = _torch()
    B, H, N, D = _prepare(q, k, v, None, lengths)
    dt = _dtype_code(q)
    need = oracle_top_workspace_bytes(B, H, N, D, dt, topk)
    if need == 0:
        _check(library().oracle_top_attention_fwd(None, None, None, None, B, H, N, D, dt, topk,
                                                  None, None, None, 0, None))
    if topk_out is not None and (topk_out.dtype != torch.int32 or not topk_out.is_cuda
                                 or not topk_out.is_contiguous()
                                 or tuple(topk_out.shape) != (B, H, N, topk)):
        raise ValueError("topk_out must be a contiguous int32 device tensor [batch, heads, n, topk]")
    ws = _workspace(need, q.device, workspace)
    if out is None:
        out = torch.empty_like(q)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(oracle_top_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), _ptr(lengths), B, H,
                                    N, D, dt, topk, out.data_ptr(), _ptr(topk_out), ws.data_ptr(),
                                    need, stream))
    return out


def _backward(q, k, v, dout, n_clusters, topk, lengths, workspace, bwd_workspace, grads):
    torch = _torch()
    B, H, N, D = _prepare(q, k, v, None, lengths)
    if dout.shape != q.shape or dout.dtype != q.dtype or not dout.is_contiguous():
        raise ValueError("dout must be a contiguous tensor like q")
    if workspace is None:
        raise ValueError("workspace: pass the buffer that the forward call used")
    dt = _dtype_code(q)
    bneed = backward_workspace_bytes(B, H, N, D, dt, n_clusters, topk)
    if bneed == 0:
        bneed = 1  # invalid sizes: the call below reports why
    bws = _workspace(bneed, q.device, bwd_workspace)
    if grads is None:
        grads = tuple(torch.empty(q.shape, dtype=torch.float32, device=q.device) for _ in range(3))
    dq, dk, dv = grads
    stream = torch.cuda.current_stream(q.device).cuda_stream
    wbytes = workspace.numel() * workspace.element_size()
    if topk > 0:
        rc = iclustered_attention_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), _ptr(lengths), B, H,
                                      N, D, dt, n_clusters, topk, dout.data_ptr(), dq.data_ptr(),
                                      dk.data_ptr(), dv.data_ptr(), workspace.data_ptr(), wbytes,
                                      bws.data_ptr(), bws.numel(), stream)
    else:
        rc = clustered_attention_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), _ptr(lengths), B, H,
                                     N, D, dt, n_clusters, dout.data_ptr(), dq.data_ptr(),
                                     dk.data_ptr(), dv.data_ptr(), workspace.data_ptr(), wbytes,
                                     bws.data_ptr(), bws.numel(), stream)
    _check(rc)
    return dq, dk, dv


def clustered_attention_backward(q, k, v, dout, n_clusters, workspace, lengths=None,
                                 bwd_workspace=None, grads=None):
    """Gradients (dq, dk, dv), fp32, of the clustered forward call that last
    used ``workspace`` with these inputs (partition held constant)."""
    return _backward(q, k, v, dout, n_clusters, 0, lengths, workspace, bwd_workspace, grads)


def iclustered_attention_backward(q, k, v, dout, n_clusters, topk, workspace, lengths=None,
                                  bwd_workspace=None, grads=None):
    """Gradients (dq, dk, dv), fp32, of the improved clustered forward call
    that last used ``workspace`` (partition and top-k sets held constant)."""
    return _backward(q, k, v, dout, n_clusters, topk, lengths, workspace, bwd_workspace, grads)

"""The allocation-free entry point (iclustered_attention_fwd_noalloc, the
library's device scratch instead of a caller workspace) against the entry
point it varies (iclustered_attention_fwd with a workspace), called through
the C ABI: two calls in a row, the second on a smaller input, must give the
same outputs and stage exports bit for bit (same kernels, deterministic),
and sizes beyond the scratch must be rejected with nothing enqueued."""
import numpy as np
import pytest

import gen
from gpu_util import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _announce(request):
    print("\n[gpu test] %s" % request.node.name, flush=True)
    yield


def _run(w, noalloc):
    import paper_2007_04825_amd as ca
    import torch
    B, H, N, D = w.q.shape
    U = B * H
    dt = ca.CA_F32 if w.dtype == "f32" else ca.CA_BF16
    q, k, v = (to_dev(x, w.dtype) for x in (w.q, w.k, w.v))
    planes = torch.from_numpy(np.ascontiguousarray(w.planes)).cuda()
    lens = torch.from_numpy(w.lengths.astype(np.int32)).cuda()
    out = torch.full_like(q, 3.0)
    ex = dict(assign_out=torch.zeros((U, N), dtype=torch.int32, device="cuda"),
              topk_out=torch.zeros((U, w.C, w.topk), dtype=torch.int32, device="cuda"),
              values_out=torch.zeros((U, w.C, D), dtype=torch.float32, device="cuda"))
    aux = ca.make_aux(**ex)
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        rc = ca.iclustered_attention_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                 lens.data_ptr(), planes.data_ptr(), B, H, N, D,
                                                 dt, w.C, w.n_bits, w.L, 0, w.topk,
                                                 out.data_ptr(), aux, stream)
    else:
        need = ca.workspace_bytes(B, H, N, D, dt, w.C, w.n_bits, w.topk)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        rc = ca.iclustered_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), lens.data_ptr(),
                                         planes.data_ptr(), B, H, N, D, dt, w.C, w.n_bits, w.L, 0,
                                         w.topk, out.data_ptr(), ws.data_ptr(), need, aux, stream)
    assert rc == ca.CA_OK, ca.library().ca_last_error()
    torch.cuda.synchronize()
    res = {key: t.cpu().numpy() for key, t in ex.items()}
    res["out"] = out.float().cpu().numpy()
    return res


def test_noalloc_equals_workspace_entry_point_on_two_calls():
    import paper_2007_04825_amd as ca
    first = gen.config_speech(B=6, H=2, N=800, d=32, C=100, L=6, topk=32, min_len=300)
    second = gen.with_dtype(gen.config_tiny(B=1, H=3, N=300, d=64, C=20, L=4, topk=16), "bf16")
    second.lengths = np.array([257], np.int32)
    for w in (first, second):
        need = ca.workspace_bytes(*w.q.shape, 0 if w.dtype == "f32" else 1, w.C, w.n_bits, w.topk)
        assert 0 < need <= ca.NOALLOC_SCRATCH_BYTES
        ref = _run(w, noalloc=False)
        got = _run(w, noalloc=True)
        for key in ref:
            assert np.array_equal(got[key], ref[key]), (w.name, key)
        print("%s: outputs and exports equal" % w.name, flush=True)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    import paper_2007_04825_amd as ca
    import torch
    B, H, N, D, C, topk = 1, 8, 65536, 64, 200, 64
    assert ca.workspace_bytes(B, H, N, D, ca.CA_BF16, C, 63, topk) > ca.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, H, N, D), dtype=torch.bfloat16, device="cuda")
    planes = torch.zeros((H, 63, D), device="cuda")
    out = torch.full_like(q, 5.0)
    rc = ca.iclustered_attention_fwd_noalloc(q.data_ptr(), q.data_ptr(), q.data_ptr(), None,
                                             planes.data_ptr(), B, H, N, D, ca.CA_BF16, C, 63, 15,
                                             0, topk, out.data_ptr(), None,
                                             torch.cuda.current_stream().cuda_stream)
    assert rc == ca.CA_ERR_UNSUPPORTED
    assert b"scratch" in ca.library().ca_last_error()
    torch.cuda.synchronize()
    assert bool((out == 5.0).all())

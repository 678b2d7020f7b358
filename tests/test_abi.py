"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function that include/clustered_attn.h declares, sizes its workspace,
and rejects invalid arguments before it would enqueue any work."""
import ctypes
import os
import re

import pytest

import paper_2007_04825_amd as ca

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "clustered_attn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_expected_functions():
    assert set(declared_functions()) == set(ca.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = ca.library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert lib.ca_version() == 200


def test_workspace_bytes():
    small = ca.workspace_bytes(1, 1, 100, 32, ca.CA_F32, 10, 63, 0)
    assert small > 0 and small % 256 == 0
    assert ca.workspace_bytes(1, 1, 100, 32, ca.CA_F32, 10, 63, 8) > small
    big = ca.workspace_bytes(1, 8, 65536, 64, ca.CA_BF16, 200, 63, 64)
    assert 0 < big < 2 ** 30
    # n_bits sizes the room for planes drawn from a seed, [heads][n_bits][d] fp32
    grow = (ca.workspace_bytes(1, 8, 1000, 64, ca.CA_F32, 10, 64, 0)
            - ca.workspace_bytes(1, 8, 1000, 64, ca.CA_F32, 10, 1, 0))
    assert grow == 8 * 64 * 64 * 4 - 8 * 1 * 64 * 4
    for bad in [(0, 1, 100, 32, 0, 10, 63, 0), (1, 1, 100, 48, 0, 10, 63, 0),
                (1, 1, 100, 32, 2, 10, 63, 0), (1, 1, 100, 32, 0, 257, 63, 0),
                (1, 1, 100, 32, 0, 10, 65, 0), (1, 1, 100, 32, 0, 10, 63, 129),
                (1, 1, 2 ** 20 + 1, 32, 0, 10, 63, 0)]:
        assert ca.workspace_bytes(*bad) == 0, bad


@pytest.mark.parametrize("args,code", [
    (dict(batch=0), ca.CA_ERR_INVALID_ARG),
    (dict(d=16), ca.CA_ERR_UNSUPPORTED),
    (dict(dtype=5), ca.CA_ERR_INVALID_ARG),
    (dict(C=0), ca.CA_ERR_INVALID_ARG),
    (dict(C=300), ca.CA_ERR_UNSUPPORTED),
    (dict(n_bits=0), ca.CA_ERR_INVALID_ARG),
    (dict(n_bits=65), ca.CA_ERR_UNSUPPORTED),
    (dict(L=0), ca.CA_ERR_INVALID_ARG),
    (dict(topk=0), ca.CA_ERR_INVALID_ARG),
    (dict(topk=200), ca.CA_ERR_UNSUPPORTED),
    (dict(q=None), ca.CA_ERR_INVALID_ARG),
    (dict(out=None), ca.CA_ERR_INVALID_ARG),
    (dict(planes=None, n_bits=65), ca.CA_ERR_UNSUPPORTED),  # planes drawn from the seed
    (dict(ws=None), ca.CA_ERR_WORKSPACE),
    (dict(ws_bytes=16), ca.CA_ERR_WORKSPACE),
    (dict(ws=0x1001), ca.CA_ERR_WORKSPACE),
])
def test_invalid_arguments_rejected_on_host(args, code):
    """Every case fails validation, which runs before any HIP call, so the
    dummy (never dereferenced) addresses below are safe without a GPU."""
    p = dict(q=0x1000, k=0x1000, v=0x1000, lengths=None, planes=0x1000, batch=1, heads=2, n=64,
             d=32, dtype=0, C=8, n_bits=63, L=2, topk=4, out=0x1000, ws=0x10000, ws_bytes=16 << 20)
    p.update(args)
    rc = ca.iclustered_attention_fwd(p["q"], p["k"], p["v"], p["lengths"], p["planes"], p["batch"],
                                     p["heads"], p["n"], p["d"], p["dtype"], p["C"], p["n_bits"],
                                     p["L"], 7, p["topk"], p["out"], p["ws"], p["ws_bytes"])
    assert rc == code
    assert len(ca.library().ca_last_error()) > 0
    if "topk" not in args:
        rc = ca.clustered_attention_fwd(p["q"], p["k"], p["v"], p["lengths"], p["planes"],
                                        p["batch"], p["heads"], p["n"], p["d"], p["dtype"], p["C"],
                                        p["n_bits"], p["L"], 7, p["out"], p["ws"], p["ws_bytes"])
        assert rc == code


def test_kmeans_path_switch_validation():
    lib = ca.library()
    assert lib.ca_set_kmeans_path(6) == ca.CA_ERR_INVALID_ARG
    assert lib.ca_set_kmeans_path(-1) == ca.CA_ERR_INVALID_ARG
    for path in (5, 4, 3, 2, 1, 0):
        assert lib.ca_set_kmeans_path(path) == ca.CA_OK


def test_oracle_top_workspace_bytes():
    one = ca.oracle_top_workspace_bytes(1, 1, 1024, 32, ca.CA_F32, 32)
    assert one >= 1024 * 32 * 4
    # several key chunks add the per-chunk candidate lists
    two = ca.oracle_top_workspace_bytes(1, 1, 2048, 32, ca.CA_F32, 32)
    assert two >= 2048 * 32 * 4 + 2 * 2048 * 2 * 32 * 4
    for bad in [(0, 1, 64, 32, 0, 8), (1, 1, 64, 16, 0, 8), (1, 1, 64, 32, 0, 0),
                (1, 1, 64, 32, 0, 200), (1, 1, 64, 32, 3, 8)]:
        assert ca.oracle_top_workspace_bytes(*bad) == 0, bad


@pytest.mark.parametrize("args,code", [
    (dict(batch=0), ca.CA_ERR_INVALID_ARG),
    (dict(d=16), ca.CA_ERR_UNSUPPORTED),
    (dict(dtype=5), ca.CA_ERR_INVALID_ARG),
    (dict(topk=0), ca.CA_ERR_INVALID_ARG),
    (dict(topk=200), ca.CA_ERR_UNSUPPORTED),
    (dict(v=None), ca.CA_ERR_INVALID_ARG),
    (dict(out=None), ca.CA_ERR_INVALID_ARG),
    (dict(ws=None), ca.CA_ERR_WORKSPACE),
    (dict(ws_bytes=16), ca.CA_ERR_WORKSPACE),
    (dict(ws=0x1001), ca.CA_ERR_WORKSPACE),
])
def test_oracle_top_invalid_arguments_rejected_on_host(args, code):
    """Validation runs before any HIP call; the dummy addresses are never used."""
    p = dict(q=0x1000, k=0x1000, v=0x1000, lengths=None, batch=1, heads=2, n=64, d=32, dtype=0,
             topk=4, out=0x1000, topk_out=None, ws=0x10000, ws_bytes=16 << 20)
    p.update(args)
    rc = ca.oracle_top_attention_fwd(p["q"], p["k"], p["v"], p["lengths"], p["batch"], p["heads"],
                                     p["n"], p["d"], p["dtype"], p["topk"], p["out"], p["topk_out"],
                                     p["ws"], p["ws_bytes"])
    assert rc == code
    assert len(ca.library().ca_last_error()) > 0

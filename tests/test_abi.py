"""CPU tests of the C ABI: the library loads, exports every symbol the header
declares, and rejects bad arguments before any HIP call (so no GPU is needed)."""

import ctypes
import os
import re

import pytest

import paper_2402_02082_amd as glide
from paper_2402_02082_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "glide.h")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_header_parses():
    fns = header_functions()
    assert {"glide_tree_attn", "cape_expand", "tree_verify", "glide_argmax_rows"} <= set(fns)


def test_every_declared_symbol_is_exported(lib):
    for name in header_functions():
        assert hasattr(lib, name), name
    assert sorted(header_functions()) == sorted(_lib.EXPORTED)


def test_strerror(lib):
    assert lib.glide_strerror(0) == b"ok"
    assert lib.glide_strerror(glide.GLIDE_EINVAL) == b"invalid argument"
    assert lib.glide_strerror(12345) == b"unknown status"
    assert lib.glide_last_hip_error() == 0


def _attn(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, lens=FAKE, parents=FAKE, out=FAKE, B=1, N=16, H=32, D=128,
             L_cap=2064, dtype=0, scale=0.0, splits=0, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return lib.glide_tree_attn(a["q"], a["k"], a["v"], a["lens"], a["parents"], a["out"], a["B"],
                               a["N"], a["H"], a["D"], a["L_cap"], a["dtype"], a["scale"],
                               a["splits"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("bad", [
    dict(q=None), dict(k=None), dict(v=None), dict(lens=None), dict(out=None),
    dict(N=0), dict(N=65), dict(D=64), dict(D=256), dict(B=0), dict(H=0), dict(dtype=2),
    dict(dtype=-1), dict(L_cap=15), dict(splits=-1), dict(splits=65),
    dict(scale=float("nan")), dict(scale=float("inf")), dict(ws=None), dict(ws_bytes=16),
    dict(L_cap=(1 << 22) + 1), dict(B=65536), dict(B=65535, N=64, H=1024),
])
def test_tree_attn_rejects(lib, bad):
    assert _attn(lib, **bad) == glide.GLIDE_EINVAL


def _noalloc(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, lens=FAKE, parents=FAKE, out=FAKE, B=1, N=16, H=32, D=128,
             L_cap=2064, dtype=0, scale=0.0, splits=0)
    a.update(kw)
    return lib.glide_tree_attn_noalloc(a["q"], a["k"], a["v"], a["lens"], a["parents"], a["out"],
                                       a["B"], a["N"], a["H"], a["D"], a["L_cap"], a["dtype"],
                                       a["scale"], a["splits"], None)


@pytest.mark.parametrize("bad", [
    dict(q=None), dict(out=None), dict(N=65), dict(D=64), dict(dtype=2), dict(splits=65),
    dict(scale=float("nan")), dict(L_cap=(1 << 22) + 1),
])
def test_tree_attn_noalloc_rejects(lib, bad):
    assert _noalloc(lib, **bad) == glide.GLIDE_EINVAL


def test_tree_attn_noalloc_scratch_limit(lib):
    """Plans needing more workspace than the fixed scratch are refused with
    their own status before any HIP call."""
    cap = lib.glide_tree_attn_noalloc_max_workspace()
    assert cap == 16 << 20
    assert lib.glide_tree_attn_workspace(8, 64, 52, 128, 8256, 64) > cap
    assert _noalloc(lib, B=8, N=64, H=52, L_cap=8256, splits=64) == glide.GLIDE_ESCRATCH
    assert lib.glide_strerror(glide.GLIDE_ESCRATCH).startswith(b"sizes need more")
    # the workloads' automatic plans fit
    for B, N, H, L_cap in ((1, 16, 32, 2064), (4, 32, 40, 4128), (8, 64, 52, 8256),
                           (16, 64, 32, 32832), (16, 5, 32, 32832)):
        assert lib.glide_tree_attn_workspace(B, N, H, 128, L_cap, 0) <= cap


def test_tree_attn_workspace_plan(lib):
    # Vicuna-7B verify layer: 32 heads, 2048 + 16 keys -> a split plan with workspace
    ws = lib.glide_tree_attn_workspace(1, 16, 32, 128, 2064, 0)
    assert ws > 0
    # one split needs no workspace
    assert lib.glide_tree_attn_workspace(1, 16, 32, 128, 2064, 1) == 0
    assert lib.glide_tree_attn_workspace(1, 16, 32, 128, 100, 0) == 0
    # invalid sizes report 0
    assert lib.glide_tree_attn_workspace(1, 65, 32, 128, 2064, 0) == 0
    assert lib.glide_tree_attn_workspace(1, 16, 32, 64, 2064, 0) == 0
    # more splits never need less workspace
    sizes = [lib.glide_tree_attn_workspace(4, 32, 40, 128, 4128, s) for s in (2, 4, 8, 16, 32, 64)]
    assert sizes == sorted(sizes)


def test_tree_attn_workspace_layout(lib):
    """A split workspace is the fixed 256 KiB counter block, then the (max,
    sum) pair and the 128-float output of every (sequence, head, split,
    query) row, and -- single-sequence calls, whose splits merge inside the
    kernel -- the 128 fp16 values of every row: the 7B verification layer's
    plan has 8 splits."""
    assert glide.ATTN_COUNTER_BYTES == 256 << 10
    units = 1 * 32 * 8 * 16
    want = (256 << 10) + units * 8 + units * 512 + units * 256
    assert lib.glide_tree_attn_workspace(1, 16, 32, 128, 2064, 8) == want
    assert lib.glide_tree_attn_workspace(1, 16, 32, 128, 2064, 0) == want
    # the counter block does not grow with the number of (sequence, head) pairs
    units = 33 * 64 * 3 * 5
    ml = (units * 8 + 255) // 256 * 256
    assert lib.glide_tree_attn_workspace(33, 5, 64, 128, 379, 3) == (256 << 10) + ml + units * 512


def _cape(lib, **kw):
    a = dict(p=FAKE, B=1, gamma=5, V=32000, k=3, fixed=0, n_max=16, t=FAKE, par=FAKE, n=FAKE,
             ws=FAKE, ws_bytes=1 << 20)
    a.update(kw)
    return lib.cape_expand(a["p"], a["B"], a["gamma"], a["V"], a["k"], a["fixed"], a["n_max"],
                           a["t"], a["par"], a["n"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("bad", [
    dict(p=None), dict(t=None), dict(par=None), dict(n=None), dict(ws=None), dict(B=0),
    dict(gamma=0), dict(gamma=17), dict(n_max=65, gamma=5), dict(V=1), dict(k=-1),
    dict(fixed=1, k=8), dict(ws_bytes=8),
    # B * gamma draft rows are a grid dimension: at most 65535
    dict(B=1025, gamma=64, n_max=64, ws_bytes=1 << 40), dict(B=65535, gamma=2, ws_bytes=1 << 40),
])
def test_cape_rejects(lib, bad):
    assert _cape(lib, **bad) == glide.GLIDE_EINVAL


def test_cape_workspace(lib):
    # 32000 tokens = 8 parts of 4096, 8 keys of 8 bytes per part and row
    assert lib.cape_expand_workspace(2, 5, 32000) == 2 * 5 * 8 * 8 * 8
    assert lib.cape_expand_workspace(1, 1, 4096) == 8 * 8
    assert lib.cape_expand_workspace(0, 5, 100) == 0
    assert lib.cape_expand_workspace(1, 65, 100) == 0
    assert lib.cape_expand_workspace(1, 5, 1) == 0
    assert lib.cape_expand_workspace(13107, 5, 100) > 0      # 65535 rows
    assert lib.cape_expand_workspace(13108, 5, 100) == 0     # 65540 rows
    assert lib.cape_expand_workspace(1025, 64, 100) == 0


def test_tree_attn_size_limit(lib):
    """The largest accepted cache, 2^22 rows, in float32 is 2^31 bytes per
    (sequence, head) slab: accepted (the kernels form that byte range
    unsigned), one row more is rejected; the same in bfloat16."""
    assert lib.glide_tree_attn_workspace(1, 1, 1, 128, 1 << 22, 2) > 0
    assert lib.glide_tree_attn_workspace(1, 1, 1, 128, (1 << 22) + 1, 2) == 0
    for dtype in (0, 1):
        assert _attn(lib, L_cap=(1 << 22) + 1, dtype=dtype, B=1, H=1, N=1) == glide.GLIDE_EINVAL


@pytest.mark.parametrize("args", [
    (None, 4, 10, FAKE), (FAKE, 0, 10, FAKE), (FAKE, 4, 0, FAKE), (FAKE, 4, 10, None),
])
def test_argmax_rejects(lib, args):
    assert lib.glide_argmax_rows(*args, None) == glide.GLIDE_EINVAL


@pytest.mark.parametrize("args", [
    (None, FAKE, FAKE, 1, 8, FAKE), (FAKE, None, FAKE, 1, 8, FAKE), (FAKE, FAKE, None, 1, 8, FAKE),
    (FAKE, FAKE, FAKE, 0, 8, FAKE), (FAKE, FAKE, FAKE, 1, 0, FAKE), (FAKE, FAKE, FAKE, 1, 65, FAKE),
    (FAKE, FAKE, FAKE, 1, 8, None),
])
def test_verify_rejects(lib, args):
    assert lib.tree_verify(*args, None, None, None) == glide.GLIDE_EINVAL


def test_binding_rejects_host_tensors():
    import torch
    q = torch.zeros(1, 4, 2, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        glide.glide_tree_attn(q, q, q, torch.zeros(1, dtype=torch.int32), None, q)


def _commit(lib, **kw):
    ptrs = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    a = dict(logits=FAKE, V=32000, cand=FAKE, par=FAKE, B=1, N=16, kc=ptrs, vc=ptrs, layers=2,
             H=32, D=128, L_cap=2064, dtype=0, lens=ctypes.c_void_p(0x3000),
             lens_out=ctypes.c_void_p(0x4000), ta=FAKE, acc=FAKE)
    a.update(kw)
    return lib.glide_verify_commit(a["logits"], a["V"], a["cand"], a["par"], a["B"], a["N"],
                                   a["kc"], a["vc"], a["layers"], a["H"], a["D"], a["L_cap"],
                                   a["dtype"], a["lens"], a["lens_out"], a["ta"], a["acc"], None,
                                   None, None, None)


@pytest.mark.parametrize("bad", [
    dict(logits=None), dict(cand=None), dict(par=None), dict(lens=None), dict(lens_out=None),
    dict(ta=None), dict(acc=None), dict(lens_out=ctypes.c_void_p(0x3000)), dict(V=0), dict(B=0),
    dict(B=65536), dict(N=0), dict(N=65), dict(layers=-1), dict(layers=129), dict(dtype=2),
    dict(H=0), dict(D=64), dict(L_cap=15), dict(kc=None), dict(vc=None),
    dict(kc=(ctypes.c_void_p * 2)(0x1000, None)),
])
def test_verify_commit_rejects(lib, bad):
    assert _commit(lib, **bad) == glide.GLIDE_EINVAL


@pytest.mark.parametrize("args", [
    (None, FAKE, FAKE, 5, 4096, 4096, 0), (FAKE, None, FAKE, 5, 4096, 4096, 0),
    (FAKE, FAKE, None, 5, 4096, 4096, 0), (ctypes.c_void_p(0x1002), FAKE, FAKE, 5, 4096, 4096, 0),
    (FAKE, ctypes.c_void_p(0x1008), FAKE, 5, 4096, 4096, 0), (FAKE, FAKE, FAKE, 0, 4096, 4096, 0),
    (FAKE, FAKE, FAKE, 5, 0, 4096, 0), (FAKE, FAKE, FAKE, 5, 12, 4096, 0),
    (FAKE, FAKE, FAKE, 5, (1 << 20) + 8, 4096, 0), (FAKE, FAKE, FAKE, 5, 4096, 0, 0),
    (FAKE, FAKE, FAKE, 5, 4096, 4096, 2),
])
def test_rows_matmul_rejects(lib, args):
    assert lib.glide_rows_matmul(*args, None) == glide.GLIDE_EINVAL


def test_rows_weights_packed_bytes(lib):
    # one 1 KB block per (16-row tile, 32-wide K step)
    assert lib.glide_rows_weights_packed_bytes(4096, 4096) == 256 * 128 * 1024
    assert lib.glide_rows_weights_packed_bytes(40, 17) == 2 * 2 * 1024
    assert lib.glide_rows_weights_packed_bytes(8, 1) == 1024
    for K, N in ((12, 16), (0, 16), (4096, 0), ((1 << 20) + 8, 16)):
        assert lib.glide_rows_weights_packed_bytes(K, N) == 0


@pytest.mark.parametrize("args", [
    (None, FAKE, 4096, 4096), (FAKE, None, 4096, 4096), (ctypes.c_void_p(0x1008), FAKE, 4096, 4096),
    (FAKE, ctypes.c_void_p(0x1004), 4096, 4096), (FAKE, FAKE, 12, 4096), (FAKE, FAKE, 0, 4096),
    (FAKE, FAKE, 4096, 0),
])
def test_pack_rows_weights_rejects(lib, args):
    assert lib.glide_pack_rows_weights(*args, None) == glide.GLIDE_EINVAL


@pytest.mark.parametrize("args", [
    (None, FAKE, FAKE, 5, 4096, 4096, 0), (FAKE, None, FAKE, 5, 4096, 4096, 0),
    (FAKE, FAKE, None, 5, 4096, 4096, 0), (FAKE, ctypes.c_void_p(0x1008), FAKE, 5, 4096, 4096, 0),
    (FAKE, FAKE, FAKE, 0, 4096, 4096, 0), (FAKE, FAKE, FAKE, 5, 12, 4096, 0),
    (FAKE, FAKE, FAKE, 5, 4096, 0, 0), (FAKE, FAKE, FAKE, 5, 4096, 4096, 2),
])
def test_rows_matmul_packed_rejects(lib, args):
    assert lib.glide_rows_matmul_packed(*args, None) == glide.GLIDE_EINVAL


def test_cross_block_workspace(lib):
    rows = 1 * 5 * 32 * 128 * 2                      # bf16 [B, Nq, H, D], 256-aligned already
    attn = lib.glide_tree_attn_workspace(1, 5, 32, 128, 2064, 0)
    assert lib.glide_cross_block_workspace(1, 5, 4096, 32, 128, 2064) == 2 * rows + attn
    assert lib.glide_cross_block_workspace(1, 5, 4096, 32, 64, 2064) == 0
    assert lib.glide_cross_block_workspace(1, 65, 4096, 32, 128, 2064) == 0
    assert lib.glide_cross_block_workspace(1, 5, 4100, 32, 128, 2064) == 0


def _xblock(lib, **kw):
    a = dict(h=FAKE, wq=FAKE, k=FAKE, v=FAKE, lens=FAKE, wo=FAKE, out=FAKE, B=1, Nq=5, dD=4096,
             H=32, D=128, L_cap=2064, scale=0.0, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return lib.glide_cross_block(a["h"], a["wq"], a["k"], a["v"], a["lens"], a["wo"], a["out"],
                                 a["B"], a["Nq"], a["dD"], a["H"], a["D"], a["L_cap"], a["scale"],
                                 a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("bad", [
    dict(h=None), dict(wq=None), dict(k=None), dict(v=None), dict(lens=None), dict(wo=None),
    dict(out=None), dict(ws=None), dict(h=ctypes.c_void_p(0x1004)), dict(ws=ctypes.c_void_p(0x1001)),
    dict(B=0), dict(Nq=0), dict(Nq=65), dict(dD=12), dict(H=0), dict(D=64), dict(L_cap=0),
    dict(scale=float("nan")), dict(ws_bytes=1024),
])
def test_cross_block_rejects(lib, bad):
    assert _xblock(lib, **bad) == glide.GLIDE_EINVAL
    a = dict(h=FAKE, wq=FAKE, k=FAKE, v=FAKE, lens=FAKE, wo=FAKE, out=FAKE, B=1, Nq=5, dD=4096,
             H=32, D=128, L_cap=2064, scale=0.0, ws=FAKE, ws_bytes=1 << 30)
    a.update(bad)
    assert lib.glide_cross_block_packed(a["h"], a["wq"], a["k"], a["v"], a["lens"], a["wo"], a["out"],
                                        a["B"], a["Nq"], a["dD"], a["H"], a["D"], a["L_cap"],
                                        a["scale"], a["ws"], a["ws_bytes"], None) == glide.GLIDE_EINVAL


@pytest.mark.parametrize("args", [
    (None, FAKE, FAKE, FAKE, 1, 5, 32000, FAKE, FAKE), (FAKE, None, FAKE, FAKE, 1, 5, 32000, FAKE, FAKE),
    (FAKE, FAKE, None, FAKE, 1, 5, 32000, FAKE, FAKE), (FAKE, FAKE, FAKE, None, 1, 5, 32000, FAKE, FAKE),
    (FAKE, FAKE, FAKE, FAKE, 1, 5, 32000, None, FAKE), (FAKE, FAKE, FAKE, FAKE, 1, 5, 32000, FAKE, None),
    (FAKE, FAKE, FAKE, FAKE, 0, 5, 32000, FAKE, FAKE), (FAKE, FAKE, FAKE, FAKE, 1, 0, 32000, FAKE, FAKE),
    (FAKE, FAKE, FAKE, FAKE, 1, 65, 32000, FAKE, FAKE), (FAKE, FAKE, FAKE, FAKE, 1, 5, 0, FAKE, FAKE),
    (FAKE, FAKE, FAKE, FAKE, 1, 5, (1 << 20) + 1, FAKE, FAKE),
])
def test_spec_sample_rejects(lib, args):
    assert lib.spec_sample_verify(*args, None) == glide.GLIDE_EINVAL


def test_expected_speedup_host_function():
    """The library's host-side E(Spd) against the oracle and Table 1."""
    import json
    import math
    from oracle import spec_sampling as S
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "table1_expected_speedup.json")))
    for r in g["rows"]:
        for a, e in zip(r["acc"], r["spd"]):
            v = glide.glide_expected_speedup(a / 100.0, g["gamma"], r["cost"] / 100.0)
            assert abs(v - S.expected_speedup(a / 100.0, g["gamma"], r["cost"] / 100.0)) < 1e-12
            assert abs(v - e) <= 0.01
    assert glide.glide_expected_speedup(1.0, 5, 0.1) == pytest.approx(6 / 1.5)
    for bad in ((-0.1, 5, 0.1), (1.1, 5, 0.1), (0.5, 0, 0.1), (0.5, 5, -1.0)):
        assert math.isnan(glide.glide_expected_speedup(*bad))


def _blk(lib, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, B=4, T=2048, H=32, D=128, L_cap=2048, block=5,
             scale=0.0)
    a.update(kw)
    return lib.glide_block_attn(a["q"], a["k"], a["v"], a["out"], a["B"], a["T"], a["H"], a["D"],
                                a["L_cap"], a["block"], a["scale"], None)


@pytest.mark.parametrize("bad", [
    dict(q=None), dict(k=None), dict(v=None), dict(out=None), dict(B=0), dict(B=65536), dict(T=0),
    dict(T=2049), dict(H=0), dict(D=64), dict(block=0), dict(scale=float("inf")),
    dict(L_cap=(1 << 22) + 1, T=4096), dict(B=65535, H=1024, T=4096, L_cap=4096),
])
def test_block_attn_rejects(lib, bad):
    assert _blk(lib, **bad) == glide.GLIDE_EINVAL

"""GPU parity of glide_rows_matmul and glide_cross_block against the float64
oracle.  rows_matmul with float32 output: max-abs error <= 1e-4 (the
accumulation error of 4096 float32 products of O(1) values is ~1e-5).  A
bfloat16 output carries one rounding to 8 significant bits, up to 2^-8 of
the value (0.016 for values in [4, 8)), so the bound for bfloat16-stored
results is 1e-2 + 2^-8 |reference|.  The block stores its projected queries
and concatenated heads in bfloat16, so the oracle rounds the same two
intermediates (store=bfloat16) and the same bound applies to its output."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import cross_block as OX
from synth import workloads as W
from tests.gpu_common import BF16_TOL, require_gpu, say, to64

pytestmark = pytest.mark.gpu

F32_OUT_TOL = 1e-4


def bf16_ok(got, want):
    """Every element within 1e-2 + 2^-8 |want|; returns the worst excess."""
    return float(np.max(np.abs(got - want) - (BF16_TOL + 2.0 ** -8 * np.abs(want))))


def _bf16(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)


@pytest.mark.parametrize("M,K,N", [(1, 8, 1), (5, 4096, 4096), (16, 4096, 4096), (17, 512, 100),
                                   (64, 1024, 333), (80, 4096, 4096), (97, 520, 200), (128, 256, 48),
                                   (130, 256, 48), (257, 64, 17), (3, 4104, 16), (5, 96, 4096)])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_rows_matmul(M, K, N, out_dtype):
    require_gpu()
    say("rows_matmul", dict(M=M, K=K, N=N, out=str(out_dtype)))
    a = _bf16((M, K), 1 + M)
    w_t = _bf16((N, K), 2 + N, 1.0 / np.sqrt(K))
    out = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
    glide.glide_rows_matmul(a.cuda(), w_t.cuda(), out)
    torch.cuda.synchronize()
    want = OX.rows_matmul(to64(a), to64(w_t))
    if out_dtype == torch.float32:
        err = float(np.abs(to64(out) - want).max())
        assert err <= F32_OUT_TOL, err
    else:
        excess = bf16_ok(to64(out), want)
        assert excess <= 0, excess


def _block_case(seed, B, Nq, H, d_D, L_cap, lens):
    dev = torch.device("cuda")
    hidden = _bf16((B, Nq, d_D), seed).to(dev)
    wq_t = _bf16((H * 128, d_D), seed + 1, 1.0 / np.sqrt(d_D)).to(dev)
    wo_t = _bf16((d_D, H * 128), seed + 2, 1.0 / np.sqrt(H * 128)).to(dev)
    k = _bf16((B, H, L_cap, 128), seed + 3).to(dev)
    v = _bf16((B, H, L_cap, 128), seed + 4).to(dev)
    return hidden, wq_t, k, v, torch.tensor(lens, dtype=torch.int32, device=dev), wo_t


@pytest.mark.parametrize("B,Nq,H,d_D,L_cap,lens", [
    (1, 5, 2, 256, 300, [300]),
    (3, 7, 4, 520, 700, [0, 1, 699]),
    (2, 16, 3, 384, 2100, [2050, 37]),
])
def test_cross_block_small(B, Nq, H, d_D, L_cap, lens):
    require_gpu()
    say("cross_block", dict(B=B, Nq=Nq, H=H, d_D=d_D, L_cap=L_cap, lens=lens))
    hidden, wq_t, k, v, sl, wo_t = _block_case(7 + B, B, Nq, H, d_D, L_cap, lens)
    out = torch.full_like(hidden, float("nan"))
    glide.glide_cross_block(hidden, wq_t, k, v, sl, wo_t, out)
    torch.cuda.synchronize()
    want = OX.cross_block(to64(hidden), to64(wq_t), to64(k), to64(v), lens, to64(wo_t),
                          store=torch.bfloat16)
    excess = bf16_ok(to64(out), want)
    assert excess <= 0, excess


@pytest.mark.parametrize("cfg", [2, 5])
def test_cross_block_workload(cfg):
    """The workload's cross layer as a full block (d_D = 4096 = H * D), on the
    seeded cache; sequences sampled for the oracle (first and last)."""
    require_gpu()
    wl = W.WORKLOADS[cfg]
    dev = torch.device("cuda")
    lens_np = W.prefix_lengths(wl, 2)
    lens = torch.from_numpy(lens_np).to(dev)
    _, k, v = W.attention_layer(wl, 2, wl.layers - 1, torch.bfloat16, dev)
    d_D = wl.heads * 128
    hidden = _bf16((wl.batch, wl.cross_queries, d_D), 31).to(dev)
    wq_t = _bf16((d_D, d_D), 32, 1.0 / np.sqrt(d_D)).to(dev)
    wo_t = _bf16((d_D, d_D), 33, 1.0 / np.sqrt(d_D)).to(dev)
    out = torch.full_like(hidden, float("nan"))
    say("cross_block workload", wl.name)
    glide.glide_cross_block(hidden, wq_t, k, v, lens, wo_t, out)
    torch.cuda.synchronize()
    for b in sorted({0, wl.batch - 1}):
        L = int(lens_np[b])
        want = OX.cross_block(to64(hidden[b:b + 1]), to64(wq_t), to64(k[b:b + 1, :, :L]),
                              to64(v[b:b + 1, :, :L]), [L], to64(wo_t), store=torch.bfloat16)
        excess = bf16_ok(to64(out[b:b + 1]), want)
        assert excess <= 0, (b, excess)


@pytest.mark.parametrize("M,K,N", [(1, 8, 1), (5, 4096, 4096), (17, 512, 100), (64, 1024, 333),
                                   (80, 4096, 4096), (113, 200, 33), (130, 256, 48), (3, 4104, 16),
                                   (5, 40, 4097)])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_rows_matmul_packed(M, K, N, out_dtype):
    """Packed weights: the same registers reach the matrix cores, so the
    result is bit-identical to the row-major call, and within the bound of the
    oracle; ragged N (partial last tile) and K (partial last step) included."""
    require_gpu()
    say("rows_matmul packed", dict(M=M, K=K, N=N, out=str(out_dtype)))
    a = _bf16((M, K), 11 + M).cuda()
    w_t = _bf16((N, K), 12 + N, 1.0 / np.sqrt(K)).cuda()
    packed = glide.pack_rows_weights(w_t)
    assert packed.numel() * 2 == ((N + 15) // 16) * ((K + 31) // 32) * 1024
    got = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
    ref = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
    glide.glide_rows_matmul_packed(a, packed, got)
    glide.glide_rows_matmul(a, w_t, ref)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32),
                       ref.view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32))
    want = OX.rows_matmul(to64(a), to64(w_t))
    if out_dtype == torch.float32:
        err = float(np.abs(to64(got) - want).max())
        assert err <= F32_OUT_TOL, err
    else:
        excess = bf16_ok(to64(got), want)
        assert excess <= 0, excess


def test_pack_layout():
    """Unit l of block (t, j) holds w_t[16t + l % 16][32j + 8 (l / 16) .. + 7],
    zeros past N and K (K = 40, N = 17: both edges)."""
    require_gpu()
    K, N = 40, 17
    w_t = (torch.arange(N * K, dtype=torch.float32).reshape(N, K) % 251).to(torch.bfloat16)
    packed = glide.pack_rows_weights(w_t.cuda()).cpu().view(-1, 8)   # 16-byte units
    ksteps = (K + 31) // 32
    for u in range(packed.shape[0]):
        blk, l = divmod(u, 64)
        t, j = divmod(blk, ksteps)
        row, k0 = 16 * t + l % 16, 32 * j + 8 * (l // 16)
        want = w_t[row, k0:k0 + 8] if row < N and k0 < K else torch.zeros(8, dtype=torch.bfloat16)
        assert torch.equal(packed[u].view(torch.int16), want.view(torch.int16)), u


@pytest.mark.parametrize("B,Nq,H,d_D,L_cap,lens", [
    (1, 5, 2, 256, 300, [300]),
    (3, 7, 4, 520, 700, [0, 1, 699]),
])
def test_cross_block_packed(B, Nq, H, d_D, L_cap, lens):
    require_gpu()
    say("cross_block packed", dict(B=B, Nq=Nq, H=H, d_D=d_D, L_cap=L_cap, lens=lens))
    hidden, wq_t, k, v, sl, wo_t = _block_case(17 + B, B, Nq, H, d_D, L_cap, lens)
    got = torch.full_like(hidden, float("nan"))
    ref = torch.full_like(hidden, float("nan"))
    glide.glide_cross_block_packed(hidden, glide.pack_rows_weights(wq_t), k, v, sl,
                                   glide.pack_rows_weights(wo_t), got)
    glide.glide_cross_block(hidden, wq_t, k, v, sl, wo_t, ref)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
    want = OX.cross_block(to64(hidden), to64(wq_t), to64(k), to64(v), lens, to64(wo_t),
                          store=torch.bfloat16)
    excess = bf16_ok(to64(got), want)
    assert excess <= 0, excess


@pytest.mark.parametrize("M", [80, 128])
def test_rows_matmul_one_pass_matches_row_blocks(M):
    """Up to 128 rows go through one launch; each output row is the same
    dot products in the same order whatever the other rows, so the one-pass
    result equals, bit for bit, the projections of the rows taken 64 and
    then M - 64 at a time (row-major and packed weights)."""
    require_gpu()
    say("rows_matmul one pass", dict(M=M))
    K, N = 4096, 1024
    a = _bf16((M, K), 41 + M).cuda()
    w_t = _bf16((N, K), 42, 1.0 / np.sqrt(K)).cuda()
    packed = glide.pack_rows_weights(w_t)
    for out_dtype in (torch.bfloat16, torch.float32):
        view = torch.int16 if out_dtype == torch.bfloat16 else torch.int32
        one = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
        parts = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
        glide.glide_rows_matmul(a, w_t, one)
        glide.glide_rows_matmul(a[:64].contiguous(), w_t, parts[:64])
        glide.glide_rows_matmul(a[64:].contiguous(), w_t, parts[64:])
        onep = torch.full_like(one, float("nan"))
        glide.glide_rows_matmul_packed(a, packed, onep)
        torch.cuda.synchronize()
        assert torch.equal(one.view(view), parts.view(view))
        assert torch.equal(onep.view(view), one.view(view))


@pytest.mark.parametrize("M,K,N", [(21, 520, 40), (32, 4104, 17), (33, 264, 17), (48, 8, 40),
                                   (100, 520, 33), (128, 4104, 64)])
def test_rows_matmul_staged_matches_direct(M, K, N):
    """From 21 rows the activations are staged through LDS in 256-wide K
    chunks (swizzled pieces, a partial last chunk, rows past M as zeros);
    each output row must still be the direct kernel's dot products in the
    same order: one launch equals, bit for bit, the rows taken 16 at a time
    (the direct kernel), and stays within the oracle's bound."""
    require_gpu()
    say("rows_matmul staged vs direct", dict(M=M, K=K, N=N))
    a = _bf16((M, K), 51 + M).cuda()
    w_t = _bf16((N, K), 52 + N, 1.0 / np.sqrt(K)).cuda()
    packed = glide.pack_rows_weights(w_t)
    for out_dtype in (torch.bfloat16, torch.float32):
        view = torch.int16 if out_dtype == torch.bfloat16 else torch.int32
        for weights, call in ((w_t, glide.glide_rows_matmul), (packed, glide.glide_rows_matmul_packed)):
            one = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
            rows = torch.full((M, N), float("nan"), dtype=out_dtype, device="cuda")
            call(a, weights, one)
            for m0 in range(0, M, 16):
                m1 = min(M, m0 + 16)
                call(a[m0:m1].contiguous(), weights, rows[m0:m1])
            torch.cuda.synchronize()
            assert torch.equal(one.view(view), rows.view(view))
    want = OX.rows_matmul(to64(a.cpu()), to64(w_t.cpu()))
    out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    glide.glide_rows_matmul(a, w_t, out)
    torch.cuda.synchronize()
    assert float(np.abs(to64(out) - want).max()) <= F32_OUT_TOL

"""GPU parity of glide_block_attn (the block-masked cross attention of draft
training) against the float64 oracle: max-abs error <= 1e-2 (bf16 inputs,
float32 accumulation, outputs averages of N(0, 1) values)."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import block_attention as OB
from tests.gpu_common import BF16_TOL, require_gpu, say, to64

pytestmark = pytest.mark.gpu


def _run(seed, B, T, H, L_cap, block, positions=None):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((B, T, H, 128), generator=g).to(torch.bfloat16)
    k = torch.randn((B, H, L_cap, 128), generator=g).to(torch.bfloat16)
    v = torch.randn((B, H, L_cap, 128), generator=g).to(torch.bfloat16)
    out = torch.full((B, T, H, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    glide.glide_block_attn(q.cuda(), k.cuda(), v.cuda(), out, block)
    torch.cuda.synchronize()
    want = OB.block_attention(to64(q), to64(k), to64(v), T, block, positions=positions)
    got = to64(out)
    rows = slice(None) if positions is None else positions
    return float(np.abs(got[:, rows] - want[:, rows]).max()), got


@pytest.mark.parametrize("B,T,H,L_cap,block", [
    (2, 37, 3, 40, 5), (1, 64, 2, 64, 1), (1, 200, 2, 210, 64), (1, 130, 1, 130, 100),
    (3, 1, 2, 8, 5), (1, 20, 2, 20, 20), (2, 129, 2, 129, 7),
])
def test_small(B, T, H, L_cap, block):
    require_gpu()
    say("block_attn", dict(B=B, T=T, H=H, L_cap=L_cap, block=block))
    err, got = _run(B * 100 + T + block, B, T, H, L_cap, block)
    assert err <= BF16_TOL, err
    assert np.all(got[:, :min(block, T)] == 0)   # the first block sees no key


def test_training_shape_sampled():
    """A training-length sequence (T = 2048, blocks of 5): sampled positions
    at block edges, early and late."""
    require_gpu()
    T = 2048
    pos = sorted({0, 4, 5, 9, 10, 63, 64, 65, 511, 512, 1000, 1024, 2043, 2044, 2045, 2047})
    say("block_attn training shape", dict(T=T, positions=len(pos)))
    err, _ = _run(7, 2, T, 4, T, 5, positions=pos)
    assert err <= BF16_TOL, err


def test_two_tile_launch_sampled():
    """Enough (sequence, head, 128-position) groups for the two-tiles-per-wave
    launch (B * H * ceil(T / 128) >= 512): T = 1100 leaves a ragged last group
    whose second tiles lie partly past the end; blocks of 5."""
    require_gpu()
    T, H = 1100, 64
    pos = sorted({0, 4, 5, 127, 128, 129, 255, 256, 600, 1023, 1024, 1050, 1087, 1088, 1095, 1099})
    say("block_attn two-tile launch", dict(T=T, H=H, positions=len(pos)))
    err, got = _run(11, 1, T, H, T, 5, positions=pos)
    assert err <= BF16_TOL, err
    assert np.all(got[:, :5] == 0)


def test_bench_shape_sampled():
    """The benchmark's shape and launch (4 sequences x 2048 positions, 32
    heads, blocks of 5: two tiles per wave, every query block of a (sequence,
    head) pair on one XCD, four pairs at a time): sampled positions in the
    first, middle and last query blocks against the oracle."""
    require_gpu()
    B, T, H = 4, 2048, 32
    pos = sorted({0, 5, 127, 128, 1000, 1024, 1919, 1920, 2040, 2047})
    say("block_attn bench shape", dict(B=B, T=T, H=H, positions=len(pos)))
    err, got = _run(13, B, T, H, T, 5, positions=pos)
    assert err <= BF16_TOL, err
    assert np.all(got[:, :5] == 0)


def test_peaked_scores():
    """Queries scaled by 24: the block kernel's lazily moved reference max is
    passed by far and often; two-tile launch (64 heads x 1100 positions)."""
    require_gpu()
    B, T, H, L_cap, block = 1, 1100, 64, 1100, 5
    g = torch.Generator().manual_seed(41)
    q = (torch.randn((B, T, H, 128), generator=g) * 24).to(torch.bfloat16)
    k = torch.randn((B, H, L_cap, 128), generator=g).to(torch.bfloat16)
    v = torch.randn((B, H, L_cap, 128), generator=g).to(torch.bfloat16)
    pos = sorted({5, 9, 127, 128, 600, 1099})
    say("block_attn peaked", dict(T=T, H=H, positions=len(pos)))
    out = torch.full((B, T, H, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    glide.glide_block_attn(q.cuda(), k.cuda(), v.cuda(), out, block)
    torch.cuda.synchronize()
    want = OB.block_attention(to64(q), to64(k), to64(v), T, block, positions=pos)
    # a peaked softmax returns nearly single value rows, not averages: the
    # bf16 probabilities and output carry 8 significant bits, so the bound
    # is 1e-2 + 2^-8 |ref|
    got = to64(out)[:, pos]
    excess = np.abs(got - want[:, pos]) - (BF16_TOL + np.abs(want[:, pos]) / 256)
    assert float(excess.max()) <= 0, float(np.abs(got - want[:, pos]).max())

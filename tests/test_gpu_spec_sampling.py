"""GPU parity of spec_sample_verify: accept lengths and emitted tokens
bit-exact against the oracle (the acceptance tests are float32 comparisons of
the same values on both sides, and the draws are integer inverse CDFs over
fixed-point weights, so the outputs are functions of the inputs alone)."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import spec_sampling as S
from tests.gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu


def make_case(seed, B, gamma, V, mode):
    """Draft/target distributions with every acceptance pattern: 'mixed'
    (target = a blend of the draft and noise, so ratios straddle 1),
    'same' (target = draft: always accepted), 'zero' (the target gives some
    proposal tokens no mass: rejected there), 'scaled' (target = half the
    draft: the residual has no weight and the draw falls back)."""
    rng = np.random.default_rng(seed)
    pd = rng.dirichlet(np.full(V, 0.3), size=(B, gamma)).astype(np.float32)
    noise = rng.dirichlet(np.full(V, 0.3), size=(B, gamma + 1)).astype(np.float32)
    pt = noise.copy()
    lam = rng.random((B, gamma, 1)).astype(np.float32)
    pt[:, :gamma] = (lam * pd + (1 - lam) * noise[:, :gamma]).astype(np.float32)
    tokens = np.zeros((B, gamma), dtype=np.int32)
    for b in range(B):
        for i in range(gamma):
            q = pd[b, i].astype(np.float64)
            tokens[b, i] = rng.choice(V, p=q / q.sum())
    if mode == "same":
        pt[:, :gamma] = pd
    elif mode == "zero":
        for b in range(B):
            i = int(rng.integers(0, gamma))
            pt[b, i, tokens[b, i]] = 0.0
    elif mode == "scaled":
        pt[:, :gamma] = pd * np.float32(0.5)
    u = rng.random((B, gamma + 1)).astype(np.float32)
    return tokens, pd, pt, u


@pytest.mark.parametrize("B,gamma,V", [(1, 5, 32000), (16, 5, 32000), (4, 1, 7), (3, 8, 1000),
                                       (2, 64, 300), (5, 5, 1), (8, 3, 1025),
                                       # the last vocabulary whose chunks are kept in LDS, the
                                       # first that reads its rows twice, and an odd one past it
                                       (2, 5, 32768), (2, 5, 32769), (2, 3, 65537)])
@pytest.mark.parametrize("mode", ["mixed", "same", "zero", "scaled"])
def test_parity(B, gamma, V, mode):
    require_gpu()
    say("spec_sample_verify", dict(B=B, gamma=gamma, V=V, mode=mode))
    tokens, pd, pt, u = make_case(B * 1000 + gamma * 10 + V % 97, B, gamma, V, mode)
    dev = torch.device("cuda")
    acc = torch.full((B,), -7, dtype=torch.int32, device=dev)
    tok = torch.full((B,), -7, dtype=torch.int32, device=dev)
    glide.spec_sample_verify(torch.from_numpy(tokens).to(dev), torch.from_numpy(pd).to(dev),
                             torch.from_numpy(pt).to(dev), torch.from_numpy(u).to(dev), acc, tok)
    torch.cuda.synchronize()
    want_acc, want_tok = S.spec_sample_verify(tokens, pd, pt, u)
    assert np.array_equal(acc.cpu().numpy(), want_acc)
    assert np.array_equal(tok.cpu().numpy(), want_tok)
    if mode == "same":
        assert (want_acc == gamma).all()


def test_uniform_sweep_boundaries():
    """Emission draws at and next to every interval boundary of a small row:
    u = k / W for each running weight, and its float32 neighbours."""
    require_gpu()
    dev = torch.device("cuda")
    V, gamma = 5, 1
    pd = np.array([[[0.2, 0.2, 0.2, 0.2, 0.2]]], dtype=np.float32)
    pt = np.array([[[0.2, 0.2, 0.2, 0.2, 0.2], [0.1, 0.3, 0.05, 0.25, 0.3]]], dtype=np.float32)
    W = int(S.fixed_weights(pt[0, 1]).sum())
    run = np.cumsum(S.fixed_weights(pt[0, 1]))
    us = []
    for r in run[:-1]:
        c = np.float32(r / W)
        us += [np.nextafter(c, np.float32(0)), c, np.nextafter(c, np.float32(1))]
    B = len(us)
    tokens = np.zeros((B, gamma), dtype=np.int32)
    u = np.stack([np.zeros(B, dtype=np.float32), np.array(us, dtype=np.float32)], axis=1)
    pdB, ptB = np.repeat(pd, B, 0), np.repeat(pt, B, 0)
    acc = torch.empty((B,), dtype=torch.int32, device=dev)
    tok = torch.empty((B,), dtype=torch.int32, device=dev)
    glide.spec_sample_verify(torch.from_numpy(tokens).to(dev), torch.from_numpy(pdB).to(dev),
                             torch.from_numpy(ptB).to(dev), torch.from_numpy(u).to(dev), acc, tok)
    torch.cuda.synchronize()
    want_acc, want_tok = S.spec_sample_verify(tokens, pdB, ptB, u)
    assert np.array_equal(acc.cpu().numpy(), want_acc) and (want_acc == 1).all()
    assert np.array_equal(tok.cpu().numpy(), want_tok)

"""Pins for the block-masked training attention oracle (CPU only).

* every query equals the inference-time cross attention over the delayed
  cache it stands for: position j in block i sees the cache up to L * i
  (the cross-attention oracle with that length);
* brute force: torch's scaled_dot_product_attention (float64) with a boolean
  mask built independently from block ids (block(j) > block(k) over an
  outer comparison), for every row that sees at least one key;
* special cases: blocks of one token give strictly-earlier attention; a block
  as long as the sequence leaves every output zero; a sequence of two blocks
  gives the second block plain attention over the first;
* planted mistakes in the oracle must fail at least one pin.
"""

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import block_attention as OB


def _case(rng, B=2, T=23, H=2, D=8):
    q = rng.standard_normal((B, T, H, D))
    k = rng.standard_normal((B, H, T + 3, D))
    v = rng.standard_normal((B, H, T + 3, D))
    return q, k, v


def delayed_cache_errors(seed=51):
    rng = np.random.default_rng(seed)
    bad = []
    for L in (1, 2, 5, 7):
        q, k, v = _case(rng)
        B, T, H, _ = q.shape
        out = OB.block_attention(q, k, v, T, L)
        for b in range(B):
            for h in range(H):
                for j in range(T):
                    want = OA.tree_attention_head(q[b, j:j + 1, h], k[b, h], v[b, h],
                                                  L * (j // L), None)[0]
                    if not np.allclose(out[b, j, h], want, atol=1e-12, rtol=0):
                        bad.append(("delayed", L, b, h, j))
    return bad


def sdpa_errors(seed=52):
    rng = np.random.default_rng(seed)
    bad = []
    for L in (3, 5):
        q, k, v = _case(rng)
        B, T, H, D = q.shape
        out = OB.block_attention(q, k, v, T, L)
        blk = np.arange(T) // L
        mask = blk[:, None] > blk[None, :]                       # [T queries, T keys]
        rows = mask.any(axis=1)
        for b in range(B):
            for h in range(H):
                ref = torch.nn.functional.scaled_dot_product_attention(
                    torch.from_numpy(q[b, :, h][rows][None]), torch.from_numpy(k[b, h, :T][None]),
                    torch.from_numpy(v[b, h, :T][None]),
                    attn_mask=torch.from_numpy(mask[rows][None])).numpy()[0]
                if not np.allclose(out[b, rows, h], ref, atol=1e-12, rtol=0):
                    bad.append(("sdpa", L, b, h))
                if not np.all(out[b, ~rows, h] == 0):
                    bad.append(("empty rows", L, b, h))
    return bad


def special_case_errors(seed=53):
    rng = np.random.default_rng(seed)
    bad = []
    q, k, v = _case(rng, T=10)
    T, D = 10, q.shape[3]
    # a block as long as the sequence: nothing visible
    if np.any(OB.block_attention(q, k, v, T, T) != 0):
        bad.append(("one block",))
    # two blocks: the second attends to all of the first
    out = OB.block_attention(q, k, v, T, 5)
    for j in range(5, 10):
        want = OA.attention_rows(q[0, j:j + 1, 0], k[0, 0, :5], v[0, 0, :5], 1 / np.sqrt(D))[0]
        if not np.allclose(out[0, j, 0], want, atol=1e-12, rtol=0):
            bad.append(("two blocks", j))
    # blocks of one: strictly earlier positions
    out = OB.block_attention(q, k, v, T, 1)
    for j in range(1, T):
        want = OA.attention_rows(q[1, j:j + 1, 1], k[1, 1, :j], v[1, 1, :j], 1 / np.sqrt(D))[0]
        if not np.allclose(out[1, j, 1], want, atol=1e-12, rtol=0):
            bad.append(("L = 1", j))
    return bad


PINS = [delayed_cache_errors, sdpa_errors, special_case_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


# ---- planted mistakes ----

def _mut_own_block(monkeypatch):
    # the query's own block up to itself is visible too (plain causal)
    monkeypatch.setattr(OB, "visible_keys", lambda j, L: list(range(j + 1)))


def _mut_off_by_one(monkeypatch):
    monkeypatch.setattr(OB, "visible_keys", lambda j, L: list(range(max(L * (j // L) - 1, 0))))


def _mut_ceil_blocks(monkeypatch):
    # block index rounded up (kept inside the sequences the pins use)
    monkeypatch.setattr(OB, "visible_keys", lambda j, L: list(range(min(L * (-(-j // L)), 20))))


def _mut_width_scale(monkeypatch):
    real = OB.block_attention
    monkeypatch.setattr(OB, "block_attention",
                        lambda q, k, v, T, L, scale=None: real(q, k, v, T, L,
                                                               1 / np.sqrt(q.shape[2] * q.shape[3])))


MUTANTS = [_mut_own_block, _mut_off_by_one, _mut_ceil_blocks, _mut_width_scale]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mutant(monkeypatch)
    failures = []
    for pin in PINS:
        failures += pin()
    assert failures

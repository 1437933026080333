"""Pins for the attention oracle (CPU only).

Each check compares ``oracle.attention`` with something that is not itself:
* brute force: every root-to-leaf path of the tree, built top-down from child
  lists, is laid out as an ordinary sequence after the prefix and run through
  torch's causal scaled-dot-product attention (float64); each path position
  must reproduce that node's tree-attention output;
* the paper's mask: for CaPE-shaped trees the dense mask_CaPE of Sec. 4.2 is
  written out from pos() and handed to the library routine as an explicit mask;
* closed forms and special cases (single visible key, identical keys, two keys,
  prefix permutation, empty cross-attention key set);
* planted mistakes: each pin battery must fail for a deliberately broken copy
  of the oracle's helpers.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import attention as A


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def _children(parents):
    ch = {m: [] for m in range(-1, len(parents))}
    for n, p in enumerate(parents):
        ch[int(p)].append(n)
    return ch


def _root_paths(parents):
    """All root-to-leaf paths, enumerated top-down (DFS over child lists)."""
    ch = _children(parents)
    paths = []

    def dfs(node, path):
        path = path + [node]
        if not ch[node]:
            paths.append(path)
        for c in ch[node]:
            dfs(c, path)

    for r in ch[-1]:
        dfs(r, [])
    return paths


def _sdpa(q, k, v, mask=None, causal=False, scale=None):
    q = torch.from_numpy(np.ascontiguousarray(q))[None, None]
    k = torch.from_numpy(np.ascontiguousarray(k))[None, None]
    v = torch.from_numpy(np.ascontiguousarray(v))[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    out = F.scaled_dot_product_attention(q, k, v, attn_mask=m, is_causal=causal, scale=scale)
    return out[0, 0].numpy()


def _random_tree(rng, n):
    return np.array([int(rng.integers(-1, i)) if i > 0 else -1 for i in range(n)], dtype=np.int64)


def bruteforce_error(fn, rng, trials=12):
    """Max |fn - causal attention over explicit root paths| on tiny trees."""
    worst = 0.0
    for _ in range(trials):
        L = int(rng.integers(0, 9))
        N = int(rng.integers(1, 9))
        D = int(rng.integers(2, 9))
        parents = _random_tree(rng, N)
        q = _rand(rng, N, D)
        k = _rand(rng, L + N, D)
        v = _rand(rng, L + N, D)
        got = fn(q, k, v, L, parents, None)
        for path in _root_paths(parents):
            rows = list(range(L)) + [L + m for m in path]
            seq_q = np.zeros((len(rows), D))
            seq_q[L:] = q[path]
            ref = _sdpa(seq_q, k[rows], v[rows], causal=True)
            for pos, node in enumerate(path):
                worst = max(worst, float(np.abs(ref[L + pos] - got[node]).max()))
    return worst


def cape_mask_error(fn, rng, trials=8):
    """Max |fn - attention under the paper's mask_CaPE| for CaPE-shaped trees."""
    worst = 0.0
    for _ in range(trials):
        gamma = int(rng.integers(1, 6))
        sizes = [int(rng.integers(0, 4)) for _ in range(gamma)]
        # pos() of the linearised proposal, 1-based as in the paper.
        pos = list(range(1, gamma + 1))
        for j, K in enumerate(sizes, start=1):
            pos += [j] * K
        beta = len(pos)
        parents = np.array([i - 1 for i in range(gamma)] +
                           [p - 2 for p in pos[gamma:]], dtype=np.int64)
        L = int(rng.integers(0, 6))
        D = 4
        q = _rand(rng, beta, D)
        k = _rand(rng, L + beta, D)
        v = _rand(rng, L + beta, D)
        allowed = np.zeros((beta, L + beta), dtype=bool)
        allowed[:, :L] = True
        for i in range(1, beta + 1):
            for j in range(1, beta + 1):
                if (j <= gamma and pos[i - 1] > j) or i == j:
                    allowed[i - 1, L + j - 1] = True
        ref = _sdpa(q, k, v, mask=allowed)
        got = fn(q, k, v, L, parents, None)
        worst = max(worst, float(np.abs(ref - got).max()))
    return worst


def chain_error(fn, rng, trials=6):
    """A chain tree must equal ordinary causal decoding of the appended tokens."""
    worst = 0.0
    for _ in range(trials):
        L, N, D = int(rng.integers(0, 10)), int(rng.integers(1, 7)), 8
        parents = np.arange(-1, N - 1)
        q, k, v = _rand(rng, N, D), _rand(rng, L + N, D), _rand(rng, L + N, D)
        seq_q = np.vstack([np.zeros((L, D)), q])
        ref = _sdpa(seq_q, k, v, causal=True)[L:]
        worst = max(worst, float(np.abs(ref - fn(q, k, v, L, parents, None)).max()))
    return worst


def cross_error(fn, rng, trials=6):
    """Cross mode: unmasked attention over the first L rows only."""
    worst = 0.0
    for _ in range(trials):
        L, N, D = int(rng.integers(1, 12)), int(rng.integers(1, 6)), 8
        q, k, v = _rand(rng, N, D), _rand(rng, L + 3, D), _rand(rng, L + 3, D)
        ref = _sdpa(q, k[:L], v[:L])
        worst = max(worst, float(np.abs(ref - fn(q, k, v, L, None, None)).max()))
    return worst


def two_key_error(fn):
    """Two visible keys: the weight of key 0 is the logistic function of the
    scaled score difference, sigma((s0 - s1) / sqrt(d))."""
    d = 4
    q = np.array([[1.0, 2.0, -1.0, 0.5]])
    k = np.array([[0.5, 1.0, 0.0, 2.0], [-1.0, 0.0, 1.0, 1.0]])
    v = np.array([[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]])
    s = (q @ k.T)[0] / np.sqrt(d)
    w0 = 1.0 / (1.0 + np.exp(-(s[0] - s[1])))
    got = fn(q, k, v, 1, np.array([-1]), None)
    return float(np.abs(got[0] - np.array([w0, 1.0 - w0, 0.0, 0.0])).max())


PINS = [bruteforce_error, cape_mask_error, chain_error, cross_error]


def _oracle(q, k, v, L, parents, scale):
    return A.tree_attention_head(q, k, v, L, parents, scale)


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin(_oracle, np.random.default_rng(1234)) < 1e-12


def test_two_keys_closed_form():
    assert two_key_error(_oracle) < 1e-15


def test_single_visible_key_is_exact():
    rng = np.random.default_rng(5)
    N, D = 6, 16
    q, k, v = _rand(rng, N, D), _rand(rng, N, D), _rand(rng, N, D)
    got = _oracle(q, k, v, 0, np.full(N, -1), None)
    assert np.array_equal(got, v)


def test_identical_keys_give_mean_of_visible_values():
    rng = np.random.default_rng(6)
    L, N, D = 5, 7, 8
    parents = _random_tree(rng, N)
    k = np.tile(_rand(rng, 1, D), (L + N, 1))
    v = _rand(rng, L + N, D)
    got = _oracle(_rand(rng, N, D), k, v, L, parents, None)
    for n in range(N):
        rows = list(range(L)) + [L + m for m in A.ancestor_or_self(parents, n)]
        assert np.abs(got[n] - v[rows].mean(axis=0)).max() < 1e-13


def test_prefix_permutation_invariance():
    rng = np.random.default_rng(7)
    L, N, D = 9, 5, 8
    parents = _random_tree(rng, N)
    q, k, v = _rand(rng, N, D), _rand(rng, L + N, D), _rand(rng, L + N, D)
    perm = np.concatenate([rng.permutation(L), np.arange(L, L + N)])
    a = _oracle(q, k, v, L, parents, None)
    b = _oracle(q, k[perm], v[perm], L, parents, None)
    assert np.abs(a - b).max() < 1e-13


def test_empty_cross_key_set_gives_zeros():
    rng = np.random.default_rng(8)
    got = _oracle(_rand(rng, 3, 8), _rand(rng, 4, 8), _rand(rng, 4, 8), 0, None, None)
    assert np.array_equal(got, np.zeros((3, 8)))


def test_batched_layout_matches_per_head():
    rng = np.random.default_rng(9)
    B, N, H, D, Lc = 2, 4, 3, 8, 12
    q = _rand(rng, B, N, H, D)
    k, v = _rand(rng, B, H, Lc, D), _rand(rng, B, H, Lc, D)
    seq = np.array([3, 8])
    parents = np.stack([_random_tree(rng, N) for _ in range(B)])
    out = A.tree_attention(q, k, v, seq, parents)
    for b in range(B):
        for h in range(H):
            ref = _oracle(q[b, :, h], k[b, h], v[b, h], seq[b], parents[b], None)
            assert np.array_equal(out[b, :, h], ref)


def test_invalid_parents_rejected():
    with pytest.raises(ValueError):
        A.ancestor_or_self(np.array([-1, 2, 0]), 1)


# ---- planted mistakes: every broken oracle must fail at least one pin ----

_REAL_ANC = A.ancestor_or_self
_REAL_ROWS = A.attention_rows

def _mut_drop_self(parents_b, n):
    return [m for m in _REAL_ANC(parents_b, n) if m != n]


def _mut_parent_only(parents_b, n):
    p = int(parents_b[n])
    return sorted([n] + ([p] if p >= 0 else []))


def _mut_off_by_one(parents_b, n):
    return [max(m - 1, 0) for m in _REAL_ANC(parents_b, n)]


def _mut_no_scale(q, k, v, scale):
    return _REAL_ROWS(q, k, v, 1.0)


def _mut_values_are_keys(q, k, v, scale):
    return _REAL_ROWS(q, k, k, scale)


def _mut_no_max_shift_and_no_norm(q, k, v, scale):
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    if k.shape[0] == 0:
        return np.zeros((q.shape[0], v.shape[1]))
    p = np.exp((q @ k.T) * scale)
    return p @ v


MUTANTS = [
    ("ancestor_or_self", _mut_drop_self),
    ("ancestor_or_self", _mut_parent_only),
    ("ancestor_or_self", _mut_off_by_one),
    ("attention_rows", _mut_no_scale),
    ("attention_rows", _mut_values_are_keys),
    ("attention_rows", _mut_no_max_shift_and_no_norm),
]


@pytest.mark.parametrize("name,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_planted_mistake_is_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(A, name, mutant)
    rng = np.random.default_rng(99)
    errors = [pin(_oracle, rng) for pin in PINS] + [two_key_error(_oracle)]
    assert max(errors) > 1e-6, errors

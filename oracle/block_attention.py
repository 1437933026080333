"""Oracle: block-wise masked cross-attention of draft training (test
infrastructure only).

What is computed (Sec. 4.1, "Block-wise Attention Mask"; the plain
definition written out):

* a training sequence of length T is cut into blocks of L tokens
  (block(j) = floor(j / L); L = 5 in the paper's experiments);
* the draft's query at position j attends, in each head, to the target's
  cached keys and values of the positions k with block(j) > block(k) --
  every position of the earlier blocks and none of its own block -- with the
  softmax(q k^T / sqrt(d_k)) v of the cross-attention sub-layer; the mask
  sends every other score to -inf.

Layout (the C ABI's): q ``[B, T, H, D]``; k_cache, v_cache ``[B, H, L_cap, D]``
holding the target's keys and values of positions 0 .. T - 1; out
``[B, T, H, D]``.  Reading: a query in the first block sees no key and its
output is zero (the softmax of an all-masked row is not defined).
"""

import numpy as np

from . import attention as OA


def block_of(j, L):
    return j // L


def visible_keys(j, L):
    """Positions k with block(j) > block(k): [0, L * block(j))."""
    return [k for k in range(L * block_of(j, L)) if block_of(j, L) > block_of(k, L)]


def block_attention(q, k_cache, v_cache, T, L, scale=None, positions=None):
    """out[b, j, h] = attention of q[b, j, h] over k_cache[b, h, visible_keys(j)],
    for every position j or only those listed (others stay zero)."""
    q = np.asarray(q, dtype=np.float64)
    B, _, H, D = q.shape
    sc = 1.0 / np.sqrt(D) if scale is None else float(scale)
    out = np.zeros((B, T, H, D), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            kh = np.asarray(k_cache[b, h], dtype=np.float64)
            vh = np.asarray(v_cache[b, h], dtype=np.float64)
            for j in (range(T) if positions is None else positions):
                keys = visible_keys(j, L)
                out[b, j, h] = OA.attention_rows(q[b, j:j + 1, h], kh[keys], vh[keys], sc)[0]
    return out

"""Oracle: tree-masked and cross softmax attention in float64 (test infrastructure only).

What is computed (no approximation, so this is the plain definition):

* Sec. 4.1, multi-head cross-attention equation: for one head,
  hd = SoftMax(Q K^T / sqrt(d_k)) V, with K, V the target model's cached rows
  of that head.  In the GliDe role the queries see every cached row up to the
  cache length and nothing else (the block mask of Sec. 4.1 is a training-time
  device only).
* Sec. 4.2, "Verification of Expanded Proposals", mask_CaPE equation: a
  proposal token attends to the proposal tokens in front of it and to itself.
  In a parent-indexed tree that is exactly the node's ancestor-or-self set; the
  target model additionally attends to the whole accepted prefix (the cache).

Layout conventions (the same as the C ABI, so tests can hand over the same
arrays):  q ``[B, N, H, D]``; k_cache, v_cache ``[B, H, L_cap, D]``; seq_lens
``[B]``; parents ``[B, N]`` with ``-1 <= parents[b, n] < n``.  Tree node ``m``
of sequence ``b`` has its key/value at cache row ``seq_lens[b] + m``.

Every input is upcast exactly to float64 before use.
"""

import numpy as np


def ancestor_or_self(parents_b, n):
    """Indices of the tree nodes visible to node ``n``: itself and every node
    reached by following parent links to a root (Sec. 4.2, mask_CaPE: the
    proposal tokens in front of a token, plus the token itself)."""
    seen = []
    m = int(n)
    if not 0 <= m < len(parents_b):
        raise ValueError("node index out of range")
    while m != -1:
        seen.append(m)
        p = int(parents_b[m])
        if not -1 <= p < m:
            raise ValueError("parents must satisfy -1 <= parents[n] < n")
        m = p
    return sorted(seen)


def attention_rows(q_rows, k_rows, v_rows, scale):
    """Softmax attention of a set of query vectors against one explicit key set.

    q_rows [Nq, D], k_rows [J, D], v_rows [J, D] -> [Nq, D] (float64).
    hd = SoftMax(q K^T * scale) V (Sec. 4.1).  An empty key set gives zeros.
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    k_rows = np.asarray(k_rows, dtype=np.float64)
    v_rows = np.asarray(v_rows, dtype=np.float64)
    if k_rows.shape[0] == 0:
        return np.zeros((q_rows.shape[0], v_rows.shape[1]), dtype=np.float64)
    s = (q_rows @ k_rows.T) * scale
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ v_rows


def tree_attention_head(q_h, k_h, v_h, seq_len, parents_b=None, scale=None, nodes=None):
    """One (sequence, head) unit of the hot path.

    q_h [N, D]: the N query rows of this head.
    k_h, v_h [L_cap, D]: this head's cache.
    seq_len: accepted prefix length L_b.
    parents_b [N] or None: tree parents (verification role) or None (GliDe
    cross-attention role: every query sees rows [0, L_b) and nothing else).
    nodes: optional subset of query rows to evaluate (the others stay 0).
    Returns [N, D] float64.
    """
    q_h = np.asarray(q_h, dtype=np.float64)
    k_h = np.asarray(k_h, dtype=np.float64)
    v_h = np.asarray(v_h, dtype=np.float64)
    n_q, d = q_h.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = int(seq_len)
    out = np.zeros((n_q, d), dtype=np.float64)
    for n in (range(n_q) if nodes is None else nodes):
        if parents_b is None:
            rows = list(range(L))
        else:
            rows = list(range(L)) + [L + m for m in ancestor_or_self(parents_b, n)]
        rows = np.asarray(rows, dtype=np.int64)
        out[n] = attention_rows(q_h[n:n + 1], k_h[rows], v_h[rows], scale)[0]
    return out


def tree_attention(q, k_cache, v_cache, seq_lens, parents=None, scale=None):
    """Whole-batch oracle: out[b, n, h] = tree_attention_head(...)[n] for every
    sequence b and head h.  Returns float64 ``[B, N, H, D]``."""
    q = np.asarray(q)
    B, N, H, D = q.shape
    out = np.zeros((B, N, H, D), dtype=np.float64)
    for b in range(B):
        pb = None if parents is None else np.asarray(parents[b])
        for h in range(H):
            out[b, :, h, :] = tree_attention_head(
                q[b, :, h, :], k_cache[b, h], v_cache[b, h], int(seq_lens[b]), pb, scale)
    return out

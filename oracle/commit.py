"""Oracle: committing a verified candidate tree to the KV cache (test
infrastructure only).

What is computed (a selection and a copy, so this is the plain definition):

* Sec. 3 (Background): verification accepts the first n proposal tokens and
  adds one token of the target's own; the accepted tokens and that extra token
  extend the prefix for the next round.
* Sec. 4.1 (GliDe): after a verification step only the KV cache of the
  accepted tokens is kept; the rows of the rejected tokens are discarded.
* Sec. 4.2 (verification of expanded proposals): the candidates of an expanded
  proposal are verified together as a tree; a candidate is accepted when its
  whole root path is (``verify.tree_verify``).

Layout (the C ABI's): node ``m`` of sequence ``b`` has its key/value at cache
row ``L_b + m`` of every layer (``L_b = seq_lens[b]``), caches ``[B, H, L_cap,
D]``.  Committing the accepted node ``n_a`` with root path ``n_1, ..., n_a``
(depths 1..a) moves those nodes' rows to ``L_b, ..., L_b + a - 1`` of every
layer's K and V cache and sets the sequence length to ``L_b + a``.  The extra
target token (the bonus) is returned; its keys and values come from the next
forward pass.

Readings where the paper is silent:
* rows outside ``[L_b, L_b + a)`` are left as they were (rejected rows past
  the new length are no longer covered by it);
* ``path[b, d]`` is the accepted node at depth ``d + 1`` for ``d < a`` and
  ``-1`` after;
* the acceptance rule is ``verify.tree_verify``'s (deepest accepted node,
  lowest index among equals).
"""

import numpy as np

from . import verify as OV


def root_path(parents_b, node):
    """The nodes from a root down to ``node``, in depth order, found by
    following parent links upwards."""
    path = []
    m = int(node)
    while m != -1:
        p = int(parents_b[m])
        if not -1 <= p < m:
            raise ValueError("parents must satisfy -1 <= parents[n] < n")
        path.append(m)
        m = p
    return path[::-1]


def verify_commit(logits, cand, parents, seq_lens, k_caches, v_caches):
    """Greedy verification followed by the cache commit.

    logits ``[B, N+1, V]`` float32 (row ``n + 1`` follows node ``n``, row 0 the
    prefix); cand, parents ``[B, N]``; seq_lens ``[B]``; k_caches, v_caches:
    one ``[B, H, L_cap, D]`` array per layer.  Inputs are not modified.

    Returns a dict: target_argmax ``[B, N+1]``, accept_len, last_node, bonus
    ``[B]``, path ``[B, N]``, seq_lens_out ``[B]`` and the committed caches
    k_out, v_out (new arrays, one per layer).
    """
    logits = np.asarray(logits, dtype=np.float32)
    cand = np.asarray(cand)
    parents = np.asarray(parents)
    B, N = cand.shape
    V = logits.shape[-1]
    ta = OV.argmax_rows(logits.reshape(B * (N + 1), V)).reshape(B, N + 1)
    accept_len, last_node, bonus = OV.tree_verify(ta, cand, parents)
    path = np.full((B, N), -1, dtype=np.int32)
    k_out = [np.array(k, copy=True) for k in k_caches]
    v_out = [np.array(v, copy=True) for v in v_caches]
    for b in range(B):
        nodes = root_path(parents[b], last_node[b]) if last_node[b] >= 0 else []
        if len(nodes) != int(accept_len[b]):
            raise AssertionError("accept length differs from the accepted node's depth")
        a = len(nodes)
        path[b, :a] = nodes
        L = int(seq_lens[b])
        for k_in, v_in, k_new, v_new in zip(k_caches, v_caches, k_out, v_out):
            if not 0 <= L <= k_in.shape[2] - N:
                raise ValueError("seq_lens[b] + N must fit the cache")
            rows = [L + n for n in nodes]
            # gather from the inputs, then write: the plain definition, with
            # no in-place ordering question
            k_new[b, :, L:L + a] = np.asarray(k_in)[b][:, rows]
            v_new[b, :, L:L + a] = np.asarray(v_in)[b][:, rows]
    seq_out = (np.asarray(seq_lens, dtype=np.int64) + accept_len).astype(np.int32)
    return {"target_argmax": ta, "accept_len": accept_len, "last_node": last_node,
            "bonus": bonus, "path": path, "seq_lens_out": seq_out, "k_out": k_out,
            "v_out": v_out}

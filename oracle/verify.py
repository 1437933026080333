"""Oracle: greedy acceptance of a candidate tree (test infrastructure only).

Sec. 3 (Background: Speculative Decoding): verification returns the first n
proposal tokens the target accepts plus one more target token for free; with
the "speculative decoding" acceptance strategy (the one Sec. 5.1 "Experiment
design" uses for every CaPE experiment) a token is accepted exactly when it is
the target's greedy choice at that point, so the output equals target greedy
search.  Sec. 4.2 verifies all candidates of the expanded proposal in one
target pass; a candidate is accepted when its whole root path is.

Slot layout of ``target_argmax`` ([N + 1] per sequence): slot 0 is the target's
greedy token after the accepted prefix (it judges depth-1 candidates), slot
n + 1 is the target's greedy token after tree node n (it judges node n's
children).  Both follow from the linearised tree: node n's logits row predicts
the token after the path ending at n.

Readings where the paper is silent: the accept length is the depth of the deepest
accepted node; when several accepted nodes share that depth the lowest node
index wins; padding nodes (token -1) never match; no node accepted gives
accept_len 0, last_node -1 and the bonus from slot 0.
"""

import numpy as np


def argmax_rows(logits):
    """Greedy token of every logits row: the first index of the maximum
    (np.argmax returns the first occurrence, i.e. ties go to the lower id)."""
    logits = np.asarray(logits, dtype=np.float32)
    return np.argmax(logits, axis=-1).astype(np.int32)


def tree_verify_one(target_argmax, cand, parents):
    """Returns (accept_len, last_node, bonus) for one sequence."""
    N = len(cand)
    accepted = [False] * N
    depth = [0] * N
    for c in range(N):
        p = int(parents[c])
        if not (-1 <= p < c):
            raise ValueError("parents must satisfy -1 <= parents[n] < n")
        depth[c] = 1 if p == -1 else depth[p] + 1
        parent_ok = (p == -1) or accepted[p]
        accepted[c] = parent_ok and int(cand[c]) == int(target_argmax[p + 1])
    accept_len, last_node = 0, -1
    for c in range(N):
        if accepted[c] and depth[c] > accept_len:
            accept_len, last_node = depth[c], c
    bonus = int(target_argmax[last_node + 1])
    return accept_len, last_node, bonus


def tree_verify(target_argmax, cand, parents):
    """Batched: target_argmax [B, N+1], cand [B, N], parents [B, N] ->
    accept_len [B], last_node [B], bonus [B] (int32)."""
    cand = np.asarray(cand)
    B = cand.shape[0]
    out = np.zeros((3, B), dtype=np.int32)
    for b in range(B):
        out[:, b] = tree_verify_one(target_argmax[b], cand[b], parents[b])
    return out[0], out[1], out[2]

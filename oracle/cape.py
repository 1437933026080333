"""Oracle: CaPE confidence-aware proposal expansion (test infrastructure only).

CaPE is a selection procedure, so this module takes the paper's steps in the
paper's order (Sec. 4.2, "Proposal Expansion" and "Verification of Expanded
Proposals"):

1. at each proposal position i the draft's most probable token x_{t+i} is the
   proposal token and its probability p_i is the confidence;
2. the expansion-set size is K_i = S(p_i) with S = 7, 5, 3, 1 on the bins
   (0, 0.3], (0.3, 0.6], (0.6, 0.8], (0.8, 1];
3. X_i holds the K_i most probable tokens other than x_{t+i};
4. expansion tokens are leaves: they are never used to predict later tokens;
5. linearisation: the proposal first, then X_1, X_2, ... appended in order.

Readings where the paper is silent:

* ties in "highest probability" go to the lower token id (a strict total order
  (prob desc, id asc)); probabilities are compared as the float32 values given;
* the S(p) bin edges are the float32 values nearest 0.3, 0.6, 0.8, upper bounds
  inclusive; p > 1 falls in the last bin and p <= 0 in the first;
* ``k`` (absent from the paper) caps |X_i|: K_i = min(S(p_i), k), with k = 0
  meaning "no cap" (S(p) <= 7 so k >= 7 is also paper-exact); ``fixed`` selects
  the fixed-size ablation of Sec. 5.4 ("The importance of confidence scores"),
  K_i = k for every i;
* K_i never exceeds V - 1 (there are only V - 1 other tokens);
* the verification budget (Sec. 5.3: at most 32 tokens per verify step) is the
  argument ``n_max``; when gamma + sum K_i exceeds it, the n_max - gamma leaf
  candidates kept are the first ones in the order (prob desc, position asc,
  rank asc); kept leaves are then emitted in linearisation order;
* unused slots up to n_max are padding: token -1, parent -1.

Tree encoding: node index = position in the linearised proposal (0-based).
Proposal token i has parent i - 1 (-1 for i = 0); a leaf of X_i has the same
parent as proposal token i, i.e. it sees the proposal tokens in front of
position i and itself, as the mask_CaPE equation requires.
"""

import numpy as np

MAX_EXPANSION = 7  # the largest value S(p) takes (Sec. 4.2)


def expansion_size(p):
    """S(p) of Sec. 4.2, evaluated in float32 against float32 bin edges."""
    p32 = np.float32(p)
    if p32 <= np.float32(0.3):
        return 7
    if p32 <= np.float32(0.6):
        return 5
    if p32 <= np.float32(0.8):
        return 3
    return 1


def rank_tokens(row):
    """Token ids of one draft distribution in the order (prob desc, id asc).

    np.lexsort sorts by the last key first: primary key -prob (float32
    negation is exact), secondary key the token id.
    """
    row = np.asarray(row, dtype=np.float32)
    ids = np.arange(row.shape[0])
    return np.lexsort((ids, -row))


def expansion_sizes(probs, k, fixed=False):
    """K_i for every position of one sequence's draft rows ``probs [gamma, V]``."""
    probs = np.asarray(probs, dtype=np.float32)
    gamma, V = probs.shape
    sizes = []
    for i in range(gamma):
        order = rank_tokens(probs[i])
        p_i = probs[i, order[0]]
        if fixed:
            K = int(k)
        else:
            K = expansion_size(p_i)
            if k > 0:
                K = min(K, int(k))
        sizes.append(min(K, V - 1))
    return sizes


def keep_within_budget(candidates, budget):
    """Leaf candidates kept under the verification budget (Sec. 5.3 caps the
    tokens verified per step): all of them when they fit, else the ``budget``
    first ones in the order (prob desc, position asc, rank asc).

    candidates: list of (position i, rank r, token, prob)."""
    if len(candidates) <= budget:
        return list(candidates)
    by_confidence = sorted(candidates, key=lambda c: (-c[3], c[0], c[1]))
    return by_confidence[:budget]


def linearise(proposal, leaves, n_max):
    """Sec. 4.2: the proposal first, then the expansion sets appended in
    position order.  Proposal token i has parent i - 1; a leaf of X_i has the
    parent of proposal token i.  Slots past the tree are padding (-1, -1)."""
    gamma = len(proposal)
    tokens = np.full(n_max, -1, dtype=np.int32)
    parents = np.full(n_max, -1, dtype=np.int32)
    for i in range(gamma):
        tokens[i] = proposal[i]
        parents[i] = i - 1
    ordered = sorted(leaves, key=lambda c: (c[0], c[1]))
    for j, (i, _r, tok, _p) in enumerate(ordered):
        tokens[gamma + j] = tok
        parents[gamma + j] = i - 1
    return tokens, parents, gamma + len(ordered)


def cape_expand_one(probs, k, n_max, fixed=False):
    """Expanded proposal of one sequence.

    probs [gamma, V] float32: draft next-token distributions p_D(. | x_<t+i).
    Returns (tokens [n_max] int32, parents [n_max] int32, n_nodes int).
    """
    probs = np.asarray(probs, dtype=np.float32)
    gamma, V = probs.shape
    if n_max < gamma:
        raise ValueError("n_max must be >= gamma")
    sizes = expansion_sizes(probs, k, fixed)

    proposal = []        # x_{t+i}: the most probable token at each position
    candidates = []      # (position i, rank r >= 1, token, prob)
    for i in range(gamma):
        order = rank_tokens(probs[i])
        proposal.append(int(order[0]))
        for r in range(1, sizes[i] + 1):
            tok = int(order[r])
            candidates.append((i, r, tok, probs[i, tok]))

    kept = keep_within_budget(candidates, n_max - gamma)
    return linearise(proposal, kept, n_max)


def cape_expand(draft_probs, k, n_max, fixed=False):
    """Batched form: draft_probs [B, gamma, V] -> tokens [B, n_max],
    parents [B, n_max], n_nodes [B] (all int32)."""
    draft_probs = np.asarray(draft_probs, dtype=np.float32)
    B = draft_probs.shape[0]
    tokens = np.zeros((B, n_max), dtype=np.int32)
    parents = np.zeros((B, n_max), dtype=np.int32)
    n_nodes = np.zeros(B, dtype=np.int32)
    for b in range(B):
        tokens[b], parents[b], n_nodes[b] = cape_expand_one(draft_probs[b], k, n_max, fixed)
    return tokens, parents, n_nodes

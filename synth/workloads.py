"""Synthetic stand-ins for the paper's decoding workloads.

The paper measures on MT-Bench, GSM8K, Finance-Alpaca, Spider and
Code-Search-Python with Vicuna / Mistral targets (Sec. 5.1); none of those are
available, so these seeded inputs stand in for them.  They keep the paper's
workload structure: batch-1 CaPE decoding with proposal length gamma = 5
(Sec. 5.1, "Experiment design"), at most 32 verified tokens per step (Sec. 5.3),
chain-plus-leaves trees (Sec. 4.2), and the Vicuna attention shapes (head_dim
128, multi-head attention) with the prefix lengths of each workload below.

Recipe (seed s):
* host arrays come from ``numpy.random.Generator(PCG64)`` streams spawned from
  ``SeedSequence(s)``: stream 0 prefix lengths, 1 draft probabilities, 2 target
  logits, 3 planting choices, 4 chain / random-tree tokens;
* draft rows are Dirichlet(0.3) over the vocabulary; in each row one token is
  then raised to twice, and one to 1.5 times, the largest raw value of the
  whole batch, and the row is renormalised.  So the proposal token and the
  first expansion token of every position are known, and every position's
  first expansion token outranks any other candidate when the verification
  budget forces a cut;
* target logits are N(0, 1) float32; acceptance is planted: a depth a ~ U{0..D}
  per sequence, the path runs down the proposal chain and, with probability
  1/2, ends on the first expansion token of position a; each logits row on the
  path gets the path token raised to (row max + 1), and the row after the
  path's last node gets a token that is none of that node's children;
* Q, K and V are bfloat16 N(0, 1) (float32 in fp32 mode) drawn in float32
  from a torch generator seeded with 1000 s + layer, in the order K cache,
  V cache, q; the GliDe cross-attention queries use layer index 999 and read
  the last layer's cache.  Tree rows [L_b, L_b + N) of the cache are part of
  the same draw.

Nothing here calls the oracle or the HIP library.
"""

from dataclasses import dataclass

import numpy as np

VOCAB = 32000
HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    heads: int
    batch: int
    prefix_lo: int
    prefix_hi: int
    nodes: int          # N: tree nodes verified per sequence
    depth: int          # gamma: proposal length = tree depth
    k: int              # expansion cap used to build the attention tree
    k_config: int       # the workload's stated top-k (separate CaPE parity runs)
    tree: str           # "chain" or "cape"
    cross: bool         # also one GliDe cross-attention layer
    cross_queries: int = 0  # its query rows per sequence (0 when there is none)
    vocab: int = VOCAB
    head_dim: int = HEAD_DIM

    @property
    def l_cap(self):
        return self.prefix_hi + self.nodes


WORKLOADS = {
    # 7B single layer, a 5-token chain, greedy verify on random logits.
    1: Workload("7b-1layer-chain5", 1, 32, 1, 512, 512, 5, 5, 0, 0, "chain", False),
    # Vicuna-7B: 32 layers, prefix 2048, 16-node CaPE tree of depth 5, k = 3,
    # plus one 5-query GliDe cross-attention layer on the same cache.
    2: Workload("vicuna7b-cape16", 32, 32, 1, 2048, 2048, 16, 5, 3, 3, "cape", True, 5),
    # Vicuna-13B: 40 layers x 40 heads, B = 4, prefixes U[1024, 4096], 32 nodes,
    # depth 6.  k = 4 gives only 6 + 24 = 30 nodes, so the attention tree uses
    # the uncapped S(p) (k = 7) to reach 32; k = 4 runs as its own CaPE case.
    3: Workload("vicuna13b-cape32", 40, 40, 4, 1024, 4096, 32, 6, 7, 4, "cape", False),
    # Vicuna-33B: 60 layers x 52 heads, B = 8, prefixes U[4096, 8192], 64 nodes,
    # depth 8 (k = 5 gives 48 nodes; the attention tree uses k = 7).
    4: Workload("vicuna33b-cape64", 60, 52, 8, 4096, 8192, 64, 8, 7, 5, "cape", False),
    # Long context at 7B head shape: 4 layers, B = 16, prefixes U[16384, 32768],
    # 64-node trees of depth 8, plus a 5-query cross-attention layer per
    # sequence (the stated query count, not the tree depth).
    5: Workload("7b-longctx-cape64", 4, 32, 16, 16384, 32768, 64, 8, 7, 7, "cape", True, 5),
}


def _streams(seed, n=5):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def prefix_lengths(wl, seed):
    rng = _streams(seed)[0]
    return rng.integers(wl.prefix_lo, wl.prefix_hi + 1, size=wl.batch).astype(np.int32)


def draft_probs(wl, seed, batch=None, gamma=None, vocab=None):
    """Draft distributions [B, gamma, V] float32 with a known proposal token
    (``chain[b, i]``) and a known first expansion token (``first_leaf[b, i]``)."""
    B = wl.batch if batch is None else batch
    G = wl.depth if gamma is None else gamma
    V = wl.vocab if vocab is None else vocab
    rng = _streams(seed)[1]
    raw = rng.dirichlet(np.full(V, 0.3), size=B * G).reshape(B, G, V)
    top = raw.max()
    chain = np.zeros((B, G), dtype=np.int64)
    first_leaf = np.zeros((B, G), dtype=np.int64)
    for b in range(B):
        for i in range(G):
            a, c = rng.choice(V, size=2, replace=False)
            chain[b, i], first_leaf[b, i] = a, c
            raw[b, i, a] = 2.0 * top
            raw[b, i, c] = 1.5 * top
            raw[b, i] /= raw[b, i].sum()
    return raw.astype(np.float32), chain, first_leaf


def peaked_probs(batch, gamma, vocab, seed, confidences):
    """Rows whose top probability is exactly one of ``confidences`` (float32),
    the rest of the mass spread over the other tokens, so that every S(p) bin
    and bin edge is exercised.  Returns float32 [batch, gamma, vocab]."""
    rng = _streams(seed)[1]
    conf = np.asarray(confidences, dtype=np.float32)
    out = np.zeros((batch, gamma, vocab), dtype=np.float32)
    for b in range(batch):
        for i in range(gamma):
            p = conf[rng.integers(0, conf.shape[0])]
            rest = rng.dirichlet(np.full(vocab - 1, 0.5)).astype(np.float32)
            rest *= (np.float32(1.0) - p) if p < 1 else np.float32(0.0)
            rest = np.minimum(rest, np.float32(p) * np.float32(0.999))
            top_id = rng.integers(0, vocab)
            row = np.insert(rest, top_id, p)
            out[b, i] = row
    return out


def chain_tokens(wl, seed):
    """Random proposal tokens for a chain tree [B, N] (int32, distinct per row)."""
    rng = _streams(seed)[4]
    return np.stack([rng.choice(wl.vocab, size=wl.nodes, replace=False)
                     for _ in range(wl.batch)]).astype(np.int32)


def random_parents(batch, nodes, max_depth, seed):
    """Uniformly random topological parent arrays: parents[n] is drawn from
    {-1} and the earlier nodes whose depth is below ``max_depth``."""
    rng = _streams(seed)[4]
    out = np.zeros((batch, nodes), dtype=np.int32)
    for b in range(batch):
        depth = []
        for n in range(nodes):
            choices = [-1] + [m for m in range(n) if depth[m] < max_depth]
            p = int(choices[rng.integers(0, len(choices))])
            out[b, n] = p
            depth.append(1 if p == -1 else depth[p] + 1)
    return out


def random_tokens(batch, nodes, vocab_used, seed):
    """Candidate tokens drawn from a small id range so that siblings collide."""
    rng = _streams(seed)[3]
    return rng.integers(0, vocab_used, size=(batch, nodes)).astype(np.int32)


def _raise_to_argmax(row, tok):
    row[tok] = row.max() + np.float32(1.0)


def planted_logits_cape(wl, seed, chain, first_leaf, probs, n_rows=None):
    """Target logits [B, N+1, V] with a planted accepted path per sequence.

    Returns (logits, planted_depth [B], ends_on_leaf [B]).  ``chain`` and
    ``first_leaf`` are the known tokens from ``draft_probs``; ``probs`` is used
    only to pick a stop token of lowest draft probability (never a candidate).
    """
    B, G = chain.shape
    V = probs.shape[-1]
    rows = (wl.nodes + 1) if n_rows is None else n_rows
    st = _streams(seed)
    logits = st[2].standard_normal((B, rows, V), dtype=np.float32)
    rng = st[3]
    depth = np.zeros(B, dtype=np.int32)
    leaf_end = np.zeros(B, dtype=bool)
    for b in range(B):
        a = int(rng.integers(0, G + 1))
        on_leaf = bool(a >= 1 and rng.integers(0, 2) == 1)
        for d in range(1, a):            # chain nodes at depths 1 .. a-1
            _raise_to_argmax(logits[b, d - 1], chain[b, d - 1])
        if a >= 1:                       # depth a: chain node or first leaf
            tok = first_leaf[b, a - 1] if on_leaf else chain[b, a - 1]
            _raise_to_argmax(logits[b, a - 1], tok)
        if not on_leaf and a < G:        # stop: a token that is no child
            stop_row = a                 # slot after chain node a-1 (0 when a == 0)
            _raise_to_argmax(logits[b, stop_row], int(np.argmin(probs[b, a])))
        depth[b], leaf_end[b] = a, on_leaf
    return logits, depth, leaf_end


def planted_logits_chain(wl, seed, cand):
    """Target logits [B, N+1, V] for a chain tree with a planted accept length."""
    B, N = cand.shape
    st = _streams(seed)
    logits = st[2].standard_normal((B, N + 1, wl.vocab), dtype=np.float32)
    rng = st[3]
    depth = np.zeros(B, dtype=np.int32)
    for b in range(B):
        a = int(rng.integers(0, N + 1))
        for d in range(a):
            _raise_to_argmax(logits[b, d], cand[b, d])
        if a < N:
            _raise_to_argmax(logits[b, a], (int(cand[b, a]) + 1) % wl.vocab)
        depth[b] = a
    return logits, depth


def torch_normal(shape, generator, dtype, device):
    """N(0, 1) tensor drawn in float32 from ``generator`` and cast to ``dtype``."""
    import torch
    x = torch.randn(shape, generator=generator, dtype=torch.float32, device=device)
    return x.to(dtype)


def layer_seed(seed, layer):
    """Seed of one layer's tensors, so any layer can be drawn on its own."""
    return int(seed) * 1000 + int(layer)


def attention_layer(wl, seed, layer, dtype, device, batch=None, heads=None, l_cap=None,
                    n_q=None):
    """(q, k_cache, v_cache) of one layer: q [B, Nq, H, D], caches
    [B, H, L_cap, D], N(0, 1) drawn in the order K cache, V cache, q."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(layer_seed(seed, layer))
    B = wl.batch if batch is None else batch
    H = wl.heads if heads is None else heads
    Lc = wl.l_cap if l_cap is None else l_cap
    Nq = wl.nodes if n_q is None else n_q
    D = wl.head_dim
    k = torch_normal((B, H, Lc, D), g, dtype, device)
    v = torch_normal((B, H, Lc, D), g, dtype, device)
    q = torch_normal((B, Nq, H, D), g, dtype, device)
    return q, k, v


def cross_queries(wl, seed, dtype, device):
    """GliDe cross-attention queries [B, Nq, H, D] (one draft layer)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(layer_seed(seed, 999))
    return torch_normal((wl.batch, wl.cross_queries, wl.heads, wl.head_dim), g, dtype, device)

"""Pins for the CaPE oracle (CPU only).

* S(p) boundary table at every float32 bin edge and its neighbours (Sec. 4.2);
* a hand-derived worked example (tests/golden/cape_worked_example.json);
* the paper's text with no budget pressure: X_i is the K_i most probable tokens
  other than x_{t+i}, ranked here with Python's own sort;
* the budget rule characterised by brute force: among all subsets of the
  candidates of the budget's size exactly one has every kept candidate ahead
  of every dropped one, and it is the oracle's;
* invariants: siblings distinct, leaves differ from the proposal token at their
  position, parents topological, node count, and the tree's visibility equal
  to the paper's mask_CaPE written out from pos();
* planted mistakes in the oracle's helpers must fail at least one pin.
"""

import itertools
import json
import os

import numpy as np
import pytest

from oracle import cape as C
from synth import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "cape_worked_example.json")
f32 = np.float32


def _next_up(x):
    return np.nextafter(f32(x), f32(2.0), dtype=np.float32)


def _next_down(x):
    return np.nextafter(f32(x), f32(-1.0), dtype=np.float32)


S_TABLE = [
    (f32(1e-30), 7), (f32(0.05), 7), (f32(0.3), 7), (_next_up(0.3), 5),
    (f32(0.45), 5), (f32(0.6), 5), (_next_up(0.6), 3), (f32(0.7), 3),
    (f32(0.8), 3), (_next_up(0.8), 1), (f32(0.95), 1), (f32(1.0), 1),
    (_next_down(0.3), 7), (_next_down(0.6), 5), (_next_down(0.8), 3),
]


def s_table_errors():
    return [(p, s, C.expansion_size(p)) for p, s in S_TABLE if C.expansion_size(p) != s]


def golden_errors():
    g = json.load(open(GOLDEN))
    probs = np.asarray(g["probs"], dtype=np.float32)
    bad = []
    for case in g["cases"]:
        t, p, n = C.cape_expand_one(probs, case["k"], case["n_max"], bool(case["fixed"]))
        if list(t) != case["tokens"] or list(p) != case["parents"] or n != case["n_nodes"]:
            bad.append((case, list(t), list(p), n))
    return bad


def _python_rank(row):
    return sorted(range(len(row)), key=lambda t: (-float(row[t]), t))


def text_errors(seed=3, trials=20):
    """No budget pressure: the tree must be the literal Sec. 4.2 construction."""
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        gamma, V = int(rng.integers(1, 5)), int(rng.integers(2, 12))
        probs = np.round(rng.random((gamma, V)) * 8).astype(np.float32) / f32(8.0)
        k = int(rng.integers(0, 9))
        tokens, parents, n = C.cape_expand_one(probs, k, gamma * 8)
        want_tokens, want_parents = [], []
        leaves_t, leaves_p = [], []
        for i in range(gamma):
            order = _python_rank(probs[i])
            x, p = order[0], probs[i][order[0]]
            size = 7 if p <= f32(0.3) else 5 if p <= f32(0.6) else 3 if p <= f32(0.8) else 1
            if k > 0:
                size = min(size, k)
            size = min(size, V - 1)
            want_tokens.append(x)
            want_parents.append(i - 1)
            leaves_t += order[1:1 + size]
            leaves_p += [i - 1] * size
        want_tokens += leaves_t
        want_parents += leaves_p
        if list(tokens[:n]) != want_tokens or list(parents[:n]) != want_parents:
            bad.append((probs, k))
    return bad


def _order_key(c):
    return (-float(c[3]), c[0], c[1])


def budget_errors(seed=4, trials=25):
    """Brute force over subsets: the kept set is the unique one whose members
    all precede every dropped candidate in (prob desc, position, rank)."""
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        gamma, V = int(rng.integers(1, 4)), int(rng.integers(3, 7))
        probs = (rng.integers(0, 4, size=(gamma, V)).astype(np.float32) / f32(4.0))
        n_max = gamma + int(rng.integers(0, 5))
        tokens, parents, n = C.cape_expand_one(probs, 0, n_max)
        cands = []
        for i in range(gamma):
            order = _python_rank(probs[i])
            size = C.expansion_sizes(probs[i:i + 1], 0)[0]
            cands += [(i, r, order[r], probs[i][order[r]]) for r in range(1, size + 1)]
        budget = min(n_max - gamma, len(cands))
        valid = []
        for subset in itertools.combinations(range(len(cands)), budget):
            kept = set(subset)
            dropped = [c for j, c in enumerate(cands) if j not in kept]
            if all(_order_key(cands[j]) < _order_key(d) for j in kept for d in dropped):
                valid.append(sorted(kept))
        if len(valid) != 1:
            bad.append(("not unique", probs, n_max))
            continue
        want = [cands[j] for j in valid[0]]  # cands are already in (i, r) order
        got = list(zip(tokens[gamma:n], parents[gamma:n]))
        if got != [(c[2], c[0] - 1) for c in want]:
            bad.append((probs, n_max, got, want))
    return bad


def _mask_from_pos(gamma, pos):
    beta = len(pos)
    m = np.zeros((beta, beta), dtype=bool)
    for i in range(1, beta + 1):
        for j in range(1, beta + 1):
            m[i - 1, j - 1] = (j <= gamma and pos[i - 1] > j) or i == j
    return m


def _visible_from_parents(parents, n_nodes):
    m = np.zeros((n_nodes, n_nodes), dtype=bool)
    for n in range(n_nodes):
        a = n
        while a != -1:
            m[n, a] = True
            a = parents[a]
    return m


def invariant_errors(seed=5, trials=12):
    bad = []
    confid = [f32(0.05), f32(0.3), _next_up(0.3), f32(0.6), _next_up(0.6), f32(0.8),
              _next_up(0.8), f32(1.0)]
    for t in range(trials):
        probs = W.peaked_probs(1, 4, 64, seed + t, confid)[0]
        n_max = [4, 10, 16, 40][t % 4]
        tokens, parents, n = C.cape_expand_one(probs, 0, n_max)
        gamma = probs.shape[0]
        sizes = C.expansion_sizes(probs, 0)
        if n != min(n_max, gamma + sum(sizes)):
            bad.append("node count")
        if any(not (-1 <= parents[j] < j) for j in range(n)):
            bad.append("topological")
        if any(tokens[j] != -1 or parents[j] != -1 for j in range(n, n_max)):
            bad.append("padding")
        pos = list(range(1, gamma + 1)) + [int(parents[j]) + 2 for j in range(gamma, n)]
        for j in range(gamma, n):
            if tokens[j] == tokens[pos[j] - 1]:
                bad.append("leaf equals proposal token")
        for i in range(1, gamma + 1):
            sib = [tokens[j] for j in range(gamma, n) if pos[j] == i]
            if len(set(sib)) != len(sib):
                bad.append("siblings repeat")
            order = _python_rank(probs[i - 1])
            if sib != order[1:1 + len(sib)]:
                bad.append("kept leaves are not the top of their position")
        if not np.array_equal(_mask_from_pos(gamma, pos), _visible_from_parents(parents, n)):
            bad.append("mask_CaPE")
    return bad


PINS = [s_table_errors, golden_errors, text_errors, budget_errors, invariant_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


def test_batched_matches_per_sequence():
    wl = W.WORKLOADS[2]
    probs, _, _ = W.draft_probs(wl, 11, batch=2, vocab=500)
    t, p, n = C.cape_expand(probs, 3, 16)
    for b in range(2):
        tb, pb, nb = C.cape_expand_one(probs[b], 3, 16)
        assert np.array_equal(t[b], tb) and np.array_equal(p[b], pb) and n[b] == nb


def test_planted_draft_rows_have_known_top_two():
    wl = W.WORKLOADS[2]
    probs, chain, leaf = W.draft_probs(wl, 12, vocab=2000)
    t, p, n = C.cape_expand(probs, wl.k, wl.nodes)
    assert n[0] == wl.nodes
    assert list(t[0, :wl.depth]) == list(chain[0])
    kept_first = [t[0, j] for j in range(wl.depth, n[0]) if p[0, j] >= -1]
    for i in range(wl.depth):
        assert leaf[0, i] in kept_first


def test_gamma_above_budget_rejected():
    with pytest.raises(ValueError):
        C.cape_expand_one(np.ones((4, 8), dtype=np.float32), 0, 3)


# ---- planted mistakes ----

def _mut_exclusive_edges(p):
    p32 = np.float32(p)
    return 7 if p32 < f32(0.3) else 5 if p32 < f32(0.6) else 3 if p32 < f32(0.8) else 1


def _mut_ties_high_id(row):
    row = np.asarray(row, dtype=np.float32)
    return np.lexsort((-np.arange(row.shape[0]), -row))


def _mut_budget_position_major(cands, budget):
    return list(cands)[:budget]


def _mut_leaf_parent_is_proposal_token(proposal, leaves, n_max):
    t, p, n = _REAL_LIN(proposal, leaves, n_max)
    g = len(proposal)
    for j in range(g, n):
        p[j] = p[j] + 1
    return t, p, n


_REAL_LIN = C.linearise

MUTANTS = [
    ("expansion_size", _mut_exclusive_edges),
    ("rank_tokens", _mut_ties_high_id),
    ("keep_within_budget", _mut_budget_position_major),
    ("linearise", _mut_leaf_parent_is_proposal_token),
]


@pytest.mark.parametrize("name,mutant", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_planted_mistake_is_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(C, name, mutant)
    failures = []
    for pin in PINS:
        try:
            failures += pin()
        except Exception as e:  # a crash is also a caught mistake
            failures.append(repr(e))
    assert failures

"""Pins for the greedy-acceptance oracle (CPU only).

* hand-derived worked example (tests/golden/verify_worked_example.json);
* a chain tree reduces to vanilla speculative decoding (Sec. 3): the accept
  length is the longest prefix of the proposal that matches the target's
  greedy tokens, computed here by a plain scan;
* brute force: every root-to-node path, enumerated top-down, is checked token
  by token; the deepest fully matching one (lowest end index on ties) wins;
* planted acceptance from the seeded generator gives a known accept length;
* accept_len <= tree depth; on CaPE trees the accepted nodes form one path;
* argmax: first index of the maximum, against a plain Python scan;
* planted mistakes in the oracle must fail at least one pin.
"""

import json
import os

import numpy as np
import pytest

from oracle import cape as C
from oracle import verify as Vf
from synth import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "verify_worked_example.json")


def golden_errors():
    g = json.load(open(GOLDEN))
    bad = []
    for case in g["cases"]:
        got = Vf.tree_verify_one(case["target_argmax"], g["tokens"], g["parents"])
        if got != (case["accept_len"], case["last_node"], case["bonus"]):
            bad.append((case, got))
    return bad


def chain_errors(seed=1, trials=200):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        N = int(rng.integers(1, 9))
        cand = rng.integers(0, 3, size=N)
        ta = rng.integers(0, 3, size=N + 1)
        n = 0
        while n < N and cand[n] == ta[n]:
            n += 1
        want = (n, n - 1, int(ta[n]))
        got = Vf.tree_verify_one(ta, cand, np.arange(-1, N - 1))
        if got != want:
            bad.append((cand, ta, got, want))
    return bad


def _paths_top_down(parents):
    ch = {m: [] for m in range(-1, len(parents))}
    for n, p in enumerate(parents):
        ch[int(p)].append(n)
    out = []

    def dfs(node, path):
        path = path + [node]
        out.append(path)
        for c in ch[node]:
            dfs(c, path)

    for r in ch[-1]:
        dfs(r, [])
    return out


def bruteforce_errors(seed=2, trials=300):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        N = int(rng.integers(1, 10))
        parents = [int(rng.integers(-1, n)) if n else -1 for n in range(N)]
        cand = rng.integers(0, 3, size=N)
        ta = rng.integers(0, 3, size=N + 1)
        best = (0, -1)
        for path in _paths_top_down(parents):
            prev = -1
            ok = True
            for node in path:
                if cand[node] != ta[prev + 1]:
                    ok = False
                    break
                prev = node
            if ok:
                key = (len(path), -path[-1])
                if key > (best[0], -best[1]):
                    best = (len(path), path[-1])
        want = (best[0], best[1], int(ta[best[1] + 1]))
        got = Vf.tree_verify_one(ta, cand, parents)
        if got != want:
            bad.append((parents, cand, ta, got, want))
    return bad


def planted_errors(seed=3):
    bad = []
    for cfg in (2, 3):
        wl = W.WORKLOADS[cfg]
        probs, chain, leaf = W.draft_probs(wl, seed, vocab=3000)
        tokens, parents, _ = C.cape_expand(probs, wl.k, wl.nodes)
        logits, depth, _ = W.planted_logits_cape(wl, seed, chain, leaf, probs)
        ta = Vf.argmax_rows(logits)
        acc, last, bonus = Vf.tree_verify(ta, tokens, parents)
        if not np.array_equal(acc, depth):
            bad.append((cfg, acc, depth))
    wl = W.WORKLOADS[1]
    cand = W.chain_tokens(wl, seed)
    logits, depth = W.planted_logits_chain(wl, seed, cand)
    acc, _, _ = Vf.tree_verify(Vf.argmax_rows(logits), cand, np.tile(np.arange(-1, wl.nodes - 1), (wl.batch, 1)))
    if not np.array_equal(acc, depth):
        bad.append((1, acc, depth))
    return bad


def depth_and_single_path_errors(seed=4, trials=40):
    rng = np.random.default_rng(seed)
    bad = []
    for t in range(trials):
        probs = rng.random((4, 12)).astype(np.float32)
        tokens, parents, n = C.cape_expand_one(probs, 0, 20)
        ta = rng.integers(0, 12, size=21)
        acc, last, _ = Vf.tree_verify_one(ta, tokens, parents)
        if acc > 4:
            bad.append("deeper than the tree")
        # on a CaPE tree the accepted nodes are one root path
        accepted = []
        for c in range(len(tokens)):
            p = parents[c]
            if tokens[c] == ta[p + 1] and (p == -1 or p in accepted):
                accepted.append(c)
        depths = {}
        for c in accepted:
            d, a = 0, c
            while a != -1:
                d, a = d + 1, parents[a]
            depths.setdefault(d, []).append(c)
        if any(len(v) > 1 for v in depths.values()):
            bad.append("two accepted nodes at one depth")
        if acc != (max(depths) if depths else 0):
            bad.append("accept length")
    return bad


def argmax_errors(seed=5):
    rng = np.random.default_rng(seed)
    bad = []
    x = rng.integers(0, 5, size=(50, 17)).astype(np.float32)
    x[3] = 2.0
    x[4, 7] = -0.0
    got = Vf.argmax_rows(x)
    for r in range(x.shape[0]):
        best = 0
        for j in range(1, x.shape[1]):
            if x[r, j] > x[r, best]:
                best = j
        if got[r] != best:
            bad.append((r, got[r], best))
    return bad


PINS = [golden_errors, chain_errors, bruteforce_errors, planted_errors,
        depth_and_single_path_errors, argmax_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


def test_invalid_parents_rejected():
    with pytest.raises(ValueError):
        Vf.tree_verify_one([0, 0, 0], [0, 0], [-1, 1])


# ---- planted mistakes ----

def _mut_wrong_slot(target_argmax, cand, parents):
    return _REAL(list(target_argmax[1:]) + [target_argmax[0]], cand, parents)


def _mut_ignore_parent(target_argmax, cand, parents):
    N = len(cand)
    depth = [0] * N
    best = (0, -1)
    for c in range(N):
        p = int(parents[c])
        depth[c] = 1 if p == -1 else depth[p] + 1
        if int(cand[c]) == int(target_argmax[p + 1]) and depth[c] > best[0]:
            best = (depth[c], c)
    return best[0], best[1], int(target_argmax[best[1] + 1])


def _mut_last_on_ties(target_argmax, cand, parents):
    acc, last, bonus = _REAL(target_argmax, cand, parents)
    N = len(cand)
    for c in range(N - 1, -1, -1):
        a, d = c, 0
        ok = True
        while a != -1:
            if int(cand[a]) != int(target_argmax[int(parents[a]) + 1]):
                ok = False
            d, a = d + 1, int(parents[a])
        if ok and d == acc and acc > 0:
            return acc, c, int(target_argmax[c + 1])
    return acc, last, bonus


_REAL = Vf.tree_verify_one

MUTANTS = [_mut_wrong_slot, _mut_ignore_parent, _mut_last_on_ties]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_planted_mistake_is_caught(monkeypatch, mutant):
    monkeypatch.setattr(Vf, "tree_verify_one", mutant)
    failures = []
    for pin in PINS:
        failures += pin()
    assert failures

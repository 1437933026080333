"""Pins for the cache-commit oracle (CPU only).

* hand-derived worked examples (tests/golden/commit_worked_example.json);
* the committed prefix is what the accepted node saw: the accepted node's
  query attending under the CaPE mask to the old cache equals the same query
  attending, with no mask, to the committed rows [0, L + a) (attention oracle,
  Sec. 4.2, against plain softmax attention);
* brute force: every root-to-node path, enumerated top-down through child
  lists, is checked token by token; the committed path is the deepest fully
  matching one (lowest end index on ties);
* rows outside [L, L + a) and other sequences are untouched; a chain that is
  accepted in full leaves the cache as it was;
* planted mistakes in the oracle must fail at least one pin.
"""

import json
import os

import numpy as np
import pytest

from oracle import attention as OA
from oracle import commit as OCm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "commit_worked_example.json")


def _logits_for(ta, V):
    B, R = ta.shape
    lg = np.zeros((B, R, V), dtype=np.float32)
    for b in range(B):
        for r in range(R):
            lg[b, r, ta[b, r]] = 1.0
    return lg


def golden_errors():
    g = json.load(open(GOLDEN))
    bad = []
    for case in g["cases"]:
        N, L, Lc = len(case["cand"]), case["seq_len"], case["L_cap"]
        k = (100.0 + np.arange(Lc, dtype=np.float64)).reshape(1, 1, Lc, 1)
        v = (200.0 + np.arange(Lc, dtype=np.float64)).reshape(1, 1, Lc, 1)
        ta = np.array([case["target_argmax"]], dtype=np.int32)
        r = OCm.verify_commit(_logits_for(ta, 100), np.array([case["cand"]]),
                              np.array([case["parents"]]), np.array([L]), [k], [v])
        got = (int(r["accept_len"][0]), int(r["last_node"][0]), int(r["bonus"][0]),
               list(r["path"][0]), int(r["seq_lens_out"][0]),
               list(r["k_out"][0][0, 0, :, 0]), list(r["v_out"][0][0, 0, :, 0]))
        want = (case["accept_len"], case["last_node"], case["bonus"], case["path"],
                case["seq_len_out"], case["k_out"], case["v_out"])
        if got != want:
            bad.append((case["name"], got))
    return bad


def _random_tree(rng, N):
    return np.array([-1] + [int(rng.integers(-1, n)) for n in range(1, N)], dtype=np.int32)


def _planted_case(rng, B, N, H, D, layers):
    """Random trees with one planted accepted node per sequence (or none)."""
    parents = np.stack([_random_tree(rng, N) for _ in range(B)])
    cand = rng.integers(0, 50, size=(B, N)).astype(np.int32)
    ta = rng.integers(50, 60, size=(B, N + 1)).astype(np.int32)  # matches nothing
    for b in range(B):
        if rng.random() < 0.15:
            continue
        target = int(rng.integers(0, N))
        m = target
        while m != -1:
            ta[b, parents[b, m] + 1] = cand[b, m]
            m = int(parents[b, m])
    lens = rng.integers(0, 6, size=B).astype(np.int32)
    L_cap = int(lens.max()) + N + 2
    ks = [rng.standard_normal((B, H, L_cap, D)) for _ in range(layers)]
    vs = [rng.standard_normal((B, H, L_cap, D)) for _ in range(layers)]
    return parents, cand, ta, lens, ks, vs


def attention_equivalence_errors(seed=11, trials=40):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        B, N, H, D = 2, int(rng.integers(1, 9)), 2, 4
        parents, cand, ta, lens, ks, vs = _planted_case(rng, B, N, H, D, 1)
        r = OCm.verify_commit(_logits_for(ta, 64), cand, parents, lens, ks, vs)
        for b in range(B):
            last = int(r["last_node"][b])
            if last < 0:
                continue
            L, a = int(lens[b]), int(r["accept_len"][b])
            for h in range(H):
                q = rng.standard_normal((N, D))
                tree = OA.tree_attention_head(q, ks[0][b, h], vs[0][b, h], L, parents[b],
                                              nodes=[last])[last]
                flat = OA.attention_rows(q[last:last + 1], r["k_out"][0][b, h, :L + a],
                                         r["v_out"][0][b, h, :L + a], 1.0 / np.sqrt(D))[0]
                if not np.allclose(tree, flat, atol=1e-12, rtol=0):
                    bad.append(("attention", b, h))
    return bad


def _paths_top_down(parents):
    kids = {n: [] for n in range(-1, len(parents))}
    for n, p in enumerate(parents):
        kids[int(p)].append(n)
    out = []

    def walk(node, path):
        for c in kids[node]:
            out.append(path + [c])
            walk(c, path + [c])
    walk(-1, [])
    return out


def bruteforce_errors(seed=12, trials=60):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        B, N = 3, int(rng.integers(1, 10))
        parents, cand, ta, lens, ks, vs = _planted_case(rng, B, N, 1, 2, 2)
        r = OCm.verify_commit(_logits_for(ta, 64), cand, parents, lens, ks, vs)
        for b in range(B):
            best = []
            for path in _paths_top_down(parents[b]):
                ok = all(cand[b, n] == ta[b, (path[i - 1] if i else -1) + 1]
                         for i, n in enumerate(path))
                if ok and (len(path) > len(best) or (len(path) == len(best) and path[-1] < best[-1])):
                    best = path
            want = best + [-1] * (N - len(best))
            if list(r["path"][b]) != want or int(r["seq_lens_out"][b]) != lens[b] + len(best):
                bad.append(("path", b, list(r["path"][b]), want))
    return bad


def untouched_errors(seed=13, trials=40):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        B, N = 3, int(rng.integers(1, 9))
        parents, cand, ta, lens, ks, vs = _planted_case(rng, B, N, 2, 3, 2)
        r = OCm.verify_commit(_logits_for(ta, 64), cand, parents, lens, ks, vs)
        for l in range(2):
            for b in range(B):
                L, a = int(lens[b]), int(r["accept_len"][b])
                keep = np.ones(ks[l].shape[2], dtype=bool)
                keep[L:L + a] = False
                for new, old in ((r["k_out"][l], ks[l]), (r["v_out"][l], vs[l])):
                    if not np.array_equal(new[b][:, keep], old[b][:, keep]):
                        bad.append(("untouched", l, b))
    # a chain accepted in full commits every row onto itself
    N, L = 6, 4
    parents = np.arange(-1, N - 1, dtype=np.int32)[None]
    cand = np.arange(1, N + 1, dtype=np.int32)[None]
    ta = np.concatenate([cand, [[42]]], axis=1).astype(np.int32)
    k = rng.standard_normal((1, 2, L + N, 3))
    v = rng.standard_normal((1, 2, L + N, 3))
    r = OCm.verify_commit(_logits_for(ta, 64), cand, parents, np.array([L]), [k], [v])
    if not (np.array_equal(r["k_out"][0], k) and np.array_equal(r["v_out"][0], v)
            and int(r["seq_lens_out"][0]) == L + N and int(r["bonus"][0]) == 42):
        bad.append(("chain",))
    return bad


PINS = [golden_errors, attention_equivalence_errors, bruteforce_errors, untouched_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


def test_cache_too_short_rejected():
    k = np.zeros((1, 1, 4, 1))
    with pytest.raises(ValueError):
        OCm.verify_commit(_logits_for(np.array([[0, 0, 0, 0]], dtype=np.int32), 4),
                          np.array([[0, 0, 0]]), np.array([[-1, 0, 1]]), np.array([2]), [k], [k])


# ---- planted mistakes ----

_REAL = OCm.verify_commit


def _rewrite(fn):
    """Runs the real oracle for the selection, then rebuilds the caches with
    ``fn(k_in, k_new, b, L, nodes)`` (both K and V)."""
    def mutant(logits, cand, parents, seq_lens, k_caches, v_caches):
        r = _REAL(logits, cand, parents, seq_lens, k_caches, v_caches)
        r["k_out"] = [np.array(k, copy=True) for k in k_caches]
        r["v_out"] = [np.array(v, copy=True) for v in v_caches]
        for b in range(len(seq_lens)):
            nodes = [int(n) for n in r["path"][b] if n >= 0]
            for src, dst in zip(list(k_caches) + list(v_caches), r["k_out"] + r["v_out"]):
                fn(np.asarray(src), dst, b, int(seq_lens[b]), nodes)
        return r
    return mutant


def _in_place_deepest_first(src, dst, b, L, nodes):
    for d in range(len(nodes) - 1, -1, -1):
        dst[b, :, L + d] = dst[b, :, L + nodes[d]]


def _off_by_one(src, dst, b, L, nodes):
    for d, n in enumerate(nodes):
        if L + d + 1 < dst.shape[2]:
            dst[b, :, L + d + 1] = src[b, :, L + n]


def _path_reversed(src, dst, b, L, nodes):
    for d, n in enumerate(nodes[::-1]):
        dst[b, :, L + d] = src[b, :, L + n]


def _length_is_depth_of_tree(logits, cand, parents, seq_lens, k_caches, v_caches):
    r = _REAL(logits, cand, parents, seq_lens, k_caches, v_caches)
    r["seq_lens_out"] = np.asarray(seq_lens, dtype=np.int32) + np.int32(np.asarray(cand).shape[1])
    return r


MUTANTS = [_rewrite(_in_place_deepest_first), _rewrite(_off_by_one), _rewrite(_path_reversed),
           _length_is_depth_of_tree]


@pytest.mark.parametrize("mutant", MUTANTS, ids=["in_place_deepest_first", "off_by_one",
                                                 "path_reversed", "length_is_node_count"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    monkeypatch.setattr(OCm, "verify_commit", mutant)
    failures = []
    for pin in PINS:
        failures += pin()
    assert failures

"""GPU parity of cape_expand, glide_argmax_rows and tree_verify: bit-exact
against the oracle on seeded inputs, boundary confidences, ties, tiny
vocabularies, budget cuts, fixed-size expansion and random trees."""

import json
import os

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import cape as OC
from oracle import verify as OV
from synth import workloads as W
from tests.gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu

f32 = np.float32
GOLDEN_CAPE = os.path.join(os.path.dirname(__file__), "golden", "cape_worked_example.json")


def gpu_cape(probs, k, n_max, fixed=False):
    dev = torch.device("cuda")
    B, gamma, V = probs.shape
    t = torch.empty((B, n_max), dtype=torch.int32, device=dev)
    p = torch.empty((B, n_max), dtype=torch.int32, device=dev)
    n = torch.empty((B,), dtype=torch.int32, device=dev)
    glide.cape_expand(torch.from_numpy(np.ascontiguousarray(probs)).to(dev), k, n_max, t, p, n,
                      fixed=fixed)
    torch.cuda.synchronize()
    return t.cpu().numpy(), p.cpu().numpy(), n.cpu().numpy()


def check_cape(probs, k, n_max, fixed=False):
    say("cape_expand", dict(shape=probs.shape, k=k, n_max=n_max, fixed=fixed))
    got = gpu_cape(probs, k, n_max, fixed)
    want = OC.cape_expand(probs, k, n_max, fixed)
    for g, w in zip(got, want):
        assert np.array_equal(g, w), (g, w)


def test_cape_golden():
    require_gpu()
    g = json.load(open(GOLDEN_CAPE))
    probs = np.asarray(g["probs"], dtype=np.float32)[None]
    for case in g["cases"]:
        t, p, n = gpu_cape(probs, case["k"], case["n_max"], bool(case["fixed"]))
        assert list(t[0]) == case["tokens"] and list(p[0]) == case["parents"]
        assert n[0] == case["n_nodes"]


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_cape_dirichlet_workloads(cfg):
    require_gpu()
    wl = W.WORKLOADS[cfg]
    probs, _, _ = W.draft_probs(wl, 100 + cfg, batch=min(wl.batch, 4))
    check_cape(probs, wl.k, wl.nodes)
    check_cape(probs, wl.k_config, wl.nodes)


def test_cape_boundary_confidences():
    require_gpu()
    up = lambda x: np.nextafter(f32(x), f32(2), dtype=np.float32)  # noqa: E731
    conf = [f32(0.05), f32(0.3), up(0.3), f32(0.6), up(0.6), f32(0.8), up(0.8), f32(1.0)]
    probs = W.peaked_probs(6, 8, 1000, 7, conf)
    for k, n_max in ((0, 64), (0, 20), (3, 30), (7, 8), (1, 12)):
        check_cape(probs, k, n_max)


@pytest.mark.parametrize("V", [2, 3, 5, 8, 9, 12, 13])
def test_cape_tiny_vocab_with_ties(V):
    require_gpu()
    rng = np.random.default_rng(V)
    probs = (rng.integers(0, 4, size=(5, 6, V)).astype(np.float32) / f32(4))
    probs[0, 0] = f32(0.25)          # a row of exact ties
    probs[1, 2, :] = f32(0.0)
    probs[1, 2, V - 1] = f32(-0.0)   # -0.0 ties with +0.0
    for k, n_max in ((0, 6 * 8), (0, 9), (2, 14), (7, 6)):
        check_cape(probs, k, n_max)


@pytest.mark.parametrize("k", range(0, 8))
def test_cape_fixed_size(k):
    require_gpu()
    probs, _, _ = W.draft_probs(W.WORKLOADS[2], 40 + k, batch=3, vocab=4099)
    check_cape(probs, k, 64, fixed=True)
    check_cape(probs, k, 12, fixed=True)


def test_cape_long_proposal():
    require_gpu()
    probs, _, _ = W.draft_probs(W.WORKLOADS[2], 55, batch=2, gamma=16, vocab=777)
    check_cape(probs, 0, 64)
    check_cape(probs, 0, 16)


def gpu_argmax(x):
    dev = torch.device("cuda")
    xt = torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    idx = torch.empty(x.shape[:-1], dtype=torch.int32, device=dev)
    glide.glide_argmax_rows(xt, idx)
    torch.cuda.synchronize()
    return idx.cpu().numpy()


@pytest.mark.parametrize("V", [1, 3, 4, 1000, 1001, 32000])
def test_argmax_rows(V):
    require_gpu()
    rng = np.random.default_rng(V)
    x = rng.integers(-3, 3, size=(37, V)).astype(np.float32)   # many ties
    x[0] = f32(-0.0)
    x[1, :] = f32(0.0)
    x[1, V // 2] = f32(-0.0)
    x[2] = -np.inf
    x[3] = rng.standard_normal(V).astype(np.float32)
    say("argmax", V)
    assert np.array_equal(gpu_argmax(x), OV.argmax_rows(x))


@pytest.mark.parametrize("V", [1001, 32000])
def test_argmax_many_rows(V):
    """More rows than two 1024-thread workgroups per CU hold (the 256-thread
    launch), ties and signed zeros included."""
    require_gpu()
    rng = np.random.default_rng(V + 7)
    x = rng.integers(-3, 3, size=(600, V)).astype(np.float32)
    x[5] = f32(-0.0)
    x[599, :] = -np.inf
    say("argmax many rows", V)
    assert np.array_equal(gpu_argmax(x), OV.argmax_rows(x))


def gpu_verify(ta, cand, parents):
    dev = torch.device("cuda")
    B, N = cand.shape
    outs = [torch.full((B,), 12345, dtype=torch.int32, device=dev) for _ in range(3)]
    glide.tree_verify(torch.from_numpy(ta.astype(np.int32)).to(dev),
                      torch.from_numpy(cand.astype(np.int32)).to(dev),
                      torch.from_numpy(parents.astype(np.int32)).to(dev), *outs)
    torch.cuda.synchronize()
    return tuple(o.cpu().numpy() for o in outs)


@pytest.mark.parametrize("N,depth,vocab", [(1, 1, 2), (5, 5, 3), (16, 5, 3), (32, 6, 2),
                                           (64, 8, 2), (64, 64, 2), (40, 3, 4)])
def test_tree_verify_random_trees(N, depth, vocab):
    require_gpu()
    B = 64
    parents = W.random_parents(B, N, depth, N * 7 + depth)
    cand = W.random_tokens(B, N, vocab, N)
    rng = np.random.default_rng(N)
    ta = rng.integers(0, vocab, size=(B, N + 1)).astype(np.int32)
    cand[0, :] = -1                      # all padding: nothing accepted
    say("tree_verify", N, depth, vocab)
    got = gpu_verify(ta, cand, parents)
    want = OV.tree_verify(ta, cand, parents)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)


def test_tree_verify_planted_cape():
    require_gpu()
    wl = W.WORKLOADS[3]
    probs, chain, leaf = W.draft_probs(wl, 9, vocab=5000)
    tokens, parents, _ = OC.cape_expand(probs, wl.k, wl.nodes)
    logits, depth, _ = W.planted_logits_cape(wl, 9, chain, leaf, probs)
    ta = gpu_argmax(logits)
    assert np.array_equal(ta, OV.argmax_rows(logits))
    acc, last, bonus = gpu_verify(ta, tokens, parents)
    assert np.array_equal(acc, depth)
    want = OV.tree_verify(ta, tokens, parents)
    assert np.array_equal(last, want[1]) and np.array_equal(bonus, want[2])

"""GPU parity of glide_verify_commit: the target argmax, the acceptance
outputs and the committed K/V caches, bit-exact against the oracle.  The
commit only moves rows, so the caches are compared as raw bits (the oracle
runs on the integer view of the same values)."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import cape as OC
from oracle import commit as OCm
from synth import workloads as W
from tests.gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu

SEED = 2  # the seed bench.py uses


def _bits(t):
    view = torch.int16 if t.dtype == torch.bfloat16 else torch.int32
    return t.contiguous().view(view).cpu().numpy()


def _random_tree(rng, N, chain_bias):
    par = [-1]
    for n in range(1, N):
        par.append(n - 1 if rng.random() < chain_bias else int(rng.integers(-1, n)))
    return par


def make_case(seed, B, N, V=97, chain_bias=0.5, none_frac=0.15, max_len=40):
    """Random trees with a planted accepted node per sequence (sometimes none)."""
    rng = np.random.default_rng(seed)
    parents = np.stack([_random_tree(rng, N, chain_bias) for _ in range(B)]).astype(np.int32)
    cand = rng.integers(0, V, size=(B, N)).astype(np.int32)
    logits = rng.standard_normal((B, N + 1, V)).astype(np.float32)
    for b in range(B):
        if rng.random() < none_frac:
            continue
        m = int(rng.integers(0, N))
        while m != -1:
            row = parents[b, m] + 1
            logits[b, row, cand[b, m]] = logits[b, row].max() + 1.0
            m = int(parents[b, m])
    lens = rng.integers(0, max_len + 1, size=B).astype(np.int32)
    return logits, cand, parents, lens


def run_and_check(logits, cand, parents, lens, k_caches, v_caches, label):
    dev = torch.device("cuda")
    B, N = cand.shape
    say("verify_commit", label, dict(B=B, N=N, layers=len(k_caches)))
    k_in = [_bits(k) for k in k_caches]
    v_in = [_bits(v) for v in v_caches]
    outs = {name: torch.full(shape, -7, dtype=torch.int32, device=dev)
            for name, shape in (("ta", (B, N + 1)), ("acc", (B,)), ("last", (B,)),
                                ("bonus", (B,)), ("path", (B, N)), ("lens_out", (B,)))}
    glide.glide_verify_commit(torch.from_numpy(logits).to(dev), torch.from_numpy(cand).to(dev),
                              torch.from_numpy(parents).to(dev), k_caches, v_caches,
                              torch.from_numpy(lens).to(dev), outs["lens_out"], outs["ta"],
                              outs["acc"], outs["last"], outs["bonus"], outs["path"])
    torch.cuda.synchronize()
    want = OCm.verify_commit(logits, cand, parents, lens, k_in, v_in)
    for name, key in (("ta", "target_argmax"), ("acc", "accept_len"), ("last", "last_node"),
                      ("bonus", "bonus"), ("path", "path"), ("lens_out", "seq_lens_out")):
        assert np.array_equal(outs[name].cpu().numpy(), want[key]), (label, name)
    for l in range(len(k_caches)):
        assert np.array_equal(_bits(k_caches[l]), want["k_out"][l]), (label, "k", l)
        assert np.array_equal(_bits(v_caches[l]), want["v_out"][l]), (label, "v", l)
    return want


def _caches(seed, B, H, L_cap, layers, dtype):
    g = torch.Generator().manual_seed(seed)
    mk = lambda: torch.randn((B, H, L_cap, 128), generator=g).to(dtype).cuda()  # noqa: E731
    return [mk() for _ in range(layers)], [mk() for _ in range(layers)]


CASES = [
    # (seed, B, N, H, layers, dtype, chain_bias)
    (1, 1, 16, 32, 2, torch.bfloat16, 0.5),
    (2, 3, 5, 3, 1, torch.float32, 0.5),
    (3, 4, 64, 5, 3, torch.bfloat16, 0.9),
    (4, 2, 64, 2, 2, torch.float32, 0.97),
    (5, 5, 1, 1, 1, torch.bfloat16, 0.5),
    (6, 16, 64, 32, 1, torch.bfloat16, 0.8),
    (7, 3, 33, 6, 2, torch.float32, 0.3),
    (8, 2, 17, 4, 0, torch.bfloat16, 0.5),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d_B%d_N%d_H%d_L%d_%s" % (
    c[0], c[1], c[2], c[3], c[4], str(c[5]).split(".")[-1]))
def test_random_trees(case):
    require_gpu()
    seed, B, N, H, layers, dtype, bias = case
    logits, cand, parents, lens = make_case(seed, B, N, chain_bias=bias)
    L_cap = int(lens.max()) + N + 3
    ks, vs = _caches(seed, B, H, L_cap, layers, dtype)
    run_and_check(logits, cand, parents, lens, ks, vs, "random")


def test_deep_paths_move_every_row():
    """Second root accepted and followed to the bottom of a 64-deep chain:
    every committed row comes from one row further down (fp32 takes two
    copy batches)."""
    require_gpu()
    N, B = 64, 2
    parents = np.array([[-1, -1] + list(range(1, N - 1))] * B, dtype=np.int32)
    cand = np.arange(1, N + 1, dtype=np.int32)[None].repeat(B, 0)
    logits = np.zeros((B, N + 1, 128), dtype=np.float32)
    logits[:, 0, 2] = 1.0                      # root slot: node 1's token
    for n in range(1, N - 1):
        logits[:, n + 1, n + 2] = 1.0          # node n's child n + 1
    logits[:, N, 7] = 1.0                      # bonus after the last node
    lens = np.array([0, 5], dtype=np.int32)
    for dtype in (torch.bfloat16, torch.float32):
        ks, vs = _caches(9, B, 3, 5 + N, 2, dtype)
        want = run_and_check(logits, cand, parents, lens, ks, vs, "deep %s" % dtype)
        assert list(want["accept_len"]) == [N - 1, N - 1]


def test_nothing_accepted_changes_nothing():
    require_gpu()
    logits, cand, parents, lens = make_case(10, 3, 8, none_frac=1.0)
    logits[:, 0, :] = 0.0
    logits[:, 0, 96] = 5.0                     # no root holds token 96 after this
    cand[cand == 96] = 0
    ks, vs = _caches(10, 3, 2, int(lens.max()) + 8, 1, torch.bfloat16)
    want = run_and_check(logits, cand, parents, lens, ks, vs, "none")
    assert list(want["accept_len"]) == [0, 0, 0]


def test_seq_lens_validation(monkeypatch):
    require_gpu()
    monkeypatch.setenv("GLIDE_VALIDATE", "1")
    dev = torch.device("cuda")
    logits, cand, parents, _ = make_case(11, 1, 4)
    ks, vs = _caches(11, 1, 1, 10, 1, torch.bfloat16)
    lens = torch.tensor([7], dtype=torch.int32, device=dev)   # 7 + 4 > 10
    out = [torch.empty(s, dtype=torch.int32, device=dev) for s in ((1,), (1, 5), (1,))]
    with pytest.raises(glide.GlideError) as e:
        glide.glide_verify_commit(torch.from_numpy(logits).to(dev), torch.from_numpy(cand).to(dev),
                                  torch.from_numpy(parents).to(dev), ks, vs, lens, out[0], out[1],
                                  out[2])
    assert e.value.status == glide.GLIDE_ERANGE


def test_out_of_range_lengths_are_clamped():
    """Without GLIDE_VALIDATE, lengths past L_cap - N (and negative ones) are
    clamped into [0, L_cap - N]; the rows move at the clamped length and the
    committed length is that clamped length plus the accepted count.  The
    expected values are the oracle's at the clamped lengths."""
    require_gpu()
    B, N = 3, 8
    logits, cand, parents, _ = make_case(12, B, N, none_frac=0.0)
    L_cap = 20
    raw = np.array([L_cap + 5, -4, L_cap - N + 1], dtype=np.int32)
    clamped = np.clip(raw, 0, L_cap - N).astype(np.int32)
    for dtype in (torch.bfloat16, torch.float32):
        ks, vs = _caches(12, B, 2, L_cap, 2, dtype)
        k_in = [_bits(k) for k in ks]
        v_in = [_bits(v) for v in vs]
        dev = torch.device("cuda")
        lens_out = torch.full((B,), -7, dtype=torch.int32, device=dev)
        acc = torch.empty((B,), dtype=torch.int32, device=dev)
        ta = torch.empty((B, N + 1), dtype=torch.int32, device=dev)
        say("verify_commit", "clamped lengths", dtype, raw.tolist())
        glide.glide_verify_commit(torch.from_numpy(logits).to(dev), torch.from_numpy(cand).to(dev),
                                  torch.from_numpy(parents).to(dev), ks, vs,
                                  torch.from_numpy(raw).to(dev), lens_out, ta, acc)
        torch.cuda.synchronize()
        want = OCm.verify_commit(logits, cand, parents, clamped, k_in, v_in)
        assert want["accept_len"].max() > 0
        assert np.array_equal(acc.cpu().numpy(), want["accept_len"])
        assert np.array_equal(lens_out.cpu().numpy(), want["seq_lens_out"])
        for l in range(len(ks)):
            assert np.array_equal(_bits(ks[l]), want["k_out"][l]), ("k", l)
            assert np.array_equal(_bits(vs[l]), want["v_out"][l]), ("v", l)


@pytest.mark.parametrize("cfg,layers", [(2, None), (3, [0, 39]), (4, [59])])
def test_workload(cfg, layers):
    """A workload's CaPE tree (built on the GPU), its planted logits and its
    caches: every layer for the 7B shape, sampled layers for the larger ones
    (the kernel does the same for every layer)."""
    require_gpu()
    wl = W.WORKLOADS[cfg]
    dev = torch.device("cuda")
    probs, chain, leaf = W.draft_probs(wl, SEED)
    logits, depth, _ = W.planted_logits_cape(wl, SEED, chain, leaf, probs)
    t = torch.empty((wl.batch, wl.nodes), dtype=torch.int32, device=dev)
    p = torch.empty_like(t)
    n = torch.empty((wl.batch,), dtype=torch.int32, device=dev)
    glide.cape_expand(torch.from_numpy(probs).to(dev), wl.k, wl.nodes, t, p, n)
    torch.cuda.synchronize()
    ot, op, _ = OC.cape_expand(probs, wl.k, wl.nodes)
    assert np.array_equal(t.cpu().numpy(), ot) and np.array_equal(p.cpu().numpy(), op)
    lens = W.prefix_lengths(wl, SEED)
    ks, vs = [], []
    for layer in (range(wl.layers) if layers is None else layers):
        _, k, v = W.attention_layer(wl, SEED, layer, torch.bfloat16, dev)
        ks.append(k)
        vs.append(v)
    want = run_and_check(logits, ot, op, lens, ks, vs, wl.name)
    assert np.array_equal(want["accept_len"], depth)

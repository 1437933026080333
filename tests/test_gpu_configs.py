"""GPU parity at the full sizes of the five workloads, in the launch
configuration bench.py uses (automatic split plan, bf16).

For every workload:
* CaPE expansion of the full draft rows (V = 32000) -- bit-exact against the
  oracle, for the tree the attention uses and for the workload's stated top-k;
* argmax over the planted target logits and greedy verification -- bit-exact,
  and the planted accept length is recovered;
* verification attention of the first and last layer with the tree the GPU
  built, and (where the workload has one) the GliDe cross-attention on the
  last layer's cache -- every sequence, heads {0, H/2, H-1} and sampled nodes
  (every chain node and a middle node of every depth) against the float64
  oracle, max-abs error <= 1e-2.
"""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import attention as OA
from oracle import cape as OC
from oracle import verify as OV
from synth import workloads as W
from tests.gpu_common import BF16_TOL, F32_TOL, require_gpu, say, to64

pytestmark = pytest.mark.gpu

SEED = 2  # the seed bench.py uses


def _gpu_tree(wl, probs, k):
    dev = torch.device("cuda")
    B = probs.shape[0]
    t = torch.empty((B, wl.nodes), dtype=torch.int32, device=dev)
    p = torch.empty_like(t)
    n = torch.empty((B,), dtype=torch.int32, device=dev)
    glide.cape_expand(torch.from_numpy(probs).to(dev), k, wl.nodes, t, p, n)
    torch.cuda.synchronize()
    return t, p, n


def _sample_nodes(parents_b, N, depth):
    """Nodes compared against the oracle: every chain node, a middle node of
    every depth (the middle leaf of that depth's expansion set when it has
    one), the middle and the last node."""
    d = np.zeros(N, dtype=np.int64)
    for n in range(N):
        p = int(parents_b[n])
        d[n] = 1 + (d[p] if p >= 0 else 0)
    pick = set(range(min(depth, N))) | {N // 2, N - 1}
    for level in range(1, int(d.max()) + 1):
        at = [n for n in range(N) if d[n] == level and n >= depth]
        if at:
            pick.add(at[len(at) // 2])
    return sorted(pick)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_integer_path(cfg):
    require_gpu()
    wl = W.WORKLOADS[cfg]
    dev = torch.device("cuda")
    say("integer path", wl.name)
    if wl.tree == "cape":
        probs, chain, leaf = W.draft_probs(wl, SEED)
        for k in sorted({wl.k, wl.k_config}):
            t, p, n = _gpu_tree(wl, probs, k)
            ot, op, on = OC.cape_expand(probs, k, wl.nodes)
            assert np.array_equal(t.cpu().numpy(), ot)
            assert np.array_equal(p.cpu().numpy(), op)
            assert np.array_equal(n.cpu().numpy(), on)
        ot, op, _ = OC.cape_expand(probs, wl.k, wl.nodes)
        logits, depth, _ = W.planted_logits_cape(wl, SEED, chain, leaf, probs)
    else:
        ot = W.chain_tokens(wl, SEED)
        op = np.tile(np.arange(-1, wl.nodes - 1, dtype=np.int32), (wl.batch, 1))
        logits, depth = W.planted_logits_chain(wl, SEED, ot)
    B, N = ot.shape
    ta = torch.empty((B, N + 1), dtype=torch.int32, device=dev)
    glide.glide_argmax_rows(torch.from_numpy(logits).to(dev), ta)
    outs = [torch.empty((B,), dtype=torch.int32, device=dev) for _ in range(3)]
    glide.tree_verify(ta, torch.from_numpy(ot).to(dev), torch.from_numpy(op).to(dev), *outs)
    torch.cuda.synchronize()
    o_ta = OV.argmax_rows(logits)
    assert np.array_equal(ta.cpu().numpy(), o_ta)
    want = OV.tree_verify(o_ta, ot, op)
    for g, w in zip(outs, want):
        assert np.array_equal(g.cpu().numpy(), w)
    assert np.array_equal(want[0], depth)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_attention(cfg):
    require_gpu()
    wl = W.WORKLOADS[cfg]
    dev = torch.device("cuda")
    lens_np = W.prefix_lengths(wl, SEED)
    lens = torch.from_numpy(lens_np).to(dev)
    if wl.tree == "cape":
        probs, _, _ = W.draft_probs(wl, SEED)
        _, par_gpu, _ = _gpu_tree(wl, probs, wl.k)
        _, par_or, _ = OC.cape_expand(probs, wl.k, wl.nodes)
        assert np.array_equal(par_gpu.cpu().numpy(), par_or)
    else:
        par_or = np.tile(np.arange(-1, wl.nodes - 1, dtype=np.int32), (wl.batch, 1))
        par_gpu = torch.from_numpy(par_or).to(dev)
    seqs = range(wl.batch)
    heads = sorted({0, wl.heads // 2, wl.heads - 1})
    for layer in sorted({0, wl.layers - 1}):
        say("attention", wl.name, "layer", layer)
        q, k, v = W.attention_layer(wl, SEED, layer, torch.bfloat16, dev)
        out = torch.full_like(q, float("nan"))
        glide.glide_tree_attn(q, k, v, lens, par_gpu, out)
        torch.cuda.synchronize()
        for b in seqs:
            nodes = _sample_nodes(par_or[b], wl.nodes, wl.depth)
            for h in heads:
                L = int(lens_np[b])
                rows = L + wl.nodes
                ref = OA.tree_attention_head(to64(q[b, :, h]), to64(k[b, h, :rows]),
                                             to64(v[b, h, :rows]), L, par_or[b], nodes=nodes)
                got = to64(out[b, :, h])
                err = float(np.abs(got[nodes] - ref[nodes]).max())
                assert err <= BF16_TOL, (layer, b, h, err)
        if wl.cross and layer == wl.layers - 1:
            say("cross attention", wl.name)
            xq = W.cross_queries(wl, SEED, torch.bfloat16, dev)
            xo = torch.full_like(xq, float("nan"))
            glide.glide_tree_attn(xq, k, v, lens, None, xo)
            torch.cuda.synchronize()
            for b in seqs:
                for h in heads:
                    L = int(lens_np[b])
                    ref = OA.tree_attention_head(to64(xq[b, :, h]), to64(k[b, h, :L]),
                                                 to64(v[b, h, :L]), L, None)
                    err = float(np.abs(to64(xo[b, :, h]) - ref).max())
                    assert err <= BF16_TOL, ("cross", b, h, err)
        del q, k, v, out
        torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_attention_f32(cfg):
    """The float32 mode on the same values (the workload's bf16 draws widened
    exactly), first layer, automatic split plan: sampled outputs against the
    float64 oracle within 1e-5."""
    require_gpu()
    wl = W.WORKLOADS[cfg]
    dev = torch.device("cuda")
    lens_np = W.prefix_lengths(wl, SEED)
    lens = torch.from_numpy(lens_np).to(dev)
    if wl.tree == "cape":
        probs, _, _ = W.draft_probs(wl, SEED)
        _, par_gpu, _ = _gpu_tree(wl, probs, wl.k)
        _, par_or, _ = OC.cape_expand(probs, wl.k, wl.nodes)
        assert np.array_equal(par_gpu.cpu().numpy(), par_or)
    else:
        par_or = np.tile(np.arange(-1, wl.nodes - 1, dtype=np.int32), (wl.batch, 1))
        par_gpu = torch.from_numpy(par_or).to(dev)
    say("attention f32", wl.name)
    q, k, v = (t.float() for t in W.attention_layer(wl, SEED, 0, torch.bfloat16, dev))
    out = torch.full_like(q, float("nan"))
    glide.glide_tree_attn(q, k, v, lens, par_gpu, out)
    torch.cuda.synchronize()
    for b in range(wl.batch):
        nodes = _sample_nodes(par_or[b], wl.nodes, wl.depth)
        for h in sorted({0, wl.heads // 2, wl.heads - 1}):
            L = int(lens_np[b])
            rows = L + wl.nodes
            ref = OA.tree_attention_head(to64(q[b, :, h]), to64(k[b, h, :rows]), to64(v[b, h, :rows]),
                                         L, par_or[b], nodes=nodes)
            err = float(np.abs(to64(out[b, :, h])[nodes] - ref[nodes]).max())
            assert err <= F32_TOL, (b, h, err)

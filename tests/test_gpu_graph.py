"""Graph capture: the hot-path calls recorded into one HIP graph (through
torch.cuda.CUDAGraph) and replayed several times, with eager work and
synchronisations between the replays.  Every replay must reproduce the eager
results bit for bit: the library records no memsets and allocates nothing
inside the calls, and every workspace is written before it is read.

Covered: CaPE expansion, tree attention on the GPU-built tree (split plan
with the merge kernel, 16 rows) and on a 32-row random tree (shared-step
kernel), cross attention, argmax and greedy verification, the verification
epilogue with its cache commit (on a copy of the caches made inside the
graph, so every replay starts from the same state), speculative sampling,
the packed cross-attention block and the block-masked attention."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from synth import workloads as W
from tests.gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu


def _inputs():
    dev = torch.device("cuda")
    wl = W.WORKLOADS[2]
    B, H, L, N, V, gamma = 2, 4, 300, wl.nodes, 2000, wl.depth
    probs, chain, leaf = W.draft_probs(wl, 5, vocab=V, batch=B)
    logits, _, _ = W.planted_logits_cape(wl, 5, chain, leaf, probs)
    q, k, v = W.attention_layer(wl, 5, 0, torch.bfloat16, dev, batch=B, heads=H, l_cap=L + 32)
    g = torch.Generator(device=dev)
    g.manual_seed(9)
    rnd = lambda *shape, s=1.0: (torch.randn(shape, generator=g, device=dev) * s).to(torch.bfloat16)  # noqa: E731
    rng = np.random.default_rng(9)
    par32 = np.array([[rng.integers(-1, n) if n else -1 for n in range(32)] for _ in range(B)], dtype=np.int32)
    d_D = H * 128
    st = dict(
        probs=torch.from_numpy(probs).to(dev), logits=torch.from_numpy(logits).to(dev),
        q=q[:, :N].contiguous(), q32=rnd(B, 32, H, 128), xq=q[:, :gamma].contiguous(), kc=k, vc=v,
        lens=torch.tensor([L, L - 37], dtype=torch.int32, device=dev),
        par32=torch.from_numpy(par32).to(dev),
        tok=torch.empty((B, N), dtype=torch.int32, device=dev),
        par=torch.empty((B, N), dtype=torch.int32, device=dev),
        nn=torch.empty((B,), dtype=torch.int32, device=dev),
        ta=torch.empty((B, N + 1), dtype=torch.int32, device=dev),
        acc=torch.empty((B,), dtype=torch.int32, device=dev),
        kc2=torch.empty_like(k), vc2=torch.empty_like(v),
        lens_out=torch.empty((B,), dtype=torch.int32, device=dev),
        ta2=torch.empty((B, N + 1), dtype=torch.int32, device=dev),
        acc2=torch.empty((B,), dtype=torch.int32, device=dev),
        path=torch.empty((B, N), dtype=torch.int32, device=dev),
        sd_tok=torch.from_numpy(rng.integers(0, V, (B, gamma)).astype(np.int32)).to(dev),
        sd_pd=torch.from_numpy(rng.dirichlet(np.full(V, 0.3), (B, gamma)).astype(np.float32)).to(dev),
        sd_pt=torch.from_numpy(rng.dirichlet(np.full(V, 0.3), (B, gamma + 1)).astype(np.float32)).to(dev),
        sd_u=torch.from_numpy(rng.random((B, gamma + 1)).astype(np.float32)).to(dev),
        sd_acc=torch.empty((B,), dtype=torch.int32, device=dev),
        sd_next=torch.empty((B,), dtype=torch.int32, device=dev),
        hidden=rnd(B, gamma, d_D), wq=rnd(d_D, d_D, s=d_D ** -0.5), wo=rnd(d_D, d_D, s=d_D ** -0.5),
        bq=rnd(1, 260, H, 128), bk=rnd(1, H, 260, 128), bv=rnd(1, H, 260, 128),
    )
    st["wq_p"] = glide.pack_rows_weights(st["wq"])
    st["wo_p"] = glide.pack_rows_weights(st["wo"])
    for name, like in (("out", st["q"]), ("out32", st["q32"]), ("xout", st["xq"]),
                       ("xb_out", st["hidden"]), ("b_out", st["bq"])):
        st[name] = torch.empty_like(like)
    return st


OUTPUTS = ["tok", "par", "nn", "out", "out32", "xout", "ta", "acc", "kc2", "vc2", "lens_out", "ta2",
           "acc2", "path", "sd_acc", "sd_next", "xb_out", "b_out"]


def _calls(st):
    glide.cape_expand(st["probs"], 7, st["tok"].shape[1], st["tok"], st["par"], st["nn"])
    glide.glide_tree_attn(st["q"], st["kc"], st["vc"], st["lens"], st["par"], st["out"])
    glide.glide_tree_attn(st["q32"], st["kc"], st["vc"], st["lens"], st["par32"], st["out32"])
    glide.glide_tree_attn(st["xq"], st["kc"], st["vc"], st["lens"], None, st["xout"])
    glide.glide_argmax_rows(st["logits"], st["ta"])
    glide.tree_verify(st["ta"], st["tok"], st["par"], st["acc"])
    st["kc2"].copy_(st["kc"])
    st["vc2"].copy_(st["vc"])
    glide.glide_verify_commit(st["logits"], st["tok"], st["par"], [st["kc2"]], [st["vc2"]], st["lens"],
                              st["lens_out"], st["ta2"], st["acc2"], path=st["path"])
    glide.spec_sample_verify(st["sd_tok"], st["sd_pd"], st["sd_pt"], st["sd_u"], st["sd_acc"], st["sd_next"])
    glide.glide_cross_block_packed(st["hidden"], st["wq_p"], st["kc"], st["vc"], st["lens"], st["wo_p"],
                                   st["xb_out"])
    glide.glide_block_attn(st["bq"], st["bk"], st["bv"], st["b_out"], 5)


def _snapshot(st):
    return {k: st[k].clone() for k in OUTPUTS}


def _scribble(st):
    for k in OUTPUTS:
        if st[k].dtype == torch.int32:
            st[k].fill_(-5)
        else:
            st[k].fill_(float("nan"))


def test_graph_replays_match_eager():
    require_gpu()
    say("graph capture of the hot-path calls")
    st = _inputs()
    _calls(st)                       # eager reference (and workspace set-up)
    torch.cuda.synchronize()
    want = _snapshot(st)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):    # warm the capture stream's workspaces
        _calls(st)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _calls(st)
    torch.cuda.synchronize()
    for rep in range(3):
        _scribble(st)                # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in OUTPUTS:
            a, b = st[k], want[k]
            same = torch.equal(a.view(torch.int16), b.view(torch.int16)) if a.dtype == torch.bfloat16 \
                else torch.equal(a, b)
            assert same, (rep, k)
    del graph


def test_two_streams_own_workspaces():
    """Split-plan attention and the cross block issued on two streams at once:
    the binding keeps one workspace per (device, stream), so the calls do not
    share partial states and each matches its single-stream result."""
    require_gpu()
    say("two streams")
    st = _inputs()
    other = _inputs()
    other["q"] = other["q"].flip(0).contiguous()        # different queries on the second stream
    other["hidden"] = (other["hidden"] * 0.5).contiguous()
    work = lambda d: (glide.glide_tree_attn(d["q"], d["kc"], d["vc"], d["lens"], d["par32"][:, :16].contiguous(),  # noqa: E731
                                             d["out"]),
                      glide.glide_cross_block_packed(d["hidden"], d["wq_p"], d["kc"], d["vc"], d["lens"],
                                                     d["wo_p"], d["xb_out"]))
    work(st)
    work(other)
    torch.cuda.synchronize()
    want = (st["out"].clone(), st["xb_out"].clone(), other["out"].clone(), other["xb_out"].clone())
    for d in (st, other):
        d["out"].fill_(float("nan"))
        d["xb_out"].fill_(float("nan"))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        with torch.cuda.stream(s1):
            work(st)
        with torch.cuda.stream(s2):
            work(other)
    torch.cuda.synchronize()
    got = (st["out"], st["xb_out"], other["out"], other["xb_out"])
    for a, b in zip(got, want):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_explicit_stream_argument():
    """Calls given stream= a stream that is not the current one: the binding
    allocates their temporary workspaces (CaPE's, the cross block's, the
    attention's cached one and the packed weights) on that stream, so memory
    the current stream then allocates and scribbles on is never one of them
    while the calls run.  Results match the calls made on the current stream."""
    require_gpu()
    say("explicit stream argument")
    st = _inputs()
    _calls(st)
    torch.cuda.synchronize()
    want = {k: st[k].clone() for k in ("tok", "par", "nn", "out", "xb_out")}
    for k in want:
        st[k].fill_(-5 if st[k].dtype == torch.int32 else float("nan"))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        glide.cape_expand(st["probs"], 7, st["tok"].shape[1], st["tok"], st["par"], st["nn"], stream=s)
        glide.glide_tree_attn(st["q"], st["kc"], st["vc"], st["lens"], st["par"], st["out"], stream=s)
        wq_p = glide.pack_rows_weights(st["wq"], stream=s)
        glide.glide_cross_block_packed(st["hidden"], wq_p, st["kc"], st["vc"], st["lens"], st["wo_p"],
                                       st["xb_out"], stream=s)
        del wq_p
        # the current stream allocates and overwrites freed memory meanwhile
        junk = [torch.full((1 << 20,), float("nan"), device="cuda") for _ in range(8)]
        del junk
    torch.cuda.synchronize()
    for k, w in want.items():
        a = st[k]
        same = torch.equal(a.view(torch.int16), w.view(torch.int16)) if a.dtype == torch.bfloat16 \
            else torch.equal(a, w)
        assert same, k

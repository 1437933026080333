"""GPU parity of glide_tree_attn against the float64 oracle.

Shapes span several 32-key steps and 128-key split chunks with ragged tails,
every query-tile count (N = 1 .. 64), empty prefixes, cross mode, forced split
counts and both element types.  Tolerances: max-abs 1e-2 (bf16 inputs, fp32
accumulation) and 1e-5 (fp32 mode).
"""

import os

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import attention as OA
from synth import workloads as W
from tests.gpu_common import BF16_TOL, F32_TOL, cpu_normal, require_gpu, say, to64

pytestmark = pytest.mark.gpu

D = 128


def _parents(kind, B, N, seed):
    if kind is None:
        return None
    if kind == "chain":
        return np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1))
    if kind == "roots":
        return np.full((B, N), -1, dtype=np.int32)
    if kind == "random":
        return W.random_parents(B, N, 8, seed)
    if kind == "cape":  # proposal chain of depth min(N, 8) then leaves on every position
        g = min(N, 8)
        p = [i - 1 for i in range(g)] + [((j - g) % g) - 1 for j in range(g, N)]
        return np.tile(np.asarray(p, dtype=np.int32), (B, 1))
    raise ValueError(kind)


def run_case(B, N, H, lens, kind, dtype, splits, seed, l_cap=None):
    require_gpu()
    say("tree_attn", dict(B=B, N=N, H=H, lens=list(lens), kind=kind, dtype=str(dtype),
                          splits=splits, seed=seed))
    tree = kind is not None
    L_cap = l_cap or (max(lens) + (N if tree else 0))
    q = cpu_normal((B, N, H, D), seed, dtype)
    k = cpu_normal((B, H, L_cap, D), seed + 1, dtype)
    v = cpu_normal((B, H, L_cap, D), seed + 2, dtype)
    parents = _parents(kind, B, N, seed)
    dev = torch.device("cuda")
    out = torch.full((B, N, H, D), float("nan"), dtype=dtype, device=dev)
    glide.glide_tree_attn(q.to(dev), k.to(dev), v.to(dev),
                          torch.tensor(lens, dtype=torch.int32, device=dev),
                          None if parents is None else torch.from_numpy(parents).to(dev),
                          out, max_splits=splits)
    torch.cuda.synchronize()
    ref = OA.tree_attention(to64(q), to64(k), to64(v), lens, parents)
    got = to64(out)
    assert np.isfinite(got).all()
    return got, ref


CASES = [
    # B, N, H, lens, kind, splits
    (1, 5, 4, [512], "chain", 0),
    (1, 5, 4, [512], "chain", 1),
    (1, 16, 4, [2048], "cape", 0),
    (1, 16, 2, [2048], "cape", 9),
    (2, 17, 2, [33, 300], "random", 0),
    (3, 32, 2, [0, 1, 129], "random", 2),
    (2, 31, 2, [255, 256], "cape", 3),
    (2, 33, 2, [257, 1000], "random", 7),
    (1, 48, 2, [500], "random", 0),
    (2, 63, 2, [127, 128], "random", 64),
    (2, 64, 2, [4096, 1500], "cape", 0),
    (1, 64, 2, [4096], "roots", 0),
    (1, 1, 3, [1], "chain", 0),
    (1, 1, 3, [777], "roots", 5),
    (2, 5, 3, [1, 2048], None, 0),      # cross mode
    (2, 5, 3, [31, 129], None, 2),
    (1, 64, 2, [3000], None, 0),
    (3, 8, 2, [0, 33, 64], None, 1),    # empty key set for b = 0
    # one split per sequence: workgroup rows take the sequences longest first
    # (B <= 64, ties among equal lengths) or in order (B > 64)
    (64, 16, 1, [(37 * i) % 300 for i in range(64)], "cape", 1),
    (5, 32, 2, [90, 300, 90, 0, 300], "random", 1),
    (70, 5, 1, [(53 * i) % 200 for i in range(70)], None, 1),
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "B%dN%dH%d-%s-%s-s%d" % (
    c[0], c[1], c[2], "_".join(map(str, c[3])), c[4], c[5]))
def test_parity(case, dtype):
    B, N, H, lens, kind, splits = case
    got, ref = run_case(B, N, H, lens, kind, dtype, splits, seed=17 + N)
    tol = BF16_TOL if dtype == torch.bfloat16 else F32_TOL
    err = float(np.abs(got - ref).max())
    assert err <= tol, err


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_single_visible_key_is_exact(dtype):
    """Empty prefix, every node a root: each row sees only its own value row,
    so the output is that row exactly (weight 1)."""
    got, ref = run_case(2, 40, 3, [0, 0], "roots", dtype, 0, seed=5, l_cap=40)
    assert np.array_equal(got, ref)


def test_empty_cross_key_set_is_zero():
    got, _ = run_case(2, 5, 2, [0, 0], None, torch.bfloat16, 0, seed=6, l_cap=64)
    assert not got.any()


def test_ragged_l_cap_slack():
    """L_cap well above the longest prefix: the unused rows are never read."""
    require_gpu()
    got, ref = run_case(2, 20, 2, [100, 333], "random", torch.bfloat16, 0, seed=7, l_cap=4096)
    assert float(np.abs(got - ref).max()) <= BF16_TOL


def test_deterministic_and_split_invariant():
    require_gpu()
    dev = torch.device("cuda")
    B, N, H, L = 2, 32, 4, 3000
    q = cpu_normal((B, N, H, D), 1, torch.bfloat16).to(dev)
    k = cpu_normal((B, H, L + N, D), 2, torch.bfloat16).to(dev)
    v = cpu_normal((B, H, L + N, D), 3, torch.bfloat16).to(dev)
    lens = torch.tensor([L, L - 777], dtype=torch.int32, device=dev)
    par = torch.from_numpy(W.random_parents(B, N, 6, 4)).to(dev)
    outs = {}
    for splits in (1, 2, 5, 16, 64, 0, 0):
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=dev)
        glide.glide_tree_attn(q, k, v, lens, par, o, max_splits=splits)
        outs.setdefault(splits, []).append(o)
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[0][1])
    base = outs[1][0].float()
    for s, os_ in outs.items():
        assert float((os_[0].float() - base).abs().max()) <= BF16_TOL


def test_workspace_reused_across_shapes():
    """One workspace serves calls of different shapes in turn: each call
    writes the partial states it reads (stale ones are garbage on purpose)
    and leaves the arrival-counter block zero."""
    require_gpu()
    dev = torch.device("cuda")
    big = glide.attn_workspace(4, 64, 8, 4160, 0, dev)
    ws = torch.full((big.numel(),), 0xFF, dtype=torch.uint8, device=dev)  # stale partial states
    cnt = ws[:glide.ATTN_COUNTER_BYTES]
    cnt.zero_()  # the counter block starts zero (include/glide.h)
    shapes = [(4, 64, 8, 4096, 0), (1, 16, 2, 2048, 9), (2, 5, 3, 1000, 3), (4, 64, 8, 4096, 0),
              (1, 16, 2, 2048, 64)]
    for i, (B, N, H, L, splits) in enumerate(shapes):
        say("ws reuse", B, N, H, L, splits)
        q = cpu_normal((B, N, H, D), 40 + i, torch.bfloat16)
        k = cpu_normal((B, H, L + N, D), 50 + i, torch.bfloat16)
        v = cpu_normal((B, H, L + N, D), 60 + i, torch.bfloat16)
        par = W.random_parents(B, N, 6, i)
        out = torch.full((B, N, H, D), float("nan"), dtype=torch.bfloat16, device=dev)
        lens = [L - 37 * b for b in range(B)]
        glide.glide_tree_attn(q.to(dev), k.to(dev), v.to(dev),
                              torch.tensor(lens, dtype=torch.int32, device=dev),
                              torch.from_numpy(par).to(dev), out, max_splits=splits, workspace=ws)
        torch.cuda.synchronize()
        assert int(cnt.count_nonzero()) == 0
        got = to64(out)
        # sample two heads per shape against the oracle
        for b in range(B):
            for h in (0, H - 1):
                ref = OA.tree_attention_head(to64(q[b, :, h]), to64(k[b, h]), to64(v[b, h]),
                                             lens[b], par[b])
                assert float(np.abs(got[b, :, h] - ref).max()) <= BF16_TOL


@pytest.mark.parametrize("tree", [True, False], ids=["tree", "cross"])
def test_many_pairs_merge_in_second_launch(tree):
    """Many sequences (and more (sequence, head) pairs than arrival counters,
    B * H > 2048) with several splits: the partial states are merged by the
    second launch;
    sampled (sequence, head) pairs against the oracle, and a workspace whose
    counter block stays zero."""
    require_gpu()
    dev = torch.device("cuda")
    B, N, H = 33, 5, 64
    lens = [150 + 7 * b for b in range(B)]
    L_cap = max(lens) + N
    say("many pairs", dict(B=B, N=N, H=H, tree=tree))
    q = cpu_normal((B, N, H, D), 70, torch.bfloat16)
    k = cpu_normal((B, H, L_cap, D), 71, torch.bfloat16)
    v = cpu_normal((B, H, L_cap, D), 72, torch.bfloat16)
    par = np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1)) if tree else None
    need = glide.load().glide_tree_attn_workspace(B, N, H, D, L_cap, 3)
    ws = torch.zeros(need, dtype=torch.uint8, device=dev)
    out = torch.full((B, N, H, D), float("nan"), dtype=torch.bfloat16, device=dev)
    glide.glide_tree_attn(q.to(dev), k.to(dev), v.to(dev), torch.tensor(lens, dtype=torch.int32, device=dev),
                          None if par is None else torch.from_numpy(par).to(dev), out, max_splits=3,
                          workspace=ws)
    torch.cuda.synchronize()
    assert int(ws[:glide.ATTN_COUNTER_BYTES].count_nonzero()) == 0
    got = to64(out)
    assert np.isfinite(got).all()
    for b in (0, 16, B - 1):
        for h in (0, 31, H - 1):
            ref = OA.tree_attention_head(to64(q[b, :, h]), to64(k[b, h]), to64(v[b, h]), lens[b],
                                         None if par is None else par[b])
            assert float(np.abs(got[b, :, h] - ref).max()) <= BF16_TOL


def test_counter_block_left_zero():
    """Every split call -- both kernels, both dtypes, tree and cross mode,
    forced split counts up to 64 -- leaves the binding's cached workspace's
    counter block zero, and a repeated call gives bit-identical results."""
    require_gpu()
    dev = torch.device("cuda")
    for i, (B, N, H, L, dtype, splits, tree) in enumerate([
            (1, 16, 32, 2048, torch.bfloat16, 0, True), (4, 32, 8, 1500, torch.bfloat16, 0, True),
            (2, 64, 4, 3000, torch.bfloat16, 7, True), (3, 5, 16, 900, torch.bfloat16, 64, False),
            (2, 40, 4, 1200, torch.float32, 5, True), (1, 16, 8, 600, torch.float32, 0, False)]):
        say("counters", dict(B=B, N=N, H=H, L=L, dtype=str(dtype), splits=splits, tree=tree))
        q = cpu_normal((B, N, H, D), 80 + i, dtype).to(dev)
        k = cpu_normal((B, H, L + N, D), 90 + i, dtype).to(dev)
        v = cpu_normal((B, H, L + N, D), 100 + i, dtype).to(dev)
        lens = torch.tensor([L - 11 * b for b in range(B)], dtype=torch.int32, device=dev)
        par = torch.from_numpy(W.random_parents(B, N, 6, i)).to(dev) if tree else None
        outs = [torch.empty_like(q) for _ in range(2)]
        for o in outs:
            glide.glide_tree_attn(q, k, v, lens, par, o, max_splits=splits)
        ws = glide.attn_workspace(B, N, H, L + N, splits, dev)
        torch.cuda.synchronize()
        assert ws is not None and int(ws[:glide.ATTN_COUNTER_BYTES].count_nonzero()) == 0
        view = torch.int16 if dtype == torch.bfloat16 else torch.int32
        assert torch.equal(outs[0].view(view), outs[1].view(view))


def test_validation_reports_bad_device_data(monkeypatch):
    require_gpu()
    dev = torch.device("cuda")
    q = torch.zeros((1, 4, 2, D), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((1, 2, 64, D), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    monkeypatch.setenv("GLIDE_VALIDATE", "1")
    bad_parents = torch.tensor([[-1, 0, 3, 1]], dtype=torch.int32, device=dev)
    lens = torch.tensor([10], dtype=torch.int32, device=dev)
    with pytest.raises(glide.GlideError) as e:
        glide.glide_tree_attn(q, k, k, lens, bad_parents, out)
    assert e.value.status == glide.GLIDE_ERANGE
    with pytest.raises(glide.GlideError) as e:
        glide.glide_tree_attn(q, k, k, torch.tensor([61], dtype=torch.int32, device=dev),
                              torch.tensor([[-1, 0, 1, 2]], dtype=torch.int32, device=dev), out)
    assert e.value.status == glide.GLIDE_ERANGE
    # valid data passes validation
    glide.glide_tree_attn(q, k, k, lens, torch.tensor([[-1, 0, 1, 1]], dtype=torch.int32,
                                                       device=dev), out)
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("N,kind", [(16, "cape"), (64, "random"), (5, None)])
def test_peaked_scores(N, kind, dtype):
    """Queries scaled by 24 (scaled scores with a spread of hundreds in log2
    units): the lazily moved reference max is passed by far, often, and by
    single keys deep in the sequence; outputs stay within the tolerance."""
    require_gpu()
    B, H = 2, 3
    lens = [1500, 700]
    tree = kind is not None
    L_cap = max(lens) + (N if tree else 0)
    say("tree_attn peaked", dict(N=N, kind=kind, dtype=str(dtype)))
    q = (cpu_normal((B, N, H, D), 31, torch.float32) * 24).to(dtype)
    k = cpu_normal((B, H, L_cap, D), 32, dtype)
    v = cpu_normal((B, H, L_cap, D), 33, dtype)
    parents = _parents(kind, B, N, 34)
    dev = torch.device("cuda")
    out = torch.full((B, N, H, D), float("nan"), dtype=dtype, device=dev)
    glide.glide_tree_attn(q.to(dev), k.to(dev), v.to(dev), torch.tensor(lens, dtype=torch.int32, device=dev),
                          None if parents is None else torch.from_numpy(parents).to(dev), out)
    torch.cuda.synchronize()
    ref = OA.tree_attention(to64(q), to64(k), to64(v), lens, parents)
    # A peaked softmax returns nearly single value rows (|v| up to ~4), not
    # averages: in bf16 the probabilities and the output are rounded to 8
    # significant bits, so the bound is 1e-2 + 2^-8 |ref| (one output rounding
    # of a value in [4, 8) alone is up to 0.016).  float32 rounding of a score
    # is relative to its size, so the float32 bound scales with the query
    # scale.
    got = to64(out)
    if dtype == torch.bfloat16:
        excess = np.abs(got - ref) - (BF16_TOL + np.abs(ref) / 256)
        assert float(excess.max()) <= 0, float(np.abs(got - ref).max())
    else:
        err = float(np.abs(got - ref).max())
        assert err <= 24 * F32_TOL, err


@pytest.mark.parametrize("splits", [1, 0])
def test_largest_float32_cache(splits):
    """L_cap = 2^22 rows in float32, the largest accepted: a (sequence, head)
    slab of exactly 2^31 bytes, which one split reads through a single byte
    range.  Zero queries give every key weight 2^-22 exactly; the values are
    1 except the node's own row (the last one), which is 2^22 + 1, so the
    exact output is 2^23 / 2^22 = 2 -- and any row left unread (a truncated
    range) would pull it towards 1.  Every partial sum is an integer below
    2^24, so float32 holds them exactly."""
    require_gpu()
    dev = torch.device("cuda")
    L_cap = 1 << 22
    say("tree_attn largest float32 cache", dict(L_cap=L_cap, splits=splits))
    q = torch.zeros((1, 1, 1, D), dtype=torch.float32, device=dev)
    k = torch.zeros((1, 1, L_cap, D), dtype=torch.float32, device=dev)
    v = torch.ones((1, 1, L_cap, D), dtype=torch.float32, device=dev)
    v[0, 0, L_cap - 1] = float(L_cap + 1)
    lens = torch.tensor([L_cap - 1], dtype=torch.int32, device=dev)
    parents = torch.tensor([[-1]], dtype=torch.int32, device=dev)
    out = torch.full_like(q, float("nan"))
    glide.glide_tree_attn(q, k, v, lens, parents, out, max_splits=splits)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    del q, k, v
    torch.cuda.empty_cache()
    assert np.all(got == 2.0), got.ravel()[:4]


def _single_and_pair(q, k, v, L, par, splits):
    """The same sequence run alone (B = 1: split states merged inside the
    kernel, fp16 o / L from bf16 inputs) and as sequence 0 of a pair whose
    second sequence is empty (B = 2: float32 states merged by the second
    launch), with the same forced split plan."""
    dev = torch.device("cuda")
    N, H = q.shape[1], q.shape[2]
    one = torch.full_like(q, float("nan"))
    glide.glide_tree_attn(q, k, v, torch.tensor([L], dtype=torch.int32, device=dev), par, one,
                          max_splits=splits)
    q2 = torch.cat([q, q]).contiguous()
    k2, v2 = torch.cat([k, k]).contiguous(), torch.cat([v, v]).contiguous()
    par2 = None if par is None else torch.cat([par, par]).contiguous()
    two = torch.full((2, N, H, D), float("nan"), dtype=q.dtype, device=dev)
    glide.glide_tree_attn(q2, k2, v2, torch.tensor([L, 0], dtype=torch.int32, device=dev), par2, two,
                          max_splits=splits)
    torch.cuda.synchronize()
    return to64(one[0]), to64(two[0])


@pytest.mark.parametrize("tree", [True, False], ids=["tree", "cross"])
def test_half_states_match_float32_states(tree):
    """Single-sequence bf16 calls of 8 or more rows keep each split's
    normalised output o / L in fp16 (rounded to nearest even: error at most 2^-11 of the value, and
    the merge is a convex combination of the splits' values); against the
    float32 states of the two-launch merge on the same splits the outputs
    differ by at most 2^-11 max |v| plus one bf16 ulp (each side rounded
    once: up to 2^-7 of the value apart).  Both are within the oracle's
    bound."""
    require_gpu()
    dev = torch.device("cuda")
    N, H, L = (16 if tree else 8), 8, 2048
    for splits in (8, 3):
        say("half states", dict(tree=tree, splits=splits))
        q = cpu_normal((1, N, H, D), 61, torch.bfloat16).to(dev)
        k = cpu_normal((1, H, L + N, D), 62, torch.bfloat16).to(dev)
        v = cpu_normal((1, H, L + N, D), 63, torch.bfloat16).to(dev)
        par = torch.from_numpy(_parents("cape", 1, N, 64)).to(dev) if tree else None
        one, two = _single_and_pair(q, k, v, L, par, splits)
        vmax = float(to64(v).__abs__().max())
        bound = 2.0 ** -11 * vmax + 2.0 ** -7 * np.maximum(np.abs(one), np.abs(two)) + 1e-6
        assert float((np.abs(one - two) - bound).max()) <= 0
        ref = OA.tree_attention(to64(q), to64(k), to64(v), [L], None if par is None else par.cpu().numpy())[0]
        assert float(np.abs(one - ref).max()) <= BF16_TOL


@pytest.mark.parametrize("where", ["one split", "every split"])
def test_half_states_fall_back_to_float32(where):
    """Value rows near 2e5 (representable in bf16, beyond fp16's 65504):
    every split whose normalised output does not fit fp16 stores float32
    rows instead (its sum stored negated).  Large rows inside one split only
    (the others keep fp16 states of N(0, 1) rows) or in every split; the
    result is finite and matches the float32-state merge within one bf16
    ulp plus 2^-11 of the fp16 splits' values, and the oracle, scaled."""
    require_gpu()
    dev = torch.device("cuda")
    N, H, L, splits = 16, 4, 2048, 8
    big = 2.0e5
    say("half states fallback", dict(where=where))
    q = cpu_normal((1, N, H, D), 71, torch.bfloat16)
    k = cpu_normal((1, H, L + N, D), 72, torch.bfloat16)
    v = cpu_normal((1, H, L + N, D), 73, torch.float32)
    rows = slice(300, 560) if where == "one split" else slice(0, L + N)  # keys 288..575: split 1
    small = float(torch.cat([v[:, :, :300], v[:, :, 560:]], dim=2).abs().max()) if where == "one split" else 0.0
    v[:, :, rows] = big * (1.0 + 0.01 * v[:, :, rows])
    v = v.to(torch.bfloat16)
    q, k, v = q.to(dev), k.to(dev), v.to(dev)
    par = torch.from_numpy(_parents("cape", 1, N, 74)).to(dev)
    one, two = _single_and_pair(q, k, v, L, par, splits)
    # split 1's states are ~2e5 either way (they would overflow fp16 to
    # infinities); with every row large so are the outputs
    assert np.isfinite(one).all()
    assert np.abs(one).max() > (65504 if where == "every split" else 1.0e4)
    bound = 2.0 ** -11 * small + 2.0 ** -7 * np.maximum(np.abs(one), np.abs(two)) + 1e-6 * big
    assert float((np.abs(one - two) - bound).max()) <= 0
    ref = OA.tree_attention(to64(q), to64(k), to64(v), [L], par.cpu().numpy())[0]
    assert float((np.abs(one - ref) - (BF16_TOL * big + 2.0 ** -8 * np.abs(ref))).max()) <= 0


def test_half_states_flags_across_batches():
    """64 splits (eight merge batches of eight, one flag word each): value
    rows near 2e5 in splits 5, 37 and 63 only, so flag words 0, 4 and 7
    carry bits and the others none; two calls in a row (the merge clears
    the words it found set).  Against the float32-state merge within one
    bf16 ulp plus 2^-11 of the fp16 splits' values, and against the oracle."""
    require_gpu()
    dev = torch.device("cuda")
    N, H, L, splits = 16, 2, 64 * 128 - 16, 64
    big = 2.0e5
    say("half states flags", dict(N=N, H=H, L=L, splits=splits))
    q = cpu_normal((1, N, H, D), 81, torch.bfloat16)
    k = cpu_normal((1, H, L + N, D), 82, torch.bfloat16)
    v = cpu_normal((1, H, L + N, D), 83, torch.float32)
    small = float(v.abs().max())
    for sp in (5, 37, 63):  # splits of 128 keys
        v[:, :, 128 * sp + 10:128 * sp + 100] = big * (1.0 + 0.01 * v[:, :, 128 * sp + 10:128 * sp + 100])
    v = v.to(torch.bfloat16)
    q, k, v = q.to(dev), k.to(dev), v.to(dev)
    par = torch.from_numpy(_parents("cape", 1, N, 84)).to(dev)
    first, two = _single_and_pair(q, k, v, L, par, splits)
    again, _ = _single_and_pair(q, k, v, L, par, splits)
    assert np.array_equal(first, again)
    assert np.isfinite(first).all()
    bound = 2.0 ** -11 * small + 2.0 ** -7 * np.maximum(np.abs(first), np.abs(two)) + 1e-6 * big
    assert float((np.abs(first - two) - bound).max()) <= 0
    ref = OA.tree_attention(to64(q), to64(k), to64(v), [L], par.cpu().numpy())[0]
    assert float((np.abs(first - ref) - (BF16_TOL * big + 2.0 ** -8 * np.abs(ref))).max()) <= 0

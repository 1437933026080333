"""The no-allocation entry point, glide_tree_attn_noalloc, through the C ABI
against glide_tree_attn (the existing entry point, same kernels): on two
calls in a row, the second with a smaller input, the outputs are bit-identical
to glide_tree_attn's and within the attention bound of the float64 oracle.
Also checked: sizes beyond the fixed scratch are refused before any HIP call
(GLIDE_ESCRATCH), and a one-split shape that needs no scratch."""

import numpy as np
import pytest
import torch

import paper_2402_02082_amd as glide
from oracle import attention as OA
from tests.gpu_common import BF16_TOL, F32_TOL, cpu_normal, require_gpu, say, to64

pytestmark = pytest.mark.gpu


def _case(B, N, H, lens, L_cap, dtype, seed, tree=True):
    dev = torch.device("cuda")
    q = cpu_normal((B, N, H, 128), seed, dtype).to(dev)
    k = cpu_normal((B, H, L_cap, 128), seed + 1, dtype).to(dev)
    v = cpu_normal((B, H, L_cap, 128), seed + 2, dtype).to(dev)
    rng = np.random.default_rng(seed)
    par = np.array([[int(rng.integers(-1, n)) if n else -1 for n in range(N)] for _ in range(B)],
                   dtype=np.int32) if tree else None
    return (q, k, v, torch.tensor(lens, dtype=torch.int32, device=dev),
            None if par is None else torch.from_numpy(par).to(dev), par)


def _same(a, b):
    view = torch.int16 if a.dtype == torch.bfloat16 else torch.int32
    return torch.equal(a.view(view), b.view(view))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_noalloc_matches_existing_entry_point(dtype):
    require_gpu()
    # a large split call, then a smaller one: the second reuses the scratch
    # the first left behind (partials are written before they are read)
    cases = [dict(B=2, N=16, H=32, lens=[2048, 1500], L_cap=2064, seed=3, splits=0),
             dict(B=1, N=5, H=4, lens=[700], L_cap=705, seed=4, splits=6)]
    for c in cases:
        say("noalloc", dict(c, dtype=str(dtype)))
        q, k, v, lens, par, par_np = _case(c["B"], c["N"], c["H"], c["lens"], c["L_cap"], dtype, c["seed"])
        assert glide.load().glide_tree_attn_workspace(c["B"], c["N"], c["H"], 128, c["L_cap"],
                                                      c["splits"]) > 0
        got = torch.full_like(q, float("nan"))
        ref = torch.full_like(q, float("nan"))
        glide.glide_tree_attn_noalloc(q, k, v, lens, par, got, max_splits=c["splits"])
        glide.glide_tree_attn(q, k, v, lens, par, ref, max_splits=c["splits"])
        torch.cuda.synchronize()
        assert _same(got, ref)
        want = OA.tree_attention(to64(q), to64(k), to64(v), c["lens"], par_np)
        err = float(np.abs(to64(got) - want).max())
        assert err <= (BF16_TOL if dtype == torch.bfloat16 else F32_TOL), err


def test_noalloc_cross_mode_and_one_split():
    require_gpu()
    q, k, v, lens, _, _ = _case(3, 5, 8, [300, 0, 17], 320, torch.bfloat16, 7, tree=False)
    for splits in (0, 1):
        say("noalloc cross", dict(splits=splits))
        got = torch.full_like(q, float("nan"))
        ref = torch.full_like(q, float("nan"))
        glide.glide_tree_attn_noalloc(q, k, v, lens, None, got, max_splits=splits)
        glide.glide_tree_attn(q, k, v, lens, None, ref, max_splits=splits)
        torch.cuda.synchronize()
        assert _same(got, ref)


def test_noalloc_refuses_plans_beyond_the_scratch():
    require_gpu()
    lib = glide.load()
    cap = lib.glide_tree_attn_noalloc_max_workspace()
    B, N, H, L_cap = 8, 64, 52, 8256
    assert lib.glide_tree_attn_workspace(B, N, H, 128, L_cap, 64) > cap
    q = torch.zeros((B, N, H, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((B, H, L_cap, 128), dtype=torch.bfloat16, device="cuda")
    lens = torch.full((B,), 100, dtype=torch.int32, device="cuda")
    with pytest.raises(glide.GlideError) as e:
        glide.glide_tree_attn_noalloc(q, k, k, lens, None, torch.empty_like(q), max_splits=64)
    assert e.value.status == glide.GLIDE_ESCRATCH

"""Pins for the GliDe cross-attention block oracle (CPU only).

* identity projections reduce the block to the cross-attention oracle;
* a head whose query projection is zero attends uniformly: its slice of the
  concatenation is the mean of that head's cached values (closed form);
* an output projection that permutes features permutes the output the same
  way (a transposed operand would apply the inverse permutation);
* the block is linear in W^O, and scaling the query projection by c equals
  attention with scale c / sqrt(d_k);
* per-head matrices W_j and W^O written out separately (the paper's shapes)
  give the same block as the stacked, transposed storage;
* rows_matmul against a plain triple loop;
* planted mistakes in the oracle must fail at least one pin.
"""

import numpy as np
import pytest

from oracle import attention as OA
from oracle import cross_block as OX


def _case(rng, B=2, Nq=3, H=3, D=4, d_D=None, L_cap=9):
    d_D = H * D if d_D is None else d_D
    hidden = rng.standard_normal((B, Nq, d_D))
    k = rng.standard_normal((B, H, L_cap, D))
    v = rng.standard_normal((B, H, L_cap, D))
    lens = rng.integers(1, L_cap + 1, size=B)
    return hidden, k, v, lens


def identity_errors(seed=21):
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng)
    B, Nq, d = hidden.shape
    H, D = k.shape[1], k.shape[3]
    got = OX.cross_block(hidden, np.eye(d), k, v, lens, np.eye(d))
    want = OA.tree_attention(hidden.reshape(B, Nq, H, D), k, v, lens, None).reshape(B, Nq, d)
    return [] if np.allclose(got, want, atol=1e-12, rtol=0) else [("identity",)]


def zero_head_errors(seed=22):
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng, d_D=7)
    H, D = k.shape[1], k.shape[3]
    wq_t = rng.standard_normal((H * D, 7))
    wq_t[D:2 * D] = 0.0                       # head 1 sees q = 0
    got = OX.cross_block(hidden, wq_t, k, v, lens, np.eye(H * D))
    bad = []
    for b in range(hidden.shape[0]):
        mean = v[b, 1, :lens[b]].mean(axis=0)
        if not np.allclose(got[b, :, D:2 * D], mean[None], atol=1e-12, rtol=0):
            bad.append(("zero head", b))
    return bad


def permutation_errors(seed=23):
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng, d_D=5)
    HD = k.shape[1] * k.shape[3]
    wq_t = rng.standard_normal((HD, 5))
    perm = np.roll(np.arange(HD), 1)          # not its own inverse
    wo_t = np.eye(HD)[perm]                   # out[:, n] = concat[:, perm[n]]
    base = OX.cross_block(hidden, wq_t, k, v, lens, np.eye(HD))
    got = OX.cross_block(hidden, wq_t, k, v, lens, wo_t)
    return [] if np.allclose(got, base[..., perm], atol=1e-12, rtol=0) else [("permutation",)]


def linearity_and_scale_errors(seed=24):
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng, d_D=6)
    H, D = k.shape[1], k.shape[3]
    wq_t = rng.standard_normal((H * D, 6))
    wo1, wo2 = rng.standard_normal((6, H * D)), rng.standard_normal((6, H * D))
    bad = []
    a = OX.cross_block(hidden, wq_t, k, v, lens, wo1 + wo2)
    b = OX.cross_block(hidden, wq_t, k, v, lens, wo1) + OX.cross_block(hidden, wq_t, k, v, lens, wo2)
    if not np.allclose(a, b, atol=1e-10, rtol=0):
        bad.append(("linearity",))
    # scaling Q by c is attention with scale c / sqrt(d_k)
    hidden2, k2, v2, lens2 = _case(rng)
    B, Nq, d = hidden2.shape
    c = 2.5
    got = OX.cross_block(hidden2, c * np.eye(d), k2, v2, lens2, np.eye(d))
    want = OA.tree_attention(hidden2.reshape(B, Nq, H, D), k2, v2, lens2, None,
                             scale=c / np.sqrt(D)).reshape(B, Nq, d)
    if not np.allclose(got, want, atol=1e-12, rtol=0):
        bad.append(("scale",))
    return bad


def per_head_errors(seed=25):
    """The paper's shapes: W_j in R^{d_D x d_k}, W^O in R^{h d_k x d_D}."""
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng)           # d_D = h * d_k: square projections
    B, Nq, d_D = hidden.shape
    H, D = k.shape[1], k.shape[3]
    Wj = [rng.standard_normal((d_D, D)) for _ in range(H)]
    WO = rng.standard_normal((H * D, d_D))
    want = np.zeros((B, Nq, d_D))
    for b in range(B):
        hd = [OA.attention_rows(hidden[b] @ Wj[j], k[b, j, :lens[b]], v[b, j, :lens[b]],
                                1.0 / np.sqrt(D)) for j in range(H)]
        want[b] = np.concatenate(hd, axis=1) @ WO
    wq_t = np.concatenate([W.T for W in Wj], axis=0)   # row j*D + c = column c of W_j
    got = OX.cross_block(hidden, wq_t, k, v, lens, WO.T)
    return [] if np.allclose(got, want, atol=1e-12, rtol=0) else [("per head",)]


def rows_matmul_errors(seed=26):
    rng = np.random.default_rng(seed)
    a, w_t = rng.standard_normal((3, 5)), rng.standard_normal((4, 5))
    got = OX.rows_matmul(a, w_t)
    for m in range(3):
        for n in range(4):
            if abs(got[m, n] - sum(float(a[m, i]) * float(w_t[n, i]) for i in range(5))) > 1e-12:
                return [("rows_matmul", m, n)]
    return []


PINS = [identity_errors, zero_head_errors, permutation_errors, linearity_and_scale_errors,
        per_head_errors, rows_matmul_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


# ---- the bfloat16-store path ----
#
# ``store=bfloat16`` rounds exactly two intermediates, the projected queries
# and the concatenated heads, to bfloat16 (round to nearest, ties to even,
# after the float32 value a kernel accumulates), and nothing else.  Two pins:
# intermediates that are bfloat16-exact make the path equal the float64 one
# bit for bit (so no other value -- the output in particular -- is rounded),
# and on general values the path equals the block computed here with each of
# the two intermediates rounded by a bfloat16 rounding written out from the
# format's definition (so the format, the rounding rule and the two points
# are the stated ones).


def bf16_round_by_hand(x):
    """float64 -> float32 (IEEE round to nearest even) -> bfloat16: keep the
    top 16 bits of the float32 pattern, rounding the dropped 16 bits to
    nearest with ties to the even kept pattern.  Written from the format's
    definition (8 exponent bits, 7 stored fraction bits), independent of
    torch's conversion."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    low = bits & 0xFFFF
    keep = bits >> 16
    up = (low > 0x8000) | ((low == 0x8000) & ((keep & 1) == 1))
    keep = keep + up.astype(np.uint64)
    return (keep << 16).astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_hand_rounding_errors():
    """The hand rounding itself against values whose bfloat16 neighbours are
    known exactly: ties go to the even pattern, just past a tie rounds up,
    the float32 step happens first, signs are symmetric, and bfloat16 (7
    fraction bits) differs from float16 (10 bits) on 1 + 2^-9."""
    e = 2.0 ** -7                      # bfloat16 spacing in [1, 2)
    cases = [(1.0, 1.0), (1.0 + e / 2, 1.0), (1.0 + 3 * e / 2, 1.0 + 2 * e),
             (1.0 + e / 2 + 2.0 ** -20, 1.0 + e), (1.0 + 2.0 ** -9, 1.0),
             (-(1.0 + 3 * e / 2), -(1.0 + 2 * e)), (3.0, 3.0), (0.0, 0.0),
             (2.0 ** -130, 2.0 ** -130), (1.0 + e / 2 + 2.0 ** -40, 1.0)]
    bad = []
    for x, want in cases:
        got = float(bf16_round_by_hand(np.array([x]))[0])
        if got != want:
            bad.append(("hand rounding", x, got, want))
    return bad


def store_exact_intermediates_errors(seed=28):
    """Projected queries and heads that bfloat16 holds exactly: small-integer
    queries (small-integer hidden rows times 0/1 weights) and one visible key
    per sequence (its value row, dyadic, is the head's output with weight 1).
    The output projection (weights k/3) is not bfloat16-exact, so rounding at
    any further point shows."""
    import torch
    rng = np.random.default_rng(seed)
    B, Nq, H, D, d_D, L_cap = 2, 3, 2, 4, 6, 5
    hidden = rng.integers(-3, 4, size=(B, Nq, d_D)).astype(np.float64)
    wq_t = rng.integers(0, 2, size=(H * D, d_D)).astype(np.float64)
    k = rng.standard_normal((B, H, L_cap, D))
    v = rng.integers(-64, 65, size=(B, H, L_cap, D)) / 16.0
    lens = [1, 1]
    wo_t = rng.integers(1, 9, size=(d_D, H * D)) / 3.0
    a = OX.cross_block(hidden, wq_t, k, v, lens, wo_t)
    b = OX.cross_block(hidden, wq_t, k, v, lens, wo_t, store=torch.bfloat16)
    if not np.array_equal(a, b):
        return [("store on exact intermediates",)]
    if np.array_equal(bf16_round_by_hand(a), a):
        return [("output happens to be bfloat16-exact: the pin would not see output rounding",)]
    return []


def store_hand_rounded_errors(seed=29):
    """General values: the store path equals the block with the projected
    queries and the concatenated heads rounded by hand, float64 elsewhere
    (per-head attention from the pinned attention oracle)."""
    import torch
    rng = np.random.default_rng(seed)
    hidden, k, v, lens = _case(rng, B=2, Nq=3, H=3, D=4, d_D=10, L_cap=9)
    B, Nq, d_D = hidden.shape
    H, D = k.shape[1], k.shape[3]
    wq_t = rng.standard_normal((H * D, d_D)) / 3
    wo_t = rng.standard_normal((d_D, H * D)) / 3
    q = bf16_round_by_hand(hidden.reshape(B * Nq, d_D) @ wq_t.T).reshape(B, Nq, H, D)
    heads = np.zeros((B, Nq, H, D))
    for b in range(B):
        for j in range(H):
            heads[b, :, j] = OA.attention_rows(q[b, :, j], k[b, j, :lens[b]], v[b, j, :lens[b]],
                                               1.0 / np.sqrt(D))
    want = (bf16_round_by_hand(heads.reshape(B * Nq, H * D)) @ wo_t.T).reshape(B, Nq, d_D)
    got = OX.cross_block(hidden, wq_t, k, v, lens, wo_t, store=torch.bfloat16)
    if not np.allclose(got, want, rtol=1e-13, atol=1e-13):
        return [("store vs hand rounding", float(np.abs(got - want).max()))]
    # and the rounding is not a no-op on these values
    if np.allclose(got, OX.cross_block(hidden, wq_t, k, v, lens, wo_t), rtol=0, atol=1e-6):
        return [("store path changed nothing",)]
    return []


STORE_PINS = [bf16_hand_rounding_errors, store_exact_intermediates_errors,
              store_hand_rounded_errors]


@pytest.mark.parametrize("pin", STORE_PINS, ids=lambda f: f.__name__)
def test_store_pin(pin):
    assert pin() == []


_REAL_ROUND = OX._round
_REAL_BLOCK = OX.cross_block


def _smut_output_rounded_too(monkeypatch):
    def block(hidden, wq_t, k, v, lens, wo_t, store=None, scale=None):
        out = _REAL_BLOCK(hidden, wq_t, k, v, lens, wo_t, store=store, scale=scale)
        return OX._round(out, store)
    monkeypatch.setattr(OX, "cross_block", block)


def _smut_float16_storage(monkeypatch):
    import torch

    def rnd(x, store):
        return _REAL_ROUND(x, None if store is None else torch.float16)
    monkeypatch.setattr(OX, "_round", rnd)


def _smut_truncating_rounding(monkeypatch):
    def rnd(x, store):
        if store is None:
            return x
        bits = np.asarray(x, dtype=np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
        return bits.view(np.float32).astype(np.float64)
    monkeypatch.setattr(OX, "_round", rnd)


def _smut_queries_only(monkeypatch):
    calls = {"n": 0}

    def rnd(x, store):
        calls["n"] += 1
        return _REAL_ROUND(x, store) if calls["n"] % 2 == 1 else x
    monkeypatch.setattr(OX, "_round", rnd)


def _smut_heads_only(monkeypatch):
    calls = {"n": 0}

    def rnd(x, store):
        calls["n"] += 1
        return _REAL_ROUND(x, store) if calls["n"] % 2 == 0 else x
    monkeypatch.setattr(OX, "_round", rnd)


STORE_MUTANTS = [_smut_output_rounded_too, _smut_float16_storage, _smut_truncating_rounding,
                 _smut_queries_only, _smut_heads_only]


@pytest.mark.parametrize("mutant", STORE_MUTANTS, ids=lambda f: f.__name__)
def test_planted_store_mistake_is_caught(monkeypatch, mutant):
    mutant(monkeypatch)
    failures = []
    for pin in STORE_PINS:
        failures += pin()
    assert failures


# ---- planted mistakes ----

_REAL_MM = OX.rows_matmul
_REAL_ATT = OA.tree_attention


def _mut_untransposed_q(monkeypatch):
    calls = {"n": 0}

    def mm(a, w_t):
        calls["n"] += 1
        if calls["n"] % 2 == 1 and w_t.shape[0] == w_t.shape[1]:   # the query projection
            return np.asarray(a, dtype=np.float64) @ np.asarray(w_t, dtype=np.float64)
        return _REAL_MM(a, w_t)
    monkeypatch.setattr(OX, "rows_matmul", mm)


def _mut_reversed_heads(monkeypatch):
    def att(q, k, v, lens, parents=None, scale=None):
        return _REAL_ATT(q, k, v, lens, parents, scale)[:, :, ::-1]
    monkeypatch.setattr(OA, "tree_attention", att)


def _mut_no_output_projection(monkeypatch):
    def block(hidden, wq_t, k, v, lens, wo_t, store=None, scale=None):
        B, Nq, _ = np.asarray(hidden).shape
        H, D = k.shape[1], k.shape[3]
        q = _REAL_MM(np.asarray(hidden).reshape(B * Nq, -1), wq_t).reshape(B, Nq, H, D)
        return OA.tree_attention(q, k, v, lens, None, scale=scale).reshape(B, Nq, H * D)
    monkeypatch.setattr(OX, "cross_block", block)


def _mut_model_width_scale(monkeypatch):
    def att(q, k, v, lens, parents=None, scale=None):
        H, D = q.shape[2], q.shape[3]
        return _REAL_ATT(q, k, v, lens, parents, 1.0 / np.sqrt(H * D) if scale is None else scale)
    monkeypatch.setattr(OA, "tree_attention", att)


MUTANTS = [_mut_untransposed_q, _mut_reversed_heads, _mut_no_output_projection,
           _mut_model_width_scale]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mutant(monkeypatch)
    failures = []
    for pin in PINS:
        failures += pin()
    assert failures

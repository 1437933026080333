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


def test_store_rounding_stays_close():
    rng = np.random.default_rng(27)
    hidden, k, v, lens = _case(rng, d_D=16)
    HD = k.shape[1] * k.shape[3]
    wq_t, wo_t = rng.standard_normal((HD, 16)) / 4, rng.standard_normal((16, HD)) / 4
    import torch
    a = OX.cross_block(hidden, wq_t, k, v, lens, wo_t)
    b = OX.cross_block(hidden, wq_t, k, v, lens, wo_t, store=torch.bfloat16)
    assert 0 < np.abs(a - b).max() < 5e-2


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

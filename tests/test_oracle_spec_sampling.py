"""Pins for the speculative-sampling and expected-speedup oracle (CPU only).

* Table 1: E(Spd) recomputed from every printed (alpha, c) pair with gamma = 5
  matches the printed expected speedup within 0.01 (44 cells;
  tests/golden/table1_expected_speedup.json);
* Sec. 3: with speculative sampling the emitted token follows the target's
  distribution: over a fine grid of the two uniforms that decide a one-token
  proposal, each token's share of the grid equals p_T within the grid
  resolution, for random tiny vocabularies;
* Sec. 5.1: the probability of accepting the first proposal token equals
  alpha = sum_x min(p_T(x), p_D(x)) (grid over its uniform);
* identical draft and target distributions accept the whole chain;
  a proposal token the target gives no mass is always rejected and the
  replacement never equals it; the fixed-point sampler's token intervals
  against explicit enumeration; a hand-worked two-step example;
* planted mistakes in the oracle must fail at least one pin.
"""

import json
import os

import numpy as np
import pytest

from oracle import spec_sampling as S

TABLE1 = os.path.join(os.path.dirname(__file__), "golden", "table1_expected_speedup.json")


def table1_errors():
    g = json.load(open(TABLE1))
    bad = []
    for r in g["rows"]:
        for a, e in zip(r["acc"], r["spd"]):
            v = S.expected_speedup(a / 100.0, g["gamma"], r["cost"] / 100.0)
            if abs(v - e) > 0.01:
                bad.append((r["target"], r["draft"], a, e, v))
    return bad


def _dist(rng, V, zero_frac=0.0):
    p = rng.dirichlet(np.full(V, 0.7))
    p[rng.random(V) < zero_frac] = 0.0
    if p.sum() == 0:
        p[0] = 1.0
    return (p / p.sum()).astype(np.float32)


GRID = 2000
_GRID = (np.arange(GRID) + 0.5) / GRID


def _accept_share(x, pd, pt):
    """Share of the r-grid that accepts proposal token x (one-token chain)."""
    return float(np.mean([S.spec_sample_verify_one([x], pd[None], np.stack([pt, pt]), [r, 0.5])[0]
                          for r in _GRID]))


def distribution_errors(seed=41, trials=6):
    """The emitted token's distribution is p_T.  Acceptance depends only on
    r and the replacement only on u, so each is measured on its own grid:
    emitted(y) = sum_x p_D(x) [acc_x 1(y = x) + (1 - acc_x) rej_x(y)]."""
    rng = np.random.default_rng(seed)
    bad = []
    r_reject = np.float32(1.0) - np.float32(2.0 ** -24)   # rejects every ratio below 1
    for _ in range(trials):
        V = int(rng.integers(2, 6))
        pd = _dist(rng, V, 0.2)
        pt = _dist(rng, V, 0.2)
        emitted = np.zeros(V)
        for x in range(V):
            if pd[x] == 0:
                continue
            acc = _accept_share(x, pd, pt)
            emitted[x] += pd[x] * acc
            if acc < 1.0:
                rej = np.zeros(V)
                for u in _GRID:
                    a, tok = S.spec_sample_verify_one([x], pd[None], np.stack([pt, pt]), [r_reject, u])
                    rej[tok] += 1.0 / GRID
                emitted += pd[x] * (1.0 - acc) * rej
        if np.abs(emitted - pt).max() > 5e-3:
            bad.append(("distribution", V, emitted, pt))
    return bad


def acceptance_rate_errors(seed=42, trials=10):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(trials):
        V = int(rng.integers(2, 8))
        pd, pt = _dist(rng, V), _dist(rng, V, 0.3)
        acc = sum(pd[x] * _accept_share(x, pd, pt) for x in range(V))
        if abs(acc - S.acceptance_rate(pt, pd)) > 1e-3:
            bad.append(("alpha", acc, S.acceptance_rate(pt, pd)))
    return bad


def special_case_errors(seed=43):
    rng = np.random.default_rng(seed)
    bad = []
    for _ in range(20):
        V, gamma = 6, 4
        p = np.stack([_dist(rng, V) for _ in range(gamma + 1)])
        x = [int(np.argmax(p[i])) for i in range(gamma)]
        u = rng.random(gamma + 1).astype(np.float32) * np.float32(0.999)
        acc, tok = S.spec_sample_verify_one(x, p[:gamma], p, u)
        if acc != gamma:
            bad.append(("same distributions", acc))
        if tok != S.sample_fixed(S.fixed_weights(p[gamma]), u[gamma]):
            bad.append(("bonus from the last target row",))
        # a token the target gives no mass is rejected and never re-emitted
        pt = p.copy()
        pt[0, x[0]] = 0.0
        acc, tok = S.spec_sample_verify_one(x, p[:gamma], pt, u)
        if acc != 0 or tok == x[0]:
            bad.append(("zero target mass", acc, tok))
    # fixed-point inverse CDF: weights [3, 0, 5] -> u in [0, 3/8) -> 0, else 2
    w = [3, 0, 5]
    for u in (0.0, 0.37, 0.375, 0.99):
        want = 0 if np.floor(np.float64(np.float32(u)) * 8) < 3 else 2
        if S.sample_fixed(w, u) != want:
            bad.append(("sampler", u))
    return bad


def worked_example_errors():
    """Two-step chain over 3 tokens, hand-derived.
    Row 0: p_D = (0.5, 0.25, 0.25), p_T = (0.25, 0.5, 0.25); proposal 1
    (p_T/p_D = 2): accepted for any r.  Row 1: p_D = (0.5, 0.5, 0), p_T =
    (0.25, 0.25, 0.5); proposal 0 (ratio 0.5): r = 0.6 rejects.  Residual
    max(0, p_T - p_D) = (0, 0, 0.5): token 2 whatever u."""
    pd = np.array([[0.5, 0.25, 0.25], [0.5, 0.5, 0.0]], dtype=np.float32)
    pt = np.array([[0.25, 0.5, 0.25], [0.25, 0.25, 0.5], [1.0, 0.0, 0.0]], dtype=np.float32)
    got = S.spec_sample_verify_one([1, 0], pd, pt, [0.99, 0.6, 0.1])
    got2 = S.spec_sample_verify_one([1, 0], pd, pt, [0.3, 0.4, 0.1])   # r = 0.4 accepts
    bad = []
    if got != (1, 2):
        bad.append(("example reject", got))
    if got2 != (2, 0):                  # all accepted: bonus from row 2 = token 0
        bad.append(("example accept", got2))
    return bad


PINS = [table1_errors, distribution_errors, acceptance_rate_errors, special_case_errors,
        worked_example_errors]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    assert pin() == []


# ---- planted mistakes ----

_REAL_ONE = S.spec_sample_verify_one
_REAL_SPD = S.expected_speedup


def _mut_ratio_inverted(monkeypatch):
    def one(dt, pd, pt, u):
        return _REAL_ONE(dt, pt[:len(dt)], np.concatenate([pd, pt[-1:]]), u)
    monkeypatch.setattr(S, "spec_sample_verify_one", one)


def _mut_residual_is_target(monkeypatch):
    def one(dt, pd, pt, u):
        acc, tok = _REAL_ONE(dt, pd, pt, u)
        if acc < len(dt):
            tok = S.sample_fixed(S.fixed_weights(np.asarray(pt)[acc]), u[len(dt)])
        return acc, tok
    monkeypatch.setattr(S, "spec_sample_verify_one", one)


def _mut_bonus_from_draft(monkeypatch):
    def one(dt, pd, pt, u):
        acc, tok = _REAL_ONE(dt, pd, pt, u)
        if acc == len(dt):
            tok = S.sample_fixed(S.fixed_weights(np.asarray(pd)[-1]), u[len(dt)])
        return acc, tok
    monkeypatch.setattr(S, "spec_sample_verify_one", one)


def _mut_speedup_exponent(monkeypatch):
    monkeypatch.setattr(S, "expected_speedup",
                        lambda a, g, c: (1 - a ** g) / ((1 - a) * (g * c + 1)))


MUTANTS = [_mut_ratio_inverted, _mut_residual_is_target, _mut_bonus_from_draft,
           _mut_speedup_exponent]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mutant(monkeypatch)
    failures = []
    for pin in PINS:
        failures += pin()
    assert failures

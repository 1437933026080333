"""Oracle: chain verification with speculative sampling, and the expected
speedup model (test infrastructure only).

What is computed:

* Sec. 3 (Background): a proposal of gamma draft tokens is verified in one
  target pass; the first n accepted tokens and one more token from the target
  extend the prefix, and with the speculative-sampling acceptance strategy the
  emitted tokens follow the target's own sampling distribution.  Sec. 5.1
  ("Experiment design") uses this strategy, with gamma = 5 chains, for the
  GliDe-only experiments.  The paper defers the rule itself to its cited
  work; restated here:
    - proposal token x_i (row i - 1 of both distributions) is accepted when
      r_i * p_D(x_i) < p_T(x_i), i.e. with probability min(1, p_T/p_D);
    - at the first rejection, at row j, the emitted token is drawn from the
      residual max(0, p_T_j - p_D_j) (renormalised) and the chain stops;
    - if all gamma tokens are accepted, the emitted token is drawn from the
      target's distribution after the last one (row gamma).
* Sec. 5.1 ("Metrics"): the acceptance rate alpha = sum_x min(p_T(x),
  p_D(x)), and the expected speedup
  E(Spd) = (1 - alpha^(gamma+1)) / ((1 - alpha) (gamma c + 1)).

Readings where the paper is silent or garbled:
* The random numbers are inputs: ``uniforms[b, i]`` (i < gamma) is r_{i+1}
  of the acceptance tests and ``uniforms[b, gamma]`` is the one draw of the
  emitted token, each in [0, 1).
* A distribution is sampled by inverse CDF over fixed-point weights
  w_v = floor(p_v * 2^32) (p as float32, exact in float64): with
  W = sum_v w_v and t = floor(u * W) (float64 product), the token is the
  first v whose running sum of weights exceeds t.  Integer sums do not
  depend on summation order, so the drawn token is a property of the inputs.
  A residual of zero weight falls back to the target row itself; a target
  row of zero weight gives token 0.
* The Metrics paragraph writes alpha as an expectation under p_D of
  min(p_T, p_D); the cited definition is the sum over tokens of
  min(p_T, p_D) (the expectation of min(1, p_T/p_D) under p_D), used here.
"""

import numpy as np

FIXED_ONE = 1 << 32


def fixed_weights(p):
    """w_v = floor(p_v * 2^32) for float32 probabilities (negatives -> 0)."""
    p = np.maximum(np.asarray(p, dtype=np.float32).astype(np.float64), 0.0)
    return np.floor(p * FIXED_ONE).astype(np.int64)


def sample_fixed(weights, u):
    """Inverse-CDF draw from integer weights with one uniform in [0, 1)."""
    w = [int(x) for x in weights]
    total = sum(w)
    if total == 0:
        return None
    t = int(np.floor(np.float64(np.float32(u)) * np.float64(total)))
    t = min(t, total - 1)
    run = 0
    for v, x in enumerate(w):
        run += x
        if run > t:
            return v
    raise AssertionError("unreachable: t < total")


def spec_sample_verify_one(draft_tokens, p_draft, p_target, uniforms):
    """One chain.  draft_tokens [gamma]; p_draft [gamma, V]; p_target
    [gamma + 1, V]; uniforms [gamma + 1].  Returns (accept_len, next_token)."""
    p_draft = np.asarray(p_draft, dtype=np.float32)
    p_target = np.asarray(p_target, dtype=np.float32)
    uniforms = np.asarray(uniforms, dtype=np.float32)
    gamma = len(draft_tokens)
    u_emit = uniforms[gamma]
    for i in range(gamma):
        x = int(draft_tokens[i])
        pd = np.float32(p_draft[i, x])
        pt = np.float32(p_target[i, x])
        # r * p_D(x) < p_T(x), both sides in float32
        if not np.float32(uniforms[i]) * pd < pt:
            residual = np.maximum(p_target[i] - p_draft[i], np.float32(0))
            tok = sample_fixed(fixed_weights(residual), u_emit)
            if tok is None:
                tok = sample_fixed(fixed_weights(p_target[i]), u_emit)
            return i, 0 if tok is None else tok
    tok = sample_fixed(fixed_weights(p_target[gamma]), u_emit)
    return gamma, 0 if tok is None else tok


def spec_sample_verify(draft_tokens, p_draft, p_target, uniforms):
    """Batched: [B, gamma], [B, gamma, V], [B, gamma + 1, V], [B, gamma + 1]
    -> accept_len [B], next_token [B] (int32)."""
    draft_tokens = np.asarray(draft_tokens)
    B = draft_tokens.shape[0]
    out = np.zeros((2, B), dtype=np.int32)
    for b in range(B):
        out[:, b] = spec_sample_verify_one(draft_tokens[b], p_draft[b], p_target[b], uniforms[b])
    return out[0], out[1]


def acceptance_rate(p_target, p_draft):
    """alpha = sum_x min(p_T(x), p_D(x)) for one position (float64)."""
    return float(np.minimum(np.asarray(p_target, dtype=np.float64),
                            np.asarray(p_draft, dtype=np.float64)).sum())


def expected_speedup(alpha, gamma, c):
    """E(Spd) = (1 - alpha^(gamma+1)) / ((1 - alpha)(gamma c + 1)); the limit
    gamma + 1 at alpha = 1."""
    alpha, c = float(alpha), float(c)
    if alpha == 1.0:
        return (gamma + 1) / (gamma * c + 1)
    return (1 - alpha ** (gamma + 1)) / ((1 - alpha) * (gamma * c + 1))

"""Oracle: the GliDe cross-attention sub-layer with its projections (test
infrastructure only).

What is computed (Sec. 4.1, the Q^{m,j} and MultiHead equations; plain
definitions, so this is the definition written out):

* for every target head j, Q^{m,j} = H^m W_j with W_j in R^{d_D x d_k};
* hd_j = SoftMax(Q^{m,j} (K^{l,j})^T / sqrt(d_k)) V^{l,j} over the target
  layer's cached rows (``attention.tree_attention`` in cross mode);
* MultiHead = Concat(hd_1, ..., hd_h) W^O with W^O in R^{h d_k x d_D}.

Weight storage (a reading; the paper gives only the mathematical shapes): the
projections are stored transposed, one row per output feature, as framework
linear layers keep them -- ``wq_t`` is ``[h*d_k, d_D]`` with row ``j*d_k + c``
equal to column ``c`` of W_j, and ``wo_t`` is ``[d_D, h*d_k]`` (the transpose
of W^O).  Hidden rows ``[B, Nq, d_D]``; caches ``[B, h, L_cap, d_k]``;
``seq_lens`` ``[B]`` rows visible to every query (the cache up to t - 1).

``store`` rounds the two stored intermediates (the projected queries and the
concatenated heads) to that dtype, as a kernel that keeps them in bf16 does;
``None`` keeps float64 throughout.
"""

import numpy as np

from . import attention as OA


def _round(x, store):
    if store is None:
        return x
    import torch
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(store).double().numpy()


def rows_matmul(a, w_t):
    """out = a @ w_t^T in float64: ``a`` ``[M, K]``, ``w_t`` ``[N, K]``."""
    return np.asarray(a, dtype=np.float64) @ np.asarray(w_t, dtype=np.float64).T


def cross_block(hidden, wq_t, k_cache, v_cache, seq_lens, wo_t, store=None, scale=None):
    """MultiHead(Q^m, K^l, V^l) for every sequence: ``[B, Nq, d_D]`` float64."""
    hidden = np.asarray(hidden, dtype=np.float64)
    B, Nq, d_D = hidden.shape
    H, D = k_cache.shape[1], k_cache.shape[3]
    q = rows_matmul(hidden.reshape(B * Nq, d_D), wq_t)            # [B*Nq, H*D]
    q = _round(q, store).reshape(B, Nq, H, D)
    heads = OA.tree_attention(q, k_cache, v_cache, seq_lens, None, scale=scale)
    concat = _round(heads.reshape(B * Nq, H * D), store)          # Concat(hd_1..hd_h)
    return rows_matmul(concat, wo_t).reshape(B, Nq, -1)

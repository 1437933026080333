"""ctypes binding of libglide.so: argument marshalling only.

Every function here checks shapes/dtypes/devices of the torch tensors it is
given, takes their device pointers and calls the C entry point of the same
name.  No computation happens in Python and there is no fallback: if the
library is missing or a call fails, an exception is raised.
"""

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# GLIDE_LIBRARY selects another build of the same library (for instance the
# AddressSanitizer build, libglide_asan.so).
LIB_PATH = os.environ.get("GLIDE_LIBRARY") or os.path.join(_PKG, "libglide.so")

GLIDE_OK, GLIDE_EINVAL, GLIDE_ERANGE, GLIDE_EHIP, GLIDE_ESCRATCH = 0, 1, 2, 3, 4
GLIDE_BF16, GLIDE_F32 = 0, 1
MAX_NODES, MAX_SPLITS, HEAD_DIM, CAPE_MAX_K = 64, 64, 128, 7

_lib = None


class GlideError(RuntimeError):
    def __init__(self, fn, status):
        lib = load()
        msg = lib.glide_strerror(status).decode()
        if status == GLIDE_EHIP:
            msg += " (hipError %d)" % lib.glide_last_hip_error()
        super().__init__("%s failed: %s" % (fn, msg))
        self.status = status


def load():
    """Load libglide.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libglide.so is not built: run `python -m paper_2402_02082_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.glide_strerror.restype = ctypes.c_char_p
    lib.glide_strerror.argtypes = [I]
    lib.glide_last_hip_error.restype = I
    lib.glide_last_hip_error.argtypes = []
    lib.glide_tree_attn_workspace.restype = Z
    lib.glide_tree_attn_workspace.argtypes = [I, I, I, I, I, I]
    lib.glide_tree_attn.restype = I
    lib.glide_tree_attn.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, F, I, P, Z, P]
    lib.glide_tree_attn_noalloc_max_workspace.restype = Z
    lib.glide_tree_attn_noalloc_max_workspace.argtypes = []
    lib.glide_tree_attn_noalloc.restype = I
    lib.glide_tree_attn_noalloc.argtypes = [P, P, P, P, P, P, I, I, I, I, I, I, F, I, P]
    lib.cape_expand_workspace.restype = Z
    lib.cape_expand_workspace.argtypes = [I, I, I]
    lib.cape_expand.restype = I
    lib.cape_expand.argtypes = [P, I, I, I, I, I, I, P, P, P, P, Z, P]
    lib.glide_argmax_rows.restype = I
    lib.glide_argmax_rows.argtypes = [P, I, I, P, P]
    lib.tree_verify.restype = I
    lib.tree_verify.argtypes = [P, P, P, I, I, P, P, P, P]
    lib.glide_rows_matmul.restype = I
    lib.glide_rows_matmul.argtypes = [P, P, P, I, I, I, I, P]
    lib.glide_rows_weights_packed_bytes.restype = Z
    lib.glide_rows_weights_packed_bytes.argtypes = [I, I]
    lib.glide_pack_rows_weights.restype = I
    lib.glide_pack_rows_weights.argtypes = [P, P, I, I, P]
    lib.glide_rows_matmul_packed.restype = I
    lib.glide_rows_matmul_packed.argtypes = [P, P, P, I, I, I, I, P]
    lib.glide_cross_block_packed.restype = I
    lib.glide_cross_block_packed.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, F, P, Z, P]
    lib.glide_cross_block_workspace.restype = Z
    lib.glide_cross_block_workspace.argtypes = [I, I, I, I, I, I]
    lib.glide_cross_block.restype = I
    lib.glide_cross_block.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, F, P, Z, P]
    lib.glide_block_attn.restype = I
    lib.glide_block_attn.argtypes = [P, P, P, P, I, I, I, I, I, I, F, P]
    lib.spec_sample_verify.restype = I
    lib.spec_sample_verify.argtypes = [P, P, P, P, I, I, I, P, P, P]
    lib.glide_expected_speedup.restype = ctypes.c_double
    lib.glide_expected_speedup.argtypes = [ctypes.c_double, I, ctypes.c_double]
    lib.glide_verify_commit.restype = I
    lib.glide_verify_commit.argtypes = [P, I, P, P, I, I, P, P, I, I, I, I, I, P, P, P, P, P, P, P,
                                        P]
    _lib = lib
    return lib


EXPORTED = ["glide_strerror", "glide_last_hip_error", "glide_tree_attn_workspace",
            "glide_tree_attn", "glide_tree_attn_noalloc_max_workspace", "glide_tree_attn_noalloc",
            "cape_expand_workspace", "cape_expand",
            "glide_argmax_rows", "tree_verify", "glide_verify_commit", "glide_rows_matmul",
            "glide_rows_weights_packed_bytes", "glide_pack_rows_weights", "glide_rows_matmul_packed",
            "glide_cross_block_workspace", "glide_cross_block", "glide_cross_block_packed",
            "glide_block_attn",
            "spec_sample_verify",
            "glide_expected_speedup"]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def _check(fn, status):
    if status != GLIDE_OK:
        raise GlideError(fn, status)


def _need(cond, what):
    if not cond:
        raise ValueError(what)


def _dev(t, name, dtype=None):
    _need(isinstance(t, torch.Tensor), "%s must be a torch tensor" % name)
    _need(t.is_cuda, "%s must be on the GPU" % name)
    _need(t.is_contiguous(), "%s must be contiguous" % name)
    if dtype is not None:
        _need(t.dtype == dtype, "%s must be %s" % (name, dtype))


def _alloc_bytes(nbytes, device, stream=None, zero=False):
    """A byte buffer allocated on the stream that will use it.  torch's caching
    allocator ties a block to the stream current at allocation and reuses it
    for that stream's later work once freed; a buffer used on another stream
    must be allocated there, or its memory could be handed to the current
    stream's work while the kernels on `stream` still use it.  zero=True
    fills it with zeros (on that stream): attention workspaces keep arrival
    counters that must start at zero, and every call leaves them so."""
    make = torch.zeros if zero else torch.empty
    if stream is None:
        return make(nbytes, dtype=torch.uint8, device=device)
    with torch.cuda.stream(stream):
        return make(nbytes, dtype=torch.uint8, device=device)


# Bytes of the arrival-counter block at the start of every attention
# workspace (include/glide.h, glide_tree_attn_workspace): zero before the
# first call, left zero by every call.
ATTN_COUNTER_BYTES = 2048 * 128

# Workspaces, kept per (device, stream) so that calls that may run
# concurrently on different streams never share partial states.  Each is
# allocated on its stream (see _alloc_bytes), so a replaced one is only
# reused after that stream's pending work.
_ws_cache = {}


def attn_workspace(B, N, H, L_cap, max_splits, device, stream=None):
    need = load().glide_tree_attn_workspace(B, N, H, HEAD_DIM, L_cap, max_splits)
    if need == 0:
        return None
    s = torch.cuda.current_stream(device) if stream is None else stream
    key = (str(device), s.cuda_stream)
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < need:
        ws = _alloc_bytes(need, device, s, zero=True)
        _ws_cache[key] = ws
    return ws


def glide_tree_attn(q, k_cache, v_cache, seq_lens, tree_parents, out, scale=0.0,
                    max_splits=0, workspace=None, stream=None):
    """out[b, n, h] = attention of q[b, n, h] over the prefix (and, with
    tree_parents, the node's ancestor-or-self tree rows).  See include/glide.h."""
    _dev(q, "q")
    _need(q.dtype in (torch.bfloat16, torch.float32), "q must be bfloat16 or float32")
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
        _dev(t, name, q.dtype)
    _dev(seq_lens, "seq_lens", torch.int32)
    B, N, H, D = q.shape
    _need(k_cache.dim() == 4 and k_cache.shape[:2] == (B, H) and k_cache.shape[3] == D,
          "k_cache must be [B, H, L_cap, D]")
    _need(v_cache.shape == k_cache.shape, "v_cache must match k_cache")
    _need(out.shape == q.shape, "out must match q")
    _need(seq_lens.shape == (B,), "seq_lens must be [B]")
    if tree_parents is not None:
        _dev(tree_parents, "tree_parents", torch.int32)
        _need(tree_parents.shape == (B, N), "tree_parents must be [B, N]")
    L_cap = k_cache.shape[2]
    dtype = GLIDE_BF16 if q.dtype == torch.bfloat16 else GLIDE_F32
    if workspace is None:
        workspace = attn_workspace(B, N, H, L_cap, max_splits, q.device, stream)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    status = load().glide_tree_attn(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(seq_lens), _ptr(tree_parents), _ptr(out),
        B, N, H, D, L_cap, dtype, float(scale), int(max_splits), _ptr(workspace), ws_bytes,
        _stream(stream, q.device))
    _check("glide_tree_attn", status)
    return out


def glide_tree_attn_noalloc(q, k_cache, v_cache, seq_lens, tree_parents, out, scale=0.0,
                            max_splits=0, stream=None):
    """glide_tree_attn without a workspace: the split partials use the
    library's fixed per-device scratch (no allocation anywhere on this path).
    Calls that overlap on one GPU race; see include/glide.h."""
    _dev(q, "q")
    _need(q.dtype in (torch.bfloat16, torch.float32), "q must be bfloat16 or float32")
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
        _dev(t, name, q.dtype)
    _dev(seq_lens, "seq_lens", torch.int32)
    B, N, H, D = q.shape
    _need(k_cache.dim() == 4 and k_cache.shape[:2] == (B, H) and k_cache.shape[3] == D,
          "k_cache must be [B, H, L_cap, D]")
    _need(v_cache.shape == k_cache.shape, "v_cache must match k_cache")
    _need(out.shape == q.shape, "out must match q")
    _need(seq_lens.shape == (B,), "seq_lens must be [B]")
    if tree_parents is not None:
        _dev(tree_parents, "tree_parents", torch.int32)
        _need(tree_parents.shape == (B, N), "tree_parents must be [B, N]")
    status = load().glide_tree_attn_noalloc(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(seq_lens), _ptr(tree_parents), _ptr(out),
        B, N, H, D, k_cache.shape[2], GLIDE_BF16 if q.dtype == torch.bfloat16 else GLIDE_F32,
        float(scale), int(max_splits), _stream(stream, q.device))
    _check("glide_tree_attn_noalloc", status)
    return out


def cape_expand(draft_probs, k, n_max, tokens_out, parents_out, n_nodes_out, fixed=False,
                workspace=None, stream=None):
    """CaPE expansion of draft_probs [B, gamma, V] into a parent-indexed tree."""
    _dev(draft_probs, "draft_probs", torch.float32)
    B, gamma, V = draft_probs.shape
    for name, t, shape in (("tokens_out", tokens_out, (B, n_max)),
                           ("parents_out", parents_out, (B, n_max)),
                           ("n_nodes_out", n_nodes_out, (B,))):
        _dev(t, name, torch.int32)
        _need(tuple(t.shape) == shape, "%s must be %s" % (name, shape))
    need = load().cape_expand_workspace(B, gamma, V)
    if workspace is None:
        workspace = _alloc_bytes(max(need, 1), draft_probs.device, stream)
    status = load().cape_expand(
        _ptr(draft_probs), B, gamma, V, int(k), 1 if fixed else 0, int(n_max), _ptr(tokens_out),
        _ptr(parents_out), _ptr(n_nodes_out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream, draft_probs.device))
    _check("cape_expand", status)
    return tokens_out, parents_out, n_nodes_out


def glide_argmax_rows(logits, idx_out, stream=None):
    """idx_out[r] = first index of the maximum of logits[r] (logits [..., V])."""
    _dev(logits, "logits", torch.float32)
    V = logits.shape[-1]
    rows = logits.numel() // max(V, 1)
    _dev(idx_out, "idx_out", torch.int32)
    _need(idx_out.numel() == rows, "idx_out must have one entry per row")
    status = load().glide_argmax_rows(_ptr(logits), rows, V, _ptr(idx_out),
                                      _stream(stream, logits.device))
    _check("glide_argmax_rows", status)
    return idx_out


def tree_verify(target_argmax, cand_tokens, parents, accept_len, last_node=None, bonus=None,
                stream=None):
    """Greedy acceptance: accept_len[b] (and optionally last_node, bonus)."""
    _dev(cand_tokens, "cand_tokens", torch.int32)
    B, N = cand_tokens.shape
    _dev(target_argmax, "target_argmax", torch.int32)
    _need(tuple(target_argmax.shape) == (B, N + 1), "target_argmax must be [B, N + 1]")
    _dev(parents, "parents", torch.int32)
    _need(tuple(parents.shape) == (B, N), "parents must be [B, N]")
    for name, t in (("accept_len", accept_len), ("last_node", last_node), ("bonus", bonus)):
        if t is not None:
            _dev(t, name, torch.int32)
            _need(tuple(t.shape) == (B,), "%s must be [B]" % name)
    status = load().tree_verify(_ptr(target_argmax), _ptr(cand_tokens), _ptr(parents), B, N,
                                _ptr(accept_len), _ptr(last_node), _ptr(bonus),
                                _stream(stream, cand_tokens.device))
    _check("tree_verify", status)
    return accept_len


def glide_verify_commit(logits, cand_tokens, parents, k_caches, v_caches, seq_lens, seq_lens_out,
                        target_argmax, accept_len, last_node=None, bonus=None, path=None,
                        stream=None):
    """Argmax of every tree row, greedy acceptance and the commit of the
    accepted path to every layer's K/V cache (in place); see include/glide.h.
    k_caches, v_caches: sequences of per-layer [B, H, L_cap, D] tensors."""
    _dev(logits, "logits", torch.float32)
    _dev(cand_tokens, "cand_tokens", torch.int32)
    B, N = cand_tokens.shape
    _need(logits.dim() == 3 and tuple(logits.shape[:2]) == (B, N + 1),
          "logits must be [B, N + 1, V]")
    V = logits.shape[2]
    _dev(parents, "parents", torch.int32)
    _need(tuple(parents.shape) == (B, N), "parents must be [B, N]")
    for name, t, shape in (("seq_lens", seq_lens, (B,)), ("seq_lens_out", seq_lens_out, (B,)),
                           ("target_argmax", target_argmax, (B, N + 1)),
                           ("accept_len", accept_len, (B,)), ("last_node", last_node, (B,)),
                           ("bonus", bonus, (B,)), ("path", path, (B, N))):
        if t is not None or name in ("seq_lens", "seq_lens_out", "target_argmax", "accept_len"):
            _dev(t, name, torch.int32)
            _need(tuple(t.shape) == shape, "%s must be %s" % (name, shape))
    k_caches, v_caches = list(k_caches), list(v_caches)
    _need(len(k_caches) == len(v_caches), "k_caches and v_caches must have one entry per layer")
    layers = len(k_caches)
    H, L_cap, D, dtype = 1, N, HEAD_DIM, GLIDE_BF16
    if layers:
        ref = k_caches[0]
        _need(ref.dtype in (torch.bfloat16, torch.float32), "caches must be bfloat16 or float32")
        _need(ref.dim() == 4 and ref.shape[0] == B, "caches must be [B, H, L_cap, D]")
        H, L_cap, D = ref.shape[1], ref.shape[2], ref.shape[3]
        dtype = GLIDE_BF16 if ref.dtype == torch.bfloat16 else GLIDE_F32
        for i, t in enumerate(k_caches + v_caches):
            _dev(t, "cache %d" % i, ref.dtype)
            _need(t.shape == ref.shape, "every cache must be [B, H, L_cap, D] like the first")
    kp = (ctypes.c_void_p * max(layers, 1))(*[t.data_ptr() for t in k_caches])
    vp = (ctypes.c_void_p * max(layers, 1))(*[t.data_ptr() for t in v_caches])
    status = load().glide_verify_commit(
        _ptr(logits), V, _ptr(cand_tokens), _ptr(parents), B, N, kp, vp, layers, H, D, L_cap,
        dtype, _ptr(seq_lens), _ptr(seq_lens_out), _ptr(target_argmax), _ptr(accept_len),
        _ptr(last_node), _ptr(bonus), _ptr(path), _stream(stream, logits.device))
    _check("glide_verify_commit", status)
    return accept_len


def glide_rows_matmul(a, w_t, out, stream=None):
    """out[m, n] = sum_k a[m, k] * w_t[n, k]; a [M, K], w_t [N, K] bfloat16,
    out [M, N] bfloat16 or float32."""
    _dev(a, "a", torch.bfloat16)
    _dev(w_t, "w_t", torch.bfloat16)
    _need(a.dim() == 2 and w_t.dim() == 2 and a.shape[1] == w_t.shape[1],
          "a must be [M, K] and w_t [N, K]")
    M, K = a.shape
    N = w_t.shape[0]
    _need(out.dtype in (torch.bfloat16, torch.float32), "out must be bfloat16 or float32")
    _dev(out, "out")
    _need(tuple(out.shape) == (M, N), "out must be [M, N]")
    status = load().glide_rows_matmul(_ptr(a), _ptr(w_t), _ptr(out), M, K, N,
                                      GLIDE_BF16 if out.dtype == torch.bfloat16 else GLIDE_F32,
                                      _stream(stream, a.device))
    _check("glide_rows_matmul", status)
    return out


def rows_weights_packed_bytes(K, N):
    return load().glide_rows_weights_packed_bytes(K, N)


def pack_rows_weights(w_t, out=None, stream=None):
    """The packed copy of w_t [N, K] bfloat16 for the *_packed calls (a flat
    bfloat16 tensor; see include/glide.h for the layout)."""
    _dev(w_t, "w_t", torch.bfloat16)
    _need(w_t.dim() == 2, "w_t must be [N, K]")
    N, K = w_t.shape
    need = rows_weights_packed_bytes(K, N)
    _need(need > 0, "unsupported projection sizes")
    if out is None:
        out = _alloc_bytes(need, w_t.device, stream).view(torch.bfloat16)
    _dev(out, "out", torch.bfloat16)
    _need(out.numel() * 2 >= need, "out is smaller than the packed copy")
    status = load().glide_pack_rows_weights(_ptr(w_t), _ptr(out), K, N, _stream(stream, w_t.device))
    _check("glide_pack_rows_weights", status)
    return out


def glide_rows_matmul_packed(a, w_packed, out, stream=None):
    """glide_rows_matmul with the packed copy of w_t; N is out.shape[1]."""
    _dev(a, "a", torch.bfloat16)
    _dev(w_packed, "w_packed", torch.bfloat16)
    _need(a.dim() == 2 and out.dim() == 2 and out.shape[0] == a.shape[0], "a must be [M, K], out [M, N]")
    M, K = a.shape
    N = out.shape[1]
    _need(out.dtype in (torch.bfloat16, torch.float32), "out must be bfloat16 or float32")
    _dev(out, "out")
    _need(w_packed.numel() * 2 >= rows_weights_packed_bytes(K, N) > 0, "w_packed does not fit [N, K]")
    status = load().glide_rows_matmul_packed(_ptr(a), _ptr(w_packed), _ptr(out), M, K, N,
                                             GLIDE_BF16 if out.dtype == torch.bfloat16 else GLIDE_F32,
                                             _stream(stream, a.device))
    _check("glide_rows_matmul_packed", status)
    return out


def cross_block_workspace(B, Nq, d_D, H, L_cap, device, stream=None):
    need = load().glide_cross_block_workspace(B, Nq, d_D, H, HEAD_DIM, L_cap)
    _need(need > 0, "unsupported cross-attention block sizes")
    return _alloc_bytes(need, device, stream, zero=True)


def glide_cross_block(hidden, wq_t, k_cache, v_cache, seq_lens, wo_t, out, scale=0.0,
                      workspace=None, stream=None):
    """The GliDe cross-attention sub-layer: hidden [B, Nq, d_D] -> out [B, Nq, d_D]
    through the query projection, cross attention over the cache and the
    output projection (bfloat16).  See include/glide.h."""
    for name, t in (("hidden", hidden), ("wq_t", wq_t), ("k_cache", k_cache),
                    ("v_cache", v_cache), ("wo_t", wo_t), ("out", out)):
        _dev(t, name, torch.bfloat16)
    _dev(seq_lens, "seq_lens", torch.int32)
    B, Nq, d_D = hidden.shape
    _need(k_cache.dim() == 4 and k_cache.shape[0] == B, "k_cache must be [B, H, L_cap, D]")
    _need(v_cache.shape == k_cache.shape, "v_cache must match k_cache")
    H, L_cap, D = k_cache.shape[1], k_cache.shape[2], k_cache.shape[3]
    _need(tuple(wq_t.shape) == (H * D, d_D), "wq_t must be [H*D, d_D]")
    _need(tuple(wo_t.shape) == (d_D, H * D), "wo_t must be [d_D, H*D]")
    _need(tuple(out.shape) == (B, Nq, d_D), "out must be [B, Nq, d_D]")
    _need(seq_lens.shape == (B,), "seq_lens must be [B]")
    if workspace is None:
        workspace = cross_block_workspace(B, Nq, d_D, H, L_cap, hidden.device, stream)
    status = load().glide_cross_block(
        _ptr(hidden), _ptr(wq_t), _ptr(k_cache), _ptr(v_cache), _ptr(seq_lens), _ptr(wo_t),
        _ptr(out), B, Nq, d_D, H, D, L_cap, float(scale), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream, hidden.device))
    _check("glide_cross_block", status)
    return out


def glide_cross_block_packed(hidden, wq_packed, k_cache, v_cache, seq_lens, wo_packed, out, scale=0.0,
                             workspace=None, stream=None):
    """glide_cross_block with both projections' weights packed
    (pack_rows_weights of wq_t and of wo_t)."""
    for name, t in (("hidden", hidden), ("wq_packed", wq_packed), ("k_cache", k_cache),
                    ("v_cache", v_cache), ("wo_packed", wo_packed), ("out", out)):
        _dev(t, name, torch.bfloat16)
    _dev(seq_lens, "seq_lens", torch.int32)
    B, Nq, d_D = hidden.shape
    _need(k_cache.dim() == 4 and k_cache.shape[0] == B, "k_cache must be [B, H, L_cap, D]")
    _need(v_cache.shape == k_cache.shape, "v_cache must match k_cache")
    H, L_cap, D = k_cache.shape[1], k_cache.shape[2], k_cache.shape[3]
    _need(wq_packed.numel() * 2 >= rows_weights_packed_bytes(d_D, H * D) > 0,
          "wq_packed does not fit [H*D, d_D]")
    _need(wo_packed.numel() * 2 >= rows_weights_packed_bytes(H * D, d_D) > 0,
          "wo_packed does not fit [d_D, H*D]")
    _need(tuple(out.shape) == (B, Nq, d_D), "out must be [B, Nq, d_D]")
    _need(seq_lens.shape == (B,), "seq_lens must be [B]")
    if workspace is None:
        workspace = cross_block_workspace(B, Nq, d_D, H, L_cap, hidden.device, stream)
    status = load().glide_cross_block_packed(
        _ptr(hidden), _ptr(wq_packed), _ptr(k_cache), _ptr(v_cache), _ptr(seq_lens), _ptr(wo_packed),
        _ptr(out), B, Nq, d_D, H, D, L_cap, float(scale), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream, hidden.device))
    _check("glide_cross_block_packed", status)
    return out


def spec_sample_verify(draft_tokens, draft_probs, target_probs, uniforms, accept_len, next_token,
                       stream=None):
    """Speculative-sampling verification of draft chains; see include/glide.h."""
    _dev(draft_tokens, "draft_tokens", torch.int32)
    B, gamma = draft_tokens.shape
    _dev(draft_probs, "draft_probs", torch.float32)
    _need(draft_probs.dim() == 3 and tuple(draft_probs.shape[:2]) == (B, gamma),
          "draft_probs must be [B, gamma, V]")
    V = draft_probs.shape[2]
    _dev(target_probs, "target_probs", torch.float32)
    _need(tuple(target_probs.shape) == (B, gamma + 1, V), "target_probs must be [B, gamma + 1, V]")
    _dev(uniforms, "uniforms", torch.float32)
    _need(tuple(uniforms.shape) == (B, gamma + 1), "uniforms must be [B, gamma + 1]")
    for name, t in (("accept_len", accept_len), ("next_token", next_token)):
        _dev(t, name, torch.int32)
        _need(tuple(t.shape) == (B,), "%s must be [B]" % name)
    status = load().spec_sample_verify(_ptr(draft_tokens), _ptr(draft_probs), _ptr(target_probs),
                                       _ptr(uniforms), B, gamma, V, _ptr(accept_len),
                                       _ptr(next_token), _stream(stream, draft_tokens.device))
    _check("spec_sample_verify", status)
    return accept_len, next_token


def glide_expected_speedup(alpha, gamma, c):
    """E(Spd) = (1 - alpha^(gamma+1)) / ((1 - alpha)(gamma c + 1))."""
    return load().glide_expected_speedup(float(alpha), int(gamma), float(c))


def glide_block_attn(q, k_cache, v_cache, out, block, scale=0.0, stream=None):
    """Block-masked training cross attention: q [B, T, H, D] over the cache's
    positions [0, block * floor(p / block)); bfloat16.  See include/glide.h."""
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
        _dev(t, name, torch.bfloat16)
    B, T, H, D = q.shape
    _need(k_cache.dim() == 4 and k_cache.shape[:2] == (B, H) and k_cache.shape[3] == D,
          "k_cache must be [B, H, L_cap, D]")
    _need(v_cache.shape == k_cache.shape, "v_cache must match k_cache")
    _need(out.shape == q.shape, "out must match q")
    status = load().glide_block_attn(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(out), B, T, H, D,
                                     k_cache.shape[2], int(block), float(scale),
                                     _stream(stream, q.device))
    _check("glide_block_attn", status)
    return out

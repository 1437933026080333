"""GliDe + CaPE decoding hot path for MI355X (gfx950).

Thin Python face of libglide.so (HIP kernels behind a C ABI, declared in
include/glide.h).  Functions carry the C names:

    glide_tree_attn   tree-masked / cross attention against a KV cache
    glide_tree_attn_noalloc  the same with the split partials in the
                      library's fixed scratch (for callers that cannot allocate)
    cape_expand       confidence-aware proposal expansion into a tree
    glide_argmax_rows the target's greedy token per logits row
    tree_verify       greedy longest-accepted-path selection
    glide_verify_commit  argmax, acceptance and the KV cache commit of the
                      accepted path in every layer
    glide_cross_block the GliDe cross-attention sub-layer (query projection,
                      cross attention, output projection)
    glide_rows_matmul its few-row projection
    pack_rows_weights, glide_rows_matmul_packed, glide_cross_block_packed
                      the same with weights packed once per 16-row operand tile
    glide_block_attn  the block-masked cross attention of draft training
    spec_sample_verify  chain verification with speculative sampling
    glide_expected_speedup  the expected-speedup model

PyTorch only provides device memory and streams.
"""

from ._lib import (  # noqa: F401
    ATTN_COUNTER_BYTES, CAPE_MAX_K, GLIDE_BF16, GLIDE_EHIP, GLIDE_EINVAL, GLIDE_ERANGE, GLIDE_ESCRATCH, GLIDE_F32,
    GLIDE_OK,
    HEAD_DIM, MAX_NODES, MAX_SPLITS, GlideError, attn_workspace, cape_expand,
    cross_block_workspace, glide_argmax_rows, glide_block_attn, glide_cross_block,
    glide_cross_block_packed, glide_rows_matmul, glide_rows_matmul_packed, pack_rows_weights,
    rows_weights_packed_bytes,
    glide_expected_speedup, glide_tree_attn, glide_tree_attn_noalloc, glide_verify_commit, load,
    spec_sample_verify,
    tree_verify,
)

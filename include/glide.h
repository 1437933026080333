/*
 * glide.h -- C ABI of the GliDe + CaPE decoding hot path for MI355X (gfx950).
 *
 * Operations (arXiv 2402.02082, "GliDe with a CaPE"):
 *   glide_tree_attn    softmax attention of a few query rows against a long
 *                      KV cache, either under the CaPE tree mask (target
 *                      verification, Sec. 4.2 "Verification of Expanded
 *                      Proposals", mask_CaPE equation) or unmasked (GliDe
 *                      cross-attention into the target cache, Sec. 4.1,
 *                      MultiHead / hd_j equations).
 *   cape_expand        confidence-aware proposal expansion and linearisation
 *                      into a parent-indexed tree (Sec. 4.2 "Proposal
 *                      Expansion", S(p) table).
 *   glide_argmax_rows  the target's greedy token per logits row (Sec. 3,
 *                      greedy "speculative decoding" acceptance).
 *   tree_verify        greedy longest-accepted-path selection (Sec. 3;
 *                      Sec. 5.1 "Experiment design": greedy acceptance for
 *                      the CaPE experiments).
 *   glide_verify_commit  argmax, acceptance and the KV cache commit of the
 *                      accepted path in every layer (Sec. 3; Sec. 4.1, the
 *                      cache kept after a verification step).
 *   spec_sample_verify chain verification with speculative sampling (Sec. 3;
 *                      Sec. 5.1, the GliDe-only experiments), and
 *                      glide_expected_speedup, the expected-speedup model
 *                      (Sec. 5.1, Metrics).
 *   glide_block_attn   the block-wise masked cross attention of draft
 *                      training (Sec. 4.1, "Block-wise Attention Mask").
 *   glide_cross_block  the GliDe cross-attention sub-layer with its query
 *                      and output projections (Sec. 4.1, Q^{m,j} and
 *                      MultiHead equations); glide_rows_matmul is its
 *                      few-row projection.
 *
 * Conventions shared by every call:
 *   - All array arguments are DEVICE pointers to memory the caller owns and
 *     allocated; the library never allocates or frees memory on these paths
 *     and never keeps a pointer after the call returns.
 *   - Work is enqueued on `stream` (NULL = the default stream) and the call
 *     returns without synchronising.  Outputs are valid once the stream
 *     reaches that point.
 *   - Every scalar/pointer argument is checked on the host BEFORE any HIP
 *     call; a bad argument returns GLIDE_EINVAL and touches nothing.  Device
 *     data (sequence lengths, parent arrays) is trusted unless the environment
 *     variable GLIDE_VALIDATE=1 is set, in which case it is copied to the host
 *     (synchronising the stream) and checked, returning GLIDE_ERANGE when out
 *     of range.  Unvalidated out-of-range data never causes an out-of-bounds
 *     access: lengths are clamped and bad parents are treated as roots.
 *   - A failed kernel launch returns GLIDE_EHIP; glide_last_hip_error() gives
 *     the HIP error code of the calling thread's last failure.
 *   - int32 tree arrays: node index = position in the linearised proposal;
 *     parents[n] in [-1, n) (-1 = child of the accepted prefix).
 */
#ifndef GLIDE_H
#define GLIDE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define GLIDE_OK      0
#define GLIDE_EINVAL  1   /* bad pointer, size, dtype or option */
#define GLIDE_ERANGE  2   /* device data out of range (GLIDE_VALIDATE=1 only) */
#define GLIDE_EHIP    3   /* a HIP call or kernel launch failed */
#define GLIDE_ESCRATCH 4  /* sizes need more than glide_tree_attn_noalloc's
                             fixed scratch holds */

/* Element types of q / k_cache / v_cache / out. */
#define GLIDE_BF16    0   /* bfloat16 in and out, float32 accumulation */
#define GLIDE_F32     1   /* float32 in and out, float32 accumulation */

#define GLIDE_MAX_NODES   64   /* tree nodes / query rows per sequence */
#define GLIDE_MAX_SPLITS  64   /* key-range splits per (sequence, head) */
#define GLIDE_HEAD_DIM    128  /* the only head dimension supported */
#define GLIDE_CAPE_MAX_K  7    /* largest expansion set, max of S(p) */

/* Human-readable name of a status code (static storage, never NULL). */
const char* glide_strerror(int status);

/* HIP error code (hipError_t as int) of the calling thread's last
 * GLIDE_EHIP, or 0. */
int glide_last_hip_error(void);

/*
 * Workspace bytes glide_tree_attn needs for these sizes (0 when the call runs
 * without a workspace, i.e. with one split).  Arguments as glide_tree_attn.
 * The workspace starts with a fixed 256 KiB block of arrival counters (one per
 * head, 128 bytes apart, with the flags of the merge below), followed by the
 * per-split partial softmax states (running max, running sum and the float32
 * output of every query row) and, for a single sequence of N >= 8 rows, the
 * same rows in fp16: such bf16 calls exchange each split's normalised output
 * in fp16, and in float32 only for the pieces whose values exceed fp16's
 * range.
 * For a single sequence (B == 1, H <= 2048, 1..16 bf16 rows or any float32
 * rows) the workgroup of a split counts itself in once its states are
 * written, and the one that completes a head merges them, so the call is a
 * single launch; other calls merge in a second launch and leave the counters
 * alone.  The counter block must be zero before the workspace's first use
 * (zero-fill the whole buffer once); every call leaves it zero, and the
 * partial states need no initialisation, so one buffer of the largest size
 * needed can serve calls of any shape in turn.  It must not be shared by
 * calls that can run concurrently.  Returns 0 for invalid sizes.
 */
size_t glide_tree_attn_workspace(int B, int N, int H, int D, int L_cap,
                                 int max_splits);

/*
 * glide_tree_attn -- one attention layer of the verification pass (tree mode)
 * or the GliDe cross-attention (cross mode).
 *
 * Sec. 4.1: hd_j = SoftMax(Q K^T / sqrt(d_k)) V per head j.
 * Tree mode (tree_parents != NULL): query row n of sequence b sees cache rows
 *   [0, seq_lens[b]) (the accepted prefix) and the rows seq_lens[b] + m of
 *   every tree node m that is node n or one of its ancestors -- the
 *   ancestor-or-self relation that mask_CaPE (Sec. 4.2) defines for a
 *   linearised expanded proposal.  The caller has written the tree nodes'
 *   keys/values at cache rows [seq_lens[b], seq_lens[b] + N).
 * Cross mode (tree_parents == NULL): every query row sees rows
 *   [0, seq_lens[b]) and nothing else (Sec. 4.1: the draft's queries attend
 *   the target cache up to position t-1; no mask at inference).
 *
 *   q            [B, N, H, D]  dtype; query rows (post-RoPE, unscaled).
 *   k_cache      [B, H, L_cap, D] dtype, contiguous.
 *   v_cache      [B, H, L_cap, D] dtype, contiguous.
 *   seq_lens     [B] int32: prefix length L_b.  Clamped to [0, L_cap - N]
 *                (tree) or [0, L_cap] (cross).
 *   tree_parents [B, N] int32 or NULL (cross mode).
 *   out          [B, N, H, D]  dtype; may not alias the inputs.  Rows of a
 *                sequence with no visible key (cross mode, L_b = 0) are 0.
 *   1 <= B <= 65535; 1 <= N <= 64; H >= 1; B * N * H < 2^31; D == 128;
 *   N (tree) or 1 <= L_cap <= 4194304 (2^22).
 *   dtype        GLIDE_BF16 or GLIDE_F32.
 *   scale        softmax scale; <= 0 selects 1/sqrt(D).
 *   max_splits   0 = choose automatically, else 1..64 key-range splits.
 *   workspace    device buffer of >= glide_tree_attn_workspace(...) bytes;
 *                may be NULL when that size is 0.
 * Precision: scores, softmax sums and outputs accumulate in float32; with
 * bf16 inputs the probabilities enter the PV product rounded to bf16, and
 * a single-sequence call of 8 or more rows with several splits exchanges
 * each split's normalised output in fp16 (at most 2^-11 of its size off;
 * float32 when out of fp16's range).  The output is rounded to dtype once.
 */
int glide_tree_attn(const void* q, const void* k_cache, const void* v_cache,
                    const int32_t* seq_lens, const int32_t* tree_parents,
                    void* out, int B, int N, int H, int D, int L_cap,
                    int dtype, float scale, int max_splits,
                    void* workspace, size_t ws_bytes, hipStream_t stream);

/*
 * glide_tree_attn_noalloc -- glide_tree_attn for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, same kernels and the
 * same results as glide_tree_attn with max_splits alike, but no workspace
 * argument: the arrival counters and split partial states live in a fixed
 * scratch array of glide_tree_attn_noalloc_max_workspace() bytes (16 MiB)
 * that the library holds on every GPU it runs on until the process ends.
 * The call allocates nothing and records no memset: the array starts zeroed
 * when the library is loaded, every call leaves its counters zero, and the
 * partials are written before they are read.  Sizes whose split plan needs
 * more than the scratch holds (glide_tree_attn_workspace(...) > the maximum)
 * return GLIDE_ESCRATCH before any HIP call; sizes that need no workspace
 * never touch it.
 * The first call on a device, with that device current, looks up the
 * scratch array's device address (hipGetSymbolAddress).
 * Every call on one GPU shares that GPU's scratch: calls that can overlap on
 * one GPU (other streams, other host threads) race and must not be issued.
 */
size_t glide_tree_attn_noalloc_max_workspace(void);
int glide_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache,
                            const int32_t* seq_lens, const int32_t* tree_parents,
                            void* out, int B, int N, int H, int D, int L_cap,
                            int dtype, float scale, int max_splits,
                            hipStream_t stream);

/* Workspace bytes cape_expand needs (the best candidates of every 4096-token
 * part of every draft row); 0 for invalid sizes (as cape_expand rejects). */
size_t cape_expand_workspace(int B, int gamma, int V);

/*
 * cape_expand -- confidence-aware proposal expansion (Sec. 4.2).
 *
 * For each sequence b and position i < gamma, with row p = draft_probs[b, i]:
 *   x_i = the most probable token (ties: lower id), p_i = its probability;
 *   K_i = S(p_i) = 7, 5, 3, 1 for p_i in (0,0.3], (0.3,0.6], (0.6,0.8],
 *         (0.8,1] (float32 edges, upper bounds inclusive), capped by k when
 *         k > 0; with fixed != 0, K_i = k for every i (the fixed-size
 *         ablation, Sec. 5.4); always K_i <= V - 1;
 *   X_i = the K_i most probable tokens other than x_i (ties: lower id).
 * Tree: node i < gamma is x_i with parent i - 1; the leaves of X_0, X_1, ...
 * follow in position order, rank order within a position, each with the
 * parent of its position's proposal token.  If gamma + sum K_i > n_max (the
 * verification budget, Sec. 5.3), the n_max - gamma leaves kept are the first
 * in the order (prob desc, position asc, rank asc).  Unused slots are
 * (token -1, parent -1).
 *
 *   draft_probs [B, gamma, V] float32, finite (no NaN).
 *   tokens_out, parents_out [B, n_max] int32; n_nodes_out [B] int32.
 *   B >= 1; 1 <= gamma <= n_max <= 64; B * gamma <= 65535; V >= 2;
 *   0 <= k (<= 7 when fixed).
 *   workspace >= cape_expand_workspace(B, gamma, V) bytes (no zero-fill needed).
 */
int cape_expand(const float* draft_probs, int B, int gamma, int V, int k,
                int fixed, int n_max, int32_t* tokens_out,
                int32_t* parents_out, int32_t* n_nodes_out,
                void* workspace, size_t ws_bytes, hipStream_t stream);

/*
 * glide_argmax_rows -- idx_out[r] = argmax_v logits[r, v], ties to the lower
 * index (Sec. 3: greedy acceptance compares against the target's greedy
 * token).  -0.0 and +0.0 compare equal; NaN is not allowed.
 *   logits [rows, V] float32 row-major; idx_out [rows] int32.
 *   rows >= 1; V >= 1.
 */
int glide_argmax_rows(const float* logits, int rows, int V, int32_t* idx_out,
                      hipStream_t stream);

/*
 * tree_verify -- greedy acceptance of a candidate tree (Sec. 3, Sec. 4.2).
 *
 * Node c is accepted when its parent is accepted (or c is a root) and
 * cand_tokens[c] == target_argmax[parents[c] + 1].  accept_len = the depth
 * of the deepest accepted node (0 if none); last_node = that node (lowest
 * index among equals; -1 if none); bonus = target_argmax[last_node + 1], the
 * free token the target contributes.
 *
 *   target_argmax [B, N + 1] int32: slot 0 = the target's greedy token after
 *                 the prefix, slot n + 1 = after tree node n.
 *   cand_tokens   [B, N] int32 (padding nodes carry -1 and never match).
 *   parents       [B, N] int32.
 *   accept_len    [B] int32 out;  last_node, bonus [B] int32 out, nullable.
 *   B >= 1; 1 <= N <= 64.
 */
int tree_verify(const int32_t* target_argmax, const int32_t* cand_tokens,
                const int32_t* parents, int B, int N, int32_t* accept_len,
                int32_t* last_node, int32_t* bonus, hipStream_t stream);

/*
 * glide_verify_commit -- the verification epilogue: the target's greedy
 * token per tree row, greedy acceptance of the tree, and the commit of the
 * accepted path to the KV cache (Sec. 3: the accepted proposal tokens plus
 * one target token extend the prefix; Sec. 4.1: after a verification step
 * only the accepted tokens' cache rows are kept; Sec. 4.2: a tree candidate
 * is accepted when its whole root path is).
 *
 * With L = seq_lens[b] clamped into [0, L_cap - N] and the accepted node's
 * root path n_1, ..., n_a (depths 1..a), every layer's K and V row L + n_d
 * moves to row L + d - 1; other rows are left as they are.
 * seq_lens_out[b] = L + a, with the same clamped L (so an out-of-range length
 * that GLIDE_VALIDATE would reject still gives a length that matches the rows
 * committed).  With layers == 0 there is no cache: L_cap is not used,
 * seq_lens[b] is taken as given (no clamp, no validation) and
 * seq_lens_out[b] = seq_lens[b] + a.
 *
 *   logits        [B, N + 1, V] float32: row 0 = the target's logits after
 *                 the prefix, row n + 1 = after tree node n.
 *   cand_tokens   [B, N] int32 (padding nodes carry -1 and never match).
 *   parents       [B, N] int32.
 *   k_caches, v_caches  HOST arrays of `layers` DEVICE pointers, each a
 *                 [B, H, L_cap, D] cache of `dtype` holding node m's key /
 *                 value at row L + m (the layout glide_tree_attn reads);
 *                 updated in place.  0 <= layers <= 128 (0: no commit).
 *   seq_lens      [B] int32 in; seq_lens_out [B] int32 out (must not be
 *                 seq_lens: the launch still reads the old lengths).
 *   target_argmax [B, N + 1] int32 out (as glide_argmax_rows).
 *   accept_len    [B] int32 out; last_node, bonus [B] and path [B, N]
 *                 (accepted node at depth d + 1 in slot d, -1 after) int32
 *                 out, nullable.
 *   B <= 65535; 1 <= N <= 64; B * N * H < 2^31; D == 128;
 *   N <= L_cap <= 4194304; seq_lens[b] + N <= L_cap when layers > 0
 *   (clamped into range unless GLIDE_VALIDATE=1).
 * Two launches (the argmax, then the acceptance and copy); no workspace.
 */
int glide_verify_commit(const float* logits, int V, const int32_t* cand_tokens,
                        const int32_t* parents, int B, int N, void* const* k_caches,
                        void* const* v_caches, int layers, int H, int D, int L_cap,
                        int dtype, const int32_t* seq_lens, int32_t* seq_lens_out,
                        int32_t* target_argmax, int32_t* accept_len, int32_t* last_node,
                        int32_t* bonus, int32_t* path, hipStream_t stream);

/*
 * glide_rows_matmul -- out[m, n] = sum_k a[m, k] * w_t[n, k], the projection
 * of a few activation rows by a weight matrix stored one row per output
 * feature (Sec. 4.1: Q^{m,j} = H^m W_j for every head j, and
 * Concat(hd_1..hd_h) W^O; w_t is the transpose of the paper's W).
 *   a   [M, K] bfloat16, 16-byte aligned;  w_t [N, K] bfloat16, 16-byte
 *       aligned;  out [M, N] of out_dtype (GLIDE_BF16 rounds to nearest
 *       even, GLIDE_F32 keeps the float32 accumulation).
 *   M >= 1 (128 rows per launch, more rows take further launches, each
 *   reading w_t again); 8 <= K <= 2^20 with K % 8 == 0; N >= 1.
 */
int glide_rows_matmul(const void* a, const void* w_t, void* out, int M, int K, int N,
                      int out_dtype, hipStream_t stream);

/*
 * Packed weights for the projections (the same operation as
 * glide_rows_matmul, Sec. 4.1).  From a row-major w_t every load of the
 * projection fetches 64 bytes from each of 16 rows K * 2 bytes apart; the
 * packed copy stores each (16-row tile, 32-wide K step) operand as one
 * contiguous 1 KB block in the order the matrix cores take it: block
 * (t, j) at byte (t * ceil(K / 32) + j) * 1024, its 16-byte unit l holding
 * w_t[16t + l % 16][32j + 8 * (l / 16) .. + 7] (zeros past N or K).  Pack
 * once (weights are static) and pass the copy to the *_packed calls; the
 * results are bit-identical to the row-major calls.
 *
 * glide_rows_weights_packed_bytes -- bytes of the packed copy of a [N, K]
 *   matrix, ceil(N / 16) * ceil(K / 32) * 1024; 0 for sizes
 *   glide_rows_matmul rejects.  Host only.
 * glide_pack_rows_weights -- writes the packed copy of w_t [N, K] bfloat16
 *   (16-byte aligned) into w_packed (that many bytes, 16-byte aligned,
 *   caller-allocated, not overlapping w_t).
 * glide_rows_matmul_packed -- glide_rows_matmul with w_packed, the packed
 *   copy of w_t for the same K and N.
 */
size_t glide_rows_weights_packed_bytes(int K, int N);
int glide_pack_rows_weights(const void* w_t, void* w_packed, int K, int N, hipStream_t stream);
int glide_rows_matmul_packed(const void* a, const void* w_packed, void* out, int M, int K, int N,
                             int out_dtype, hipStream_t stream);

/*
 * glide_cross_block -- MultiHead(Q^m, K^l, V^l) = Concat(hd_1..hd_h) W^O with
 * hd_j = SoftMax(Q^{m,j} (K^{l,j})^T / sqrt(d_k)) V^{l,j} and Q^{m,j} = H^m W_j
 * (Sec. 4.1): the draft's hidden rows projected into one query per target
 * head, attended over the target layer's cache (rows [0, seq_lens[b]), as
 * glide_tree_attn in cross mode) and projected back.  bfloat16 throughout;
 * the projected queries and the concatenated heads are stored in bfloat16
 * in the workspace between the three launches.
 *   hidden [B, Nq, d_D];  wq_t [H*D, d_D] (row j*D + c = column c of W_j);
 *   k_cache, v_cache [B, H, L_cap, D];  seq_lens [B] int32;
 *   wo_t [d_D, H*D] (the transpose of W^O);  out [B, Nq, d_D].
 *   D == 128; 1 <= Nq <= 64; d_D % 8 == 0; scale <= 0 means 1/sqrt(D);
 *   workspace of glide_cross_block_workspace() bytes, 16-byte aligned (0 for
 *   invalid sizes); it begins with the attention's workspace, so its first
 *   256 KiB must be zero before its first use, and every call leaves them so
 *   (see glide_tree_attn_workspace).
 */
size_t glide_cross_block_workspace(int B, int Nq, int d_D, int H, int D, int L_cap);
int glide_cross_block(const void* hidden, const void* wq_t, const void* k_cache,
                      const void* v_cache, const int32_t* seq_lens, const void* wo_t, void* out,
                      int B, int Nq, int d_D, int H, int D, int L_cap, float scale,
                      void* workspace, size_t ws_bytes, hipStream_t stream);

/*
 * glide_cross_block_packed -- glide_cross_block with the two projections'
 * weights in packed form: wq_packed the packed copy of wq_t (K = d_D,
 * N = H*D) and wo_packed that of wo_t (K = H*D, N = d_D), as written by
 * glide_pack_rows_weights.  Same workspace, results bit-identical.
 */
int glide_cross_block_packed(const void* hidden, const void* wq_packed, const void* k_cache,
                             const void* v_cache, const int32_t* seq_lens, const void* wo_packed,
                             void* out, int B, int Nq, int d_D, int H, int D, int L_cap, float scale,
                             void* workspace, size_t ws_bytes, hipStream_t stream);

/*
 * spec_sample_verify -- verification of a gamma-token draft chain with
 * speculative sampling (Sec. 3: the accepted tokens plus one target token
 * extend the prefix, and the emitted tokens follow the target's sampling
 * distribution; Sec. 5.1: gamma = 5 chains in the GliDe-only experiments).
 * Token x_i is accepted when uniforms[b, i-1] * p_D(x_i) < p_T(x_i) (float32);
 * at the first rejection, at row j, next_token is drawn from max(0, p_T_j -
 * p_D_j); if all are accepted it is drawn from p_T row gamma.  Draws use
 * uniforms[b, gamma] by inverse CDF over the fixed-point weights
 * floor(p * 2^32): with W their sum, the token is the first whose running
 * weight exceeds floor(u * W) (a residual of weight 0 falls back to the
 * target row; a target row of weight 0 gives token 0).
 *   draft_tokens [B, gamma] int32 in [0, V) (clamped);  draft_probs
 *   [B, gamma, V] and target_probs [B, gamma + 1, V] float32 (row i of the
 *   target follows draft token i; row 0 follows the prefix);  uniforms
 *   [B, gamma + 1] float32 in [0, 1);  accept_len, next_token [B] int32 out.
 *   1 <= gamma <= 64; 1 <= V <= 2^20.
 */
int spec_sample_verify(const int32_t* draft_tokens, const float* draft_probs,
                       const float* target_probs, const float* uniforms, int B, int gamma,
                       int V, int32_t* accept_len, int32_t* next_token, hipStream_t stream);

/*
 * glide_block_attn -- the cross attention of draft training under the
 * block-wise mask (Sec. 4.1, "Block-wise Attention Mask"): with positions cut
 * into blocks of `block` tokens, the query at position p attends to the
 * target's keys and values of the positions k with block(p) > block(k),
 * i.e. [0, block * floor(p / block)); a query of the first block sees none
 * and gets zeros.  bfloat16 in and out, float32 accumulation.
 *   q   [B, T, H, D] (the draft's projected queries of a training sequence);
 *   k_cache, v_cache [B, H, L_cap, D] holding positions 0 .. T - 1;
 *   out [B, T, H, D].  D == 128; 1 <= T <= L_cap <= 4194304; block >= 1;
 *   B <= 65535; B * H * ceil(T / 64) < 2^31;
 *   scale <= 0 means 1/sqrt(D).
 */
int glide_block_attn(const void* q, const void* k_cache, const void* v_cache, void* out, int B,
                     int T, int H, int D, int L_cap, int block, float scale, hipStream_t stream);

/*
 * glide_expected_speedup -- E(Spd) = (1 - alpha^(gamma+1)) /
 * ((1 - alpha)(gamma c + 1)) for acceptance rate alpha in [0, 1], proposal
 * length gamma >= 1 and cost coefficient c >= 0 (Sec. 5.1, Metrics); NaN
 * for arguments outside those ranges.  Host function, no GPU work.
 */
double glide_expected_speedup(double alpha, int gamma, double c);

#ifdef __cplusplus
}
#endif

#endif /* GLIDE_H */

/*
 * treeflash.h -- C ABI of the TreeFlash drafting library for AMD MI355X (gfx950).
 *
 * TreeFlash (arXiv 2606.03819) drafts a speculative-decoding tree from a
 * one-shot block drafter in two stages (Appendix B, "AR-approximated OPT-Tree
 * Construction"):
 *
 *   Part 1 (treeflash_marginal_topk + treeflash_arapprox_expand)
 *     stage 1: q_{t+i} = LMHead(h_{t+i}) for every draft depth i, top-M ids;
 *     stage 2: for depth 1 (conditioned on the root token x_t) and for every
 *              (depth i >= 2, candidate m of depth i-1) pair, Eq. 1
 *                h' = h_i + SwiGLU( rms(h_i) :: rms(Embd(prev)) )
 *              then the LM head, a log-softmax and the best entries per row.
 *   Part 2 (treeflash_build_tree)
 *     best-first (OPT-Tree) selection of B nodes by path probability; a node
 *     is expanded only when its token is one of the M candidates of its depth.
 *
 * Conventions shared by every call
 *   - Every tensor pointer is a DEVICE pointer to a dense row-major array owned
 *     by the caller; the library never allocates, frees or keeps a pointer
 *     after the call returns.  h, h', lm_head, w_gate, w_up, w_down and the
 *     workspace must be 16-byte aligned (they are read with 16-byte loads);
 *     every other array needs 4-byte alignment.
 *   - Calls are asynchronous and ordered on `stream` (0 = the null stream).
 *     They never synchronise the device.  Arguments are validated before any
 *     HIP call; an invalid argument returns an error and launches nothing.
 *     After launching, the library checks hipGetLastError and maps a failure
 *     to TF_ERR_HIP.  Nothing is thrown or aborted across the ABI.
 *   - `dt` is the element type of h, the embedding, the gains and every weight
 *     matrix: TF_BF16 (bf16 operands, fp32 accumulation, bf16 rounding of the
 *     x and h' operands; the SwiGLU activation enters the down projection as
 *     a bf16 hi/lo pair, about 16 significant bits) or TF_F32 (fp32 throughout).
 *   - Shapes: b sequences, hidden size d, vocabulary V, draft depth gamma,
 *     M = k stage-1 candidates per depth, SwiGLU width I, draft budget B.
 *     R = 1 + (gamma-1)*k conditional rows per sequence.  Row 0 is depth 1
 *     conditioned on the root token; row 1 + (i-2)*k + m is depth i (2..gamma)
 *     conditioned on candidate m of depth i-1.
 *   - Requirements (else TF_ERR_INVALID_ARG): b >= 1, gamma >= 1, 1 <= k <= V,
 *     k <= 1024, d >= 16 and d % 16 == 0, I >= 16 and I % 16 == 0,
 *     inv_temperature > 0 and finite.  b*gamma*... products must fit in int32.
 *   - Ordering: every top-k list is sorted by (value desc, token id asc).
 *   - Non-finite inputs give unspecified (but memory-safe) results.
 *   - Calls that share a workspace must not overlap in time.
 */
#ifndef TREEFLASH_H
#define TREEFLASH_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TF_OK = 0,
    TF_ERR_INVALID_ARG = 1,  /* a NULL required pointer, a bad shape or parameter */
    TF_ERR_UNSUPPORTED = 2,  /* valid request outside what this build implements  */
    TF_ERR_WORKSPACE = 3,    /* workspace NULL or smaller than required           */
    TF_ERR_HIP = 4           /* a HIP launch or runtime error                     */
} tf_status_t;

typedef enum { TF_F32 = 0, TF_BF16 = 1 } tf_dtype_t;

/* Bytes of device workspace the two Part-1 calls need for these shapes (the
 * larger of the two).  `topk2` is the stage-2 list length (see below).
 * Returns 0 if the shapes are invalid.  The first 64 bytes of the workspace
 * hold diagnostic counters: int32 at byte offset 0 counts the (row, vocabulary
 * slice) pairs the last call re-evaluated on its exact slow path. */
size_t treeflash_workspace_bytes(int b, int gamma, int d, int I, int V, int k, int topk2,
                                 tf_dtype_t dt);

/* Part 1, stage 1 (Appendix B, first loop of Part 1): marginal LM head and top-k.
 *   h             [b, gamma, d]  drafter hidden states h_{t+1..t+gamma}
 *   lm_head       [V, d]         output embedding; row v belongs to token v
 *   inv_temperature              logits are multiplied by it before the softmax
 *   topk_idx      out [b, gamma, k] int32: the k best ids per depth (logit desc, id asc)
 *   topk_logprob  out [b, gamma, k] fp32 log-softmax values of those ids; may be NULL
 *   lse           out [b, gamma] fp32 log-sum-exp of the scaled logits; may be NULL
 * bf16: the order and the listed log-probs use each logit with its 7 lowest
 * mantissa bits cleared (a monotone change below 2^-16 relative), so logits
 * that close rank by id; the log-sum-exp uses the full values.
 * The [b*gamma, V] logits are never written to memory.  The operation is the
 * same for any set of rows: called on h' viewed as [b, R, d] with k = topk2 it
 * is the LM-head half of the conditional stage (here `gamma` only counts rows
 * and may exceed 255). */
tf_status_t treeflash_marginal_topk(const void *h, const void *lm_head,
                                    int b, int gamma, int d, int V, int k,
                                    float inv_temperature, tf_dtype_t dt,
                                    int32_t *topk_idx, float *topk_logprob, float *lse,
                                    void *workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/* treeflash_marginal_topk with its LM-head product timed: `ev_begin` and
 * `ev_end` (events created by the caller; either may be NULL) are recorded on
 * `stream` right before and right after the kernel that streams lm_head, so
 * the per-row merge kernel that follows lies outside the pair.  For callers
 * that measure that kernel's bandwidth; arguments, results and errors are
 * otherwise those of treeflash_marginal_topk (on an invalid argument nothing
 * is recorded). */
tf_status_t treeflash_marginal_topk_timed(const void *h, const void *lm_head,
                                          int b, int gamma, int d, int V, int k,
                                          float inv_temperature, tf_dtype_t dt,
                                          int32_t *topk_idx, float *topk_logprob, float *lse,
                                          void *workspace, size_t workspace_bytes,
                                          hipStream_t stream, hipEvent_t ev_begin,
                                          hipEvent_t ev_end);

/* treeflash_marginal_topk for callers that cannot allocate memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid it):
 * the same computation and outputs, with its scratch taken from a device
 * array the library owns instead of a caller workspace.  The array holds
 * treeflash_static_scratch_bytes() bytes (16 MiB: stage 1 of up to 16
 * sequences at the Qwen3-8B shape, or one sequence's conditional rows); a
 * call that needs more returns TF_ERR_WORKSPACE and launches nothing.  It
 * calls no allocator.  Each GPU holds one copy of the array until the process
 * ends, shared by every call on that GPU: calls that overlap in time on one
 * GPU (several streams or host threads) race and must be serialised by the
 * caller.  The first call on a GPU resolves the array's device address
 * (TF_ERR_HIP if the runtime cannot). */
tf_status_t treeflash_marginal_topk_static(const void *h, const void *lm_head,
                                           int b, int gamma, int d, int V, int k,
                                           float inv_temperature, tf_dtype_t dt,
                                           int32_t *topk_idx, float *topk_logprob, float *lse,
                                           hipStream_t stream);
size_t treeflash_static_scratch_bytes(void);

/* Part 1, stage 2, first half (Method, Eq. 1): the AR-approximated hidden
 * state of every conditional row,
 *   h'_r = h_{depth(r)} + W_down( silu(W_gate x_r) * (W_up x_r) ),
 *   x_r  = [ rms(h_{depth(r)}) * norm_h_gain ; rms(Embd(prev_r)) * norm_e_gain ].
 * Arguments as in treeflash_arapprox_expand below;
 *   hprime        out [b, R, d] (dtype dt; bf16 values are rounded to nearest even)
 * The workspace must be sized by treeflash_workspace_bytes. */
tf_status_t treeflash_arapprox_hidden(const void *h, const int32_t *root_token,
                                      const int32_t *topk_idx, const void *emb,
                                      const void *norm_h_gain, const void *norm_e_gain,
                                      const void *w_gate, const void *w_up, const void *w_down,
                                      int b, int gamma, int d, int I, int V, int k,
                                      float rms_eps, tf_dtype_t dt, void *hprime,
                                      void *workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/* The paper's "w/ Linear" ablation (Ablations, Model Design): the SwiGLU of
 * Eq. 1 replaced by one linear layer on the same normalised input,
 *   h'_r = h_{depth(r)} + W_lin x_r,  x_r as above,
 *   w_lin  [d, 2d] (columns 0..d-1 act on the normalised h, d..2d-1 on the
 *          normalised embedding; no bias)
 * Other arguments as in treeflash_arapprox_hidden (no SwiGLU width); bf16
 * rounds x and h'.  The workspace must hold
 * treeflash_workspace_bytes(b, gamma, d, 16, V, k, topk2, dt) bytes for any
 * valid topk2 (the SwiGLU width does not enter). */
tf_status_t treeflash_arapprox_linear_hidden(const void *h, const int32_t *root_token,
                                             const int32_t *topk_idx, const void *emb,
                                             const void *norm_h_gain, const void *norm_e_gain,
                                             const void *w_lin, int b, int gamma, int d, int V, int k,
                                             float rms_eps, tf_dtype_t dt, void *hprime,
                                             void *workspace, size_t workspace_bytes,
                                             hipStream_t stream);

/* Part 1, stage 2 (Method, Eq. 1; Appendix B, rest of Part 1): AR approximation
 * of every conditional row, LM head, log-softmax, top-topk2.  Equivalent to
 * treeflash_arapprox_hidden followed by treeflash_marginal_topk on h'.
 *   h             [b, gamma, d]  drafter hidden states
 *   root_token    [b] int32      x_t, the token that conditions depth 1
 *   topk_idx      [b, gamma, k]  int32 stage-1 candidates (ids must be < V)
 *   emb           [V, d]         input embedding Embd
 *   norm_h_gain   [d] or NULL    RMSNorm gain applied to h (NULL = ones)
 *   norm_e_gain   [d] or NULL    RMSNorm gain applied to Embd(prev) (NULL = ones)
 *   w_gate, w_up  [I, 2d]        SwiGLU input projections; columns 0..d-1 act on
 *                                the normalised h, columns d..2d-1 on the
 *                                normalised embedding
 *   w_down        [d, I]         SwiGLU output projection
 *   lm_head       [V, d]         output embedding (as in stage 1)
 *   topk2                        entries kept per row; min(B, V) <= topk2 <= V,
 *                                topk2 <= 1024.  topk2 >= min(B, V) makes the
 *                                tree of Part 2 equal to the tree of full rows.
 *   rms_eps                      RMSNorm epsilon (the paper's models use 1e-6), >= 0
 *   cond_idx      out [b, R, topk2] int32 best ids per row (log-prob desc, id asc)
 *   cond_logprob  out [b, R, topk2] fp32 log-softmax of those ids
 *   cond_lse      out [b, R] fp32 log-sum-exp of the scaled logits, or NULL
 * The [b*R, V] logits are never written to memory. */
tf_status_t treeflash_arapprox_expand(const void *h, const int32_t *root_token,
                                      const int32_t *topk_idx, const void *emb,
                                      const void *norm_h_gain, const void *norm_e_gain,
                                      const void *w_gate, const void *w_up,
                                      const void *w_down, const void *lm_head,
                                      int b, int gamma, int d, int I, int V, int k, int topk2,
                                      float inv_temperature, float rms_eps, tf_dtype_t dt,
                                      int32_t *cond_idx, float *cond_logprob, float *cond_lse,
                                      void *workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/* Part 2 (Appendix B): OPT-Tree selection.  Needs no workspace.
 *   cond_idx, cond_logprob  [b, R, topk2] rows as produced by the call above
 *                           (each row sorted by log-prob desc, id asc; log-probs <= 0)
 *   topk_idx                [b, gamma, k] stage-1 candidates
 *   B                       draft budget: nodes besides the root, 1 <= B <= 4095,
 *                           B <= V * (1 + k + ... + k^(gamma-1)), and topk2 >= min(B, V);
 *                           TF_ERR_UNSUPPORTED when the node table and frontier
 *                           (44*B + 20 + 4*gamma*k bytes) exceed the kernel's 144 KiB of
 *                           LDS, i.e. from about B = 3300 on
 * Outputs, per sequence, in pop order (best first), arrays [b, B]:
 *   node_token      token id
 *   node_parent     index of the parent node in the same array, -1 = the root x_t
 *   node_depth      1..gamma
 *   node_score      fp32 path log-probability: parent score + row log-prob, added in fp32
 *   node_child_row  row (0..R-1) holding this node's children, -1 if it is not
 *                   expandable (depth gamma, or not a stage-1 candidate); may be NULL
 * Ties in path score go to the shallower node, then to the lexicographically
 * smaller path of row ranks (rank = position in the parent's sorted row).
 * Rows shorter than the vocabulary (topk2 < B) may hold fewer admissible
 * nodes than B when they omit a depth's candidates: the selection then stops
 * when its frontier is empty and the remaining entries read token and parent
 * -1, depth 0, score -inf, child_row -1 (the count of real nodes is the
 * number of entries with depth > 0). */
tf_status_t treeflash_build_tree(const int32_t *cond_idx, const float *cond_logprob,
                                 const int32_t *topk_idx,
                                 int b, int gamma, int k, int topk2, int B,
                                 int32_t *node_token, int32_t *node_parent, int32_t *node_depth,
                                 float *node_score, int32_t *node_child_row,
                                 hipStream_t stream);

/* The paper's "w/ 2-prev" ablation (Ablations, Model Design): the AR
 * approximator reads the previous bigram instead of one token.
 *   R2 = 1 + k + (gamma-2)*k*k conditional rows per sequence (1 when gamma = 1):
 *   row 0: depth 1, previous tokens (context_token, root_token);
 *   rows 1..k: depth 2, (root_token, candidate m of depth 1), row 1 + m;
 *   depth i >= 3: (candidate m2 of depth i-2, candidate m1 of depth i-1),
 *   row 1 + k + (i-3)*k*k + m2*k + m1.
 * x_r = [ rms(h)*g_h ; rms(Embd(prev1))*g_e ; rms(Embd(prev2))*g_e ] with prev1
 * the token right before the drafted position, then Eq. 1's SwiGLU and
 * residual.  b*R2 must not exceed 2^20. */

/* Workspace bytes of treeflash_arapprox_2prev_hidden and of the LM-head call
 * on its rows (treeflash_marginal_topk on h' viewed as [b, R2, d] with k =
 * topk2); 0 for invalid shapes. */
size_t treeflash_workspace_bytes_2prev(int b, int gamma, int d, int I, int V, int k, int topk2,
                                       tf_dtype_t dt);

/* h' of every bigram row.
 *   context_token [b] int32: the token before each root (x_{t-1})
 *   w_gate, w_up  [I, 3d]  (columns: h~, then e~(prev1), then e~(prev2))
 *   w_down        [d, I]
 *   hprime        out [b, R2, d]
 * Other arguments, rounding and errors as treeflash_arapprox_hidden. */
tf_status_t treeflash_arapprox_2prev_hidden(const void *h, const int32_t *context_token,
                                            const int32_t *root_token, const int32_t *topk_idx,
                                            const void *emb, const void *norm_h_gain,
                                            const void *norm_e_gain, const void *w_gate,
                                            const void *w_up, const void *w_down, int b, int gamma,
                                            int d, int I, int V, int k, float rms_eps, tf_dtype_t dt,
                                            void *hprime, void *workspace, size_t workspace_bytes,
                                            hipStream_t stream);

/* OPT-Tree selection over the bigram rows [b, R2, topk2]: as treeflash_build_tree,
 * except that a node of depth i < gamma whose token is candidate m1 of its
 * depth expands into row 1 + m1 (i = 1) or 1 + k + (i-2)*k*k + m2*k + m1,
 * m2 being its parent's candidate index. */
tf_status_t treeflash_build_tree_2prev(const int32_t *cond_idx, const float *cond_logprob,
                                       const int32_t *topk_idx, int b, int gamma, int k, int topk2,
                                       int B, int32_t *node_token, int32_t *node_parent,
                                       int32_t *node_depth, float *node_score,
                                       int32_t *node_child_row, hipStream_t stream);

/* The marginal OPT-Tree (the paper's DDTree comparison, Related Work;
 * Appendix C): the same best-first selection on the drafter's marginal
 * distributions alone.  Every node above depth gamma expands into the
 * marginal row of the next depth, so all paths share one child ranking.
 * Needs no workspace.
 *   marg_idx, marg_logprob  [b, gamma, K] stage-1 lists from
 *                           treeflash_marginal_topk with k = K (row i-1 is
 *                           depth i, sorted by log-prob desc, id asc)
 *   K                       list length, 1 <= K <= 4096; K >= min(B, V) gives
 *                           the tree of full rows
 *   B                       1 <= B <= 4095 and B <= K + K^2 + ... + K^gamma;
 *                           TF_ERR_UNSUPPORTED past the kernel's LDS, as for
 *                           treeflash_build_tree
 * Outputs as for treeflash_build_tree; node_child_row is the row a node
 * expands into (its depth, 0-based row of depth+1) or -1 at depth gamma.
 * Ties: as for treeflash_build_tree. */
tf_status_t treeflash_build_tree_marginal(const int32_t *marg_idx, const float *marg_logprob,
                                          int b, int gamma, int K, int B,
                                          int32_t *node_token, int32_t *node_parent,
                                          int32_t *node_depth, float *node_score,
                                          int32_t *node_child_row, hipStream_t stream);

/* Verification hand-off, part 1 (Method, "Inference": the draft is verified
 * in one verifier pass with tree attention and an equality check): the tree
 * as that pass's input.  Position 0 is the root token x_t, position 1 + j is
 * node j of the tree (pop order, as produced by treeflash_build_tree or
 * treeflash_build_tree_marginal).  Needs no workspace.
 *   root_token      [b] int32
 *   node_token, node_parent, node_depth  [b, B] int32 (a parent precedes its
 *                   child; parent -1 = the root)
 *   tokens          out [b, B+1] int32: root token, then the node tokens
 *   positions       out [b, B+1] int32: depth of each position (root 0); add
 *                   the root's sequence position for absolute positions
 *   mask            out [b, B+1, B+1] uint8: mask[i][j] = 1 when position j
 *                   is position i or one of its ancestors (what i attends to
 *                   inside the tree), else 0
 * Requirements: 1 <= B <= 4095; int32 arrays 4-byte aligned. */
tf_status_t treeflash_tree_attention_inputs(const int32_t *root_token, const int32_t *node_token,
                                            const int32_t *node_parent, const int32_t *node_depth,
                                            int b, int B, int32_t *tokens, int32_t *positions,
                                            uint8_t *mask, hipStream_t stream);

/* Verification hand-off, part 2 (Method, "Inference"; Experiments, "Metrics":
 * block efficiency tau = accepted tokens + the verifier's residual token):
 * the greedy equality walk.  Needs no workspace.
 *   node_token, node_parent  [b, B] int32, as above
 *   target          [b, B+1] int32: the verifier's next token at every
 *                   position of the tree input above (position 0 = after the
 *                   root)
 *   gamma           longest acceptable path (the draft depth), 1..255
 *   accepted        out [b, gamma] int32: accepted node ids, root to leaf,
 *                   then -1
 *   accept_len      out [b] int32: number of accepted nodes; tau = accept_len + 1
 *   bonus           out [b] int32: the verifier's token after the last
 *                   accepted node (the residual token)
 * From the root, the walk moves to the child whose token equals the current
 * position's target while there is one (siblings carry distinct tokens). */
tf_status_t treeflash_accept(const int32_t *node_token, const int32_t *node_parent, const int32_t *target,
                             int b, int B, int gamma, int32_t *accepted, int32_t *accept_len,
                             int32_t *bonus, hipStream_t stream);

/* Static description of a status code. */
const char *treeflash_status_string(tf_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* TREEFLASH_H */

// Host launchers of the TreeFlash kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tf {

// LM head over `rows` activation rows [rows, d] (row stride ldx elements),
// followed by the per-row merge: top-K ids and log-probs, log-sum-exp.
// `lm_ws` holds lm_scratch_bytes(rows, V, d, bf16) bytes.
hipError_t launch_lmhead_topk(const void* x, long ldx, const void* w, int rows, int d, int V, int K,
                              float inv_t, bool bf16, unsigned char* lm_ws, int32_t* out_idx, float* out_lp,
                              float* out_lse, int* diag, hipStream_t stream, hipEvent_t ev_begin = nullptr,
                              hipEvent_t ev_end = nullptr);

// Eq. 1 for every conditional row: RMSNorm of h and of the previous token's
// embedding, SwiGLU, residual.  Writes h' [b*R, d] into `hp`.  `bigram`: the
// w/ 2-prev rows (rows.hpp), x = [h~ ; e~(prev1) ; e~(prev2)], W_gate/W_up
// [I, 3d], `context` [b] the token before each root (unused otherwise).
hipError_t launch_arapprox(const void* h, const int32_t* root, const int32_t* context, const int32_t* topk_idx,
                           const void* emb, const void* gain_h, const void* gain_e, const void* w_gate,
                           const void* w_up, const void* w_down, int b, int gamma, int d, int I, int V, int k,
                           bool bigram, float eps, bool bf16, void* ht, void* et, void* act, void* hp,
                           float* mlp_partial, int* counters, float* hh, int* diag, hipStream_t stream);

// The "w/ Linear" approximator for every conditional row: RMSNorm of h and
// of the previous token's embedding, h' = h + W_lin [h~ ; e~].
hipError_t launch_arapprox_linear(const void* h, const int32_t* root, const int32_t* topk_idx, const void* emb,
                                  const void* gain_h, const void* gain_e, const void* w_lin, int b, int gamma, int d,
                                  int V, int k, float eps, bool bf16, void* ht, void* et, void* hp,
                                  float* mlp_partial, int* counters, float* hh, int* diag, hipStream_t stream);

// Best-first tree selection, one workgroup per sequence.  `mode` 0: the
// single-token rows; 1: the rows are the gamma marginal rows [b, gamma,
// topk2] and every node above depth gamma expands into the next depth's row
// (topk_idx and k unused); 2: the bigram rows of the w/ 2-prev ablation.
hipError_t launch_build_tree(const int32_t* cond_idx, const float* cond_lp, const int32_t* topk_idx, int b,
                             int gamma, int k, int topk2, int B, int mode, int32_t* node_token,
                             int32_t* node_parent, int32_t* node_depth, float* node_score, int32_t* node_child_row,
                             hipStream_t stream);
size_t tree_lds_bytes(int B, int gamma, int M, int Rs, int K2, int* cached_ranks);

// Verifier input of a draft tree: tokens and positions [b, B+1], ancestor
// mask [b, B+1, B+1] (uint8).
hipError_t launch_tree_inputs(const int32_t* root_token, const int32_t* node_token, const int32_t* node_parent,
                              const int32_t* node_depth, int b, int B, int32_t* tokens, int32_t* positions,
                              uint8_t* mask, hipStream_t stream);

// Greedy acceptance walk: accepted node ids [b, max_depth], lengths and the
// verifier's bonus token per sequence.
hipError_t launch_accept(const int32_t* node_token, const int32_t* node_parent, const int32_t* target, int b, int B,
                         int max_depth, int32_t* accepted, int32_t* accept_len, int32_t* bonus, hipStream_t stream);

}  // namespace tf

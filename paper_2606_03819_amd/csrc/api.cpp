// C ABI of the TreeFlash drafting library: argument checks, workspace layout,
// launches.  Every argument is checked before the first HIP call.
#include <math.h>
#include <stdint.h>

#include <initializer_list>
#include <mutex>

#include "treeflash.h"
#include "launch.hpp"
#include "plan.hpp"

namespace {

using namespace tf;

constexpr long long kMaxRows = 1 << 20;

// Alignment.  An array not aligned to its element size is an invalid
// argument.  Operands read with 16-byte vector loads (h, h', the weights, the
// LM head) must also be 16-byte aligned; an element-aligned pointer that is
// not is a valid request this build does not implement (TF_ERR_UNSUPPORTED).
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool dtype_ok(tf_dtype_t dt) { return dt == TF_F32 || dt == TF_BF16; }
size_t elem_bytes(tf_dtype_t dt) { return dt == TF_BF16 ? 2 : 4; }
bool elem_aligned(const void* p, tf_dtype_t dt) { return (reinterpret_cast<uintptr_t>(p) % elem_bytes(dt)) == 0; }
// a vector-loaded operand of type dt (non-null)
tf_status_t vec_status(const void* p, tf_dtype_t dt) {
    if (!elem_aligned(p, dt)) return TF_ERR_INVALID_ARG;
    return aligned16(p) ? TF_OK : TF_ERR_UNSUPPORTED;
}
// the first non-OK status of a list of vector-loaded operands, invalid before unsupported
tf_status_t vec_status_all(std::initializer_list<const void*> ps, tf_dtype_t dt) {
    tf_status_t worst = TF_OK;
    for (const void* p : ps) {
        const tf_status_t st = vec_status(p, dt);
        if (st == TF_ERR_INVALID_ARG) return st;
        if (st != TF_OK) worst = st;
    }
    return worst;
}

// Widths: d (and I) must be positive; the kernels step through them 16 at a
// time (the MFMA's k), so other values are unsupported.
tf_status_t width_status(int w) {
    if (w < 1) return TF_ERR_INVALID_ARG;
    return w % 16 == 0 ? TF_OK : TF_ERR_UNSUPPORTED;
}

// `gamma` is a draft depth (at most 255) unless `rows_only`, where it only
// counts rows per sequence (the LM-head call on h' viewed as [b, R, d]).
tf_status_t common_shapes(int b, int gamma, int d, int V, int k, bool rows_only = false) {
    if (b < 1 || gamma < 1 || (!rows_only && gamma > 255) || V < 1 || k < 1 || k > V || k > kMaxTopk)
        return TF_ERR_INVALID_ARG;
    const tf_status_t wd = width_status(d);
    if (wd != TF_OK) return wd;
    if ((long long)b * gamma > kMaxRows) return TF_ERR_INVALID_ARG;
    if (!rows_only && (long long)b * (1 + (long long)(gamma - 1) * k) > kMaxRows) return TF_ERR_INVALID_ARG;
    if ((long long)V * d >= (1ll << 40)) return TF_ERR_INVALID_ARG;
    return TF_OK;
}

size_t stage1_bytes(int b, int gamma, int d, int V, bool bf16) {
    return 256 + lm_scratch_bytes(b * gamma, V, d, bf16);
}

}  // namespace

extern "C" {

size_t treeflash_workspace_bytes(int b, int gamma, int d, int I, int V, int k, int topk2, tf_dtype_t dt) {
    if (!dtype_ok(dt) || common_shapes(b, gamma, d, V, k) != TF_OK) return 0;
    if (width_status(I) != TF_OK || topk2 < 1 || topk2 > V || topk2 > kMaxTopk) return 0;
    return workspace_layout(b, gamma, d, I, V, k, dt == TF_BF16).total;
}

// Every argument of the LM-head call but its workspace.
static tf_status_t check_marginal_args(const void* h, const void* lm_head, int b, int gamma, int d, int V, int k,
                                       float inv_temperature, tf_dtype_t dt, const int32_t* topk_idx,
                                       const float* topk_logprob, const float* lse) {
    if (h == nullptr || lm_head == nullptr || topk_idx == nullptr) return TF_ERR_INVALID_ARG;
    if (!dtype_ok(dt)) return TF_ERR_INVALID_ARG;
    const tf_status_t shp = common_shapes(b, gamma, d, V, k, true);
    if (shp != TF_OK) return shp;
    if (!(inv_temperature > 0.f) || !isfinite(inv_temperature)) return TF_ERR_INVALID_ARG;
    if (!aligned4(topk_idx) || (topk_logprob != nullptr && !aligned4(topk_logprob)) || (lse != nullptr && !aligned4(lse)))
        return TF_ERR_INVALID_ARG;
    return vec_status_all({h, lm_head}, dt);
}

static tf_status_t marginal_topk(const void* h, const void* lm_head, int b, int gamma, int d, int V, int k,
                                 float inv_temperature, tf_dtype_t dt, int32_t* topk_idx, float* topk_logprob,
                                 float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 hipEvent_t ev_begin, hipEvent_t ev_end) {
    const tf_status_t chk =
        check_marginal_args(h, lm_head, b, gamma, d, V, k, inv_temperature, dt, topk_idx, topk_logprob, lse);
    if (chk != TF_OK) return chk;
    const bool bf16 = dt == TF_BF16;
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < stage1_bytes(b, gamma, d, V, bf16))
        return TF_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    int* diag = reinterpret_cast<int*>(ws);
    const hipError_t e = launch_lmhead_topk(h, d, lm_head, b * gamma, d, V, k, inv_temperature, bf16, ws + 256,
                                            topk_idx, topk_logprob, lse, diag, stream, ev_begin, ev_end);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

tf_status_t treeflash_marginal_topk(const void* h, const void* lm_head, int b, int gamma, int d, int V, int k,
                                    float inv_temperature, tf_dtype_t dt, int32_t* topk_idx,
                                    float* topk_logprob, float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    return marginal_topk(h, lm_head, b, gamma, d, V, k, inv_temperature, dt, topk_idx, topk_logprob, lse, workspace,
                         workspace_bytes, stream, nullptr, nullptr);
}

}  // extern "C"

// ------------------------------------------- the allocation-free variant
//
// treeflash_marginal_topk_static draws its scratch (the diagnostic counter
// and the (row, vocabulary slice) partials) from a device array of
// kStaticScratchBytes owned by the library, not from a caller workspace.
// Every call on a GPU shares that GPU's copy of the array, so calls that
// overlap in time on one GPU (other streams, other host threads) race.  The
// LM-head kernel zeroes the diagnostic counter itself and writes every
// partial the merge reads, so nothing left by an earlier call is read.
namespace {

constexpr size_t kStaticScratchBytes = 16u << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// This device's address of `scratch`, resolved once per device (each GPU
// holds its own copy of the array); nullptr when the runtime cannot.
void* device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

tf_status_t treeflash_marginal_topk_static(const void* h, const void* lm_head, int b, int gamma, int d, int V,
                                           int k, float inv_temperature, tf_dtype_t dt, int32_t* topk_idx,
                                           float* topk_logprob, float* lse, hipStream_t stream) {
    // every argument and the scratch size before any HIP call
    const tf_status_t chk =
        check_marginal_args(h, lm_head, b, gamma, d, V, k, inv_temperature, dt, topk_idx, topk_logprob, lse);
    if (chk != TF_OK) return chk;
    if (stage1_bytes(b, gamma, d, V, dt == TF_BF16) > kStaticScratchBytes) return TF_ERR_WORKSPACE;
    void* ws = device_scratch();
    if (ws == nullptr) return TF_ERR_HIP;
    return marginal_topk(h, lm_head, b, gamma, d, V, k, inv_temperature, dt, topk_idx, topk_logprob, lse, ws,
                         kStaticScratchBytes, stream, nullptr, nullptr);
}

size_t treeflash_static_scratch_bytes(void) { return kStaticScratchBytes; }

tf_status_t treeflash_marginal_topk_timed(const void* h, const void* lm_head, int b, int gamma, int d, int V, int k,
                                          float inv_temperature, tf_dtype_t dt, int32_t* topk_idx,
                                          float* topk_logprob, float* lse, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream, hipEvent_t ev_begin,
                                          hipEvent_t ev_end) {
    return marginal_topk(h, lm_head, b, gamma, d, V, k, inv_temperature, dt, topk_idx, topk_logprob, lse, workspace,
                         workspace_bytes, stream, ev_begin, ev_end);
}

}  // extern "C"

namespace {

// w_up may be null (the plain SiLU MLP) when `up_optional`.
tf_status_t check_hidden_args(const void* h, const int32_t* root_token, const int32_t* topk_idx, const void* emb,
                              const void* norm_h_gain, const void* norm_e_gain, const void* w_gate,
                              const void* w_up, const void* w_down, int b, int gamma, int d, int I, int V, int k,
                              float rms_eps, tf_dtype_t dt, bool up_optional = false) {
    if (h == nullptr || root_token == nullptr || topk_idx == nullptr || emb == nullptr || w_gate == nullptr ||
        (w_up == nullptr && !up_optional) || w_down == nullptr)
        return TF_ERR_INVALID_ARG;
    if (!dtype_ok(dt)) return TF_ERR_INVALID_ARG;
    tf_status_t st = common_shapes(b, gamma, d, V, k);
    if (st != TF_OK) return st;
    if ((st = width_status(I)) != TF_OK) return st;
    if (!(rms_eps >= 0.f) || !isfinite(rms_eps)) return TF_ERR_INVALID_ARG;
    if (!aligned4(root_token) || !aligned4(topk_idx) || !elem_aligned(emb, dt)) return TF_ERR_INVALID_ARG;
    if ((norm_h_gain != nullptr && !elem_aligned(norm_h_gain, dt)) ||
        (norm_e_gain != nullptr && !elem_aligned(norm_e_gain, dt)))
        return TF_ERR_INVALID_ARG;
    return vec_status_all({h, w_gate, w_up != nullptr ? w_up : w_gate, w_down}, dt);
}

}  // namespace

extern "C" {

tf_status_t treeflash_arapprox_hidden(const void* h, const int32_t* root_token, const int32_t* topk_idx,
                                      const void* emb, const void* norm_h_gain, const void* norm_e_gain,
                                      const void* w_gate, const void* w_up, const void* w_down, int b, int gamma,
                                      int d, int I, int V, int k, float rms_eps, tf_dtype_t dt, void* hprime,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
    const tf_status_t chk = check_hidden_args(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up,
                                              w_down, b, gamma, d, I, V, k, rms_eps, dt, true);
    if (chk != TF_OK) return chk;
    if (hprime == nullptr) return TF_ERR_INVALID_ARG;
    if (vec_status(hprime, dt) != TF_OK) return vec_status(hprime, dt);
    const bool bf16 = dt == TF_BF16;
    const Workspace lay = workspace_layout(b, gamma, d, I, V, k, bf16);
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < lay.total) return TF_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    const hipError_t e = launch_arapprox(h, root_token, nullptr, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate,
                                         w_up, w_down, b, gamma, d, I, V, k, false, rms_eps, bf16, ws + lay.ht, ws + lay.et,
                                         ws + lay.act, hprime, reinterpret_cast<float*>(ws + lay.mlp_part),
                                         reinterpret_cast<int*>(ws + lay.counters), reinterpret_cast<float*>(ws + lay.hh),
                                         reinterpret_cast<int*>(ws + lay.diag), stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

size_t treeflash_workspace_bytes_2prev(int b, int gamma, int d, int I, int V, int k, int topk2, tf_dtype_t dt) {
    if (!dtype_ok(dt) || common_shapes(b, gamma, d, V, k) != TF_OK) return 0;
    if (width_status(I) != TF_OK || topk2 < 1 || topk2 > V || topk2 > kMaxTopk) return 0;
    if ((long long)b * cond_rows(gamma, k, 1) > kMaxRows) return 0;
    return workspace_layout(b, gamma, d, I, V, k, dt == TF_BF16, true).total;
}

tf_status_t treeflash_arapprox_2prev_hidden(const void* h, const int32_t* context_token, const int32_t* root_token,
                                            const int32_t* topk_idx, const void* emb, const void* norm_h_gain,
                                            const void* norm_e_gain, const void* w_gate, const void* w_up,
                                            const void* w_down, int b, int gamma, int d, int I, int V, int k,
                                            float rms_eps, tf_dtype_t dt, void* hprime, void* workspace,
                                            size_t workspace_bytes, hipStream_t stream) {
    const tf_status_t chk = check_hidden_args(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up,
                                              w_down, b, gamma, d, I, V, k, rms_eps, dt);
    if (chk != TF_OK) return chk;
    if (context_token == nullptr || !aligned4(context_token)) return TF_ERR_INVALID_ARG;
    if ((long long)b * cond_rows(gamma, k, 1) > kMaxRows) return TF_ERR_INVALID_ARG;
    if (hprime == nullptr) return TF_ERR_INVALID_ARG;
    if (vec_status(hprime, dt) != TF_OK) return vec_status(hprime, dt);
    const bool bf16 = dt == TF_BF16;
    const Workspace lay = workspace_layout(b, gamma, d, I, V, k, bf16, true);
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < lay.total) return TF_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    const hipError_t e = launch_arapprox(h, root_token, context_token, topk_idx, emb, norm_h_gain, norm_e_gain,
                                         w_gate, w_up, w_down, b, gamma, d, I, V, k, true, rms_eps, bf16,
                                         ws + lay.ht, ws + lay.et, ws + lay.act, hprime,
                                         reinterpret_cast<float*>(ws + lay.mlp_part),
                                         reinterpret_cast<int*>(ws + lay.counters),
                                         reinterpret_cast<float*>(ws + lay.hh), reinterpret_cast<int*>(ws + lay.diag),
                                         stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

tf_status_t treeflash_arapprox_linear_hidden(const void* h, const int32_t* root_token, const int32_t* topk_idx,
                                             const void* emb, const void* norm_h_gain, const void* norm_e_gain,
                                             const void* w_lin, int b, int gamma, int d, int V, int k, float rms_eps,
                                             tf_dtype_t dt, void* hprime, void* workspace, size_t workspace_bytes,
                                             hipStream_t stream) {
    // the SwiGLU checks with w_lin standing in for the three projections and the smallest width
    const tf_status_t chk = check_hidden_args(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_lin, w_lin,
                                              w_lin, b, gamma, d, 16, V, k, rms_eps, dt);
    if (chk != TF_OK) return chk;
    if (hprime == nullptr) return TF_ERR_INVALID_ARG;
    if (vec_status(hprime, dt) != TF_OK) return vec_status(hprime, dt);
    const bool bf16 = dt == TF_BF16;
    const Workspace lay = workspace_layout(b, gamma, d, 16, V, k, bf16);
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < lay.total) return TF_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    const hipError_t e = launch_arapprox_linear(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_lin, b,
                                                gamma, d, V, k, rms_eps, bf16, ws + lay.ht, ws + lay.et, hprime,
                                                reinterpret_cast<float*>(ws + lay.mlp_part),
                                                reinterpret_cast<int*>(ws + lay.counters),
                                                reinterpret_cast<float*>(ws + lay.hh),
                                                reinterpret_cast<int*>(ws + lay.diag), stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

tf_status_t treeflash_arapprox_expand(const void* h, const int32_t* root_token, const int32_t* topk_idx,
                                      const void* emb, const void* norm_h_gain, const void* norm_e_gain,
                                      const void* w_gate, const void* w_up, const void* w_down,
                                      const void* lm_head, int b, int gamma, int d, int I, int V, int k, int topk2,
                                      float inv_temperature, float rms_eps, tf_dtype_t dt, int32_t* cond_idx,
                                      float* cond_logprob, float* cond_lse, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream) {
    const tf_status_t chk = check_hidden_args(h, root_token, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up,
                                              w_down, b, gamma, d, I, V, k, rms_eps, dt, true);
    if (chk != TF_OK) return chk;
    if (lm_head == nullptr || cond_idx == nullptr || cond_logprob == nullptr) return TF_ERR_INVALID_ARG;
    if (topk2 < 1 || topk2 > V || topk2 > kMaxTopk) return TF_ERR_INVALID_ARG;
    if (!(inv_temperature > 0.f) || !isfinite(inv_temperature)) return TF_ERR_INVALID_ARG;
    if (!aligned4(cond_idx) || !aligned4(cond_logprob) || (cond_lse != nullptr && !aligned4(cond_lse)))
        return TF_ERR_INVALID_ARG;
    if (vec_status(lm_head, dt) != TF_OK) return vec_status(lm_head, dt);
    const bool bf16 = dt == TF_BF16;
    const Workspace lay = workspace_layout(b, gamma, d, I, V, k, bf16);
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < lay.total) return TF_ERR_WORKSPACE;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    int* diag = reinterpret_cast<int*>(ws + lay.diag);
    hipError_t e = launch_arapprox(h, root_token, nullptr, topk_idx, emb, norm_h_gain, norm_e_gain, w_gate, w_up,
                                   w_down, b, gamma, d, I, V, k, false, rms_eps, bf16, ws + lay.ht, ws + lay.et,
                                   ws + lay.act,
                                   ws + lay.hp, reinterpret_cast<float*>(ws + lay.mlp_part),
                                   reinterpret_cast<int*>(ws + lay.counters), reinterpret_cast<float*>(ws + lay.hh), diag,
                                   stream);
    if (e != hipSuccess) return TF_ERR_HIP;
    const int rows = b * (1 + (gamma - 1) * k);
    e = launch_lmhead_topk(ws + lay.hp, d, lm_head, rows, d, V, topk2, inv_temperature, bf16, ws + lay.lm,
                           cond_idx, cond_logprob, cond_lse, diag, stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

}  // extern "C"

namespace {

// The selection over single-token or bigram conditional rows.
tf_status_t build_tree_rows(const int32_t* cond_idx, const float* cond_logprob, const int32_t* topk_idx, int b,
                            int gamma, int k, int topk2, int B, bool bigram, int32_t* node_token,
                            int32_t* node_parent, int32_t* node_depth, float* node_score, int32_t* node_child_row,
                            hipStream_t stream) {
    if (cond_idx == nullptr || cond_logprob == nullptr || topk_idx == nullptr || node_token == nullptr ||
        node_parent == nullptr || node_depth == nullptr || node_score == nullptr)
        return TF_ERR_INVALID_ARG;
    if (b < 1 || gamma < 1 || gamma > 255 || k < 1 || k > kMaxTopk || topk2 < 1 || topk2 > 4096) return TF_ERR_INVALID_ARG;
    if (B < 1 || B > kMaxBudget) return TF_ERR_INVALID_ARG;
    const long long Rs = cond_rows(gamma, k, bigram ? 1 : 0);
    if ((long long)b * Rs > kMaxRows) return TF_ERR_INVALID_ARG;
    if (topk2 < B) {
        // Rows shorter than B are only meaningful when they are full rows
        // (topk2 == V); then the tree can hold topk2 * (1 + k + ... + k^(gamma-1)) nodes.
        long long cap = 0, pw = 1;
        for (int j = 0; j < gamma && cap < B; ++j) {
            cap += pw * topk2;
            pw = pw * k > (1ll << 40) ? (1ll << 40) : pw * k;
        }
        if (cap < B) return TF_ERR_INVALID_ARG;
    }
    const void* ptrs[] = {cond_idx, cond_logprob, topk_idx, node_token, node_parent, node_depth, node_score};
    for (const void* p : ptrs)
        if (!aligned4(p)) return TF_ERR_INVALID_ARG;
    if (node_child_row != nullptr && !aligned4(node_child_row)) return TF_ERR_INVALID_ARG;
    if (tree_lds_bytes(B, gamma, k, (int)Rs, topk2, nullptr) == 0) return TF_ERR_UNSUPPORTED;
    const hipError_t e = launch_build_tree(cond_idx, cond_logprob, topk_idx, b, gamma, k, topk2, B, bigram ? 2 : 0,
                                           node_token, node_parent, node_depth, node_score, node_child_row, stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

}  // namespace

extern "C" {

tf_status_t treeflash_build_tree(const int32_t* cond_idx, const float* cond_logprob, const int32_t* topk_idx, int b,
                                 int gamma, int k, int topk2, int B, int32_t* node_token, int32_t* node_parent,
                                 int32_t* node_depth, float* node_score, int32_t* node_child_row,
                                 hipStream_t stream) {
    return build_tree_rows(cond_idx, cond_logprob, topk_idx, b, gamma, k, topk2, B, false, node_token, node_parent,
                           node_depth, node_score, node_child_row, stream);
}

tf_status_t treeflash_build_tree_2prev(const int32_t* cond_idx, const float* cond_logprob, const int32_t* topk_idx,
                                       int b, int gamma, int k, int topk2, int B, int32_t* node_token,
                                       int32_t* node_parent, int32_t* node_depth, float* node_score,
                                       int32_t* node_child_row, hipStream_t stream) {
    return build_tree_rows(cond_idx, cond_logprob, topk_idx, b, gamma, k, topk2, B, true, node_token, node_parent,
                           node_depth, node_score, node_child_row, stream);
}

tf_status_t treeflash_build_tree_marginal(const int32_t* marg_idx, const float* marg_logprob, int b, int gamma,
                                          int K, int B, int32_t* node_token, int32_t* node_parent,
                                          int32_t* node_depth, float* node_score, int32_t* node_child_row,
                                          hipStream_t stream) {
    if (marg_idx == nullptr || marg_logprob == nullptr || node_token == nullptr || node_parent == nullptr ||
        node_depth == nullptr || node_score == nullptr)
        return TF_ERR_INVALID_ARG;
    if (b < 1 || gamma < 1 || gamma > 255 || K < 1 || K > 4096 || B < 1 || B > kMaxBudget)
        return TF_ERR_INVALID_ARG;
    if ((long long)b * gamma > kMaxRows) return TF_ERR_INVALID_ARG;
    // every path of length 1..gamma over the rows is a node: K + K^2 + ... + K^gamma of them
    long long cap = 0, pw = K;
    for (int j = 0; j < gamma && cap < B; ++j) {
        cap += pw;
        pw = pw * K > (1ll << 40) ? (1ll << 40) : pw * K;
    }
    if (cap < B) return TF_ERR_INVALID_ARG;
    const void* ptrs[] = {marg_idx, marg_logprob, node_token, node_parent, node_depth, node_score};
    for (const void* p : ptrs)
        if (!aligned4(p)) return TF_ERR_INVALID_ARG;
    if (node_child_row != nullptr && !aligned4(node_child_row)) return TF_ERR_INVALID_ARG;
    if (tree_lds_bytes(B, gamma, 0, gamma, K, nullptr) == 0) return TF_ERR_UNSUPPORTED;
    const hipError_t e = launch_build_tree(marg_idx, marg_logprob, nullptr, b, gamma, 0, K, B, 1, node_token,
                                           node_parent, node_depth, node_score, node_child_row, stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

tf_status_t treeflash_tree_attention_inputs(const int32_t* root_token, const int32_t* node_token,
                                            const int32_t* node_parent, const int32_t* node_depth, int b, int B,
                                            int32_t* tokens, int32_t* positions, uint8_t* mask,
                                            hipStream_t stream) {
    if (root_token == nullptr || node_token == nullptr || node_parent == nullptr || node_depth == nullptr ||
        tokens == nullptr || positions == nullptr || mask == nullptr)
        return TF_ERR_INVALID_ARG;
    if (b < 1 || B < 1 || B > kMaxBudget || (long long)b * (B + 1) * (B + 1) > (1ll << 40)) return TF_ERR_INVALID_ARG;
    const void* ptrs[] = {root_token, node_token, node_parent, node_depth, tokens, positions};
    for (const void* p : ptrs)
        if (!aligned4(p)) return TF_ERR_INVALID_ARG;
    const hipError_t e = launch_tree_inputs(root_token, node_token, node_parent, node_depth, b, B, tokens,
                                            positions, mask, stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

tf_status_t treeflash_accept(const int32_t* node_token, const int32_t* node_parent, const int32_t* target, int b,
                             int B, int gamma, int32_t* accepted, int32_t* accept_len, int32_t* bonus,
                             hipStream_t stream) {
    if (node_token == nullptr || node_parent == nullptr || target == nullptr || accepted == nullptr ||
        accept_len == nullptr || bonus == nullptr)
        return TF_ERR_INVALID_ARG;
    if (b < 1 || B < 1 || B > kMaxBudget || gamma < 1 || gamma > 255) return TF_ERR_INVALID_ARG;
    const void* ptrs[] = {node_token, node_parent, target, accepted, accept_len, bonus};
    for (const void* p : ptrs)
        if (!aligned4(p)) return TF_ERR_INVALID_ARG;
    const hipError_t e = launch_accept(node_token, node_parent, target, b, B, gamma, accepted, accept_len, bonus,
                                       stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

const char* treeflash_status_string(tf_status_t status) {
    switch (status) {
        case TF_OK: return "success";
        case TF_ERR_INVALID_ARG: return "invalid argument";
        case TF_ERR_UNSUPPORTED: return "unsupported configuration";
        case TF_ERR_WORKSPACE: return "workspace missing or too small";
        case TF_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

}  // extern "C"

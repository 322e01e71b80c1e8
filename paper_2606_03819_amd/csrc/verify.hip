// Verification hand-off (Method, "Inference": the draft tree is verified in
// one pass with an equality check; Experiments, "Metrics": block efficiency
// counts the accepted tokens plus the verifier's residual token).
//
// tree_inputs_kernel lays a draft tree out for a verifier pass with tree
// attention: position 0 is the root token, position 1 + j node j (pop
// order); positions are depths; mask[i][j] = 1 when position j is position i
// or one of its ancestors.  accept_kernel walks the tree with the verifier's
// next token at every position: from the root, to the child carrying the
// current position's target, while there is one.
#include "common.hpp"
#include "launch.hpp"

namespace tf {

constexpr int kVerifyThreads = 256;

// One workgroup per sequence.  Parents are staged in LDS; a node's parent
// must precede it (pop order), which also bounds every ancestor walk.
__global__ __launch_bounds__(kVerifyThreads) void tree_inputs_kernel(const int32_t* __restrict__ root_token,
                                                                     const int32_t* __restrict__ node_token,
                                                                     const int32_t* __restrict__ node_parent,
                                                                     const int32_t* __restrict__ node_depth, int B,
                                                                     int32_t* __restrict__ tokens,
                                                                     int32_t* __restrict__ positions,
                                                                     uint8_t* __restrict__ mask) {
    extern __shared__ int32_t par[];
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int n = B + 1;
    const int32_t* tk = node_token + (size_t)s * B;
    const int32_t* pa = node_parent + (size_t)s * B;
    const int32_t* dp = node_depth + (size_t)s * B;
    int32_t* to = tokens + (size_t)s * n;
    int32_t* po = positions + (size_t)s * n;
    uint8_t* m = mask + (size_t)s * n * n;

    for (int j = tid; j < B; j += kVerifyThreads) par[j] = pa[j];
    for (int i = tid; i < n; i += kVerifyThreads) {
        to[i] = i == 0 ? root_token[s] : tk[i - 1];
        po[i] = i == 0 ? 0 : dp[i - 1];
    }
    // zero the n x n mask: 16-byte stores on the aligned middle, bytes at the ends
    const size_t total = (size_t)n * n;
    const size_t head = (16 - (reinterpret_cast<uintptr_t>(m) & 15)) & 15;
    const size_t h = head < total ? head : total;
    for (size_t e = tid; e < h; e += kVerifyThreads) m[e] = 0;
    const size_t nvec = (total - h) / 16;
    uint4* mv = reinterpret_cast<uint4*>(m + h);
    for (size_t e = tid; e < nvec; e += kVerifyThreads) mv[e] = uint4{0u, 0u, 0u, 0u};
    for (size_t e = h + nvec * 16 + tid; e < total; e += kVerifyThreads) m[e] = 0;
    __syncthreads();   // zeros stored and parents staged before the ones below

    for (int i = tid; i < n; i += kVerifyThreads) {
        uint8_t* row = m + (size_t)i * n;
        row[0] = 1;
        if (i == 0) continue;
        row[i] = 1;
        int child = i - 1;
        int p = par[child];
        while (p >= 0 && p < child) {   // ancestors in pop order always precede
            row[1 + p] = 1;
            child = p;
            p = par[p];
        }
    }
}

// One wave per sequence.
__global__ __launch_bounds__(64) void accept_kernel(const int32_t* __restrict__ node_token,
                                                    const int32_t* __restrict__ node_parent,
                                                    const int32_t* __restrict__ target, int B, int max_depth,
                                                    int32_t* __restrict__ accepted, int32_t* __restrict__ accept_len,
                                                    int32_t* __restrict__ bonus) {
    extern __shared__ int32_t lds[];
    int32_t* par = lds;
    int32_t* tok = lds + B;
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    const int32_t* tg = target + (size_t)s * (B + 1);
    for (int j = lane; j < B; j += 64) {
        par[j] = node_parent[(size_t)s * B + j];
        tok[j] = node_token[(size_t)s * B + j];
    }
    __syncthreads();
    int cur = -1, len = 0;
    while (len < max_depth) {
        const int want = tg[1 + cur];
        int hit = -1;
        for (int j0 = 0; j0 < B && hit < 0; j0 += 64) {
            const int j = j0 + lane;
            const bool ok = j < B && par[j] == cur && tok[j] == want;
            const unsigned long long bal = __ballot(ok);
            if (bal != 0ull) hit = j0 + __ffsll((long long)bal) - 1;
        }
        if (hit < 0) break;
        if (lane == 0) accepted[(size_t)s * max_depth + len] = hit;
        cur = hit;
        ++len;
    }
    for (int i = len + lane; i < max_depth; i += 64) accepted[(size_t)s * max_depth + i] = -1;
    if (lane == 0) {
        accept_len[s] = len;
        bonus[s] = tg[1 + cur];
    }
}

hipError_t launch_tree_inputs(const int32_t* root_token, const int32_t* node_token, const int32_t* node_parent,
                              const int32_t* node_depth, int b, int B, int32_t* tokens, int32_t* positions,
                              uint8_t* mask, hipStream_t stream) {
    hipLaunchKernelGGL(tree_inputs_kernel, dim3(b), dim3(kVerifyThreads), (size_t)B * 4, stream, root_token,
                       node_token, node_parent, node_depth, B, tokens, positions, mask);
    return hipGetLastError();
}

hipError_t launch_accept(const int32_t* node_token, const int32_t* node_parent, const int32_t* target, int b, int B,
                         int max_depth, int32_t* accepted, int32_t* accept_len, int32_t* bonus, hipStream_t stream) {
    hipLaunchKernelGGL(accept_kernel, dim3(b), dim3(64), (size_t)B * 8, stream, node_token, node_parent, target, B,
                       max_depth, accepted, accept_len, bonus);
    return hipGetLastError();
}

}  // namespace tf

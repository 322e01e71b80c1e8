// OPT-Tree selection (Appendix B, Part 2) on the GPU, one wave per sequence.
//
// The paper's queue holds every child of every expanded node.  Because each
// conditional row arrives sorted, a node's children are popped in row order,
// so the frontier only needs each expanded node's best child not yet popped:
// slot 0 holds the root's next child, slot n+1 node n's next child.  A pop is
// an argmax over at most B+1 slots (a 64-lane butterfly), then the popped
// slot advances to its next sibling and, if the popped token is a stage-1
// candidate of its depth, slot n+1 opens on the first entry of its row.
//
// Candidate order: path score (fp32 running sum) desc, depth asc, then the
// lexicographic order of the rank paths (ranks of the nodes in their parents'
// rows, root to node).  Siblings compare by rank; nodes of different parents
// at equal depth compare at the first ancestor where their paths diverge.
#include "common.hpp"
#include "launch.hpp"
#include "plan.hpp"

namespace tf {

constexpr int kTreeLdsBudget = 64 * 1024;

struct TreeArgs {
    const int32_t* cond_idx;
    const float* cond_lp;
    const int32_t* topk;
    int gamma, M, K2, B, Rs, P;   // P = leading ranks of each row cached in LDS
    int32_t* tok;
    int32_t* par;
    int32_t* dep;
    float* score;
    int32_t* crow;
};

struct TreeLds {
    int32_t *n_tok, *n_par, *n_rank, *n_dep, *n_crow;
    float* n_score;
    float *f_score, *f_pscore;
    int32_t *f_depth, *f_rank, *f_row;
    int32_t* tk;
    float* c_lp;
    int32_t* c_idx;
};

// Byte size of the fixed part (nodes, frontier, candidate table).
__host__ __device__ inline size_t tree_fixed_bytes(int B, int gamma, int M) {
    return (size_t)24 * B + (size_t)20 * (B + 1) + (size_t)4 * gamma * M;
}

__device__ inline TreeLds tree_lds(unsigned char* base, const TreeArgs& a) {
    TreeLds t;
    int32_t* p = reinterpret_cast<int32_t*>(base);
    t.n_tok = p; p += a.B;
    t.n_par = p; p += a.B;
    t.n_rank = p; p += a.B;
    t.n_dep = p; p += a.B;
    t.n_crow = p; p += a.B;
    t.n_score = reinterpret_cast<float*>(p); p += a.B;
    t.f_score = reinterpret_cast<float*>(p); p += a.B + 1;
    t.f_pscore = reinterpret_cast<float*>(p); p += a.B + 1;
    t.f_depth = p; p += a.B + 1;
    t.f_rank = p; p += a.B + 1;
    t.f_row = p; p += a.B + 1;
    t.tk = p; p += a.gamma * a.M;
    t.c_lp = reinterpret_cast<float*>(p); p += a.Rs * a.P;
    t.c_idx = p;
    return t;
}

struct Cand {
    float score;
    uint32_t meta;   // depth << 24 | slot << 12 | rank; depth 0 = empty
};

__device__ __forceinline__ int c_depth(uint32_t m) { return (int)(m >> 24); }
__device__ __forceinline__ int c_slot(uint32_t m) { return (int)((m >> 12) & 0xfffu); }
__device__ __forceinline__ int c_rank(uint32_t m) { return (int)(m & 0xfffu); }

__device__ __forceinline__ bool cand_before(const Cand& x, const Cand& y, const TreeLds& t) {
    const int dx = c_depth(x.meta), dy = c_depth(y.meta);
    if (dx == 0) return false;
    if (dy == 0) return true;
    if (x.score != y.score) return x.score > y.score;
    if (dx != dy) return dx < dy;
    int px = c_slot(x.meta) - 1, py = c_slot(y.meta) - 1;
    int rx = c_rank(x.meta), ry = c_rank(y.meta);
    while (px != py) {   // equal depths: both reach the common ancestor together
        rx = t.n_rank[px];
        ry = t.n_rank[py];
        px = t.n_par[px];
        py = t.n_par[py];
    }
    return rx < ry;
}

__global__ __launch_bounds__(64) void build_tree_kernel(TreeArgs a) {
    extern __shared__ __align__(16) unsigned char dyn[];
    const TreeLds t = tree_lds(dyn, a);
    const int seq = blockIdx.x;
    const int lane = threadIdx.x;
    const int32_t* ridx = a.cond_idx + (size_t)seq * a.Rs * a.K2;
    const float* rlp = a.cond_lp + (size_t)seq * a.Rs * a.K2;

    for (int s = lane; s <= a.B; s += 64) t.f_depth[s] = 0;
    for (int e = lane; e < a.gamma * a.M; e += 64) t.tk[e] = a.topk[(size_t)seq * a.gamma * a.M + e];
    for (int e = lane; e < a.Rs * a.P; e += 64) {
        const int r = e / a.P, c = e - r * a.P;
        t.c_lp[e] = rlp[(size_t)r * a.K2 + c];
        t.c_idx[e] = ridx[(size_t)r * a.K2 + c];
    }
    __syncthreads();
    auto get_lp = [&](int r, int c) -> float {
        return c < a.P ? t.c_lp[r * a.P + c] : rlp[(size_t)r * a.K2 + c];
    };
    auto get_idx = [&](int r, int c) -> int {
        return c < a.P ? t.c_idx[r * a.P + c] : ridx[(size_t)r * a.K2 + c];
    };
    if (lane == 0) {
        t.f_depth[0] = 1;
        t.f_rank[0] = 0;
        t.f_row[0] = 0;
        t.f_pscore[0] = 0.f;
        t.f_score[0] = 0.f + get_lp(0, 0);
    }
    __syncthreads();

    int n = 0;
    for (; n < a.B; ++n) {
        Cand best{0.f, 0u};
        for (int s = lane; s <= n; s += 64) {
            const int dp = t.f_depth[s];
            if (dp > 0) {
                Cand c{t.f_score[s], ((uint32_t)dp << 24) | ((uint32_t)s << 12) | (uint32_t)t.f_rank[s]};
                if (cand_before(c, best, t)) best = c;
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            Cand other{__shfl_xor(best.score, o), (uint32_t)__shfl_xor((int)best.meta, o)};
            if (cand_before(other, best, t)) best = other;
        }
        const int depth = c_depth(best.meta);
        if (depth == 0) break;   // frontier exhausted (excluded by argument checks)
        const int slot = c_slot(best.meta), rank = c_rank(best.meta);
        const int row = t.f_row[slot];
        const int tok = get_idx(row, rank);
        int child_row = -1;
        if (depth < a.gamma) {
            for (int m0 = 0; m0 < a.M; m0 += 64) {
                const int m = m0 + lane;
                const bool hit = m < a.M && t.tk[(depth - 1) * a.M + m] == tok;
                const unsigned long long bal = __ballot(hit);
                if (bal != 0ull) {
                    child_row = 1 + (depth - 1) * a.M + m0 + (__ffsll((long long)bal) - 1);
                    break;
                }
            }
        }
        __syncthreads();   // every lane has read the frontier before it changes
        if (lane == 0) {
            t.n_tok[n] = tok;
            t.n_par[n] = slot - 1;
            t.n_rank[n] = rank;
            t.n_dep[n] = depth;
            t.n_score[n] = best.score;
            t.n_crow[n] = child_row;
            if (rank + 1 < a.K2) {
                t.f_rank[slot] = rank + 1;
                t.f_score[slot] = t.f_pscore[slot] + get_lp(row, rank + 1);
            } else {
                t.f_depth[slot] = 0;
            }
            if (child_row >= 0) {
                t.f_depth[n + 1] = depth + 1;
                t.f_rank[n + 1] = 0;
                t.f_row[n + 1] = child_row;
                t.f_pscore[n + 1] = best.score;
                t.f_score[n + 1] = best.score + get_lp(child_row, 0);
            }
        }
        __syncthreads();
    }
    const size_t o = (size_t)seq * a.B;
    for (int i = lane; i < a.B; i += 64) {
        const bool ok = i < n;
        a.tok[o + i] = ok ? t.n_tok[i] : -1;
        a.par[o + i] = ok ? t.n_par[i] : -1;
        a.dep[o + i] = ok ? t.n_dep[i] : 0;
        a.score[o + i] = ok ? t.n_score[i] : neg_inf();
        if (a.crow != nullptr) a.crow[o + i] = ok ? t.n_crow[i] : -1;
    }
}

size_t tree_lds_bytes(int B, int gamma, int M, int Rs, int K2, int* cached_ranks) {
    const size_t fixed = tree_fixed_bytes(B, gamma, M);
    if (fixed > (size_t)kTreeLdsBudget) return 0;
    size_t P = ((size_t)kTreeLdsBudget - fixed) / ((size_t)8 * Rs);
    if (P > (size_t)K2) P = K2;
    if (cached_ranks) *cached_ranks = (int)P;
    return fixed + (size_t)8 * Rs * P;
}

hipError_t launch_build_tree(const int32_t* cond_idx, const float* cond_lp, const int32_t* topk_idx, int b,
                             int gamma, int k, int topk2, int B, int32_t* node_token, int32_t* node_parent,
                             int32_t* node_depth, float* node_score, int32_t* node_child_row,
                             hipStream_t stream) {
    const int Rs = 1 + (gamma - 1) * k;
    int P = 0;
    const size_t lds = tree_lds_bytes(B, gamma, k, Rs, topk2, &P);
    if (lds == 0) return hipErrorInvalidValue;
    TreeArgs a{cond_idx, cond_lp, topk_idx, gamma, k, topk2, B, Rs, P,
               node_token, node_parent, node_depth, node_score, node_child_row};
    hipLaunchKernelGGL(build_tree_kernel, dim3(b), dim3(64), lds, stream, a);
    return hipGetLastError();
}

}  // namespace tf

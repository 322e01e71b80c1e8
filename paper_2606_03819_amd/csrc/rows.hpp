// Conditional rows of one sequence (Appendix B, Part 1; the bigram table of
// the w/ 2-prev ablation in Ablations, Model Design).
//
// Single previous token (bigram == 0): row 0 is depth 1, conditioned on the
// root token; row 1 + (i-2)*M + m is depth i, conditioned on candidate m of
// depth i-1.  Previous bigram (bigram == 1): row 0 is depth 1, conditioned on
// (context token, root); rows 1..M are depth 2, conditioned on (root,
// candidate m of depth 1); from depth 3 on, row 1 + M + (i-3)*M*M + m2*M + m1
// is conditioned on (candidate m2 of depth i-2, candidate m1 of depth i-1).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tf {

// rows per sequence (int64: callers range-check before narrowing)
__host__ __device__ inline long long cond_rows(int gamma, int M, int bigram) {
    if (!bigram) return 1 + (long long)(gamma - 1) * M;
    if (gamma == 1) return 1;
    return 1 + (long long)M + (long long)(gamma - 2) * M * M;
}

struct RowTable {
    int Rs;       // rows per sequence
    int gamma;    // draft depth
    int M;        // stage-1 candidates per depth
    int bigram;   // 1: rows read the previous bigram

    __host__ __device__ int depth(int rl) const {
        if (rl == 0) return 1;
        if (!bigram) return 2 + (rl - 1) / M;
        return rl <= M ? 2 : 3 + (rl - 1 - M) / (M * M);
    }

    // Previous token `which` (0: the token right before the drafted position,
    // 1: the one before it; 1 only for bigram rows) of local row rl of
    // sequence s.  topk is [b, gamma, M].
    __device__ int prev_token(int s, int rl, int which, const int32_t* root, const int32_t* context,
                              const int32_t* topk) const {
        const int32_t* tk = topk + (size_t)s * gamma * M;
        if (!bigram) return rl == 0 ? root[s] : tk[rl - 1];
        if (rl == 0) return which == 0 ? root[s] : context[s];
        if (rl <= M) return which == 0 ? tk[rl - 1] : root[s];
        const int q = rl - 1 - M;
        const int i = 3 + q / (M * M);
        const int r2 = q - (i - 3) * M * M;
        return which == 0 ? tk[(i - 2) * M + r2 % M] : tk[(i - 3) * M + r2 / M];
    }
};

inline RowTable make_row_table(int gamma, int M, int bigram) {
    return RowTable{(int)cond_rows(gamma, M, bigram), gamma, M, bigram};
}

}  // namespace tf

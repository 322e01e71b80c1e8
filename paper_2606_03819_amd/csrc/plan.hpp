// Launch plans and workspace layout shared by the C ABI and the launchers.
// Host-only; every function here is a pure function of the shapes, so the
// workspace size the caller is told and the layout the kernels use agree.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "limits.hpp"

namespace tf {

constexpr int kMaxSplits = 2048;       // vocabulary slices (partials per row); kMaxSplits*kKeep <= merge capacity
constexpr int kTargetWorkgroups = 512; // two 256-thread workgroups per CU on 256 CUs
constexpr int kMaxTopk = 1024;         // longest top-k list the merge kernel sorts
constexpr int kMaxBudget = 4095;       // tree nodes per sequence
constexpr int kMaxSplitK = 8;          // k-parts of a SwiGLU product

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

struct GemmPlan {
    int NT;       // 32-row activation tiles per workgroup
    int WM;       // 32-row weight tiles per wave (bf16)
    int chunk;    // weight tiles per workgroup
    int nrb;      // activation-row blocks
    int ntiles;   // 32-row weight tiles
    int nchunks;  // workgroup chunks of weight tiles (= vocabulary slices for the LM head)
    int nkp;      // k-parts
    bool wnt;     // non-temporal weight loads (weights read by one row block only)
    int blocks() const { return nchunks * nkp * nrb; }
};

// Pipeline depth (k-chunks of loads in flight per wave) when a single row
// block reads each weight once at NT = 4, and otherwise; the launchers pick
// the kernel instance from NT and wnt.
#ifndef TF_PIPE_SINGLE_NT4
#define TF_PIPE_SINGLE_NT4 3
#endif
#ifndef TF_PIPE_DEFAULT
#define TF_PIPE_DEFAULT 2
#endif
#ifndef TF_MLP_WNT
#define TF_MLP_WNT 0
#endif

inline int plan_nt(int rows) { return rows <= 32 ? 1 : (rows <= 64 ? 2 : 4); }
// one weight tile per wave at NT = 4 keeps two workgroups per CU
inline int plan_wm(int NT) { return NT == 4 ? 1 : 2; }

// LM-head tile shape (weight tiles per wave) per activation-tile count.
#ifndef TF_LM_WM_NT1
#define TF_LM_WM_NT1 2
#endif
#ifndef TF_LM_WM_NT2
#define TF_LM_WM_NT2 2
#endif
#ifndef TF_LM_WM_NT4
#define TF_LM_WM_NT4 1
#endif
inline int lm_wm(int NT) { return NT == 1 ? TF_LM_WM_NT1 : (NT == 2 ? TF_LM_WM_NT2 : TF_LM_WM_NT4); }

// LM head: one chunk of the vocabulary per workgroup, so every workgroup
// streams the same bytes.  fp32: 32 rows and 8 tiles (256 tokens) per workgroup.
inline GemmPlan lm_plan(int rows, int V, bool bf16) {
    GemmPlan p;
    p.NT = bf16 ? plan_nt(rows) : 1;
    p.WM = bf16 ? lm_wm(p.NT) : 2;
    p.chunk = 4 * p.WM;
    p.nrb = cdiv(rows, 32 * p.NT);
    p.ntiles = cdiv(V, 32);
    p.nchunks = cdiv(p.ntiles, p.chunk);
    p.nkp = 1;
    p.wnt = p.nrb == 1;
    return p;
}

// SwiGLU products (bf16): few weight tiles, so the reduction is split over
// up to kMaxSplitK workgroups until about kTargetWorkgroups are in flight.
inline GemmPlan mlp_plan(int rows, int ntiles, int K) {
    GemmPlan p;
    p.NT = plan_nt(rows);
    p.WM = plan_wm(p.NT);
    p.chunk = 4 * p.WM;
    p.nrb = cdiv(rows, 32 * p.NT);
    p.ntiles = ntiles;
    p.nchunks = cdiv(ntiles, p.chunk);
    int nkp = kTargetWorkgroups / (p.nchunks * p.nrb);
    const int nkc = cdiv(K, 64);
    if (nkp > kMaxSplitK) nkp = kMaxSplitK;
    if (nkp > nkc) nkp = nkc;
    if (nkp < 1) nkp = 1;
    p.nkp = nkp;
    p.wnt = TF_MLP_WNT && p.nrb == 1;
    return p;
}

inline size_t mlp_partial_floats(const GemmPlan& p) {
    if (p.nkp == 1) return 0;
    return (size_t)p.nchunks * p.nrb * p.nkp * (4 * p.WM * p.NT * 16 * 64);
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Workspace {
    size_t diag, part, ht, et, act, hp, mlp_part, counters, total;
    int ncounters;
};

// Layout: [diag counters | LM-head partials | normalised h | normalised
// embeddings | SwiGLU activation | h' | split-K partials | split-K counters].
// Stage 1 uses the first two only.
inline Workspace workspace_layout(int b, int gamma, int d, int I, int V, int k, bool bf16) {
    const int R = 1 + (gamma - 1) * k;
    const size_t es = bf16 ? 2 : 4;
    const int rows1 = b * gamma, rows2 = b * R;
    const GemmPlan p1 = lm_plan(rows1, V, bf16), p2 = lm_plan(rows2, V, bf16);
    const size_t part1 = (size_t)rows1 * p1.nchunks, part2 = (size_t)rows2 * p2.nchunks;
    Workspace w;
    size_t off = 0;
    w.diag = off;
    off += 256;
    w.part = off;
    off += align256((part1 > part2 ? part1 : part2) * kPartStride * 4);
    w.ht = off;
    off += align256((size_t)rows1 * d * es);
    w.et = off;
    off += align256((size_t)rows2 * d * es);
    w.act = off;
    off += align256((size_t)rows2 * I * es);
    w.hp = off;
    off += align256((size_t)rows2 * d * es);
    size_t mp = 0;
    w.ncounters = 0;
    if (bf16) {
        const GemmPlan pg = mlp_plan(rows2, cdiv(I, 16), 2 * d), pd = mlp_plan(rows2, cdiv(d, 32), I);
        const size_t a = mlp_partial_floats(pg), c = mlp_partial_floats(pd);
        mp = a > c ? a : c;
        w.ncounters = pg.nchunks * pg.nrb + pd.nchunks * pd.nrb;
    }
    w.mlp_part = off;
    off += align256(mp * 4);
    w.counters = off;
    off += align256((size_t)w.ncounters * 4);
    w.total = off;
    return w;
}

}  // namespace tf

// Launch plans and workspace layout shared by the C ABI and the launchers.
// Host-only; every function here is a pure function of the shapes, so the
// workspace size the caller is told and the layout the kernels use agree.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "limits.hpp"

namespace tf {

constexpr int kMaxSplits = 512;        // vocabulary slices per row block (partials per row)
constexpr int kTargetWorkgroups = 512; // two 256-thread workgroups per CU on 256 CUs
constexpr int kMaxTopk = 1024;         // longest top-k list the merge kernel sorts
constexpr int kMaxBudget = 4095;       // tree nodes per sequence

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

struct LmPlan {
    int NT;       // 32-row activation tiles per workgroup (bf16 path)
    int nrb;      // activation-row blocks
    int ntiles;   // 32-row vocabulary tiles
    int nsplit;   // vocabulary slices
};

inline LmPlan lm_plan(int rows, int V, bool bf16) {
    LmPlan p;
    if (bf16) {
        p.NT = rows <= 32 ? 1 : (rows <= 64 ? 2 : 4);
    } else {
        p.NT = 1;
    }
    p.nrb = cdiv(rows, 32 * p.NT);
    p.ntiles = cdiv(V, 32);
    int ns = kTargetWorkgroups / p.nrb;
    if (ns < 1) ns = 1;
    if (ns > p.ntiles) ns = p.ntiles;
    if (ns > kMaxSplits) ns = kMaxSplits;
    p.nsplit = ns;
    return p;
}

// Plan for the streaming products of the SwiGLU (no per-row state across
// tiles, so every slice is independent).
inline LmPlan mlp_plan(int rows, int ntiles) {
    LmPlan p;
    p.NT = rows <= 32 ? 1 : (rows <= 64 ? 2 : 4);
    p.nrb = cdiv(rows, 32 * p.NT);
    p.ntiles = ntiles;
    int ns = kTargetWorkgroups / p.nrb;
    if (ns < 1) ns = 1;
    if (ns > ntiles) ns = ntiles;
    p.nsplit = ns;
    return p;
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Workspace {
    size_t diag, part, ht, et, act, hp, total;
};

// Layout: [diag counters | partials | normalised h | normalised embeddings |
//          SwiGLU activation | h'].  Stage 1 uses the first two only.
inline Workspace workspace_layout(int b, int gamma, int d, int I, int V, int k, bool bf16) {
    const int R = 1 + (gamma - 1) * k;
    const size_t es = bf16 ? 2 : 4;
    const int rows1 = b * gamma, rows2 = b * R;
    const LmPlan p1 = lm_plan(rows1, V, bf16), p2 = lm_plan(rows2, V, bf16);
    const size_t part1 = (size_t)rows1 * p1.nsplit, part2 = (size_t)rows2 * p2.nsplit;
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
    w.total = off;
    return w;
}

}  // namespace tf

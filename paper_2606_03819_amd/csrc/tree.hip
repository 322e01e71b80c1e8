// OPT-Tree selection (Appendix B, Part 2) on the GPU, one workgroup per
// sequence: every wave preloads the sequence's rows into LDS, then one wave
// selects.
//
// The paper's queue holds every child of every expanded node.  Because each
// conditional row arrives sorted, a node's children are popped in row order,
// so the frontier only needs each expanded node's best child not yet popped:
// slot 0 holds the root's next child, slot n+1 node n's next child.  A pop is
// an argmax over at most B+1 slots, then the popped slot advances to its next
// sibling and, if the popped token is a stage-1 candidate of its depth, slot
// n+1 opens on the first entry of its row.
//
// Up to 1024 slots the frontier lives in registers (slot s in lane s % 64)
// and the argmax is a DPP maximum of the lanes' score keys; only an exact
// score tie between lanes runs the full comparison.  Larger budgets keep the
// frontier in LDS.  Below 128 slots, with every row in LDS, the stage-1
// candidates and the rows' first log-probs sit in registers too and runs of
// siblings from one slot are popped in one step (see the lane-table kernel).
//
// Candidate order: path score (fp32 running sum) desc, depth asc, then the
// lexicographic order of the rank paths (ranks of the nodes in their parents'
// rows, root to node).  Siblings compare by rank; nodes of different parents
// at equal depth compare at the first ancestor where their paths diverge.
#include "common.hpp"
#include "launch.hpp"
#include "plan.hpp"
#include "rows.hpp"

namespace tf {

// LDS for the node table, the frontier and the cached leading ranks of every
// row (gfx950 gives a workgroup up to 160 KB).
constexpr int kTreeLdsBudget = 144 * 1024;
constexpr int kTreeThreads = 1024;  // all waves preload; wave 0 alone selects
constexpr int kTreeRegSlots = 16;   // frontier slots per lane held in registers

// Row tables the selection expands into.  Single: a node whose token is
// candidate m of its depth i expands into row 1 + (i-1)*M + m.  Marginal:
// every node above depth gamma expands into the marginal row of the next
// depth.  Bigram (w/ 2-prev): row 1 + m at depth 1, else
// 1 + M + (i-2)*M*M + m2*M + m with m2 the parent's candidate index.
constexpr int kTreeSingle = 0;
constexpr int kTreeMarginal = 1;
constexpr int kTreeBigram = 2;

struct TreeArgs {
    const int32_t* cond_idx;
    const float* cond_lp;
    const int32_t* topk;
    int gamma, M, K2, B, Rs, P;   // P = leading ranks of each row cached in LDS
    int mode;                     // kTreeSingle, kTreeMarginal or kTreeBigram
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

// Orders this wave's LDS accesses (the selection runs in one wave, whose LDS
// operations complete in issue order).
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Rows of this sequence's leading ranks and its stage-1 candidates into LDS,
// every thread with several independent loads in flight.
__device__ __forceinline__ void tree_preload(const TreeArgs& a, const TreeLds& t, int seq, const float* rlp,
                                             const int32_t* ridx) {
    const int tid = threadIdx.x;
    for (int s = tid; s <= a.B; s += kTreeThreads) t.f_depth[s] = 0;
    if (a.mode != kTreeMarginal)
        for (int e = tid; e < a.gamma * a.M; e += kTreeThreads) t.tk[e] = a.topk[(size_t)seq * a.gamma * a.M + e];
    const int ncache = a.Rs * a.P;
    for (int e0 = tid; e0 < ncache; e0 += 4 * kTreeThreads) {
        float lp[4];
        int ix[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * kTreeThreads;
            const int r = e / a.P, c = e - r * a.P;
            const size_t gi = e < ncache ? (size_t)r * a.K2 + c : 0;
            lp[u] = rlp[gi];
            ix[u] = ridx[gi];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * kTreeThreads;
            if (e < ncache) {
                t.c_lp[e] = lp[u];
                t.c_idx[e] = ix[u];
            }
        }
    }
}

// Child row of a node popped from row `row` (see the row tables above), -1
// if it does not expand.  In bigram mode the parent's candidate index is read
// off `row`: a depth-2 row 1 + m2, a deeper row 1 + M + ... + m2*M + m1 whose
// last index is the parent's.  Uniform across the wave.
__device__ __forceinline__ int tree_child_row(const TreeArgs& a, const TreeLds& t, int depth, int tok, int row,
                                              int lane) {
    if (depth >= a.gamma) return -1;
    if (a.mode == kTreeMarginal) return depth;
    for (int m0 = 0; m0 < a.M; m0 += 64) {
        const int m = m0 + lane;
        const bool hit = m < a.M && t.tk[(depth - 1) * a.M + m] == tok;
        const unsigned long long bal = __ballot(hit);
        if (bal != 0ull) {
            const int mc = m0 + (__ffsll((long long)bal) - 1);
            if (a.mode == kTreeSingle) return 1 + (depth - 1) * a.M + mc;
            if (depth == 1) return 1 + mc;
            const int mp = depth == 2 ? row - 1 : (row - 1 - a.M) % a.M;
            return 1 + a.M + (depth - 2) * a.M * a.M + mp * a.M + mc;
        }
    }
    return -1;
}

// Node table -> outputs (slots past the last pop get the empty values).
__device__ __forceinline__ void tree_store(const TreeArgs& a, const TreeLds& t, int seq, int n, int lane) {
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

// Wave maximum through DPP: quad swaps, half-row and row mirrors give every
// lane its 16-lane row maximum; four readlanes combine the rows.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return max(max(r0, r1), max(r2, r3));
}

// Best candidate of the wave under the full order (butterfly).
__device__ __forceinline__ Cand wave_best(Cand best, const TreeLds& t) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        Cand other{__shfl_xor(best.score, o), (uint32_t)__shfl_xor((int)best.meta, o)};
        if (cand_before(other, best, t)) best = other;
    }
    return best;
}

// Frontier in registers: slot s = lane + 64*j, j < FS (B + 1 <= 64*FS).
// ALL: every rank of every row is cached (P = K2), so the row reads are LDS
// reads only (a read that may go to either memory compiles to a flat load,
// whose latency is that of the vector-memory path).
template <int FS, bool ALL>
__global__ __launch_bounds__(kTreeThreads) void build_tree_reg_kernel(TreeArgs a) {
    extern __shared__ __align__(16) unsigned char dyn[];
    const TreeLds t = tree_lds(dyn, a);
    const int seq = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int32_t* ridx = a.cond_idx + (size_t)seq * a.Rs * a.K2;
    const float* rlp = a.cond_lp + (size_t)seq * a.Rs * a.K2;
    tree_preload(a, t, seq, rlp, ridx);
    __syncthreads();
    if (threadIdx.x >= 64) return;
    auto get_lp = [&](int r, int c) -> float {
        if constexpr (ALL) return t.c_lp[r * a.P + c];
        return c < a.P ? t.c_lp[r * a.P + c] : rlp[(size_t)r * a.K2 + c];
    };
    auto get_idx = [&](int r, int c) -> int {
        if constexpr (ALL) return t.c_idx[r * a.P + c];
        return c < a.P ? t.c_idx[r * a.P + c] : ridx[(size_t)r * a.K2 + c];
    };
    float f_score[FS], f_pscore[FS];
    int f_depth[FS], f_rank[FS], f_row[FS];
#pragma unroll
    for (int j = 0; j < FS; ++j) {
        f_score[j] = f_pscore[j] = 0.f;
        f_depth[j] = f_rank[j] = f_row[j] = 0;
    }
    {
        const float first = get_lp(0, 0);
        if (lane == 0) {
            f_depth[0] = 1;
            f_score[0] = 0.f + first;   // a -0.0 log-prob scores +0.0, as in the LDS kernel
        }
    }

    int n = 0;
    for (; n < a.B; ++n) {
        Cand lb{0.f, 0u};
#pragma unroll
        for (int j = 0; j < FS; ++j)
            if (f_depth[j] > 0) {
                const Cand c{f_score[j],
                             ((uint32_t)f_depth[j] << 24) | ((uint32_t)(lane + 64 * j) << 12) | (uint32_t)f_rank[j]};
                if (cand_before(c, lb, t)) lb = c;
            }
        // keys on score + 0: -0.0 and +0.0 tie here as they do in cand_before
        const uint32_t key = c_depth(lb.meta) != 0 ? f32_key(lb.score + 0.f) : 0u;
        const uint32_t mx = wave_max_u32(key);
        if (mx == 0u) break;   // frontier exhausted: rows too short for B nodes; the rest stay -1
        const unsigned long long tied = __ballot(key == mx);
        Cand best;
        if (__popcll(tied) == 1) {
            const int wl = __ffsll((long long)tied) - 1;
            best.score = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lb.score), wl));
            best.meta = (uint32_t)__builtin_amdgcn_readlane((int)lb.meta, wl);
        } else {   // exact score tie between lanes: the full order decides
            best = wave_best(key == mx ? lb : Cand{0.f, 0u}, t);
        }
        const int depth = c_depth(best.meta), slot = c_slot(best.meta), rank = c_rank(best.meta);
        const int owner = slot & 63, js = slot >> 6;
        int my_row = 0;
        float my_ps = 0.f;
#pragma unroll
        for (int j = 0; j < FS; ++j)
            if (j == js) {
                my_row = f_row[j];
                my_ps = f_pscore[j];
            }
        const int row = __builtin_amdgcn_readlane(my_row, owner);
        const float pscore = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_ps), owner));
        // both reads of the popped row together, so that ranks past the LDS
        // cache cost one memory round trip per pop rather than two
        const int tok = get_idx(row, rank);
        const bool more = rank + 1 < a.K2;
        const float next_lp = more ? get_lp(row, rank + 1) : 0.f;
        const int child_row = tree_child_row(a, t, depth, tok, row, lane);
        if (lane == 0) {
            t.n_tok[n] = tok;
            t.n_par[n] = slot - 1;
            t.n_rank[n] = rank;
            t.n_dep[n] = depth;
            t.n_score[n] = best.score;
            t.n_crow[n] = child_row;
        }
        // the popped slot moves to its next sibling (owner lane)
        if (lane == owner) {
#pragma unroll
            for (int j = 0; j < FS; ++j)
                if (j == js) {
                    f_rank[j] = rank + 1;
                    f_score[j] = pscore + next_lp;
                    f_depth[j] = more ? f_depth[j] : 0;
                }
        }
        // an expandable node opens slot n + 1 on the first entry of its row
        if (child_row >= 0) {
            const float first = get_lp(child_row, 0);
            const int jn = (n + 1) >> 6;
            if (lane == ((n + 1) & 63)) {
#pragma unroll
                for (int j = 0; j < FS; ++j)
                    if (j == jn) {
                        f_depth[j] = depth + 1;
                        f_rank[j] = 0;
                        f_row[j] = child_row;
                        f_pscore[j] = best.score;
                        f_score[j] = best.score + first;
                    }
            }
        }
        wave_lds_sync();   // node n is in LDS before a later tie walk reads it
    }
    tree_store(a, t, seq, n, lane);
}

// Frontier in LDS, for budgets beyond the register frontier.
__global__ __launch_bounds__(kTreeThreads) void build_tree_kernel(TreeArgs a) {
    extern __shared__ __align__(16) unsigned char dyn[];
    const TreeLds t = tree_lds(dyn, a);
    const int seq = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int32_t* ridx = a.cond_idx + (size_t)seq * a.Rs * a.K2;
    const float* rlp = a.cond_lp + (size_t)seq * a.Rs * a.K2;
    tree_preload(a, t, seq, rlp, ridx);
    __syncthreads();
    if (threadIdx.x >= 64) return;
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
    wave_lds_sync();

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
        best = wave_best(best, t);
        const int depth = c_depth(best.meta);
        if (depth == 0) break;   // frontier exhausted: rows too short for B nodes; the rest stay -1
        const int slot = c_slot(best.meta), rank = c_rank(best.meta);
        const int row = t.f_row[slot];
        // both reads of the popped row together (one round trip past the cache)
        const int tok = get_idx(row, rank);
        const float next_lp = rank + 1 < a.K2 ? get_lp(row, rank + 1) : 0.f;
        const int child_row = tree_child_row(a, t, depth, tok, row, lane);
        wave_lds_sync();   // every lane has read the frontier before it changes
        if (lane == 0) {
            t.n_tok[n] = tok;
            t.n_par[n] = slot - 1;
            t.n_rank[n] = rank;
            t.n_dep[n] = depth;
            t.n_score[n] = best.score;
            t.n_crow[n] = child_row;
            if (rank + 1 < a.K2) {
                t.f_rank[slot] = rank + 1;
                t.f_score[slot] = t.f_pscore[slot] + next_lp;
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
        wave_lds_sync();
    }
    tree_store(a, t, seq, n, lane);
}

// ------------------------------------------------ lane tables and sibling runs
//
// For budgets below 128 with every rank of every row in LDS, the selecting
// wave also keeps in registers the stage-1 candidates (flat index
// (depth-1)*M + m in lane index % 64 of register index / 64) and the first
// log-prob of every row (row r in lane r % 64 of register r / 64).  Each
// frontier slot holds its candidate's key, parent score, depth and rank,
// entry index and the first row of its entries' children (single rows:
// 1 + (depth-1)*M; bigram rows: 1 + M + (depth-2)*M^2 + m2*M, m2 the
// parent's candidate index; marginal: the next depth's row).  At the top of
// every pop each lane reads its slots' tokens and next log-probs from LDS,
// so that the read overlaps the wave maximum; the popped node's child row is
// then a ballot of the candidate registers against its token and the first
// log-prob of that row a readlane.
//
// Sibling runs.  When a pop comes from the same slot as the one before, the
// best key of the other slots (a second wave maximum) bounds what may come
// next: the slot's following siblings are popped in order for as long as
// each beats that bound and every child opened by the siblings popped before
// it (ties stop the run; the next pop then takes the full order).  All 64
// lanes evaluate the next 64 siblings at once (score, child row, child key),
// a prefix maximum over the lanes gives the run's length, and the run is
// committed in one step: its nodes written by their lanes, its children
// moved into their slots by a lane permutation.  Nodes go to the outputs as
// they are popped; LDS keeps only their parents and ranks, which the full
// order reads on ties.  Rows whose leading entries
// dominate the frontier (flat conditional distributions make star-shaped
// trees) then cost one step instead of one pop per node.
//
// A node's score is the key's float: scores are sums of a +0.0 root score
// and log-probs, never -0.0, so the key (which folds -0.0 into +0.0) loses
// nothing.
constexpr int kLaneSlotsMax = 8;   // frontier slots per lane (B <= 512)
constexpr int kLaneTabMax = 4;     // table registers (rows and candidates <= 256)

// LDS of the lane-table kernel: the nodes' parents and ranks, then the
// leading P ranks of every row (ids and log-probs), P as many as fit.
__host__ __device__ inline int tree_lane_ranks(int B, int Rs, int K2) {
    const long long room = (long long)kTreeLdsBudget - 8ll * B;
    if (room < 8ll * Rs) return 0;
    const long long P = room / (8ll * Rs);
    return (int)(P < K2 ? P : K2);
}
__host__ __device__ inline size_t tree_lane_lds_bytes(int B, int Rs, int P) {
    return (size_t)8 * B + (size_t)8 * Rs * P;
}

// Key of a candidate score: -0.0 keys as +0.0, as cand_before compares.
__device__ __forceinline__ uint32_t score_key(float s) {
    const int u = __float_as_int(s + 0.f);
    return (uint32_t)(u ^ ((u >> 31) | (int)0x80000000));   // f32_key
}

// Inclusive prefix maximum over the wave's lanes (0 is the identity).
__device__ __forceinline__ uint32_t wave_prefix_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, true));   // row_shr:1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, true));   // row_shr:2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, true));   // row_shr:4
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, true));   // row_shr:8
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));  // row_bcast:15
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));  // row_bcast:31
    return v;
}

// FS frontier slots per lane (B <= 64 * FS: a child slot past the last one,
// opened by the B-th pop, is never popped and is dropped), T table
// registers; ALL: every rank of every
// row is in LDS (a.P == a.K2), else ranks from a.P on are read from memory
// (only when some lane needs one: a ballot guards those loads).
template <int FS, int T, bool ALL>
__global__ __launch_bounds__(kTreeThreads) void build_tree_lane_kernel(TreeArgs a) {
    extern __shared__ __align__(16) unsigned char dyn[];
    TreeLds t{};   // parents and ranks of the nodes (for ties), and the rows' leading ranks
    {
        int32_t* p = reinterpret_cast<int32_t*>(dyn);
        t.n_par = p; p += a.B;
        t.n_rank = p; p += a.B;
        t.c_lp = reinterpret_cast<float*>(p); p += a.Rs * a.P;
        t.c_idx = p;
    }
    const int nent = a.Rs * a.K2;   // entries in memory
    const int ncache = a.Rs * a.P;  // entries in LDS
    const int seq = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int32_t* ridx = a.cond_idx + (size_t)seq * nent;
    const float* rlp = a.cond_lp + (size_t)seq * nent;
    // outputs of this sequence, written as the nodes are popped
    int32_t* o_tok = a.tok + (size_t)seq * a.B;
    int32_t* o_par = a.par + (size_t)seq * a.B;
    int32_t* o_dep = a.dep + (size_t)seq * a.B;
    float* o_score = a.score + (size_t)seq * a.B;
    int32_t* o_crow = a.crow != nullptr ? a.crow + (size_t)seq * a.B : nullptr;
    const bool marginal = a.mode == kTreeMarginal;
    const int nflat = marginal ? 0 : a.gamma * a.M;
    // first child row of the entries of a slot opened by a node of depth d
    // and candidate index m: c0 + c1*d + c2*m
    const int c0 = a.mode == kTreeBigram ? 1 + a.M - a.M * a.M : 1;
    const int c1 = a.mode == kTreeSingle ? a.M : a.mode == kTreeBigram ? a.M * a.M : 1;
    const int c2 = a.mode == kTreeBigram ? a.M : 0;

    // the selecting wave's tables, loaded beside the rows
    int tkr[T], tkd[T];
    float rfr[T];
    if (tid < 64) {
#pragma unroll
        for (int r = 0; r < T; ++r) {
            const int f = 64 * r + lane;
            tkr[r] = f < nflat ? a.topk[(size_t)seq * nflat + f] : -1;
            tkd[r] = f < nflat ? f / a.M + 1 : 0;
            rfr[r] = rlp[(size_t)min(f, a.Rs - 1) * a.K2];
        }
    }
    for (int e0 = tid; e0 < ncache; e0 += 4 * kTreeThreads) {
        float lp[4];
        int ix[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = min(e0 + u * kTreeThreads, ncache - 1);
            int ge = e;
            if constexpr (!ALL) {
                const int r = e / a.P;
                ge = r * a.K2 + (e - r * a.P);
            }
            lp[u] = rlp[ge];
            ix[u] = ridx[ge];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * kTreeThreads;
            if (e < ncache) {
                t.c_lp[e] = lp[u];
                t.c_idx[e] = ix[u];
            }
        }
    }
    __syncthreads();
    if (tid >= 64) return;

    // frontier: slot s = lane + 64*j; key 0 = empty
    uint32_t skey[FS];
    float sps[FS];
    int sdr[FS], sea[FS], slc[FS], scb[FS];   // sdr = depth << 16 | rank; sea / slc = entry index in memory / LDS
#pragma unroll
    for (int j = 0; j < FS; ++j) {
        skey[j] = 0u;
        sps[j] = 0.f;
        sdr[j] = sea[j] = slc[j] = scb[j] = 0;
    }
    {
        const float first = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(rfr[0])));
        if (lane == 0) {
            skey[0] = score_key(0.f + first);
            sdr[0] = 1 << 16;
            scb[0] = 1;   // depth-1 entries expand into rows 1 + m (marginal: row 1)
        }
    }

    int n = 0, prev = -1;
    while (n < a.B) {
        // every slot's token and next log-prob, read while the maximum runs
        int tokv[FS];
        float nlpv[FS];
#pragma unroll
        for (int j = 0; j < FS; ++j) {
            tokv[j] = t.c_idx[min(slc[j], ncache - 1)];
            nlpv[j] = t.c_lp[min(slc[j] + 1, ncache - 1)];
        }
        if constexpr (!ALL) {
            // ranks past the LDS copy come from memory (a slot at rank P - 1 needs its next log-prob)
            bool far = false;
#pragma unroll
            for (int j = 0; j < FS; ++j) far = far || (skey[j] != 0u && (sdr[j] & 0xffff) + 1 >= a.P);
            if (__ballot(far) != 0ull) {
#pragma unroll
                for (int j = 0; j < FS; ++j) {
                    const int rk = sdr[j] & 0xffff;
                    if (skey[j] != 0u && rk >= a.P) tokv[j] = ridx[sea[j]];
                    if (skey[j] != 0u && rk + 1 >= a.P) nlpv[j] = rlp[min(sea[j] + 1, nent - 1)];
                }
            }
        }
        asm volatile("" ::: "memory");   // keep the reads above the maximum
        uint32_t lk = skey[0];
        int lj = 0, ldup = 0;
#pragma unroll
        for (int j = 1; j < FS; ++j) {
            if (skey[j] > lk) {
                lk = skey[j];
                lj = j;
                ldup = 0;
            } else if (skey[j] == lk) {
                ldup = 1;
            }
        }
        const uint32_t mx = wave_max_u32(lk);
        if (mx == 0u) break;   // frontier exhausted: rows too short for B nodes; the rest stay -1
        const unsigned long long tied = __ballot(lk == mx);
        int wl, js;
        if (__builtin_expect(__popcll(tied) == 1 &&
                                 (FS == 1 || __builtin_amdgcn_readlane(ldup, __ffsll((long long)tied) - 1) == 0),
                             1)) {
            wl = __ffsll((long long)tied) - 1;
            js = FS == 1 ? 0 : __builtin_amdgcn_readlane(lj, wl);
        } else {   // exact score tie: the full order decides (rank paths from the node table)
            Cand lb{0.f, 0u};
#pragma unroll
            for (int j = 0; j < FS; ++j)
                if (skey[j] == mx) {
                    const Cand c{key_f32(skey[j]), ((uint32_t)(sdr[j] >> 16) << 24) |
                                                       ((uint32_t)(lane + 64 * j) << 12) | (uint32_t)(sdr[j] & 0xffff)};
                    if (cand_before(c, lb, t)) lb = c;
                }
            const Cand best = wave_best(lb, t);
            wl = __builtin_amdgcn_readfirstlane(c_slot(best.meta) & 63);
            js = __builtin_amdgcn_readfirstlane(c_slot(best.meta) >> 6);
        }
        // the winning slot's fields
        float g_ps = sps[0], g_nl = nlpv[0];
        int g_dr = sdr[0], g_cb = scb[0], g_tok = tokv[0], g_ea = sea[0], g_lc = slc[0];
#pragma unroll
        for (int j = 1; j < FS; ++j)
            if (j == js) {
                g_ps = sps[j];
                g_nl = nlpv[j];
                g_dr = sdr[j];
                g_cb = scb[j];
                g_tok = tokv[j];
                g_ea = sea[j];
                g_lc = slc[j];
            }
        const float score = key_f32(mx);
        const int dr = __builtin_amdgcn_readlane(g_dr, wl);
        const int cb = __builtin_amdgcn_readlane(g_cb, wl);
        const int tok = __builtin_amdgcn_readlane(g_tok, wl);
        const int depth = dr >> 16, rank = dr & 0xffff;
        const int slot = wl + 64 * js;
        const bool more = rank + 1 < a.K2;
        // child row: the node's token among the candidates of its depth
        int f = -1;
#pragma unroll
        for (int r = T - 1; r >= 0; --r) {
            const unsigned long long hit = __ballot(((tkr[r] ^ tok) | (tkd[r] ^ depth)) == 0);
            if (hit != 0ull) f = 64 * r + __ffsll((long long)hit) - 1;
        }
        const int m = marginal ? 0 : f - (depth - 1) * a.M;
        const int child_row = depth < a.gamma && (marginal || f >= 0) ? cb + m : -1;
        float cfirst = 0.f;
        if (child_row >= 0) {
            cfirst = rfr[0];
#pragma unroll
            for (int r = 1; r < T; ++r)
                if (r == (child_row >> 6)) cfirst = rfr[r];
            cfirst = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cfirst), child_row & 63));
        }
        const float cs = score + cfirst;
        const uint32_t ck = child_row >= 0 ? score_key(cs) : 0u;

        // a second pop in a row from this slot: try a sibling run
        int L = 1;
        if (slot == prev && more && n + 1 < a.B) {
            uint32_t lo = 0u;
#pragma unroll
            for (int j = 0; j < FS; ++j) lo = max(lo, lane + 64 * j == slot ? 0u : skey[j]);
            const uint32_t k2 = wave_max_u32(lo);
            const float ps = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g_ps), wl));
            const float nl = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g_nl), wl));
            const uint32_t ka = score_key(ps + nl);
            if (ka > k2 && ka > ck) {
                const int ea = __builtin_amdgcn_readlane(g_ea, wl);
                const int lc = __builtin_amdgcn_readlane(g_lc, wl);
                // sibling i of this pop in lane i
                const bool valid = rank + lane < a.K2;
                float lpi;
                int toki;
                if (ALL || rank + 63 < a.P) {
                    const int e = min(lc + lane, ncache - 1);
                    lpi = t.c_lp[e];
                    toki = t.c_idx[e];
                } else {
                    const int e = min(ea + lane, nent - 1);
                    const int c = min(lc + lane, ncache - 1);
                    lpi = t.c_lp[c];
                    toki = t.c_idx[c];
                    if (rank + lane >= a.P) {   // past the LDS copy
                        lpi = rlp[e];
                        toki = ridx[e];
                    }
                }
                const float si = ps + lpi;
                const uint32_t ki = valid ? score_key(si) : 0u;
                int mi = -1;
                if (depth < a.gamma) {
                    if (marginal) {
                        mi = 0;
                    } else {
                        for (int q = 0; q < a.M; ++q) {
                            const int fq = (depth - 1) * a.M + q;
                            int cand = tkr[0];
#pragma unroll
                            for (int r = 1; r < T; ++r)
                                if (r == (fq >> 6)) cand = tkr[r];
                            cand = __builtin_amdgcn_readlane(cand, fq & 63);
                            mi = mi < 0 && toki == cand ? q : mi;
                        }
                    }
                }
                const int crowi = mi >= 0 ? cb + mi : -1;
                const float cfi = t.c_lp[max(crowi, 0) * a.P];   // rank 0 of a row is always in LDS
                const uint32_t cki = crowi >= 0 && valid ? score_key(si + cfi) : 0u;
                // a sibling is popped if it beats the other slots and every child opened before it
                const uint32_t before = (uint32_t)__builtin_amdgcn_update_dpp(
                    0, (int)wave_prefix_max_u32(cki), 0x138, 0xF, 0xF, true);   // wave_shr:1
                const bool ok = lane == 0 || (ki > max(k2, before) && lane < a.B - n);
                const unsigned long long bad = ~__ballot(ok);
                L = bad == 0ull ? 63 : min(__ffsll((long long)bad) - 1, 63);
                // the run's nodes
                if (lane < L) {
                    t.n_par[n + lane] = slot - 1;
                    t.n_rank[n + lane] = rank + lane;
                    o_tok[n + lane] = toki;
                    o_par[n + lane] = slot - 1;
                    o_dep[n + lane] = depth;
                    o_score[n + lane] = si;
                    if (o_crow != nullptr) o_crow[n + lane] = crowi;
                }
                // their children into slots n + 1 + i
                const int ncbi = c0 + c1 * depth + c2 * mi;
                const int srci_ea = max(crowi, 0) * a.K2, srci_lc = max(crowi, 0) * a.P;
#pragma unroll
                for (int j = 0; j < FS; ++j) {
                    if (64 * j + 63 < n + 1 || 64 * j > n + L) continue;   // no slot of this register changes
                    const int s = lane + 64 * j;
                    const int src = ((s - n - 1) & 63) << 2;
                    const uint32_t pk = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)cki);
                    const float pps = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(si)));
                    const int pea = __builtin_amdgcn_ds_bpermute(src, srci_ea);
                    const int plc = __builtin_amdgcn_ds_bpermute(src, srci_lc);
                    const int pcb = __builtin_amdgcn_ds_bpermute(src, ncbi);
                    const bool in = s >= n + 1 && s <= n + L;
                    skey[j] = in ? pk : skey[j];
                    sps[j] = in ? pps : sps[j];
                    sdr[j] = in ? (depth + 1) << 16 : sdr[j];
                    sea[j] = in ? pea : sea[j];
                    slc[j] = in ? plc : slc[j];
                    scb[j] = in ? pcb : scb[j];
                }
                // the slot moves past the run
                const uint32_t kl = (uint32_t)__builtin_amdgcn_readlane((int)ki, L);
#pragma unroll
                for (int j = 0; j < FS; ++j) {
                    const bool own = lane + 64 * j == slot;
                    skey[j] = own ? kl : skey[j];
                    sdr[j] = own ? sdr[j] + L : sdr[j];
                    sea[j] = own ? sea[j] + L : sea[j];
                    slc[j] = own ? slc[j] + L : slc[j];
                }
            }
        }
        if (L == 1) {
            if (lane == 0) {
                t.n_par[n] = slot - 1;
                t.n_rank[n] = rank;
                o_tok[n] = tok;
                o_par[n] = slot - 1;
                o_dep[n] = depth;
                o_score[n] = score;
                if (o_crow != nullptr) o_crow[n] = child_row;
            }
            // the popped slot moves to its next sibling (its lane has read that entry's log-prob)
#pragma unroll
            for (int j = 0; j < FS; ++j) {
                const bool own = lane + 64 * j == slot;
                const float ns = sps[j] + nlpv[j];
                skey[j] = own ? (more ? score_key(ns) : 0u) : skey[j];
                sdr[j] = own ? sdr[j] + 1 : sdr[j];
                sea[j] = own ? sea[j] + (more ? 1 : 0) : sea[j];
                slc[j] = own ? slc[j] + (more ? 1 : 0) : slc[j];
            }
            // an expandable node opens slot n + 1 on the first entry of its row
            if (child_row >= 0) {
                const int ncb = c0 + c1 * depth + c2 * m;
#pragma unroll
                for (int j = 0; j < FS; ++j) {
                    const bool ch = lane + 64 * j == n + 1;
                    skey[j] = ch ? ck : skey[j];
                    sps[j] = ch ? score : sps[j];
                    sdr[j] = ch ? (depth + 1) << 16 : sdr[j];
                    sea[j] = ch ? child_row * a.K2 : sea[j];
                    slc[j] = ch ? child_row * a.P : slc[j];
                    scb[j] = ch ? ncb : scb[j];
                }
            }
        }
        prev = slot;
        n += L;
    }
    // slots past the last pop get the empty values
    for (int i = n + lane; i < a.B; i += 64) {
        o_tok[i] = -1;
        o_par[i] = -1;
        o_dep[i] = 0;
        o_score[i] = neg_inf();
        if (o_crow != nullptr) o_crow[i] = -1;
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
                             int gamma, int k, int topk2, int B, int mode, int32_t* node_token,
                             int32_t* node_parent, int32_t* node_depth, float* node_score, int32_t* node_child_row,
                             hipStream_t stream) {
    const int M = mode == kTreeMarginal ? 0 : k;
    const int Rs = mode == kTreeMarginal ? gamma : (int)cond_rows(gamma, k, mode == kTreeBigram ? 1 : 0);
    int P = 0;
    const size_t lds = tree_lds_bytes(B, gamma, M, Rs, topk2, &P);
    if (lds == 0) return hipErrorInvalidValue;
    TreeArgs a{cond_idx, cond_lp, topk_idx, gamma, M, topk2, B, Rs, P, mode,
               node_token, node_parent, node_depth, node_score, node_child_row};
    const void* fn;
    const bool all = P >= topk2;
    size_t lds_used = lds;
    const int tab = std::max(Rs, mode == kTreeMarginal ? 0 : gamma * M);
    const int PL = tree_lane_ranks(B, Rs, topk2);
    // B slots suffice: the slot the last pop opens is never popped
    if (PL >= 1 && B <= 64 * kLaneSlotsMax && tab <= 64 * kLaneTabMax) {
        // frontier, candidates and first log-probs in registers; sibling runs
        lds_used = tree_lane_lds_bytes(B, Rs, PL);
        a.P = PL;
        const bool lall = PL >= topk2, t2 = tab <= 128;
        const int fs = B <= 64 ? 1 : B <= 128 ? 2 : B <= 256 ? 4 : 8;
#define TF_LANE(FSV, TV, AV) reinterpret_cast<const void*>(build_tree_lane_kernel<FSV, TV, AV>)
#define TF_LANE_FS(FSV) (lall ? (t2 ? TF_LANE(FSV, 2, true) : TF_LANE(FSV, 4, true)) \
                              : (t2 ? TF_LANE(FSV, 2, false) : TF_LANE(FSV, 4, false)))
        fn = fs == 1 ? TF_LANE_FS(1) : fs == 2 ? TF_LANE_FS(2) : fs == 4 ? TF_LANE_FS(4) : TF_LANE_FS(8);
#undef TF_LANE_FS
#undef TF_LANE
    } else if (B + 1 <= 64)
        fn = all ? reinterpret_cast<const void*>(build_tree_reg_kernel<1, true>)
                 : reinterpret_cast<const void*>(build_tree_reg_kernel<1, false>);
    else if (B + 1 <= 128)
        fn = all ? reinterpret_cast<const void*>(build_tree_reg_kernel<2, true>)
                 : reinterpret_cast<const void*>(build_tree_reg_kernel<2, false>);
    else if (B + 1 <= 256)
        fn = all ? reinterpret_cast<const void*>(build_tree_reg_kernel<4, true>)
                 : reinterpret_cast<const void*>(build_tree_reg_kernel<4, false>);
    else if (B + 1 <= 512)
        fn = all ? reinterpret_cast<const void*>(build_tree_reg_kernel<8, true>)
                 : reinterpret_cast<const void*>(build_tree_reg_kernel<8, false>);
    else if (B + 1 <= 64 * kTreeRegSlots)
        fn = all ? reinterpret_cast<const void*>(build_tree_reg_kernel<kTreeRegSlots, true>)
                 : reinterpret_cast<const void*>(build_tree_reg_kernel<kTreeRegSlots, false>);
    else
        fn = reinterpret_cast<const void*>(build_tree_kernel);
    // dynamic LDS beyond the 64 KiB default
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kTreeLdsBudget) != hipSuccess)
        return hipErrorInvalidValue;
    void* args[] = {&a};
    const hipError_t e = hipLaunchKernel(fn, dim3(b), dim3(kTreeThreads), args, lds_used, stream);
    if (e != hipSuccess) return e;
    return hipGetLastError();
}

}  // namespace tf

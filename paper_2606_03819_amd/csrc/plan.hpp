// Launch plans and workspace layout shared by the C ABI and the launchers.
// Host-only; every function here is a pure function of the shapes, so the
// workspace size the caller is told and the layout the kernels use agree.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "limits.hpp"
#include "rows.hpp"
#include "work.hpp"

namespace tf {

constexpr int kMaxSplits = 2048;       // vocabulary slices (partials per row); kMaxSplits*kKeep <= merge capacity
constexpr int kMaxSplitsLong = 1024;   // slices up to which a launch may keep long lists
constexpr int kMaxTopk = 1024;         // longest top-k list the merge kernel sorts
constexpr int kMaxBudget = 4095;       // tree nodes per sequence
constexpr int kNumCUs = 256;           // compute units of an MI355X

// Waves per workgroup of the bf16 streaming products with several row
// blocks; one such workgroup fills a CU's register file at two waves per
// SIMD.  A single row block uses half the waves (two workgroups per CU): the
// k-range is cut there, and a smaller workgroup leaves the last piece's
// workgroup less partial sum to read back.
#ifndef TF_NW
#define TF_NW 8
#endif
#ifndef TF_NW_SINGLE
#define TF_NW_SINGLE 4
#endif
// Tile ranges (workgroups) of the LM head when a single row block streams
// the whole vocabulary.
#ifndef TF_LM_WORKGROUPS
#define TF_LM_WORKGROUPS 256
#endif
// Workgroups of the SwiGLU gate/up and down products when a single row
// block leaves too few weight tiles to occupy every CU (their k-range is
// then cut; every cut adds a partial-sum round trip, so the smaller down
// product uses fewer workgroups).
#ifndef TF_MLP_WORKGROUPS
#define TF_MLP_WORKGROUPS 512
#endif
#ifndef TF_DOWN_WORKGROUPS
#define TF_DOWN_WORKGROUPS 256
#endif
// Pipeline depth (k-chunks of loads in flight per wave) when a single row
// block streams the weights once at NT = 4, and otherwise; the launchers pick
// the kernel instance from NT and wnt.
#ifndef TF_PIPE_SINGLE_NT4
#define TF_PIPE_SINGLE_NT4 3
#endif
#ifndef TF_PIPE_DEFAULT
#define TF_PIPE_DEFAULT 2
#endif

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

struct GemmPlan {
    int NT;       // 32-row activation tiles per workgroup
    int WM;       // 32-row weight tiles per wave (bf16)
    int NW;       // waves per workgroup
    int chunk;    // weight tiles per chunk (NW * WM)
    int nrb;      // activation-row blocks
    int ntiles;   // 32-row weight tiles
    int nchunks;  // chunks (= vocabulary slices for the LM head)
    int nk;       // 64-wide k-chunks
    int G;        // workgroups
    bool wnt;     // non-temporal weight loads (weights read by one row block only)
    bool pieces;  // some item is cut between workgroups
    int items() const { return nchunks * nrb; }
    int blocks() const { return G; }
    GemmShape shape(int R, int K) const { return GemmShape{R, K, ntiles, nchunks, nrb, nk, G}; }
    // accumulators of one workgroup, in floats
    size_t part_floats() const { return (size_t)NW * WM * NT * 16 * 64; }
    // partial sums of cut items: two slots per workgroup
    size_t fix_floats() const { return pieces ? 2 * (size_t)G * part_floats() : 0; }
    size_t counter_ints() const { return pieces ? (size_t)items() : 0; }
};

inline int plan_nt(int rows) { return rows <= 32 ? 1 : (rows <= 64 ? 2 : 4); }
// two weight tiles per wave at NT = 1; one otherwise keeps the accumulators,
// the load pipeline and the epilogue within 256 registers
inline int plan_wm(int NT) { return NT == 1 ? 2 : 1; }

// bf16 product of `rows` activation rows with `ntiles` weight tiles over K.
// Enough (chunk, row block) items of eight-wave workgroups to give every CU
// one: one item per workgroup, the row blocks of a chunk on consecutive
// workgroups so that they share the chunk through L2.  Fewer (one row block,
// or a few): four-wave workgroups, the units cut evenly over `wg_single`
// workgroups.
inline GemmPlan gemm_plan(int rows, int ntiles, int K, int wg_single) {
    GemmPlan p;
    p.NT = plan_nt(rows);
    p.WM = plan_wm(p.NT);
    p.nrb = cdiv(rows, 32 * p.NT);
    const bool whole = p.nrb > 1 && (long long)cdiv(ntiles, TF_NW * p.WM) * p.nrb >= kNumCUs;
    p.NW = whole ? TF_NW : TF_NW_SINGLE;
    p.chunk = p.NW * p.WM;
    p.ntiles = ntiles;
    p.nchunks = cdiv(ntiles, p.chunk);
    p.nk = cdiv(K, 64);
    if (!whole) {
        const long long units = (long long)p.items() * p.nk;
        p.G = (int)(units < wg_single ? units : wg_single);
        if (p.G < p.items()) p.G = p.items();
    } else {
        p.G = p.items();
    }
    p.wnt = p.nrb == 1;
    p.pieces = gemm_has_pieces(p.shape(rows, K));
    return p;
}

// LM head over [rows, d] x [V, d]: vocabulary slices (see SliceMap), one
// workgroup per (tile range, row block), the row blocks of a range on
// consecutive workgroups so that they share its tiles through L2.  One row
// block, or up to TF_LM_GRID_NRB on the DMA kernel's wave grid: the tiles
// spread over TF_LM_WORKGROUPS workgroups in all; more row blocks: one
// chunk per range.  fp32 (small workloads, SIMT kernel): 32 rows and at most
// 8 tiles (256 tokens) per workgroup.
struct LmPlan {
    int NT, WM, NW, chunk, nrb, ntiles, nk;
    int WB = 1;   // waves along the activation tiles (a grid of NW / WB x WB waves)
    bool grid = false;   // the DMA kernel's 2 x 2 wave grid (up to TF_LM_GRID_NRB row blocks)
    SliceMap map;
    bool wnt;
    bool dma;   // the LDS-DMA kernel (32-row tiles, the grid, or 256-row blocks)
    int nsplit() const { return map.G * map.rmax; }
    int blocks() const { return map.G * nrb; }
};

// LM-head tile shape per activation-tile count: waves per workgroup and
// weight tiles per wave (one wave per SIMD when NW = 4, so that a wave may
// hold 128 accumulator registers).
#ifndef TF_LM_NW_NT1
#define TF_LM_NW_NT1 4
#endif
#ifndef TF_LM_WM_NT1
#define TF_LM_WM_NT1 4
#endif
#ifndef TF_LM_NW_NT2
#define TF_LM_NW_NT2 8
#endif
#ifndef TF_LM_WM_NT2
#define TF_LM_WM_NT2 1
#endif
#ifndef TF_LM_NW_NT4
#define TF_LM_NW_NT4 8
#endif
#ifndef TF_LM_WM_NT4
#define TF_LM_WM_NT4 1
#endif
// A single row block: four waves, one per SIMD, in a 2 x 2 grid (two along
// the weight tiles, two along the activation tiles), each with 5 weight
// tiles x 2 activation tiles: ten tiles per round, so the 256 ranges of the
// Qwen vocabularies take two rounds, and every SIMD issues the same MFMAs
// and fragment reads (five waves of 2 x 4 tiles left one SIMD with two
// waves' work, which set the pace of every k step).
#ifndef TF_LM_DMA_WM
#define TF_LM_DMA_WM 5
#endif
#ifndef TF_LM_DMA_NW_SINGLE
#define TF_LM_DMA_NW_SINGLE 4
#endif
#ifndef TF_LM_DMA_SINGLE_WB
#define TF_LM_DMA_SINGLE_WB 2
#endif
// Row blocks up to which the grid shape serves the LM head: the row blocks
// of a tile range run on consecutive workgroups (one XCD), so the second
// reads the weights the first brought into L2 (plain loads, not
// non-temporal).
#ifndef TF_LM_GRID_NRB
#define TF_LM_GRID_NRB 2
#endif
// Several row blocks (MFMA-bound): 256-row blocks of eight waves in a 4 x 2
// grid (2 weight x 4 activation tiles each), one workgroup per CU.  Each
// copied weight tile then meets 256 activation rows and each copied
// activation tile 8 weight tiles: 0.5 KiB of copies per 32 x 32 tile pair of
// MFMA work against 0.75 KiB with 128-row blocks of four waves (+6% on the
// 1936-row batched step); 64-wide k steps fill the 160 KiB of LDS (+1.5%
// against 32-wide).
#ifndef TF_LM_DMA_MULTI_WM
#define TF_LM_DMA_MULTI_WM 2
#endif
#ifndef TF_LM_DMA_KC
#define TF_LM_DMA_KC 64
#endif
#ifndef TF_LM_DMA_STAGES
#define TF_LM_DMA_STAGES 3
#endif
// 32-row tiles (stage 1): four waves of three tiles (twelve per round, two
// rounds per range, 152 KiB of rings), about 1% faster per step than the
// register-staged kernel at the 8B shape
#ifndef TF_LM_DMA_NT1_WM
#define TF_LM_DMA_NT1_WM 3
#endif
#ifndef TF_LM_DMA_NT1_NW
#define TF_LM_DMA_NT1_NW 4
#endif
inline int lm_nw(int NT) { return NT == 1 ? TF_LM_NW_NT1 : (NT == 2 ? TF_LM_NW_NT2 : TF_LM_NW_NT4); }
inline int lm_wm(int NT) { return NT == 1 ? TF_LM_WM_NT1 : (NT == 2 ? TF_LM_WM_NT2 : TF_LM_WM_NT4); }

inline LmPlan lm_plan(int rows, int V, int d, bool bf16) {
    LmPlan p;
    p.ntiles = cdiv(V, 32);
    p.nk = cdiv(d, 64);
    p.dma = false;
    if (bf16) {
        p.NT = plan_nt(rows);
        // k in whole 64-wide steps: the DMA kernel -- 32-row tiles, the 2 x 2
        // wave grid up to TF_LM_GRID_NRB row blocks, else 256-row blocks
        p.nrb = cdiv(rows, 32 * p.NT);
        p.grid = p.NT >= 2 && p.nrb <= TF_LM_GRID_NRB && d % TF_LM_DMA_KC == 0;
        const bool multi = p.NT == 4 && p.nrb > 1 && !p.grid && d % TF_LM_DMA_KC == 0;
        p.dma = p.grid || multi || (p.NT == 1 && d % TF_LM_DMA_KC == 0);
        if (p.dma && p.NT == 1) {
            p.WM = TF_LM_DMA_NT1_WM;
            p.NW = TF_LM_DMA_NT1_NW;
        } else if (p.grid) {
            p.WM = TF_LM_DMA_WM;
            p.NW = TF_LM_DMA_NW_SINGLE;
            p.WB = TF_LM_DMA_SINGLE_WB;
        } else if (p.dma) {
            // 256-row blocks: eight waves in a 4 x 2 grid of 2 weight x 4
            // activation tiles, one workgroup per CU
            p.NT = 8;
            p.nrb = cdiv(rows, 256);
            p.WM = TF_LM_DMA_MULTI_WM;
            p.NW = 8;
            p.WB = 2;
        } else {
            p.WM = lm_wm(p.NT);
            p.NW = lm_nw(p.NT);
        }
        p.chunk = p.NW / p.WB * p.WM;
        // one row block, or the grid kernel: TF_LM_WORKGROUPS workgroups in
        // all, the row blocks of a tile range on consecutive ones
        const int gw = TF_LM_WORKGROUPS / p.nrb;
        const int G = p.nrb == 1 || p.grid ? (p.ntiles < gw ? p.ntiles : gw) : cdiv(p.ntiles, p.chunk);
        p.map = make_slice_map(p.ntiles, G, p.chunk);
        p.wnt = p.nrb == 1;
    } else {
        p.NT = 1;
        p.WM = 2;
        p.NW = 4;
        p.chunk = 8;
        p.nrb = cdiv(rows, 32);
        p.map = make_slice_map(p.ntiles, cdiv(p.ntiles, p.chunk), p.chunk);
        p.wnt = false;
    }
    return p;
}

// SwiGLU products (bf16).
inline GemmPlan mlp_plan(int rows, int ntiles, int K, int wg_single) {
    GemmPlan p = gemm_plan(rows, ntiles, K, wg_single);
    p.wnt = false;   // every workgroup of a row block re-reads its weights from L2
    return p;
}
// gate/up over x = [h~ ; e~], K = 2d (3d for the bigram rows)
inline GemmPlan gateup_plan(int rows, int K, int I) { return mlp_plan(rows, cdiv(I, 16), K, TF_MLP_WORKGROUPS); }
// the gate alone (plain SiLU MLP): tiles of 32 gate rows
inline GemmPlan silu_gate_plan(int rows, int K, int I) { return mlp_plan(rows, cdiv(I, 32), K, TF_MLP_WORKGROUPS); }
// down projection over the activation's bf16 hi/lo pairs: K = 2I
inline GemmPlan down_plan(int rows, int d, int I) { return mlp_plan(rows, cdiv(d, 32), 2 * I, TF_DOWN_WORKGROUPS); }
// the linear approximator: [rows, 2d] x [d, 2d]^T
inline GemmPlan linear_plan(int rows, int d) { return mlp_plan(rows, cdiv(d, 32), 2 * d, TF_DOWN_WORKGROUPS); }
// one half (h~ or e~) of the linear layer's input: [rows, d] x [d, d]^T
inline GemmPlan linear_half_plan(int rows, int d) { return mlp_plan(rows, cdiv(d, 32), d, TF_DOWN_WORKGROUPS); }

// The input projections over several activation row blocks, split at the
// h~ / e~ boundary of x (Eq. 1): the h~ half once per drafter state
// ([b*gamma, d] into an fp32 table of ldh() columns), the e~ half for every
// row (K = ew), whose epilogue adds its state's entry of the table.
struct SplitPlans {
    GemmPlan ph, pe;
    int ldh() const { return ph.ntiles * 32; }
    size_t fix_floats() const { return ph.fix_floats() > pe.fix_floats() ? ph.fix_floats() : pe.fix_floats(); }
    size_t counter_ints() const { return ph.counter_ints() + pe.counter_ints(); }
};
// kind 0: SwiGLU gate/up, 1: the plain SiLU gate, 2: the linear layer
inline SplitPlans split_plans(int kind, int states, int rows, int d, int ew, int I) {
    if (kind == 0) return SplitPlans{gateup_plan(states, d, I), gateup_plan(rows, ew, I)};
    if (kind == 1) return SplitPlans{silu_gate_plan(states, d, I), silu_gate_plan(rows, ew, I)};
    return SplitPlans{linear_half_plan(states, d), linear_half_plan(rows, d)};
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The products of the AR approximator when one row block holds every
// conditional row (mlp_dma.hpp): items of TG weight tiles over their whole
// reduction range (an h phase of nkh and an e phase of nke 64-column
// chunks), dealt out to G workgroups of at least kMlpDmaMinUnits chunks.
// The input projections take four tiles per item, the down projection (its
// activation rows twice as long: bf16 hi/lo pairs) two, so that one chunk
// carries 16 MFMAs per wave and 8-16 KiB of weights: fewer, fatter chunks
// than with one tile, whose per-chunk barrier and latencies otherwise set
// the pace.
#ifndef TF_MLP_DMA_TG_IN
#define TF_MLP_DMA_TG_IN 4
#endif
#ifndef TF_MLP_DMA_TG_DOWN
#define TF_MLP_DMA_TG_DOWN 2
#endif
constexpr int kMlpDmaMinUnits = 12;
constexpr int kMlpDmaMaxRows = 128;    // conditional rows (four activation tiles)
constexpr int kMlpDmaMaxGateRows = 256; // the input projections alone (eight activation tiles)
constexpr int kMlpDmaMaxStates = 32;   // drafter states (one activation tile)
struct MlpDmaPlan {
    int TG;       // weight tiles per item
    int NTE;      // 32-row activation tiles of the e phase (1, 2 or 4)
    int ntiles;   // 32-row weight tiles
    int items, nkh, nke, G;
    int wh, we;   // cost of an h chunk and of an e chunk in the split (work.hpp)
    size_t part_floats() const { return (size_t)2 * G * TG * 1024 * (1 + NTE); }
};
inline MlpDmaPlan mlp_dma_plan(int rows, int ntiles, int nkh, int nke, int TG) {
    MlpDmaPlan p;
    p.TG = TG;
    p.NTE = rows <= 32 ? 1 : (rows <= 64 ? 2 : (rows <= 128 ? 4 : 8));
    p.ntiles = ntiles;
    p.items = cdiv(ntiles, TG);
    p.nkh = nkh;
    p.nke = nke;
    const long long U = (long long)p.items * (nkh + nke);
    long long G = U / kMlpDmaMinUnits;
    G = G < kNumCUs ? G : kNumCUs;
    p.G = (int)(G < 1 ? 1 : G);
    // An e chunk against four activation tiles streams its weights at about
    // three fifths of an h chunk's rate (the activation copies from L2 share
    // the CU's load path with the weight stream; 5:3 measured best against
    // 3:2 and 9:5); two tiles take a ratio between that and 1, and one tile,
    // like the h phase, costs the same; eight tiles (the input
    // projections of 129-256 rows) 5:2.
    p.wh = nkh == 0 ? 1 : (p.NTE == 8 ? 2 : (p.NTE == 4 ? 3 : (p.NTE == 2 ? 4 : 1)));
    p.we = nkh == 0 ? 1 : (p.NTE == 8 ? 5 : (p.NTE == 4 ? 5 : (p.NTE == 2 ? 5 : 1)));
    if (!cost_split_valid(p.items, nkh, nke, p.wh, p.we, p.G)) p.wh = p.we = 1;
    return p;
}
inline bool mlp_dma_plan_ok(const MlpDmaPlan& p) {
    return cost_split_valid(p.items, p.nkh, p.nke, p.wh, p.we, p.G);
}
// gate/up (SwiGLU: tiles of 16 gate + 16 up rows) or the gate alone (the
// plain SiLU MLP: tiles of 32 gate rows) over [h~ ; e~], e~ ew wide
inline MlpDmaPlan mlp_dma_gate_plan(int rows, int d, int ew, int I, bool swiglu) {
    return mlp_dma_plan(rows, swiglu ? cdiv(I, 16) : cdiv(I, 32), d / 64, ew / 64, TF_MLP_DMA_TG_IN);
}
// down projection over the activation's hi/lo pairs (no h phase)
inline MlpDmaPlan mlp_dma_down_plan(int rows, int d, int I) {
    return mlp_dma_plan(rows, cdiv(d, 32), 0, I / 64, TF_MLP_DMA_TG_DOWN);
}
// the linear approximator W_lin [d, 2d] over [h~ ; e~]
inline MlpDmaPlan mlp_dma_linear_plan(int rows, int d) {
    return mlp_dma_plan(rows, cdiv(d, 32), d / 64, d / 64, TF_MLP_DMA_TG_IN);
}
// One row block holds every conditional row and each plan the path may
// launch (either gate plan, the down projection, the linear layer) keeps its
// split in 32-bit arithmetic.
// 129-256 conditional rows: the input projections on the one-row-block kernel
// (eight activation tiles), the down projection on the kernel for several
// row blocks (its activation pairs for eight tiles do not fit the LDS).
inline bool mlp_dma_gate_applies(bool bf16, int b, int gamma, int R, int d, int I, int ew) {
    if (!(bf16 && (long long)b * gamma <= kMlpDmaMaxStates && (long long)b * R > kMlpDmaMaxRows &&
          (long long)b * R <= kMlpDmaMaxGateRows && d % 64 == 0 && I % 64 == 0 && ew % 64 == 0))
        return false;
    const int rows = b * R;
    return mlp_dma_plan_ok(mlp_dma_gate_plan(rows, d, ew, I, true)) &&
           mlp_dma_plan_ok(mlp_dma_gate_plan(rows, d, ew, I, false));
}
inline bool mlp_dma_applies(bool bf16, int b, int gamma, int R, int d, int I, int ew) {
    if (!(bf16 && (long long)b * gamma <= kMlpDmaMaxStates && (long long)b * R <= kMlpDmaMaxRows && d % 64 == 0 &&
          I % 64 == 0 && ew % 64 == 0))
        return false;
    const int rows = b * R;
    return mlp_dma_plan_ok(mlp_dma_gate_plan(rows, d, ew, I, true)) &&
           mlp_dma_plan_ok(mlp_dma_gate_plan(rows, d, ew, I, false)) && mlp_dma_plan_ok(mlp_dma_down_plan(rows, d, I)) &&
           mlp_dma_plan_ok(mlp_dma_linear_plan(rows, d));
}

// Long (row, slice) lists for top-k lists of at least kLongListK entries
// (bf16 kernels, while the merge's candidate buffer holds every entry).
inline bool lm_long_lists(const LmPlan& p, bool bf16, int K) {
    return bf16 && K >= kLongListK && p.nsplit() <= kMaxSplitsLong;
}

// LM-head scratch: the (row, slice) partials, sized for the long lists
// whenever a launch could keep them.
inline size_t lm_scratch_bytes(int rows, int V, int d, bool bf16) {
    const LmPlan p = lm_plan(rows, V, d, bf16);
    const int stride = bf16 && p.nsplit() <= kMaxSplitsLong ? kPartStrideLong : kPartStride;
    return align256((size_t)rows * p.nsplit() * stride * 4);
}

struct Workspace {
    size_t diag, lm, ht, et, act, hp, mlp_part, counters, hh, total;
    int ncounters;
};

// Layout: [diag counters | LM-head scratch (stage 1 or stage 2) | normalised
// h | normalised embeddings | SwiGLU activation | h' | SwiGLU partial sums |
// SwiGLU arrival counters | h~-half table of the split input projections].
// Stage 1 uses the first two only.  `bigram` sizes the w/ 2-prev rows (two
// embeddings per row, a 3d-wide input).
inline Workspace workspace_layout(int b, int gamma, int d, int I, int V, int k, bool bf16, bool bigram = false) {
    const int R = (int)cond_rows(gamma, k, bigram ? 1 : 0);
    const int npre = bigram ? 2 : 1;
    const size_t es = bf16 ? 2 : 4;
    const int rows1 = b * gamma, rows2 = b * R;
    const size_t lm1 = lm_scratch_bytes(rows1, V, d, bf16), lm2 = lm_scratch_bytes(rows2, V, d, bf16);
    Workspace w;
    size_t off = 0;
    w.diag = off;
    off += 256;
    w.lm = off;
    off += lm1 > lm2 ? lm1 : lm2;
    w.ht = off;
    off += align256((size_t)rows1 * d * es);
    w.et = off;
    off += align256((size_t)rows2 * npre * d * es);
    w.act = off;
    off += align256((size_t)rows2 * I * es * (bf16 ? 2 : 1));   // bf16: hi/lo pairs
    w.hp = off;
    off += align256((size_t)rows2 * d * es);
    size_t mp = 0;
    w.ncounters = 0;
    size_t hhf = 0;
    if (bf16) {
        const SplitPlans sg = split_plans(0, rows1, rows2, d, npre * d, I), ss = split_plans(1, rows1, rows2, d, npre * d, I),
                         sl = split_plans(2, rows1, rows2, d, d, I);
        const GemmPlan pd = down_plan(rows2, d, I);
        const size_t fx[] = {sg.fix_floats(), ss.fix_floats(), sl.fix_floats(), pd.fix_floats()};
        for (size_t x : fx) mp = mp > x ? mp : x;
        size_t nc = sg.counter_ints() + pd.counter_ints();
        nc = nc > ss.counter_ints() + pd.counter_ints() ? nc : ss.counter_ints() + pd.counter_ints();
        nc = nc > sl.counter_ints() ? nc : sl.counter_ints();
        const int ldh[] = {sg.ldh(), ss.ldh(), sl.ldh()};
        for (int x : ldh) hhf = hhf > (size_t)rows1 * x ? hhf : (size_t)rows1 * x;
        if (mlp_dma_applies(bf16, b, gamma, R, d, I, npre * d)) {
            // either the SwiGLU or the SiLU gate plan (the SwiGLU one has more
            // items), the down projection, the linear approximator
            const MlpDmaPlan qg = mlp_dma_gate_plan(rows2, d, npre * d, I, true),
                             qs = mlp_dma_gate_plan(rows2, d, npre * d, I, false), qd = mlp_dma_down_plan(rows2, d, I),
                             ql = mlp_dma_linear_plan(rows2, d);
            const size_t pf[] = {qg.part_floats(), qs.part_floats(), qd.part_floats(), ql.part_floats()};
            for (size_t x : pf) mp = mp > x ? mp : x;
            const size_t qc = (size_t)qg.items + qd.items;
            nc = nc > qc ? nc : qc;
            nc = nc > (size_t)ql.items ? nc : (size_t)ql.items;
        }
        if (mlp_dma_gate_applies(bf16, b, gamma, R, d, I, npre * d)) {
            // either gate plan on the one-row-block kernel, then the down
            // projection of several row blocks
            const MlpDmaPlan qg = mlp_dma_gate_plan(rows2, d, npre * d, I, true),
                             qs = mlp_dma_gate_plan(rows2, d, npre * d, I, false);
            mp = mp > qg.part_floats() ? mp : qg.part_floats();
            mp = mp > qs.part_floats() ? mp : qs.part_floats();
            const size_t qc = (size_t)qg.items + pd.counter_ints();
            nc = nc > qc ? nc : qc;
        }
        w.ncounters = (int)nc;
    }
    w.mlp_part = off;
    off += align256(mp * 4);
    w.counters = off;
    off += align256((size_t)w.ncounters * 4);
    w.hh = off;
    off += align256(hhf * 4);
    w.total = off;
    return w;
}

}  // namespace tf

// Work split of a weight-streaming product, shared by the host plans and the
// kernels so both derive the same pieces from the same shape.
//
// SwiGLU products (few weight tiles): the k-range is cut.  The weight tiles
// (32 rows each) are grouped into chunks, the activation rows
// into row blocks.  An item is one (chunk, row block) pair; a unit is one
// 64-wide k-chunk of an item.  The U = items * nk units are ordered item-major
// (row block fastest within a chunk, then k) and workgroup g owns the
// contiguous range [g*U/G, (g+1)*U/G), so every workgroup streams the same
// number of weight bytes, up to one k-chunk.  An item cut by a range boundary
// is computed in pieces by consecutive workgroups; the last of them to finish
// sums the pieces in workgroup order and runs the epilogue.
#pragma once

#include <hip/hip_runtime.h>

namespace tf {

struct GemmShape {
    int R;        // activation rows
    int K;        // reduction length (multiple of 16)
    int ntiles;   // 32-row weight tiles
    int nchunks;  // chunks of weight tiles
    int nrb;      // activation-row blocks
    int nk;       // 64-wide k-chunks, ceil(K / 64)
    int G;        // workgroups
};

__host__ __device__ inline long long gemm_units(const GemmShape& s) {
    return (long long)s.nchunks * s.nrb * s.nk;
}

// first unit of workgroup g (g = G gives the end of the last range)
__host__ __device__ inline long long unit_start(const GemmShape& s, int g) {
    return (long long)g * gemm_units(s) / s.G;
}

// workgroup whose range holds unit u: the largest g with unit_start(g) <= u
__host__ __device__ inline int unit_owner(const GemmShape& s, long long u) {
    return (int)(((u + 1) * s.G - 1) / gemm_units(s));
}

// Partial-sum slot of workgroup g's piece of `item`: a workgroup holds at most
// two cut items, the one its range starts in (slot 2g) and the one it ends in
// (slot 2g + 1).
__host__ __device__ inline int piece_slot(const GemmShape& s, int g, int item) {
    return 2 * g + (item != (int)(unit_start(s, g) / s.nk) ? 1 : 0);
}

// Does any range boundary fall inside an item?
inline bool gemm_has_pieces(const GemmShape& s) {
    for (int g = 1; g < s.G; ++g)
        if (unit_start(s, g) % s.nk != 0) return true;
    return false;
}

// One-row-block products (every activation row in one block): an item's k-
// chunks come in two phases, first nkh chunks of the h~ half of x against the
// drafter states' one row tile, then nke chunks against every row (the e~
// half, or the whole input of a product without the split).  An e chunk costs
// more than an h chunk (more activation tiles per weight byte), so the units
// (item-major, as above) are dealt out by cost: an h chunk costs wh, an e
// chunk we, and workgroup g owns the units whose cost offset falls in
// [ceil(g*C/G), ceil((g+1)*C/G)), C the total.  Every workgroup then carries
// the same work up to one chunk; the pieces of a cut item are consecutive
// workgroups as before, and a workgroup holds at most two cut items.  Ranges
// are never empty while C/G >= max(wh, we), and the arithmetic stays in 32
// bits while C*G < 2^31 (cost_split_valid).
struct CostSplit {
    int nk, nkh, wh, we, G;
    int citem, ctot;   // cost of one item, of all items
};

__host__ __device__ inline CostSplit cost_split(int items, int nkh, int nke, int wh, int we, int G) {
    const int citem = nkh * wh + nke * we;
    return CostSplit{nkh + nke, nkh, wh, we, G, citem, citem * items};
}

// cost offset of chunk c of `item` (the cost of every unit before it)
__host__ __device__ inline int split_cost(const CostSplit& s, int item, int c) {
    const int ch = c < s.nkh ? c : s.nkh;
    return item * s.citem + ch * s.wh + (c - ch) * s.we;
}

// first unit of workgroup g (g = G gives the end of the last range): the
// first unit whose cost offset reaches ceil(g*C/G)
__host__ __device__ inline int unit_start(const CostSplit& s, int g) {
    const int x = (g * s.ctot + s.G - 1) / s.G;
    const int it = x / s.citem;
    const int o = x - it * s.citem, oh = s.nkh * s.wh;
    const int c = o <= oh ? (o + s.wh - 1) / s.wh : s.nkh + (o - oh + s.we - 1) / s.we;
    return it * s.nk + c;
}

// workgroup whose range holds chunk c of `item`
__host__ __device__ inline int unit_owner(const CostSplit& s, int item, int c) {
    return split_cost(s, item, c) * s.G / s.ctot;
}

// partial-sum slot of workgroup g's piece of `item`: slot 2g for the item its
// range starts in, 2g + 1 for the one it ends in (as piece_slot above)
__host__ __device__ inline int piece_slot(const CostSplit& s, int g, int item) {
    return 2 * g + (item != unit_start(s, g) / s.nk ? 1 : 0);
}

// The pieces of a cut item: workgroups gfirst .. gfirst + npieces - 1.  Piece
// i > 0 starts its range inside the item (slot 2(gfirst + i)); the first may
// have started in an earlier item (then slot 2 gfirst + 1).  Pieces [0, ph1)
// cover h chunks, pieces [pe0, npieces) e chunks (one piece may do both).
struct CutPieces {
    int gfirst, npieces, slot0, ph1, pe0;
    __host__ __device__ int slot(int i) const { return i == 0 ? slot0 : 2 * (gfirst + i); }
};

__host__ __device__ inline CutPieces cut_pieces(const CostSplit& s, int item) {
    CutPieces p;
    p.gfirst = unit_owner(s, item, 0);
    p.npieces = unit_owner(s, item, s.nk - 1) - p.gfirst + 1;
    p.slot0 = 2 * p.gfirst + (unit_start(s, p.gfirst) < item * s.nk ? 1 : 0);
    p.ph1 = s.nkh > 0 ? unit_owner(s, item, (s.nkh < s.nk ? s.nkh : s.nk) - 1) - p.gfirst + 1 : 0;
    p.pe0 = s.nkh < s.nk ? unit_owner(s, item, s.nkh) - p.gfirst : p.npieces;
    return p;
}

inline bool cost_split_valid(int items, int nkh, int nke, int wh, int we, int G) {
    const long long c = ((long long)nkh * wh + (long long)nke * we) * items;
    return c > 0 && c * G < (1LL << 31) && c >= (long long)G * (wh > we ? wh : we);
}

// LM head (many weight tiles): the vocabulary is cut instead.
//
// Vocabulary slices of the LM head.  The T weight tiles are cut into G
// contiguous ranges of floor(T/G) or ceil(T/G) tiles (one per workgroup
// column); range g is streamed in rounds(g) = ceil(n_g / chunk) near-equal
// rounds of at most `chunk` tiles, each a full pass over K.  Slice g*rmax + r
// is round r of range g and is empty when r >= rounds(g).  Every workgroup
// thus streams the same number of weight tiles (up to one), and no slice
// needs partial sums from another workgroup.
struct SliceMap {
    int T;       // weight tiles
    int G;       // tile ranges
    int chunk;   // most tiles per round
    int rmax;    // slices per range
};

__host__ __device__ inline int slice_range_begin(const SliceMap& m, int g) {
    return (int)((long long)g * m.T / m.G);
}

// tiles [t0, t1) of slice s (t0 == t1 for an empty slice)
__host__ __device__ inline void slice_tiles(const SliceMap& m, int s, int& t0, int& t1) {
    const int g = s / m.rmax, r = s - g * m.rmax;
    const int a = slice_range_begin(m, g);
    const int n = slice_range_begin(m, g + 1) - a;
    const int rounds = (n + m.chunk - 1) / m.chunk;
    if (r >= rounds) {
        t0 = t1 = a;
        return;
    }
    t0 = a + (int)((long long)r * n / rounds);
    t1 = a + (int)((long long)(r + 1) * n / rounds);
}

inline SliceMap make_slice_map(int T, int G, int chunk) {
    const int per = (T + G - 1) / G;
    return SliceMap{T, G, chunk, (per + chunk - 1) / chunk};
}

}  // namespace tf

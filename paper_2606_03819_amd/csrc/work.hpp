// Work split of a weight-streaming product, shared by the host plans and the
// kernels so both derive the same pieces from the same shape.
//
// The weight tiles (32 rows each) are grouped into chunks, the activation rows
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

}  // namespace tf

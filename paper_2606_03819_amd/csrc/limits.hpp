// Compile-time constants shared by host planning code and device kernels.
#pragma once

namespace tf {

// Entries each (row, vocabulary slice) partial keeps, and the partial layout:
// [max, sum, bound, count, val[keep], idx[keep]] (raw, unscaled logits).
// Long lists (kKeepLong per slice, kLaneMfmaLong per lane and row in the
// MFMA epilogue) serve top-k lists of at least kLongListK entries: with
// short ones a row's best logits overflow a slice's or a lane's list often
// enough there that the exact re-evaluation dominates.
constexpr int kKeep = 4;
constexpr int kKeepLong = 8;
constexpr int kPartStride = 4 + 2 * kKeep;
constexpr int kPartStrideLong = 4 + 2 * kKeepLong;
constexpr int kLongListK = 64;
constexpr int part_stride(int keep) { return 4 + 2 * keep; }
// Per-thread running list lengths inside the LM-head epilogues (SIMT fp32
// kernel, MFMA bf16 kernel; "wide": a lane holds more than 64 logits of a
// row, so it more often holds several of the row's best and needs a longer
// list for the same rate of overflowing lanes).
constexpr int kLane = 4;
constexpr int kLaneMfma = 2;
// 256-row blocks (the batched steps: thousands of rows, so a lane holding
// three of a row's best 32 logits, which a two-entry list flags for the
// exact slow path, turns up in a sizeable share of launches)
constexpr int kLaneMfmaMulti = 3;
constexpr int kLaneMfmaLong = 3;
constexpr int kLaneMfmaWide = 3;
constexpr int kLaneMfmaWideLong = 5;

}  // namespace tf

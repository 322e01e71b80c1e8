// Compile-time constants shared by host planning code and device kernels.
#pragma once

namespace tf {

// Entries each (row, vocabulary slice) partial keeps, and the partial layout:
// [max, sum, bound, count, val[kKeep], idx[kKeep]] (raw, unscaled logits).
constexpr int kKeep = 4;
constexpr int kPartStride = 4 + 2 * kKeep;
// Per-thread running list lengths inside the LM-head epilogues (SIMT fp32
// kernel, MFMA bf16 kernel).
constexpr int kLane = 4;
constexpr int kLaneMfma = 2;

}  // namespace tf

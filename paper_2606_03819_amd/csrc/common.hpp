// Shared device helpers of the TreeFlash HIP library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "limits.hpp"

namespace tf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Vocabulary rows per MFMA tile.
constexpr int kTile = 32;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t u16) { return __uint_as_float(u16 << 16); }

// float -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Two floats to bf16 with round-to-nearest-even in one instruction
// (v_cvt_pk_bf16_f32): a in the low half, b in the high half.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2_bits(float a, float b) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){a, b}, b2));
}

// Monotone map float -> uint32 (larger float <=> larger key).
__device__ __forceinline__ uint32_t f32_key(float f) {
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_f32(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

// (value desc, id asc) order: is (va, ia) strictly before (vb, ib)?
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
    return va > vb || (va == vb && ia < ib);
}
// The same order with the three comparisons combined as lane masks, so that
// a wave evaluates it without branches.
__device__ __forceinline__ bool better_masks(float va, int ia, float vb, int ib) {
    return (va > vb) | ((va == vb) & (ia < ib));
}

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// A bf16 LM-head logit as the lists carry and compare it: the fp32 value
// with its low kLogitTagBits mantissa bits cleared (monotone, relative change
// below 2^-16).  The MFMA epilogue stores a token's lane-local position in
// those bits, so that one float max or median ranks (value, position) pairs;
// every comparison of bf16 logits (epilogue, merge, exact re-evaluation) is
// made on this value, so that the lists' bounds stay exact.
constexpr int kLogitTagBits = 7;
__device__ __forceinline__ float logit_trunc(float x) {
    return __int_as_float(__float_as_int(x) & ~((1 << kLogitTagBits) - 1));
}

__device__ __forceinline__ f32x16 mfma_32x32x16_bf16(const u32x4& a, const u32x4& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Row of a 32x32 MFMA accumulator held in register j of lane `lane`
// (the column is lane % 32).
__device__ __forceinline__ int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

// The value that lane (lane ^ J) of this wave holds, J a power of two below
// 64, without a trip through the LDS crossbar: DPP quad permutes (J = 1, 2),
// rotations within a 16-lane row (J = 4, 8), and the row and half-wave swaps
// of gfx950 (J = 16, 32).  Every lane must be active.
template <int J>
__device__ __forceinline__ int lane_xor(int v) {
    static_assert(J == 1 || J == 2 || J == 4 || J == 8 || J == 16 || J == 32, "xor distance");
    if constexpr (J == 1) {
        return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
    } else if constexpr (J == 2) {
        return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
    } else if constexpr (J == 4) {
        const int up = __builtin_amdgcn_mov_dpp(v, 0x12C, 0xF, 0xF, false);   // row_ror:12, lane + 4
        const int dn = __builtin_amdgcn_mov_dpp(v, 0x124, 0xF, 0xF, false);   // row_ror:4, lane - 4
        return (threadIdx.x & 4) ? dn : up;
    } else if constexpr (J == 8) {
        return __builtin_amdgcn_mov_dpp(v, 0x128, 0xF, 0xF, false);   // row_ror:8
    } else if constexpr (J == 16) {
        // odd rows of the first copy trade places with even rows of the second
        const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (threadIdx.x & 16) ? (int)p[0] : (int)p[1];
    } else {
        // the upper half of the first copy trades places with the lower half of the second
        const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (threadIdx.x & 32) ? (int)p[0] : (int)p[1];
    }
}
template <int J>
__device__ __forceinline__ float lane_xor(float v) {
    return __int_as_float(lane_xor<J>(__float_as_int(v)));
}
// lane_xor with a distance known once the caller's loops are unrolled
template <class T>
__device__ __forceinline__ T lane_xor_n(T v, int j) {
    switch (j) {
        case 1: return lane_xor<1>(v);
        case 2: return lane_xor<2>(v);
        case 4: return lane_xor<4>(v);
        case 8: return lane_xor<8>(v);
        case 16: return lane_xor<16>(v);
        default: return lane_xor<32>(v);
    }
}

__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, lane_xor<32>(v));
    v = fmaxf(v, lane_xor<16>(v));
    v = fmaxf(v, lane_xor<8>(v));
    v = fmaxf(v, lane_xor<4>(v));
    v = fmaxf(v, lane_xor<2>(v));
    return fmaxf(v, lane_xor<1>(v));
}
__device__ __forceinline__ float wave_sum(float v) {
    v += lane_xor<32>(v);
    v += lane_xor<16>(v);
    v += lane_xor<8>(v);
    v += lane_xor<4>(v);
    v += lane_xor<2>(v);
    return v + lane_xor<1>(v);
}

}  // namespace tf

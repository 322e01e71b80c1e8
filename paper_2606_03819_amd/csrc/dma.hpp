// Copies from global memory straight into LDS (gfx950 global_load_lds), and
// the waits and barriers the kernels built on them use.
#pragma once

#include <hip/hip_runtime.h>

namespace tf {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void global_void_t;

// cache-policy bit of a non-temporal load (weights that one workgroup alone
// streams); weights shared through L2 by several workgroups load normally
constexpr int kCpolNt = 2;

// One DMA instruction: every lane copies 16 bytes from `src` to LDS; the 64
// lanes fill 1 KiB at `dst` in lane order (lane l at dst + 16 l).
__device__ __forceinline__ void dma16(const void* src, void* dst, int cpol) {
    if (cpol == kCpolNt)
        __builtin_amdgcn_global_load_lds((global_void_t*)src, (lds_void_t*)dst, 16, 0, kCpolNt);
    else
        __builtin_amdgcn_global_load_lds((global_void_t*)src, (lds_void_t*)dst, 16, 0, 0);
}

// wait until at most N of this wave's memory loads are outstanding (also a
// compiler barrier for memory operations)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
    asm volatile("" ::: "memory");
}

// The same with a count known only at run time (uniform across the wave);
// counts past 62 wait for 62.
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
    switch (n) {
#define TF_WAIT_CASE(N) \
    case N: wait_vmcnt<N>(); break;
        TF_WAIT_CASE(0) TF_WAIT_CASE(1) TF_WAIT_CASE(2) TF_WAIT_CASE(3) TF_WAIT_CASE(4) TF_WAIT_CASE(5)
        TF_WAIT_CASE(6) TF_WAIT_CASE(7) TF_WAIT_CASE(8) TF_WAIT_CASE(9) TF_WAIT_CASE(10) TF_WAIT_CASE(11)
        TF_WAIT_CASE(12) TF_WAIT_CASE(13) TF_WAIT_CASE(14) TF_WAIT_CASE(15) TF_WAIT_CASE(16) TF_WAIT_CASE(17)
        TF_WAIT_CASE(18) TF_WAIT_CASE(19) TF_WAIT_CASE(20) TF_WAIT_CASE(21) TF_WAIT_CASE(22) TF_WAIT_CASE(23)
        TF_WAIT_CASE(24) TF_WAIT_CASE(25) TF_WAIT_CASE(26) TF_WAIT_CASE(27) TF_WAIT_CASE(28) TF_WAIT_CASE(29)
        TF_WAIT_CASE(30) TF_WAIT_CASE(31) TF_WAIT_CASE(32) TF_WAIT_CASE(33) TF_WAIT_CASE(34) TF_WAIT_CASE(35)
        TF_WAIT_CASE(36) TF_WAIT_CASE(37) TF_WAIT_CASE(38) TF_WAIT_CASE(39) TF_WAIT_CASE(40) TF_WAIT_CASE(41)
        TF_WAIT_CASE(42) TF_WAIT_CASE(43) TF_WAIT_CASE(44) TF_WAIT_CASE(45) TF_WAIT_CASE(46) TF_WAIT_CASE(47)
        TF_WAIT_CASE(48) TF_WAIT_CASE(49) TF_WAIT_CASE(50) TF_WAIT_CASE(51) TF_WAIT_CASE(52) TF_WAIT_CASE(53)
        TF_WAIT_CASE(54) TF_WAIT_CASE(55) TF_WAIT_CASE(56) TF_WAIT_CASE(57) TF_WAIT_CASE(58) TF_WAIT_CASE(59)
        TF_WAIT_CASE(60) TF_WAIT_CASE(61) TF_WAIT_CASE(62)
#undef TF_WAIT_CASE
        default: wait_vmcnt<62>(); break;
    }
}

__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }


}  // namespace tf

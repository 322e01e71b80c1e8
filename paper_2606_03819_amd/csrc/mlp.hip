// The AR approximator of Eq. 1 for every conditional row:
//   h'_r = h_{depth(r)} + W_down( silu(W_gate x_r) * (W_up x_r) ),
//   x_r  = [ rms(h_{depth(r)}) * g_h ; rms(Embd(prev_r)) * g_e ],
// the w/ Linear ablation h'_r = h_{depth(r)} + W_lin x_r, and the w/ 2-prev
// ablation whose x_r appends the normalised embedding of the token before
// prev_r (Ablations, Model Design).  Rows follow the tables in rows.hpp.
#include "common.hpp"
#include "launch.hpp"
#include "mlp_dma.hpp"
#include "plan.hpp"
#include "rows.hpp"
#include "stream_gemm.hpp"

namespace tf {

__device__ __forceinline__ float load_elem(const uint16_t* p, size_t i) { return bf16_bits_to_f32(p[i]); }
__device__ __forceinline__ float load_elem(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ void store_elem(uint16_t* p, size_t i, float v) { p[i] = (uint16_t)f32_to_bf16_bits(v); }
__device__ __forceinline__ void store_elem(float* p, size_t i, float v) { p[i] = v; }

// RMSNorm of the b*gamma drafter states (into ht) and of the npre previous-
// token embeddings of each of the b*R rows (into et, [b*R, npre*d], the
// nearer token first); one workgroup per vector.  bf16 outputs are rounded to
// nearest even: they are the bf16 operand x of the products that follow.
template <class T>
__global__ __launch_bounds__(256) void rmsnorm_rows_kernel(const T* __restrict__ h, const int32_t* __restrict__ root,
                                                           const int32_t* __restrict__ context,
                                                           const int32_t* __restrict__ topk,
                                                           const T* __restrict__ emb, const T* __restrict__ gh,
                                                           const T* __restrict__ ge, int b, int d, int V, RowTable rt,
                                                           int npre, float eps, T* __restrict__ ht,
                                                           T* __restrict__ et, int* __restrict__ diag,
                                                           int* __restrict__ counters, int ncounters) {
    __shared__ float red[4];
    if (diag != nullptr && blockIdx.x == 0 && threadIdx.x == 0) diag[0] = 0;
    if (blockIdx.x == 0)   // arrival counters of the products that follow on this stream
        for (int i = threadIdx.x; i < ncounters; i += 256) counters[i] = 0;
    const int row = blockIdx.x;
    const T* src;
    const T* gain;
    T* dst;
    if (row < b * rt.gamma) {
        src = h + (size_t)row * d;
        gain = gh;
        dst = ht + (size_t)row * d;
    } else {
        const int e = row - b * rt.gamma;
        const int rr = e / npre, which = e - rr * npre;
        const int s = rr / rt.Rs;
        int prev = rt.prev_token(s, rr - s * rt.Rs, which, root, context, topk);
        prev = min(max(prev, 0), V - 1);   // ids are documented to be < V; never read out of bounds
        src = emb + (size_t)prev * d;
        gain = ge;
        dst = et + (size_t)rr * npre * d + (size_t)which * d;
    }
    float ss = 0.f;
    for (int k = threadIdx.x; k < d; k += 256) {
        const float x = load_elem(src, k);
        ss = fmaf(x, x, ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = (red[0] + red[1]) + (red[2] + red[3]);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    for (int k = threadIdx.x; k < d; k += 256) {
        float y = load_elem(src, k) * inv;
        if (gain != nullptr) y *= load_elem(gain, k);
        store_elem(dst, k, y);
    }
}

// bf16 with every row 16-byte aligned: one wave per vector; each lane keeps
// its 16-byte pieces (pieces lane, lane + 64, ...; at most MAXC of them) in
// registers between the sum of squares and the scaling, so the vector is
// read once and the reduction needs no barrier.
template <int MAXC>
__global__ __launch_bounds__(256) void rmsnorm_rows_bf16_kernel(const uint16_t* __restrict__ h,
                                                                const int32_t* __restrict__ root,
                                                                const int32_t* __restrict__ context,
                                                                const int32_t* __restrict__ topk,
                                                                const uint16_t* __restrict__ emb,
                                                                const uint16_t* __restrict__ gh,
                                                                const uint16_t* __restrict__ ge, int b, int d, int V,
                                                                RowTable rt, int npre, float eps,
                                                                uint16_t* __restrict__ ht, uint16_t* __restrict__ et,
                                                                int* __restrict__ diag, int* __restrict__ counters,
                                                                int ncounters) {
    if (diag != nullptr && blockIdx.x == 0 && threadIdx.x == 0) diag[0] = 0;
    if (blockIdx.x == 0)   // arrival counters of the products that follow on this stream
        for (int i = threadIdx.x; i < ncounters; i += 256) counters[i] = 0;
    const int lane = threadIdx.x & 63;
    const int vec = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int nvec = b * rt.gamma + b * rt.Rs * npre;
    if (vec >= nvec) return;
    const uint16_t* src;
    const uint16_t* gain;
    uint16_t* dst;
    if (vec < b * rt.gamma) {
        src = h + (size_t)vec * d;
        gain = gh;
        dst = ht + (size_t)vec * d;
    } else {
        const int e = vec - b * rt.gamma;
        const int rr = e / npre, which = e - rr * npre;
        const int s = rr / rt.Rs;
        int prev = rt.prev_token(s, rr - s * rt.Rs, which, root, context, topk);
        prev = min(max(prev, 0), V - 1);   // ids are documented to be < V; never read out of bounds
        src = emb + (size_t)prev * d;
        gain = ge;
        dst = et + (size_t)rr * npre * d + (size_t)which * d;
    }
    const int npc = d >> 3;   // 16-byte pieces
    u32x4 v[MAXC], gv[MAXC];
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int pc = lane + 64 * c;
        if (pc < npc) {
            v[c] = *reinterpret_cast<const u32x4*>(src + 8 * pc);
            // the gains travel with the vector: one round trip for both
            gv[c] = gain != nullptr ? *reinterpret_cast<const u32x4*>(gain + 8 * pc)
                                    : u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};   // bf16 ones
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float lo = bf16_bits_to_f32(v[c][q] & 0xffffu), hi = bf16_bits_to_f32(v[c][q] >> 16);
                ss = fmaf(lo, lo, ss);
                ss = fmaf(hi, hi, ss);
            }
        }
    }
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int pc = lane + 64 * c;
        if (pc < npc) {
            u32x4 o;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float lo = bf16_bits_to_f32(v[c][q] & 0xffffu) * inv * bf16_bits_to_f32(gv[c][q] & 0xffffu);
                const float hi = bf16_bits_to_f32(v[c][q] >> 16) * inv * bf16_bits_to_f32(gv[c][q] >> 16);
                o[q] = f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
            }
            *reinterpret_cast<u32x4*>(dst + 8 * pc) = o;
        }
    }
}

// ------------------------------------------------------------------ bf16

template <int WM, int NT, int NW, int PIPE, bool WNT>
__global__ __launch_bounds__(64 * NW, 512 / (64 * NW)) void gateup_bf16_kernel(WRowsGateUp ws, XRowsConcat xs, GemmShape sh,
                                                                 uint16_t* __restrict__ act, int I, float* partial,
                                                                 int* counter) {
    __shared__ __align__(16) unsigned char smem[GemmTraits<WM, NT, NW>::SMEM_BYTES];
    EpiFixup<WM, NT, NW, EpiSwiGLU<WM, NT>> epi{EpiSwiGLU<WM, NT>{act, I}, partial, counter};
    stream_gemm<WM, NT, NW, PIPE, WNT>(ws, xs, epi, sh, smem);
}

// the plain SiLU MLP's input projection: tiles of 32 gate rows
template <int WM, int NT, int NW, int PIPE, bool WNT>
__global__ __launch_bounds__(64 * NW, 512 / (64 * NW)) void silu_gate_bf16_kernel(WRowsPlain ws, XRowsConcat xs,
                                                                                  GemmShape sh,
                                                                                  uint16_t* __restrict__ act, int I,
                                                                                  float* partial, int* counter) {
    __shared__ __align__(16) unsigned char smem[GemmTraits<WM, NT, NW>::SMEM_BYTES];
    EpiFixup<WM, NT, NW, EpiSiLU<WM, NT>> epi{EpiSiLU<WM, NT>{act, I}, partial, counter};
    stream_gemm<WM, NT, NW, PIPE, WNT>(ws, xs, epi, sh, smem);
}

template <int WM, int NT, int NW, int PIPE, bool WNT>
__global__ __launch_bounds__(64 * NW, 512 / (64 * NW)) void down_bf16_kernel(WRowsPairedK ws, XRowsPlain xs, GemmShape sh,
                                                               uint16_t* __restrict__ hp, const uint16_t* __restrict__ h,
                                                               int d, RowTable rt, float* partial, int* counter) {
    __shared__ __align__(16) unsigned char smem[GemmTraits<WM, NT, NW>::SMEM_BYTES];
    EpiFixup<WM, NT, NW, EpiResidual<WM, NT>> epi{EpiResidual<WM, NT>{hp, h, d, rt}, partial, counter};
    stream_gemm<WM, NT, NW, PIPE, WNT>(ws, xs, epi, sh, smem);
}

// The linear approximator: h' = h + W_lin [h~ ; e~].
template <int WM, int NT, int NW, int PIPE, bool WNT>
__global__ __launch_bounds__(64 * NW, 512 / (64 * NW)) void linear_bf16_kernel(WRowsPlain ws, XRowsConcat xs,
                                                                              GemmShape sh,
                                                                              uint16_t* __restrict__ hp,
                                                                              const uint16_t* __restrict__ h, int d,
                                                                              RowTable rt, float* partial,
                                                                              int* counter) {
    __shared__ __align__(16) unsigned char smem[GemmTraits<WM, NT, NW>::SMEM_BYTES];
    EpiFixup<WM, NT, NW, EpiResidual<WM, NT>> epi{EpiResidual<WM, NT>{hp, h, d, rt}, partial, counter};
    stream_gemm<WM, NT, NW, PIPE, WNT>(ws, xs, epi, sh, smem);
}

// ------------------------------------------------------------------ fp32

// x_r = [ht(depth) ; et(r)] is K = d + ew wide.
__global__ __launch_bounds__(256) void gateup_f32_kernel(const float* __restrict__ wg, const float* wu,
                                                         const float* __restrict__ ht, const float* __restrict__ et,
                                                         int rows, int d, int ew, int I, RowTable rt,
                                                         float* __restrict__ act) {
    const int r = blockIdx.y * 4 + (threadIdx.x >> 6);
    const int i = blockIdx.x * 64 + (threadIdx.x & 63);
    if (r >= rows || i >= I) return;
    const int s = r / rt.Rs;
    const int rl = r - s * rt.Rs;
    const int K = d + ew;
    const float* hr = ht + (size_t)(s * rt.gamma + rt.depth(rl) - 1) * d;
    const float* er = et + (size_t)r * ew;
    const float* g_row = wg + (size_t)i * K;
    float g = 0.f;
    for (int k = 0; k < d; ++k) g = fmaf(hr[k], g_row[k], g);
    for (int k = 0; k < ew; ++k) g = fmaf(er[k], g_row[d + k], g);
    float a = g / (1.0f + expf(-g));
    if (wu != nullptr) {   // SwiGLU; without it the plain SiLU MLP
        const float* u_row = wu + (size_t)i * K;
        float u = 0.f;
        for (int k = 0; k < d; ++k) u = fmaf(hr[k], u_row[k], u);
        for (int k = 0; k < ew; ++k) u = fmaf(er[k], u_row[d + k], u);
        a *= u;
    }
    act[(size_t)r * I + i] = a;
}

__global__ __launch_bounds__(256) void down_f32_kernel(const float* __restrict__ wd, const float* __restrict__ act,
                                                       const float* __restrict__ h, int rows, int d, int I,
                                                       RowTable rt, float* __restrict__ hp) {
    const int r = blockIdx.y * 4 + (threadIdx.x >> 6);
    const int n = blockIdx.x * 64 + (threadIdx.x & 63);
    if (r >= rows || n >= d) return;
    const int s = r / rt.Rs;
    const int rl = r - s * rt.Rs;
    const float* ar = act + (size_t)r * I;
    const float* wr = wd + (size_t)n * I;
    float y = 0.f;
    for (int i = 0; i < I; ++i) y = fmaf(ar[i], wr[i], y);
    hp[(size_t)r * d + n] = h[(size_t)(s * rt.gamma + rt.depth(rl) - 1) * d + n] + y;
}

__global__ __launch_bounds__(256) void linear_f32_kernel(const float* __restrict__ wl, const float* __restrict__ ht,
                                                         const float* __restrict__ et, const float* __restrict__ h,
                                                         int rows, int d, RowTable rt, float* __restrict__ hp) {
    const int r = blockIdx.y * 4 + (threadIdx.x >> 6);
    const int n = blockIdx.x * 64 + (threadIdx.x & 63);
    if (r >= rows || n >= d) return;
    const int s = r / rt.Rs;
    const int rl = r - s * rt.Rs;
    const int hrow = s * rt.gamma + rt.depth(rl) - 1;
    const float* hr = ht + (size_t)hrow * d;
    const float* er = et + (size_t)r * d;
    const float* w = wl + (size_t)n * 2 * d;
    float y = 0.f;
    for (int k = 0; k < d; ++k) y = fmaf(hr[k], w[k], y);
    for (int k = 0; k < d; ++k) y = fmaf(er[k], w[d + k], y);
    hp[(size_t)r * d + n] = h[(size_t)hrow * d + n] + y;
}

// ------------------------------------------------------------------ launcher

// SwiGLU gate/up, or the gate alone when wu is null (plain SiLU MLP)
template <int WM, int NT, int NW, int PIPE, bool WNT>
static void launch_gateup(const uint16_t* wg, const uint16_t* wu, const uint16_t* ht, const uint16_t* et,
                          uint16_t* act, int rows, int d, int ew, int I, const RowTable& rt, const GemmPlan& pg,
                          float* partial, int* counters, hipStream_t st) {
    XRowsConcat xc{ht, et, d, ew, rt};
    const GemmShape shg = pg.shape(rows, d + ew);
    if (wu != nullptr) {
        WRowsGateUp wgu{wg, wu, I, d + ew};
        hipLaunchKernelGGL((gateup_bf16_kernel<WM, NT, NW, PIPE, WNT>), dim3(shg.G), dim3(64 * NW), 0, st, wgu, xc,
                           shg, act, I, partial, counters);
    } else {
        WRowsPlain wgp{wg, I, d + ew};
        hipLaunchKernelGGL((silu_gate_bf16_kernel<WM, NT, NW, PIPE, WNT>), dim3(shg.G), dim3(64 * NW), 0, st, wgp,
                           xc, shg, act, I, partial, counters);
    }
}

// the activation is [rows, 2I] bf16 hi/lo pairs
template <int WM, int NT, int NW, int PIPE, bool WNT>
static void launch_down(const uint16_t* h, const uint16_t* wd, const uint16_t* act, uint16_t* hp, int rows, int d,
                        int I, const RowTable& rt, const GemmPlan& pd, float* partial, int* counters,
                        hipStream_t st) {
    WRowsPairedK wdn{wd, d, I};
    XRowsPlain xa{act, 2l * I};
    const GemmShape shd = pd.shape(rows, 2 * I);
    hipLaunchKernelGGL((down_bf16_kernel<WM, NT, NW, PIPE, WNT>), dim3(shd.G), dim3(64 * NW), 0, st, wdn, xa, shd,
                       hp, h, d, rt, partial, counters);
}

// Both products share the row blocking (same rows); each plan picks its own
// waves per workgroup.
template <int WM, int NT>
static void launch_mlp_bf16(const uint16_t* h, const uint16_t* wg, const uint16_t* wu, const uint16_t* wd,
                            const uint16_t* ht, const uint16_t* et, uint16_t* act, uint16_t* hp, int rows, int d,
                            int ew, int I, const RowTable& rt, const GemmPlan& pg, const GemmPlan& pd,
                            float* partial, int* counters, hipStream_t st) {
    constexpr int S = TF_NW_SINGLE, P = TF_PIPE_DEFAULT;
    if (pg.NW != S)
        launch_gateup<WM, NT, TF_NW, P, false>(wg, wu, ht, et, act, rows, d, ew, I, rt, pg, partial, counters, st);
    else
        launch_gateup<WM, NT, S, P, false>(wg, wu, ht, et, act, rows, d, ew, I, rt, pg, partial, counters, st);
    int* cd = counters + pg.counter_ints();
    if (pd.NW != S)
        launch_down<WM, NT, TF_NW, P, false>(h, wd, act, hp, rows, d, I, rt, pd, partial, cd, st);
    else
        launch_down<WM, NT, S, P, false>(h, wd, act, hp, rows, d, I, rt, pd, partial, cd, st);
}

static bool aligned16p(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <class T>
static void launch_norms(const void* h, const int32_t* root, const int32_t* context, const int32_t* topk,
                         const void* emb, const void* gh, const void* ge, int b, int d, int V, const RowTable& rt,
                         int npre, float eps, void* ht, void* et, int* diag, int* counters, int ncounters,
                         hipStream_t stream) {
    const int nvec = b * rt.gamma + b * rt.Rs * npre;
    constexpr int kMaxPieces = 16;   // d <= 16 * 64 * 8 = 8192 in registers
    if constexpr (sizeof(T) == 2) {
        // h rows are 16-byte aligned (checked at the boundary); the embedding and gains are only
        // required to be 4-byte aligned, so this path is taken when they happen to be 16-byte aligned
        if (d <= kMaxPieces * 64 * 8 && aligned16p(emb) && (gh == nullptr || aligned16p(gh)) &&
            (ge == nullptr || aligned16p(ge))) {
            hipLaunchKernelGGL(rmsnorm_rows_bf16_kernel<kMaxPieces>, dim3(cdiv(nvec, 4)), dim3(256), 0, stream,
                               static_cast<const uint16_t*>(h), root, context, topk,
                               static_cast<const uint16_t*>(emb), static_cast<const uint16_t*>(gh),
                               static_cast<const uint16_t*>(ge), b, d, V, rt, npre, eps,
                               static_cast<uint16_t*>(ht), static_cast<uint16_t*>(et), diag, counters, ncounters);
            return;
        }
    }
    hipLaunchKernelGGL(rmsnorm_rows_kernel<T>, dim3(nvec), dim3(256), 0, stream, static_cast<const T*>(h), root,
                       context, topk, static_cast<const T*>(emb), static_cast<const T*>(gh),
                       static_cast<const T*>(ge), b, d, V, rt, npre, eps, static_cast<T*>(ht), static_cast<T*>(et),
                       diag, counters, ncounters);
}

// ------------------------------------------------ one row block (mlp_dma.hpp)

// Ring depths: 40-70 KiB of weights in flight (SW - 1 stages of TG tiles,
// 4 KiB each), and two activation chunks; the down projection's 256-byte
// activation rows leave room for fewer weight stages.
template <int TG, bool PAIRED>
constexpr int mlp_dma_sw() {
    return PAIRED ? (TG == 2 ? 6 : 4) : (TG == 2 ? 10 : 5);
}
constexpr int kMlpDmaSX = 3;

template <int TG, int NTE, bool PAIRED, int WMAP, int EPI>
static hipError_t launch_mlp_dma_nte(const MlpDmaArgs& a, hipStream_t st) {
    constexpr int SW = mlp_dma_sw<TG, PAIRED>(), SX = kMlpDmaSX;
    using T = MlpDmaTraits<TG, NTE, PAIRED, SW, SX>;
    static_assert(T::SMEM <= 152 * 1024, "LDS of one workgroup");
    auto kern = mlp_dma_kernel<TG, NTE, PAIRED, SW, SX, WMAP, EPI>;
    const hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, T::SMEM);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.G), dim3(256), T::SMEM, st, a);
    return hipGetLastError();
}

template <bool PAIRED, int WMAP, int EPI>
static hipError_t launch_mlp_dma(const MlpDmaArgs& a, const MlpDmaPlan& p, hipStream_t st) {
    constexpr int TG = PAIRED ? TF_MLP_DMA_TG_DOWN : TF_MLP_DMA_TG_IN;
    if (p.TG != TG) return hipErrorInvalidValue;
    if (p.NTE == 1) return launch_mlp_dma_nte<TG, 1, PAIRED, WMAP, EPI>(a, st);
    if (p.NTE == 2) return launch_mlp_dma_nte<TG, 2, PAIRED, WMAP, EPI>(a, st);
    return launch_mlp_dma_nte<TG, 4, PAIRED, WMAP, EPI>(a, st);
}

static MlpDmaArgs mlp_dma_args(const MlpDmaPlan& p, const uint16_t* w, const uint16_t* wu, int N, int Kw,
                               const uint16_t* xh, const uint16_t* xe, long lde, int Rh, int Re, uint16_t* out,
                               int Nout, const uint16_t* h, const RowTable& rt, float* partial, int* counter) {
    return MlpDmaArgs{w,      wu,     N,       Kw,    xh,   xe,   lde,  Rh, Re,      p.ntiles, p.items,
                      p.nkh,  p.nke,  p.G,     out,   Nout, h,    rt,   partial, counter};
}

// Eq. 1 (or the plain SiLU MLP when w_up is null) for at most 128 rows and
// 32 drafter states: gate/up with the h~ half once per drafter state, then
// the down projection with the residual.
static hipError_t launch_arapprox_dma(const void* h, const int32_t* root, const int32_t* context,
                                      const int32_t* topk_idx, const void* emb, const void* gain_h,
                                      const void* gain_e, const void* w_gate, const void* w_up, const void* w_down,
                                      int b, int d, int I, int V, const RowTable& rt, int npre, float eps, void* ht,
                                      void* et, void* act, void* hp, float* partial, int* counters, int* diag,
                                      hipStream_t stream);

hipError_t launch_arapprox(const void* h, const int32_t* root, const int32_t* context, const int32_t* topk_idx,
                           const void* emb, const void* gain_h, const void* gain_e, const void* w_gate,
                           const void* w_up, const void* w_down, int b, int gamma, int d, int I, int V, int k,
                           bool bigram, float eps, bool bf16, void* ht, void* et, void* act, void* hp,
                           float* mlp_partial, int* counters, int* diag, hipStream_t stream) {
    const RowTable rt = make_row_table(gamma, k, bigram ? 1 : 0);
    const int npre = bigram ? 2 : 1;
    const int ew = npre * d;
    const int rows = b * rt.Rs;
    if (bf16) {
        if (mlp_dma_applies(true, b, gamma, rt.Rs, d, I, ew))
            return launch_arapprox_dma(h, root, context, topk_idx, emb, gain_h, gain_e, w_gate, w_up, w_down, b, d,
                                       I, V, rt, npre, eps, ht, et, act, hp, mlp_partial, counters, diag, stream);
        const GemmPlan pg = w_up != nullptr ? gateup_plan(rows, d + ew, I) : silu_gate_plan(rows, d + ew, I);
        const GemmPlan pd = down_plan(rows, d, I);
        const int ncounters = (int)(pg.counter_ints() + pd.counter_ints());
        launch_norms<uint16_t>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et, diag,
                               counters, ncounters, stream);
        const uint16_t* hb = static_cast<const uint16_t*>(h);
        const uint16_t* wg = static_cast<const uint16_t*>(w_gate);
        const uint16_t* wu = static_cast<const uint16_t*>(w_up);
        const uint16_t* wd = static_cast<const uint16_t*>(w_down);
        const uint16_t* htb = static_cast<const uint16_t*>(ht);
        const uint16_t* etb = static_cast<const uint16_t*>(et);
        uint16_t* actb = static_cast<uint16_t*>(act);
        uint16_t* hpb = static_cast<uint16_t*>(hp);
        if (pg.NT == 1)
            launch_mlp_bf16<2, 1>(hb, wg, wu, wd, htb, etb, actb, hpb, rows, d, ew, I, rt, pg, pd, mlp_partial,
                                  counters, stream);
        else if (pg.NT == 2)
            launch_mlp_bf16<1, 2>(hb, wg, wu, wd, htb, etb, actb, hpb, rows, d, ew, I, rt, pg, pd, mlp_partial,
                                  counters, stream);
        else
            launch_mlp_bf16<1, 4>(hb, wg, wu, wd, htb, etb, actb, hpb, rows, d, ew, I, rt, pg, pd, mlp_partial,
                                  counters, stream);
    } else {
        launch_norms<float>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et, diag,
                            counters, 0, stream);
        hipLaunchKernelGGL(gateup_f32_kernel, dim3(cdiv(I, 64), cdiv(rows, 4)), dim3(256), 0, stream,
                           static_cast<const float*>(w_gate), static_cast<const float*>(w_up),
                           static_cast<const float*>(ht), static_cast<const float*>(et), rows, d, ew, I, rt,
                           static_cast<float*>(act));
        hipLaunchKernelGGL(down_f32_kernel, dim3(cdiv(d, 64), cdiv(rows, 4)), dim3(256), 0, stream,
                           static_cast<const float*>(w_down), static_cast<const float*>(act),
                           static_cast<const float*>(h), rows, d, I, rt, static_cast<float*>(hp));
    }
    return hipGetLastError();
}

hipError_t launch_arapprox_linear(const void* h, const int32_t* root, const int32_t* topk_idx, const void* emb,
                                  const void* gain_h, const void* gain_e, const void* w_lin, int b, int gamma, int d,
                                  int V, int k, float eps, bool bf16, void* ht, void* et, void* hp,
                                  float* mlp_partial, int* counters, int* diag, hipStream_t stream) {
    const RowTable rt = make_row_table(gamma, k, 0);
    const int rows = b * rt.Rs;
    if (mlp_dma_applies(bf16, b, gamma, rt.Rs, d, 64, d)) {
        // one row block: the h~ half once per drafter state, residual epilogue
        const MlpDmaPlan pl = mlp_dma_linear_plan(rows, d);
        launch_norms<uint16_t>(h, root, nullptr, topk_idx, emb, gain_h, gain_e, b, d, V, rt, 1, eps, ht, et, diag,
                               counters, pl.items, stream);
        const uint16_t* hb = static_cast<const uint16_t*>(h);
        const MlpDmaArgs al = mlp_dma_args(pl, static_cast<const uint16_t*>(w_lin), nullptr, d, 2 * d,
                                           static_cast<const uint16_t*>(ht), static_cast<const uint16_t*>(et), d,
                                           b * gamma, rows, static_cast<uint16_t*>(hp), d, hb, rt, mlp_partial,
                                           counters);
        return launch_mlp_dma<false, kMlpWPlain, kMlpEpiResidual>(al, pl, stream);
    }
    if (bf16) {
        const GemmPlan pl = linear_plan(rows, d);
        launch_norms<uint16_t>(h, root, nullptr, topk_idx, emb, gain_h, gain_e, b, d, V, rt, 1, eps, ht, et, diag,
                               counters, (int)pl.counter_ints(), stream);
        WRowsPlain wr{static_cast<const uint16_t*>(w_lin), d, 2 * d};
        XRowsConcat xc{static_cast<const uint16_t*>(ht), static_cast<const uint16_t*>(et), d, d, rt};
        const GemmShape sh = pl.shape(rows, 2 * d);
        uint16_t* hpb = static_cast<uint16_t*>(hp);
        const uint16_t* hb = static_cast<const uint16_t*>(h);
        constexpr int S = TF_NW_SINGLE;
        if (pl.NT == 1)
            hipLaunchKernelGGL((linear_bf16_kernel<2, 1, S, TF_PIPE_DEFAULT, false>), dim3(sh.G), dim3(64 * S), 0,
                               stream, wr, xc, sh, hpb, hb, d, rt, mlp_partial, counters);
        else if (pl.NT == 2)
            hipLaunchKernelGGL((linear_bf16_kernel<1, 2, S, TF_PIPE_DEFAULT, false>), dim3(sh.G), dim3(64 * S), 0,
                               stream, wr, xc, sh, hpb, hb, d, rt, mlp_partial, counters);
        else if (pl.NW == S)
            hipLaunchKernelGGL((linear_bf16_kernel<1, 4, S, TF_PIPE_DEFAULT, false>), dim3(sh.G), dim3(64 * S), 0,
                               stream, wr, xc, sh, hpb, hb, d, rt, mlp_partial, counters);
        else
            hipLaunchKernelGGL((linear_bf16_kernel<1, 4, TF_NW, TF_PIPE_DEFAULT, false>), dim3(sh.G), dim3(64 * TF_NW),
                               0, stream, wr, xc, sh, hpb, hb, d, rt, mlp_partial, counters);
    } else {
        launch_norms<float>(h, root, nullptr, topk_idx, emb, gain_h, gain_e, b, d, V, rt, 1, eps, ht, et, diag,
                            counters, 0, stream);
        hipLaunchKernelGGL(linear_f32_kernel, dim3(cdiv(d, 64), cdiv(rows, 4)), dim3(256), 0, stream,
                           static_cast<const float*>(w_lin), static_cast<const float*>(ht),
                           static_cast<const float*>(et), static_cast<const float*>(h), rows, d, rt,
                           static_cast<float*>(hp));
    }
    return hipGetLastError();
}

static hipError_t launch_arapprox_dma(const void* h, const int32_t* root, const int32_t* context,
                                      const int32_t* topk_idx, const void* emb, const void* gain_h,
                                      const void* gain_e, const void* w_gate, const void* w_up, const void* w_down,
                                      int b, int d, int I, int V, const RowTable& rt, int npre, float eps, void* ht,
                                      void* et, void* act, void* hp, float* partial, int* counters, int* diag,
                                      hipStream_t stream) {
    const int ew = npre * d;
    const int rows = b * rt.Rs;
    const bool swiglu = w_up != nullptr;
    const MlpDmaPlan pg = mlp_dma_gate_plan(rows, d, ew, I, swiglu);
    const MlpDmaPlan pd = mlp_dma_down_plan(rows, d, I);
    launch_norms<uint16_t>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et, diag,
                           counters, pg.items + pd.items, stream);
    const uint16_t* hb = static_cast<const uint16_t*>(h);
    const uint16_t* htb = static_cast<const uint16_t*>(ht);
    const uint16_t* etb = static_cast<const uint16_t*>(et);
    uint16_t* actb = static_cast<uint16_t*>(act);
    const MlpDmaArgs ag = mlp_dma_args(pg, static_cast<const uint16_t*>(w_gate), static_cast<const uint16_t*>(w_up),
                                       I, d + ew, htb, etb, ew, b * rt.gamma, rows, actb, I, hb, rt, partial, counters);
    hipError_t e = swiglu ? launch_mlp_dma<false, kMlpWGateUp, kMlpEpiSwiGLU>(ag, pg, stream)
                          : launch_mlp_dma<false, kMlpWPlain, kMlpEpiSiLU>(ag, pg, stream);
    if (e != hipSuccess) return e;
    const MlpDmaArgs ad = mlp_dma_args(pd, static_cast<const uint16_t*>(w_down), nullptr, d, I, nullptr, actb, 2l * I,
                                       0, rows, static_cast<uint16_t*>(hp), d, hb, rt, partial, counters + pg.items);
    return launch_mlp_dma<true, kMlpWPlain, kMlpEpiResidual>(ad, pd, stream);
}

}  // namespace tf

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
#pragma unroll 4   // four loads in flight before the first use
    for (int k = threadIdx.x; k < d; k += 256) {
        const float x = load_elem(src, k);
        ss = fmaf(x, x, ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = (red[0] + red[1]) + (red[2] + red[3]);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    if (gain != nullptr) {
#pragma unroll 4
        for (int k = threadIdx.x; k < d; k += 256) store_elem(dst, k, load_elem(src, k) * inv * load_elem(gain, k));
    } else {
#pragma unroll 4
        for (int k = threadIdx.x; k < d; k += 256) store_elem(dst, k, load_elem(src, k) * inv);
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
    // Every load is issued before the first use: the branch per piece is
    // uniform and a lane past the row re-reads its last piece (its values are
    // dropped below), so the row and its gains take one round trip.
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        if (64 * c < npc) {
            const int pc = min(lane + 64 * c, npc - 1);
            v[c] = *reinterpret_cast<const u32x4*>(src + 8 * pc);
            gv[c] = gain != nullptr ? *reinterpret_cast<const u32x4*>(gain + 8 * pc)
                                    : u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};   // bf16 ones
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        if (64 * c < npc && lane + 64 * c < npc) {
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
                o[q] = f32x2_to_bf16x2_bits(lo, hi);
            }
            *reinterpret_cast<u32x4*>(dst + 8 * pc) = o;
        }
    }
}

// ------------------------------------------------------------------ bf16

// Any product of the approximator over several row blocks: `ws` weight rows
// against `xs` activation rows, the epilogue behind the split-k fix-up.
template <int WM, int NT, int NW, int PIPE, bool WNT, class WSrc, class XSrc, class Epi>
__global__ __launch_bounds__(64 * NW, 512 / (64 * NW)) void product_bf16_kernel(WSrc ws, XSrc xs, GemmShape sh,
                                                                              Epi epi) {
    __shared__ __align__(16) unsigned char smem[GemmTraits<WM, NT, NW>::SMEM_BYTES];
    stream_gemm<WM, NT, NW, PIPE, WNT>(ws, xs, epi, sh, smem);
}

// ------------------------------------------------------------------ fp32

// The approximator's fp32 products (small models): out[r, n] = epi( x_r . W[n] )
// with x_r = [x0 row of r's drafter state (d0 wide) ; x1 row r (K - d0 wide)].
// A workgroup holds 16 rows x 16 output columns; the reduction range streams
// through LDS in 64-wide chunks (every thread copies four activation and four
// weight values per chunk, consecutive threads consecutive k, the next
// chunk's loads in flight while this one is multiplied), and each thread
// accumulates its output with one fmaf chain in k order.
//   GATE:  act = silu(x . W_gate[n]) * (x . W_up[n])  (W_up null: silu alone)
//   else:  out = h[r's drafter state, n] + x . W[n]   (down projection, linear)
template <bool GATE>
__global__ __launch_bounds__(256) void mlp_f32_kernel(const float* __restrict__ wa, const float* __restrict__ wb,
                                                      int N, int K, const float* __restrict__ x0, int d0,
                                                      const float* __restrict__ x1, int ld1, RowTable rt, int rows,
                                                      const float* __restrict__ h, float* __restrict__ out,
                                                      int ldo) {
    __shared__ float xs[16][65];
    __shared__ float ws[2][16][65];
    const int tid = threadIdx.x;
    const int n0 = blockIdx.x * 16, r0 = blockIdx.y * 16;
    const int tx = tid & 15, ty = tid >> 4;
    const bool two = GATE && wb != nullptr;
    // the x0 row (drafter state) of each of the tile's rows
    auto state_of = [&](int r) {
        const int s = r / rt.Rs;
        return s * rt.gamma + rt.depth(r - s * rt.Rs) - 1;
    };
    // this thread's copies of a chunk: rows (and weight rows) e / 64, k e % 64, e = tid + 256 j
    int xrow[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = r0 + ((tid + 256 * j) >> 6);
        xrow[j] = r < rows ? state_of(r) : -1;
    }
    float px[4], pw[4], pw2[4];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = tid + 256 * j;
            const int rr = e >> 6, k = k0 + (e & 63);
            const int r = r0 + rr, n = n0 + rr;
            px[j] = pw[j] = pw2[j] = 0.f;
            if (xrow[j] >= 0 && k < K) px[j] = k < d0 ? x0[(size_t)xrow[j] * d0 + k] : x1[(size_t)r * ld1 + (k - d0)];
            if (n < N && k < K) {
                pw[j] = wa[(size_t)n * K + k];
                if (two) pw2[j] = wb[(size_t)n * K + k];
            }
        }
    };
    float acc_a = 0.f, acc_b = 0.f;
    fetch(0);
    for (int k0 = 0; k0 < K; k0 += 64) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = tid + 256 * j;
            xs[e >> 6][e & 63] = px[j];
            ws[0][e >> 6][e & 63] = pw[j];
            ws[1][e >> 6][e & 63] = pw2[j];
        }
        __syncthreads();
        if (k0 + 64 < K) fetch(k0 + 64);   // the next chunk's loads run under this chunk's products
        const int kn = min(64, K - k0);
        for (int kk = 0; kk < kn; ++kk) {
            const float xv = xs[ty][kk];
            acc_a = fmaf(xv, ws[0][tx][kk], acc_a);
            if (two) acc_b = fmaf(xv, ws[1][tx][kk], acc_b);
        }
        __syncthreads();
    }
    const int r = r0 + ty, n = n0 + tx;
    if (r >= rows || n >= N) return;
    if constexpr (GATE) {
        float a = acc_a / (1.0f + expf(-acc_a));
        if (two) a *= acc_b;
        out[(size_t)r * ldo + n] = a;
    } else {
        out[(size_t)r * ldo + n] = h[(size_t)state_of(r) * N + n] + acc_a;
    }
}

// ------------------------------------------------------------------ launcher

// Epilogue makers: each product's epilogue for the (WM, NT) its plan picks.
struct MakeStoreH {   // the h~ half: fp32 table, one row per drafter state
    float* out;
    int ldo;
    template <int WM, int NT>
    EpiStoreF32<WM, NT> make() const { return EpiStoreF32<WM, NT>{out, ldo}; }
};
struct MakeSwiGLUH {   // the e~ half of gate/up: + h~ half, SwiGLU
    uint16_t* act;
    int I;
    const float* hh;
    int ldh;
    RowTable rt;
    template <int WM, int NT>
    EpiAddH<WM, NT, EpiSwiGLU<WM, NT>> make() const {
        return EpiAddH<WM, NT, EpiSwiGLU<WM, NT>>{EpiSwiGLU<WM, NT>{act, I}, hh, ldh, rt};
    }
};
struct MakeSiLUH {   // the e~ half of the plain SiLU gate
    uint16_t* act;
    int I;
    const float* hh;
    int ldh;
    RowTable rt;
    template <int WM, int NT>
    EpiAddH<WM, NT, EpiSiLU<WM, NT>> make() const {
        return EpiAddH<WM, NT, EpiSiLU<WM, NT>>{EpiSiLU<WM, NT>{act, I}, hh, ldh, rt};
    }
};
struct MakeResidual {   // the down projection: + h
    uint16_t* hp;
    const uint16_t* h;
    int d;
    RowTable rt;
    template <int WM, int NT>
    EpiResidual<WM, NT> make() const { return EpiResidual<WM, NT>{hp, h, d, rt}; }
};
struct MakeResidualH {   // the e~ half of the linear layer: + h~ half, + h
    uint16_t* hp;
    const uint16_t* h;
    int d;
    RowTable rt;
    const float* hh;
    int ldh;
    template <int WM, int NT>
    EpiAddH<WM, NT, EpiResidual<WM, NT>> make() const {
        return EpiAddH<WM, NT, EpiResidual<WM, NT>>{EpiResidual<WM, NT>{hp, h, d, rt}, hh, ldh, rt};
    }
};

template <int WM, int NT, class WSrc, class XSrc, class Maker>
static void run_product_nt(const GemmPlan& p, const WSrc& ws, const XSrc& xs, int rows, int K, const Maker& mk,
                           float* partial, int* counters, hipStream_t st) {
    constexpr int S = TF_NW_SINGLE, P = TF_PIPE_DEFAULT;
    using Inner = decltype(mk.template make<WM, NT>());
    const GemmShape sh = p.shape(rows, K);
    if (p.NW != S) {
        using E = EpiFixup<WM, NT, TF_NW, Inner>;
        hipLaunchKernelGGL((product_bf16_kernel<WM, NT, TF_NW, P, false, WSrc, XSrc, E>), dim3(sh.G),
                           dim3(64 * TF_NW), 0, st, ws, xs, sh, E{mk.template make<WM, NT>(), partial, counters});
    } else {
        using E = EpiFixup<WM, NT, S, Inner>;
        hipLaunchKernelGGL((product_bf16_kernel<WM, NT, S, P, false, WSrc, XSrc, E>), dim3(sh.G), dim3(64 * S), 0,
                           st, ws, xs, sh, E{mk.template make<WM, NT>(), partial, counters});
    }
}

// One product with the tile shape its plan picks (plan_nt / plan_wm).
template <class WSrc, class XSrc, class Maker>
static void run_product(const GemmPlan& p, const WSrc& ws, const XSrc& xs, int rows, int K, const Maker& mk,
                        float* partial, int* counters, hipStream_t st) {
    if (p.NT == 1)
        run_product_nt<2, 1>(p, ws, xs, rows, K, mk, partial, counters, st);
    else if (p.NT == 2)
        run_product_nt<1, 2>(p, ws, xs, rows, K, mk, partial, counters, st);
    else
        run_product_nt<1, 4>(p, ws, xs, rows, K, mk, partial, counters, st);
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

// Ring depths: SW - 1 weight stages in flight (TG tiles of 4 KiB each) and
// two activation chunks.  Every copy of a workgroup fills LDS through the
// same per-CU path (~45 GB/s measured for weights and activations alike), so
// the down projection, whose 256-byte activation rows make the activation
// four fifths of its bytes, keeps three weight stages in flight (measured
// faster than four or five); the input projections are insensitive to
// four to six.
template <int TG, bool PAIRED, int NTE>
constexpr int mlp_dma_sw() {
    return PAIRED ? 4 : (TG == 2 ? 10 : (NTE == 8 ? 4 : 5));
}
// activation stages: eight tiles' 32 KiB chunks leave room for one in flight
template <int NTE>
constexpr int mlp_dma_sx() {
    return NTE == 8 ? 2 : 3;
}

template <int TG, int NTE, bool PAIRED, int WMAP, int EPI>
static hipError_t launch_mlp_dma_nte(const MlpDmaArgs& a, hipStream_t st) {
    constexpr int SW = mlp_dma_sw<TG, PAIRED, NTE>(), SX = mlp_dma_sx<NTE>();
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
    if constexpr (!PAIRED && EPI != kMlpEpiResidual) {   // eight tiles: the input projections only
        if (p.NTE == 8) return launch_mlp_dma_nte<TG, 8, PAIRED, WMAP, EPI>(a, st);
    }
    if (p.NTE != 4) return hipErrorInvalidValue;
    return launch_mlp_dma_nte<TG, 4, PAIRED, WMAP, EPI>(a, st);
}

static MlpDmaArgs mlp_dma_args(const MlpDmaPlan& p, const uint16_t* w, const uint16_t* wu, int N, int Kw,
                               const uint16_t* xh, const uint16_t* xe, long lde, int Rh, int Re, uint16_t* out,
                               int Nout, const uint16_t* h, const RowTable& rt, float* partial, int* counter) {
    return MlpDmaArgs{w,     wu,    N,   Kw,   xh,   xe,   lde, Rh,   Re,      p.ntiles, p.items, p.nkh,
                      p.nke, p.G,   p.wh, p.we, out, Nout, h,  rt,   partial, counter};
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
                           float* mlp_partial, int* counters, float* hh, int* diag, hipStream_t stream) {
    const RowTable rt = make_row_table(gamma, k, bigram ? 1 : 0);
    const int npre = bigram ? 2 : 1;
    const int ew = npre * d;
    const int rows = b * rt.Rs;
    if (bf16) {
        if (mlp_dma_applies(true, b, gamma, rt.Rs, d, I, ew))
            return launch_arapprox_dma(h, root, context, topk_idx, emb, gain_h, gain_e, w_gate, w_up, w_down, b, d,
                                       I, V, rt, npre, eps, ht, et, act, hp, mlp_partial, counters, diag, stream);
        if (mlp_dma_gate_applies(true, b, gamma, rt.Rs, d, I, ew)) {
            // 129-256 rows: the input projections on the one-row-block kernel
            // (eight activation tiles), the down projection over several row blocks
            const bool swiglu = w_up != nullptr;
            const MlpDmaPlan pg = mlp_dma_gate_plan(rows, d, ew, I, swiglu);
            const GemmPlan pd = down_plan(rows, d, I);
            launch_norms<uint16_t>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et,
                                   diag, counters, (int)(pg.items + pd.counter_ints()), stream);
            const uint16_t* hb = static_cast<const uint16_t*>(h);
            uint16_t* actb = static_cast<uint16_t*>(act);
            const MlpDmaArgs ag = mlp_dma_args(pg, static_cast<const uint16_t*>(w_gate),
                                               static_cast<const uint16_t*>(w_up), I, d + ew,
                                               static_cast<const uint16_t*>(ht), static_cast<const uint16_t*>(et),
                                               ew, b * rt.gamma, rows, actb, I, hb, rt, mlp_partial, counters);
            const hipError_t e = swiglu ? launch_mlp_dma<false, kMlpWGateUp, kMlpEpiSwiGLU>(ag, pg, stream)
                                        : launch_mlp_dma<false, kMlpWPlain, kMlpEpiSiLU>(ag, pg, stream);
            if (e != hipSuccess) return e;
            run_product(pd, WRowsPairedK{static_cast<const uint16_t*>(w_down), d, I}, XRowsPlain{actb, 2l * I},
                        rows, 2 * I, MakeResidual{static_cast<uint16_t*>(hp), hb, d, rt}, mlp_partial,
                        counters + pg.items, stream);
            return hipGetLastError();
        }
        // several row blocks: the input projection split at the h~ / e~ boundary
        // (the h~ half once per drafter state), then the down projection
        const bool swiglu = w_up != nullptr;
        const int states = b * rt.gamma;
        const SplitPlans sp = split_plans(swiglu ? 0 : 1, states, rows, d, ew, I);
        const GemmPlan pd = down_plan(rows, d, I);
        launch_norms<uint16_t>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et, diag,
                               counters, (int)(sp.counter_ints() + pd.counter_ints()), stream);
        const uint16_t* hb = static_cast<const uint16_t*>(h);
        const uint16_t* wg = static_cast<const uint16_t*>(w_gate);
        const uint16_t* wu = static_cast<const uint16_t*>(w_up);
        const XRowsPlain xh{static_cast<const uint16_t*>(ht), d};
        const XRowsPlain xe{static_cast<const uint16_t*>(et), ew};
        uint16_t* actb = static_cast<uint16_t*>(act);
        int* ce = counters + sp.ph.counter_ints();
        int* cd = ce + sp.pe.counter_ints();
        if (swiglu) {
            run_product(sp.ph, WRowsGateUp{wg, wu, I, d + ew}, xh, states, d, MakeStoreH{hh, sp.ldh()}, mlp_partial,
                        counters, stream);
            run_product(sp.pe, WRowsGateUp{wg + d, wu + d, I, d + ew}, xe, rows, ew,
                        MakeSwiGLUH{actb, I, hh, sp.ldh(), rt}, mlp_partial, ce, stream);
        } else {
            run_product(sp.ph, WRowsPlain{wg, I, d + ew}, xh, states, d, MakeStoreH{hh, sp.ldh()}, mlp_partial,
                        counters, stream);
            run_product(sp.pe, WRowsPlain{wg + d, I, d + ew}, xe, rows, ew, MakeSiLUH{actb, I, hh, sp.ldh(), rt},
                        mlp_partial, ce, stream);
        }
        run_product(pd, WRowsPairedK{static_cast<const uint16_t*>(w_down), d, I}, XRowsPlain{actb, 2l * I}, rows,
                    2 * I, MakeResidual{static_cast<uint16_t*>(hp), hb, d, rt}, mlp_partial, cd, stream);
    } else {
        launch_norms<float>(h, root, context, topk_idx, emb, gain_h, gain_e, b, d, V, rt, npre, eps, ht, et, diag,
                            counters, 0, stream);
        hipLaunchKernelGGL(mlp_f32_kernel<true>, dim3(cdiv(I, 16), cdiv(rows, 16)), dim3(256), 0, stream,
                           static_cast<const float*>(w_gate), static_cast<const float*>(w_up), I, d + ew,
                           static_cast<const float*>(ht), d, static_cast<const float*>(et), ew, rt, rows, nullptr,
                           static_cast<float*>(act), I);
        hipLaunchKernelGGL(mlp_f32_kernel<false>, dim3(cdiv(d, 16), cdiv(rows, 16)), dim3(256), 0, stream,
                           static_cast<const float*>(w_down), nullptr, d, I, nullptr, 0,
                           static_cast<const float*>(act), I, rt, rows, static_cast<const float*>(h),
                           static_cast<float*>(hp), d);
    }
    return hipGetLastError();
}

hipError_t launch_arapprox_linear(const void* h, const int32_t* root, const int32_t* topk_idx, const void* emb,
                                  const void* gain_h, const void* gain_e, const void* w_lin, int b, int gamma, int d,
                                  int V, int k, float eps, bool bf16, void* ht, void* et, void* hp,
                                  float* mlp_partial, int* counters, float* hh, int* diag, hipStream_t stream) {
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
        // several row blocks: the h~ half once per drafter state, then the e~ half with the residual
        const int states = b * gamma;
        const SplitPlans sp = split_plans(2, states, rows, d, d, d);
        launch_norms<uint16_t>(h, root, nullptr, topk_idx, emb, gain_h, gain_e, b, d, V, rt, 1, eps, ht, et, diag,
                               counters, (int)sp.counter_ints(), stream);
        const uint16_t* wl = static_cast<const uint16_t*>(w_lin);
        run_product(sp.ph, WRowsPlain{wl, d, 2 * d}, XRowsPlain{static_cast<const uint16_t*>(ht), d}, states, d,
                    MakeStoreH{hh, sp.ldh()}, mlp_partial, counters, stream);
        run_product(sp.pe, WRowsPlain{wl + d, d, 2 * d}, XRowsPlain{static_cast<const uint16_t*>(et), d}, rows, d,
                    MakeResidualH{static_cast<uint16_t*>(hp), static_cast<const uint16_t*>(h), d, rt, hh, sp.ldh()},
                    mlp_partial, counters + sp.ph.counter_ints(), stream);
    } else {
        launch_norms<float>(h, root, nullptr, topk_idx, emb, gain_h, gain_e, b, d, V, rt, 1, eps, ht, et, diag,
                            counters, 0, stream);
        hipLaunchKernelGGL(mlp_f32_kernel<false>, dim3(cdiv(d, 16), cdiv(rows, 16)), dim3(256), 0, stream,
                           static_cast<const float*>(w_lin), nullptr, d, 2 * d, static_cast<const float*>(ht), d,
                           static_cast<const float*>(et), d, rt, rows, static_cast<const float*>(h),
                           static_cast<float*>(hp), d);
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

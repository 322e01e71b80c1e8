// LM head with online log-sum-exp and top-k (Appendix B, Part 1: q = LMHead(h),
// TopM, and the conditional rows q').  The [rows, V] logits never reach
// memory: each workgroup reduces its vocabulary slice to a (row, slice)
// partial, and one merge workgroup per row turns the partials into the row's
// log-sum-exp and exact top-k.
#include "common.hpp"
#include "dma.hpp"
#include "launch.hpp"
#include "plan.hpp"
#include "stream_gemm.hpp"

namespace tf {

// ------------------------------------------------------------ bf16 / MFMA

// One workgroup per (tile range, row block): the range's rounds in turn, each
// a full pass over K reduced to a (row, slice) partial.
template <int WM, int NT, int NW, int PIPE, bool WNT, bool LONG>
__global__ __launch_bounds__(64 * NW, 1) void lmhead_bf16_kernel(const uint16_t* __restrict__ x, long ldx,
                                                                               const uint16_t* __restrict__ w,
                                                                               GemmShape sh, SliceMap map, int V,
                                                                               float sl2, float* __restrict__ part,
                                                                               int* __restrict__ diag) {
    using Tr = GemmTraits<WM, NT, NW>;
    using E = EpiLmHead<WM, NT, NW, LONG>;
    constexpr int SMEM = Tr::SMEM_BYTES > E::MERGE_BYTES ? Tr::SMEM_BYTES : E::MERGE_BYTES;
    __shared__ __align__(16) unsigned char smem[SMEM];
    if (diag != nullptr && blockIdx.x == 0 && threadIdx.x == 0) diag[0] = 0;
    WRowsPlain ws{w, V, sh.K};
    XRowsPlain xs{x, ldx};
    E epi{part, V, sl2};
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int rb = L % sh.nrb;
    const int g = L / sh.nrb;
    GemmShape se = sh;   // the epilogue indexes partials by slice
    se.nchunks = map.G * map.rmax;
    for (int r = 0; r < map.rmax; ++r) {
        Segment seg;
        seg.g = L;
        seg.item = seg.chunk = g * map.rmax + r;
        seg.rb = rb;
        slice_tiles(map, seg.chunk, seg.t0, seg.t1);
        seg.kc0 = 0;
        seg.kc1 = sh.nk;
        seg.row0 = rb * Tr::TR;
        seg.gfirst = L;
        seg.npieces = 1;
        if (seg.t0 == seg.t1) {   // empty slice: a partial the merge skips
            const int t = threadIdx.x;
            if (t < Tr::TR && seg.row0 + t < sh.R) {
                float* o = part + ((size_t)(seg.row0 + t) * se.nchunks + seg.chunk) * part_stride(E::KEEP);
                o[0] = neg_inf();
                o[1] = 0.f;
                o[2] = neg_inf();
                o[3] = __int_as_float(0);
            }
            continue;
        }
        f32x16 acc[WM][NT];
        gemm_segment<WM, NT, NW, PIPE, WNT>(ws, xs, sh, seg, acc, smem);
        __syncthreads();  // LDS tiles no longer needed
        epi.apply(acc, seg, smem, se);
        lds_barrier();  // the epilogue's LDS use ends before the next round's tiles land
    }
}

// ------------------------------------------------ bf16 / MFMA, LDS DMA
//
// The same vocabulary slices with the weight and activation tiles copied
// from memory straight into LDS (global_load_lds_dwordx4, no register
// staging), so that the registers go to accumulators.  The NW waves form a
// grid of NW / WB along the weight tiles (WM each) times WB along the
// activation tiles (NT / WB each); the WB waves of a weight column split its
// copies (WNT: they carry the non-temporal hint).  k advances KC at a time.
// The weight tiles ([32 rows][KC] per tile) go through a ring of S stages,
// copied S - 1 steps ahead; the activation tile ([32*NT rows][KC]) through a
// ring of two, copied one step ahead from L2.  After the step's barrier a
// wave issues the next activation copies, then spreads the weight copies of
// step j + S - 1 over its MFMA sub-steps; waiting for the activation copies
// (issue order) also retires the older weight copies.  One
// DMA instruction fills 1 KiB: 1024 / (2 KC) whole rows, lane l taking
// 16-byte slot l % (KC / 8) of row l / (KC / 8).  Slots are XOR-swizzled per
// row so that the 16 rows one quarter-wave reads at one logical slot cover
// all 64 banks.

template <int WM, int NT, int NW, int KC, int S, int WB = 1>
struct DmaTraits {
    static constexpr int WA = NW / WB;                        // waves along the weight tiles
    static constexpr int NTW = NT / WB;                       // activation tiles per wave
    static constexpr int ROWB = KC * 2;                       // bytes of one tile row in one stage
    static constexpr int SLOTS = KC / 8;                      // 16-byte slots per row
    static constexpr int RPI = 1024 / ROWB;                   // rows per DMA instruction
    static constexpr int WTILE = 32 * ROWB;                   // one weight tile of one stage
    static constexpr int WINSTR = 32 / RPI;                   // DMA instructions per weight tile
    static constexpr int WSTAGE = WA * WM * WTILE;            // all waves' weight tiles of one stage
    static constexpr int XSTAGE = 32 * NT * ROWB;             // the activation tile of one stage
    static constexpr int XINSTR = XSTAGE / 1024;              // its DMA instructions, spread over the waves
    static constexpr int XOFF = S * WSTAGE;                   // activation ring after the weight ring
    static constexpr int RING = S * WSTAGE + 2 * XSTAGE;
    static constexpr int WPI = WINSTR / WB;                   // DMA instructions of a shared tile per wave
    static constexpr int WPS = WPI * WM;                      // weight DMA instructions per wave per step
    static_assert(NW % WB == 0 && NT % WB == 0 && WINSTR % WB == 0, "wave grid");
    static_assert(KC == 32 || KC == 64, "k step");
    // Copies are issued in the order w(0) .. w(S-3), x(0), w(S-2), then
    // during step j: x(j+1), w(j+S-1).  S >= 3 puts w(j) before x(j), and
    // after x(j) come only the WPS copies of w(j+S-2).
    static_assert(S >= 3 && WPS < 64, "ring depth, vmcnt range");
    // byte offset of 16-byte logical slot `ls` of row `r`
    __device__ static __forceinline__ int slot(int r, int ls) {
        const int sw = KC == 32 ? ((r >> 2) & 3) : ((r >> 1) & 7);
        return r * ROWB + ((ls ^ sw) << 4);
    }
};


template <int WM, int NT, int NW, int KC, int S, bool WNT, int MINB, bool LONG, int WB>
__global__ __launch_bounds__(64 * NW, MINB) void lmhead_dma_kernel(const uint16_t* __restrict__ x, long ldx,
                                                                const uint16_t* __restrict__ w, GemmShape sh,
                                                                SliceMap map, int V, float sl2,
                                                                float* __restrict__ part, int* __restrict__ diag) {
    using T = DmaTraits<WM, NT, NW, KC, S, WB>;
    using E = EpiLmHead<WM, NT, NW, LONG, WB>;
    constexpr int NTW = T::NTW;
    static_assert(E::MERGE_BYTES <= T::RING, "the epilogue reuses the rings");
    extern __shared__ __align__(16) unsigned char dyn[];
    if (diag != nullptr && blockIdx.x == 0 && threadIdx.x == 0) diag[0] = 0;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // wave grid: WA waves along the weight tiles times WB along the activation
    // tiles; the WB waves of one weight column share its tiles' copies
    const int wa = wave % T::WA, wb = wave / T::WA;
    E epi{part, V, sl2};
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int rb = L % sh.nrb;
    const int g = L / sh.nrb;
    GemmShape se = sh;   // the epilogue indexes partials by slice
    se.nchunks = map.G * map.rmax;
    const int nsteps = sh.K / KC;
    // this lane's piece of every 1 KiB DMA block
    const int lrow = lane / T::SLOTS;
    const int lphys = lane % T::SLOTS;

    for (int r = 0; r < map.rmax; ++r) {
        Segment seg;
        seg.g = L;
        seg.item = seg.chunk = g * map.rmax + r;
        seg.rb = rb;
        slice_tiles(map, seg.chunk, seg.t0, seg.t1);
        seg.kc0 = 0;
        seg.kc1 = sh.nk;
        seg.row0 = rb * 32 * NT;
        seg.gfirst = L;
        seg.npieces = 1;
        if (seg.t0 == seg.t1) {   // empty slice: a partial the merge skips
            const int t = threadIdx.x;
            if (t < 32 * NT && seg.row0 + t < sh.R) {
                float* o = part + ((size_t)(seg.row0 + t) * se.nchunks + seg.chunk) * part_stride(E::KEEP);
                o[0] = neg_inf();
                o[1] = 0.f;
                o[2] = neg_inf();
                o[3] = __int_as_float(0);
            }
            continue;
        }
        // global sources of this lane's DMA pieces (k offset added per step):
        // the piece landing at physical slot lphys of row `row` is logical
        // slot lphys ^ swizzle(row).  Tiles past the slice repeat its last
        // tile and vocabulary rows past V repeat row V-1, so every load stays
        // inside w; the epilogue masks those products.  (They are computed
        // anyway: a per-tile branch in the k loop costs more in MFMA-bound
        // launches, whose slices are all full, than the spare products cost
        // in the memory-bound ones.)
        const int tw = seg.t0 + wa * WM;
        const uint16_t* wsrc[WM][T::WPI];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int hi = 0; hi < T::WPI; ++hi) {
                const int row = T::RPI * (wb * T::WPI + hi) + lrow;
                const int tile = min(tw + mt, seg.t1 - 1);
                const int v = min(tile * 32 + row, V - 1);
                wsrc[mt][hi] = w + (size_t)v * sh.K + (T::slot(row, lphys) - row * T::ROWB) / 2;
            }
        constexpr int XPW = (T::XINSTR + NW - 1) / NW;   // activation instructions of this wave (at most)
        const uint16_t* xsrc[XPW];
#pragma unroll
        for (int i = 0; i < XPW; ++i) {
            const int blk = min(wave + NW * i, T::XINSTR - 1);   // block of RPI activation rows
            const int row = T::RPI * blk + lrow;
            const int gr = min(seg.row0 + row, sh.R - 1);
            xsrc[i] = x + (size_t)gr * ldx + (T::slot(row, lphys) - row * T::ROWB) / 2;
        }
        auto issue_w = [&](int step) {
            unsigned char* st = dyn + (step % S) * T::WSTAGE;
            const int k0 = step * KC;
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int hi = 0; hi < T::WPI; ++hi)
                    __builtin_amdgcn_global_load_lds(
                        (global_void_t*)(wsrc[mt][hi] + k0),
                        (lds_void_t*)(st + (wa * WM + mt) * T::WTILE + (wb * T::WPI + hi) * 1024), 16, 0,
                        WNT ? kCpolNt : 0);
        };
        // the weight copies q = mt * WPI + hi of step `step` with q % (KC / 16) == part
        auto issue_w_part = [&](int step, int part) {
            unsigned char* st = dyn + (step % S) * T::WSTAGE;
            const int k0 = step * KC;
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int hi = 0; hi < T::WPI; ++hi)
                    if ((mt * T::WPI + hi) % (KC / 16) == part)
                        __builtin_amdgcn_global_load_lds(
                            (global_void_t*)(wsrc[mt][hi] + k0),
                            (lds_void_t*)(st + (wa * WM + mt) * T::WTILE + (wb * T::WPI + hi) * 1024), 16, 0,
                            WNT ? kCpolNt : 0);
        };
        auto issue_x = [&](int step) {
            unsigned char* st = dyn + T::XOFF + (step & 1) * T::XSTAGE;
            const int k0 = step * KC;
#pragma unroll
            for (int i = 0; i < XPW; ++i)
                if (wave + NW * i < T::XINSTR)   // uniform per wave
                    __builtin_amdgcn_global_load_lds((global_void_t*)(xsrc[i] + k0),
                                                     (lds_void_t*)(st + (wave + NW * i) * 1024), 16, 0, 0);
        };
        f32x16 acc[WM][NTW];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
                for (int j = 0; j < 16; ++j) acc[mt][nt][j] = 0.f;

        // prologue: weight steps 0 .. S-3, activation step 0, weight step S-2
#pragma unroll
        for (int p = 0; p < S - 2; ++p)
            if (p < nsteps) issue_w(p);
        issue_x(0);
        if (S - 2 < nsteps) issue_w(S - 2);
        for (int j = 0; j < nsteps; ++j) {
            // this wave's copies of step j have landed (only w(j+S-2) may
            // still be out); the other waves' too after the barrier, which
            // also frees the stages read in step j - 1
            if (j + S - 2 < nsteps)
                wait_vmcnt<T::WPS>();
            else
                wait_vmcnt<0>();
            block_barrier();
            const unsigned char* wt = dyn + (j % S) * T::WSTAGE + wa * WM * T::WTILE;
            const unsigned char* xt = dyn + T::XOFF + (j & 1) * T::XSTAGE + wb * NTW * 32 * T::ROWB;
#pragma unroll
            for (int ks = 0; ks < KC / 16; ++ks) {
                const int ls = 2 * ks + (lane >> 5);
                u32x4 afr[WM], bfr[NTW];
                // refill the freed stages between the MFMAs: the activation
                // step first, the weight copies spread over the k sub-steps
                // (issued in one burst they held the wave off its MFMAs)
                if (ks == 0 && j + 1 < nsteps) issue_x(j + 1);
                if (j + S - 1 < nsteps) issue_w_part(j + S - 1, ks);
#pragma unroll
                for (int mt = 0; mt < WM; ++mt)
                    afr[mt] = *reinterpret_cast<const u32x4*>(wt + mt * T::WTILE + T::slot(lane & 31, ls));
#pragma unroll
                for (int nt = 0; nt < NTW; ++nt)
                    bfr[nt] = *reinterpret_cast<const u32x4*>(xt + T::slot(nt * 32 + (lane & 31), ls));
#pragma unroll
                for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                    for (int nt = 0; nt < NTW; ++nt) acc[mt][nt] = mfma_32x32x16_bf16(afr[mt], bfr[nt], acc[mt][nt]);
            }
        }
        __syncthreads();  // ring reads done before the epilogue reuses the LDS
        epi.apply(acc, seg, dyn, se);
        lds_barrier();  // the epilogue's LDS use ends before the next round's copies land
    }
}

// ------------------------------------------------------------ fp32 / SIMT
//
// The fp32 workloads are small; this kernel keeps the same partial format
// with plain FMA: a workgroup holds 32 activation rows, each thread one
// vocabulary row of the current 256-row step, and every (row, 1/8 of the
// step) pair is one contributor list.
__global__ __launch_bounds__(256) void lmhead_f32_kernel(const float* __restrict__ x, long ldx,
                                                         const float* __restrict__ w, GemmShape sh, SliceMap map,
                                                         int V, float sl2, float* __restrict__ part,
                                                         int* __restrict__ diag) {
    __shared__ float xs[32][65];
    __shared__ float lt[32][257];
    if (diag != nullptr && blockIdx.x == 0 && threadIdx.x == 0) diag[0] = 0;
    const int tid = threadIdx.x;
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int split = L / sh.nrb;   // one tile range of at most 8 tiles, one slice (rmax = 1)
    const int rb = L - split * sh.nrb;
    const int row0 = rb * 32;
    int t0, t1;
    slice_tiles(map, split, t0, t1);
    const int vend = min(V, t1 * 32);
    const int srow = tid >> 3, sub = tid & 7;

    float m = neg_inf(), s = 0.f;
    float lv[kLane];
    int li[kLane];
#pragma unroll
    for (int q = 0; q < kLane; ++q) {
        lv[q] = neg_inf();
        li[q] = -1;
    }
    int seen = 0;

    for (int ct = t0; ct < t1; ct += 8) {
        const int v = ct * 32 + tid;
        const bool vok = v < vend;
        float acc[32];
#pragma unroll
        for (int r = 0; r < 32; ++r) acc[r] = 0.f;
        for (int k0 = 0; k0 < sh.K; k0 += 64) {
            __syncthreads();
            for (int i = 0; i < 8; ++i) {
                const int e = tid + 256 * i;
                const int r = e >> 6, c = e & 63;
                const int gr = row0 + r, k = k0 + c;
                xs[r][c] = (gr < sh.R && k < sh.K) ? x[(size_t)gr * ldx + k] : 0.f;
            }
            __syncthreads();
            if (vok) {
                const float* wr = w + (size_t)v * sh.K + k0;
                const int kn = min(64, sh.K - k0);
                for (int c = 0; c < kn; ++c) {
                    const float wv = wr[c];
#pragma unroll
                    for (int r = 0; r < 32; ++r) acc[r] = fmaf(wv, xs[r][c], acc[r]);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < 32; ++r) lt[r][tid] = acc[r];
        __syncthreads();
        float cm = neg_inf();
        int nv = 0;
        for (int j = 0; j < 32; ++j) {
            const int vv = ct * 32 + sub + 8 * j;
            if (vv < vend) {
                cm = fmaxf(cm, lt[srow][sub + 8 * j]);
                ++nv;
            }
        }
        if (nv > 0) {
            seen += nv;
            const float mn = fmaxf(m, cm);
            float sum = s * exp2f((m - mn) * sl2);
            for (int j = 0; j < 32; ++j) {
                const int vv = ct * 32 + sub + 8 * j;
                if (vv >= vend) continue;
                float cv = lt[srow][sub + 8 * j];
                sum += exp2f((cv - mn) * sl2);
                if (cv > lv[kLane - 1]) {
                    int ci = vv;
#pragma unroll
                    for (int q = 0; q < kLane; ++q) {
                        const bool sw = cv > lv[q];
                        const float tv = sw ? lv[q] : cv;
                        const int ti = sw ? li[q] : ci;
                        lv[q] = sw ? cv : lv[q];
                        li[q] = sw ? ci : li[q];
                        cv = tv;
                        ci = ti;
                    }
                }
            }
            s = sum;
            m = mn;
        }
    }
    __syncthreads();
    constexpr int W = 3 + 2 * kLane;
    float* cmrg = &lt[0][0];   // [32 rows][8 contributors][W]
    float* c = cmrg + (srow * 8 + sub) * W;
    c[0] = m;
    c[1] = s;
    c[2] = seen > kLane ? lv[kLane - 1] : neg_inf();
#pragma unroll
    for (int e = 0; e < kLane; ++e) {
        c[3 + e] = lv[e];
        c[3 + kLane + e] = __int_as_float(li[e]);
    }
    __syncthreads();
    lm_merge_contributors<8, kLane, kKeep, 8>(cmrg, 8 * W, 32, row0, split, sh.nchunks, sh.R, sl2, part);
}

// ------------------------------------------------------------------ merge

struct MergeArgs {
    const float* part;
    int nsplit;
    SliceMap map;
    int K, V, d;
    float inv_t, sl2;
    int32_t* out_idx;
    float* out_lp;
    float* out_lse;
    const void* x;   // activation rows (slow path)
    long ldx;
    const void* w;   // LM head (slow path)
    int* diag;
};

// Exact logits of one activation row with the 32 vocabulary rows of each of
// NTL tiles (ids 32t .. 32t+31; ids past V repeat row V-1), computed as the
// bf16 LM-head kernels compute them: one chain per logit, an MFMA 32x32x16
// per 16-wide k block in increasing k from zero, the weights as the A
// operand and the activation as B, so that every value is bit for bit the
// one the fast path saw (exact ties order the same way on both paths).  The
// row fills all 32 B columns, so every lane holds the logits of ids
// 32t + acc_row(j, lane) in acc[j].  Loads go in batches of P k blocks, two
// batches in flight: one lands while the other feeds the MFMAs (a batch
// reaching past d re-reads the last block and is not used).
template <int NTL, int P>
__device__ __forceinline__ void tile_logits_mfma(const uint16_t* xr, const uint16_t* w, int d, int V,
                                                 const int (&t)[NTL], f32x16 (&acc)[NTL]) {
    const int lane = threadIdx.x & 63;
    const int h8 = 8 * (lane >> 5);
    const uint16_t* wp[NTL];
#pragma unroll
    for (int i = 0; i < NTL; ++i) {
        wp[i] = w + (size_t)min(t[i] * 32 + (lane & 31), V - 1) * d + h8;
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[i][j] = 0.f;
    }
    const uint16_t* xp = xr + h8;
    const int nblk = d / 16;
    auto load = [&](int blk, u32x4 (&xv)[P], u32x4 (&wv)[NTL][P]) {
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int k0 = min(blk + p, nblk - 1) * 16;
            xv[p] = *reinterpret_cast<const u32x4*>(xp + k0);
#pragma unroll
            for (int i = 0; i < NTL; ++i) wv[i][p] = *reinterpret_cast<const u32x4*>(wp[i] + k0);
        }
    };
    auto mma = [&](int blk, const u32x4 (&xv)[P], const u32x4 (&wv)[NTL][P]) {
#pragma unroll
        for (int p = 0; p < P; ++p)
            if (blk + p < nblk)
#pragma unroll
                for (int i = 0; i < NTL; ++i) acc[i] = mfma_32x32x16_bf16(wv[i][p], xv[p], acc[i]);
    };
    u32x4 xa[P], wa[NTL][P], xb[P], wb[NTL][P];
    load(0, xa, wa);
    for (int blk = 0; blk < nblk; blk += 2 * P) {
        load(blk + P, xb, wb);
        mma(blk, xa, wa);
        if (blk + 2 * P < nblk) load(blk + 2 * P, xa, wa);
        mma(blk + P, xb, wb);
    }
}

// Logits of tiles [tg, tend) (at most 16) into colv[(t - tg) * 32 + m]: wave
// w takes tiles tg + w + 4i, i < NTL; a slot past tend repeats the last tile
// and is not read.
template <int NTL>
__device__ __forceinline__ void slice_logits(const uint16_t* xr, const uint16_t* w, int d, int V, int tg, int tend,
                                             float* colv) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int tl[NTL];
#pragma unroll
    for (int i = 0; i < NTL; ++i) tl[i] = min(tg + wave + 4 * i, tend - 1);
    f32x16 lg[NTL];
    tile_logits_mfma<NTL, (NTL >= 4 ? 2 : 3)>(xr, w, d, V, tl, lg);
    if ((lane & 31) == 0)
#pragma unroll
        for (int i = 0; i < NTL; ++i)
#pragma unroll
            for (int j = 0; j < 16; ++j) colv[(wave + 4 * i) * 32 + acc_row(j, lane)] = lg[i][j];
}

__device__ __forceinline__ float dot_row(const float* a, const float* b, int d) {
    float acc = 0.f;
    for (int k = 0; k < d; ++k) acc = fmaf(a[k], b[k], acc);
    return acc;
}

// Descending bitonic sort of one value per lane across a wave.
__device__ __forceinline__ float wave_sort_desc(float v, int lane) {
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            const float o = lane_xor_n(v, j);
            const bool keep_max = ((lane & j) == 0) == ((lane & k) == 0);
            v = keep_max ? fmaxf(v, o) : fminf(v, o);
        }
    return v;
}

// The best 64 of two wave lists sorted in opposite directions, sorted
// descending (DESC) or ascending: the larger of a[l] and b[l] per lane form a
// bitonic sequence holding them, and half-cleaners sort it.
template <bool DESC>
__device__ __forceinline__ float wave_merge(float a, float b, int lane) {
    float v = fmaxf(a, b);
#pragma unroll
    for (int j = 32; j > 0; j >>= 1) {
        const float o = lane_xor_n(v, j);
        v = ((lane & j) == 0) == DESC ? fmaxf(v, o) : fminf(v, o);
    }
    return v;
}

// Order-preserving unsigned image of a float: a larger float has a larger
// image, and -0 shares +0's (they compare equal).
__device__ __forceinline__ unsigned ord_bits(float v) {
    const unsigned b = v == 0.f ? 0u : __float_as_uint(v);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// ord_bits of the K-th largest of vals[0, n) (1 <= K <= n), found by a radix
// select over four 8-bit digits from the top: each pass counts, in LDS, the
// values that match the digits found so far by their next digit, and wave 0
// locates the digit holding the wanted rank.  Called by all 256 threads.
__device__ unsigned kth_largest_ord(const float* vals, int n, int K, int* hist, int* sel) {
    const int tid = threadIdx.x;
    unsigned prefix = 0, mask = 0;
    int need = K;   // rank wanted among the values that match the prefix
    for (int shift = 24; shift >= 0; shift -= 8) {
        hist[tid] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += 256) {
            const unsigned u = ord_bits(vals[i]);
            if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
        }
        __syncthreads();
        if (tid < 64) {
            // lane l holds digits 255 - 4l .. 252 - 4l, largest first
            int h[4], tot = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                h[q] = hist[255 - (4 * tid + q)];
                tot += h[q];
            }
            int incl = tot;
            for (int o = 1; o < 64; o <<= 1) {
                const int t = __shfl_up(incl, o);
                if (tid >= o) incl += t;
            }
            int acc = incl - tot;
            if (acc < need && need <= incl) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (acc < need && need <= acc + h[q]) {
                        sel[0] = 255 - (4 * tid + q);
                        sel[1] = need - acc;
                    }
                    acc += h[q];
                }
            }
        }
        __syncthreads();
        prefix |= (unsigned)sel[0] << shift;
        mask |= 255u << shift;
        need = sel[1];
        __syncthreads();   // sel and hist are rewritten by the next pass
    }
    return prefix;
}

// (value, id) pairs of a wave sorted in the (value desc, id asc) order, lane
// 0 first: a bitonic network (ids are distinct, so the order is total;
// padding pairs are equal and stay put).
__device__ __forceinline__ void wave_sort_pairs(float& v, int& i, int lane) {
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            const float ov = lane_xor_n(v, j);
            const int oi = lane_xor_n(i, j);
            const bool keep_better = ((lane & j) == 0) == ((lane & k) == 0);
            const bool ob = better_masks(ov, oi, v, i);
            if (keep_better == ob) {
                v = ov;
                i = oi;
            }
        }
}

// The best 64 of two pair lists sorted in opposite orders, in the (value
// desc, id asc) order (DESC) or its reverse: the better of a[l] and b[l] per
// lane form a bitonic sequence holding them, and half-cleaners sort it.
template <bool DESC>
__device__ __forceinline__ void wave_merge_pairs(float& v, int& i, float bv, int bi, int lane) {
    if (better_masks(bv, bi, v, i)) {
        v = bv;
        i = bi;
    }
#pragma unroll
    for (int j = 32; j > 0; j >>= 1) {
        const float ov = lane_xor_n(v, j);
        const int oi = lane_xor_n(i, j);
        const bool keep_better = ((lane & j) == 0) == DESC;
        const bool ob = better_masks(ov, oi, v, i);
        if (keep_better == ob) {
            v = ov;
            i = oi;
        }
    }
}

// candidate buffer: every slice entry fits (long lists: at most kMaxSplitsLong slices)
constexpr int kMergeCap = kMaxSplits * kKeep;
static_assert(kMaxSplitsLong * kKeepLong <= kMergeCap, "long-list slices fit the candidate buffer");

// One workgroup per row.
//  1. log-sum-exp of the row from the slices' (max, sum) pairs;
//  2. a lower bound t0 on the row's k-th best value: the k-th best of the
//     threads' heads (a thread's head is the best entry of its slices); k
//     threads, so k distinct slices, reach it, so at least k candidates are
//     >= it (k <= 64; otherwise t0 = -inf);
//  3. every slice entry >= t0 goes to LDS; when more than 2k qualify and
//     they would not fit the register sort, a radix select finds the exact
//     k-th largest of them and only those at or above it stay; the rest is
//     sorted (in registers when k <= 64 and at most 256 remain), and the
//     first k are the row's top-k among the candidates;
//  4. a slice whose bound (everything it dropped is <= bound) reaches the k-th
//     value is re-evaluated exactly from memory, so the result is the exact
//     top-k of the row for any data, ties included.
// SPT: slices per thread (nsplit <= 256 * SPT), so that a launch with few
// slices keeps no idle slice slots in its registers.
template <class T, int KEEP, int SPT>
__global__ __launch_bounds__(256) void merge_topk_kernel(MergeArgs a) {
    constexpr int PS = part_stride(KEEP);
    constexpr int NQ = PS / 4;   // 16-byte words of one partial
    static_assert(PS % 4 == 0, "partials are whole 16-byte words");
    __shared__ float s_max[4], s_sum[4];
    __shared__ float s_bound[4];
    __shared__ float s_heads[256];
    __shared__ int s_hist[256];
    __shared__ int s_sel[2];
    __shared__ int s_count, s_nflag, s_ncand;
    // candidate buffer: every entry of the launch's slices fits (the last
    // slot takes discarded stores); sized by SPT so that launches with few
    // slices keep more workgroups per CU
    constexpr int CAP = 256 * SPT * KEEP;
    static_assert(CAP >= kMaxTopk + 256 && CAP <= kMergeCap, "sorted head and slow-path scratch fit");
    __shared__ float cand_v[CAP + 1];
    __shared__ int cand_i[CAP + 1];
    __shared__ int s_flag[256 * SPT];
    __shared__ float s_colv[512];   // logits of a re-evaluated group of 16 tiles (bf16)

    const int row = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int K = a.K;
    const float* P = a.part + (size_t)row * a.nsplit * PS;

    // every slice's whole partial (max, sum, bound, count, values, ids), read
    // in one batch (the slices of a thread are tid, tid + 256, ...)
    static_assert(256 * SPT <= (KEEP == kKeep ? kMaxSplits : kMaxSplitsLong), "slices per thread");
    f32x4 rec[SPT][NQ];
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int s = tid + 256 * j;
        if (s < a.nsplit) {
#pragma unroll
            for (int w = 0; w < NQ; ++w) rec[j][w] = *reinterpret_cast<const f32x4*>(P + s * PS + 4 * w);
        } else {
            rec[j][0] = f32x4{neg_inf(), 0.f, neg_inf(), 0.f};   // count 0
#pragma unroll
            for (int w = 1; w < NQ; ++w) rec[j][w] = f32x4{neg_inf(), neg_inf(), neg_inf(), neg_inf()};
        }
    }
    auto field = [&](int j, int f) { return rec[j][f >> 2][f & 3]; };   // f a constant after unrolling
    if (tid == 0) {
        s_count = 0;
        s_nflag = 0;
    }
    float M = neg_inf(), head = neg_inf();
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        M = fmaxf(M, field(j, 0));
        if (__float_as_int(field(j, 3)) > 0) head = fmaxf(head, field(j, 4));
    }
    // lower bound on the k-th best value: the k-th best of the 256 thread
    // heads (each wave sorts its 64, wave 0 merges the four sorted lists)
    const float sorted = wave_sort_desc(head, lane);
    s_heads[tid] = sorted;
    M = wave_max(M);
    if (lane == 0) s_max[wave] = M;
    __syncthreads();
    M = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
    float S = 0.f;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const float ms = field(j, 0);
        if (ms != neg_inf()) S += field(j, 1) * exp2f((ms - M) * a.sl2);
    }
    S = wave_sum(S);
    if (lane == 0) s_sum[wave] = S;
    if (wave == 0) {
        // lists 0 and 1 into one descending list, 2 and 3 into an ascending
        // one (each second list read back to front), then those two
        float v = wave_merge<true>(sorted, s_heads[64 + 63 - lane], lane);
        const float v23 = wave_merge<false>(s_heads[128 + lane], s_heads[192 + 63 - lane], lane);
        v = wave_merge<true>(v, v23, lane);
        const float kth = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), (K <= 64 ? K : 64) - 1));
        if (lane == 0) s_bound[0] = K <= 64 ? kth : neg_inf();
    }
    __syncthreads();
    S = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
    const float logS = logf(S);
    const float t0 = s_bound[0];

    // every entry >= t0 to LDS (lists are sorted: an entry qualifies only if
    // the ones before it do), one slot reservation per thread; an entry past
    // its slice's count (whose slot may hold stale words) reads as NaN, which
    // never qualifies, and the stores of the entries that do not qualify go
    // to a dump slot, so the pass runs without branches
    int nq[SPT], ntot = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int n = __float_as_int(field(j, 3));
        int m = 0;
#pragma unroll
        for (int e = 0; e < KEEP; ++e) {
            const float v = e < n ? field(j, 4 + e) : __builtin_nanf("");
            m += v >= t0 ? 1 : 0;
        }
        nq[j] = m;
        ntot += m;
    }
    int pos = ntot > 0 ? atomicAdd(&s_count, ntot) : 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
#pragma unroll
        for (int e = 0; e < KEEP; ++e) {
            const bool q = e < nq[j];
            const int dst = q ? pos : CAP;
            cand_v[dst] = field(j, 4 + e);
            cand_i[dst] = __float_as_int(field(j, 4 + KEEP + e));
            pos += q ? 1 : 0;
        }
    __syncthreads();
    int c = s_count;
    if ((K > 64 || c > 256) && c > 2 * K) {
        // many candidates: keep those at or above the exact K-th largest
        // value (at least K of them; more only with ties)
        const unsigned tk = kth_largest_ord(cand_v, c, K, s_hist, s_sel);
        constexpr int CPT = CAP / 256;
        float rv[CPT];
        int ri[CPT];
#pragma unroll
        for (int m = 0; m < CPT; ++m) {
            const int i = tid + 256 * m;
            rv[m] = i < c ? cand_v[i] : neg_inf();
            ri[m] = i < c ? cand_i[i] : 0;
        }
        if (tid == 0) s_count = 0;
        __syncthreads();   // every candidate read before any is moved
#pragma unroll
        for (int m = 0; m < CPT; ++m) {
            const int i = tid + 256 * m;
            if (i < c && ord_bits(rv[m]) >= tk) {
                const int pos = atomicAdd(&s_count, 1);
                cand_v[pos] = rv[m];
                cand_i[pos] = ri[m];
            }
        }
        __syncthreads();
        c = s_count;
    }
    if (K <= 64 && c <= 256) {
        // each wave sorts 64 candidates in registers, wave 0 merges the four
        // lists: the best 64 land sorted at the front of the buffer
        const int e = 64 * wave + lane;
        float v = e < c ? cand_v[e] : neg_inf();
        int i = e < c ? cand_i[e] : 0x7fffffff;
        wave_sort_pairs(v, i, lane);
        cand_v[e] = v;
        cand_i[e] = i;
        __syncthreads();
        if (wave == 0) {
            // a wave whose 64 slots all lie past c holds padding only, which
            // no merge takes over a candidate: merge only the waves in use.
            // Lists 0 and 1 into one sorted list, 2 and 3 into a reversed
            // one (each second list read back to front), then those two.
            if (c > 128) {
                float v2 = cand_v[128 + lane];
                int i2 = cand_i[128 + lane];
                wave_merge_pairs<false>(v2, i2, cand_v[192 + 63 - lane], cand_i[192 + 63 - lane], lane);
                wave_merge_pairs<true>(v, i, cand_v[64 + 63 - lane], cand_i[64 + 63 - lane], lane);
                wave_merge_pairs<true>(v, i, v2, i2, lane);
            } else if (c > 64) {
                wave_merge_pairs<true>(v, i, cand_v[64 + 63 - lane], cand_i[64 + 63 - lane], lane);
            }
            cand_v[lane] = v;
            cand_i[lane] = i;
        }
        __syncthreads();
    } else {
    int pw = 1;
    while (pw < c) pw <<= 1;
    for (int i = c + tid; i < pw; i += 256) {
        cand_v[i] = neg_inf();
        cand_i[i] = 0x7fffffff;
    }
    __syncthreads();
    for (int size = 2; size <= pw; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < (pw >> 1); i += 256) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const bool up = (lo & size) == 0;
                const float vl = cand_v[lo], vh = cand_v[hi];
                const int il = cand_i[lo], ih = cand_i[hi];
                const bool sw = up ? better(vh, ih, vl, il) : better(vl, il, vh, ih);
                if (sw) {
                    cand_v[lo] = vh;
                    cand_i[lo] = ih;
                    cand_v[hi] = vl;
                    cand_i[hi] = il;
                }
            }
            __syncthreads();
        }
    }
    }
    int cnt = min(c, K);
    float* sel_v = cand_v;   // the best cnt entries, sorted
    int* sel_i = cand_i;

    const float tval = cnt == K ? sel_v[K - 1] : neg_inf();
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const float U = field(j, 2);
        if (U != neg_inf() && U >= tval) s_flag[atomicAdd(&s_nflag, 1)] = tid + 256 * j;
    }
    __syncthreads();

    // exact slow path for slices that may hide a qualifying logit
    const int nflag = s_nflag;
    if (nflag > 0) {
        float* buf_v = cand_v + CAP - 256;   // scratch past the sorted head (K <= kMaxTopk)
        int* buf_i = cand_i + CAP - 256;
        const T* xr = reinterpret_cast<const T*>(a.x) + (size_t)row * a.ldx;
        const T* wb = reinterpret_cast<const T*>(a.w);
        for (int f = 0; f < nflag; ++f) {
            const int s = s_flag[f];
            int t0s, t1s;
            slice_tiles(a.map, s, t0s, t1s);
            // groups of 16 tiles (every slice the plans make is one group)
            for (int tg = t0s; tg < t1s; tg += 16) {
                const int tend = min(t1s, tg + 16);
                const int v0 = tg * 32, v1 = min(a.V, tend * 32);
                if constexpr (sizeof(T) == 2) {
                    const int ntl = (tend - tg + 3) / 4;   // tiles per wave
                    if (ntl == 1)
                        slice_logits<1>(xr, wb, a.d, a.V, tg, tend, s_colv);
                    else if (ntl == 2)
                        slice_logits<2>(xr, wb, a.d, a.V, tg, tend, s_colv);
                    else if (ntl == 3)
                        slice_logits<3>(xr, wb, a.d, a.V, tg, tend, s_colv);
                    else
                        slice_logits<4>(xr, wb, a.d, a.V, tg, tend, s_colv);
                }
                for (int vb = v0; vb < v1; vb += 256) {
                    if (tid == 0) s_ncand = 0;
                    __syncthreads();
                    const int v = vb + tid;
                    if (v < v1) {
                        float val;
                        if constexpr (sizeof(T) == 2)   // compared as the fast path's lists are
                            val = logit_trunc(s_colv[v - v0]);
                        else   // the fp32 kernel's chain: fmaf over k in increasing order
                            val = dot_row(xr, wb + (size_t)v * a.d, a.d);
                        bool take = cnt < K || better(val, v, sel_v[K - 1], sel_i[K - 1]);
                        if (take)
                            for (int j = 0; j < cnt; ++j)
                                if (sel_i[j] == v) {
                                    take = false;
                                    break;
                                }
                        if (take) {
                            const int p = atomicAdd(&s_ncand, 1);
                            buf_v[p] = val;
                            buf_i[p] = v;
                        }
                    }
                    __syncthreads();
                    if (tid == 0) {
                        int cc = cnt;
                        for (int q = 0; q < s_ncand; ++q) {
                            const float cv = buf_v[q];
                            const int ci = buf_i[q];
                            int pos;
                            if (cc < K) {
                                pos = cc++;
                            } else if (better(cv, ci, sel_v[K - 1], sel_i[K - 1])) {
                                pos = K - 1;
                            } else {
                                continue;
                            }
                            while (pos > 0 && better(cv, ci, sel_v[pos - 1], sel_i[pos - 1])) {
                                sel_v[pos] = sel_v[pos - 1];
                                sel_i[pos] = sel_i[pos - 1];
                                --pos;
                            }
                            sel_v[pos] = cv;
                            sel_i[pos] = ci;
                        }
                        s_count = cc;
                    }
                    __syncthreads();
                    cnt = s_count;
                }
            }
        }
        if (tid == 0 && a.diag != nullptr) atomicAdd(a.diag, nflag);
    }

    for (int j = tid; j < K; j += 256) {
        const bool ok = j < cnt;
        a.out_idx[(size_t)row * K + j] = ok ? sel_i[j] : -1;
        if (a.out_lp != nullptr)
            a.out_lp[(size_t)row * K + j] = ok ? a.inv_t * (sel_v[j] - M) - logS : neg_inf();
    }
    if (a.out_lse != nullptr && tid == 0) a.out_lse[row] = a.inv_t * M + logS;
}

// ------------------------------------------------------------------ launchers

template <bool LONG, int WM, int NT, int NW, int PIPE, bool WNT>
static void launch_lm_bf16(const uint16_t* x, long ldx, const uint16_t* w, const GemmShape& sh, const SliceMap& map,
                           int blocks, int V, float sl2, float* part, int* diag, hipStream_t st) {
    hipLaunchKernelGGL((lmhead_bf16_kernel<WM, NT, NW, PIPE, WNT, LONG>), dim3(blocks), dim3(64 * NW), 0, st, x, ldx,
                       w, sh, map, V, sl2, part, diag);
}

template <bool LONG, int WM, int NT, int NW, int KC, bool WNT, int MINB = 1, int WB = 1>
static hipError_t launch_lm_dma(const uint16_t* x, long ldx, const uint16_t* w, const GemmShape& sh,
                                const SliceMap& map, int blocks, int V, float sl2, float* part, int* diag,
                                hipStream_t st) {
    using T = DmaTraits<WM, NT, NW, KC, TF_LM_DMA_STAGES, WB>;
    auto kern = lmhead_dma_kernel<WM, NT, NW, KC, TF_LM_DMA_STAGES, WNT, MINB, LONG, WB>;
    // dynamic LDS beyond the 64 KiB default
    const hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, T::RING);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * NW), T::RING, st, x, ldx, w, sh, map, V, sl2, part, diag);
    return hipSuccess;
}

// tile shape and pipeline variants the plans can ask for
template <bool LONG>
static hipError_t dispatch_lm_bf16(const LmPlan& p, const uint16_t* x, long ldx, const uint16_t* w,
                                   const GemmShape& sh, int V, float sl2, float* part, int* diag, hipStream_t st) {
    const int nb = p.blocks();
    if (p.dma) {   // the shapes the plans use (see lm_plan)
        if (p.NT == 1)
            return launch_lm_dma<LONG, TF_LM_DMA_NT1_WM, 1, TF_LM_DMA_NT1_NW, TF_LM_DMA_KC, true>(x, ldx, w, sh, p.map, nb,
                                                                                            V, sl2, part, diag, st);
        if (p.grid && p.NT == 2)   // 33..64 rows: one activation tile per wave of the grid
            return launch_lm_dma<LONG, TF_LM_DMA_WM, 2, TF_LM_DMA_NW_SINGLE, TF_LM_DMA_KC, true, 1, TF_LM_DMA_SINGLE_WB>(
                x, ldx, w, sh, p.map, nb, V, sl2, part, diag, st);
        if (p.grid && p.wnt)   // a single row block
            return launch_lm_dma<LONG, TF_LM_DMA_WM, 4, TF_LM_DMA_NW_SINGLE, TF_LM_DMA_KC, true, 1, TF_LM_DMA_SINGLE_WB>(
                x, ldx, w, sh, p.map, nb, V, sl2, part, diag, st);
        if (p.grid)   // a few row blocks sharing each range's weights through L2
            return launch_lm_dma<LONG, TF_LM_DMA_WM, 4, TF_LM_DMA_NW_SINGLE, TF_LM_DMA_KC, false, 1, TF_LM_DMA_SINGLE_WB>(
                x, ldx, w, sh, p.map, nb, V, sl2, part, diag, st);
        // several row blocks: 256-row blocks (lm_plan)
        return launch_lm_dma<LONG, TF_LM_DMA_MULTI_WM, 8, 8, TF_LM_DMA_KC, false, 1, 2>(x, ldx, w, sh, p.map, nb, V,
                                                                                    sl2, part, diag, st);
    }
    if (p.NT == 1)
        launch_lm_bf16<LONG, TF_LM_WM_NT1, 1, TF_LM_NW_NT1, TF_PIPE_DEFAULT, true>(x, ldx, w, sh, p.map, nb, V, sl2, part,
                                                                           diag, st);
    else if (p.NT == 2)
        launch_lm_bf16<LONG, TF_LM_WM_NT2, 2, TF_LM_NW_NT2, TF_PIPE_DEFAULT, true>(x, ldx, w, sh, p.map, nb, V, sl2, part,
                                                                           diag, st);
    else if (p.wnt)
        launch_lm_bf16<LONG, TF_LM_WM_NT4, 4, TF_LM_NW_NT4, TF_PIPE_SINGLE_NT4, true>(x, ldx, w, sh, p.map, nb, V, sl2,
                                                                              part, diag, st);
    else
        launch_lm_bf16<LONG, TF_LM_WM_NT4, 4, TF_LM_NW_NT4, TF_PIPE_DEFAULT, false>(x, ldx, w, sh, p.map, nb, V, sl2, part,
                                                                            diag, st);
    return hipSuccess;
}

hipError_t launch_lmhead_topk(const void* x, long ldx, const void* w, int rows, int d, int V, int K,
                              float inv_t, bool bf16, unsigned char* lm_ws, int32_t* out_idx, float* out_lp,
                              float* out_lse, int* diag, hipStream_t stream, hipEvent_t ev_begin,
                              hipEvent_t ev_end) {
    const LmPlan p = lm_plan(rows, V, d, bf16);
    if (p.nsplit() > kMaxSplits) return hipErrorInvalidValue;
    float* part = reinterpret_cast<float*>(lm_ws);
    // the LM kernels read R, K, ntiles, nrb and nk; G counts workgroups
    const GemmShape sh{rows, d, p.ntiles, p.map.G, p.nrb, p.nk, p.blocks()};
    const float sl2 = inv_t * kLog2e;
    if (ev_begin != nullptr && hipEventRecord(ev_begin, stream) != hipSuccess) return hipErrorInvalidHandle;
    const bool longl = lm_long_lists(p, bf16, K);
    if (bf16) {
        const hipError_t de =
            longl ? dispatch_lm_bf16<true>(p, static_cast<const uint16_t*>(x), ldx, static_cast<const uint16_t*>(w),
                                           sh, V, sl2, part, diag, stream)
                  : dispatch_lm_bf16<false>(p, static_cast<const uint16_t*>(x), ldx, static_cast<const uint16_t*>(w),
                                            sh, V, sl2, part, diag, stream);
        if (de != hipSuccess) return de;
    } else
        hipLaunchKernelGGL(lmhead_f32_kernel, dim3(p.blocks()), dim3(256), 0, stream, static_cast<const float*>(x),
                           ldx, static_cast<const float*>(w), sh, p.map, V, sl2, part, diag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ev_end != nullptr && hipEventRecord(ev_end, stream) != hipSuccess) return hipErrorInvalidHandle;
    MergeArgs ma{part, p.nsplit(), p.map, K, V, d, inv_t, sl2, out_idx, out_lp, out_lse, x, ldx, w, diag};
    // slices per thread: two, four or the most a launch may have
    const int ns = p.nsplit();
    if (bf16 && longl) {
        if (ns <= 512)
            hipLaunchKernelGGL((merge_topk_kernel<uint16_t, kKeepLong, 2>), dim3(rows), dim3(256), 0, stream, ma);
        else
            hipLaunchKernelGGL((merge_topk_kernel<uint16_t, kKeepLong, kMaxSplitsLong / 256>), dim3(rows), dim3(256),
                               0, stream, ma);
    } else if (bf16) {
        if (ns <= 512)
            hipLaunchKernelGGL((merge_topk_kernel<uint16_t, kKeep, 2>), dim3(rows), dim3(256), 0, stream, ma);
        else if (ns <= 1024)
            hipLaunchKernelGGL((merge_topk_kernel<uint16_t, kKeep, 4>), dim3(rows), dim3(256), 0, stream, ma);
        else
            hipLaunchKernelGGL((merge_topk_kernel<uint16_t, kKeep, kMaxSplits / 256>), dim3(rows), dim3(256), 0,
                               stream, ma);
    } else {
        hipLaunchKernelGGL((merge_topk_kernel<float, kKeep, kMaxSplits / 256>), dim3(rows), dim3(256), 0, stream, ma);
    }
    return hipGetLastError();
}

}  // namespace tf

// Weight-streaming GEMM for gfx950: Y[r, n] = sum_k X[r, k] * W[n, k].
//
// Every product on the drafting path has this shape: a large weight matrix
// (LM head [V, d], SwiGLU gate/up [I, 2d], down [d, I]) streamed once from HBM
// against a small set of activation rows (b*gamma or b*R rows).  The weight
// side is the MFMA "A" operand (32 weight rows per tile), the activation rows
// the "B" operand (32 rows per N-tile).  Each lane of a 32x32 accumulator then
// owns one activation row (lane % 32) and 16 weight rows, so per-row
// reductions over the vocabulary (max, sum-exp, running top-k) stay inside a
// lane.
//
// Work decomposition (see work.hpp): a workgroup of NW waves streams chunks
// of NW*WM weight tiles (WM per wave) against blocks of 32*NT activation rows.
// The LM head cuts the vocabulary into equal tile ranges, one per workgroup,
// streamed in rounds; the small SwiGLU products cut their k-range instead.
// Per 64-wide k-chunk the activation tile [32*NT x 64] is staged in LDS
// (double buffered, rows padded to 144 B so the 16-byte fragment reads are
// bank-conflict free) and shared by all NW*WM weight tiles of the workgroup.
// Each wave streams its own weight rows with fully coalesced loads -- one
// instruction covers 8 rows x 128 B, i.e. whole cache lines -- several
// k-chunks ahead of the MFMAs, and transposes them into fragment order
// through a wave-private LDS tile whose 16-byte slots are XOR-swizzled by
// row (see wswz), so both the writes and the fragment reads are conflict
// free.  (Loading fragments directly -- 32 rows x 32 B per instruction --
// measured ~17% less HBM bandwidth on MI355X.)
//
// What bounds these kernels on MI355X is the vector-memory path of each CU:
// weight bytes (from HBM) plus activation bytes (re-read from L2 once per
// round of a workgroup) together top out near 6.5-7 TB/s, the rate of a
// plain streaming read.  The activation share therefore shrinks with more
// weight tiles per round (more accumulators per CU).
#pragma once

#include "common.hpp"
#include "rows.hpp"
#include "work.hpp"

namespace tf {

// One contiguous k-range of one item, computed by one workgroup.
struct Segment {
    int g;         // workgroup (logical id)
    int item, chunk, rb;
    int t0, t1;    // weight tiles [t0, t1)
    int kc0, kc1;  // 64-wide k-chunks [kc0, kc1)
    int row0;      // first activation row
    int gfirst;    // first workgroup holding a piece of the item
    int npieces;   // workgroups holding a piece of the item
};

// Workgroups are dispatched round-robin over the 8 XCDs of an MI355X.
// Renumber them so consecutive logical ids share an XCD (and its L2): the
// row blocks of one weight chunk, and the pieces of a cut item, then meet in
// the same L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    if ((nblocks & 7) != 0) return bid;
    return (bid & 7) * (nblocks >> 3) + (bid >> 3);
}


template <int WM, int NT, int NW>
struct GemmTraits {
    static constexpr int TR = 32 * NT;           // activation rows per workgroup
    static constexpr int KC = 64;                // k per LDS stage
    static constexpr int LDSW = KC + 8;          // padded LDS row (144 B), bf16 elements
    static constexpr int XS_BYTES = 2 * TR * LDSW * 2;
    static constexpr int WROWS = 32 * WM;        // weight rows per wave
    static constexpr int WS_BYTES = NW * WROWS * KC * 2;   // wave-private weight tiles
    static constexpr int SMEM_BYTES = XS_BYTES + WS_BYTES;
    static constexpr int NWL = WROWS / 8;        // coalesced weight loads per wave per k-chunk
    static constexpr int CHUNK = NW * WM;        // weight tiles per chunk
    static constexpr int NTHREADS = 64 * NW;
    static constexpr int XPIECES = TR * 8;       // 16-byte pieces of an activation tile
    static constexpr int XPT = (XPIECES + NTHREADS - 1) / NTHREADS;
    static constexpr int PART_FLOATS = NW * WM * NT * 16 * 64;   // one workgroup's accumulators
};

// The segment of workgroup g that starts at unit u (u < end of g's range).
template <int WM, int NT, int NW>
__device__ __forceinline__ Segment make_segment(const GemmShape& sh, int g, long long u, long long u_end) {
    using T = GemmTraits<WM, NT, NW>;
    Segment s;
    s.g = g;
    s.item = (int)(u / sh.nk);
    s.chunk = s.item / sh.nrb;
    s.rb = s.item - s.chunk * sh.nrb;
    const long long ib = (long long)s.item * sh.nk;
    s.kc0 = (int)(u - ib);
    s.kc1 = (int)((u_end - ib) < sh.nk ? (u_end - ib) : sh.nk);
    s.t0 = s.chunk * T::CHUNK;
    s.t1 = min(s.t0 + T::CHUNK, sh.ntiles);
    s.row0 = s.rb * T::TR;
    s.gfirst = unit_owner(sh, ib);
    s.npieces = unit_owner(sh, ib + sh.nk - 1) - s.gfirst + 1;
    return s;
}

__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// XOR swizzle of the 16-byte slots of a 128-byte weight row in LDS.  gfx950
// serves a 16-lane quarter of a 128-bit LDS access from 64 four-byte banks,
// i.e. two 128-byte rows per cycle: consecutive rows sit in opposite bank
// halves and (row / 2) % 8 spreads the 8 rows of each half over all slots.
// Fragment reads (16 consecutive rows, one logical slot) and the coalesced
// writes (2 rows x 8 slots per quarter) are then both conflict free.
__device__ __forceinline__ int wswz(int row) { return (row >> 1) & 7; }

// Workgroup barrier for LDS traffic only.  __syncthreads() also waits for
// every outstanding global load (its release fence), which would drain the
// weight prefetch at each k-chunk; here only this wave's LDS operations are
// waited for before the barrier.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Accumulate one segment: acc[mt][nt] = X[rows of nt] . W[tiles of mt] over
// the segment's 64-wide k-chunks.  PIPE: k-chunks of loads in flight per
// wave.  WNT: weight loads carry the non-temporal hint, for weights that one
// workgroup alone reads (a single activation row block), so they do not
// evict the activations that every workgroup re-reads from L2.
template <int WM, int NT, int NW, int PIPE, bool WNT, class WSrc, class XSrc>
__device__ __forceinline__ void gemm_segment(const WSrc& wsrc, const XSrc& xsrc, const GemmShape& sh,
                                             const Segment& it, f32x16 (&acc)[WM][NT], unsigned char* smem) {
    using T = GemmTraits<WM, NT, NW>;
    constexpr int TR = T::TR, KC = T::KC, LDSW = T::LDSW, NWL = T::NWL, NTH = T::NTHREADS, XPT = T::XPT;
    uint16_t* xs = reinterpret_cast<uint16_t*>(smem);   // [2 buffers][TR][LDSW]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // this wave's weight tile: [WROWS][KC]
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem + T::XS_BYTES) + wave * T::WROWS * KC;
    const int nk = it.kc1 - it.kc0;
    const int slot = lane & 7;          // 16-byte slot of a 128-byte row segment this lane loads
    // wave-uniform: does this wave own a weight tile of the segment?  Idle
    // waves (a segment narrower than the workgroup) still stage activations
    // and meet the barriers, but load no weights and issue no MFMAs.
    const bool wact = it.t0 + wave * WM < it.t1;

    // Coalesced weight loads: instruction q covers wave rows 8q..8q+7.  Every
    // load is unconditional and in bounds: rows past the matrix read its first
    // row (their outputs are discarded by the epilogue) and k past K is
    // clamped; the activation side is zeroed there, so those products vanish.
    // Conditional "load or zero" would make the compiler wait for all loads
    // in flight before re-zeroing a register.
    const uint16_t* gw[NWL];
#pragma unroll
    for (int q = 0; q < NWL; ++q) {
        const int row = 8 * q + (lane >> 3);
        const int tile = it.t0 + wave * WM + (row >> 5);
        const uint16_t* p = (tile < it.t1) ? wsrc.row(tile, row & 31) : nullptr;
        gw[q] = p != nullptr ? p : wsrc.row(0, 0);
    }
#pragma unroll
    for (int mt = 0; mt < WM; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[mt][nt][j] = 0.f;

    // activation rows of this thread's 16-byte pieces (clamped into [0, R))
    const int kmax = sh.K - 8;
    // activation pieces p = tid + NTH*i: row p / 8, 16-byte slot p % 8
    constexpr bool XFULL = T::XPIECES % NTH == 0;
    auto load_x = [&](u32x4 (&xr)[XPT], int kc) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            const int p = tid + NTH * i;
            if (XFULL || p < T::XPIECES) {
                const int gr = min(it.row0 + (p >> 3), sh.R - 1);
                const int k = min(kc * KC + (p & 7) * 8, kmax);
                xr[i] = *reinterpret_cast<const u32x4*>(xsrc.ptr(gr, k));
            }
        }
    };
    // chunk kc into activation buffer `buf`; zero outside the matrix
    auto store_x = [&](const u32x4 (&xr)[XPT], int buf, int kc) {
        uint16_t* dst = xs + buf * TR * LDSW;
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            const int p = tid + NTH * i;
            if (XFULL || p < T::XPIECES) {
                const bool ok = it.row0 + (p >> 3) < sh.R && kc * KC + (p & 7) * 8 < sh.K;
                *reinterpret_cast<u32x4*>(dst + (p >> 3) * LDSW + (p & 7) * 8) =
                    ok ? xr[i] : u32x4{0u, 0u, 0u, 0u};
            }
        }
    };
    auto load_w = [&](u32x4 (&w)[NWL], int kc) {
        if (!wact) return;
        const int k = min(kc * KC + slot * 8, kmax);
#pragma unroll
        for (int q = 0; q < NWL; ++q) {
            const u32x4* src = reinterpret_cast<const u32x4*>(gw[q] + wsrc.kcol(k));
            if constexpr (WNT)
                w[q] = __builtin_nontemporal_load(src);
            else
                w[q] = *src;
        }
    };
    auto store_w = [&](const u32x4 (&w)[NWL]) {
        if (!wact) return;
#pragma unroll
        for (int q = 0; q < NWL; ++q) {
            const int row = 8 * q + (lane >> 3);
            *reinterpret_cast<u32x4*>(wl + row * KC + ((slot ^ wswz(row)) * 8)) = w[q];
        }
    };

    // Software pipeline of depth PIPE: the loads of k-chunk j are issued at
    // the start of step j-PIPE+1 (their register set held chunk j-PIPE+1,
    // already in LDS), so they run under that step's MFMAs, and are stored
    // to LDS at the end of step j-1.  Within a step the stores wait only for
    // the loads of the chunk they store (loads return in order), leaving the
    // later chunks in flight.
    static_assert(PIPE >= 2 && PIPE <= 4, "pipeline depth");
    u32x4 xr[PIPE][XPT];
    u32x4 wr[PIPE][NWL];
    auto load_step = [&](int r, int i) {
        load_x(xr[r], it.kc0 + i);
        load_w(wr[r], it.kc0 + i);
    };
    // MFMAs of k-chunk i from LDS (activation buffer i & 1, the wave's weight tile)
    auto compute = [&](int i) {
        if (!wact) return;
        const uint16_t* xb = xs + (i & 1) * TR * LDSW;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            u32x4 afr[WM], bfr[NT];
#pragma unroll
            for (int mt = 0; mt < WM; ++mt) {
                const int row = mt * 32 + (lane & 31);
                const int ls = 2 * ks + (lane >> 5);
                afr[mt] = *reinterpret_cast<const u32x4*>(wl + row * KC + ((ls ^ wswz(row)) * 8));
            }
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                bfr[nt] = *reinterpret_cast<const u32x4*>(
                    xb + (nt * 32 + (lane & 31)) * LDSW + (2 * ks + (lane >> 5)) * 8);
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[mt][nt] = mfma_32x32x16_bf16(afr[mt], bfr[nt], acc[mt][nt]);
        }
    };
    // store register set r (k-chunk i) into LDS after this wave's reads of the
    // previous chunk (LDS operations of a wave complete in order)
    auto stage = [&](int r, int i) {
        compiler_fence();
        store_w(wr[r]);
        store_x(xr[r], i & 1, it.kc0 + i);
        compiler_fence();
    };
    const int nsteps = nk;
    if (nsteps > 0) {
#pragma unroll
        for (int j = 0; j < PIPE; ++j)
            if (j < nsteps) load_step(j, j);
        stage(0, 0);
        int i0 = 0;
        // steady state, branch free: every step refills the register set it
        // freed, computes, and stages the next chunk
        for (; i0 + 2 * PIPE <= nsteps; i0 += PIPE) {
#pragma unroll
            for (int u = 0; u < PIPE; ++u) {
                const int i = i0 + u;
                // register set u held step i, already in LDS: refill it first,
                // so the loads run under this step's MFMAs
                load_step(u, i + PIPE);
                lds_barrier();  // step i visible; the other activation buffer is free
                compute(i);
                stage((u + 1) % PIPE, i + 1);
            }
        }
        // tail: fewer than 2*PIPE steps left
#pragma unroll
        for (int u = 0; u < 2 * PIPE; ++u) {
            const int i = i0 + u;
            if (i < nsteps) {
                if (i + PIPE < nsteps) load_step(u % PIPE, i + PIPE);
                lds_barrier();
                compute(i);
                if (i + 1 < nsteps) stage((u + 1) % PIPE, i + 1);
            }
        }
    }
}

// Every segment of this workgroup: accumulate, then hand the accumulators to
// the epilogue (which may reuse the LDS tiles).
template <int WM, int NT, int NW, int PIPE, bool WNT, class WSrc, class XSrc, class Epi>
__device__ __forceinline__ void stream_gemm(const WSrc& wsrc, const XSrc& xsrc, Epi& epi, const GemmShape& sh,
                                            unsigned char* smem) {
    const int g = xcd_logical_id(blockIdx.x, gridDim.x);
    const long long u_end = unit_start(sh, g + 1);
    long long u = unit_start(sh, g);
    while (u < u_end) {
        const Segment seg = make_segment<WM, NT, NW>(sh, g, u, u_end);
        f32x16 acc[WM][NT];
        gemm_segment<WM, NT, NW, PIPE, WNT>(wsrc, xsrc, sh, seg, acc, smem);
        __syncthreads();  // LDS tiles no longer needed
        epi.apply(acc, seg, smem, sh);
        u = (long long)(seg.item + 1) * sh.nk;
        if (u < u_end) lds_barrier();  // the epilogue's LDS use ends before the next tiles land
    }
}

// ----------------------------------------------------------- weight sources

// Plain [N, K] weight matrix, one weight row per tile row.
struct WRowsPlain {
    const uint16_t* w;
    int N, K;
    __device__ __forceinline__ const uint16_t* row(int tile, int r) const {
        const int n = tile * 32 + r;
        return n < N ? w + (size_t)n * K : nullptr;
    }
    __device__ __forceinline__ int kcol(int k) const { return k; }
};

// Weight rows [N, K] read against an activation stored as bf16 hi/lo pairs
// interleaved by 8 (activation column k' holds the hi part of element
// (k'/16)*8 + k'%8 when (k'/8) is even, the lo part when odd): reduction
// column k' reads weight column kcol(k').  The two lanes that load the hi
// and lo columns of the same 8 weights read the same 16 bytes, so the weight
// bytes fetched do not change.
struct WRowsPairedK {
    const uint16_t* w;
    int N, K;   // K: weight columns (half the activation width)
    __device__ __forceinline__ const uint16_t* row(int tile, int r) const {
        const int n = tile * 32 + r;
        return n < N ? w + (size_t)n * K : nullptr;
    }
    __device__ __forceinline__ int kcol(int k) const { return ((k >> 4) << 3) | (k & 7); }
};

// SwiGLU input projections: tile rows 0..15 are gate rows 16*tile.., tile
// rows 16..31 the up rows with the same indices, so lane j of the accumulator
// holds a gate value in register j and the matching up value in register j+8.
struct WRowsGateUp {
    const uint16_t* gate;
    const uint16_t* up;
    int I, K;
    __device__ __forceinline__ const uint16_t* row(int tile, int r) const {
        const int i = tile * 16 + (r & 15);
        if (i >= I) return nullptr;
        return (r < 16 ? gate : up) + (size_t)i * K;
    }
    __device__ __forceinline__ int kcol(int k) const { return k; }
};

// -------------------------------------------------------- activation sources

struct XRowsPlain {
    const uint16_t* x;
    long ld;
    __device__ __forceinline__ const uint16_t* ptr(int r, int k) const { return x + (size_t)r * ld + k; }
};

// Input of the SwiGLU (or linear layer): row r is [ h~(depth of r) ; e~(r) ]
// (Eq. 1), where e~(r) holds the normalised embeddings of the row's previous
// token(s): ew = d for one token, 2d for the bigram of the w/ 2-prev rows.
struct XRowsConcat {
    const uint16_t* ht;   // [b*gamma, d] normalised drafter states
    const uint16_t* et;   // [b*R, ew] normalised embeddings of the previous tokens
    int d, ew;
    RowTable t;
    __device__ __forceinline__ const uint16_t* ptr(int r, int k) const {
        if (k >= d) return et + (size_t)r * ew + (k - d);
        const int s = r / t.Rs;
        const int rl = r - s * t.Rs;
        return ht + (size_t)(s * t.gamma + t.depth(rl) - 1) * d + k;
    }
};

// ------------------------------------------------------------------ epilogues

// Merge the NC contributor lists of each activation row (written to `cm` as
// [rows][NC][3 + 2*KL] = max, sum, bound, KL values, KL ids; `bound` is at
// least every value the contributor saw but did not list) into the row's
// (row, slice) partial of KEEP entries.  T consecutive lanes per row, each
// taking NC / T contributors: a lane picks the KEEP + 1 best of its own
// entries by (value desc, id asc), then the row's picks are the heads' best,
// found by maxima and minima across the T lanes (DPP), the winning lane
// moving to its next entry.  The (KEEP + 1)-th pick bounds every entry a lane
// left out (that lane still holds an unpicked entry at least as large), so
// it and the contributors' bounds bound the slice's unlisted logits.
template <int NC, int KL, int KEEP = kKeep, int T = 1>
__device__ __forceinline__ void lm_merge_contributors(const float* cm, int rstride, int rows, int row0, int split,
                                                      int nsplit, int R, float sl2, float* part) {
    static_assert(NC % T == 0 && (T == 1 || T == 2 || T == 4 || T == 8), "lanes per row");
    constexpr int W = 3 + 2 * KL;
    constexpr int NCT = NC / T;          // contributors of one lane
    constexpr int NCAND = NCT * KL;
    constexpr int NL = KEEP + 1;         // a lane's picks: KEEP to list, one to bound the rest
    const int r = threadIdx.x / T, t = threadIdx.x % T;
    if (r >= rows) return;               // whole groups of T lanes leave together
    const int grow = row0 + r;
    if (grow >= R) return;
    // this lane's contributors' words at once (one batch of LDS reads)
    const float* c = cm + r * rstride + t * NCT * W;
    float cmax[NCT], csum[NCT], cbnd[NCT], v[NCAND];
    int id[NCAND];
#pragma unroll
    for (int p = 0; p < NCT; ++p) {
        cmax[p] = c[p * W + 0];
        csum[p] = c[p * W + 1];
        cbnd[p] = c[p * W + 2];
#pragma unroll
        for (int q = 0; q < KL; ++q) {
            v[p * KL + q] = c[p * W + 3 + q];
            id[p * KL + q] = __float_as_int(c[p * W + 3 + KL + q]);
        }
    }
    float M = neg_inf(), U = neg_inf();
#pragma unroll
    for (int p = 0; p < NCT; ++p) {
        M = fmaxf(M, cmax[p]);
        U = fmaxf(U, cbnd[p]);
    }
#pragma unroll
    for (int o = 1; o < T; o <<= 1) {
        M = fmaxf(M, lane_xor_n(M, o));
        U = fmaxf(U, lane_xor_n(U, o));
    }
    float S = 0.f;
#pragma unroll
    for (int p = 0; p < NCT; ++p) S += (cmax[p] == neg_inf()) ? 0.f : csum[p] * exp2f((cmax[p] - M) * sl2);
#pragma unroll
    for (int o = 1; o < T; o <<= 1) S += lane_xor_n(S, o);
    // this lane's picks, in order: the largest value, then the smallest id
    // holding it (an empty or picked entry holds -inf, and listed logits are
    // finite), by maxima, minima and selects alone
    float lv[NL];
    int li[NL];
#pragma unroll
    for (int e = 0; e < NL; ++e) {
        float bv = neg_inf();
#pragma unroll
        for (int j = 0; j < NCAND; ++j) bv = fmaxf(bv, v[j]);
        int bi = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < NCAND; ++j) bi = min(bi, v[j] == bv ? id[j] : 0x7fffffff);
        lv[e] = bv;
        li[e] = bi;
        if (e + 1 < NL) {
#pragma unroll
            for (int j = 0; j < NCAND; ++j) v[j] = id[j] == bi ? neg_inf() : v[j];
        }
    }
    float* out = part + ((size_t)grow * nsplit + split) * part_stride(KEEP);
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < NL; ++e) {
        float bv = lv[0];
        int bi = li[0];
        if constexpr (T > 1) {
#pragma unroll
            for (int o = 1; o < T; o <<= 1) bv = fmaxf(bv, lane_xor_n(bv, o));
            bi = lv[0] == bv ? li[0] : 0x7fffffff;
#pragma unroll
            for (int o = 1; o < T; o <<= 1) bi = min(bi, lane_xor_n(bi, o));
            if (e + 1 < NL) {
                // the winning lane moves to its next pick (ids are distinct in a slice)
                const bool mine = lv[0] == bv && li[0] == bi;
#pragma unroll
                for (int q = 0; q + 1 < NL; ++q) {
                    lv[q] = mine ? lv[q + 1] : lv[q];
                    li[q] = mine ? li[q + 1] : li[q];
                }
                lv[NL - 1] = mine ? neg_inf() : lv[NL - 1];
            }
        } else if (e + 1 < NL) {
#pragma unroll
            for (int q = 0; q + 1 < NL; ++q) {
                lv[q] = lv[q + 1];
                li[q] = li[q + 1];
            }
        }
        const bool any = bv != neg_inf();
        if (e < KEEP) {
            // the e-th entry, or the empty entry once the lists are exhausted
            if (t == 0) {
                out[4 + e] = bv;
                out[4 + KEEP + e] = __int_as_float(any ? bi : -1);
            }
            cnt += any ? 1 : 0;
        } else if (any) {
            U = fmaxf(U, bv);   // the best entry left out bounds the slice's other logits
        }
    }
    if (t == 0) {
        out[0] = M;
        out[1] = S;
        out[2] = U;
        out[3] = __int_as_float(cnt);
    }
}

// LM head: per lane and row, the maximum, the sum of exponentials, the KL
// best logits with their token ids and a bound on the rest (the largest logit
// the lane drops); merged per workgroup into a (row, slice) partial of KEEP
// entries, the slice being the workgroup's chunk of the vocabulary (LONG:
// the long lists for large top-k).  WB > 1: the waves form a grid of
// NW / WB waves along the weight tiles times WB along the activation tiles,
// each wave holding NT / WB activation tiles, so a row has 2 * NW / WB
// contributor lists.
//
// The partial's `bound` is an upper bound on every logit of the slice that is
// not in its list: a lane drops only values no larger than its bound, and the
// workgroup merge drops only values no larger than the (kKeep+1)-th entry of
// the union.  The merge kernel uses it to prove the global top-k exact, or to
// re-evaluate the slice when it cannot.  Short lists (two or three entries
// per lane, by how many logits of a row a lane holds) keep this pass cheap
// (it runs on the vector ALUs after every item); a slice is re-evaluated
// only if one lane holds KL + 1 of the row's best k logits or the slice
// KEEP + 1 of them.
template <int WM, int NT, int NW, bool LONG = false, int WB = 1>
struct EpiLmHead {
    static constexpr int WA = NW / WB;            // waves along the weight tiles
    static constexpr int NTW = NT / WB;           // activation tiles per wave
    float* part;     // [R, nchunks, part_stride(KEEP)]
    int V;
    float sl2;       // inv_temperature * log2(e)
    static constexpr bool WIDE = WM * 16 > 64;
    static constexpr int KL = LONG ? (WIDE ? kLaneMfmaWideLong : kLaneMfmaLong)
                                   : (WIDE ? kLaneMfmaWide : (NT >= 8 ? kLaneMfmaMulti : kLaneMfma));
    static constexpr int KEEP = LONG ? kKeepLong : kKeep;
    static constexpr int NC = 2 * WA;             // contributor lists per row
    static constexpr int MERGE_WORDS = 3 + 2 * KL;
    // odd row stride: the lanes of a wave (consecutive rows) hit distinct banks
    static constexpr int RSTRIDE = NC * MERGE_WORDS + 1;
    static constexpr int MERGE_BYTES = 32 * NT * RSTRIDE * 4;
    // lanes per row in the merge: the workgroup's threads over the rows, at
    // most one contributor each
    static constexpr int MT_ALL = (64 * NW) / (32 * NT);
    static constexpr int MT = MT_ALL >= NC ? NC : (MT_ALL >= 1 ? MT_ALL : 1);

    // One row (accumulator column nt) of this lane: the tiles [tw, tw + WM)
    // of which those before t1 lie in the slice (a wave-uniform test) and
    // tokens from V on are left out.  Each logit becomes a key: its truncated
    // value (logit_trunc) with the lane-local position p (tokens in
    // increasing id) stored as PB - p in the cleared bits, PB the last
    // position (so most tags are inline constants of the and-or that forms
    // the key, one instruction instead of two).  Keys are
    // distinct, and for positive values their order is the (value desc, id
    // asc) order; equal negative values rank the larger id first, and when
    // that drops the smaller one the bound reaches the listed value, so the
    // merge re-evaluates the slice and the result stays exact.  The KL + 1
    // best keys cost KL + 1 medians per logit (the maximum as a median with
    // +inf, held in a scalar register the compiler cannot see through: as a
    // max it would first quiet each key, one more instruction per logit), the
    // lists' ids coming from the tags at the end; the exponentials follow in
    // the same pass, tile by tile (below).
    __device__ __forceinline__ void lane_row(const f32x16 (&acc)[WM][NTW], int nt, int vbase0, int tw, int t1,
                                             float* c) const {
        constexpr int TAG = (1 << kLogitTagBits) - 1;
        constexpr int PB = WM * 16 - 1;   // last lane-local position
        static_assert(PB <= TAG && 16 > KL, "positions fit the tag bits; one tile fills a list");
        float k[KL + 1];
#pragma unroll
        for (int q = 0; q <= KL; ++q) k[q] = neg_inf();
        float pinf;
        asm("s_mov_b32 %0, 0x7f800000" : "=s"(pinf));
        auto insert = [&](float key) {
            float n[KL + 1];
            n[0] = __builtin_amdgcn_fmed3f(k[0], key, pinf);
#pragma unroll
            for (int q = 1; q <= KL; ++q) n[q] = __builtin_amdgcn_fmed3f(k[q - 1], k[q], key);
#pragma unroll
            for (int q = 0; q <= KL; ++q) k[q] = n[q];
        };
        // one pass: a tile's logits are read once, ranked, then summed as
        // exponentials relative to the running maximum (the truncated best
        // key so far), the sum so far rescaled when the maximum grows; the
        // hardware exp2 flushes terms below 2^-126 of the maximum's to zero
        float m = neg_inf(), s = 0.f;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            if (tw + mt >= t1) continue;   // wave-uniform: a tile past the slice
            const bool full = (tw + mt + 1) * 32 <= V;   // wave-uniform: else the per-token test
            float xv[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) xv[j] = acc[mt][nt][j];
            auto key = [&](int j) { return __int_as_float((__float_as_int(xv[j]) & ~TAG) | (PB - (mt * 16 + j))); };
            auto valid = [&](int j) { return vbase0 + 32 * mt + 8 * (j >> 2) + (j & 3) < V; };
            if (full) {
#pragma unroll
                for (int j = 0; j < 16; ++j) insert(key(j));
            } else {
#pragma unroll
                for (int j = 0; j < 16; ++j) insert(valid(j) ? key(j) : neg_inf());
            }
            const float mn = logit_trunc(k[0]);
            if (mn != neg_inf()) {
                const float ms = mn * sl2;
                float t = 0.f;
                if (full) {
#pragma unroll
                    for (int j = 0; j < 16; ++j) t += __builtin_amdgcn_exp2f(fmaf(xv[j], sl2, -ms));
                } else {
#pragma unroll
                    for (int j = 0; j < 16; ++j)
                        if (valid(j)) t += __builtin_amdgcn_exp2f(fmaf(xv[j], sl2, -ms));
                }
                s = s * __builtin_amdgcn_exp2f((m - mn) * sl2) + t;   // m = -inf: s is still 0
                m = mn;
            }
        }
        c[0] = m;
        c[1] = s;
        c[2] = logit_trunc(k[KL]);
#pragma unroll
        for (int q = 0; q < KL; ++q) {
            const bool ok = k[q] != neg_inf();
            const int p = PB - (__float_as_int(k[q]) & TAG);
            c[3 + q] = ok ? logit_trunc(k[q]) : neg_inf();
            c[3 + KL + q] = __int_as_float(ok ? vbase0 + 32 * (p >> 4) + 8 * ((p >> 2) & 3) + (p & 3) : -1);
        }
    }

    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NTW], const Segment& it, unsigned char* smem,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
        const int wa = wave % WA, wb = wave / WA;
        float* cm = reinterpret_cast<float*>(smem);   // [32*NT rows, stride RSTRIDE][NC contributors][MERGE_WORDS]
        const int q = wa * 2 + (lane >> 5);
        // this lane's row of accumulator column 0
        float* crow = cm + (wb * NTW * 32 + (lane & 31)) * RSTRIDE + q * MERGE_WORDS;
        const int tw = it.t0 + wa * WM;              // this wave's first tile
        const int vbase0 = tw * 32 + 4 * (lane >> 5);
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) lane_row(acc, nt, vbase0, tw, it.t1, crow + nt * 32 * RSTRIDE);
        lds_barrier();
        lm_merge_contributors<NC, KL, KEEP, MT>(cm, RSTRIDE, 32 * NT, it.row0, it.chunk, sh.nchunks, sh.R, sl2, part);
    }
};

// Cut items: every workgroup holding a piece stores its accumulators, and
// the last one to arrive sums the pieces in workgroup order (so the result
// does not depend on arrival order) and runs the real epilogue.  The arrival
// counters are zeroed before the product starts.
//
// The pieces may sit on different XCDs, whose L2 caches are not coherent
// with each other.  A device-scope fence would write back and invalidate the
// whole L2 of the XCD (stalling every workgroup there), so only this
// traffic is made device-coherent: the partial sums are written and read with
// device-scope relaxed atomics (write-through stores and loads that do not
// hit stale lines), the writer waits for its stores to complete before it
// bumps the counter, and the reader loads only after seeing the count.
__device__ __forceinline__ void store_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// every memory operation of this thread issued so far has completed
__device__ __forceinline__ void wait_memory() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int WM, int NT, int NW, class Inner>
struct EpiFixup {
    Inner inner;
    float* partial;   // [2 * G][PART_FLOATS]
    int* counter;     // [items]

    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char* smem,
                                          const GemmShape& sh) {
        if (it.npieces > 1 && !combine(acc, it, smem, sh)) return;
        inner.apply(acc, it, smem, sh);
    }

    // Store this piece; if it is the last to arrive, replace acc by the sum
    // of all pieces and return true.
    __device__ __forceinline__ bool combine(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char* smem,
                                         const GemmShape& sh) {
        constexpr int PF = GemmTraits<WM, NT, NW>::PART_FLOATS;
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
        // register j of accumulator (mt, nt) of all 64 lanes: one 256-byte row
        auto idx = [&](int mt, int nt, int j) { return (((wave * WM + mt) * NT + nt) * 16 + j) * 64 + lane; };
        float* mine = partial + (size_t)piece_slot(sh, it.g, it.item) * PF;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int j = 0; j < 16; ++j) store_coherent(mine + idx(mt, nt, j), acc[mt][nt][j]);
        wait_memory();
        __syncthreads();   // every thread's piece is stored
        int* flag = reinterpret_cast<int*>(smem);
        if (threadIdx.x == 0)
            flag[0] = (__hip_atomic_fetch_add(counter + it.item, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                       it.npieces - 1)
                          ? 1
                          : 0;
        __syncthreads();
        const bool last = flag[0] != 0;
        __syncthreads();   // flag read by all before the epilogue reuses the LDS
        if (!last) return false;
        // pieces in workgroup order (this workgroup's own one re-read from
        // memory, so every sum is the same chain of additions); the loads of
        // one piece are independent, so each piece costs one round trip
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int j = 0; j < 16; ++j) acc[mt][nt][j] = 0.f;
        for (int pc = 0; pc < it.npieces; ++pc) {
            const float* src = partial + (size_t)piece_slot(sh, it.gfirst + pc, it.item) * PF;
            f32x16 v[WM][NT];
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                    for (int j = 0; j < 16; ++j) v[mt][nt][j] = load_coherent(src + idx(mt, nt, j));
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                    for (int j = 0; j < 16; ++j) acc[mt][nt][j] += v[mt][nt][j];
        }
        return true;
    }
};

// SwiGLU activation: a[r, i] = bf16( silu(g) * u ).
template <int WM, int NT>
struct EpiSwiGLU {
    // [R, 2I]: a = silu(g) * u as bf16 pairs, hi = bf16(a), lo = bf16(a - hi),
    // interleaved by 8 (hi of elements 8j..8j+7, then their lo), so the down
    // projection reads the activation at about 16 significant bits
    uint16_t* out;
    int I;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char*,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = it.t0 + wave * WM + mt;
            if (tile >= it.t1) continue;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = it.row0 + nt * 32 + (lane & 31);
                if (r >= sh.R) continue;
#pragma unroll
                for (int jg = 0; jg < 2; ++jg) {
                    const int i = tile * 16 + 8 * jg + 4 * (lane >> 5);
                    if (i >= I) continue;
                    uint32_t hi2[2], lo2[2];
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        float a[2];
#pragma unroll
                        for (int e = 0; e < 2; ++e) {
                            const float g = acc[mt][nt][4 * jg + 2 * q + e];
                            const float u = acc[mt][nt][4 * jg + 2 * q + e + 8];
                            // silu(g) = g / (1 + e^-g), the quotient by the hardware reciprocal
                            a[e] = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
                        }
                        hi2[q] = f32x2_to_bf16x2_bits(a[0], a[1]);
                        lo2[q] = f32x2_to_bf16x2_bits(a[0] - bf16_bits_to_f32(hi2[q] & 0xffffu),
                                                      a[1] - bf16_bits_to_f32(hi2[q] >> 16));
                    }
                    uint16_t* o = out + (size_t)r * 2 * I + (size_t)(i >> 3) * 16 + (i & 7);
                    *reinterpret_cast<uint2*>(o) = uint2{hi2[0], hi2[1]};
                    *reinterpret_cast<uint2*>(o + 8) = uint2{lo2[0], lo2[1]};
                }
            }
        }
    }
};

// Plain SiLU activation (no up projection): a[r, i] = silu(g) for tiles of
// 32 gate rows, written as bf16 hi/lo pairs interleaved by 8 like EpiSwiGLU.
template <int WM, int NT>
struct EpiSiLU {
    uint16_t* out;   // [R, 2I]
    int I;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char*,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = it.t0 + wave * WM + mt;
            if (tile >= it.t1) continue;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = it.row0 + nt * 32 + (lane & 31);
                if (r >= sh.R) continue;
#pragma unroll
                for (int jg = 0; jg < 4; ++jg) {
                    const int i = tile * 32 + 8 * jg + 4 * (lane >> 5);
                    if (i >= I) continue;
                    uint32_t hi2[2], lo2[2];
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        float a[2];
#pragma unroll
                        for (int e = 0; e < 2; ++e) {
                            const float g = acc[mt][nt][4 * jg + 2 * q + e];
                            a[e] = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
                        }
                        hi2[q] = f32x2_to_bf16x2_bits(a[0], a[1]);
                        lo2[q] = f32x2_to_bf16x2_bits(a[0] - bf16_bits_to_f32(hi2[q] & 0xffffu),
                                                      a[1] - bf16_bits_to_f32(hi2[q] >> 16));
                    }
                    uint16_t* o = out + (size_t)r * 2 * I + (size_t)(i >> 3) * 16 + (i & 7);
                    *reinterpret_cast<uint2*>(o) = uint2{hi2[0], hi2[1]};
                    *reinterpret_cast<uint2*>(o + 8) = uint2{lo2[0], lo2[1]};
                }
            }
        }
    }
};

// fp32 store of the product: out[r, tile*32 + row of the tile] (the h~
// half of an input projection, one row per drafter state).
template <int WM, int NT>
struct EpiStoreF32 {
    float* out;
    int ldo;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char*,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = it.t0 + wave * WM + mt;
            if (tile >= it.t1) continue;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = it.row0 + nt * 32 + (lane & 31);
                if (r >= sh.R) continue;
#pragma unroll
                for (int jg = 0; jg < 4; ++jg) {
                    const int n = tile * 32 + 8 * jg + 4 * (lane >> 5);
                    *reinterpret_cast<f32x4*>(out + (size_t)r * ldo + n) =
                        f32x4{acc[mt][nt][4 * jg], acc[mt][nt][4 * jg + 1], acc[mt][nt][4 * jg + 2],
                              acc[mt][nt][4 * jg + 3]};
                }
            }
        }
    }
};

// Adds to every row's product the h~-half product of its drafter state
// (EpiStoreF32's layout, the same weight tiles), then runs `inner`: the
// product over x = [h~ ; e~] (Eq. 1) with the h~ half computed once per
// (sequence, depth).
template <int WM, int NT, class Inner>
struct EpiAddH {
    Inner inner;
    const float* H;   // [b*gamma, ldh]
    int ldh;
    RowTable t;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char* smem,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = it.row0 + nt * 32 + (lane & 31);
            if (r >= sh.R) continue;
            const int s = r / t.Rs;
            const float* hrow = H + (size_t)(s * t.gamma + t.depth(r - s * t.Rs) - 1) * ldh;
#pragma unroll
            for (int mt = 0; mt < WM; ++mt) {
                const int tile = it.t0 + wave * WM + mt;
                if (tile >= it.t1) continue;
#pragma unroll
                for (int jg = 0; jg < 4; ++jg) {
                    const f32x4 hv = *reinterpret_cast<const f32x4*>(hrow + tile * 32 + 8 * jg + 4 * (lane >> 5));
#pragma unroll
                    for (int q = 0; q < 4; ++q) acc[mt][nt][4 * jg + q] += hv[q];
                }
            }
        }
        inner.apply(acc, it, smem, sh);
    }
};

// Residual: h'[r, n] = bf16( h[seq, depth-1, n] + y[r, n] ).
template <int WM, int NT>
struct EpiResidual {
    uint16_t* out;        // [R, d]
    const uint16_t* h;    // [b, gamma, d]
    int d;
    RowTable t;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const Segment& it, unsigned char*,
                                          const GemmShape& sh) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = it.row0 + nt * 32 + (lane & 31);
            if (r >= sh.R) continue;
            const int s = r / t.Rs;
            const int rl = r - s * t.Rs;
            const uint16_t* hrow = h + (size_t)(s * t.gamma + t.depth(rl) - 1) * d;
#pragma unroll
            for (int mt = 0; mt < WM; ++mt) {
                const int tile = it.t0 + wave * WM + mt;
                if (tile >= it.t1) continue;
#pragma unroll
                for (int jg = 0; jg < 4; ++jg) {
                    const int n = tile * 32 + 8 * jg + 4 * (lane >> 5);
                    if (n >= d) continue;
                    const uint2 hv = *reinterpret_cast<const uint2*>(hrow + n);
                    const float h0 = bf16_bits_to_f32(hv.x & 0xffffu), h1 = bf16_bits_to_f32(hv.x >> 16);
                    const float h2 = bf16_bits_to_f32(hv.y & 0xffffu), h3 = bf16_bits_to_f32(hv.y >> 16);
                    const uint32_t o01 = f32x2_to_bf16x2_bits(h0 + acc[mt][nt][4 * jg + 0], h1 + acc[mt][nt][4 * jg + 1]);
                    const uint32_t o23 = f32x2_to_bf16x2_bits(h2 + acc[mt][nt][4 * jg + 2], h3 + acc[mt][nt][4 * jg + 3]);
                    *reinterpret_cast<uint2*>(out + (size_t)r * d + n) = uint2{o01, o23};
                }
            }
        }
    }
};

}  // namespace tf

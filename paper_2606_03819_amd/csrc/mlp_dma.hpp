// The AR approximator's products when one activation row block holds every
// conditional row (at most 128 rows, at most 32 drafter states): the batch-1
// drafting step.
//
// Every product streams a weight matrix once against few activation rows, so
// it is bound by HBM.  An item is TG weight tiles of 32 rows over the whole
// reduction range; the range runs in 64-column chunks ("units"), and the
// units of all items are dealt out in contiguous ranges to G workgroups, so
// every workgroup streams the same weight bytes.  An item cut by a range
// boundary is computed in pieces whose sums the last piece to arrive adds
// in piece order (the same device-coherent hand-off as the SwiGLU products
// of several row blocks).
//
// The reduction range has up to two phases (Eq. 1, x = [h~ ; e~]):
//   h phase  columns 0..d-1 of W_gate / W_up / W_lin against the b*gamma
//            normalised drafter states h~: every row of depth i of a
//            sequence shares h~_i, so this half is computed once per
//            (sequence, depth) on one 32-row activation tile;
//   e phase  the remaining columns against the rows' own inputs: the
//            normalised previous-token embeddings e~ (gate/up, SiLU, linear)
//            or the SwiGLU activation as bf16 hi/lo pairs (down projection).
// The epilogue adds the h-phase sum of a row's (sequence, depth) state to its
// e-phase sum, so the result is the full product over x.
//
// Copies go from memory straight into LDS (global_load_lds): a weight ring of
// SW stages (each TG tiles x 64 columns) fed far ahead, since one item has
// few weight bytes per chunk, and an activation ring of SX stages (the chunk's
// activation tile, re-read from L2 by every workgroup).  Four waves: in the e
// phase wave w holds activation tile w % NTE and the k sub-steps of group
// w / NTE; in the h phase wave w holds the single tile and sub-steps w (mod
// 4).  Waves that share a tile sum their accumulators in wave order after the
// loop.
#pragma once

#include <type_traits>

#include "common.hpp"
#include "dma.hpp"
#include "rows.hpp"
#include "stream_gemm.hpp"
#include "work.hpp"

namespace tf {

// weight rows of a tile: gate rows 16t.. then the up rows with the same
// indices (SwiGLU), or 32 consecutive rows (every other product)
constexpr int kMlpWGateUp = 0;
constexpr int kMlpWPlain = 1;
// epilogues
constexpr int kMlpEpiSwiGLU = 0;    // a = silu(g) * u as bf16 hi/lo pairs
constexpr int kMlpEpiSiLU = 1;      // a = silu(g) as bf16 hi/lo pairs (no up projection)
constexpr int kMlpEpiResidual = 2;  // h' = bf16(h + y)

struct MlpDmaArgs {
    const uint16_t* w;    // plain weights [N, Kw], or the gate rows (gate/up)
    const uint16_t* wu;   // the up rows [N, Kw] (gate/up)
    int N;                // rows of w (and wu)
    int Kw;               // weight columns
    const uint16_t* xh;   // h phase: [Rh, d] normalised drafter states
    const uint16_t* xe;   // e phase: [Re, lde]
    long lde;
    int Rh, Re;
    int ntiles, items, nkh, nke, G;
    int wh, we;           // split costs of an h and an e chunk (CostSplit)
    uint16_t* out;        // [Re, 2 * Nout] hi/lo pairs, or [Re, Nout] (residual)
    int Nout;             // output width: I (activations) or d (residual)
    const uint16_t* h;    // residual source [b * gamma, d] (raw drafter states)
    RowTable rt;
    float* partial;       // [2G][PF] pieces of cut items
    int* counter;         // [items] arrival counters, zero before the launch
};

// 16-byte slot swizzle of 128-byte rows (below)
__device__ __forceinline__ int mlp_swz128(int r) { return (r >> 1) & 7; }

template <int TG, int NTE, bool PAIRED, int SW, int SX>
struct MlpDmaTraits {
    static constexpr int NTHREADS = 256;
    static constexpr int WTILE = 32 * 128;                  // one weight tile of one stage (64 columns)
    static constexpr int WSTAGE = TG * WTILE;
    static constexpr int XROWB = PAIRED ? 256 : 128;        // bytes of an activation row in one stage
    static constexpr int XRPI = 1024 / XROWB;               // activation rows per DMA instruction
    static constexpr int XSTAGE_E = 32 * NTE * XROWB;
    static constexpr int XSTAGE_H = 32 * 128;
    static constexpr int XSTAGE = XSTAGE_E > XSTAGE_H ? XSTAGE_E : XSTAGE_H;
    static constexpr int XOFF = SW * WSTAGE;
    static constexpr int RING = SW * WSTAGE + SX * XSTAGE;
    static constexpr int QS = PAIRED ? 8 : 4;               // MFMA k sub-steps per chunk (e phase)
    // every wave copies a quarter of each chunk (8-row blocks of 1 KiB)
    static constexpr int WPW = TG;                          // weight DMA instructions per wave per chunk
    static constexpr int XPW_H = 1;                         // activation DMA instructions per wave (h phase)
    static constexpr int XPW_E = XSTAGE_E / 1024 / 4;       // ... (e phase)
    static_assert((SW - 1) * WPW + (SX - 1) * XPW_E <= 62, "vmcnt range");
    // 2 x 2 wave grid: two waves along the weight tiles (TW each), two
    // along the activation tiles (NTW each, or both on the single tile of
    // the h phase / of NTE = 1, splitting its k sub-steps)
    static constexpr int TW = TG / 2;
    static constexpr int NTW = NTE >= 2 ? NTE / 2 : 1;
    // after the loop the piece's sums (PF floats) reuse the ring's LDS
    static constexpr int TILE_F = 1024;                     // floats of one 32x32 accumulator
    static constexpr int PF = TG * TILE_F * (1 + NTE);      // floats of one item's sums (h, then e)
    static constexpr int SCR_C = PF * 4;
    static constexpr int SMEM = RING > SCR_C ? RING : SCR_C;
    static constexpr int HC = 4 * TG;                       // summed h floats per thread
    static constexpr int EC = 4 * TG * NTE;                 // summed e floats per thread
    static_assert(TG % 2 == 0, "weight tiles split over two waves");
    static_assert(NTE == 1 || NTE == 2 || NTE == 4 || NTE == 8, "activation tiles");
    static_assert(XPW_E >= 1 && XSTAGE_E % 4096 == 0, "whole DMA instructions per wave");
    static_assert(SW > SX && SX >= 2, "ring depths: a chunk's weights are copied before its activations");
    // 16-byte slot swizzles: 128-byte rows (weights, plain activations) and
    // 256-byte rows (paired activations) keep a quarter-wave's 16 fragment
    // reads at one logical slot on 16 distinct bank groups
    __device__ static __forceinline__ int swz128(int r) { return mlp_swz128(r); }
    __device__ static __forceinline__ int swz256(int r) { return r & 15; }
};

// ------------------------------------------------------------------ outputs
//
// An item's sums are in MFMA register order: value j of lane L of a 32 x 32
// tile is weight row 8(j/4) + 4(L/32) + j%4, activation row L%32.  The
// epilogue walks an item in units of (row, weight tile, group of 8 outputs);
// a group's 8 sums sit in registers jbase + e2 % 4 of lanes c + 32 (e2 / 4),
// e2 = 0..7.  Row r of sequence s at depth i adds the h-phase sum of drafter
// state s*gamma + i - 1.

// An item's sums in LDS: hs [TG][1024] (h phase), es [TG][NTE][1024] (e phase).
struct MlpLdsSums {
    const float* hs;
    const float* es;
    template <int TG, int NTE, bool HASH>
    __device__ __forceinline__ void get(int t, int n, int c, int hr, int jbase, float (&v)[8]) const {
#pragma unroll
        for (int e2 = 0; e2 < 8; ++e2) {
            const int j = jbase + (e2 & 3), hi = 32 * (e2 >> 2);
            float x = es[(t * NTE + n) * 1024 + j * 64 + c + hi];
            if constexpr (HASH) x += hs[t * 1024 + j * 64 + hr + hi];
            v[e2] = x;
        }
    }
};

// Outputs of `item`, one epilogue unit per thread at a time, from `src`:
// unit e = tid + 256 it is row e % (32 NTE), tile and group e / (32 NTE);
// 256 is a multiple of 32 NTE, so a thread keeps one row (and its drafter
// state) for every unit.  The residual rows are read before any sum, the
// sums of a unit are all loaded before the arithmetic.
template <int TG, int NTE, int EPI, bool HASH, class Src>
__device__ __forceinline__ void mlp_epilogue(const MlpDmaArgs& a, int item, const Src& src) {
    constexpr int GPT = EPI == kMlpEpiSwiGLU ? 2 : 4;   // groups of 8 outputs per tile
    constexpr int NE = 32 * NTE * TG * GPT;             // units of the item
    constexpr int NIT = (NE + 255) / 256;
    constexpr int RPI = 32 * NTE;                       // rows of a unit row block
    static_assert(256 % RPI == 0, "a thread keeps its row");
    struct Unit {
        int r, t, q, tile, hr;
        bool ok;
    };
    const int tid = threadIdx.x;
    const int r = tid % RPI;
    const int sq = r / a.rt.Rs;
    const int hr = sq * a.rt.gamma + a.rt.depth(r - sq * a.rt.Rs) - 1;
    auto unit = [&](int it) {
        Unit u;
        u.r = r;
        const int tg = tid / RPI + it * (256 / RPI);
        u.t = tg / GPT;
        u.q = tg - u.t * GPT;
        u.tile = item * TG + u.t;
        const int o0 = EPI == kMlpEpiSwiGLU ? u.tile * 16 + 8 * u.q : u.tile * 32 + 8 * u.q;
        u.ok = tg < NE / RPI && r < a.Re && u.tile < a.ntiles && o0 < a.Nout;
        u.hr = hr;
        return u;
    };
    if constexpr (EPI == kMlpEpiResidual) {
        u32x4 hv[NIT];
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const Unit u = unit(it);
            if (u.ok) hv[it] = *reinterpret_cast<const u32x4*>(a.h + (size_t)u.hr * a.Nout + u.tile * 32 + 8 * u.q);
        }
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const Unit u = unit(it);
            if (!u.ok) continue;
            float v[8];
            src.template get<TG, NTE, HASH>(u.t, u.r >> 5, u.r & 31, u.hr, 4 * u.q, v);
            u32x4 o;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const float y0 = bf16_bits_to_f32(hv[it][p] & 0xffffu) + v[2 * p];
                const float y1 = bf16_bits_to_f32(hv[it][p] >> 16) + v[2 * p + 1];
                o[p] = f32x2_to_bf16x2_bits(y0, y1);
            }
            *reinterpret_cast<u32x4*>(a.out + (size_t)u.r * a.Nout + u.tile * 32 + 8 * u.q) = o;
        }
    } else {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const Unit u = unit(it);
            if (!u.ok) continue;
            // activation i0..i0+7 as bf16 hi/lo pairs interleaved by 8
            const int i0 = EPI == kMlpEpiSwiGLU ? u.tile * 16 + 8 * u.q : u.tile * 32 + 8 * u.q;
            float gv[8], uv[8];
            src.template get<TG, NTE, HASH>(u.t, u.r >> 5, u.r & 31, u.hr, 4 * u.q, gv);
            if constexpr (EPI == kMlpEpiSwiGLU)   // up rows 16.. of the tile
                src.template get<TG, NTE, HASH>(u.t, u.r >> 5, u.r & 31, u.hr, 4 * u.q + 8, uv);
            u32x4 hi4, lo4;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                float av[2];
#pragma unroll
                for (int z = 0; z < 2; ++z) {
                    const int e2 = 2 * p + z;
                    // silu(g) = g / (1 + e^-g), the quotient by the hardware reciprocal
                    av[z] = gv[e2] * __builtin_amdgcn_rcpf(1.0f + __expf(-gv[e2]));
                    if constexpr (EPI == kMlpEpiSwiGLU) av[z] *= uv[e2];
                }
                hi4[p] = f32x2_to_bf16x2_bits(av[0], av[1]);
                lo4[p] = f32x2_to_bf16x2_bits(av[0] - bf16_bits_to_f32(hi4[p] & 0xffffu),
                                              av[1] - bf16_bits_to_f32(hi4[p] >> 16));
            }
            uint16_t* o = a.out + (size_t)u.r * 2 * a.Nout + (size_t)(i0 >> 3) * 16;
            *reinterpret_cast<u32x4*>(o) = hi4;
            *reinterpret_cast<u32x4*>(o + 8) = lo4;
        }
    }
}

// Copy cursors of one segment: the next chunk (segment-relative) of each
// stream and its ring stage, and the stages the next chunk is read from.
struct MlpCursor {
    int wnext, wstage, xnext, xstage, rw, rx;
};

// One chunk of weights: this wave's 8-row block c of every tile of the item.
// One workgroup alone reads a weight tile, so the copies are non-temporal
// (they do not displace the activation rows every workgroup re-reads from L2).
template <int TG>
__device__ __forceinline__ void mlp_copy_w(const uint16_t* const (&wsrc)[TG], int chunk, unsigned char* st, int wtile,
                                           int c) {
#pragma unroll
    for (int t = 0; t < TG; ++t) dma16(wsrc[t] + 64 * chunk, st + t * wtile + c * 1024, kCpolNt);
}

// One chunk of activations: this wave's 8-row block of the h~ rows in the h
// phase, else its DMA instructions q = c + 4v of the e-phase rows.
template <int XPW_E, bool PAIRED>
__device__ __forceinline__ void mlp_copy_x(const uint16_t* hsrc, const uint16_t* const (&esrc)[XPW_E], bool hphase,
                                           int chunk, unsigned char* st, int c) {
    if (hphase) {
        dma16(hsrc + 64 * chunk, st + c * 1024, 0);
    } else {
#pragma unroll
        for (int v = 0; v < XPW_E; ++v)
            dma16(esrc[v] + (long)(PAIRED ? 128 : 64) * chunk, st + (c + 4 * v) * 1024, 0);
    }
}

// Copy order.  Every wave copies its share of both streams; step s (after
// its barrier) copies the activations of chunk s + SX - 1, then the weights
// of chunk s + SW - 1, and the prologue issues the copies the steps
// 1 - SW .. -1 would have, in the same order.  A wave's loads complete in
// issue order, so at step s waiting for its activation copies of chunk s
// (issued after those of the weights of chunk s, SW > SX) waits for both:
// at most the copies issued after them may be outstanding, the weights of
// chunk s + SW - SX and the activations and weights of the SX - 2 steps
// between (chunks past the segment are never copied).
template <class T, int SW, int SX>
__device__ __forceinline__ int mlp_wait_count(int s, int nsteps, int c0, int nkh) {
    int n = s + SW - SX < nsteps ? T::WPW : 0;
#pragma unroll
    for (int j = 1; j <= SX - 2; ++j) {
        if (s + j < nsteps) n += c0 + s + j < nkh ? T::XPW_H : T::XPW_E;
        if (s + j + SW - SX < nsteps) n += T::WPW;
    }
    return n;
}

// The copies of (emulated) step s: activations of chunk s + SX - 1 (when that
// is a chunk of the segment), then weights of chunk s + SW - 1.
template <class T, int SW, int SX, bool PAIRED, int TG = T::TW * 2>
__device__ __forceinline__ void mlp_step_copies(MlpCursor& cur, int s, int nsteps, int c0, int nkh, int c,
                                                const uint16_t* const (&wsrc)[TG], const uint16_t* hsrc,
                                                const uint16_t* const (&esrc)[T::XPW_E], unsigned char* dyn) {
    if (s + SX - 1 >= 0 && cur.xnext < nsteps) {
        mlp_copy_x<T::XPW_E, PAIRED>(hsrc, esrc, c0 + cur.xnext < nkh, cur.xnext,
                                     dyn + T::XOFF + cur.xstage * T::XSTAGE, c);
        ++cur.xnext;
        cur.xstage = cur.xstage + 1 == SX ? 0 : cur.xstage + 1;
    }
    if (cur.wnext < nsteps) {
        mlp_copy_w<TG>(wsrc, cur.wnext, dyn + cur.wstage * T::WSTAGE, T::WTILE, c);
        ++cur.wnext;
        cur.wstage = cur.wstage + 1 == SW ? 0 : cur.wstage + 1;
    }
}

// The start of step s: wait for this wave's copies of chunk s, meet the
// barrier (every wave's copies have landed; the stages chunk s - 1 used are
// free), then copy into the freed stages.
template <class T, int SW, int SX, bool PAIRED, int TG = T::TW * 2>
__device__ __forceinline__ void mlp_step_begin(MlpCursor& cur, int s, int nsteps, int c0, int nkh, int c,
                                               const uint16_t* const (&wsrc)[TG], const uint16_t* hsrc,
                                               const uint16_t* const (&esrc)[T::XPW_E], unsigned char* dyn) {
    wait_vmcnt_dyn(mlp_wait_count<T, SW, SX>(s, nsteps, c0, nkh));
    block_barrier();
    mlp_step_copies<T, SW, SX, PAIRED>(cur, s, nsteps, c0, nkh, c, wsrc, hsrc, esrc, dyn);
}

__device__ __forceinline__ CostSplit mlp_shape(const MlpDmaArgs& a) {
    return cost_split(a.items, a.nkh, a.nke, a.wh, a.we, a.G);
}

// Weight DMA sources of wave c (rows 8c..8c+7 of every tile) at chunk c0 of
// `item`.
template <int TG, int WMAP>
__device__ __forceinline__ void mlp_weight_sources(const MlpDmaArgs& a, int item, int c0, int c, int lane,
                                                   const uint16_t* (&wsrc)[TG]) {
    const int lrow = lane >> 3, lslot = lane & 7;
    const int row = 8 * c + lrow;
#pragma unroll
    for (int t = 0; t < TG; ++t) {
        const int tile = min(item * TG + t, a.ntiles - 1);
        const uint16_t* base;
        if constexpr (WMAP == kMlpWGateUp) {
            const int i = min(tile * 16 + (row & 15), a.N - 1);
            base = (row < 16 ? a.w : a.wu) + (size_t)i * a.Kw;
        } else {
            base = a.w + (size_t)min(tile * 32 + row, a.N - 1) * a.Kw;
        }
        wsrc[t] = base + 8 * (lslot ^ mlp_swz128(row)) + 64 * c0;
    }
}

// The copy state of one item piece, chunks [c0, c1) of `item`: this lane's
// DMA sources at chunk c0 and the ring cursors.
template <int TG, int XPW>
struct MlpSegment {
    const uint16_t* wsrc[TG];
    const uint16_t* hsrc;
    const uint16_t* esrc[XPW];
    MlpCursor cur;
    int c0, nsteps;
};

// A piece's sources and the ring prologue (the copies of the emulated steps
// 1 - SW .. -1).  Issued apart from the piece's loop so that a workgroup's
// first copies leave before any set-up of its own.
template <int TG, int NTE, bool PAIRED, int SW, int SX, int WMAP>
__device__ __forceinline__ void mlp_piece_begin(const MlpDmaArgs& a, int item, int c0, int c1, unsigned char* dyn,
                                                MlpSegment<TG, MlpDmaTraits<TG, NTE, PAIRED, SW, SX>::XPW_E>& sg) {
    using T = MlpDmaTraits<TG, NTE, PAIRED, SW, SX>;
    const int lane = threadIdx.x & 63;
    const int c = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // this wave's quarter of every chunk
    // this lane's row and physical slot in a 1 KiB DMA block of 128-byte rows
    const int lrow = lane >> 3, lslot = lane & 7;
    sg.c0 = c0;
    sg.nsteps = c1 - c0;
    mlp_weight_sources<TG, WMAP>(a, item, c0, c, lane, sg.wsrc);
    // h phase: 32 rows of h~ in four 8-row blocks, block c
    {
        const int row = 8 * c + lrow;
        sg.hsrc = a.xh != nullptr ? a.xh + (size_t)min(row, a.Rh - 1) * (a.nkh * 64) + 8 * (lslot ^ T::swz128(row)) +
                                        64 * c0
                                  : nullptr;
    }
    // e phase: DMA instruction q = c + 4v covers rows XRPI*q ..
    const int ce0 = c0 - a.nkh;   // e chunk of the segment's first chunk (negative in the h phase)
#pragma unroll
    for (int v = 0; v < T::XPW_E; ++v) {
        const int q = c + 4 * v;
        int row, ps;
        if constexpr (PAIRED) {
            row = 4 * q + (lane >> 4);
            ps = (lane & 15) ^ T::swz256(row);
        } else {
            row = 8 * q + lrow;
            ps = lslot ^ T::swz128(row);
        }
        sg.esrc[v] = a.xe + (size_t)min(row, a.Re - 1) * a.lde + 8 * ps + (long)(PAIRED ? 128 : 64) * ce0;
    }
    sg.cur = MlpCursor{0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int s = 1 - SW; s < 0; ++s)
        mlp_step_copies<T, SW, SX, PAIRED>(sg.cur, s, sg.nsteps, c0, a.nkh, c, sg.wsrc, sg.hsrc, sg.esrc, dyn);
}

// The rest of the piece begun by mlp_piece_begin, streamed through the rings
// in `dyn`.  On return every copy has landed, the LDS is free, and hc / ec
// hold this thread's part of the piece's sums, the waves' accumulators added
// in wave order: hc[i] is the 16-byte group 4 tid + 1024 i of [TG][1024] (h
// phase), ec[i] that of [TG][NTE][1024] (e phase).
template <int TG, int NTE, bool PAIRED, int SW, int SX>
__device__ __forceinline__ void mlp_piece_run(const MlpDmaArgs& a,
                                              MlpSegment<TG, MlpDmaTraits<TG, NTE, PAIRED, SW, SX>::XPW_E>& sg,
                                              unsigned char* dyn, f32x4 (&hc)[TG], f32x4 (&ec)[TG * NTE]) {
    using T = MlpDmaTraits<TG, NTE, PAIRED, SW, SX>;
    constexpr int TW = T::TW, NTW = T::NTW;
    static_assert(SX == 2 || SX == 3, "one or two activation chunks in flight");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // the wave's place in the 2 x 2 grid: weight tiles wa*TW.., activation tiles wb*NTW..
    const int wa = wave & 1, wb = wave >> 1;
    const int fr = lane & 31;
    const int c0 = sg.c0, nsteps = sg.nsteps;
    const auto& wsrc = sg.wsrc;
    const auto& esrc = sg.esrc;
    MlpCursor& cur = sg.cur;

    f32x16 acc_h[TW], acc_e[TW][NTW];
#pragma unroll
    for (int t = 0; t < TW; ++t)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            acc_h[t][j] = 0.f;
#pragma unroll
            for (int n = 0; n < NTW; ++n) acc_e[t][n][j] = 0.f;
        }

    // The two phases run in loops of their own: each updates only its own
    // accumulators, so none of them is copied between iterations.  A step
    // first waits for this wave's copies of chunk s and meets the barrier
    // (every wave's copies of chunk s have landed; the stages of chunk
    // s - 1 are free), then refills the freed stages.
    const int nh = max(0, min(nsteps, a.nkh - c0));   // h-phase chunks of the segment
    for (int s = 0; s < nh; ++s) {
        mlp_step_begin<T, SW, SX, PAIRED>(cur, s, nsteps, c0, a.nkh, wave, wsrc, sg.hsrc, esrc, dyn);
        const unsigned char* wt = dyn + cur.rw * T::WSTAGE + wa * TW * T::WTILE;
        const unsigned char* xt = dyn + T::XOFF + cur.rx * T::XSTAGE;
        cur.rw = cur.rw + 1 == SW ? 0 : cur.rw + 1;
        cur.rx = cur.rx + 1 == SX ? 0 : cur.rx + 1;
        // the single activation tile, sub-steps wb and wb + 2
#pragma unroll
        for (int qq = 0; qq < 2; ++qq) {
            const int ls = 2 * (wb + 2 * qq) + (lane >> 5);
            const u32x4 b = *reinterpret_cast<const u32x4*>(xt + fr * 128 + ((ls ^ T::swz128(fr)) << 4));
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                const u32x4 af =
                    *reinterpret_cast<const u32x4*>(wt + t * T::WTILE + fr * 128 + ((ls ^ T::swz128(fr)) << 4));
                acc_h[t] = mfma_32x32x16_bf16(af, b, acc_h[t]);
            }
        }
    }
    for (int s = nh; s < nsteps; ++s) {
        mlp_step_begin<T, SW, SX, PAIRED>(cur, s, nsteps, c0, a.nkh, wave, wsrc, sg.hsrc, esrc, dyn);
        const unsigned char* wt = dyn + cur.rw * T::WSTAGE + wa * TW * T::WTILE;
        const unsigned char* xt = dyn + T::XOFF + cur.rx * T::XSTAGE;
        cur.rw = cur.rw + 1 == SW ? 0 : cur.rw + 1;
        cur.rx = cur.rx + 1 == SX ? 0 : cur.rx + 1;
        // activation tiles wb*NTW.. over every sub-step (NTE = 1: the
        // single tile, sub-steps of parity wb)
        constexpr int QSTEP = NTE >= 2 ? 1 : 2;
#pragma unroll
        for (int qq = 0; qq < T::QS / QSTEP; ++qq) {
            const int q = NTE >= 2 ? qq : wb + 2 * qq;
            u32x4 b[NTW], af[TW];
#pragma unroll
            for (int n = 0; n < NTW; ++n) {
                const int xr = 32 * (NTE >= 2 ? wb * NTW + n : 0) + fr;
                const int ls = 2 * q + (lane >> 5);
                if constexpr (PAIRED)
                    b[n] = *reinterpret_cast<const u32x4*>(xt + xr * 256 + ((ls ^ T::swz256(xr)) << 4));
                else
                    b[n] = *reinterpret_cast<const u32x4*>(xt + xr * 128 + ((ls ^ T::swz128(xr)) << 4));
            }
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                // paired: sub-step q takes hi (lanes 0-31) and lo (32-63) of weight slot q
                const int lw = PAIRED ? q : 2 * q + (lane >> 5);
                af[t] = *reinterpret_cast<const u32x4*>(wt + t * T::WTILE + fr * 128 + ((lw ^ T::swz128(fr)) << 4));
            }
#pragma unroll
            for (int t = 0; t < TW; ++t)
#pragma unroll
                for (int n = 0; n < NTW; ++n) acc_e[t][n] = mfma_32x32x16_bf16(af[t], b[n], acc_e[t][n]);
        }
    }
    __syncthreads();   // every copy has landed and every ring read is done

    // ---- the piece's sums, in LDS in their final layout (fs: [TG][1024] h,
    // then [TG][NTE][1024] e; element j * 64 + lane of a tile is the MFMA
    // register order).  With NTE >= 2 every (weight tile, activation tile)
    // of the e phase belongs to one wave, which writes it in place; the h
    // tile (and NTE = 1's e tile) is split over the two waves of a grid
    // column (k sub-steps), so the second writes and the first adds its own.
    float* fs = reinterpret_cast<float*>(dyn);
    float* const fe = fs + TG * 1024;
    if constexpr (NTE >= 2) {
#pragma unroll
        for (int t = 0; t < TW; ++t)
#pragma unroll
            for (int n = 0; n < NTW; ++n)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    fe[((wa * TW + t) * NTE + wb * NTW + n) * 1024 + j * 64 + lane] = acc_e[t][n][j];
    }
    if (wb == 1) {
#pragma unroll
        for (int t = 0; t < TW; ++t)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                fs[(wa * TW + t) * 1024 + j * 64 + lane] = acc_h[t][j];
                if constexpr (NTE == 1) fe[(wa * TW + t) * 1024 + j * 64 + lane] = acc_e[t][0][j];
            }
    }
    __syncthreads();
    if (wb == 0) {
#pragma unroll
        for (int t = 0; t < TW; ++t)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                float* ph = fs + (wa * TW + t) * 1024 + j * 64 + lane;
                *ph = acc_h[t][j] + *ph;
                if constexpr (NTE == 1) {
                    float* pe = fe + (wa * TW + t) * 1024 + j * 64 + lane;
                    *pe = acc_e[t][0][j] + *pe;
                }
            }
    }
    __syncthreads();
    // 16-byte group tid + 256 i of each phase
#pragma unroll
    for (int i = 0; i < TG; ++i) hc[i] = *reinterpret_cast<const f32x4*>(fs + 4 * tid + 1024 * i);
#pragma unroll
    for (int i = 0; i < TG * NTE; ++i) ec[i] = *reinterpret_cast<const f32x4*>(fe + 4 * tid + 1024 * i);
    __syncthreads();   // the per-wave sums are read; the LDS is free
}

// A cut item's piece: store its sums (the phases it covers) in its slot of
// PF floats, 16 bytes per lane with the cache-policy bit of a device-scope
// store (written through to memory, where the last piece's device-coherent
// loads find them on any XCD).
template <int TG, int NTE, int PF>
__device__ __forceinline__ void mlp_store_piece(float* slot, bool has_h, bool has_e, const f32x4 (&hc)[TG],
                                                const f32x4 (&ec)[TG * NTE]) {
    constexpr int kSc1 = 16;   // cache-policy bits of a device-coherent store
    const int tid = threadIdx.x;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(slot, (short)0, PF * 4, 0x00020000);
    if (has_h) {
#pragma unroll
        for (int i = 0; i < TG; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, hc[i]), rs, (4 * tid + 1024 * i) * 4, 0,
                                                   kSc1);
    }
    if (has_e) {
#pragma unroll
        for (int i = 0; i < TG * NTE; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, ec[i]), rs,
                                                   (TG * 1024 + 4 * tid + 1024 * i) * 4, 0, kSc1);
    }
}

// The last piece of a cut item to arrive: the pieces' sums into csc ([TG][1024]
// h phase, then [TG][NTE][1024] e phase), each phase added over the pieces
// that cover it (pcs), in piece order.  The loads are 16 bytes per lane and
// device-coherent (buffer loads with the sc1 bit the device-scope atomic
// loads carry); one batch holds the h sums of two pieces and the e sums of
// BE, so the usual item (two pieces with h chunks, up to BE with e chunks)
// takes a single round trip.  Each thread owns the 16-byte groups
// tid + 256 i of a phase.
template <int TG, int NTE, int PF, int BE>
__device__ __forceinline__ void mlp_combine_pieces(const float* partial, int nslots, const CutPieces& pcs,
                                                   float* csc) {
    constexpr int kSc1 = 16;   // cache-policy bits of a device-coherent load
    constexpr int H4 = TG, E4 = TG * NTE;   // 16-byte groups per thread of each phase
    constexpr int BH = 2;                   // pieces per batch of the h phase (BE: of the e phase)
    const int tid = threadIdx.x;
    // The descriptor spans the nslots slots: a batch's missing pieces read
    // slot nslots, past the range, which returns zeros without a memory
    // access, so every load of a batch is issued unconditionally.
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(partial), (short)0, nslots * PF * 4, 0x00020000);
    auto ld = [&](int slot, int f) {
        return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (slot * PF + f) * 4, 0, kSc1));
    };
    const f32x4 zero{0.f, 0.f, 0.f, 0.f};
    f32x4 sh[H4], se[E4];
#pragma unroll
    for (int i = 0; i < H4; ++i) sh[i] = zero;
#pragma unroll
    for (int i = 0; i < E4; ++i) se[i] = zero;
    const int nh = pcs.ph1, ne = pcs.npieces - pcs.pe0;
    for (int ph = 0, pe = 0; ph < nh || pe < ne; ph += BH, pe += BE) {
        f32x4 vh[BH][H4], ve[BE][E4];
#pragma unroll
        for (int k = 0; k < BH; ++k) {
            const int slot = ph + k < nh ? pcs.slot(ph + k) : nslots;
#pragma unroll
            for (int i = 0; i < H4; ++i) vh[k][i] = ld(slot, 4 * tid + 1024 * i);
        }
#pragma unroll
        for (int k = 0; k < BE; ++k) {
            const int slot = pe + k < ne ? pcs.slot(pcs.pe0 + pe + k) : nslots;
#pragma unroll
            for (int i = 0; i < E4; ++i) ve[k][i] = ld(slot, TG * 1024 + 4 * tid + 1024 * i);
        }
#pragma unroll
        for (int k = 0; k < BH; ++k)
#pragma unroll
            for (int i = 0; i < H4; ++i) sh[i] += vh[k][i];
#pragma unroll
        for (int k = 0; k < BE; ++k)
#pragma unroll
            for (int i = 0; i < E4; ++i) se[i] += ve[k][i];
    }
#pragma unroll
    for (int i = 0; i < H4; ++i) *reinterpret_cast<f32x4*>(csc + 4 * tid + 1024 * i) = sh[i];
#pragma unroll
    for (int i = 0; i < E4; ++i) *reinterpret_cast<f32x4*>(csc + TG * 1024 + 4 * tid + 1024 * i) = se[i];
}

// Every item piece of this workgroup's range; a cut item is summed by its
// last piece to arrive, in piece order, then written by the epilogue.
template <int TG, int NTE, bool PAIRED, int SW, int SX, int WMAP, int EPI>
__global__ __launch_bounds__(256, 1) void mlp_dma_kernel(MlpDmaArgs a) {
    using T = MlpDmaTraits<TG, NTE, PAIRED, SW, SX>;
    constexpr bool HASH = !PAIRED;   // the down projection alone has no h phase
    extern __shared__ __align__(16) unsigned char dyn[];
    const int tid = threadIdx.x;
    const CostSplit sh = mlp_shape(a);
    const int nk = sh.nk;
    const int g = xcd_logical_id(blockIdx.x, gridDim.x);
    const int u_end = unit_start(sh, g + 1);
    int u = unit_start(sh, g);
    MlpSegment<TG, T::XPW_E> sg;
    if (u < u_end) mlp_piece_begin<TG, NTE, PAIRED, SW, SX, WMAP>(a, u / nk, u % nk, min(nk, u_end - u / nk * nk), dyn, sg);
    while (u < u_end) {
        const int item = u / nk;
        const int c0 = u - item * nk;
        const int c1 = min(nk, u_end - item * nk);
        CutPieces pcs = cut_pieces(sh, item);   // uniform: kept in scalar registers
        pcs.gfirst = __builtin_amdgcn_readfirstlane(pcs.gfirst);
        pcs.npieces = __builtin_amdgcn_readfirstlane(pcs.npieces);
        pcs.slot0 = __builtin_amdgcn_readfirstlane(pcs.slot0);
        pcs.ph1 = __builtin_amdgcn_readfirstlane(pcs.ph1);
        pcs.pe0 = __builtin_amdgcn_readfirstlane(pcs.pe0);
        f32x4 hc[TG], ec[TG * NTE];
        mlp_piece_run<TG, NTE, PAIRED, SW, SX>(a, sg, dyn, hc, ec);

        // ---- a cut item: store this piece; the last to arrive sums them
        float* csc = reinterpret_cast<float*>(dyn);   // [TG][1024] h, then [TG][NTE][1024] e
        bool last = true;
        if (pcs.npieces > 1) {
            mlp_store_piece<TG, NTE, T::PF>(a.partial + (size_t)pcs.slot(g - pcs.gfirst) * T::PF, c0 < a.nkh,
                                            c1 > a.nkh, hc, ec);
            wait_memory();
            __syncthreads();   // every thread's piece is stored
            int* flag = reinterpret_cast<int*>(csc);
            if (tid == 0)
                flag[0] = __hip_atomic_fetch_add(a.counter + item, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                                  pcs.npieces - 1
                              ? 1
                              : 0;
            __syncthreads();
            last = flag[0] != 0;
            __syncthreads();
            if (last) {
                // the pieces' sums in piece order, then the epilogue
                // e pieces per batch: three for SwiGLU over four tiles (an item's
                // e half usually spans three pieces), one for the widest residual
                // epilogue and for eight tiles (registers), else two
                constexpr int BE = NTE == 8 ? 1 : (NTE == 4 ? (EPI == kMlpEpiSwiGLU ? 3 : (EPI == kMlpEpiResidual && HASH ? 1 : 2)) : 2);
                mlp_combine_pieces<TG, NTE, T::PF, BE>(a.partial, 2 * a.G, pcs, csc);
                __syncthreads();
                mlp_epilogue<TG, NTE, EPI, HASH>(a, item, MlpLdsSums{csc, csc + T::HC * 256});
            }
        } else {
            // a whole item: its sums are in LDS as the piece left them
            mlp_epilogue<TG, NTE, EPI, HASH>(a, item, MlpLdsSums{csc, csc + T::HC * 256});
        }
        u = (item + 1) * nk;
        if (u < u_end) {
            __syncthreads();   // the epilogue's LDS use ends before the next item's copies land
            mlp_piece_begin<TG, NTE, PAIRED, SW, SX, WMAP>(a, item + 1, 0, min(nk, u_end - u), dyn, sg);
        }
    }
}

}  // namespace tf

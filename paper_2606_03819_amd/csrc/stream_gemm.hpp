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
// Work decomposition: a workgroup (4 waves) owns one chunk of 4*WM weight
// tiles (WM per wave), one block of 32*NT activation rows and one k-range
// (split-K for the short SwiGLU matrices; the LM head never splits K).  Every
// workgroup therefore streams the same amount of weights.  Per 64-wide
// k-chunk the activation tile [32*NT x 64] is staged in LDS (double buffered,
// rows padded to 144 B so the 16-byte fragment reads are bank-conflict free).
// Each wave streams its own weight rows with fully coalesced loads -- one
// instruction covers 8 rows x 128 B, i.e. whole cache lines -- several
// k-chunks ahead of the MFMAs, and transposes them into fragment order through a
// wave-private LDS tile whose 16-byte slots are XOR-swizzled by row (see
// wswz), so both the writes and the fragment reads are conflict free.  (Loading fragments
// directly -- 32 rows x 32 B per instruction -- measured ~17% less HBM
// bandwidth on MI355X.)
#pragma once

#include "common.hpp"

namespace tf {

struct GemmShape {
    int R;        // activation rows
    int K;        // reduction length (multiple of 16)
    int ntiles;   // 32-row weight tiles
    int nchunks;  // workgroup chunks along the weight tiles
    int nkp;      // k-parts (split-K); each a whole number of 64-wide k-chunks
    int nrb;      // activation-row blocks
};

struct WorkItem {
    int chunk, kp, rb;
    int t0, t1;    // weight tiles [t0, t1)
    int kc0, kc1;  // 64-wide k-chunks [kc0, kc1)
    int row0;      // first activation row
};

// Workgroups are dispatched round-robin over the 8 XCDs of an MI355X.
// Renumber them so consecutive logical ids share an XCD (and its L2): the
// row blocks of one weight chunk then read the same weight tiles through the
// same L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    if ((nblocks & 7) != 0) return bid;
    return (bid & 7) * (nblocks >> 3) + (bid >> 3);
}

template <int WM, int NT>
struct GemmTraits {
    static constexpr int TR = 32 * NT;           // activation rows per workgroup
    static constexpr int KC = 64;                // k per LDS stage
    static constexpr int LDSW = KC + 8;          // padded LDS row, bf16 elements
    static constexpr int XS_BYTES = 2 * TR * LDSW * 2;
    static constexpr int WROWS = 32 * WM;        // weight rows per wave
    static constexpr int WS_BYTES = 4 * WROWS * KC * 2;   // wave-private weight tiles
    static constexpr int SMEM_BYTES = XS_BYTES + WS_BYTES;
    static constexpr int NWL = WROWS / 8;        // coalesced weight loads per wave per k-chunk
    static constexpr int CHUNK = 4 * WM;         // weight tiles per workgroup
    static constexpr int PART_FLOATS = 4 * WM * NT * 16 * 64;   // one workgroup's accumulators
};

template <int WM, int NT>
__device__ __forceinline__ WorkItem work_item(const GemmShape& sh) {
    using T = GemmTraits<WM, NT>;
    WorkItem w;
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    w.rb = L % sh.nrb;
    const int rest = L / sh.nrb;
    w.kp = rest % sh.nkp;
    w.chunk = rest / sh.nkp;
    w.t0 = w.chunk * T::CHUNK;
    w.t1 = min(w.t0 + T::CHUNK, sh.ntiles);
    const int nkc = (sh.K + T::KC - 1) / T::KC;
    w.kc0 = (int)(((long long)w.kp * nkc) / sh.nkp);
    w.kc1 = (int)(((long long)(w.kp + 1) * nkc) / sh.nkp);
    w.row0 = w.rb * T::TR;
    return w;
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

// PIPE: k-chunks of loads in flight per wave.  WNT: weight loads carry the
// non-temporal hint, for weights that one workgroup alone reads (a single
// activation row block), so they do not evict the activations that every
// workgroup re-reads from L2.
template <int WM, int NT, int PIPE, bool WNT, class WSrc, class XSrc, class Epi>
__device__ __forceinline__ void stream_gemm_body(const WSrc& wsrc, const XSrc& xsrc, Epi& epi,
                                                 const GemmShape& sh, unsigned char* smem) {
    using T = GemmTraits<WM, NT>;
    constexpr int TR = T::TR, KC = T::KC, LDSW = T::LDSW, NWL = T::NWL;
    uint16_t* xs = reinterpret_cast<uint16_t*>(smem);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem + T::XS_BYTES) + wave * T::WROWS * KC;
    const WorkItem it = work_item<WM, NT>(sh);
    const int nk = it.kc1 - it.kc0;
    const int slot = lane & 7;          // 16-byte slot of a 128-byte row segment this lane loads

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
    f32x16 acc[WM][NT];
#pragma unroll
    for (int mt = 0; mt < WM; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[mt][nt][j] = 0.f;

    // activation rows of this thread's 16-byte pieces (clamped into [0, R))
    const int kmax = sh.K - 8;
    auto load_x = [&](u32x4 (&xr)[NT], int kc) {
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const int p = tid + 256 * i;
            const int gr = min(it.row0 + (p >> 3), sh.R - 1);
            const int k = min(kc * KC + (p & 7) * 8, kmax);
            xr[i] = *reinterpret_cast<const u32x4*>(xsrc.ptr(gr, k));
        }
    };
    auto store_x = [&](const u32x4 (&xr)[NT], int buf, int kc) {
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const int p = tid + 256 * i;
            const bool ok = it.row0 + (p >> 3) < sh.R && kc * KC + (p & 7) * 8 < sh.K;
            *reinterpret_cast<u32x4*>(xs + buf * TR * LDSW + (p >> 3) * LDSW + (p & 7) * 8) =
                ok ? xr[i] : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto load_w = [&](u32x4 (&w)[NWL], int kc) {
        const int k = min(kc * KC + slot * 8, kmax);
#pragma unroll
        for (int q = 0; q < NWL; ++q) {
            const u32x4* src = reinterpret_cast<const u32x4*>(gw[q] + k);
            if constexpr (WNT)
                w[q] = __builtin_nontemporal_load(src);
            else
                w[q] = *src;
        }
    };
    auto store_w = [&](const u32x4 (&w)[NWL]) {
#pragma unroll
        for (int q = 0; q < NWL; ++q) {
            const int row = 8 * q + (lane >> 3);
            *reinterpret_cast<u32x4*>(wl + row * KC + ((slot ^ wswz(row)) * 8)) = w[q];
        }
    };

    // Software pipeline of depth PIPE: the loads of k-chunk j are issued at the
    // end of step j-PIPE and stored to LDS at the end of step j-1, so each load
    // has PIPE-1 steps to arrive.  Within a step the stores wait only for the
    // loads of the chunk they store (loads return in order), leaving the
    // later chunks in flight.
    static_assert(PIPE >= 2 && PIPE <= 4, "pipeline depth");
    u32x4 xr[PIPE][NT];
    u32x4 wr[PIPE][NWL];
    // MFMAs of k-chunk i from LDS (activation buffer i & 1, the wave's weight tile)
    auto compute = [&](int i) {
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
                bfr[nt] = *reinterpret_cast<const u32x4*>(xb + (nt * 32 + (lane & 31)) * LDSW + ks * 16 +
                                                          (lane >> 5) * 8);
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[mt][nt] = mfma_32x32x16_bf16(afr[mt], bfr[nt], acc[mt][nt]);
        }
    };
    // store register set s (k-chunk i) into LDS after this wave's reads of the
    // previous chunk (LDS operations of a wave complete in order)
    auto stage = [&](int s, int i) {
        compiler_fence();
        store_w(wr[s]);
        store_x(xr[s], i & 1, it.kc0 + i);
        compiler_fence();
    };
    if (nk > 0) {
#pragma unroll
        for (int j = 0; j < PIPE; ++j)
            if (j < nk) {
                load_x(xr[j], it.kc0 + j);
                load_w(wr[j], it.kc0 + j);
            }
        stage(0, 0);
        int i0 = 0;
        // steady state, branch free: every step computes, stages the next
        // chunk and issues the loads PIPE chunks ahead
        for (; i0 + 2 * PIPE <= nk; i0 += PIPE) {
#pragma unroll
            for (int u = 0; u < PIPE; ++u) {
                const int i = i0 + u;
                lds_barrier();  // chunk i visible; the other activation buffer is free
                compute(i);
                stage((u + 1) % PIPE, i + 1);
                load_x(xr[u], it.kc0 + i + PIPE);
                load_w(wr[u], it.kc0 + i + PIPE);
            }
        }
        // tail: fewer than 2*PIPE chunks left
#pragma unroll
        for (int u = 0; u < 2 * PIPE; ++u) {
            const int i = i0 + u;
            if (i < nk) {
                lds_barrier();
                compute(i);
                if (i + 1 < nk) stage((u + 1) % PIPE, i + 1);
                if (i + PIPE < nk) {
                    load_x(xr[u % PIPE], it.kc0 + i + PIPE);
                    load_w(wr[u % PIPE], it.kc0 + i + PIPE);
                }
            }
        }
    }
    __syncthreads();  // LDS tiles no longer needed: the epilogue may reuse them
    epi.apply(acc, it, wave, lane, smem, sh);
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
};

// -------------------------------------------------------- activation sources

struct XRowsPlain {
    const uint16_t* x;
    long ld;
    __device__ __forceinline__ const uint16_t* ptr(int r, int k) const { return x + (size_t)r * ld + k; }
};

// Input of the SwiGLU: row r is [ h~(depth of r) ; e~(r) ] (Eq. 1).
struct XRowsConcat {
    const uint16_t* ht;   // [b*gamma, d] normalised drafter states
    const uint16_t* et;   // [b*R, d] normalised embeddings of the previous tokens
    int d, Rs, gamma, M;
    __device__ __forceinline__ const uint16_t* ptr(int r, int k) const {
        if (k >= d) return et + (size_t)r * d + (k - d);
        const int s = r / Rs;
        const int rl = r - s * Rs;
        const int depth = rl == 0 ? 1 : 2 + (rl - 1) / M;
        return ht + (size_t)(s * gamma + depth - 1) * d + k;
    }
};

// ------------------------------------------------------------------ epilogues

// Merge the 8 contributor lists of each activation row (written to `cm` as
// [rows][8][3 + 2*kLane] = max, sum, bound, values, ids) into the row's
// (row, slice) partial.  One thread per row.
__device__ inline void lm_merge_contributors(const float* cm, int rows, int row0, int split, int nsplit, int R,
                                             float sl2, float* part) {
    constexpr int W = 3 + 2 * kLane;
    const int tid = threadIdx.x;
    if (tid >= rows) return;
    const int grow = row0 + tid;
    if (grow >= R) return;
    const float* c = cm + tid * 8 * W;
    float M = neg_inf(), U = neg_inf();
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        M = fmaxf(M, c[p * W + 0]);
        U = fmaxf(U, c[p * W + 2]);
    }
    float S = 0.f;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const float mp = c[p * W + 0];
        S += (mp == neg_inf()) ? 0.f : c[p * W + 1] * exp2f((mp - M) * sl2);
    }
    float* out = part + ((size_t)grow * nsplit + split) * kPartStride;
    int ptr[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) ptr[p] = 0;
    int cnt = 0;
    for (int e = 0; e <= kKeep; ++e) {
        float bv = neg_inf();
        int bi = -1, bp = -1;
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            if (ptr[p] < kLane) {
                const float v = c[p * W + 3 + ptr[p]];
                const int i = __float_as_int(c[p * W + 3 + kLane + ptr[p]]);
                if (i >= 0 && (bp < 0 || better(v, i, bv, bi))) {
                    bv = v;
                    bi = i;
                    bp = p;
                }
            }
        }
        if (bp < 0) break;
        if (e == kKeep) {
            U = fmaxf(U, bv);
            break;
        }
#pragma unroll
        for (int p = 0; p < 8; ++p) ptr[p] += (p == bp) ? 1 : 0;
        out[4 + e] = bv;
        out[4 + kKeep + e] = __int_as_float(bi);
        ++cnt;
    }
    for (int e = cnt; e < kKeep; ++e) {
        out[4 + e] = neg_inf();
        out[4 + kKeep + e] = __int_as_float(-1);
    }
    out[0] = M;
    out[1] = S;
    out[2] = U;
    out[3] = __int_as_float(cnt);
}

// LM head: online log-sum-exp and a top-kLane list per lane and row, merged
// per workgroup into a (row, slice) partial of kKeep entries; the slice is the
// workgroup's chunk of the vocabulary.
//
// The partial's `bound` is an upper bound on every logit of the slice that is
// not in its list: a lane drops only values no larger than its kLane-th entry,
// and the workgroup merge drops only values no larger than the (kKeep+1)-th
// entry of the union.  The merge kernel uses it to prove the global top-k
// exact, or to re-evaluate the slice when it cannot.
template <int WM, int NT>
struct EpiLmHead {
    float* part;     // [R, nchunks, kPartStride]
    int V;
    float sl2;       // inv_temperature * log2(e)
    static constexpr int MERGE_WORDS = 3 + 2 * kLane;
    static constexpr int MERGE_BYTES = 32 * NT * 8 * MERGE_WORDS * 4;

    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const WorkItem& it, int wave, int lane,
                                          unsigned char* smem, const GemmShape& sh) {
        float* cm = reinterpret_cast<float*>(smem);   // [32*NT rows][8 contributors][MERGE_WORDS]
        const int q = wave * 2 + (lane >> 5);
        int vbase[WM];
        bool tv[WM];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = it.t0 + wave * WM + mt;
            tv[mt] = tile < it.t1;
            vbase[mt] = tile * 32 + 4 * (lane >> 5);
        }
        int seen = 0;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int j = 0; j < 16; ++j) seen += (tv[mt] && vbase[mt] + 8 * (j >> 2) + (j & 3) < V) ? 1 : 0;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            float m = neg_inf();
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const bool ok = tv[mt] && vbase[mt] + 8 * (j >> 2) + (j & 3) < V;
                    m = ok ? fmaxf(m, acc[mt][nt][j]) : m;
                }
            float s = 0.f;
            float lv[kLane];
            int li[kLane];
#pragma unroll
            for (int e = 0; e < kLane; ++e) {
                lv[e] = neg_inf();
                li[e] = -1;
            }
            // running top-kLane, visited in increasing token id so that equal
            // values keep the smaller id first
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int v = vbase[mt] + 8 * (j >> 2) + (j & 3);
                    const bool ok = tv[mt] && v < V;
                    float cv = acc[mt][nt][j];
                    s += ok ? exp2f((cv - m) * sl2) : 0.f;
                    if (ok && cv > lv[kLane - 1]) {
                        int ci = v;
#pragma unroll
                        for (int e = 0; e < kLane; ++e) {
                            const bool sw = cv > lv[e];
                            const float tvv = sw ? lv[e] : cv;
                            const int tii = sw ? li[e] : ci;
                            lv[e] = sw ? cv : lv[e];
                            li[e] = sw ? ci : li[e];
                            cv = tvv;
                            ci = tii;
                        }
                    }
                }
            float* c = cm + ((nt * 32 + (lane & 31)) * 8 + q) * MERGE_WORDS;
            c[0] = m;
            c[1] = seen > 0 ? s : 0.f;
            c[2] = seen > kLane ? lv[kLane - 1] : neg_inf();
#pragma unroll
            for (int e = 0; e < kLane; ++e) {
                c[3 + e] = lv[e];
                c[3 + kLane + e] = __int_as_float(li[e]);
            }
        }
        __syncthreads();
        lm_merge_contributors(cm, 32 * NT, it.row0, it.chunk, sh.nchunks, sh.R, sl2, part);
    }
};

// Split-K: each workgroup stores its accumulators, and the last of the nkp
// workgroups of a (chunk, row block) sums them in k-part order (so the result
// does not depend on arrival order) and runs the real epilogue.  The counters
// are zeroed before the first product of every call and reset by their last
// user.
template <int WM, int NT, class Inner>
struct EpiSplitK {
    Inner inner;
    float* partial;   // [nchunks * nrb][nkp][PART_FLOATS]
    int* counter;     // [nchunks * nrb]

    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const WorkItem& it, int wave, int lane,
                                          unsigned char* smem, const GemmShape& sh) {
        if (sh.nkp == 1) {
            inner.apply(acc, it, wave, lane, sh);
            return;
        }
        constexpr int PF = GemmTraits<WM, NT>::PART_FLOATS;
        const int slotid = it.chunk * sh.nrb + it.rb;
        float* base = partial + (size_t)slotid * sh.nkp * PF;
        auto idx = [&](int mt, int nt, int j4) {
            return ((((wave * WM + mt) * NT + nt) * 4 + j4) * 64 + lane) * 4;
        };
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4)
                    *reinterpret_cast<float4*>(base + (size_t)it.kp * PF + idx(mt, nt, j4)) =
                        float4{acc[mt][nt][4 * j4], acc[mt][nt][4 * j4 + 1], acc[mt][nt][4 * j4 + 2],
                               acc[mt][nt][4 * j4 + 3]};
        __threadfence();
        __syncthreads();
        int* flag = reinterpret_cast<int*>(smem);
        if (threadIdx.x == 0) flag[0] = (atomicAdd(counter + slotid, 1) == sh.nkp - 1) ? 1 : 0;
        __syncthreads();
        if (flag[0] == 0) return;
        __threadfence();
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) {
                    float4 sum = float4{0.f, 0.f, 0.f, 0.f};
                    for (int p = 0; p < sh.nkp; ++p) {
                        const float4 v = *reinterpret_cast<const float4*>(base + (size_t)p * PF + idx(mt, nt, j4));
                        sum.x += v.x;
                        sum.y += v.y;
                        sum.z += v.z;
                        sum.w += v.w;
                    }
                    acc[mt][nt][4 * j4] = sum.x;
                    acc[mt][nt][4 * j4 + 1] = sum.y;
                    acc[mt][nt][4 * j4 + 2] = sum.z;
                    acc[mt][nt][4 * j4 + 3] = sum.w;
                }
        if (threadIdx.x == 0) counter[slotid] = 0;
        inner.apply(acc, it, wave, lane, sh);
    }
};

// SwiGLU activation: a[r, i] = bf16( silu(g) * u ).
template <int WM, int NT>
struct EpiSwiGLU {
    uint16_t* out;   // [R, I]
    int I;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const WorkItem& it, int wave, int lane,
                                          const GemmShape& sh) {
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
                    uint32_t packed[2];
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        uint32_t lo, hi;
                        {
                            const float g = acc[mt][nt][4 * jg + 2 * q];
                            const float u = acc[mt][nt][4 * jg + 2 * q + 8];
                            lo = f32_to_bf16_bits(g / (1.0f + __expf(-g)) * u);
                        }
                        {
                            const float g = acc[mt][nt][4 * jg + 2 * q + 1];
                            const float u = acc[mt][nt][4 * jg + 2 * q + 9];
                            hi = f32_to_bf16_bits(g / (1.0f + __expf(-g)) * u);
                        }
                        packed[q] = lo | (hi << 16);
                    }
                    *reinterpret_cast<uint2*>(out + (size_t)r * I + i) = uint2{packed[0], packed[1]};
                }
            }
        }
    }
};

// Residual: h'[r, n] = bf16( h[seq, depth-1, n] + y[r, n] ).
template <int WM, int NT>
struct EpiResidual {
    uint16_t* out;        // [R, d]
    const uint16_t* h;    // [b, gamma, d]
    int d, Rs, gamma, M;
    __device__ __forceinline__ void apply(f32x16 (&acc)[WM][NT], const WorkItem& it, int wave, int lane,
                                          const GemmShape& sh) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = it.row0 + nt * 32 + (lane & 31);
            if (r >= sh.R) continue;
            const int s = r / Rs;
            const int rl = r - s * Rs;
            const int depth = rl == 0 ? 1 : 2 + (rl - 1) / M;
            const uint16_t* hrow = h + (size_t)(s * gamma + depth - 1) * d;
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
                    const uint32_t o0 = f32_to_bf16_bits(h0 + acc[mt][nt][4 * jg + 0]);
                    const uint32_t o1 = f32_to_bf16_bits(h1 + acc[mt][nt][4 * jg + 1]);
                    const uint32_t o2 = f32_to_bf16_bits(h2 + acc[mt][nt][4 * jg + 2]);
                    const uint32_t o3 = f32_to_bf16_bits(h3 + acc[mt][nt][4 * jg + 3]);
                    *reinterpret_cast<uint2*>(out + (size_t)r * d + n) = uint2{o0 | (o1 << 16), o2 | (o3 << 16)};
                }
            }
        }
    }
};

}  // namespace tf

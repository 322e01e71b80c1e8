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
// Work decomposition: the weight tiles are cut into `nsplit` contiguous slices
// balanced to within one tile; a workgroup (4 waves) owns one slice and one
// block of 32*NT activation rows and walks its slice in chunks of 4*WM tiles
// (WM tiles per wave).  Per 64-wide k-chunk the activation tile [32*NT x 64]
// is staged in LDS (double buffered, rows padded to 144 B so the 16-byte
// fragment reads are bank-conflict free) while each wave loads its own weight
// fragments straight into VGPRs one k-chunk ahead of the MFMAs.
#pragma once

#include "common.hpp"

namespace tf {

struct GemmShape {
    int R;        // activation rows
    int K;        // reduction length (multiple of 16)
    int ntiles;   // 32-row weight tiles
    int nsplit;   // weight slices (workgroups per activation-row block)
    int nrb;      // activation-row blocks
};

// Workgroups are dispatched round-robin over the 8 XCDs of an MI355X.
// Renumber them so consecutive logical ids share an XCD (and its L2): the
// row blocks of one weight slice then read the same weight tiles through the
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
    static constexpr int CHUNK = 4 * WM;         // weight tiles per workgroup step
};

template <int WM, int NT, class WSrc, class XSrc, class Epi>
__device__ __forceinline__ void stream_gemm_body(const WSrc& wsrc, const XSrc& xsrc, Epi& epi,
                                                 const GemmShape& sh, unsigned char* smem) {
    using T = GemmTraits<WM, NT>;
    constexpr int TR = T::TR, KC = T::KC, LDSW = T::LDSW;
    uint16_t* xs = reinterpret_cast<uint16_t*>(smem);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int split = L / sh.nrb;
    const int rb = L - split * sh.nrb;
    const int row0 = rb * TR;
    const int t0 = (int)(((long long)split * sh.ntiles) / sh.nsplit);
    const int t1 = (int)(((long long)(split + 1) * sh.ntiles) / sh.nsplit);
    const int nk = (sh.K + KC - 1) / KC;

    typename Epi::State st;
    epi.init(st);

    for (int ct = t0; ct < t1; ct += T::CHUNK) {
        const uint16_t* wp[WM];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = ct + wave * WM + mt;
            wp[mt] = (tile < t1) ? wsrc.row(tile, lane & 31) : nullptr;
        }
        f32x16 acc[WM][NT];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int j = 0; j < 16; ++j) acc[mt][nt][j] = 0.f;

        auto load_x = [&](u32x4 (&xr)[NT], int kc) {
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                const int p = tid + 256 * i;
                const int r = p >> 3;
                const int k = kc * KC + (p & 7) * 8;
                const int gr = row0 + r;
                if (gr < sh.R && k < sh.K)
                    xr[i] = *reinterpret_cast<const u32x4*>(xsrc.ptr(gr, k));
                else
                    xr[i] = u32x4{0u, 0u, 0u, 0u};
            }
        };
        auto store_x = [&](const u32x4 (&xr)[NT], int buf) {
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                const int p = tid + 256 * i;
                *reinterpret_cast<u32x4*>(xs + buf * TR * LDSW + (p >> 3) * LDSW + (p & 7) * 8) = xr[i];
            }
        };
        auto load_w = [&](u32x4 (&w)[WM][4], int kc) {
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const int k = kc * KC + ks * 16 + (lane >> 5) * 8;
                    if (wp[mt] != nullptr && k < sh.K)
                        w[mt][ks] = *reinterpret_cast<const u32x4*>(wp[mt] + k);
                    else
                        w[mt][ks] = u32x4{0u, 0u, 0u, 0u};
                }
        };

        u32x4 xr[NT];
        u32x4 wa[WM][4];
        __syncthreads();  // every wave is done with the LDS tiles of the previous chunk
        load_x(xr, 0);
        load_w(wa, 0);
        store_x(xr, 0);
        for (int kc = 0; kc < nk; ++kc) {
            __syncthreads();  // tile kc visible; the other buffer is free
            u32x4 wn[WM][4];
            const bool more = kc + 1 < nk;
            if (more) {
                load_x(xr, kc + 1);
                load_w(wn, kc + 1);
            }
            const uint16_t* xb = xs + (kc & 1) * TR * LDSW;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                u32x4 bfr[NT];
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    bfr[nt] = *reinterpret_cast<const u32x4*>(
                        xb + (nt * 32 + (lane & 31)) * LDSW + ks * 16 + (lane >> 5) * 8);
#pragma unroll
                for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
                        acc[mt][nt] = mfma_32x32x16_bf16(wa[mt][ks], bfr[nt], acc[mt][nt]);
            }
            if (more) {
                store_x(xr, (kc + 1) & 1);
#pragma unroll
                for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks) wa[mt][ks] = wn[mt][ks];
            }
        }
        epi.chunk(st, acc, ct, t1, wave, lane, row0, sh);
    }
    __syncthreads();  // LDS tiles no longer needed: the epilogue may reuse them
    epi.finish(st, smem, split, row0, wave, lane, sh);
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


// Merge the 8 contributor lists of each activation row (written to `cm` as
// [rows][8][3 + 2*kLane] = max, sum, bound, values, ids) into the row's
// (row, slice) partial.  One thread per row.
__device__ inline void lm_merge_contributors(const float* cm, int rows, int row0, int split, float sl2,
                                             float* part, const GemmShape& sh) {
    constexpr int W = 3 + 2 * kLane;
    const int tid = threadIdx.x;
    if (tid >= rows) return;
    const int grow = row0 + tid;
    if (grow >= sh.R) return;
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
    float* out = part + ((size_t)grow * sh.nsplit + split) * kPartStride;
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

// ------------------------------------------------------------------ epilogues

// SwiGLU activation: a[r, i] = bf16( silu(g) * u ).
template <int WM, int NT>
struct EpiSwiGLU {
    uint16_t* out;   // [R, I]
    int I;
    struct State {};
    __device__ void init(State&) {}
    __device__ __forceinline__ void chunk(State&, f32x16 (&acc)[WM][NT], int ct, int t1, int wave,
                                          int lane, int row0, const GemmShape& sh) {
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = ct + wave * WM + mt;
            if (tile >= t1) continue;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = row0 + nt * 32 + (lane & 31);
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
    __device__ void finish(State&, unsigned char*, int, int, int, int, const GemmShape&) {}
};

// Residual: h'[r, n] = bf16( h[seq, depth-1, n] + y[r, n] ).
template <int WM, int NT>
struct EpiResidual {
    uint16_t* out;        // [R, d]
    const uint16_t* h;    // [b, gamma, d]
    int d, Rs, gamma, M;
    struct State {};
    __device__ void init(State&) {}
    __device__ __forceinline__ void chunk(State&, f32x16 (&acc)[WM][NT], int ct, int t1, int wave,
                                          int lane, int row0, const GemmShape& sh) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = row0 + nt * 32 + (lane & 31);
            if (r >= sh.R) continue;
            const int s = r / Rs;
            const int rl = r - s * Rs;
            const int depth = rl == 0 ? 1 : 2 + (rl - 1) / M;
            const uint16_t* hrow = h + (size_t)(s * gamma + depth - 1) * d;
#pragma unroll
            for (int mt = 0; mt < WM; ++mt) {
                const int tile = ct + wave * WM + mt;
                if (tile >= t1) continue;
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
    __device__ void finish(State&, unsigned char*, int, int, int, int, const GemmShape&) {}
};

// LM head: online log-sum-exp and a running top-kLane list per lane and row,
// merged per workgroup into a (row, slice) partial of kKeep entries.
//
// The partial's `bound` is an upper bound on every logit of the slice that is
// not in its list: a lane drops only values no larger than its kLane-th entry,
// and the workgroup merge drops only values no larger than the (kKeep+1)-th
// entry of the union.  The merge kernel uses it to prove the global top-k
// exact, or to re-evaluate the slice when it cannot.
template <int WM, int NT>
struct EpiLmHead {
    float* part;     // [R, nsplit, kPartStride]
    int V;
    float sl2;       // inv_temperature * log2(e)
    struct State {
        float m[NT], s[NT];
        float lv[NT][kLane];
        int li[NT][kLane];
        int seen;
    };
    static constexpr int MERGE_WORDS = 3 + 2 * kLane;
    static constexpr int MERGE_BYTES = 32 * NT * 8 * MERGE_WORDS * 4;

    __device__ void init(State& st) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            st.m[nt] = neg_inf();
            st.s[nt] = 0.f;
#pragma unroll
            for (int q = 0; q < kLane; ++q) {
                st.lv[nt][q] = neg_inf();
                st.li[nt][q] = -1;
            }
        }
        st.seen = 0;
    }

    __device__ __forceinline__ void chunk(State& st, f32x16 (&acc)[WM][NT], int ct, int t1, int wave,
                                          int lane, int, const GemmShape&) {
        int vbase[WM];
        bool tv[WM];
#pragma unroll
        for (int mt = 0; mt < WM; ++mt) {
            const int tile = ct + wave * WM + mt;
            tv[mt] = tile < t1;
            vbase[mt] = tile * 32 + 4 * (lane >> 5);
        }
        int nvalid = 0;
#pragma unroll
        for (int mt = 0; mt < WM; ++mt)
#pragma unroll
            for (int j = 0; j < 16; ++j)
                nvalid += (tv[mt] && vbase[mt] + 8 * (j >> 2) + (j & 3) < V) ? 1 : 0;
        st.seen += nvalid;
        if (nvalid == 0) return;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            float cm = neg_inf();
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const bool ok = tv[mt] && vbase[mt] + 8 * (j >> 2) + (j & 3) < V;
                    cm = ok ? fmaxf(cm, acc[mt][nt][j]) : cm;
                }
            const float mn = fmaxf(st.m[nt], cm);
            float sum = st.s[nt] * exp2f((st.m[nt] - mn) * sl2);
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const bool ok = tv[mt] && vbase[mt] + 8 * (j >> 2) + (j & 3) < V;
                    sum += ok ? exp2f((acc[mt][nt][j] - mn) * sl2) : 0.f;
                }
            st.s[nt] = sum;
            st.m[nt] = mn;
            // running top-kLane, visited in increasing token id so that equal
            // values keep the smaller id first
#pragma unroll
            for (int mt = 0; mt < WM; ++mt)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int v = vbase[mt] + 8 * (j >> 2) + (j & 3);
                    float cv = acc[mt][nt][j];
                    const bool ok = tv[mt] && v < V;
                    if (ok && cv > st.lv[nt][kLane - 1]) {
                        int ci = v;
#pragma unroll
                        for (int q = 0; q < kLane; ++q) {
                            const bool sw = cv > st.lv[nt][q];
                            const float tvv = sw ? st.lv[nt][q] : cv;
                            const int tii = sw ? st.li[nt][q] : ci;
                            st.lv[nt][q] = sw ? cv : st.lv[nt][q];
                            st.li[nt][q] = sw ? ci : st.li[nt][q];
                            cv = tvv;
                            ci = tii;
                        }
                    }
                }
        }
    }

    __device__ void finish(State& st, unsigned char* smem, int split, int row0, int wave, int lane,
                           const GemmShape& sh) {
        float* cm = reinterpret_cast<float*>(smem);   // [32*NT rows][8 contributors][MERGE_WORDS]
        const int q = wave * 2 + (lane >> 5);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = nt * 32 + (lane & 31);
            float* c = cm + (r * 8 + q) * MERGE_WORDS;
            c[0] = st.m[nt];
            c[1] = st.s[nt];
            c[2] = st.seen > kLane ? st.lv[nt][kLane - 1] : neg_inf();
#pragma unroll
            for (int e = 0; e < kLane; ++e) {
                c[3 + e] = st.lv[nt][e];
                c[3 + kLane + e] = __int_as_float(st.li[nt][e]);
            }
        }
        __syncthreads();
        lm_merge_contributors(cm, 32 * NT, row0, split, sl2, part, sh);
    }
};

}  // namespace tf

// Host-side check of the work split of the one-row-block approximator
// products (work.hpp, plan.hpp): for every plan the path can build over a
// grid of widths, intermediate sizes and row counts, the workgroup ranges
// tile the units without gaps or empty ranges, unit_owner agrees with
// unit_start, the per-workgroup costs are balanced to within one chunk, a
// workgroup holds at most two cut items, and the closed-form description of
// each cut item's pieces (cut_pieces: first piece, count, partial-sum slots,
// the pieces of each phase) equals the one found by walking the item's units.
// Prints "<plans> plans, <items> items, <failures> failures" and exits 1 on
// any failure.
#include <cstdio>
#include <vector>

#include "plan.hpp"

using namespace tf;

static int fails = 0;
#define CHECK(c, ...)                        \
    do {                                     \
        if (!(c)) {                          \
            if (fails++ < 20) {              \
                std::printf("FAIL %s: ", #c); \
                std::printf(__VA_ARGS__);    \
                std::printf("\n");           \
            }                                \
        }                                    \
    } while (0)

static int owner_of(const CostSplit& s, int u) { return unit_owner(s, u / s.nk, u % s.nk); }

static void check(int rows, int ntiles, int nkh, int nke, int TG, long long& nitems) {
    const MlpDmaPlan p = mlp_dma_plan(rows, ntiles, nkh, nke, TG);
    if (!mlp_dma_plan_ok(p)) return;   // the path is not taken for this plan
    const CostSplit s = cost_split(p.items, p.nkh, p.nke, p.wh, p.we, p.G);
    const int U = p.items * s.nk;
    CHECK(unit_start(s, 0) == 0, "first range starts at 0");
    CHECK(unit_start(s, p.G) == U, "last range ends at %d, not %d", unit_start(s, p.G), U);
    long long cmax = 0, cmin = 1LL << 60;
    for (int g = 0; g < p.G; ++g) {
        const int a = unit_start(s, g), b = unit_start(s, g + 1);
        CHECK(a < b, "empty range g=%d (rows %d tiles %d nkh %d nke %d)", g, rows, ntiles, nkh, nke);
        for (int u = a; u < b; ++u) CHECK(owner_of(s, u) == g, "owner of unit %d is %d, not %d", u, owner_of(s, u), g);
        const long long cb = b < U ? split_cost(s, b / s.nk, b % s.nk) : s.ctot;
        const long long c = cb - split_cost(s, a / s.nk, a % s.nk);
        cmax = c > cmax ? c : cmax;
        cmin = c < cmin ? c : cmin;
        const int first = a / s.nk, last = (b - 1) / s.nk;
        int ncut = 0;
        for (int it = first; it <= last; ++it)
            if (owner_of(s, it * s.nk) != owner_of(s, it * s.nk + s.nk - 1)) {
                ++ncut;
                CHECK(piece_slot(s, g, it) == 2 * g + (it == first ? 0 : 1), "slot of g=%d item %d", g, it);
            }
        CHECK(ncut <= 2, "g=%d holds %d cut items", g, ncut);
    }
    CHECK(cmax - cmin <= 2 * (s.wh > s.we ? s.wh : s.we), "costs %lld..%lld", cmin, cmax);
    for (int it = 0; it < p.items; ++it) {
        const CutPieces cp = cut_pieces(s, it);
        std::vector<int> gs;   // the workgroups owning the item's units, in order
        for (int c = 0; c < s.nk; ++c) {
            const int o = unit_owner(s, it, c);
            if (gs.empty() || gs.back() != o) gs.push_back(o);
        }
        CHECK(cp.gfirst == gs[0] && cp.npieces == (int)gs.size(), "pieces of item %d", it);
        const int ib = it * s.nk;
        for (int i = 0; i < (int)gs.size(); ++i) {
            const int g = gs[i];
            CHECK(g == cp.gfirst + i, "pieces of item %d are consecutive workgroups", it);
            CHECK(cp.slot(i) == piece_slot(s, g, it), "slot of piece %d of item %d", i, it);
            int a = unit_start(s, g), b = unit_start(s, g + 1);
            a = a > ib ? a : ib;
            b = b < ib + s.nk ? b : ib + s.nk;
            CHECK((a < ib + nkh) == (i < cp.ph1), "h pieces of item %d", it);
            CHECK((b > ib + nkh) == (i >= cp.pe0), "e pieces of item %d", it);
        }
        ++nitems;
    }
}

int main() {
    long long nplans = 0, nitems = 0;
    const int ds[] = {64, 192, 640, 1024, 1088, 2048, 2560, 4096, 5120, 8192, 16384};
    const int Is[] = {64, 256, 1088, 1536, 3072, 4096, 6144, 9728, 12288, 28672};
    const int rowsv[] = {1, 16, 31, 32, 33, 61, 64, 65, 100, 121, 128, 129, 200, 241, 256};
    for (int d : ds)
        for (int I : Is)
            for (int rows : rowsv)
                for (int npre = 1; npre <= 2; ++npre) {
                    check(rows, cdiv(I, 16), d / 64, npre * d / 64, TF_MLP_DMA_TG_IN, nitems);   // gate/up
                    check(rows, cdiv(I, 32), d / 64, npre * d / 64, TF_MLP_DMA_TG_IN, nitems);   // SiLU gate
                    check(rows, cdiv(d, 32), 0, I / 64, TF_MLP_DMA_TG_DOWN, nitems);            // down
                    check(rows, cdiv(d, 32), d / 64, d / 64, TF_MLP_DMA_TG_IN, nitems);          // linear
                    nplans += 4;
                }
    std::printf("%lld plans, %lld items, %d failures\n", nplans, nitems, fails);
    return fails != 0;
}

// Host check of the edge kernels' batched AllToAll costing (csrc/taps_device.h,
// compiled for the host): every closure of every tops mask on n <= 8 binary
// levels, at every shard shift and node boundary, costed by the closed forms
// (byte dot products against the shard-fraction tables) and axis by axis from
// the definitions (Eq. 10 and Eq. 14: an axis of width w moves all but 2^-w of
// the shard, across the inter-node link when its groups cross a node, with the
// group count of Algorithm 3; the axis straddling the node boundary sends only
// its members outside the node), for the two-class model and for hierarchies
// of link classes.  Prints "N closures, 0 mismatches".
#include <cstdio>
#include <cstdlib>
#include <cstdint>
#include <cstring>

#include "taps_device.h"

namespace {

uint32_t rng_state = 12345u;
uint32_t rnd() {
    rng_state = rng_state * 1664525u + 1013904223u;
    return rng_state >> 8;
}

// Widths of the unified axes by tops mask, from the definition (an axis runs
// from one above the next lower top up to its own top).
uint32_t width_of(uint32_t tp, uint32_t t) {
    uint32_t lo = 0;
    for (uint32_t l = 0; l < t; ++l)
        if ((tp >> l) & 1u) lo = l + 1u;
    return t + 1u - lo;
}

// Two classes, axis by axis.
taps_fac two_class_reference(uint32_t tp, uint32_t x, uint32_t lam, uint32_t sh, uint32_t unused,
                             uint32_t n) {
    taps_fac c;
    taps_fac_zero(c);
    for (uint32_t t = 0; t < 8u; ++t) {
        if (!((x >> t) & 1u)) continue;
        const uint32_t w = width_of(tp, t), lo = t + 1u - w;
        const uint32_t V = (1u << sh) - (1u << (sh - w));
        c.vol += V;
        if (t < lam) {   // the group lies inside one node
            c.intra += V;
            continue;
        }
        if (lo < lam && lam < n) {   // straddles the node boundary: 2^(lam - lo) members inside
            const uint32_t kap = lam - lo;
            const uint32_t link = ((1u << w) - (1u << kap)) << (kap + sh - w);
            uint32_t used_below = 0;   // levels below lo that some dimension uses
            for (uint32_t l = 0; l < lo; ++l) used_below += ((unused >> l) & 1u) ? 0u : 1u;
            c.inter += link << used_below;
            c.ct += 1u << used_below;
            continue;
        }
        uint32_t used_below = 0;   // levels below lam that some dimension uses
        for (uint32_t l = 0; l < lam; ++l) used_below += ((unused >> l) & 1u) ? 0u : 1u;
        c.inter += V << used_below;
        c.ct += 1u << used_below;
    }
    return c;
}

bool same(const taps_fac &a, const taps_fac &b) {
    return a.vol == b.vol && a.intra == b.intra && a.inter == b.inter && a.ct == b.ct;
}

}  // namespace

int main() {
    const taps_width_table widths = taps_make_widths();
    const taps_a2a_table a2a = taps_make_a2a();
    const taps_expand_table ex = taps_make_expand();
    static taps_pair expand[256];
    for (uint32_t m = 0; m < 256u; ++m) expand[m] = taps_pair{ex.lo[m], ex.hi[m]};
    uint64_t closures = 0, bad = 0;

    // two classes: every n, lam, tops mask with the top level set, closure x of it
    for (uint32_t n = 1; n <= 8u; ++n) {
        for (uint32_t lam = 0; lam <= n; ++lam) {
            static taps_a2a_row rows[256];
            const uint32_t in_lo = lam >= 4u ? ~0u : (1u << (8u * lam)) - 1u;
            const uint32_t in_hi = lam <= 4u ? 0u : lam >= 8u ? ~0u : (1u << (8u * (lam - 4u))) - 1u;
            for (uint32_t m = 0; m < 256u; ++m)
                rows[m] = taps_a2a_row{a2a.lo[m], a2a.hi[m], a2a.lo[m] & in_lo, a2a.hi[m] & in_hi};
            const uint32_t full = (1u << n) - 1u, low = (1u << lam) - 1u;
            for (uint32_t tp = 1u << (n - 1u); tp <= full; ++tp) {
                if (!((tp >> (n - 1u)) & 1u)) continue;
                taps_lv L;
                L.tp = tp;
                L.wt = widths.v[tp];
                L.lo_s = taps_msb(((tp & low) << 1) | 1u);
                const bool st = lam >= 1u && lam < n && !((tp >> (lam - 1u)) & 1u);
                L.st = st ? 1u << taps_ctz((tp & ~low) | 0x100u) : 0u;
                for (uint32_t x = tp; ; x = (x - 1u) & tp) {   // every subset of the tops
                    for (uint32_t rep = 0; rep < 3u; ++rep) {
                        const uint32_t sh = 8u + rnd() % (n + 1u);
                        const uint32_t unused = rnd() & full;
                        taps_fac got;
                        taps_fac_zero(got);
                        taps_a2a_batch(got, x, L, lam, taps_below(lam), sh, unused, rows, expand);
                        const taps_fac want = two_class_reference(tp, x, lam, sh, unused, n);
                        ++closures;
                        if (!same(got, want)) {
                            if (bad < 5)
                                printf("two classes: n %u lam %u tops %02x x %02x sh %u unused %02x: "
                                       "%u %u %u %u against %u %u %u %u\n", n, lam, tp, x, sh, unused,
                                       got.vol, got.intra, got.inter, got.ct, want.vol, want.intra,
                                       want.inter, want.ct);
                            ++bad;
                        }
                    }
                    if (x == 0) break;
                }
            }
        }
    }

    // link classes: random hierarchies of 1-4 classes on n levels; the closed
    // form of the hierarchy model against its axis-by-axis costing
    for (uint32_t trial = 0; trial < 400u; ++trial) {
        const uint32_t n = 1u + rnd() % 8u;
        const uint32_t C = 1u + rnd() % 4u;
        taps_hier H;
        std::memset(&H, 0, sizeof(H));
        H.n_classes = C;
        uint32_t b[TAPS_D_MAX_CLASSES] = {0, 0, 0, 0};   // boundaries, non-decreasing
        for (uint32_t c = 0; c + 1u < C; ++c) b[c] = rnd() % (n + 1u);
        for (uint32_t c = 1; c + 1u < C; ++c)
            if (b[c] < b[c - 1u]) b[c] = b[c - 1u];
        for (uint32_t l = 0; l < 8u; ++l) {
            uint32_t cls = 0, beta = 0;
            for (uint32_t c = 0; c + 1u < C; ++c)
                if (b[c] <= l) {
                    ++cls;
                    beta = b[c];
                }
            H.cls_of_top |= cls << (4u * l);
            H.beta_of_top |= beta << (4u * l);
            H.levels_of_cls[cls] |= 1u << l;
            H.beta_of_cls[cls] = beta;
        }
        H.a2a_own = rnd() & 1u;
        static taps_pair cls_rows[256 * TAPS_D_MAX_CLASSES];
        for (uint32_t m = 0; m < 256u; ++m)
            for (uint32_t c = 0; c < TAPS_D_MAX_CLASSES; ++c) {
                const uint32_t lv = c < C ? H.levels_of_cls[c] & 0xFFu : 0u;
                cls_rows[m * TAPS_D_MAX_CLASSES + c] =
                    taps_pair{a2a.lo[m] & (ex.lo[lv] * 0xFFu), a2a.hi[m] & (ex.hi[lv] * 0xFFu)};
            }
        const taps_hier_model_t<TAPS_D_MAX_CLASSES> M{&H, 0, 0, false, cls_rows, expand};
        const uint32_t full = (1u << n) - 1u;
        for (uint32_t k = 0; k < 64u; ++k) {
            const uint32_t tp = ((rnd() & full) | (1u << (n - 1u))) & full;
            taps_lv L;
            L.tp = tp;
            L.wt = widths.v[tp];
            const uint32_t x = rnd() & tp, sh = 8u + rnd() % (n + 1u), unused = rnd() & full;
            taps_fach got, want;
            taps_fac_zero(got);
            taps_fac_zero(want);
            M.a2a(got, x, L, sh, unused);
            for (uint32_t r = x; r; r &= r - 1u) {   // axis by axis
                const uint32_t top = taps_ctz(r);
                const uint32_t w = width_of(tp, top), lo = top + 1u - w;
                const uint32_t V = (1u << sh) - (1u << (sh - w));
                const uint32_t cls = (H.cls_of_top >> (4u * top)) & 15u;
                want.vol += V;
                if (!cls) {
                    (H.a2a_own ? want.xa : want.x0) += V;
                    continue;
                }
                const uint32_t beta = (H.beta_of_top >> (4u * top)) & 15u;
                const uint32_t kap = beta > lo ? beta - lo : 0u;
                const uint32_t link = ((1u << w) - (1u << kap)) << (kap + sh - w);
                const uint32_t mlow = lo < beta ? lo : beta;
                uint32_t lct = 0;
                for (uint32_t l = 0; l < mlow; ++l) lct += ((unused >> l) & 1u) ? 0u : 1u;
                (cls == 1 ? want.x1 : cls == 2 ? want.x2 : want.x3) += link << lct;
                want.ct += 1u << lct;
            }
            ++closures;
            if (got.vol != want.vol || got.x0 != want.x0 || got.x1 != want.x1 || got.x2 != want.x2 ||
                got.x3 != want.x3 || got.xa != want.xa || got.ct != want.ct) {
                if (bad < 10)
                    printf("link classes: n %u C %u tops %02x x %02x sh %u: vol %u/%u x0 %u/%u x1 "
                           "%u/%u x2 %u/%u x3 %u/%u xa %u/%u ct %u/%u\n", n, C, tp, x, sh, got.vol,
                           want.vol, got.x0, want.x0, got.x1, want.x1, got.x2, want.x2, got.x3,
                           want.x3, got.xa, want.xa, got.ct, want.ct);
                ++bad;
            }
        }
    }
    printf("%llu closures, %llu mismatches\n", (unsigned long long)closures,
           (unsigned long long)bad);
    return bad != 0;
}

// taps_device.h -- per-item arithmetic of the TAPS cost tables on binary levels.
//
// Every device count here is a power of two, N = 2^n devices with L = 2^lam
// per node, so a device matrix is described by its binary levels 0..n-1
// (level 0 innermost; a device's rank bit l is its coordinate bit on level
// l; levels < lam lie inside one node).  A strategy gives each split op axis
// a contiguous run of levels; a tensor dimension inherits the run of its op
// axis.  All set operations of the cost model become bit operations on
// masks of at most 8 levels:
//
//   * intra-op AllReduce of a tensor (Eq. 5-7, Algorithm 2): the group spans
//     the levels G the tensor does not use; ct is 0 when G lies below lam,
//     else 2^(lam - |G below lam|);
//   * unification of two strategies' device matrices and tensor shapes
//     (Table 1): a least fixpoint over "cuts" (boundaries between adjacent
//     levels), where a cut inside one side's run of a dimension forces the
//     cut at the same bit of that dimension on the other side;
//   * the tensor maps become per-axis "positions" key = dim * 8 + bit, and
//     Algorithm 1's Infer* steps become operations on 64-bit position masks;
//   * AllGather / AllToAll group counts (Algorithm 3, the AllToAll
//     paragraph) and Eq. 9, 10, 14 volumes become shifts and popcounts.
//
// Volumes are integers in "nb" (bytes x N), which makes every per-device
// volume exact.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define TAPS_D_MAX_AXES 8
#define TAPS_D_MAX_RANK 8
#define TAPS_D_MAX_LEVELS 8
#define TAPS_D_NONE 0xFFu

// A strategy on binary levels: per op axis the lowest level of its run and
// the run's width (0 = not split), 4 bits each; per level the op axis that
// owns it, 4 bits each; and the strategy's cut mask (bit c set when levels
// c-1 and c belong to different op axes, 1 <= c < n).
struct taps_desc {
    uint32_t lo;     // nibble a: lowest level of op axis a
    uint32_t width;  // nibble a: log2(degree) of op axis a
    uint32_t owner;  // nibble l: op axis owning level l
    uint32_t cuts;
};

__host__ __device__ inline uint32_t taps_nib(uint32_t v, uint32_t k) { return (v >> (4u * k)) & 15u; }

__host__ __device__ inline uint32_t taps_popc(uint32_t v) { return (uint32_t)__builtin_popcount(v); }

__host__ __device__ inline uint32_t taps_ctz(uint32_t v) { return (uint32_t)__builtin_ctz(v); }

__host__ __device__ inline uint32_t taps_low_mask(uint32_t k) { return k >= 32u ? ~0u : ((1u << k) - 1u); }

// ---------------------------------------------------------------------------
// GenerateStrategySet in canonical order (Auxiliary Graph section, Table 3).
//
// Order: the exponent tuple (log2 degree per op axis, axis 0 most
// significant) ascending; within one exponent tuple the device-map tuple
// (position per split axis, in axis order) descending.  Counting is done
// with w(k, s, z) = the number of strategies that complete a prefix with z
// split axes so far, s levels still to hand out and k partitionable axes
// left: sum_j C(k, j) C(s-1, j-1) (z+j)!  (s = 0: z!).  With k = p, s = n,
// z = 0 this is the paper's count sum_i i! C(p,i) C(n-1,i-1).
// ---------------------------------------------------------------------------

__host__ __device__ inline uint64_t taps_binom(uint32_t a, uint32_t b) {
    if (b > a) return 0;
    uint64_t r = 1;
    for (uint32_t x = 1; x <= b; ++x) r = r * (a - b + x) / x;
    return r;
}

__host__ __device__ inline uint64_t taps_fact(uint32_t a) {
    uint64_t r = 1;
    for (uint32_t x = 2; x <= a; ++x) r *= x;
    return r;
}

__host__ __device__ inline uint64_t taps_completions(uint32_t k, uint32_t s, uint32_t z) {
    if (s == 0) return taps_fact(z);
    uint64_t tot = 0;
    uint32_t jmax = k < s ? k : s;
    for (uint32_t j = 1; j <= jmax; ++j)
        tot += taps_binom(k, j) * taps_binom(s - 1, j - 1) * taps_fact(z + j);
    return tot;
}

// Decodes candidate r (0 <= r < taps_completions(p, n, 0)) into per-axis
// exponents and device-map positions.  part: partitionable-axis mask.
// Returns false if r is out of range.
template <class W>
__host__ __device__ inline bool taps_unrank(uint32_t n_axes, uint32_t part, uint32_t n, uint64_t r,
                                            const W &w, uint32_t *expo, int32_t *pos) {
    uint32_t s = n, z = 0;
    for (uint32_t a = 0; a < n_axes; ++a) {
        expo[a] = 0;
        pos[a] = -1;
        if (!((part >> a) & 1u)) continue;
        uint32_t k = taps_popc(part >> (a + 1));
        bool placed = false;
        for (uint32_t e = 0; e <= s; ++e) {
            uint32_t z2 = z + (e > 0 ? 1u : 0u);
            uint64_t c = w(k, s - e, z2);
            if (r < c) {
                expo[a] = e;
                s -= e;
                z = z2;
                placed = true;
                break;
            }
            r -= c;
        }
        if (!placed) return false;
    }
    if (s != 0) return false;
    // r is now the rank of the position tuple among the z! orderings, in
    // descending order; decode the (z! - 1 - r)-th ascending permutation.
    uint64_t q = taps_fact(z) - 1 - r;
    uint32_t free_pos = taps_low_mask(z);
    uint32_t t = 0;
    for (uint32_t a = 0; a < n_axes; ++a) {
        if (expo[a] == 0) continue;
        uint64_t f = taps_fact(z - 1 - t);
        uint32_t idx = (uint32_t)(q / f);
        q -= (uint64_t)idx * f;
        uint32_t m = free_pos;
        for (uint32_t x = 0; x < idx; ++x) m &= m - 1;   // drop the idx lowest free positions
        uint32_t p = taps_ctz(m);
        free_pos &= ~(1u << p);
        pos[a] = (int32_t)p;
        ++t;
    }
    return true;
}

// Level runs of a strategy: the axis at position 0 owns the lowest levels.
// Positions outside 0..7 and runs past level 7 are ignored, so malformed
// input yields meaningless numbers but never an out-of-range index.
__host__ __device__ inline taps_desc taps_describe(uint32_t n_axes, const uint32_t *expo,
                                                   const int32_t *pos) {
    taps_desc d = {0u, 0u, 0u, 0u};
    uint32_t width_of_pos[TAPS_D_MAX_AXES];
#pragma unroll
    for (uint32_t q = 0; q < TAPS_D_MAX_AXES; ++q) width_of_pos[q] = 0;
    for (uint32_t a = 0; a < n_axes && a < TAPS_D_MAX_AXES; ++a)
        if (pos[a] >= 0 && pos[a] < (int32_t)TAPS_D_MAX_AXES)
            width_of_pos[pos[a]] = expo[a] & 15u;
    for (uint32_t a = 0; a < n_axes && a < TAPS_D_MAX_AXES; ++a) {
        if (pos[a] < 0 || pos[a] >= (int32_t)TAPS_D_MAX_AXES) continue;
        uint32_t lo = 0;
        for (uint32_t q = 0; q < (uint32_t)pos[a]; ++q) lo += width_of_pos[q];
        uint32_t w = expo[a] & 15u;
        if (lo >= TAPS_D_MAX_LEVELS) continue;
        d.lo |= lo << (4u * a);
        d.width |= w << (4u * a);
        for (uint32_t l = lo; l < lo + w && l < TAPS_D_MAX_LEVELS; ++l) d.owner |= a << (4u * l);
        if (lo > 0) d.cuts |= 1u << lo;
    }
    return d;
}

// ---------------------------------------------------------------------------
// Records
// ---------------------------------------------------------------------------

struct taps_acc {
    uint64_t vol, intra, inter;
    uint32_t n_coll, n_inter, sum_ct;
};

__host__ __device__ inline void taps_acc_zero(taps_acc &c) {
    c.vol = c.intra = c.inter = 0;
    c.n_coll = c.n_inter = c.sum_ct = 0;
}

__host__ __device__ inline uint32_t taps_meta(uint32_t cand, const taps_acc &c) {
    return cand | (c.n_coll << 2) | (c.n_inter << 7) | (c.sum_ct << 12);
}

// ---------------------------------------------------------------------------
// Intra-op cost (Eq. 5-8 with Algorithm 2 and Eq. 11-12): one ring AllReduce
// over the levels a tensor does not use.  bytes = elements x dtype bytes.
// ---------------------------------------------------------------------------
__host__ __device__ inline void taps_allreduce(taps_acc &c, uint32_t missing, uint64_t bytes,
                                               uint32_t lam) {
    if (!missing) return;
    uint32_t lg = taps_popc(missing);
    uint64_t V = ((bytes << lg) - bytes) << 1;   // 2 (g - 1) |tensor| bytes, in nb
    c.vol += V;
    c.n_coll += 1;
    if ((missing >> lam) == 0) {
        c.intra += V;
        return;
    }
    uint32_t lct = lam - taps_popc(missing & taps_low_mask(lam));
    c.inter += V << lct;
    c.n_inter += 1;
    c.sum_ct += 1u << lct;
}

// ---------------------------------------------------------------------------
// A collective of the redistribution along the unified axis [lo, lo + w):
// an AllGather (Eq. 9) or an AllToAll (Eq. 10, Eq. 14), with ct from the
// levels no tensor dimension uses at that point (Algorithm 3): groups that
// hold the same data inside a node share one inter-node transfer.
// S = per-device data size before the collective, in nb.
// ---------------------------------------------------------------------------
__host__ __device__ inline void taps_collective(taps_acc &c, bool a2a, uint32_t lo, uint32_t w,
                                                uint64_t S, uint32_t unused, uint32_t lam) {
    uint64_t V = a2a ? S - (S >> w) : (S << w) - S;
    c.vol += V;
    c.n_coll += 1;
    if (lo + w <= lam) {
        c.intra += V;
        return;
    }
    uint32_t m = lo < lam ? lo : lam;
    uint32_t lct = m - taps_popc(unused & taps_low_mask(m));
    uint64_t link = V;
    if (a2a) {
        uint32_t kap = lam > lo ? lam - lo : 0u;   // log2 of group members inside a node
        link = ((S >> w) << kap) * (uint64_t)((1u << w) - (1u << kap));
    }
    c.inter += link << lct;
    c.n_inter += 1;
    c.sum_ct += 1u << lct;
}

// ---------------------------------------------------------------------------
// One edge entry: the tensor of rank R leaves its producer under strategy P
// and enters its consumer under strategy C.
//
// Inputs per tensor dimension d: the level run [plo[d], plo[d]+pw[d]) of its
// producer axis and [clo[d], clo[d]+cw[d]) of its consumer axis (width 0 =
// whole).  pcuts / ccuts: the strategies' cut masks.  tbytes = |T| x dtype.
// ---------------------------------------------------------------------------

struct taps_edge_problem {
    uint32_t rank, n, lam;
    uint32_t plo[TAPS_D_MAX_RANK], pw[TAPS_D_MAX_RANK];
    uint32_t clo[TAPS_D_MAX_RANK], cw[TAPS_D_MAX_RANK];
    uint32_t pcuts, ccuts;
    uint64_t tbytes;
};

// Per unified axis (indexed by its lowest level) after unification.
struct taps_axes {
    uint32_t start;                      // bit l: a unified axis starts at level l
    uint32_t has_src, has_dst, home;     // axis sets (bit = its start level)
    uint32_t width[TAPS_D_MAX_LEVELS];
    uint32_t skey[TAPS_D_MAX_LEVELS];    // producer position dim*8+bit, or NONE
    uint32_t dkey[TAPS_D_MAX_LEVELS];    // consumer position, or NONE
    uint64_t tgt;                        // positions the consumer map uses
    uint64_t occ0;                       // positions the producer map uses
    uint32_t used0;                      // levels the producer map uses
    uint64_t S0;                         // producer shard, nb
};

__host__ __device__ inline uint64_t taps_bit64(uint32_t k) { return (uint64_t)1 << k; }

// Unification (Table 1) as a least fixpoint over cuts, then the position of
// every unified axis in the unified producer and consumer tensor maps.
__host__ __device__ inline void taps_unify(const taps_edge_problem &p, taps_axes &ax) {
    const uint32_t inner = taps_low_mask(p.n) & ~1u;   // valid cut bits 1..n-1
    uint32_t C = (p.pcuts | p.ccuts) & inner;
    for (uint32_t it = 0; it < TAPS_D_MAX_LEVELS; ++it) {
        uint32_t before = C;
#pragma unroll
        for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
            if (d >= p.rank) break;
            uint32_t m = p.pw[d] < p.cw[d] ? p.pw[d] : p.cw[d];
            if (m < 2) continue;
            uint32_t phi = p.plo[d] + p.pw[d], chi = p.clo[d] + p.cw[d];
            uint32_t win = taps_low_mask(m - 1);
            uint32_t pwin = win << (phi - m + 1), cwin = win << (chi - m + 1);
            if (chi >= phi) {
                uint32_t sh = chi - phi;
                C |= ((C & pwin) << sh) | ((C & cwin) >> sh);
            } else {
                uint32_t sh = phi - chi;
                C |= ((C & pwin) >> sh) | ((C & cwin) << sh);
            }
        }
        if (C == before) break;
    }
    ax.start = (C | 1u) & taps_low_mask(p.n);
    if (p.n == 0) ax.start = 0;
    ax.has_src = ax.has_dst = ax.home = 0;
    ax.tgt = ax.occ0 = 0;
    ax.used0 = 0;
    uint32_t usedw = 0;
#pragma unroll
    for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
        ax.skey[l] = TAPS_D_NONE;
        ax.dkey[l] = TAPS_D_NONE;
        ax.width[l] = 0;
        if (!((ax.start >> l) & 1u)) continue;
        uint32_t above = ax.start & ~taps_low_mask(l + 1);
        uint32_t hi = above ? taps_ctz(above) : p.n;
        ax.width[l] = hi - l;
#pragma unroll
        for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
            if (d >= p.rank) break;
            if (p.pw[d] && l >= p.plo[d] && l < p.plo[d] + p.pw[d])
                ax.skey[l] = d * 8u + (p.plo[d] + p.pw[d] - hi);
            if (p.cw[d] && l >= p.clo[d] && l < p.clo[d] + p.cw[d])
                ax.dkey[l] = d * 8u + (p.clo[d] + p.cw[d] - hi);
        }
        if (ax.skey[l] != TAPS_D_NONE) {
            ax.has_src |= 1u << l;
            ax.occ0 |= taps_bit64(ax.skey[l]);
            ax.used0 |= taps_low_mask(hi) & ~taps_low_mask(l);
        }
        if (ax.dkey[l] != TAPS_D_NONE) {
            ax.has_dst |= 1u << l;
            ax.tgt |= taps_bit64(ax.dkey[l]);
        }
        if (ax.skey[l] != TAPS_D_NONE && ax.skey[l] == ax.dkey[l]) ax.home |= 1u << l;
    }
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d)
        if (d < p.rank) usedw += p.pw[d];
    ax.S0 = p.tbytes << (p.n - usedw);
}

__host__ __device__ inline uint32_t taps_levels(uint32_t lo, uint32_t w) {
    return taps_low_mask(lo + w) & ~taps_low_mask(lo);
}

// Algorithm 1 (use_a2a) or its variant without AllToAll ("rearrange").
// Returns the number of AllToAlls issued; *ok = false if the loop did not
// settle (cannot happen for a unified problem).
__host__ __device__ inline uint32_t taps_alg1(const taps_axes &ax, uint32_t lam, bool use_a2a,
                                              taps_acc &c, bool *ok) {
    uint32_t at_src = ax.has_src & ~ax.home;    // mapped by the producer, not at its target
    uint32_t at_dst = ax.home;                  // at its target position
    uint64_t occ = ax.occ0;
    uint32_t unused = ~ax.used0;
    uint64_t S = ax.S0;
    uint32_t n_a2a = 0;
    *ok = true;
    for (uint32_t guard = 0;; ++guard) {
        if (at_src == 0 && at_dst == ax.has_dst) break;
        if (guard > 4 * TAPS_D_MAX_LEVELS) {
            *ok = false;
            break;
        }
        bool sliced;
        do {
            // InferSlice: every target position that is free and whose axis
            // no dimension uses yet
            uint32_t sl = 0;
#pragma unroll
            for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
                uint32_t b = 1u << l;
                if ((ax.has_dst & b) && !((at_src | at_dst) & b) && !((occ >> ax.dkey[l]) & 1u))
                    sl |= b;
            }
#pragma unroll
            for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
                if (!((sl >> l) & 1u)) continue;
                occ |= taps_bit64(ax.dkey[l]);
                S >>= ax.width[l];
                unused &= ~taps_levels(l, ax.width[l]);
            }
            at_dst |= sl;
            sliced = sl != 0;
            // InferAll2All until none: an axis held elsewhere moves to its
            // target position once that position is free
            while (use_a2a) {
                uint32_t mv = 0;
#pragma unroll
                for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
                    uint32_t b = 1u << l;
                    if ((at_src & ax.has_dst & b) && !((occ >> ax.dkey[l]) & 1u)) mv |= b;
                }
                if (!mv) break;
#pragma unroll
                for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
                    if (!((mv >> l) & 1u)) continue;
                    taps_collective(c, true, l, ax.width[l], S, unused, lam);
                    occ ^= taps_bit64(ax.skey[l]) | taps_bit64(ax.dkey[l]);
                    ++n_a2a;
                }
                at_src &= ~mv;
                at_dst |= mv;
            }
        } while (sliced);
        // InferAllGather: the lowest producer position the consumer does not
        // use; else AllGatherFirstUndoneDim: the lowest one not yet right
        // key = position << 8 | level << 4 | width keeps the choice in registers
        uint32_t best = 0xFFFFFu, best_any = 0xFFFFFu;
#pragma unroll
        for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
            if (!((at_src >> l) & 1u)) continue;
            uint32_t key = (ax.skey[l] << 8) | (l << 4) | ax.width[l];
            if (!((ax.tgt >> ax.skey[l]) & 1u) && key < best) best = key;
            if (key < best_any) best_any = key;
        }
        if (best == 0xFFFFFu) best = best_any;
        if (best != 0xFFFFFu) {
            uint32_t l = (best >> 4) & 15u, w = best & 15u;
            taps_collective(c, false, l, w, S, unused, lam);
            occ &= ~taps_bit64(best >> 8);
            at_src &= ~(1u << l);
            S <<= w;
            unused |= taps_levels(l, w);
        }
    }
    return n_a2a;
}

// "remove" (Table 2): gather every producer-mapped axis that is not at its
// target, lowest position first, then slice (free).
__host__ __device__ inline void taps_remove(const taps_axes &ax, uint32_t lam, taps_acc &c) {
    uint32_t todo = ax.has_src & ~ax.home;
    uint32_t unused = ~ax.used0;
    uint64_t S = ax.S0;
    while (todo) {
        uint32_t best = 0xFFFFFu;
#pragma unroll
        for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l) {
            if (!((todo >> l) & 1u)) continue;
            uint32_t key = (ax.skey[l] << 8) | (l << 4) | ax.width[l];
            if (key < best) best = key;
        }
        uint32_t l = (best >> 4) & 15u, w = best & 15u;
        taps_collective(c, false, l, w, S, unused, lam);
        todo &= ~(1u << l);
        S <<= w;
        unused |= taps_levels(l, w);
    }
}

// Exact comparison of intra/(N B_intra) + inter/(N B_inter) between two
// candidates: compare intra * bi + inter * ba with bi = B_inter / g,
// ba = B_intra / g (g = gcd of the two bandwidths), in 128 bits.
__host__ __device__ inline unsigned __int128 taps_key(const taps_acc &c, uint64_t b_inter_red,
                                                      uint64_t b_intra_red) {
    return (unsigned __int128)c.intra * b_inter_red + (unsigned __int128)c.inter * b_intra_red;
}

struct taps_entry_out {
    double t;
    uint64_t vol, intra, inter;
    uint32_t meta;
    bool ok;
};

// The cheapest of Algorithm 1, Algorithm 1 without AllToAll, and "remove"
// (the naive sequence gathers a superset of what "remove" gathers, in the
// same order, so it is never cheaper in either model and never wins a tie);
// vol is the smallest volume among them.
__host__ __device__ inline taps_entry_out taps_edge_entry(const taps_edge_problem &p,
                                                          uint64_t b_inter_red,
                                                          uint64_t b_intra_red, double inv_n_bintra,
                                                          double inv_n_binter) {
    taps_axes ax;
    taps_unify(p, ax);
    taps_acc c0, c1, c2;
    taps_acc_zero(c0);
    taps_acc_zero(c1);
    taps_acc_zero(c2);
    bool ok0 = true, ok1 = true;
    uint32_t n_a2a = taps_alg1(ax, p.lam, true, c0, &ok0);
    if (n_a2a)
        taps_alg1(ax, p.lam, false, c1, &ok1);
    else
        c1 = c0;
    taps_remove(ax, p.lam, c2);
    unsigned __int128 k0 = taps_key(c0, b_inter_red, b_intra_red);
    unsigned __int128 k1 = taps_key(c1, b_inter_red, b_intra_red);
    unsigned __int128 k2 = taps_key(c2, b_inter_red, b_intra_red);
    taps_acc best = c0;
    uint32_t cand = 0;
    unsigned __int128 kb = k0;
    if (k1 < kb) {
        best = c1;
        cand = 1;
        kb = k1;
    }
    if (k2 < kb) {
        best = c2;
        cand = 2;
    }
    taps_entry_out o;
    uint64_t v = c0.vol < c1.vol ? c0.vol : c1.vol;
    o.vol = v < c2.vol ? v : c2.vol;
    o.intra = best.intra;
    o.inter = best.inter;
    o.t = (double)best.intra * inv_n_bintra + (double)best.inter * inv_n_binter;
    o.meta = taps_meta(cand, best);
    o.ok = ok0 && ok1;
    return o;
}

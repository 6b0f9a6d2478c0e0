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
#define TAPS_D_MAX_CLASSES 4

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

// Bits 0..k-1 for k < 32.
__host__ __device__ inline uint32_t taps_below(uint32_t k) { return (1u << k) - 1u; }

// x << k for x < 2^16, k < 16 and a result below 2^16: one v_lshlrev_b16 on the
// device (it writes zeros to the upper half), which gfx950 issues at the rate
// of a 32-bit add, where v_lshlrev_b32 takes about twice as long.
__host__ __device__ inline uint32_t taps_shl16(uint32_t x, uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_lshlrev_b16 %0, %1, %2" : "=v"(r) : "v"(k), "v"(x));
    return r;
#else
    return (x << k) & 0xFFFFu;
#endif
}

// w one-bits starting at bit o, ((1 << w) - 1) << o, for w, o < 32 and w + o <= 32:
// one v_bfm_b32 on the device.
__host__ __device__ inline uint32_t taps_bfm(uint32_t w, uint32_t o) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_bfm_b32 %0, %1, %2" : "=v"(r) : "v"(w), "v"(o));
    return r;
#else
    return ((1u << w) - 1u) << o;
#endif
}

// The low w bits, (1 << w) - 1 for w < 32: taps_bfm(w, 0) with the offset as
// an inline constant (no register holding the zero).
__host__ __device__ inline uint32_t taps_low(uint32_t w) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_bfm_b32 %0, %1, 0" : "=v"(r) : "v"(w));
    return r;
#else
    return (1u << w) - 1u;
#endif
}

// x << K for a result below 2^16, the shift an inline constant.
template <uint32_t K>
__host__ __device__ inline uint32_t taps_shl16c(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_lshlrev_b16 %0, %2, %1" : "=v"(r) : "v"(x), "i"(K));
    return r;
#else
    return (x << K) & 0xFFFFu;
#endif
}

// 4 k for k < 16 (a nibble's bit offset).
__host__ __device__ inline uint32_t taps_x4(uint32_t k) { return taps_shl16c<2>(k); }

// Nibble k (< 8) of v, k per lane: one bit-field extract at a 16-bit-shifted offset.
__host__ __device__ inline uint32_t taps_nib_at(uint32_t v, uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_ubfe(v, taps_x4(k), 4u);
#else
    return (v >> (4u * k)) & 15u;
#endif
}

// Entry i (< 2^16 / sizeof(T)) of a small table: the byte offset by a 16-bit shift.
template <uint32_t LogSize, typename T>
__host__ __device__ inline const T &taps_entry(const T *tab, uint32_t i) {
    static_assert(sizeof(T) == (1u << LogSize), "entry size");
    return *(const T *)((const char *)tab + taps_shl16c<LogSize>(i));
}

// A uniform value copied into a vector register: the per-lane arithmetic then
// reads it from there (gfx950 issues a simple 32-bit operation with a scalar
// register operand at about half the rate of one with vector operands).  x
// must be the same in every lane of the wavefront (it is read from a scalar
// register): taps_make_row, its only caller, runs on one row per wavefront.
__host__ __device__ inline uint32_t taps_vcopy(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_mov_b32 %0, %1" : "=v"(r) : "s"(x));
    return r;
#else
    return x;
#endif
}

// (a & b) | c and a | b | c as one v_bitop3_b32 each: gfx950 issues it at the
// rate of a 32-bit add, where v_and_or_b32 and v_or3_b32 take about twice as
// long.  The immediate is the truth table, bit 4a + 2b + c.
__host__ __device__ inline uint32_t taps_and_or(uint32_t a, uint32_t b, uint32_t c) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0xEA);
#else
    return (a & b) | c;
#endif
}

__host__ __device__ inline uint32_t taps_or3(uint32_t a, uint32_t b, uint32_t c) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0xFE);
#else
    return a | b | c;
#endif
}

// 1 << k for k < 16: taps_shl16(1, k) with the one as an inline constant.
__host__ __device__ inline uint32_t taps_bit16(uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t r;
    __asm__("v_lshlrev_b16_e64 %0, %1, 1" : "=v"(r) : "v"(k));
    return r;
#else
    return (1u << k) & 0xFFFFu;
#endif
}

// Levels lo .. lo+w-1 (lo + w <= 8).
__host__ __device__ inline uint32_t taps_levels(uint32_t lo, uint32_t w) {
    return taps_below(lo + w) & ~taps_below(lo);
}

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

__host__ __device__ constexpr uint32_t taps_binom(uint32_t a, uint32_t b) {
    if (b > a) return 0;
    uint32_t r = 1;
    for (uint32_t x = 1; x <= b; ++x) r = r * (a - b + x) / x;
    return r;
}

__host__ __device__ constexpr uint32_t taps_fact(uint32_t a) {
    uint32_t r = 1;
    for (uint32_t x = 2; x <= a; ++x) r *= x;
    return r;
}

// w(k, s, z); only states with z + s <= 8 occur (each split axis takes at
// least one level), where every term has z + j <= 8 and the sum stays below
// 2^32; other entries are never read.
__host__ __device__ constexpr uint32_t taps_completions(uint32_t k, uint32_t s, uint32_t z) {
    if (z + s > TAPS_D_MAX_LEVELS) return 0;
    if (s == 0) return taps_fact(z);
    uint32_t tot = 0;
    const uint32_t jmax = k < s ? k : s;
    for (uint32_t j = 1; j <= jmax; ++j)
        tot += taps_binom(k, j) * taps_binom(s - 1, j - 1) * taps_fact(z + j);
    return tot;
}

struct taps_completion_table {
    uint32_t v[9 * 9 * 9];   // index (k * 9 + s) * 9 + z
};

__host__ __device__ constexpr taps_completion_table taps_make_completions() {
    taps_completion_table t{};
    for (uint32_t x = 0; x < 9u * 9u * 9u; ++x) t.v[x] = taps_completions(x / 81u, (x / 9u) % 9u, x % 9u);
    return t;
}

// Decodes candidate r (0 <= r < w(p, n, 0)) into per-axis exponents and
// device-map positions.  part: partitionable-axis mask; W: the completion
// table.  Returns false if r is out of range.
__host__ __device__ inline bool taps_unrank(uint32_t n_axes, uint32_t part, uint32_t n, uint32_t r,
                                            const uint32_t *W, uint32_t *expo, int32_t *pos) {
    uint32_t s = n, z = 0;
    for (uint32_t a = 0; a < n_axes; ++a) {
        expo[a] = 0;
        pos[a] = -1;
        if (!((part >> a) & 1u)) continue;
        const uint32_t k = taps_popc(part >> (a + 1));
        bool placed = false;
        for (uint32_t e = 0; e <= s; ++e) {
            const uint32_t z2 = z + (e > 0 ? 1u : 0u);
            const uint32_t c = W[(k * 9u + (s - e)) * 9u + z2];
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
    uint32_t q = taps_fact(z) - 1u - r;
    uint32_t free_pos = taps_low_mask(z);
    uint32_t t = 0;
    for (uint32_t a = 0; a < n_axes; ++a) {
        if (expo[a] == 0) continue;
        const uint32_t f = taps_fact(z - 1u - t);
        const uint32_t idx = q / f;
        q -= idx * f;
        uint32_t m = free_pos;
        for (uint32_t x = 0; x < idx; ++x) m &= m - 1u;   // drop the idx lowest free positions
        const uint32_t p = taps_ctz(m);
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
// Edge entries.
//
// The edge tensor T (rank R) leaves its producer under strategy P and enters
// its consumer under strategy Q.  Dimension d of T occupies the run of levels
// of its producer axis, mask pr[d] with top phi[d]-1 (0 if whole), and on the
// consumer side cr[d] with top chi[d]-1 (taps_col holds it as cr8 = cr << 8).
//
// Positions.  In the unified tensor, the sub-dimension that starts at bit t
// of dimension d is held, on the producer side, by the unified axis whose top
// level is phi[d]-1-t, and on the consumer side by the one whose top is
// chi[d]-1-t.  So one position corresponds to producer top l and consumer
// top l + dl[d] with dl[d] = chi[d] - phi[d]: every relation between the two
// tensor maps that Algorithm 1 needs is a per-dimension shift of an 8-bit
// level mask.  A unified axis is named by its top level; sets of axes are
// masks of tops.
//
// Volumes.  The producer's per-device shard is S = tbytes * 2^e nb with
// e = n - (levels the current map uses), and every volume of Eq. 9, 10 and
// 14 is tbytes times a power of two times a small integer.  Candidates are
// therefore accumulated as 32-bit integers in units of tbytes/256 ("factor"
// units) and scaled by tbytes once, exactly, at the end; comparing two
// candidates of one entry does not need tbytes at all.
// ---------------------------------------------------------------------------

__host__ __device__ inline uint32_t taps_msb(uint32_t v) { return 31u - (uint32_t)__builtin_clz(v); }

// Widths of the unified axes, by their tops: for every mask tp of top levels,
// nibble t of entry tp is the width of the axis whose top level is t (it
// starts one level above the next lower top, or at level 0), 0 when t is not
// a top.  Kernels keep a copy in LDS: one lookup per entry replaces a
// leading-zero count per axis.
struct taps_width_table {
    uint32_t v[256];
};

__host__ __device__ constexpr taps_width_table taps_make_widths() {
    taps_width_table t{};
    for (uint32_t m = 0; m < 256u; ++m) {
        uint32_t w = 0, lo = 0;
        for (uint32_t l = 0; l < 8u; ++l)
            if ((m >> l) & 1u) {
                w |= (l + 1u - lo) << (4u * l);
                lo = l + 1u;
            }
        t.v[m] = w;
    }
    return t;
}

// AllToAll shard fractions by tops mask: byte t of (lo, hi) is 2^(8 - w_t) for
// every top t of the mask (w_t the width of the axis with top t, as in
// taps_make_widths), 0 for the other levels; bytes 0-3 in lo, 4-7 in hi.
struct taps_a2a_table {
    uint32_t lo[256], hi[256];
};

__host__ __device__ constexpr taps_a2a_table taps_make_a2a() {
    taps_a2a_table t{};
    for (uint32_t m = 0; m < 256u; ++m) {
        uint32_t lo = 0, bytes[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (uint32_t l = 0; l < 8u; ++l)
            if ((m >> l) & 1u) {
                bytes[l] = 1u << (8u - (l + 1u - lo));
                lo = l + 1u;
            }
        t.lo[m] = bytes[0] | (bytes[1] << 8) | (bytes[2] << 16) | (bytes[3] << 24);
        t.hi[m] = bytes[4] | (bytes[5] << 8) | (bytes[6] << 16) | (bytes[7] << 24);
    }
    return t;
}

// Bit masks as byte vectors: byte t of (lo, hi) is bit t of the mask.
struct taps_expand_table {
    uint32_t lo[256], hi[256];
};

__host__ __device__ constexpr taps_expand_table taps_make_expand() {
    taps_expand_table t{};
    for (uint32_t m = 0; m < 256u; ++m) {
        t.lo[m] = t.hi[m] = 0;
        for (uint32_t l = 0; l < 4u; ++l) {
            t.lo[m] |= ((m >> l) & 1u) << (8u * l);
            t.hi[m] |= ((m >> (l + 4u)) & 1u) << (8u * l);
        }
    }
    return t;
}

// Sum of the four byte products of a and b, plus c: one v_dot4_u32_u8.
__host__ __device__ inline uint32_t taps_dot4(uint32_t a, uint32_t b, uint32_t c) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_udot4(a, b, c, false);
#else
    for (uint32_t k = 0; k < 32u; k += 8u) c += ((a >> k) & 0xFFu) * ((b >> k) & 0xFFu);
    return c;
#endif
}

struct taps_pair {
    uint32_t lo, hi;
};

// Per tops mask, in LDS: the shard fractions of every axis (x, y: taps_make_a2a)
// and of the axes inside one node (z, w: the same bytes below lam, 0 above).
struct taps_a2a_row {
    uint32_t all_lo, all_hi, in_lo, in_hi;
};

// Producer side of one table row (uniform across a wavefront).
struct taps_row {
    uint32_t rank, n, lam, full;
    uint32_t pr[TAPS_D_MAX_RANK];   // level run of dimension d (0 if whole)
    uint32_t phi[TAPS_D_MAX_RANK];  // top level + 1 of that run
    uint32_t pw[TAPS_D_MAX_RANK];   // its width
    uint32_t pcuts;                 // cut mask of the producer strategy
    uint32_t pru;                   // levels the producer map uses
    uint32_t e0;                    // n - |pru|
    uint32_t dstr;                  // dimension whose run holds levels lam - 1 and lam (8: none)
    uint32_t split;                 // bit d: the producer splits dimension d (pr[d] != 0)
    uint32_t vlam, vlow;            // lam and taps_below(lam) for the per-lane arithmetic (taps_vcopy)
    uint32_t vpr[TAPS_D_MAX_RANK];  // pr, likewise
    // Producer positions in order (dimension ascending, then bit ascending,
    // i.e. level descending): rank r holds level nibble r of `order`;
    // to_rank[x] is the level mask x with level l moved to bit rank(l).
    uint32_t order;
    const uint8_t *to_rank;
    const uint32_t *widths;      // taps_make_widths()
    const taps_a2a_row *a2a;     // by tops mask (taps_make_a2a, split at lam)
    const taps_pair *expand;     // by mask (taps_make_expand)
    // by tops mask, TAPS_D_MAX_CLASSES entries each: taps_make_a2a's bytes of
    // the tops in link class c (hierarchies of link classes)
    const taps_pair *a2a_cls;
};

// Consumer side of one table column.
struct taps_col {
    uint32_t cr8[TAPS_D_MAX_RANK];   // level run of dimension d (0 if whole), shifted up by 8
    uint32_t clo[TAPS_D_MAX_RANK];   // its lowest level
    uint32_t cw[TAPS_D_MAX_RANK];    // its width
    uint32_t ccuts;
};

// The unified problem of one entry.
struct taps_lv {
    uint32_t tp;            // tops of the unified axes
    uint32_t p1, p2, p4;    // "same axis as the level above" masks for taps_fill
    uint32_t src, dst;      // axes the producer / consumer maps use
    uint32_t home;          // axes at the same position in both maps
    uint32_t tgtsrc;        // producer positions the consumer map also uses
    uint32_t st;            // top of the axis holding levels lam - 1 and lam (0 if none)
    uint32_t lo_s;          // its lowest level
    uint32_t wt;            // nibble t: width of the axis with top t (taps_make_widths)
    // Positions: producer level l of dimension d and consumer level l + dl[d]
    // hold the same bit of d.  sh[d] = 8 + dl[d], so that a producer mask m of
    // d moves to the consumer side as (m << sh[d]) >> 8 (no signed shifts).
    uint32_t sh[TAPS_D_MAX_RANK];
    uint32_t pt[TAPS_D_MAX_RANK];   // producer levels of d whose position the consumer splits too
};

// One candidate sequence, in factor units, and the sum of the inter-node
// group counts (Algorithm 3's ct) of its collectives.  The number of
// collectives and of inter-node ones is the same for every candidate (each
// axis held off its target is moved once, by an AllToAll or an AllGather, and
// its collective crosses nodes exactly when its top is at or above lam), so
// it is counted once per entry (taps_collectives).
struct taps_fac {
    uint32_t vol, intra, inter;
    uint32_t ct;
};

__host__ __device__ inline void taps_fac_zero(taps_fac &c) {
    c.vol = c.intra = c.inter = 0;
    c.ct = 0;
}

// All levels of the axes whose tops are in x.
__host__ __device__ inline uint32_t taps_fill(const taps_lv &L, uint32_t x) {
    x = taps_and_or(x >> 1, L.p1, x);
    x = taps_and_or(x >> 2, L.p2, x);
    x = taps_and_or(x >> 4, L.p4, x);
    return x;
}

// Unification (Table 1) as a least fixpoint over cuts: a cut inside the part
// of a dimension both maps split forces the cut at the same bit of that
// dimension on the other side.  Then the axes and their positions.
__host__ __device__ inline void taps_unify(const taps_row &P, const taps_col &Q, taps_lv &L) {
    uint32_t pwin[TAPS_D_MAX_RANK], cwin[TAPS_D_MAX_RANK], back[TAPS_D_MAX_RANK];
    uint32_t cru = 0, home = 0, tgt = 0;
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
        pwin[d] = cwin[d] = 0;
        L.sh[d] = back[d] = 8u;
        L.pt[d] = 0;
        if (d >= P.rank) continue;
        cru |= Q.cr8[d];
        // When either side leaves d whole its run mask is 0, and so is every
        // mask below: no case split on which sides split d.
        // 8 + dl, in 0 .. 16 (dl: consumer top + 1 minus the producer's)
        const uint32_t sh = Q.clo[d] + Q.cw[d] + (8u - P.phi[d]);
        L.sh[d] = sh;
        back[d] = 16u - sh;
        // producer levels whose consumer level (l + dl) the consumer splits in
        // d: the top min(pw, cw) levels of the producer's run (the run moved
        // down by dl: (cr << 8) >> sh)
        const uint32_t pt = P.vpr[d] & (Q.cr8[d] >> sh);
        L.pt[d] = pt;
        tgt |= pt;
        // the cut positions inside that part (all its levels but the lowest),
        // on each side (l + sh <= 15 for every level l of pt, and sh = 16 only
        // where pt is 0: 16-bit shifts suffice here and in the fixpoint)
        pwin[d] = pt & (pt - 1u);
        cwin[d] = taps_shl16(pwin[d], sh) >> 8;
        // at the same position on both sides when dl = 0
        home |= sh == 8u ? pt : 0u;
    }
    // least fixpoint: each pass moves the cuts inside every window to the other
    // side (at most 7 cuts exist, so at most 8 passes)
    uint32_t C = (P.pcuts | Q.ccuts) & P.full & ~1u;
    for (uint32_t it = 0; it < TAPS_D_MAX_LEVELS; ++it) {
        // dimension 0 unconditionally (its windows are 0 without one)
        uint32_t acc = taps_shl16(C & pwin[0], L.sh[0]) | taps_shl16(C & cwin[0], back[0]);
#pragma unroll
        for (uint32_t d = 1; d < TAPS_D_MAX_RANK; ++d) {
            if (d >= P.rank) break;
            acc = taps_or3(taps_shl16(C & pwin[d], L.sh[d]), taps_shl16(C & cwin[d], back[d]), acc);
        }
        const uint32_t next = C | (acc >> 8);
        if (next == C) break;
        C = next;
    }
    const uint32_t starts = (C | 1u) & P.full;
    L.tp = P.n ? ((starts >> 1) | (1u << (P.n - 1))) & P.full : 0u;
    L.wt = taps_entry<2>(P.widths, L.tp);
    L.p1 = ~(starts >> 1) & P.full;
    L.p2 = L.p1 & (L.p1 >> 1);
    L.p4 = L.p2 & (L.p2 >> 2);
    L.src = L.tp & P.pru;
    L.dst = L.tp & (cru >> 8);
    L.home = L.tp & home;
    L.tgtsrc = L.tp & tgt;
    const uint32_t lam = P.lam;
    const uint32_t low = P.vlow;
    L.lo_s = taps_msb(((L.tp & low) << 1) | 1u);
    const bool st = lam >= 1u && lam < P.n && !((L.tp >> (lam - 1u)) & 1u);
    L.st = st ? 1u << taps_ctz((L.tp & ~low) | 0x100u) : 0u;
}

// Consumer tops whose target position an axis in ats (producer tops) holds.
// Each term lies in bits 8-15 (16-bit shifts; pt[d] is 0 where sh[d] is 16 or
// d >= rank), and two dimensions at a time join the sum in one three-way or.
__host__ __device__ inline uint32_t taps_blocked(const taps_row &P, const taps_lv &L,
                                                 uint32_t ats) {
    // dimension 0 unconditionally: without one, pt[0] is 0 and so is its term
    uint32_t acc = taps_shl16(ats & L.pt[0], L.sh[0]);
#pragma unroll
    for (uint32_t d = 1; d < TAPS_D_MAX_RANK; d += 2) {
        if (d >= P.rank) break;
        const uint32_t t = taps_shl16(ats & L.pt[d], L.sh[d]);
        const uint32_t u = d + 1u < TAPS_D_MAX_RANK ? taps_shl16(ats & L.pt[d + 1u], L.sh[d + 1u]) : 0u;
        acc = taps_or3(t, u, acc);
    }
    return acc >> 8;
}

// The level holding producer-order rank k.
__host__ __device__ inline uint32_t taps_rank_level(const taps_row &P, uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_ubfe(P.order, taps_x4(k), 4u);
#else
    return (P.order >> (4u * k)) & 15u;
#endif
}

// The level holding producer-order rank k mod 8 (k < 16): v_bfe_u32 reads
// the low five bits of its offset, so 4k needs no reduction on the device.
__host__ __device__ inline uint32_t taps_rank_level_mod8(const taps_row &P, uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_ubfe(P.order, taps_x4(k), 4u);
#else
    return (P.order >> (4u * (k & 7u))) & 15u;
#endif
}

// All ones when bit k of x is set, else 0 (k < 32): one v_bfe_i32 on the device.
__host__ __device__ inline uint32_t taps_bit_mask(uint32_t x, uint32_t k) {
#if defined(__HIP_DEVICE_COMPILE__)
    return (uint32_t)__builtin_amdgcn_sbfe((int32_t)x, k, 1u);
#else
    return 0u - ((x >> k) & 1u);
#endif
}

// The axis of x (non-empty, producer levels) at the lowest producer position.
__host__ __device__ inline uint32_t taps_first_src(const taps_row &P, uint32_t x) {
    return taps_rank_level(P, taps_ctz(P.to_rank[x]));
}

// The unified axis with top level `top`: lowest level (one above the next
// lower top, 0 if none), width and level mask.
struct taps_ax {
    uint32_t lo, w, lv;
};

__host__ __device__ inline taps_ax taps_axis(const taps_lv &L, uint32_t top) {
    taps_ax a;
#if defined(__HIP_DEVICE_COMPILE__)
    a.w = __builtin_amdgcn_ubfe(L.wt, taps_x4(top), 4u);
#else
    a.w = (L.wt >> (4u * top)) & 15u;
#endif
    a.lo = top + 1u - a.w;
    a.lv = taps_bfm(a.w, a.lo);
    return a;
}

// An AllGather (Eq. 9) of the axis with top level `top`, shard 2^sh factor
// units (taps_state), with the inter-node group count of Algorithm 3: groups
// holding the same data inside a node (replicas along levels no dimension
// uses) share one inter-node transfer.
__host__ __device__ inline void taps_cost(taps_fac &c, uint32_t top, const taps_ax &a,
                                          uint32_t lam, uint32_t low, uint32_t sh,
                                          uint32_t unused) {
    const uint32_t V = taps_bfm(a.w, sh);
    // all ones when the whole group lies inside one node (top < lam)
    const uint32_t in_node = (uint32_t)((int32_t)(top - lam) >> 31);
    // groups of replicas inside a node share one transfer: the levels below
    // min(lo, lam) that some dimension uses count
    const uint32_t lct = taps_popc(taps_low(a.lo) & low & ~unused);
    c.vol += V;
    c.intra += V & in_node;
    c.inter += (V << lct) & ~in_node;
    c.ct += taps_bit16(lct) & ~in_node;
}

// AllToAlls (Eq. 10, Eq. 14) of every axis whose top is in x, all issued at
// one state (shard 2^sh factor units, free levels `unused`; low = the levels
// below lam): an AllToAll changes
// neither, so the axes of one closure are costed together.  An axis wholly
// above the node boundary sends V over the inter-node link with the group
// count of Algorithm 3 that all such axes share; an in-node axis costs V
// inside the node; the straddling axis (at most one) keeps its group
// members inside a node out of the inter-node link.
__host__ __device__ inline void taps_a2a_batch(taps_fac &c, uint32_t x, const taps_lv &L,
                                               uint32_t lam, uint32_t low, uint32_t sh,
                                               uint32_t unused, const taps_a2a_row *a2a,
                                               const taps_pair *expand) {
    // Axis t keeps 2^-w_t of the shard: V_t = 2^sh - 2^(sh - w_t), and over the
    // axes of m, sum V_t = |m| 2^sh - 2^(sh - 8) sum 2^(8 - w_t) (w_t <= 8 <= sh,
    // so every term is whole).  The bytes 2^(8 - w_t) of the tops come from a
    // table by tops mask, m's bits as bytes from another; two byte dot products
    // sum them, all axes and the in-node ones (tops below lam).
    const uint32_t m = x & ~L.st;
    const taps_a2a_row W = taps_entry<4>(a2a, L.tp);
    const taps_pair X = taps_entry<3>(expand, m);
    const uint32_t f_all = taps_dot4(W.all_hi, X.hi, taps_dot4(W.all_lo, X.lo, 0u));
    const uint32_t f_in = taps_dot4(W.in_hi, X.hi, taps_dot4(W.in_lo, X.lo, 0u));
    const uint32_t n_in = taps_popc(m & low), n_out = taps_popc(m & ~low);
    const uint32_t e = sh - 8u;
    const uint32_t sum = ((n_in + n_out) << sh) - (f_all << e);
    const uint32_t sum_in = (n_in << sh) - (f_in << e);
    const uint32_t lct = taps_popc(low & ~unused);
    c.vol += sum;
    c.intra += sum_in;
    c.inter += (sum - sum_in) << lct;
    c.ct += n_out << lct;
    if (x & L.st) {
        const uint32_t t = taps_ctz(L.st), lo = L.lo_s;
        const uint32_t w = t + 1u - lo, kap = lam - lo;
        const uint32_t V = (1u << sh) - (1u << (sh - w));
        const uint32_t link = ((1u << w) - (1u << kap)) << (kap + sh - w);
        const uint32_t lcts = lo - taps_popc(unused & taps_below(lo));
        c.vol += V;
        c.inter += link << lcts;
        c.ct += 1u << lcts;
    }
}

// Exact order of intra/(N B_intra) + inter/(N B_inter) between candidates:
// intra * bi + inter * ba with bi = B_inter / g, ba = B_intra / g
// (g = gcd of the two).  Both products fit 64 bits when bi, ba < 2^32.
struct taps_keys {
    uint64_t b_inter_red, b_intra_red;
    bool narrow;   // both reduced bandwidths below 2^32
};

__host__ __device__ inline uint64_t taps_key64(const taps_fac &a, const taps_keys &K) {
    return (uint64_t)a.intra * (uint32_t)K.b_inter_red + (uint64_t)a.inter * (uint32_t)K.b_intra_red;
}

__host__ __device__ inline bool taps_less(const taps_fac &a, const taps_fac &b,
                                          const taps_keys &K) {
    if (K.narrow) return taps_key64(a, K) < taps_key64(b, K);
    const unsigned __int128 ka =
        (unsigned __int128)a.intra * K.b_inter_red + (unsigned __int128)a.inter * K.b_intra_red;
    const unsigned __int128 kb =
        (unsigned __int128)b.intra * K.b_inter_red + (unsigned __int128)b.inter * K.b_intra_red;
    return ka < kb;
}

// A later candidate can stop early: every collective adds to both its key
// and its volume, so once the running key reaches the best key so far and
// the running volume reaches the smallest volume so far it can neither be
// chosen (ties go to the earlier candidate) nor lower the volume.
// Without a single key (several bandwidth points) a candidate is hopeless
// once its intra- and inter-node bytes both reach the first candidate's:
// then its key is at least as large under every pair of bandwidths.
struct taps_limit {
    bool on;          // compare keys
    bool dominated;   // compare intra and inter
    uint64_t key;
    uint32_t vol, intra, inter;
};

__host__ __device__ inline bool taps_hopeless(const taps_fac &c, const taps_limit &lim,
                                              const taps_keys &K) {
    // every comparison made (no short circuit): one branch on their conjunction
    if (lim.dominated)
        return (c.vol >= lim.vol) & (c.intra >= lim.intra) & (c.inter >= lim.inter);
    return lim.on && ((c.vol >= lim.vol) & (taps_key64(c, K) >= lim.key));
}

template <class Fac>
struct taps_run_t {
    Fac c;
    uint32_t a2a_tops;   // tops of the axes moved by an AllToAll (0: none)
    bool ok;          // false if the loop did not settle (cannot happen)
    bool stopped;     // stopped early: cannot beat the limit it was given
};
using taps_run = taps_run_t<taps_fac>;

// The paper's two link classes (Eq. 11-14 with Algorithm 3): the cost of one
// AllGather and of the AllToAlls of one closure, and the early stop of a later
// candidate.  Algorithm 1 and "rearrange" below are written over such a model.
struct taps_two_class {
    using fac = taps_fac;
    uint32_t lam, low;   // lam and taps_below(lam)
    const taps_keys *K;
    const taps_limit *lim;
    const taps_a2a_row *a2a_rows;   // the row's AllToAll tables (taps_row)
    const taps_pair *expand;
    __host__ __device__ void gather(fac &c, uint32_t top, const taps_ax &a, uint32_t sh,
                                    uint32_t unused) const;
    __host__ __device__ void a2a(fac &c, uint32_t x, const taps_lv &L, uint32_t sh,
                                 uint32_t unused) const;
    __host__ __device__ bool hopeless(const fac &c) const;
};

// Running state of one sequence: axes held at their producer position (ats)
// and at their target (atd), consumer tops whose target an at-src axis holds
// (blk), free levels (unused) and the shard as a shift, sh = e + 8 for a shard
// of tbytes 2^e (taps_row's e0 at the start): 2^sh factor units.
struct taps_state {
    uint32_t ats, atd, blk, unused, sh;
};

__host__ __device__ inline void taps_two_class::gather(fac &c, uint32_t top, const taps_ax &a,
                                                      uint32_t sh, uint32_t unused) const {
    taps_cost(c, top, a, lam, low, sh, unused);
}

__host__ __device__ inline void taps_two_class::a2a(fac &c, uint32_t x, const taps_lv &L,
                                                   uint32_t sh, uint32_t unused) const {
    taps_a2a_batch(c, x, L, lam, low, sh, unused, a2a_rows, expand);
}

__host__ __device__ inline bool taps_two_class::hopeless(const fac &c) const {
    return taps_hopeless(c, *lim, *K);
}

template <class Cm>
__host__ __device__ inline void taps_gather(const taps_lv &L, taps_state &s, typename Cm::fac &c,
                                            uint32_t top, const Cm &M) {
    const taps_ax a = taps_axis(L, top);
    M.gather(c, top, a, s.sh, s.unused);
    s.ats &= ~taps_bit16(top);
    s.unused |= a.lv;
    s.sh += a.w;
}

// Every free target position whose axis no dimension uses is sliced.
__host__ __device__ inline uint32_t taps_slice(const taps_lv &L, taps_state &s) {
    const uint32_t sl = L.dst & ~(s.ats | s.atd) & ~s.blk;
    if (sl) {
        const uint32_t lv = taps_fill(L, sl);
        s.atd |= sl;
        s.unused &= ~lv;
        s.sh -= taps_popc(lv);
    }
    return sl;
}

// Algorithm 1 ("replace" in Table 2).
//
// Equivalent schedule of the printed loop:
//   * one pass of the inner loop is InferSlice, then InferAll2All until
//     nothing moves; a slice never frees a position, so a second pass can
//     only slice (targets the AllToAlls freed) and a third finds nothing;
//   * an AllGather of an axis whose producer position no consumer axis
//     targets frees no position anyone wants, and the axis itself cannot be
//     sliced (a held axis with a free target has already moved), so the
//     next inner loop does nothing: such gathers run back to back, lowest
//     position first, unless the last AllToAlls left a slice pending, in
//     which case only the first runs before it;
//   * once no axis is held at a producer position only slices remain (no
//     held axis blocks a target), and slices cost nothing: the sequence's
//     cost is final there.
// One pass of the printed inner loop: InferSlice, then InferAll2All until
// nothing moves (the AllToAlls of one closure share one state and are costed
// together), then, if the first InferSlice sliced, the slices the AllToAlls
// made possible (a slice frees no position, so a third round finds nothing).
template <class Cm>
__host__ __device__ inline void taps_alg1_settle(const taps_row &P, const taps_lv &L,
                                                 taps_state &s, typename Cm::fac &c,
                                                 uint32_t &a2a_tops, const Cm &M, uint32_t sl) {
    // The closure as a frontier: the held axes with a target whose target is
    // free move first; each move frees the target its position blocked (each
    // target is blocked by at most one held axis), and exactly the held axes
    // with a target among those move next.
    const uint32_t A = L.dst & s.ats;
    uint32_t F = A & ~s.blk, moved = 0, freed = 0;
    while (F) {
        moved |= F;
        const uint32_t fr = taps_blocked(P, L, F);
        freed |= fr;
        F = fr & A;
    }
    if (moved) {
        s.ats &= ~moved;
        s.blk &= ~freed;
        s.atd |= moved;
        a2a_tops |= moved;
        M.a2a(c, moved, L, s.sh, s.unused);
    }
    if (sl) taps_slice(L, s);
}

template <class Cm>
__host__ __device__ inline void taps_alg1_pass(const taps_row &P, const taps_lv &L, taps_state &s,
                                               typename Cm::fac &c, uint32_t &a2a_tops,
                                               const Cm &M) {
    const uint32_t sl = taps_slice(L, s);
    taps_alg1_settle(P, L, s, c, a2a_tops, M, sl);
}

// The common start of the sequences: every axis not at its target held at its
// producer position, the home axes placed, and the first InferSlice done
// (slice = what it sliced).  Algorithm 1 and "rearrange" both begin here.
struct taps_start {
    taps_state s;
    uint32_t slice;
};

__host__ __device__ inline taps_start taps_begin(const taps_row &P, const taps_lv &L) {
    taps_start b;
    b.s.ats = L.src & ~L.home;
    b.s.atd = L.home;
    b.s.blk = taps_blocked(P, L, b.s.ats);
    b.s.unused = P.full & ~P.pru;
    b.s.sh = P.e0 + 8u;
    b.slice = taps_slice(L, b.s);
    return b;
}

template <class Cm>
__host__ __device__ inline taps_run_t<typename Cm::fac> taps_alg1_t(const taps_row &P,
                                                                    const taps_col &Q,
                                                                    const taps_lv &L,
                                                                    const Cm &M,
                                                                    const taps_start &b) {
    typename Cm::fac c;
    taps_fac_zero(c);
    taps_state s = b.s;
    uint32_t a2a_tops = 0;
    taps_alg1_settle(P, L, s, c, a2a_tops, M, b.slice);
    // Nothing held at a producer position: only slices remain, and they cost
    // nothing.  Otherwise InferAllGather first gathers the held axes at
    // positions no consumer axis targets.  Such a gather frees no position
    // anyone wants, and the axis cannot be sliced back (its target is still
    // blocked, else it would have moved), so the passes between these gathers
    // only perform the slices left pending by the last AllToAlls: they run back
    // to back in producer order, the first alone before the pending slices.
    uint32_t ug = s.ats & ~L.tgtsrc;
    if (ug) {
        if (L.dst & ~(s.ats | s.atd) & ~s.blk) {
            taps_gather(L, s, c, taps_first_src(P, ug), M);
            taps_slice(L, s);
            ug = s.ats & ~L.tgtsrc;
        }
        for (uint32_t x = P.to_rank[ug]; x; x &= x - 1u)
            taps_gather(L, s, c, taps_rank_level(P, taps_ctz(x)), M);
    }
    // Held axes now sit only at targeted positions (the held set only shrinks):
    // AllGatherFirstUndoneDim gathers the first in producer order, which frees
    // its position for the axis targeting it, and a pass follows.  Each round
    // gathers one held axis, so at most |held| rounds run.
    while (s.ats) {
        const uint32_t top = taps_first_src(P, s.ats);
        s.blk &= ~taps_blocked(P, L, taps_bit16(top));
        taps_gather(L, s, c, top, M);
        if (!s.ats) break;
        taps_alg1_pass(P, L, s, c, a2a_tops, M);
    }
    taps_run_t<typename Cm::fac> r;
    r.c = c;
    r.a2a_tops = a2a_tops;
    r.ok = true;
    r.stopped = false;
    return r;
}

__host__ __device__ inline taps_run taps_alg1(const taps_row &P, const taps_col &Q,
                                              const taps_lv &L, const taps_start &b) {
    const taps_two_class M{P.vlam, P.vlow, nullptr, nullptr, P.a2a, P.expand};
    return taps_alg1_t(P, Q, L, M, b);
}

__host__ __device__ inline taps_run taps_alg1(const taps_row &P, const taps_col &Q,
                                              const taps_lv &L) {
    return taps_alg1(P, Q, L, taps_begin(P, L));
}

// Algorithm 1 without AllToAll ("rearrange" in Table 2).  Without AllToAll
// the printed loop reduces to:
//   1. InferSlice once (a second pass finds nothing: no AllToAll frees a
//      position);
//   2. every held axis whose position no consumer axis targets is gathered,
//      lowest position first; one whose own target is free is sliced back
//      right away (the slice undoes the gather's change of shard and free
//      levels), the others stay whole;
//   3. the remaining held axes (all at targeted positions) are gathered,
//      lowest position first; after each, the axis itself is sliced back if
//      its target is free, and the axis targeting the freed position is
//      sliced if no dimension uses it.
// Step 2 is step 3 on positions no consumer axis targets (nothing is freed
// for anyone there), so both run as one loop over the held axes: the
// untargeted ones in producer order, then the targeted ones.
template <class Cm>
__host__ __device__ inline taps_run_t<typename Cm::fac> taps_rearrange_t(const taps_row &P,
                                                                         const taps_col &Q,
                                                                         const taps_lv &L,
                                                                         const Cm &M,
                                                                         const taps_start &b) {
    typename Cm::fac c;
    taps_fac_zero(c);
    taps_state s = b.s;   // InferSlice once
    bool stopped = false;
    // producer ranks of the untargeted held axes in bits 0-7, of the targeted ones in bits 8-15
    uint32_t x = (uint32_t)P.to_rank[s.ats & ~L.tgtsrc] |
                 ((uint32_t)P.to_rank[s.ats & L.tgtsrc] << 8);
    while (x) {
        if (M.hopeless(c)) {
            stopped = true;
            break;
        }
        const uint32_t top = taps_rank_level_mod8(P, taps_ctz(x));
        x &= x - 1u;
        const uint32_t b = taps_bit16(top);
        const taps_ax a = taps_axis(L, top);
        M.gather(c, top, a, s.sh, s.unused);
        const uint32_t freed_for = taps_blocked(P, L, b);   // the axis targeting that position
        s.ats &= ~b;
        s.blk &= ~freed_for;
        // sliced back into its own target if that is free (shard and free levels
        // as before: all ones then), else kept whole
        const uint32_t back = taps_bit_mask(L.dst & ~s.blk, top);
        s.atd = taps_and_or(b, back, s.atd);
        s.unused |= a.lv & ~back;
        s.sh += a.w & ~back;
        const uint32_t sf = freed_for & ~(s.ats | s.atd);   // sliced into the freed position
        if (sf) {
            const uint32_t lv = taps_fill(L, sf);
            s.atd |= sf;
            s.unused &= ~lv;
            s.sh -= taps_popc(lv);
        }
    }
    taps_run_t<typename Cm::fac> r;
    r.c = c;
    r.a2a_tops = 0;
    r.ok = true;
    r.stopped = stopped;
    return r;
}

__host__ __device__ inline taps_run taps_rearrange(const taps_row &P, const taps_col &Q,
                                                   const taps_lv &L, const taps_limit &lim,
                                                   const taps_keys &K) {
    const taps_two_class M{P.vlam, P.vlow, &K, &lim, P.a2a, P.expand};
    return taps_rearrange_t(P, Q, L, M, taps_begin(P, L));
}

__host__ __device__ inline taps_run taps_rearrange(const taps_row &P, const taps_col &Q,
                                                   const taps_lv &L, const taps_limit &lim,
                                                   const taps_keys &K, const taps_start &b) {
    const taps_two_class M{P.vlam, P.vlow, &K, &lim, P.a2a, P.expand};
    return taps_rearrange_t(P, Q, L, M, b);
}

// "remove" (Table 2): gather every held axis not at its target, lowest
// position first (dimensions ascending, each from its top level down); the
// slices that follow are free.  The run is uninterrupted, so it has a
// closed form:
//   * each gather multiplies the shard by 2^w, so all volumes together
//     telescope to (2^W - 1) S0 with W the gathered levels;
//   * inside one dimension the axes wholly above the node boundary come
//     first; they leave the free levels below lam alone, so they share one
//     inter-node group count (Algorithm 3) and cost (2^W_A - 1) S together;
//   * at most one unified axis straddles the boundary (the one holding
//     levels lam - 1 and lam), and it lies in the producer dimension whose
//     run holds those levels;
//   * the in-node axes come last and cost (2^W_B - 1) S' together.
__host__ __device__ inline taps_fac taps_remove(const taps_row &P, const taps_lv &L) {
    const uint32_t low = P.vlow;
    const uint32_t G = taps_fill(L, L.src & ~L.home);
    // the straddling axis (levels lo_s .. its top); only dimension P.dstr can hold it
    const uint32_t lo_s = L.lo_s;
    const uint32_t S = L.st && P.dstr < TAPS_D_MAX_RANK ? taps_fill(L, L.st) : 0u;
    const uint32_t GA = G & ~low & ~S, GB = G & low & ~S;
    const uint32_t TA = L.tp & GA;
    taps_fac c;
    c.vol = taps_bfm(taps_popc(G), P.e0 + 8u);
    c.intra = c.inter = 0;
    c.ct = 0;
    uint32_t sh = P.e0 + 8u;
    uint32_t unused = P.full & ~P.pru;
    // levels below lam some dimension still uses: the inter-node group count of
    // the axes above the node boundary (they leave these levels alone)
    uint32_t lctA = taps_popc(low & ~unused);
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
        if (!((P.split >> d) & 1u)) continue;   // nothing of G in a dimension left whole
        const uint32_t pd = P.vpr[d];
        const uint32_t WA = taps_popc(GA & pd), WB = taps_popc(GB & pd);
        const uint32_t nA = taps_popc(TA & pd);
        uint32_t WS = 0, WL = WB;   // WL: gathered levels of d below lam
        if (d == P.dstr) {   // uniform: the only dimension that can hold the straddler
            // without one (WS = 0) both terms are 0
            WS = taps_popc(G & S);
            WL += taps_popc(G & S & low);
            const uint32_t lctS = taps_popc(taps_low(lo_s) & ~unused);
            c.inter += taps_bfm(WS, sh + WA) << lctS;
            c.ct += (WS < 1u ? WS : 1u) << lctS;
        }
        c.intra += taps_bfm(WB, sh + WA + WS);
        c.inter += taps_bfm(WA, sh) << lctA;
        c.ct += nA << lctA;
        sh += WA + WB + WS;
        unused |= G & pd;
        lctA -= WL;
    }
    return c;
}

// How the factor-unit sums of one edge become record numbers (uniform over
// the edge): volumes are tbytes * f / 256 nb, exact; t uses the per-unit
// seconds a = tbytes / 256 / (N B).
struct taps_scaler {
    uint64_t tbytes;
    uint32_t q;         // tbytes / 256 when that is exact and below 2^32, else 0
    double a_intra;     // tbytes / 256 / (N B_intra)
    double a_inter;     // tbytes / 256 / (N B_inter)
};

__host__ __device__ inline taps_scaler taps_make_scaler(uint64_t tbytes, double inv_n_bintra,
                                                        double inv_n_binter) {
    taps_scaler S;
    S.tbytes = tbytes;
    S.q = (tbytes & 255u) == 0 && (tbytes >> 40) == 0 ? (uint32_t)(tbytes >> 8) : 0u;
    const double unit = (double)tbytes * (1.0 / 256.0);   // exact: tbytes < 2^53
    S.a_intra = unit * inv_n_bintra;
    S.a_inter = unit * inv_n_binter;
    return S;
}

// tbytes * f / 256, exact (the result is an integer volume in nb < 2^64).
__host__ __device__ inline uint64_t taps_scale(const taps_scaler &S, uint32_t f) {
    if (S.q) return (uint64_t)S.q * f;
    return (((S.tbytes & 0xFFFFFFFFull) * f) >> 8) + (((S.tbytes >> 32) * f) << 24);
}

// The chosen candidate of one entry, in factor units.
struct taps_pick {
    taps_fac best;
    uint32_t vmin;   // smallest volume among the candidates
    uint32_t cand;   // 0 Algorithm 1, 1 without AllToAll, 2 remove
    uint32_t coll;   // taps_collectives
    bool ok;
};

// Collectives of every candidate of an entry (bits 0-7) and the inter-node
// ones among them (bits 8-15): one per axis held off its target, inter-node
// when its top is at or above lam.
__host__ __device__ inline uint32_t taps_collectives(const taps_lv &L, uint32_t lam) {
    const uint32_t x = L.src & ~L.home;
    return taps_popc(x) | (taps_popc(x & ~taps_below(lam)) << 8);
}

struct taps_entry_out {
    double t;
    uint64_t vol, intra, inter;
    uint32_t meta;
    bool ok;
};

// The cheapest of Algorithm 1, Algorithm 1 without AllToAll, and "remove"
// (the naive sequence of Table 2 gathers a superset of what "remove"
// gathers, in the same order, so it is never cheaper in either model and
// never wins a tie); vol is the smallest volume among them.  The second
// candidate stops as soon as it cannot change the record.
__host__ __device__ inline taps_pick taps_edge_select(const taps_row &P, const taps_col &Q,
                                                      const taps_keys &K) {
    taps_lv L;
    taps_unify(P, Q, L);
    const taps_start b = taps_begin(P, L);
    const taps_run r0 = taps_alg1(P, Q, L, b);
    taps_pick k;
    k.best = r0.c;
    k.cand = 0;
    k.vmin = r0.c.vol;
    k.coll = taps_collectives(L, P.lam);
    k.ok = r0.ok;
    taps_limit lim;
    lim.on = K.narrow;
    lim.dominated = false;
    lim.key = taps_key64(k.best, K);
    lim.vol = k.vmin;
    lim.intra = lim.inter = 0;
    if (r0.a2a_tops) {   // without AllToAll the sequence would be the same
        const taps_run r1 = taps_rearrange(P, Q, L, lim, K, b);
        k.ok = k.ok && r1.ok;
        if (!r1.stopped) {
            if (taps_less(r1.c, k.best, K)) {
                k.best = r1.c;
                k.cand = 1;
            }
            k.vmin = r1.c.vol < k.vmin ? r1.c.vol : k.vmin;
        }
    }
    const taps_fac c2 = taps_remove(P, L);
    if (taps_less(c2, k.best, K)) {
        k.best = c2;
        k.cand = 2;
    }
    k.vmin = c2.vol < k.vmin ? c2.vol : k.vmin;
    return k;
}

// The candidates of one entry costed once for several bandwidth points: the
// factor integers of a sequence do not depend on the bandwidths, only the
// order of two candidates does.  The rearrange candidate stops early only
// once it can neither be chosen at any point (its intra- and inter-node
// bytes have reached the first candidate's; ties go to the first) nor lower
// the volume, so every selection below equals taps_edge_select under its
// own keys.
struct taps_cands {
    taps_fac c[3];   // replace, rearrange, remove
    uint32_t vmin;   // smallest volume among them
    uint32_t coll;   // taps_collectives
    bool has_rearrange;
    bool ok;
};

__host__ __device__ inline taps_cands taps_edge_candidates(const taps_row &P, const taps_col &Q,
                                                           const taps_keys &any) {
    taps_lv L;
    taps_unify(P, Q, L);
    const taps_start b = taps_begin(P, L);
    const taps_run r0 = taps_alg1(P, Q, L, b);
    taps_cands k;
    k.c[0] = r0.c;
    k.ok = r0.ok;
    k.vmin = r0.c.vol;
    k.coll = taps_collectives(L, P.lam);
    k.has_rearrange = r0.a2a_tops != 0;   // without AllToAll the sequence would be the same
    taps_fac_zero(k.c[1]);
    if (k.has_rearrange) {
        taps_limit lim;
        lim.on = false;
        lim.dominated = true;
        lim.key = 0;
        lim.vol = r0.c.vol;
        lim.intra = r0.c.intra;
        lim.inter = r0.c.inter;
        const taps_run r1 = taps_rearrange(P, Q, L, lim, any, b);
        k.ok = k.ok && r1.ok;
        if (r1.stopped) {
            k.has_rearrange = false;
        } else {
            k.c[1] = r1.c;
            k.vmin = r1.c.vol < k.vmin ? r1.c.vol : k.vmin;
        }
    }
    k.c[2] = taps_remove(P, L);
    k.vmin = k.c[2].vol < k.vmin ? k.c[2].vol : k.vmin;
    return k;
}

// Selection of taps_edge_select among precomputed candidates, under the
// keys of one bandwidth point (ties go to the earlier candidate).
__host__ __device__ inline taps_pick taps_pick_for(const taps_cands &k, const taps_keys &K) {
    taps_pick p;
    p.best = k.c[0];
    p.cand = 0;
    if (K.narrow) {   // each candidate's key once
        uint64_t best = taps_key64(k.c[0], K);
        const uint64_t k1 = taps_key64(k.c[1], K), k2 = taps_key64(k.c[2], K);
        if (k.has_rearrange && k1 < best) {
            p.best = k.c[1];
            p.cand = 1;
            best = k1;
        }
        if (k2 < best) {
            p.best = k.c[2];
            p.cand = 2;
        }
    } else {
        if (k.has_rearrange && taps_less(k.c[1], p.best, K)) {
            p.best = k.c[1];
            p.cand = 1;
        }
        if (taps_less(k.c[2], p.best, K)) {
            p.best = k.c[2];
            p.cand = 2;
        }
    }
    p.vmin = k.vmin;
    p.coll = k.coll;
    p.ok = k.ok;
    return p;
}

__host__ __device__ inline taps_entry_out taps_entry_finish(const taps_pick &k,
                                                            const taps_scaler &S) {
    taps_entry_out o;
    o.vol = taps_scale(S, k.vmin);
    o.intra = taps_scale(S, k.best.intra);
    o.inter = taps_scale(S, k.best.inter);
    o.t = (double)k.best.intra * S.a_intra + (double)k.best.inter * S.a_inter;
    o.meta = k.cand | ((k.coll & 0xFFu) << 2) | ((k.coll >> 8) << 7) | (k.best.ct << 12);
    o.ok = k.ok;
    return o;
}

__host__ __device__ inline taps_entry_out taps_edge_entry(const taps_row &P, const taps_col &Q,
                                                          const taps_scaler &S,
                                                          const taps_keys &K) {
    return taps_entry_finish(taps_edge_select(P, Q, K), S);
}

// Producer side of a row from a strategy descriptor and the tensor's axes
// (nibble d of `axes` = op axis of dimension d).
__host__ __device__ inline void taps_make_row(taps_row &P, const taps_desc &D, uint32_t axes,
                                              uint32_t rank, uint32_t n, uint32_t lam) {
    P.rank = rank;
    P.n = n;
    P.lam = lam;
    P.full = taps_low_mask(n);
    P.pcuts = D.cuts;
    P.pru = 0;
    uint32_t used = 0;
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
        const uint32_t a = taps_nib(axes, d);
        const uint32_t lo = taps_nib(D.lo, a), w = d < rank ? taps_nib(D.width, a) : 0u;
        P.pw[d] = w;
        P.phi[d] = lo + w;
        P.pr[d] = taps_levels(lo, w);
        P.pru |= P.pr[d];
        used += w;
    }
    P.e0 = n - used;
    P.vlam = taps_vcopy(lam);
    P.vlow = taps_vcopy(taps_below(lam));
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) P.vpr[d] = taps_vcopy(P.pr[d]);
    P.split = 0;
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) P.split |= (P.pr[d] ? 1u : 0u) << d;
    P.dstr = TAPS_D_MAX_RANK;
    if (lam >= 1u && lam < n) {
        const uint32_t two = 3u << (lam - 1u);
#pragma unroll
        for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d)
            if ((P.pr[d] & two) == two) P.dstr = d;
    }
    // producer order: dimensions ascending, each from its top level down
    P.order = 0;
    uint32_t k = 0;
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d)
        for (uint32_t t = 0; t < P.pw[d]; ++t) P.order |= (P.phi[d] - 1u - t) << (4u * k++);
    P.to_rank = nullptr;
    P.widths = nullptr;
    P.a2a = nullptr;
    P.expand = nullptr;
    P.a2a_cls = nullptr;
}

// to_rank table of a row: tab[x] = level mask x permuted into producer order.
// Entries x = first, first + step, ... < 256.
__host__ __device__ inline void taps_fill_rank_table(const taps_row &P, uint8_t *tab, uint32_t first,
                                                     uint32_t step) {
    // nibble l: producer-order rank of level l (8 = not a producer level)
    uint32_t rank_of = 0x88888888u;
    const uint32_t used = taps_popc(P.pru);
    for (uint32_t k = 0; k < used; ++k) {
        const uint32_t l = taps_rank_level(P, k);
        rank_of = (rank_of & ~(15u << (4u * l))) | (k << (4u * l));
    }
    for (uint32_t x = first; x < 256u; x += step) {
        uint32_t y = 0;
#pragma unroll
        for (uint32_t l = 0; l < TAPS_D_MAX_LEVELS; ++l)
            if ((x >> l) & 1u) y |= (1u << ((rank_of >> (4u * l)) & 15u)) & 0xFFu;
        tab[x] = (uint8_t)y;
    }
}

// Dimensions d >= rank are left as they come (nothing reads them).
__host__ __device__ inline void taps_make_col(taps_col &Q, const taps_desc &D, uint32_t axes,
                                              uint32_t rank) {
    (void)rank;
    Q.ccuts = D.cuts;
#pragma unroll
    for (uint32_t d = 0; d < TAPS_D_MAX_RANK; ++d) {
        const uint32_t a = taps_nib(axes, d);
        const uint32_t lo = taps_nib(D.lo, a), w = taps_nib(D.width, a);
        Q.cw[d] = w;
        Q.clo[d] = lo;
        Q.cr8[d] = taps_bfm(w, lo + 8u);
    }
}

// ---------------------------------------------------------------------------
// Link-class hierarchies (an extension of the paper's two classes).
//
// Blocks of 2^beta_0 <= 2^beta_1 <= ... consecutive ranks (a node, a group of
// nodes, ...; the last class spans all devices).  A collective belongs to
// the smallest block that holds each of its groups: with top level t that is
// class c = the number of boundaries beta <= t; it pays bw[c] divided by the
// number of groups sharing the uplink of one block of the largest boundary
// beta <= t (Algorithm 2 / 3 and the AllToAll paragraph with "node" read as
// that block).  With one boundary (beta = lam) this is the two-class model.
// Every collective is costed on its own (no closed forms over the node
// boundary); volumes are the same factor units as above, accumulated per
// class, and candidates compare by the exact key sum_c x_c w_c with
// w_c = lcm(bw) / bw_c.
// ---------------------------------------------------------------------------
struct taps_hier {
    uint32_t n_classes;     // 1 .. TAPS_D_MAX_CLASSES
    uint32_t cls_of_top;    // nibble t: class of a collective whose top level is t
    uint32_t beta_of_top;   // nibble t: the largest boundary <= t (0 for class 0)
    uint32_t pad;
    uint64_t w[TAPS_D_MAX_CLASSES];        // exact-order weights, each below 2^30
    double inv_n_bw[TAPS_D_MAX_CLASSES];   // 1 / (N bw[c])
    uint64_t w_a2a;          // weight of the in-block AllToAll volume (0: priced as class 0)
    double inv_n_bw_a2a;     // 1 / (N bw_a2a)
    uint32_t a2a_own;        // 1: in-block AllToAlls go to xa at their own bandwidth
    uint32_t pad2;
    uint32_t levels_of_cls[TAPS_D_MAX_CLASSES];   // bit l: cls_of_top's nibble l is c
    uint32_t beta_of_cls[TAPS_D_MAX_CLASSES];     // the boundary of class c (0 for class 0)
};

// One candidate in factor units, per link class (x0: inside the innermost block).
// ct: the sum of the inter-block group counts of its collectives (the number
// of collectives and of inter-block ones is the same for every candidate, as
// for taps_fac: taps_collectives_h).
struct taps_fach {
    uint32_t vol, x0, x1, x2, x3;
    uint32_t xa;   // in-block AllToAll volume priced at its own bandwidth
    uint32_t ct;
};

__host__ __device__ inline void taps_fac_zero(taps_fach &c) {
    c.vol = c.x0 = c.x1 = c.x2 = c.x3 = c.xa = 0;
    c.ct = 0;
}

// x_cls += v (selects, no indexed register arrays).  C: the hierarchy's
// number of classes (every class index is below it, so x_C .. x_3 stay 0 and
// are not touched).
template <uint32_t C = TAPS_D_MAX_CLASSES>
__host__ __device__ inline void taps_fach_add(taps_fach &c, uint32_t cls, uint32_t v) {
    c.x0 += cls == 0 ? v : 0u;
    if (C > 1) c.x1 += cls == 1 ? v : 0u;
    if (C > 2) c.x2 += cls == 2 ? v : 0u;
    if (C > 3) c.x3 += cls == 3 ? v : 0u;
}

template <uint32_t C = TAPS_D_MAX_CLASSES>
__host__ __device__ inline uint64_t taps_fach_key(const taps_fach &c, const taps_hier &H) {
    uint64_t k = (uint64_t)c.x0 * H.w[0];
    if (C > 1) k += (uint64_t)c.x1 * H.w[1];
    if (C > 2) k += (uint64_t)c.x2 * H.w[2];
    if (C > 3) k += (uint64_t)c.x3 * H.w[3];
    return k + (uint64_t)c.xa * H.w_a2a;
}

// The shared uplinks of a collective of width w at lowest level lo whose
// class is cls under the boundary beta: 2^lct groups, with the free levels
// below min(lo, beta) letting replicas share one transfer (Algorithm 3).
__host__ __device__ inline uint32_t taps_hier_lct(uint32_t lo, uint32_t beta, uint32_t unused) {
    const uint32_t m = lo < beta ? lo : beta;
    return m - taps_popc(unused & taps_below(m));
}

template <uint32_t C>
struct taps_hier_model_t {
    using fac = taps_fach;
    const taps_hier *H;
    uint64_t lim_key;   // a later candidate stops once its key and volume reach these
    uint32_t lim_vol;
    bool lim_on;
    const taps_pair *a2a_cls;   // the row's AllToAll tables by class (taps_row)
    const taps_pair *expand;

    // AllGather (Eq. 9) of the axis with top level `top`.
    __host__ __device__ void gather(fac &c, uint32_t top, const taps_ax &a, uint32_t sh,
                                    uint32_t unused) const {
        const uint32_t V = taps_bfm(a.w, sh);
        const uint32_t cls = taps_nib_at(H->cls_of_top, top);
        const uint32_t lct = cls ? taps_hier_lct(a.lo, taps_nib_at(H->beta_of_top, top), unused) : 0u;
        c.vol += V;
        taps_fach_add<C>(c, cls, V << lct);
        c.ct += cls ? taps_bit16(lct) : 0u;
    }

    // AllToAlls (Eq. 10, Eq. 14) of every axis whose top is in x, at one state:
    // k = 2^kap members of a group inside one block of the boundary beta, the
    // uplink carries k (p - k) / p of the shard per group.
    //
    // An axis whose levels all lie at or above its class's boundary (kap = 0)
    // sends its whole V = 2^sh - 2^(sh - w) over its class's link, with the
    // group count the free levels below the boundary give every such axis of
    // the class: per class, sum V = n 2^sh - 2^(sh - 8) sum 2^(8 - w), the last
    // sum one byte dot product per half against a table of the row's tops
    // split by class (as taps_a2a_batch).  Only the lowest axis of a class can
    // reach below its boundary (when the level under the boundary is not a
    // top); those axes (at most one per class) are costed one by one.
    __host__ __device__ void a2a(fac &c, uint32_t x, const taps_lv &L, uint32_t sh,
                                 uint32_t unused) const {
        uint32_t cross = 0;
#pragma unroll
        for (uint32_t k = 1; k < C; ++k) {
            const uint32_t b = H->beta_of_cls[k];   // uniform
            if (b == 0) continue;                   // nothing reaches below level 0
            const uint32_t low_top = L.tp & H->levels_of_cls[k];
            cross |= (low_top & (0u - low_top)) & (((L.tp >> (b - 1u)) & 1u) - 1u);
        }
        const uint32_t m = x & ~cross;
        const taps_pair X = taps_entry<3>(expand, m);
        static_assert(sizeof(taps_pair) * TAPS_D_MAX_CLASSES == 32u, "class table row");
        const taps_pair *W = (const taps_pair *)((const char *)a2a_cls + taps_shl16c<5>(L.tp));
        const uint32_t e = sh - 8u;
#pragma unroll
        for (uint32_t k = 0; k < C; ++k) {
            const uint32_t mk = m & H->levels_of_cls[k];
            const uint32_t nk = taps_popc(mk);
            const uint32_t f = taps_dot4(W[k].hi, X.hi, taps_dot4(W[k].lo, X.lo, 0u));
            const uint32_t sum = (nk << sh) - (f << e);
            c.vol += sum;
            if (k == 0) {
                c.x0 += H->a2a_own ? 0u : sum;
                c.xa += H->a2a_own ? sum : 0u;
                continue;
            }
            const uint32_t b = H->beta_of_cls[k];
            const uint32_t lct = b - taps_popc(unused & taps_below(b));
            taps_fach_add<C>(c, k, sum << lct);
            c.ct += nk << lct;
        }
        for (uint32_t r = x & cross; r; r &= r - 1u) {
            const uint32_t top = taps_ctz(r);
            const taps_ax a = taps_axis(L, top);
            const uint32_t V = (1u << sh) - (1u << (sh - a.w));
            const uint32_t cls = taps_nib_at(H->cls_of_top, top);
            const uint32_t beta = taps_nib_at(H->beta_of_top, top);
            const uint32_t kap = beta - a.lo;   // lo < beta for a crossing axis
            const uint32_t link = ((1u << a.w) - (1u << kap)) << (kap + sh - a.w);
            const uint32_t lct = taps_hier_lct(a.lo, beta, unused);
            c.vol += V;
            taps_fach_add<C>(c, cls, link << lct);
            c.ct += 1u << lct;
        }
    }

    __host__ __device__ bool hopeless(const fac &c) const {
        return lim_on && ((c.vol >= lim_vol) & (taps_fach_key<C>(c, *H) >= lim_key));
    }
};
using taps_hier_model = taps_hier_model_t<TAPS_D_MAX_CLASSES>;

// "remove" (Table 2): every held axis not at its target gathered in producer
// order (dimensions ascending, each from its top level down), one by one.
template <class Mh>
__host__ __device__ inline taps_fach taps_remove_h(const taps_row &P, const taps_lv &L,
                                                   const Mh &M) {
    taps_fach c;
    taps_fac_zero(c);
    uint32_t sh = P.e0 + 8u, unused = P.full & ~P.pru;
    for (uint32_t x = P.to_rank[L.src & ~L.home]; x; x &= x - 1u) {
        const uint32_t top = taps_rank_level(P, taps_ctz(x));
        const taps_ax a = taps_axis(L, top);
        M.gather(c, top, a, sh, unused);
        unused |= a.lv;
        sh += a.w;
    }
    return c;
}

struct taps_pickh {
    taps_fach best;
    uint32_t vmin, cand;
    uint32_t coll;   // taps_collectives_h
    bool ok;
};

// Collectives of every candidate of an entry (bits 0-7) and the inter-block
// ones among them (bits 8-15): one per axis held off its target, inter-block
// when its top is in a class above 0.
__host__ __device__ inline uint32_t taps_collectives_h(const taps_lv &L, const taps_hier &H) {
    const uint32_t x = L.src & ~L.home;
    return taps_popc(x) | (taps_popc(x & ~H.levels_of_cls[0]) << 8);
}

// The cheapest of Algorithm 1, the same without AllToAll, and "remove" under
// the link classes of H (ties to the lower index); vmin the smallest volume.
template <uint32_t C = TAPS_D_MAX_CLASSES>
__host__ __device__ inline taps_pickh taps_edge_select_h(const taps_row &P, const taps_col &Q,
                                                         const taps_hier &H) {
    taps_lv L;
    taps_unify(P, Q, L);
    taps_hier_model_t<C> M{&H, 0, 0, false, P.a2a_cls, P.expand};
    const taps_start b = taps_begin(P, L);
    const taps_run_t<taps_fach> r0 = taps_alg1_t(P, Q, L, M, b);
    taps_pickh k;
    k.best = r0.c;
    k.cand = 0;
    k.vmin = r0.c.vol;
    k.coll = taps_collectives_h(L, H);
    k.ok = r0.ok;
    uint64_t best_key = taps_fach_key<C>(r0.c, H);
    if (r0.a2a_tops) {   // without AllToAll the sequence would be the same
        M.lim_on = true;
        M.lim_key = best_key;
        M.lim_vol = k.vmin;
        const taps_run_t<taps_fach> r1 = taps_rearrange_t(P, Q, L, M, b);
        if (!r1.stopped) {
            const uint64_t k1 = taps_fach_key<C>(r1.c, H);
            if (k1 < best_key) {
                k.best = r1.c;
                k.cand = 1;
                best_key = k1;
            }
            k.vmin = r1.c.vol < k.vmin ? r1.c.vol : k.vmin;
        }
        M.lim_on = false;
    }
    const taps_fach c2 = taps_remove_h(P, L, M);
    if (taps_fach_key<C>(c2, H) < best_key) {
        k.best = c2;
        k.cand = 2;
    }
    k.vmin = c2.vol < k.vmin ? c2.vol : k.vmin;
    return k;
}

__host__ __device__ inline taps_entry_out taps_entry_finish_h(const taps_pickh &k,
                                                              const taps_scaler &S,
                                                              const taps_hier &H) {
    taps_entry_out o;
    const double unit = (double)S.tbytes * (1.0 / 256.0);
    o.vol = taps_scale(S, k.vmin);
    o.intra = taps_scale(S, k.best.x0) + taps_scale(S, k.best.xa);
    o.inter = taps_scale(S, k.best.x1) + taps_scale(S, k.best.x2) + taps_scale(S, k.best.x3);
    o.t = (double)k.best.x0 * (unit * H.inv_n_bw[0]) + (double)k.best.x1 * (unit * H.inv_n_bw[1]) +
          (double)k.best.x2 * (unit * H.inv_n_bw[2]) + (double)k.best.x3 * (unit * H.inv_n_bw[3]) +
          (double)k.best.xa * (unit * H.inv_n_bw_a2a);
    o.meta = k.cand | ((k.coll & 0xFFu) << 2) | ((k.coll >> 8) << 7) | (k.best.ct << 12);
    o.ok = k.ok;
    return o;
}

// Intra-op AllReduce (Eq. 5-8) of a tensor missing the levels `missing`,
// under link classes: nb volumes per class.
struct taps_acch {
    uint64_t vol, x0, x1, x2, x3;
    uint32_t n_coll, n_inter, sum_ct;
};

__host__ __device__ inline void taps_allreduce_h(taps_acch &c, uint32_t missing, uint64_t bytes,
                                                 const taps_hier &H) {
    if (!missing) return;
    const uint32_t lg = taps_popc(missing);
    const uint64_t V = ((bytes << lg) - bytes) << 1;   // 2 (g - 1) |tensor| bytes, in nb
    const uint32_t top = taps_msb(missing);
    const uint32_t cls = taps_nib(H.cls_of_top, top);
    c.vol += V;
    c.n_coll += 1;
    if (!cls) {
        c.x0 += V;
        return;
    }
    const uint32_t beta = taps_nib(H.beta_of_top, top);
    const uint32_t lct = beta - taps_popc(missing & taps_below(beta));
    const uint64_t X = V << lct;
    c.x1 += cls == 1 ? X : 0u;
    c.x2 += cls == 2 ? X : 0u;
    c.x3 += cls == 3 ? X : 0u;
    c.n_inter += 1;
    c.sum_ct += 1u << lct;
}

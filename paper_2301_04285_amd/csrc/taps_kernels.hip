// taps_kernels.hip -- gfx950 kernels of the TAPS cost tables.
//
//   k_build_strategies  one workgroup per chunk of 256 candidate ranks of an
//                 operator: GenerateStrategySet in canonical order at
//                 host-counted offsets (ballot, LDS scan), optionally each
//                 strategy's descriptor and node record
//   k_describe    one thread per strategy: level runs, owners and cuts
//   k_node_costs  one thread per strategy: the intra-op AllReduces
//   k_memory_costs one thread per strategy: weight and output shard bytes
//   k_edge_plan   one thread per edge (its constants), then one thread per
//                 row segment (its edge, producer strategy and consumer
//                 range: every edge's full-length segments first, the rows'
//                 remainders last, longest first)
//   k_build_front k_build_strategies and k_edge_plan in one launch
//   k_edge_costs  one wavefront per row segment (one producer strategy,
//                 uniform: its descriptor sits in scalar registers; 2 or 8
//                 tiles of 64 consumer strategies, one per lane, the
//                 next 64 prefetched), TAPS_ROWS_PER_BLOCK segments per workgroup; five
//                 coalesced SoA stores per entry
//   k_edge_costs_sweep_win  several bandwidth points: one wavefront per
//                 aligned 64-entry window of the tables (row by row where a
//                 window crosses rows), the candidates once per entry, one
//                 selection and store per point; k_window_edges maps windows
//                 to edges
//   k_copy_tables shared tables: one workgroup per chunk of a computed
//                 table, written to every table that shares it
//   k_pull        a call's upload, read from pinned host memory
#include "taps_internal.h"

namespace {

constexpr uint32_t kWave = 64;

// Completion counts w(k, s, z) for k, s, z in 0..8 (see taps_completions),
// evaluated by the compiler.
__constant__ taps_completion_table kCompletions = taps_make_completions();
// Widths of unified axes by their tops (taps_make_widths), copied to LDS by the
// edge kernels.
__constant__ taps_width_table kWidths = taps_make_widths();
// AllToAll shard fractions by tops mask and masks as bytes (taps_make_a2a,
// taps_make_expand), copied to LDS by the two-class edge kernels.
__constant__ taps_a2a_table kA2a = taps_make_a2a();
__constant__ taps_expand_table kExpand = taps_make_expand();

// The per-workgroup LDS tables of the two-class AllToAll costing: the shard
// fractions split at the node boundary lam (bytes below lam: in-node tops).
__device__ inline void fill_a2a_tables(taps_a2a_row *a2a, taps_pair *expand, uint32_t lam) {
    const uint32_t in_lo = lam >= 4u ? ~0u : (1u << (8u * lam)) - 1u;
    const uint32_t in_hi = lam <= 4u ? 0u : lam >= 8u ? ~0u : (1u << (8u * (lam - 4u))) - 1u;
    for (uint32_t x = threadIdx.x; x < 256u; x += blockDim.x) {
        const uint32_t lo = kA2a.lo[x], hi = kA2a.hi[x];
        a2a[x] = taps_a2a_row{lo, hi, lo & in_lo, hi & in_hi};
        expand[x] = taps_pair{kExpand.lo[x], kExpand.hi[x]};
    }
}

// The per-workgroup LDS tables of the link-class AllToAll costing: per tops
// mask, the shard-fraction bytes of the tops in each class (a level's byte
// kept where the level's class is c).
__device__ inline void fill_a2a_class_tables(taps_pair *a2a_cls, taps_pair *expand,
                                             const taps_hier &H) {
    uint32_t lo_mask[TAPS_D_MAX_CLASSES], hi_mask[TAPS_D_MAX_CLASSES];
#pragma unroll
    for (uint32_t c = 0; c < TAPS_D_MAX_CLASSES; ++c) {
        const uint32_t m = c < H.n_classes ? H.levels_of_cls[c] & 0xFFu : 0u;
        lo_mask[c] = kExpand.lo[m] * 0xFFu;
        hi_mask[c] = kExpand.hi[m] * 0xFFu;
    }
    for (uint32_t x = threadIdx.x; x < 256u; x += blockDim.x) {
        const uint32_t lo = kA2a.lo[x], hi = kA2a.hi[x];
#pragma unroll
        for (uint32_t c = 0; c < TAPS_D_MAX_CLASSES; ++c)
            a2a_cls[x * TAPS_D_MAX_CLASSES + c] = taps_pair{lo & lo_mask[c], hi & hi_mask[c]};
        expand[x] = taps_pair{kExpand.lo[x], kExpand.hi[x]};
    }
}

template <typename T>
__device__ inline T *at_byte(T *base, uint32_t offset) {
    return (T *)((char *)base + offset);
}

// Entry j of a row whose records start at `row` (uniform): 32-bit byte offsets
// from the uniform row bases, j < 2^21 (8 axes on 8 levels give at most
// 1,047,376 strategies per operator); five cached stores (L2 merges the
// partial 128-byte lines where neighbouring segments meet; measured faster
// than non-temporal stores, by a third on the stores alone).
__device__ inline void store_entry(const taps_table &out, uint64_t row, uint32_t j,
                                   const taps_entry_out &o, uint32_t meta) {
    const uint32_t o8 = j * 8u, o4 = j * 4u;
    *at_byte(out.t + row, o8) = o.t;
    *at_byte(out.vol + row, o8) = o.vol;
    *at_byte(out.intra + row, o8) = o.intra;
    *at_byte(out.inter + row, o8) = o.inter;
    *at_byte(out.meta + row, o4) = meta;
}

__device__ inline uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__global__ __launch_bounds__(256) void k_describe(const taps_strategy *__restrict__ s,
                                                  uint64_t total, taps_desc *__restrict__ desc) {
    const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const taps_strategy st = s[idx];
    uint32_t expo[TAPS_D_MAX_AXES];
    int32_t pos[TAPS_D_MAX_AXES];
#pragma unroll
    for (uint32_t a = 0; a < TAPS_D_MAX_AXES; ++a) {
        expo[a] = st.log2_deg[a];
        pos[a] = st.pos[a];
    }
    desc[idx] = taps_describe(TAPS_D_MAX_AXES, expo, pos);
}

// largest k in [0, n) with offsets[k] <= x
__device__ inline uint32_t find_owner(const uint64_t *offsets, uint32_t n, uint64_t x) {
    uint32_t lo = 0, hi = n;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (offsets[mid] <= x)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__device__ inline void node_tensor(taps_acc &c, const taps_op &op, const taps_tensor &t,
                                   const taps_desc &D, uint32_t full, uint32_t lam) {
    uint32_t used = 0;
    uint64_t bytes = op.dtype_bytes;
    for (uint32_t d = 0; d < t.rank && d < TAPS_MAX_RANK; ++d) {
        const uint32_t a = t.axis[d] & 7u;
        used |= taps_levels(taps_nib(D.lo, a), taps_nib(D.width, a));
        bytes *= (uint64_t)op.axis_len[a];
    }
    taps_allreduce(c, full & ~used, bytes, lam);
}

__global__ __launch_bounds__(256) void k_node_costs(const taps_op *__restrict__ ops, uint32_t n_ops,
                                                    const uint64_t *__restrict__ offsets,
                                                    const taps_desc *__restrict__ desc,
                                                    uint64_t total, taps_launch lp, taps_table out) {
    const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const taps_op &op = ops[find_owner(offsets, n_ops, idx)];
    const taps_desc D = desc[idx];
    const uint32_t full = taps_low_mask(lp.n);
    taps_acc c;
    taps_acc_zero(c);
    node_tensor(c, op, op.out, D, full, lp.lam);
    for (uint32_t k = 0; k < op.n_in && k < TAPS_MAX_INPUTS; ++k)
        node_tensor(c, op, op.in[k], D, full, lp.lam);
    for (uint32_t k = 0; k < op.n_w && k < TAPS_MAX_WEIGHTS; ++k)
        node_tensor(c, op, op.w[k], D, full, lp.lam);
    out.t[idx] = (double)c.intra * lp.inv_n_bintra + (double)c.inter * lp.inv_n_binter;
    out.vol[idx] = c.vol;
    out.intra[idx] = c.intra;
    out.inter[idx] = c.inter;
    out.meta[idx] = taps_meta(0, c);
}

// GenerateStrategySet, and the whole strategy side of a single-call build, in
// one launch: one workgroup per chunk of 256 consecutive candidate ranks of
// one operator (only chunks that hold a strategy are launched) tests its
// candidates in canonical order (a ballot per wavefront, the four wavefront
// counts scanned in LDS) and writes every valid strategy together with, when
// asked (desc and node.t not NULL), its descriptor and its node (intra-op)
// record.  A chunk's strategies go to [base, base + count), where the host
// counted them with the same unranking and filter (plan_build checks the
// chunks' counts against the exact per-operator count); nothing is written
// outside that range.
constexpr uint32_t kBuildThreads = TAPS_BUILD_CHUNK;

// The strategies of one chunk of candidate ranks (a whole workgroup).
__device__ inline void build_chunk(const taps_build_chunk &ck, const taps_op *__restrict__ ops,
                                   uint32_t allowed_cuts, const taps_launch &lp,
                                   taps_strategy *__restrict__ out, taps_desc *__restrict__ desc,
                                   const taps_table &node) {
    __shared__ uint32_t W[9 * 9 * 9];
    __shared__ uint32_t wave_count[kBuildThreads / kWave];
    const uint32_t tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    for (uint32_t x = tid; x < 9u * 9u * 9u; x += blockDim.x) W[x] = kCompletions.v[x];
    __syncthreads();
    const taps_op &op = ops[ck.op];
    const uint32_t n_axes = op.n_axes, part = op.part_mask;
    const uint32_t total = W[(taps_popc(part) * 9u + lp.n) * 9u];
    const uint32_t full = taps_low_mask(lp.n);
    const uint32_t r = ck.first + tid;
    uint32_t expo[TAPS_D_MAX_AXES];
    int32_t pos[TAPS_D_MAX_AXES];
    bool valid = r < total && taps_unrank(n_axes, part, lp.n, r, W, expo, pos);
    if (valid)
        for (uint32_t a = 0; a < n_axes; ++a)
            if (op.axis_len[a] & (((int64_t)1 << expo[a]) - 1)) valid = false;
    taps_desc D = {0u, 0u, 0u, 0u};
    if (valid) {
        D = taps_describe(n_axes, expo, pos);
        if (D.cuts & ~allowed_cuts) valid = false;
    }
    const uint64_t m = __ballot(valid);
    if (lane == 0) wave_count[wave] = (uint32_t)__builtin_popcountll(m);
    __syncthreads();
    uint32_t before = 0;
    for (uint32_t w = 0; w < wave; ++w) before += wave_count[w];
    const uint32_t k = before + lanes_below(m);
    if (valid && k < ck.count) {
        const uint64_t idx = ck.base + k;
        taps_strategy st;
        for (uint32_t a = 0; a < TAPS_MAX_AXES; ++a) {
            st.log2_deg[a] = a < n_axes ? (uint8_t)expo[a] : 0;
            st.pos[a] = a < n_axes ? (int8_t)pos[a] : (int8_t)-1;
        }
        out[idx] = st;
        if (desc) desc[idx] = D;   // uniform: descriptors and node records are optional
        if (node.t) {
            taps_acc c;
            taps_acc_zero(c);
            node_tensor(c, op, op.out, D, full, lp.lam);
            for (uint32_t q = 0; q < op.n_in && q < TAPS_MAX_INPUTS; ++q)
                node_tensor(c, op, op.in[q], D, full, lp.lam);
            for (uint32_t q = 0; q < op.n_w && q < TAPS_MAX_WEIGHTS; ++q)
                node_tensor(c, op, op.w[q], D, full, lp.lam);
            node.t[idx] = (double)c.intra * lp.inv_n_bintra + (double)c.inter * lp.inv_n_binter;
            node.vol[idx] = c.vol;
            node.intra[idx] = c.intra;
            node.inter[idx] = c.inter;
            node.meta[idx] = taps_meta(0, c);
        }
    }
}

__global__ __launch_bounds__(kBuildThreads) void k_build_strategies(
    const taps_op *__restrict__ ops, const taps_build_chunk *__restrict__ chunks,
    uint32_t allowed_cuts, taps_launch lp, taps_strategy *__restrict__ out,
    taps_desc *__restrict__ desc, taps_table node) {
    build_chunk(chunks[blockIdx.x], ops, allowed_cuts, lp, out, desc, node);
}

// Bytes of one shard of tensor t under strategy s: each dimension's length
// divided by its split degree, times the element size.
__device__ inline uint64_t shard_bytes(const taps_op &op, const taps_tensor &t,
                                       const taps_strategy &s) {
    uint64_t b = op.dtype_bytes;
    for (uint32_t d = 0; d < t.rank && d < TAPS_MAX_RANK; ++d) {
        const uint32_t a = t.axis[d] & 7u;
        const uint32_t e = s.pos[a] >= 0 ? (s.log2_deg[a] & 15u) : 0u;
        b *= (uint64_t)op.axis_len[a] >> e;
    }
    return b;
}

__global__ __launch_bounds__(256) void k_memory_costs(const taps_op *__restrict__ ops,
                                                      uint32_t n_ops,
                                                      const uint64_t *__restrict__ offsets,
                                                      const taps_strategy *__restrict__ strategies,
                                                      uint64_t total, uint64_t *__restrict__ memory) {
    const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const taps_op &op = ops[find_owner(offsets, n_ops, idx)];
    const taps_strategy s = strategies[idx];
    uint64_t m = shard_bytes(op, op.out, s);
    for (uint32_t k = 0; k < op.n_w && k < TAPS_MAX_WEIGHTS; ++k) m += shard_bytes(op, op.w[k], s);
    memory[idx] = m;
}

// Per-edge constants of edge e.
__device__ inline void edge_setup_one(uint32_t e, const taps_plan_args &pa, const taps_launch &lp) {
    const taps_edge E = pa.edges[e];
    const taps_op &src = pa.ops[E.src_op];
    const taps_op &dst = pa.ops[E.dst_op];
    const taps_tensor &T = src.out;
    const taps_tensor &Tc = dst.in[E.dst_slot];
    taps_edge_params p;
    p.out_offset = pa.edge_offsets[e];
    uint64_t bytes = src.dtype_bytes;
    uint32_t pax = 0, cax = 0;
    for (uint32_t d = 0; d < T.rank && d < TAPS_MAX_RANK; ++d) {
        bytes *= (uint64_t)src.axis_len[T.axis[d] & 7u];
        pax |= (uint32_t)(T.axis[d] & 7u) << (4u * d);
        cax |= (uint32_t)(Tc.axis[d] & 7u) << (4u * d);
    }
    p.scale = taps_make_scaler(bytes, lp.inv_n_bintra, lp.inv_n_binter);
    // the source side of the redistribution: the producer's output map, or for
    // the backward tables the consumer's input map (the gradient moves back)
    const uint32_t from = pa.reverse ? E.dst_op : E.src_op, to = pa.reverse ? E.src_op : E.dst_op;
    p.src_base = (uint32_t)pa.op_offsets[from];
    p.dst_base = (uint32_t)pa.op_offsets[to];
    p.ns = (uint32_t)(pa.op_offsets[from + 1] - pa.op_offsets[from]);
    p.nd = (uint32_t)(pa.op_offsets[to + 1] - pa.op_offsets[to]);
    p.rank = T.rank;
    p.paxes = pa.reverse ? cax : pax;
    p.caxes = pa.reverse ? pax : cax;
    p.pad = 0;
    pa.params[e] = p;
}

// Row segment r: its edge, producer strategy and consumer range (from the
// strategy offsets, so it does not wait for the edge constants).
__device__ inline void row_map_one(uint64_t r, const taps_plan_args &pa) {
    // the last group starting at or before r (groups[0].start == 0)
    uint32_t lo = 0, hi = pa.n_groups - 1;
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) / 2;
        if (pa.groups[mid].start <= r)
            lo = mid;
        else
            hi = mid - 1;
    }
    const taps_seg_group G = pa.groups[lo];
    const taps_edge E = pa.edges[G.edge];
    const uint32_t from = pa.reverse ? E.dst_op : E.src_op, to = pa.reverse ? E.src_op : E.dst_op;
    const uint32_t nd = (uint32_t)(pa.op_offsets[to + 1] - pa.op_offsets[to]);
    const uint64_t k = r - G.start;
    taps_row_ref ref;
    ref.edge = G.edge;
    ref.strategy = (uint32_t)(pa.op_offsets[from] + k / G.per_row);
    ref.first_col = G.first_col + (uint32_t)(k % G.per_row) * G.cols;
    ref.last_col = nd - ref.first_col < G.cols ? nd : ref.first_col + G.cols;
    pa.segs[r] = ref;
}

// The edge plan in one launch: blocks [0, setup_blocks) set up the edges, the
// rest map the row segments.
__global__ __launch_bounds__(256) void k_edge_plan(taps_plan_args pa, taps_launch lp,
                                                   uint32_t setup_blocks) {
    if (blockIdx.x < setup_blocks) {
        const uint32_t e = blockIdx.x * blockDim.x + threadIdx.x;
        if (e < pa.n_edges) edge_setup_one(e, pa, lp);
    } else {
        const uint64_t r = (uint64_t)(blockIdx.x - setup_blocks) * blockDim.x + threadIdx.x;
        if (r < pa.n_segs) row_map_one(r, pa);
    }
}

// The front of a single-call build: the strategy chunks, then the edge plan
// (the edge setup and the row map need only the strategy offsets, which the
// host counted), in one launch.
__global__ __launch_bounds__(kBuildThreads) void k_build_front(
    const taps_build_chunk *__restrict__ chunks, uint32_t n_chunks, uint32_t allowed_cuts,
    taps_launch lp, taps_strategy *__restrict__ out, taps_desc *__restrict__ desc,
    taps_table node, taps_plan_args pa, uint32_t setup_blocks) {
    if (blockIdx.x < n_chunks) {
        build_chunk(chunks[blockIdx.x], pa.ops, allowed_cuts, lp, out, desc, node);
        return;
    }
    const uint32_t b = blockIdx.x - n_chunks;
    if (b < setup_blocks) {
        const uint32_t e = b * blockDim.x + threadIdx.x;
        if (e < pa.n_edges) edge_setup_one(e, pa, lp);
    } else {
        const uint64_t r = (uint64_t)(b - setup_blocks) * blockDim.x + threadIdx.x;
        if (r < pa.n_segs) row_map_one(r, pa);
    }
}

// R: the launch's tensors have rank R at most; Narrow: both reduced
// bandwidths are below 2^32 (64-bit keys), so the other order is not compiled.
template <uint32_t R, bool Narrow>
__global__ __launch_bounds__(TAPS_TILE_COLS *TAPS_ROWS_PER_BLOCK) void k_edge_costs(
    const taps_edge_params *__restrict__ params, const taps_row_ref *__restrict__ rows,
    uint32_t n_segs, const taps_desc *__restrict__ desc, taps_launch lp, taps_table out) {
    __shared__ uint8_t rank_tab[TAPS_ROWS_PER_BLOCK][256];
    __shared__ uint32_t width_tab[256];
    __shared__ taps_a2a_row a2a_tab[256];
    __shared__ taps_pair expand_tab[256];
    const uint32_t lane = threadIdx.x % TAPS_TILE_COLS;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / TAPS_TILE_COLS);
    const uint32_t r = blockIdx.x * TAPS_ROWS_PER_BLOCK + wave;
    const bool live = r < n_segs;
    const taps_row_ref ref = rows[live ? r : 0u];
    const taps_edge_params E = params[ref.edge];
    __builtin_assume(E.rank <= R);   // the launch's tensors have rank R at most
    const taps_desc Dp = desc[ref.strategy];
    const uint32_t i = ref.strategy - E.src_base;
    taps_row P;
    taps_make_row(P, Dp, E.paxes, E.rank, lp.n, lp.lam);
    taps_fill_rank_table(P, rank_tab[wave], lane, TAPS_TILE_COLS);
    fill_a2a_tables(a2a_tab, expand_tab, lp.lam);
    for (uint32_t x = threadIdx.x; x < 256u; x += blockDim.x) width_tab[x] = kWidths.v[x];
    __syncthreads();
    if (!live) return;
    P.to_rank = rank_tab[wave];
    P.widths = width_tab;
    P.a2a = a2a_tab;
    P.expand = expand_tab;
    taps_keys K;
    K.b_inter_red = lp.b_inter_red;
    K.b_intra_red = lp.b_intra_red;
    K.narrow = Narrow;
    // the row's records start here; lane j writes entry j
    const uint64_t row_out = E.out_offset + (uint64_t)i * E.nd;
    const taps_desc *col = desc + E.dst_base;
    const uint32_t c0 = ref.first_col;
    const uint32_t c1 = ref.last_col;
    // consumer descriptors one tile ahead
    taps_desc next = col[c0 + lane < c1 ? c0 + lane : c0];
    for (uint32_t j0 = c0; j0 < c1; j0 += TAPS_TILE_COLS) {
        const taps_desc cur = next;
        const uint32_t j = j0 + lane;
        const uint32_t jn = j + TAPS_TILE_COLS;
        if (jn < c1) next = col[jn];
        if (j < c1) {
            taps_col Q;
            taps_make_col(Q, cur, E.caxes, E.rank);
            const taps_entry_out o = taps_entry_finish(taps_edge_select(P, Q, K), E.scale);
            store_entry(out, row_out, j, o, o.ok ? o.meta : 0xFFFFFFFFu);
        }
    }
}

// Several bandwidth points: the candidates of each entry are costed once and
// selected, scaled and stored once per point.
//
// The sweep runs over aligned windows: wavefront w handles the entries
// [64 T w, 64 T (w + 1)) of the concatenated tables (T = TAPS_WIN_TILES), one
// 64-entry tile at a time (lane l entry 64 t + l of the tile), so every store
// covers whole 128-byte lines (store-only kernels of the sweep's four tables:
// 5.75 TB/s this way against 2.7-3.4 TB/s for row segments that start inside a
// line).  A tile that crosses rows (or edges) is taken row by row; the
// wavefront builds a row's producer side once and keeps it while the row
// continues into the next tile.  win_edge[w] is the edge holding entry 64 T w.
__global__ void k_window_edges(const uint64_t *__restrict__ eoff, uint32_t n_edges,
                               uint64_t n_windows, uint32_t *__restrict__ win_edge) {
    const uint64_t w = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= n_windows) return;
    const uint64_t g = w * (TAPS_TILE_COLS * TAPS_WIN_TILES);
    // the last edge e with eoff[e] <= g (edges without entries share an offset
    // with the next one, so this is the edge that holds g)
    uint32_t lo = 0, hi = n_edges;   // eoff[lo] <= g < eoff[hi]
    while (hi - lo > 1u) {
        const uint32_t mid = (lo + hi) / 2u;
        if (eoff[mid] <= g) lo = mid; else hi = mid;
    }
    win_edge[w] = lo;
}

template <uint32_t R, bool Narrow>
__global__ __launch_bounds__(TAPS_TILE_COLS *TAPS_ROWS_PER_BLOCK) void k_edge_costs_sweep_win(
    const taps_edge_params *__restrict__ params, uint32_t n_edges,
    const uint32_t *__restrict__ win_edge, uint64_t n_windows, uint64_t total,
    const taps_desc *__restrict__ desc, taps_launch lp, taps_sweep sw) {
    __shared__ uint8_t rank_tab[TAPS_ROWS_PER_BLOCK][256];
    __shared__ uint32_t width_tab[256];
    __shared__ taps_a2a_row a2a_tab[256];
    __shared__ taps_pair expand_tab[256];
    const uint32_t lane = threadIdx.x % TAPS_TILE_COLS;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / TAPS_TILE_COLS);
    const uint64_t w = (uint64_t)blockIdx.x * TAPS_ROWS_PER_BLOCK + wave;
    fill_a2a_tables(a2a_tab, expand_tab, lp.lam);
    for (uint32_t x = threadIdx.x; x < 256u; x += blockDim.x) width_tab[x] = kWidths.v[x];
    __syncthreads();
    if (w >= n_windows) return;
    taps_keys any;
    any.b_inter_red = sw.b_inter_red[0];
    any.b_intra_red = sw.b_intra_red[0];
    any.narrow = sw.narrow[0] != 0;
    // the window: TAPS_WIN_TILES aligned tiles of 64 entries, [g_begin, g_end)
    const uint64_t g_begin = w * (TAPS_TILE_COLS * TAPS_WIN_TILES);
    const uint64_t g_end = total - g_begin < TAPS_TILE_COLS * TAPS_WIN_TILES
                               ? total : g_begin + TAPS_TILE_COLS * TAPS_WIN_TILES;
    uint32_t e = win_edge[w];
    taps_edge_params E = params[e];
    const uint64_t local = g_begin - E.out_offset;   // below ns * nd
    uint32_t i = (uint32_t)(local / E.nd), j0 = (uint32_t)(local % E.nd);
    taps_row P;
    bool built = false;   // P (and this wavefront's rank table) hold row i of edge e
    for (uint64_t g0 = g_begin; g0 < g_end; g0 += TAPS_TILE_COLS) {
        const uint32_t n_here = (uint32_t)(g_end - g0 < TAPS_TILE_COLS ? g_end - g0 : TAPS_TILE_COLS);
        uint32_t done = 0;   // lanes below this are handled
        while (done < n_here) {   // uniform: one row of one edge per pass
            __builtin_assume(E.rank <= R);
            const uint32_t len = n_here - done < E.nd - j0 ? n_here - done : E.nd - j0;
            if (len == 0) break;   // (cannot happen: entries remain only in edges that hold them)
            if (!built) {
                taps_make_row(P, desc[E.src_base + i], E.paxes, E.rank, lp.n, lp.lam);
                // the row's producer-order table, written and read by this wavefront only
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                taps_fill_rank_table(P, rank_tab[wave], lane, TAPS_TILE_COLS);
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                P.to_rank = rank_tab[wave];
                P.widths = width_tab;
                P.a2a = a2a_tab;
                P.expand = expand_tab;
                built = true;
            }
            if (lane >= done && lane < done + len) {
                const uint32_t j = j0 + (lane - done);
                taps_col Q;
                taps_make_col(Q, desc[E.dst_base + j], E.caxes, E.rank);
                const taps_cands cands = taps_edge_candidates(P, Q, any);
                for (uint32_t k = 0; k < sw.count; ++k) {
                    taps_keys K;
                    K.b_inter_red = sw.b_inter_red[k];
                    K.b_intra_red = sw.b_intra_red[k];
                    K.narrow = Narrow || sw.narrow[k] != 0;   // Narrow: 64-bit keys at every point
                    const taps_scaler S = taps_make_scaler(E.scale.tbytes, sw.inv_n_bintra[k],
                                                           sw.inv_n_binter[k]);
                    const taps_entry_out o = taps_entry_finish(taps_pick_for(cands, K), S);
                    store_entry(sw.out[k], g0, lane, o, o.ok ? o.meta : 0xFFFFFFFFu);
                }
            }
            done += len;
            j0 += len;
            // the row is done and entries remain in the window: the next row, or
            // the first row of the next edge with entries
            if (j0 == E.nd && g0 + done < g_end) {
                j0 = 0;
                built = false;
                if (++i == E.ns) {
                    i = 0;
                    do {
                        ++e;
                        E = params[e];
                    } while (e + 1u < n_edges && (uint64_t)E.ns * E.nd == 0u);
                }
            }
        }
    }
}

// Link-class hierarchies: as k_edge_costs, each entry selected and scaled
// under the classes of H.
// C: the hierarchy's number of classes.
template <uint32_t R, uint32_t C>
__global__ __launch_bounds__(TAPS_TILE_COLS *TAPS_ROWS_PER_BLOCK) void k_edge_costs_h(
    const taps_edge_params *__restrict__ params, const taps_row_ref *__restrict__ rows,
    uint32_t n_segs, const taps_desc *__restrict__ desc, taps_launch lp, taps_hier H,
    taps_table out) {
    __shared__ uint8_t rank_tab[TAPS_ROWS_PER_BLOCK][256];
    __shared__ uint32_t width_tab[256];
    __shared__ taps_pair a2a_cls_tab[256 * TAPS_D_MAX_CLASSES];
    __shared__ taps_pair expand_tab[256];
    const uint32_t lane = threadIdx.x % TAPS_TILE_COLS;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / TAPS_TILE_COLS);
    const uint32_t r = blockIdx.x * TAPS_ROWS_PER_BLOCK + wave;
    const bool live = r < n_segs;
    const taps_row_ref ref = rows[live ? r : 0u];
    const taps_edge_params E = params[ref.edge];
    __builtin_assume(E.rank <= R);   // the launch's tensors have rank R at most
    const taps_desc Dp = desc[ref.strategy];
    const uint32_t i = ref.strategy - E.src_base;
    taps_row P;
    taps_make_row(P, Dp, E.paxes, E.rank, lp.n, lp.lam);
    taps_fill_rank_table(P, rank_tab[wave], lane, TAPS_TILE_COLS);
    for (uint32_t x = threadIdx.x; x < 256u; x += blockDim.x) width_tab[x] = kWidths.v[x];
    fill_a2a_class_tables(a2a_cls_tab, expand_tab, H);
    __syncthreads();
    if (!live) return;
    P.to_rank = rank_tab[wave];
    P.widths = width_tab;
    P.a2a_cls = a2a_cls_tab;
    P.expand = expand_tab;
    const uint64_t row_out = E.out_offset + (uint64_t)i * E.nd;
    const taps_desc *col = desc + E.dst_base;
    const uint32_t c0 = ref.first_col;
    const uint32_t c1 = ref.last_col;
    for (uint32_t j = c0 + lane; j < c1; j += TAPS_TILE_COLS) {
        taps_col Q;
        taps_make_col(Q, col[j], E.caxes, E.rank);
        const taps_entry_out o = taps_entry_finish_h(taps_edge_select_h<C>(P, Q, H), E.scale, H);
        store_entry(out, row_out, j, o, o.ok ? o.meta : 0xFFFFFFFFu);
    }
}

__global__ __launch_bounds__(256) void k_node_costs_h(const taps_op *__restrict__ ops,
                                                      uint32_t n_ops,
                                                      const uint64_t *__restrict__ offsets,
                                                      const taps_desc *__restrict__ desc,
                                                      uint64_t total, uint32_t n, taps_hier H,
                                                      taps_table out) {
    const uint64_t idx = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const taps_op &op = ops[find_owner(offsets, n_ops, idx)];
    const taps_desc D = desc[idx];
    const uint32_t full = taps_low_mask(n);
    taps_acch c = {0, 0, 0, 0, 0, 0, 0, 0};
    auto tensor = [&](const taps_tensor &t) {
        uint32_t used = 0;
        uint64_t bytes = op.dtype_bytes;
        for (uint32_t d = 0; d < t.rank && d < TAPS_MAX_RANK; ++d) {
            const uint32_t a = t.axis[d] & 7u;
            used |= taps_levels(taps_nib(D.lo, a), taps_nib(D.width, a));
            bytes *= (uint64_t)op.axis_len[a];
        }
        taps_allreduce_h(c, full & ~used, bytes, H);
    };
    tensor(op.out);
    for (uint32_t k = 0; k < op.n_in && k < TAPS_MAX_INPUTS; ++k) tensor(op.in[k]);
    for (uint32_t k = 0; k < op.n_w && k < TAPS_MAX_WEIGHTS; ++k) tensor(op.w[k]);
    out.t[idx] = (double)c.x0 * H.inv_n_bw[0] + (double)c.x1 * H.inv_n_bw[1] +
                 (double)c.x2 * H.inv_n_bw[2] + (double)c.x3 * H.inv_n_bw[3];
    out.vol[idx] = c.vol;
    out.intra[idx] = c.x0;
    out.inter[idx] = c.x1 + c.x2 + c.x3;
    out.meta[idx] = (c.n_coll << 2) | (c.n_inter << 7) | (c.sum_ct << 12);
}

// Shared tables: each task holds `count` (<= TAPS_COPY_CHUNK) consecutive
// entries of a computed table, staged once in LDS and stored into every table
// that shares it, at the same offset; blockIdx.y picks the array.  The tables
// start at arbitrary entries, so each destination is written with 16-byte
// stores aligned to its own 16-byte boundaries (LDS absorbs the difference in
// alignment between source and destination), plus single-entry stores for the
// head and tail.
struct alignas(16) vec16 {
    uint32_t w[4];
};

template <typename T>
__device__ inline void copy_range(T *base, const taps_copy_task &c,
                                  const uint64_t *__restrict__ dst_list, T *stage) {
    constexpr uint32_t kV = 16 / sizeof(T);   // entries per 16-byte store
    const T *s = base + c.src;
    for (uint32_t x = threadIdx.x; x < c.count; x += blockDim.x) stage[x] = s[x];
    __syncthreads();
    for (uint32_t k = 0; k < c.n_dst; ++k) {
        T *d = base + dst_list[c.dst_begin + k] + c.offset;
        const uint32_t mis = (uint32_t)(((uintptr_t)d & 15u) / sizeof(T));
        const uint32_t head = mis ? (kV - mis < c.count ? kV - mis : c.count) : 0u;
        const uint32_t n_vec = (c.count - head) / kV;
        const uint32_t tail = head + n_vec * kV;
        if (threadIdx.x < head) d[threadIdx.x] = stage[threadIdx.x];
        vec16 *dv = (vec16 *)(d + head);
        for (uint32_t v = threadIdx.x; v < n_vec; v += blockDim.x) {
            vec16 val;
            __builtin_memcpy(&val, stage + head + v * kV, 16);
            dv[v] = val;
        }
        if (tail + threadIdx.x < c.count) d[tail + threadIdx.x] = stage[tail + threadIdx.x];
    }
}

// An upload without the copy engine: the plan is read straight from
// fine-grained pinned host memory, 16 bytes per thread and step, so the
// build's kernels follow it on the same queue with no hand-over.
__global__ __launch_bounds__(256) void k_pull(const uint4 *__restrict__ src,
                                              uint4 *__restrict__ dst, uint32_t n16) {
    for (uint32_t k = blockIdx.x * 256u + threadIdx.x; k < n16; k += gridDim.x * 256u)
        dst[k] = src[k];
}

__global__ __launch_bounds__(256) void k_copy_tables(const taps_copy_task *__restrict__ tasks,
                                                     const uint64_t *__restrict__ dst_list,
                                                     taps_table out) {
    __shared__ uint64_t stage[TAPS_COPY_CHUNK];
    const taps_copy_task c = tasks[blockIdx.x];
    switch (blockIdx.y) {
    case 0: copy_range(out.t, c, dst_list, (double *)stage); break;
    case 1: copy_range(out.vol, c, dst_list, stage); break;
    case 2: copy_range(out.intra, c, dst_list, stage); break;
    case 3: copy_range(out.inter, c, dst_list, stage); break;
    default: copy_range(out.meta, c, dst_list, (uint32_t *)stage); break;
    }
}

// One workgroup per pair of strategy ranges; flags[p] = any entry differs.
__global__ __launch_bounds__(256) void k_same_ranges(const taps_strategy *__restrict__ s,
                                                     const uint64_t *__restrict__ pairs,
                                                     uint32_t *__restrict__ flags) {
    const uint64_t a = pairs[3 * blockIdx.x], b = pairs[3 * blockIdx.x + 1];
    const uint64_t count = pairs[3 * blockIdx.x + 2];
    int differ = 0;
    for (uint64_t k = threadIdx.x; k < count; k += blockDim.x) {
        const taps_strategy x = s[a + k], y = s[b + k];
        for (uint32_t q = 0; q < TAPS_MAX_AXES; ++q)
            differ |= (x.log2_deg[q] != y.log2_deg[q]) | (x.pos[q] != y.pos[q]);
    }
    differ = __syncthreads_or(differ);
    if (threadIdx.x == 0) flags[blockIdx.x] = differ ? 1u : 0u;
}

inline uint32_t blocks_for(uint64_t n, uint32_t per) { return (uint32_t)((n + per - 1) / per); }

}  // namespace

hipError_t taps_launch_describe(const taps_strategy *s, uint64_t total, taps_desc *desc,
                                hipStream_t stream) {
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(k_describe, dim3(blocks_for(total, 256)), dim3(256), 0, stream, s, total,
                       desc);
    return hipGetLastError();
}

hipError_t taps_launch_node_costs(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                  const taps_desc *desc, uint64_t total, const taps_launch &lp,
                                  taps_table out, hipStream_t stream) {
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(k_node_costs, dim3(blocks_for(total, 256)), dim3(256), 0, stream, ops,
                       n_ops, offsets, desc, total, lp, out);
    return hipGetLastError();
}

hipError_t taps_launch_memory_costs(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                   const taps_strategy *s, uint64_t total, uint64_t *memory,
                                   hipStream_t stream) {
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(k_memory_costs, dim3(blocks_for(total, 256)), dim3(256), 0, stream, ops,
                       n_ops, offsets, s, total, memory);
    return hipGetLastError();
}

hipError_t taps_launch_edge_setup(const taps_plan_args &pa, const taps_launch &lp,
                                  hipStream_t stream) {
    if (pa.n_edges == 0) return hipSuccess;
    const uint32_t setup_blocks = blocks_for(pa.n_edges, 256);
    const uint64_t map_blocks = pa.n_groups ? blocks_for(pa.n_segs, 256) : 0;
    hipLaunchKernelGGL(k_edge_plan, dim3((uint32_t)(setup_blocks + map_blocks)), dim3(256), 0,
                       stream, pa, lp, setup_blocks);
    return hipGetLastError();
}

hipError_t taps_launch_edge_costs(const taps_edge_params *params, const taps_row_ref *segs,
                                  uint64_t n_segs, const taps_desc *desc, const taps_launch &lp,
                                  uint32_t max_rank, taps_table out, hipStream_t stream) {
    if (n_segs == 0) return hipSuccess;
    const dim3 grid(blocks_for(n_segs, TAPS_ROWS_PER_BLOCK)), block(TAPS_TILE_COLS * TAPS_ROWS_PER_BLOCK);
    const bool low = max_rank <= TAPS_LOW_RANK, narrow = lp.narrow != 0;
    if (low && narrow)
        hipLaunchKernelGGL((k_edge_costs<TAPS_LOW_RANK, true>), grid, block, 0, stream, params,
                           segs, (uint32_t)n_segs, desc, lp, out);
    else if (low)
        hipLaunchKernelGGL((k_edge_costs<TAPS_LOW_RANK, false>), grid, block, 0, stream, params,
                           segs, (uint32_t)n_segs, desc, lp, out);
    else if (narrow)
        hipLaunchKernelGGL((k_edge_costs<TAPS_D_MAX_RANK, true>), grid, block, 0, stream, params,
                           segs, (uint32_t)n_segs, desc, lp, out);
    else
        hipLaunchKernelGGL((k_edge_costs<TAPS_D_MAX_RANK, false>), grid, block, 0, stream, params,
                           segs, (uint32_t)n_segs, desc, lp, out);
    return hipGetLastError();
}

hipError_t taps_launch_edge_costs_sweep_win(const taps_edge_params *params, uint32_t n_edges,
                                            const uint64_t *eoff, uint64_t total,
                                            uint32_t *win_edge, const taps_desc *desc,
                                            const taps_launch &lp, uint32_t max_rank,
                                            const taps_sweep &sw, hipStream_t stream) {
    if (total == 0) return hipSuccess;
    const uint64_t span = TAPS_TILE_COLS * TAPS_WIN_TILES;
    const uint64_t n_windows = (total + span - 1) / span;
    hipLaunchKernelGGL(k_window_edges, dim3(blocks_for(n_windows, 256)), dim3(256), 0, stream, eoff,
                       n_edges, n_windows, win_edge);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const dim3 grid(blocks_for(n_windows, TAPS_ROWS_PER_BLOCK)), block(TAPS_TILE_COLS * TAPS_ROWS_PER_BLOCK);
    bool narrow = true;
    for (uint32_t k = 0; k < sw.count; ++k) narrow = narrow && sw.narrow[k] != 0;
    const bool low = max_rank <= TAPS_LOW_RANK;
#define TAPS_WIN_LAUNCH(RR, NN)                                                                  \
    hipLaunchKernelGGL((k_edge_costs_sweep_win<RR, NN>), grid, block, 0, stream, params, n_edges, \
                       win_edge, n_windows, total, desc, lp, sw)
    if (low && narrow) TAPS_WIN_LAUNCH(TAPS_LOW_RANK, true);
    else if (low) TAPS_WIN_LAUNCH(TAPS_LOW_RANK, false);
    else if (narrow) TAPS_WIN_LAUNCH(TAPS_D_MAX_RANK, true);
    else TAPS_WIN_LAUNCH(TAPS_D_MAX_RANK, false);
#undef TAPS_WIN_LAUNCH
    return hipGetLastError();
}

hipError_t taps_launch_build_strategies(const taps_op *ops, const taps_build_chunk *chunks,
                                        uint32_t n_chunks, uint32_t allowed_cuts,
                                        const taps_launch &lp, taps_strategy *out, taps_desc *desc,
                                        taps_table node, hipStream_t stream) {
    if (n_chunks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_build_strategies, dim3(n_chunks), dim3(kBuildThreads), 0, stream, ops,
                       chunks, allowed_cuts, lp, out, desc, node);
    return hipGetLastError();
}

hipError_t taps_launch_build_front(const taps_build_chunk *chunks, uint32_t n_chunks,
                                   uint32_t allowed_cuts, const taps_launch &lp, taps_strategy *out,
                                   taps_desc *desc, taps_table node, const taps_plan_args &pa,
                                   hipStream_t stream) {
    const uint32_t setup_blocks = pa.n_edges ? blocks_for(pa.n_edges, 256) : 0;
    const uint64_t map_blocks = pa.n_groups ? blocks_for(pa.n_segs, 256) : 0;
    const uint64_t blocks = n_chunks + setup_blocks + map_blocks;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_build_front, dim3((uint32_t)blocks), dim3(kBuildThreads), 0, stream,
                       chunks, n_chunks, allowed_cuts, lp, out, desc, node, pa, setup_blocks);
    return hipGetLastError();
}

hipError_t taps_launch_edge_costs_h(const taps_edge_params *params, const taps_row_ref *rows,
                                    uint64_t n_rows, const taps_desc *desc, const taps_launch &lp,
                                    uint32_t max_rank, const taps_hier &H, taps_table out,
                                    hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    const dim3 grid(blocks_for(n_rows, TAPS_ROWS_PER_BLOCK)), block(TAPS_TILE_COLS * TAPS_ROWS_PER_BLOCK);
    const bool low = max_rank <= TAPS_LOW_RANK;
#define TAPS_H_LAUNCH(RR, CC)                                                                    \
    hipLaunchKernelGGL((k_edge_costs_h<RR, CC>), grid, block, 0, stream, params, rows,            \
                       (uint32_t)n_rows, desc, lp, H, out)
    switch (H.n_classes * 2 + (low ? 0 : 1)) {
    case 2: TAPS_H_LAUNCH(TAPS_LOW_RANK, 1); break;
    case 3: TAPS_H_LAUNCH(TAPS_D_MAX_RANK, 1); break;
    case 4: TAPS_H_LAUNCH(TAPS_LOW_RANK, 2); break;
    case 5: TAPS_H_LAUNCH(TAPS_D_MAX_RANK, 2); break;
    case 6: TAPS_H_LAUNCH(TAPS_LOW_RANK, 3); break;
    case 7: TAPS_H_LAUNCH(TAPS_D_MAX_RANK, 3); break;
    case 8: TAPS_H_LAUNCH(TAPS_LOW_RANK, 4); break;
    default: TAPS_H_LAUNCH(TAPS_D_MAX_RANK, 4); break;
    }
#undef TAPS_H_LAUNCH
    return hipGetLastError();
}

hipError_t taps_launch_node_costs_h(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                    const taps_desc *desc, uint64_t total, uint32_t n,
                                    const taps_hier &H, taps_table out, hipStream_t stream) {
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(k_node_costs_h, dim3(blocks_for(total, 256)), dim3(256), 0, stream, ops,
                       n_ops, offsets, desc, total, n, H, out);
    return hipGetLastError();
}

hipError_t taps_launch_pull(const void *src, void *dst, uint64_t bytes, hipStream_t stream) {
    const uint64_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    const uint64_t blocks = (n16 + 255) / 256 < 256 ? (n16 + 255) / 256 : 256;
    hipLaunchKernelGGL(k_pull, dim3((uint32_t)blocks), dim3(256), 0, stream, (const uint4 *)src,
                       (uint4 *)dst, (uint32_t)n16);
    return hipGetLastError();
}

hipError_t taps_launch_copy_tables(const taps_copy_task *tasks, uint32_t n_tasks,
                                   const uint64_t *dst_list, taps_table out, hipStream_t stream) {
    if (n_tasks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_copy_tables, dim3(n_tasks, 5), dim3(256), 0, stream, tasks, dst_list,
                       out);
    return hipGetLastError();
}

hipError_t taps_launch_same_ranges(const taps_strategy *strategies, const uint64_t *pairs,
                                   uint32_t n_pairs, uint32_t *flags, hipStream_t stream) {
    if (n_pairs == 0) return hipSuccess;
    hipLaunchKernelGGL(k_same_ranges, dim3(n_pairs), dim3(256), 0, stream, strategies, pairs,
                       flags);
    return hipGetLastError();
}

// taps_internal.h -- launch interface between the C ABI and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "taps.h"
#include "taps_device.h"

// Uniform parameters of a table launch.
struct taps_launch {
    uint32_t n;             // log2 N
    uint32_t lam;           // log2 L
    uint64_t b_inter_red;   // B_inter / gcd(B_intra, B_inter)
    uint64_t b_intra_red;   // B_intra / gcd(B_intra, B_inter)
    double inv_n_bintra;    // 1 / (N B_intra)
    double inv_n_binter;    // 1 / (N B_inter)
    uint32_t narrow;        // both reduced bandwidths below 2^32
};

// Per-edge constants of the edge-table kernel.
struct taps_edge_params {
    uint64_t out_offset;   // first entry of the edge's table
    taps_scaler scale;     // tbytes and the per-unit seconds of the edge tensor
    uint32_t src_base;     // first strategy of the source side (producer; consumer for
    uint32_t dst_base;     //   the backward tables) and of the target side
    uint32_t ns, nd;       // their strategy counts
    uint32_t rank;
    uint32_t paxes;        // nibble d: source op axis of tensor dimension d
    uint32_t caxes;        // nibble d: target op axis of tensor dimension d
    uint32_t pad;
};

// Shared tables: entries [src, src + count) of every array are copied to
// [dst[k] + offset, dst[k] + offset + count) for the n_dst table starts
// dst[k] = dst_list[dst_begin + k].
struct taps_copy_task {
    uint64_t src, offset;
    uint32_t count, dst_begin, n_dst, pad;
};
#define TAPS_COPY_CHUNK 2048    // entries per copy task (8 per thread of 256)
#define TAPS_COPY_DSTS 6        // tables one copy task writes (4-6 measured best, 16 is 20 % slower)

// One wavefront per row segment: producer strategy i of one edge and the
// consumer strategies [first_col, last_col) of its row, walked 64 at a time.
// A workgroup holds TAPS_ROWS_PER_BLOCK segments.  A segment builds its
// producer side once (about 0.15 ms of the 96-layer GPT's launch at two
// tiles per segment); TAPS_SEG_TILES_LONG tiles amortise that in launches of
// many segments, and launching the full-length segments before the shorter
// remainders keeps the longer segments from stretching the end of the launch
// (1, 2, 4, 8, 16 and 32 tiles measured).  Launches with few segments use
// TAPS_SEG_TILES_SHORT.  The bandwidth sweep, bound by its four sets of
// stores per entry, does not use segments: it runs one wavefront per window of
// TAPS_WIN_TILES aligned 64-entry tiles of the tables (k_edge_costs_sweep_win).
#define TAPS_TILE_COLS 64
#define TAPS_SEG_TILES_LONG 8
#define TAPS_SEG_TILES_SHORT 2
#ifndef TAPS_WIN_TILES
#define TAPS_WIN_TILES 2
#endif
#define TAPS_LONG_SEGS_MIN 32768   // long segments only when there are at least this many
#define TAPS_ROWS_PER_BLOCK 2

// A run of row segments of one edge: every row of the edge's table cut into
// per_row segments of `cols` consumer strategies from first_col, the last
// one ending at the row's end at the latest.  Segment r of a launch belongs
// to the last group whose start is at most r: row (r - start) / per_row,
// first consumer first_col + ((r - start) % per_row) * cols.
struct taps_seg_group {
    uint64_t start;
    uint32_t edge, per_row, first_col, cols;
};

// Segment r of a launch: its edge, the global index of its producer strategy
// and its consumer strategies [first_col, last_col).
struct taps_row_ref {
    uint32_t edge;
    uint32_t strategy;
    uint32_t first_col;
    uint32_t last_col;
};

hipError_t taps_launch_describe(const taps_strategy *s, uint64_t total, taps_desc *desc,
                                hipStream_t stream);
hipError_t taps_launch_node_costs(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                  const taps_desc *desc, uint64_t total, const taps_launch &lp,
                                  taps_table out, hipStream_t stream);
// The edge plan of a launch (device arrays): per-edge constants into params
// and the row segments of the groups into segs; reverse: the backward tables
// (source side = the consumer's input map).
struct taps_plan_args {
    const taps_op *ops;
    const taps_edge *edges;
    const uint64_t *op_offsets;
    const uint64_t *edge_offsets;
    const taps_seg_group *groups;
    taps_edge_params *params;
    taps_row_ref *segs;
    uint64_t n_segs;
    uint32_t n_edges, n_groups, reverse, pad;
};
hipError_t taps_launch_edge_setup(const taps_plan_args &pa, const taps_launch &lp,
                                  hipStream_t stream);
// max_rank: the largest tensor rank of the launch's edges; up to
// TAPS_LOW_RANK the kernels are compiled for that many dimensions (fewer
// registers for the producer side, shorter per-dimension loops).
#define TAPS_LOW_RANK 4
hipError_t taps_launch_edge_costs(const taps_edge_params *params, const taps_row_ref *rows,
                                  uint64_t n_rows, const taps_desc *desc, const taps_launch &lp,
                                  uint32_t max_rank, taps_table out, hipStream_t stream);
hipError_t taps_launch_memory_costs(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                   const taps_strategy *s, uint64_t total, uint64_t *memory,
                                   hipStream_t stream);
// Bandwidth points of one sweep: the keys and per-unit seconds of each, and
// the table each writes.
struct taps_sweep {
    uint32_t count;
    uint32_t narrow[TAPS_MAX_SWEEP];
    uint64_t b_inter_red[TAPS_MAX_SWEEP];
    uint64_t b_intra_red[TAPS_MAX_SWEEP];
    double inv_n_bintra[TAPS_MAX_SWEEP];
    double inv_n_binter[TAPS_MAX_SWEEP];
    taps_table out[TAPS_MAX_SWEEP];
};
// The sweep over aligned windows of TAPS_WIN_TILES 64-entry tiles of the
// concatenated tables (eoff: device, n_edges + 1 entry offsets; win_edge:
// device scratch of one uint32 per window, ceil(total / (64 TAPS_WIN_TILES))).
hipError_t taps_launch_edge_costs_sweep_win(const taps_edge_params *params, uint32_t n_edges,
                                            const uint64_t *eoff, uint64_t total,
                                            uint32_t *win_edge, const taps_desc *desc,
                                            const taps_launch &lp, uint32_t max_rank,
                                            const taps_sweep &sw, hipStream_t stream);
// One workgroup of k_build_strategies: candidate ranks [first, first +
// TAPS_BUILD_CHUNK) of operator `op`, of which `count` pass the filter; they
// are strategies base, base + 1, ... in rank order.
#define TAPS_BUILD_CHUNK 256
struct taps_build_chunk {
    uint64_t base;
    uint32_t op, first, count, pad;
};
// Strategies of every operator in one launch (one workgroup per chunk of
// candidate ranks that holds a strategy), with their descriptors and node
// records unless desc / node.t are NULL.
hipError_t taps_launch_build_strategies(const taps_op *ops, const taps_build_chunk *chunks,
                                        uint32_t n_chunks, uint32_t allowed_cuts,
                                        const taps_launch &lp, taps_strategy *out, taps_desc *desc,
                                        taps_table node, hipStream_t stream);
// taps_launch_build_strategies and taps_launch_edge_setup as one launch (the
// plan needs only the host-counted strategy offsets).
hipError_t taps_launch_build_front(const taps_build_chunk *chunks, uint32_t n_chunks,
                                   uint32_t allowed_cuts, const taps_launch &lp, taps_strategy *out,
                                   taps_desc *desc, taps_table node, const taps_plan_args &pa,
                                   hipStream_t stream);
// Link-class hierarchies: the edge and node tables under the classes of H.
hipError_t taps_launch_edge_costs_h(const taps_edge_params *params, const taps_row_ref *rows,
                                    uint64_t n_rows, const taps_desc *desc, const taps_launch &lp,
                                    uint32_t max_rank, const taps_hier &H, taps_table out,
                                    hipStream_t stream);
hipError_t taps_launch_node_costs_h(const taps_op *ops, uint32_t n_ops, const uint64_t *offsets,
                                    const taps_desc *desc, uint64_t total, uint32_t n,
                                    const taps_hier &H, taps_table out, hipStream_t stream);
// Copies `bytes` (a multiple of 16, below 2^36) from src, fine-grained pinned
// host memory mapped for the device, to device memory at dst.
hipError_t taps_launch_pull(const void *src, void *dst, uint64_t bytes, hipStream_t stream);
hipError_t taps_launch_copy_tables(const taps_copy_task *tasks, uint32_t n_tasks,
                                   const uint64_t *dst_list, taps_table out, hipStream_t stream);
// For each pair p: flags[p] = 0 if strategies[first_a .. +count) equals
// strategies[first_b .. +count), else 1.  pairs: (first_a, first_b, count) as
// three uint64 each.
hipError_t taps_launch_same_ranges(const taps_strategy *strategies, const uint64_t *pairs,
                                   uint32_t n_pairs, uint32_t *flags, hipStream_t stream);

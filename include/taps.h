/*
 * taps.h -- C ABI of the MI355X TAPS cost-table library.
 *
 * TAPS (Liang et al., "TAPS: Topology-Aware Intra-Operator Parallelism
 * Strategy Searching Algorithm for Deep Neural Networks", arXiv 2301.04285)
 * chooses one intra-operator sharding strategy per operator of a computation
 * graph by solving an integer program over an auxiliary graph whose
 * vertices are (operator, strategy) pairs and whose edges are (producer
 * strategy, consumer strategy) pairs.  This library builds, on one GPU, the
 * tables that program consumes:
 *
 *   1. taps_enumerate_strategies -- every strategy of every operator
 *      (GenerateStrategySet, Auxiliary Graph section, Table 3), or with
 *      taps_enumerate_strategies_mesh those a fixed device mesh expresses;
 *   2. taps_node_costs -- the intra-operator communication cost of every
 *      strategy (Communication Cost Model section: Eq. 5-8, Algorithm 2,
 *      Eq. 11-12);
 *   3. taps_edge_costs -- for every graph edge and every (producer strategy,
 *      consumer strategy) pair the cost of redistributing the edge tensor
 *      (Table 1 unification, Table 2 / Algorithm 1 sequences, Eq. 9-14,
 *      Algorithm 3; Algorithm 4 gives the pair loop).
 *
 * The inputs follow the paper's problem statement (Overview section): a
 * computation graph whose operators carry shapes and types, and a device
 * graph reduced to what the cost model uses -- the device count, the devices
 * per node and the intra- and inter-node bandwidths.
 *
 * Conventions
 *   - N = nodes * devices_per_node devices, L = devices_per_node; both must be
 *     powers of two and N <= 2^TAPS_MAX_LEVELS.  Device rank r is mixed-radix
 *     over the device matrix with its innermost axis fastest and lives on
 *     node r / L.
 *   - A strategy splits some partitionable op axes; the degrees are powers of
 *     two that multiply to N; pos orders the split axes on the device matrix
 *     (pos 0 innermost = adjacent devices).  A degree must divide its axis.
 *   - Volumes are unsigned integers in units of bytes x N ("nb"), so every
 *     per-device volume of the paper's formulas is exact.  Times are seconds.
 *   - Every record has five fields, stored as five separate arrays (SoA):
 *       t      double   cost in seconds = intra/(N B_intra) + inter/(N B_inter)
 *       vol    uint64   communication volume (nb) -- the volume-based model
 *       intra  uint64   nb carried by intra-node links
 *       inter  uint64   nb carried by inter-node links, each collective's
 *                       link volume multiplied by its inter-node group count
 *       meta   uint32   bits 0-1: chosen sequence (edges; 0 for nodes)
 *                       bits 2-6: number of collectives
 *                       bits 7-11: collectives that leave a node
 *                       bits 12-31: sum of their inter-node group counts
 *
 * Memory and streams
 *   - Graph, cluster and offset arrays are host memory owned by the caller
 *     and read only during the call.  Strategy and table arrays are device
 *     memory (HIP) owned by the caller.  The library keeps one device scratch
 *     block per (device, stream), reused by the next call on that stream
 *     (stream order makes the reuse safe) and grown in stream order when a
 *     call needs more; at most 16 such blocks are kept (the least recently
 *     used idle one is freed).  Host arrays a call uploads are copied into
 *     one of at most 8 pinned staging buffers (1 MiB or more each, kept until
 *     the process ends) and read from there by a kernel in stream order.  Calls
 *     on one stream from several threads are queued one after the other.  No
 *     pointer of the caller is kept after the call returns.
 *   - Kernels are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream): the tables are complete once that stream has been
 *     synchronised.  Every size (strategies per operator, entries per edge)
 *     is computed on the host, so only taps_edge_costs_shared synchronises
 *     (to read back a device comparison of strategy ranges).
 *   - Calls on distinct outputs may run concurrently from several threads.
 *
 * Errors
 *   - Every call returns a taps_status; arguments are validated before any
 *     GPU work and nothing is written on a validation error.
 *     taps_last_error() returns a thread-local description of the last
 *     failure of the calling thread.
 */
#ifndef TAPS_H
#define TAPS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TAPS_MAX_AXES 8     /* axes of one operator */
#define TAPS_MAX_RANK 8     /* dimensions of one tensor */
#define TAPS_MAX_INPUTS 4   /* activation inputs of one operator */
#define TAPS_MAX_WEIGHTS 4  /* weights of one operator */
#define TAPS_MAX_LEVELS 8   /* N <= 2^8 = 256 devices */
#define TAPS_MAX_SWEEP 8    /* bandwidth points of one taps_edge_costs_sweep call */
#define TAPS_MAX_TENSOR_BYTES (1ull << 40) /* keeps every volume exact in 64 bits */

typedef enum {
    TAPS_OK = 0,
    TAPS_ERR_ARG = 1,         /* NULL pointer, index out of range, malformed operator */
    TAPS_ERR_TOPOLOGY = 2,    /* nodes or devices per node not a power of two,
                                 N > 2^TAPS_MAX_LEVELS, a zero bandwidth */
    TAPS_ERR_SHAPE = 3,       /* an edge's two tensor shapes disagree */
    TAPS_ERR_NO_STRATEGY = 4, /* an operator has no strategy on N devices */
    TAPS_ERR_CAPACITY = 5,    /* the output arrays are too small */
    TAPS_ERR_DEVICE = 6       /* a HIP runtime error */
} taps_status;

/* The modeled cluster (device graph of the problem statement). */
typedef struct {
    uint32_t nodes;
    uint32_t devices_per_node; /* L */
    uint64_t bw_intra;         /* bytes per second between devices of one node */
    uint64_t bw_inter;         /* bytes per second of one node's inter-node link */
} taps_cluster;

/* A tensor of an operator: dimension d is op axis axis[d]. */
typedef struct {
    uint8_t rank;
    uint8_t axis[TAPS_MAX_RANK];
} taps_tensor;

/* An operator as an einsum over its axes: `out` is produced, `in` are
 * activations (edges attach to them), `w` are weights.  Bit a of part_mask
 * marks axis a as partitionable.  dtype_bytes is the element size of every
 * tensor of the operator. */
typedef struct {
    uint8_t n_axes, part_mask, dtype_bytes, n_in, n_w;
    int64_t axis_len[TAPS_MAX_AXES];
    taps_tensor in[TAPS_MAX_INPUTS];
    taps_tensor w[TAPS_MAX_WEIGHTS];
    taps_tensor out;
} taps_op;

/* ops[src_op].out feeds ops[dst_op].in[dst_slot]; both ends must have the
 * same rank and the same length in every dimension. */
typedef struct {
    uint32_t src_op, dst_op, dst_slot;
} taps_edge;

typedef struct {
    uint32_t n_ops, n_edges;
    const taps_op *ops;
    const taps_edge *edges;
} taps_graph;

/* One strategy: per op axis, log2 of its degree (0 = not split) and its
 * device-matrix position (-1 = not split). */
typedef struct {
    uint8_t log2_deg[TAPS_MAX_AXES];
    int8_t pos[TAPS_MAX_AXES];
} taps_strategy;

/* A fixed device mesh: dims[0] (innermost) x dims[1] x ... x dims[n_dims - 1]
 * devices, each size a power of two >= 2, the product N = nodes * L.  N = 1
 * takes n_dims = 0. */
typedef struct {
    uint32_t n_dims;
    uint32_t dims[TAPS_MAX_LEVELS];
} taps_mesh;

/* A hierarchy of link classes, an extension of the paper's two (intra- and
 * inter-node, Eq. 11-14): blocks of domain[0] <= domain[1] <= ... <=
 * domain[n_classes - 1] = N consecutive device ranks (a node, a group of
 * nodes, ...).  Class 0 links join the devices of one domain[0] block; class
 * c >= 1 links join the domain[c-1] blocks of one domain[c] block, bw[c]
 * bytes per second each.  The paper's cluster is {2, {L, N}, {B_intra,
 * B_inter}, 0}. */
#define TAPS_MAX_CLASSES 4
typedef struct {
    uint32_t n_classes;                 /* 1 .. TAPS_MAX_CLASSES */
    uint32_t domain[TAPS_MAX_CLASSES];  /* powers of two, non-decreasing, the last N */
    uint64_t bw[TAPS_MAX_CLASSES];      /* bytes per second, > 0 */
    uint64_t bw_a2a;                    /* bytes per second of an AllToAll inside one domain[0]
                                           block (peer to peer over every link of the block,
                                           where a ring uses one); 0: bw[0] */
} taps_topology;

/* Device arrays of one table, one element per record. */
typedef struct {
    double *t;
    uint64_t *vol;
    uint64_t *intra;
    uint64_t *inter;
    uint32_t *meta;
} taps_table;

/* GenerateStrategySet for every operator (Auxiliary Graph section; the
 * count sum_{i=1}^{min(p,n)} i! C(p,i) C(n-1,i-1) and the example of
 * Table 3), on N = 2^n devices.
 *   op_offsets  host, n_ops + 1 entries, written: op k's strategies are
 *               strategies[op_offsets[k] .. op_offsets[k+1]).
 *   strategies  device, `capacity` entries, written in canonical order (the
 *               degree tuple ascending, then the device-map tuple
 *               descending -- the order of Table 3).  NULL: only op_offsets
 *               is written (size query).
 * Strategies whose degree does not divide its axis are left out; with N = 1
 * the single strategy splits nothing.  The counts come from an exact count of
 * that filter on the host (ordered runs of distinct partitionable axes over
 * the n levels, each at most as wide as its length allows); the strategies
 * themselves are enumerated on the device, one workgroup per chunk of 256
 * candidate ranks of an operator, each writing at the offset the host counted
 * for that chunk (the same unranking and filter, checked against the exact
 * count), and the call does not synchronise.  TAPS_ERR_NO_STRATEGY if an operator has
 * none, TAPS_ERR_CAPACITY if op_offsets[n_ops] > capacity (op_offsets is
 * still written, the strategies are not). */
taps_status taps_enumerate_strategies(const taps_graph *graph, const taps_cluster *cluster,
                                      uint64_t *op_offsets, taps_strategy *strategies,
                                      uint64_t capacity, void *stream);

/* The strategies of taps_enumerate_strategies that a search over a fixed
 * device mesh can express (an extension: the paper's device matrices are
 * free, Auxiliary Graph section): every split axis is sharded over whole,
 * consecutive mesh dimensions, i.e. each prefix product of the strategy's
 * device matrix (innermost first) is a prefix product of the mesh.  Same
 * canonical order, a subsequence of the unrestricted set; before the
 * divisibility filter the count is the paper's formula with n replaced by
 * mesh->n_dims.  The tables of taps_node_costs, taps_edge_costs and the
 * other calls take these strategies as they take any others.
 *   mesh  host; TAPS_ERR_TOPOLOGY if a size is not a power of two >= 2, the
 *         product differs from N, or n_dims > TAPS_MAX_LEVELS.
 * Other arguments, outputs and errors as taps_enumerate_strategies. */
taps_status taps_enumerate_strategies_mesh(const taps_graph *graph, const taps_cluster *cluster,
                                           const taps_mesh *mesh, uint64_t *op_offsets,
                                           taps_strategy *strategies, uint64_t capacity,
                                           void *stream);

/* The whole build in one call, without a host synchronisation: the strategies
 * of taps_enumerate_strategies (or, with a mesh, of
 * taps_enumerate_strategies_mesh), the node table of taps_node_costs and the
 * edge table of taps_edge_costs, bit for bit.  The per-operator strategy
 * counts are computed on the host by an exact count of the same filter
 * (ordered runs of distinct partitionable axes covering the n levels, each
 * at most as wide as its length allows, each boundary a mesh boundary), so
 * op_offsets and edge_offsets are known before any GPU work and the whole
 * build is queued on `stream` at once (a caller can queue the next build
 * while this one runs).
 *   mesh          host, or NULL for every device matrix.
 *   op_offsets    host, n_ops + 1 entries, written.
 *   strategies    device, strategy_capacity entries; node: device arrays of
 *                 strategy_capacity records.
 *   edge_offsets  host, n_edges + 1 entries, written; edge: device arrays of
 *                 edge_capacity records, layout as taps_edge_costs.
 *   strategies NULL and every table array NULL: size query (host only).  The
 *   edge arrays may be NULL when the graph has no edge entries.
 *   flags         0, or TAPS_BUILD_SHARED: edges described alike (as for
 *                 taps_edge_costs_shared) share one computed table, copied to
 *                 the others; the strategies here are the library's own, so the
 *                 grouping needs no device comparison and the call still does
 *                 not synchronise.  The tables are the same either way.
 * TAPS_ERR_NO_STRATEGY, TAPS_ERR_CAPACITY (either capacity), TAPS_ERR_TOPOLOGY
 * (cluster or mesh) and TAPS_ERR_ARG (also for unknown flags) as the separate
 * calls, all before any GPU work; outputs are valid after a stream
 * synchronisation.  The events of taps_set_edge_kernel_events bracket the
 * edge-table kernel and, when shared, the copies after it. */
#define TAPS_BUILD_SHARED 1u
taps_status taps_build_tables(const taps_graph *graph, const taps_cluster *cluster,
                              const taps_mesh *mesh, uint64_t *op_offsets,
                              taps_strategy *strategies, uint64_t strategy_capacity, taps_table node,
                              uint64_t *edge_offsets, taps_table edge, uint64_t edge_capacity,
                              uint32_t flags, void *stream);

/* taps_build_tables for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, outputs and errors, the same tables bit for
 * bit; the caller still provides every output array.  The call's device
 * workspace (the uploaded graph and plan, strategy descriptors, per-edge
 * constants, row segments) lives in a fixed array of
 * TAPS_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until
 * the process ends; the plan is uploaded with one hipMemcpyAsync from
 * pageable host memory.  No hipMalloc, hipFree, hipHostMalloc or other
 * allocating routine is called.
 * TAPS_ERR_CAPACITY, before any GPU work, if a build needs more workspace
 * than that (the 96-layer GPT on 128 devices needs about 21 MB).
 * Every call on one GPU uses that GPU's single array: calls that overlap on
 * one GPU (other streams, other threads) race and must be serialised by the
 * caller; consecutive calls on one stream are ordered and safe. */
#define TAPS_NOALLOC_SCRATCH_BYTES ((uint64_t)32 << 20)
taps_status taps_build_tables_noalloc(const taps_graph *graph, const taps_cluster *cluster,
                                      const taps_mesh *mesh, uint64_t *op_offsets,
                                      taps_strategy *strategies, uint64_t strategy_capacity,
                                      taps_table node, uint64_t *edge_offsets, taps_table edge,
                                      uint64_t edge_capacity, uint32_t flags, void *stream);

/* Intra-operator cost of every strategy (Eq. 5-8 generalised to any
 * operator: one ring AllReduce per tensor that lacks some split axis -- the
 * forward partial sum of the output, the backward gradient of an input or
 * weight -- with volume 2(g-1)/g of its shard; Algorithm 2 gives the
 * inter-node groups, Eq. 11-12 the cost).
 *   strategies  device, from taps_enumerate_strategies for the same graph
 *               and cluster; op_offsets host, as that call returned it.
 *   out         device arrays of op_offsets[n_ops] records, one per strategy. */
taps_status taps_node_costs(const taps_graph *graph, const taps_cluster *cluster,
                            const taps_strategy *strategies, const uint64_t *op_offsets,
                            taps_table out, void *stream);

/* Redistribution cost of every (producer strategy i, consumer strategy j)
 * pair of every edge (Algorithm 4's pair loop).  Per pair: the device
 * matrices and tensor shapes are unified (Table 1); Algorithm 1's sequence,
 * the same without AllToAll and the "remove" sequence of Table 2 are costed
 * with Eq. 9-10 volumes and Algorithm 3 / Eq. 14 inter-node groups
 * (Eq. 11, 13, 14); the record keeps the cheapest in seconds (exact
 * comparison, ties to the lower index), and vol the smallest volume.
 *   edge_offsets  host, n_edges + 1 entries, written: edge e's table is
 *                 entries [edge_offsets[e], edge_offsets[e+1]), row-major,
 *                 entry edge_offsets[e] + i * S_dst + j.
 *   out           device arrays of `capacity` records; all five NULL: only
 *                 edge_offsets is written (size query).
 * TAPS_ERR_CAPACITY if edge_offsets[n_edges] > capacity. */
taps_status taps_edge_costs(const taps_graph *graph, const taps_cluster *cluster,
                            const taps_strategy *strategies, const uint64_t *op_offsets,
                            uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                            void *stream);

/* The same tables as taps_edge_costs, written with each distinct table
 * computed once.  Edges with the same producer (axes, lengths, partitionable
 * axes, element size, output tensor) and the same consumer (axes, lengths,
 * partitionable axes, the input tensor the edge feeds) have the same table
 * whenever their operators' strategy ranges are equal -- which holds for the
 * strategies taps_enumerate_strategies writes and is checked on the device
 * for any others.  The paper relies on the same fact when it searches one
 * layer of a stack of identical transformer layers (searching runtime
 * subsection).  Each group's first edge is computed and every other member's
 * range is copied from it.  Unlike taps_edge_costs this call synchronises the
 * stream once (to read back the strategy comparison) when some edges share.
 * Arguments, layout and errors as taps_edge_costs. */
taps_status taps_edge_costs_shared(const taps_graph *graph, const taps_cluster *cluster,
                                   const taps_strategy *strategies, const uint64_t *op_offsets,
                                   uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                   void *stream);

/* The backward direction of every edge: in the backward pass the gradient of
 * the edge tensor leaves the consumer in the consumer's input map (fully
 * reduced: its AllReduce is in the consumer's node cost) and must reach the
 * producer in the producer's output map.  The same candidates and selection
 * as taps_edge_costs, with the roles of the two maps swapped; same shape and
 * element size.  The paper costs only the forward direction (the edge-weight
 * paragraph after Algorithm 4); a search that also charges the backward
 * redistribution adds these tables.
 *   edge_offsets  as taps_edge_costs (S_src * S_dst entries per edge);
 *                 edge e's table is consumer-major: entry
 *                 edge_offsets[e] + j * S_src + i for producer strategy i and
 *                 consumer strategy j.
 * Other arguments and errors as taps_edge_costs. */
taps_status taps_edge_costs_backward(const taps_graph *graph, const taps_cluster *cluster,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                     void *stream);

/* The node and edge tables under a hierarchy of link classes (an extension
 * of Eq. 11-14).  A collective belongs to the smallest block size that holds
 * each of its groups (class c: the first domain[c] whose Algorithm 2 / 3
 * inter-block count is zero); it pays bw[c] divided by ct, the number of its
 * groups that share the uplink of one domain[c-1] block (Algorithm 2 / 3 and
 * the AllToAll paragraph with "node" read as that block; an AllToAll's uplink
 * carries k(p-k)/p of the shard per group, k = members in one block).  Fields:
 * t = sum over classes of (link volume x ct) / (N bw[c]); intra = the class-0
 * volume; inter = the sum over the other classes of link volume x ct; vol and
 * meta as before ("inter-node" read as "leaving a domain[0] block").
 * Candidates compare exactly by sum_c x_c lcm(bw) / bw[c] (bw_a2a, if set,
 * prices the in-block AllToAll volume, which stays in intra).  With the
 * domains (L, N) and bw_a2a 0 the tables equal those of taps_node_costs /
 * taps_edge_costs.
 *   topology  host; TAPS_ERR_TOPOLOGY unless n_classes is 1..TAPS_MAX_CLASSES,
 *             every domain is a power of two, non-decreasing, the last one
 *             N <= 2^TAPS_MAX_LEVELS, every bw > 0 and lcm(bw) / bw[c] < 2^30
 *             for every c, bw_a2a included (bandwidths in round ratios).
 *   strategies from taps_enumerate_strategies(_mesh) on N devices.
 * Other arguments, layouts and errors as taps_node_costs / taps_edge_costs. */
taps_status taps_node_costs_topology(const taps_graph *graph, const taps_topology *topology,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     taps_table out, void *stream);
taps_status taps_edge_costs_topology(const taps_graph *graph, const taps_topology *topology,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                     void *stream);

/* Per-device memory of every strategy: the memory cost that the ILP's
 * device-memory constraint (Eq. 18) sums, which the paper names but never
 * defines.  Reading used here: a strategy keeps on each device one shard of
 * each of the operator's weights and one shard of its output (an input is
 * another operator's output and is counted there); a tensor dimension on op
 * axis a is cut into 2^log2_deg[a] equal parts when the strategy splits a
 * (pos[a] >= 0), so a shard holds prod_d (axis_len / 2^log2_deg) elements of
 * dtype_bytes bytes.  Exact for strategies whose degrees divide their axes
 * (every strategy taps_enumerate_strategies writes); for others each
 * dimension's length is divided with the remainder dropped.
 *   strategies  device, op_offsets[n_ops] entries; op_offsets host.
 *   memory      device, op_offsets[n_ops] bytes per device, one per strategy.
 * TAPS_ERR_ARG on NULL arguments (strategies and memory may be NULL when
 * there are no strategies); TAPS_ERR_DEVICE if the launch fails. */
taps_status taps_memory_costs(const taps_graph *graph, const taps_strategy *strategies,
                              const uint64_t *op_offsets, uint64_t *memory, void *stream);

/* The tables of taps_edge_costs at several bandwidth points in one pass:
 * clusters[k] (k < n_points <= TAPS_MAX_SWEEP) must have the same nodes and
 * devices_per_node and may differ in bw_intra and bw_inter.  The candidate
 * sequences of an entry (Table 2) and their volumes, intra- and inter-node
 * bytes and collective counts do not depend on the bandwidths; only the
 * choice among them (Eq. 9, 10, 14 times) and t do.  So each entry's
 * candidates are costed once and the choice, scaling and store are made once
 * per point -- the bandwidth sweep of the evaluation (the wide-MLP workload
 * is costed at several inter-node bandwidths).  out[k] receives the table of
 * clusters[k], bit for bit what taps_edge_costs(graph, &clusters[k], ...)
 * writes.
 *   out           host array of n_points tables (device arrays of `capacity`
 *                 records each, same layout as taps_edge_costs); out NULL or
 *                 every array of every table NULL: size query.
 * TAPS_ERR_ARG if n_points is 0 or above TAPS_MAX_SWEEP, if the points differ
 * in nodes or devices_per_node, or if some but not all arrays are NULL; other
 * arguments and errors as taps_edge_costs. */
taps_status taps_edge_costs_sweep(const taps_graph *graph, const taps_cluster *clusters,
                                  uint32_t n_points, const taps_strategy *strategies,
                                  const uint64_t *op_offsets, uint64_t *edge_offsets,
                                  const taps_table *out, uint64_t capacity, void *stream);

/* Profiling aid, not part of the method: `before` and `after` are HIP events
 * (hipEvent_t, created by the caller, passed as plain pointers) that the
 * calling thread's next taps_edge_costs, taps_edge_costs_shared,
 * taps_edge_costs_backward, taps_edge_costs_sweep, taps_edge_costs_topology
 * or taps_build_tables call that launches the edge-table kernel records on
 * its stream immediately before and after that
 * kernel (and, for shared tables, the copies after it), so that
 * the caller can time the kernel alone.  The setting is thread-local,
 * used once and then cleared; two NULLs clear it.  The events stay owned by
 * the caller.  TAPS_ERR_ARG if exactly one of them is NULL. */
taps_status taps_set_edge_kernel_events(void *before, void *after);

/* Launch-shape setting, not part of the method: single-table edge launches
 * (taps_edge_costs, taps_edge_costs_shared, taps_edge_costs_backward,
 * taps_edge_costs_topology, taps_build_tables) whose tables hold at least
 * `min_segments` row segments of eight 64-entry tiles run those long segments
 * (each edge's full-length segments first, the rows' remainders last, longest
 * first); smaller launches run segments of at most two tiles in row order (the
 * bandwidth sweep runs aligned 64-entry windows of its tables instead).  Every
 * shape writes the same tables; the setting only moves the size at which a
 * single-table launch changes shape (default 32768; 0 or 1: every launch with at least one segment
 * runs long ones).  Process-wide, read when a
 * launch is planned; returns the previous value.  Never fails. */
uint64_t taps_set_long_segments_min(uint64_t min_segments);

/* Static name of a status code. */
const char *taps_status_str(taps_status status);

/* Description of the calling thread's last failure ("" if none). */
const char *taps_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TAPS_H */

/*
 * taps_oracle.c -- CPU oracle for the TAPS cost tables.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * statement of what the cost tables contain.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg load it.  The library's GPU path
 * never calls it, and the two share no code: this file works on explicit
 * device matrices and tensor maps in the paper's notation, the GPU path on
 * packed binary-level masks.
 *
 * Paper: P. Liang, H. Zheng, T. Su, L. Qiao, D. Li, "TAPS: Topology-Aware
 * Intra-Operator Parallelism Strategy Searching Algorithm for Deep Neural
 * Networks", arXiv 2301.04285.
 *
 * Notation, as in the paper:
 *   device matrix  D = [d_{h-1}, ..., d_0]  (stored here as D[0..h-1], D[0]
 *                  innermost, i.e. the axis whose devices are adjacent);
 *   tensor map     M = [m_0, ..., m_{n-1}], m_i = the device-matrix axis that
 *                  splits tensor dimension i, or -1 when dimension i is whole
 *                  (replicated along every axis that no dimension uses).
 * A device's rank is mixed-radix over D with axis 0 fastest; with L devices
 * per node, rank r lives on node floor(r / L).
 *
 * Units.  Every volume is an integer number of "nb" = bytes x N, where N is
 * the device count: all group sizes divide N, so per-device volumes such as
 * 2(g-1)/g * data_size become exact integers.  Time costs (seconds) are fp64
 * and are computed with the paper's own formula, cost = volume / B_e.
 *
 * Readings of the paper that this file takes (each is stated again at the
 * function that uses it):
 *   R-a  strategies whose degree does not divide the axis length are dropped;
 *        with one device the only strategy leaves every axis whole;
 *   R-b  enumeration order: degree tuple ascending, then device-map tuple
 *        descending (reproduces Table 3's order);
 *   R-c  intra-op cost: one ring AllReduce per tensor that lacks some split
 *        axis (forward partial sum for the output, backward gradient for
 *        inputs and weights), generalising Eq. 5-7; ops whose tensors all
 *        carry every split axis cost nothing;
 *   R-d  Algorithm 2's in-node factor multiplies instead of replacing the
 *        running product when an axis straddles the node boundary;
 *   R-e  Algorithm 3 loops over the device axes inside the gathered axis and
 *        counts as shareable replicas only the part of an unused axis that
 *        lies inside one node; AllToAll takes k and r from the same place;
 *   R-f  Table 1's two-step unification is repeated until neither step
 *        changes anything;
 *   R-g  InferSlice and InferAll2All make one pass over the dimensions in
 *        ascending order, InferAllGather emits a single AllGather (lowest
 *        dimension), AllGatherFirstUndoneDim does nothing when every split
 *        dimension already has its target axis;
 *   R-h  the redistribution cost of an edge is the cheapest of the four
 *        sequences Table 2 shows (replace = Algorithm 1, rearrange = without
 *        AllToAll, remove, naive), ties to the first; the volume table takes
 *        the smallest volume of the four;
 *   R-i  partial sums of the producer are resolved inside the producer's own
 *        intra-op cost, so the edge sees those axes as replicated;
 *   R-j  (an extension) a hierarchy of link classes: blocks of domain[0] <=
 *        domain[1] <= ... <= domain[C-1] = N consecutive ranks; a collective
 *        belongs to the smallest domain whose Algorithm 2 / 3 count is zero
 *        (its group fits inside one block), takes that class's bandwidth and
 *        the count of the next smaller domain as its ct; with the domains
 *        (L, N) this is the paper's two-class model.  An AllToAll inside one
 *        domain[0] block may take its own bandwidth (peer to peer over every
 *        link of the block, where a ring uses one).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_MAX_AXES 8
#define OR_MAX_RANK 8
#define OR_MAX_IN 4
#define OR_MAX_W 4
#define OR_MAX_DEV 16   /* axes of a (unified) device matrix */
#define OR_MAX_SUB 48   /* dimensions of a unified tensor     */
#define OR_MAX_SEQ 96   /* operators in one redistribution    */

typedef struct {
    int32_t rank;
    int32_t axis[OR_MAX_RANK];
} or_tensor;

typedef struct {
    int32_t n_axes, part_mask, dtype_bytes, n_in, n_w;
    int32_t pad_;
    int64_t axis_len[OR_MAX_AXES];
    or_tensor in[OR_MAX_IN], w[OR_MAX_W], out;
} or_op;

/* A parallelism strategy (Table 3): per op axis, its degree (1 = not split)
 * and its device-map entry (-1 = not split; 0 = innermost device axis). */
typedef struct {
    int32_t degree[OR_MAX_AXES];
    int32_t pos[OR_MAX_AXES];
} or_strategy;

typedef struct {
    double t;           /* seconds */
    uint64_t vol;       /* nb, communication volume */
    uint64_t intra;     /* nb sent over intra-node links */
    uint64_t inter;     /* nb x ct sent over inter-node links */
    uint32_t meta;      /* candidate | collectives<<2 | inter collectives<<7 | sum ct<<12 */
    uint32_t pad_;
} or_record;

enum { OR_SLICE = 0, OR_ALLGATHER = 1, OR_ALLTOALL = 2 };

typedef struct {
    int32_t kind, axis, from_dim, to_dim;  /* Slice(axis, to_dim); AllGather(axis, from_dim);
                                             AllToAll(axis, from_dim -> to_dim) */
    int32_t ct, k_in;                       /* inter-node groups per node; members per node */
    uint64_t shard_nb;                      /* per-device data size before the op, in nb */
    uint64_t volume_nb;                     /* Eq. 9 / Eq. 10 volume */
    uint64_t link_nb;                       /* volume carried by the link class (Eq. 14 for AllToAll) */
    double cost;                            /* seconds */
} or_redop;

/* Link classes (reading R-j).  Class 0: links inside one block of domain[0]
 * consecutive ranks (a node); class c >= 1: links between the domain[c-1]
 * blocks of one domain[c] block, bw[c] bytes/s each.  domain[] is
 * non-decreasing, domain[n_classes - 1] = N.  The paper's cluster is
 * {2, {L, N}, {B_intra, B_inter}}. */
#define OR_MAX_CLASSES 4
typedef struct {
    int32_t n_classes;
    int32_t pad_;
    int64_t domain[OR_MAX_CLASSES];
    uint64_t bw[OR_MAX_CLASSES];
    uint64_t bw_a2a;   /* an AllToAll inside one domain[0] block: bytes/s (0: bw[0]) */
} or_topology;

static or_topology two_class(int64_t N, int64_t L, uint64_t Bintra, uint64_t Binter) {
    or_topology t;
    memset(&t, 0, sizeof t);
    t.n_classes = 2;
    t.domain[0] = L;
    t.domain[1] = N;
    t.bw[0] = Bintra;
    t.bw[1] = Binter;
    return t;
}

typedef struct {
    int32_t h;                  /* depth of the unified device matrix */
    int32_t r;                  /* rank of the unified tensor */
    int64_t D[OR_MAX_DEV];      /* unified device matrix, D[0] innermost */
    int32_t orig[OR_MAX_SUB];   /* original tensor dimension of each unified dimension */
    int64_t size[OR_MAX_SUB];   /* unified shape */
    int32_t m_from[OR_MAX_SUB]; /* tensor map on the producer side */
    int32_t m_to[OR_MAX_SUB];   /* tensor map on the consumer side */
} or_unified;

/* ---------------------------------------------------------------------------
 * GenerateStrategySet (Auxiliary Graph section; Table 3).
 *
 * A strategy picks i of the p partitionable axes, gives each a degree that is
 * a power of two greater than one, with the degrees multiplying to N = 2^n,
 * and orders the chosen axes on device-matrix positions 0..i-1.  Before
 * filtering there are sum_i i! C(p,i) C(n-1,i-1) of them.  Reading R-a drops a
 * strategy whose degree does not divide the axis length; reading R-b fixes
 * the order.
 * ------------------------------------------------------------------------- */

typedef struct {
    or_strategy *buf;
    int64_t len, cap;
} strat_vec;

static int vec_push(strat_vec *v, const or_strategy *s) {
    if (v->len == v->cap) {
        int64_t nc = v->cap ? 2 * v->cap : 64;
        or_strategy *nb = (or_strategy *)realloc(v->buf, (size_t)nc * sizeof(or_strategy));
        if (!nb) return -1;
        v->buf = nb;
        v->cap = nc;
    }
    v->buf[v->len++] = *s;
    return 0;
}

static int g_sort_axes;

static int strategy_order(const void *pa, const void *pb) {
    const or_strategy *a = (const or_strategy *)pa, *b = (const or_strategy *)pb;
    for (int x = 0; x < g_sort_axes; ++x)          /* degree tuple, ascending */
        if (a->degree[x] != b->degree[x]) return a->degree[x] < b->degree[x] ? -1 : 1;
    for (int x = 0; x < g_sort_axes; ++x)          /* device-map tuple, descending */
        if (a->pos[x] != b->pos[x]) return a->pos[x] > b->pos[x] ? -1 : 1;
    return 0;
}

/* all orderings of the split axes onto positions 0..i-1 */
static int emit_orderings(const or_op *op, or_strategy *s, const int *split, int i, int depth,
                          int used_pos, int filter, strat_vec *v) {
    if (depth == i) {
        if (filter)
            for (int x = 0; x < op->n_axes; ++x)
                if (op->axis_len[x] % s->degree[x] != 0) return 0;
        return vec_push(v, s);
    }
    for (int q = 0; q < i; ++q) {
        if (used_pos & (1 << q)) continue;
        s->pos[split[depth]] = q;
        if (emit_orderings(op, s, split, i, depth + 1, used_pos | (1 << q), filter, v)) return -1;
    }
    s->pos[split[depth]] = -1;
    return 0;
}

/* choose the degree of axis x, given the product still to place */
static int choose_degrees(const or_op *op, or_strategy *s, int x, int64_t remaining, int filter,
                          strat_vec *v) {
    if (x == op->n_axes) {
        if (remaining != 1) return 0;
        int split[OR_MAX_AXES], i = 0;
        for (int y = 0; y < op->n_axes; ++y)
            if (s->degree[y] > 1) split[i++] = y;
        return emit_orderings(op, s, split, i, 0, 0, filter, v);
    }
    s->degree[x] = 1;
    s->pos[x] = -1;
    if (choose_degrees(op, s, x + 1, remaining, filter, v)) return -1;
    if (op->part_mask & (1 << x)) {
        for (int64_t deg = 2; deg <= remaining; deg *= 2) {
            if (remaining % deg) break;
            s->degree[x] = (int32_t)deg;
            if (choose_degrees(op, s, x + 1, remaining / deg, filter, v)) return -1;
        }
    }
    s->degree[x] = 1;
    s->pos[x] = -1;
    return 0;
}

/* Writes up to cap strategies in canonical order; returns how many there are
 * (or -1 on allocation failure).  filter = 0 keeps non-dividing degrees (used
 * to check the count formula). */
int64_t or_enumerate(const or_op *op, int64_t N, int filter, or_strategy *out, int64_t cap) {
    strat_vec v = {0, 0, 0};
    or_strategy s;
    memset(&s, 0, sizeof s);
    for (int x = 0; x < OR_MAX_AXES; ++x) {
        s.degree[x] = 1;
        s.pos[x] = -1;
    }
    if (choose_degrees(op, &s, 0, N, filter, &v)) {
        free(v.buf);
        return -1;
    }
    g_sort_axes = op->n_axes;
    if (v.len > 1) qsort(v.buf, (size_t)v.len, sizeof(or_strategy), strategy_order);
    for (int64_t k = 0; k < v.len && k < cap; ++k) out[k] = v.buf[k];
    int64_t n = v.len;
    free(v.buf);
    return n;
}

/* ---------------------------------------------------------------------------
 * Device matrix and tensor maps of one strategy.
 * ------------------------------------------------------------------------- */

static int device_matrix(const or_op *op, const or_strategy *s, int64_t *D) {
    int h = 0;
    for (int x = 0; x < op->n_axes; ++x)
        if (s->degree[x] > 1) ++h;
    for (int x = 0; x < op->n_axes; ++x)
        if (s->degree[x] > 1) D[s->pos[x]] = s->degree[x];
    return h;
}

/* ---------------------------------------------------------------------------
 * Fixed-mesh strategy spaces (an extension; the paper's device matrix is
 * free).
 *
 * A search over a fixed physical mesh [m_0, m_1, ..., m_{k-1}] (m_0 innermost,
 * the product is N) shards an operator axis over whole mesh dimensions only:
 * the strategy's device matrix D = [d_{h-1}, ..., d_0] must group consecutive
 * mesh dimensions, i.e. every prefix product d_0 ... d_j is a prefix product
 * m_0 ... m_i of the mesh.  The candidates before the divisibility filter are
 * then counted by the paper's formula with n replaced by k: a strategy picks i
 * axes, an ordering, and a composition of the k mesh dimensions into i runs.
 * ------------------------------------------------------------------------- */

static int on_mesh(const or_op *op, const or_strategy *s, const int64_t *mesh, int k) {
    int64_t D[OR_MAX_DEV];
    const int h = device_matrix(op, s, D);
    int i = 0;
    int64_t mp = 1, dp = 1;
    for (int j = 0; j < h; ++j) {
        dp *= D[j];
        while (i < k && mp < dp) mp *= mesh[i++];
        if (mp != dp) return 0;
    }
    return 1;
}

/* The strategies of or_enumerate on N = prod(mesh) devices that lie on the
 * mesh, in the same (canonical) order; returns how many (-1 on allocation
 * failure). */
int64_t or_enumerate_mesh(const or_op *op, const int64_t *mesh, int k, int filter,
                          or_strategy *out, int64_t cap) {
    int64_t N = 1;
    for (int i = 0; i < k; ++i) N *= mesh[i];
    const int64_t all = or_enumerate(op, N, filter, NULL, 0);
    if (all < 0) return -1;
    or_strategy *buf = (or_strategy *)malloc((size_t)(all ? all : 1) * sizeof(or_strategy));
    if (!buf) return -1;
    or_enumerate(op, N, filter, buf, all);
    int64_t n = 0;
    for (int64_t x = 0; x < all; ++x) {
        if (!on_mesh(op, &buf[x], mesh, k)) continue;
        if (n < cap) out[n] = buf[x];
        ++n;
    }
    free(buf);
    return n;
}

static void tensor_map(const or_tensor *t, const or_strategy *s, int32_t *M) {
    for (int d = 0; d < t->rank; ++d) {
        int a = t->axis[d];
        M[d] = s->degree[a] > 1 ? s->pos[a] : -1;
    }
}

static int map_uses(const int32_t *M, int r, int k) {
    for (int d = 0; d < r; ++d)
        if (M[d] == k) return 1;
    return 0;
}

static int64_t tensor_elems(const or_op *op, const or_tensor *t) {
    int64_t e = 1;
    for (int d = 0; d < t->rank; ++d) e *= op->axis_len[t->axis[d]];
    return e;
}

/* ---------------------------------------------------------------------------
 * Where the devices of one node sit in the device matrix (the rank layout of
 * reading R-a: axis 0 fastest, node = rank / L).  Axis k advances the rank
 * in steps of stride_k = D[0] ... D[k-1]; every size is a power of two, so
 * the ranks of one node (L consecutive ranks, or all N when N < L) take
 * in_node(k) = min(D[k], max(1, L / stride_k)) distinct coordinates of axis
 * k, the same ones on every node.
 * ------------------------------------------------------------------------- */
static int64_t axis_stride(const int64_t *D, int k) {
    int64_t s = 1;
    for (int j = 0; j < k; ++j) s *= D[j];
    return s;
}

static int64_t in_node(const int64_t *D, int k, int64_t L) {
    const int64_t per_node = L / axis_stride(D, k);
    return per_node <= 1 ? 1 : (per_node < D[k] ? per_node : D[k]);
}

static int64_t devices_per_node(const int64_t *D, int h, int64_t L) {
    const int64_t N = axis_stride(D, h);
    return N < L ? N : L;
}

/* ---------------------------------------------------------------------------
 * Algorithm 2 (inter-node groups of the AllReduce of a tensor with map M over
 * the axes M does not use), from the layout above.  A group is the set of
 * devices that agree on every axis M uses; it has prod D[k] members over the
 * unused axes k, prod in_node(k) of them on one node.  If that is all of
 * them, the group never leaves its node: 0.  Otherwise every group that
 * touches a node crosses to other nodes, and the node's devices belong to
 * devices_per_node / (members on the node) such groups: the count of groups
 * sharing the node's uplink (Eq. 11-12).  Multiplying the in-node parts of
 * all unused axes is reading R-d.
 * ------------------------------------------------------------------------- */
int64_t or_allreduce_ct(const int64_t *D, int h, const int32_t *M, int r, int64_t L) {
    int64_t members = 1, on_node = 1;
    for (int k = 0; k < h; ++k) {
        if (map_uses(M, r, k)) continue;
        members *= D[k];
        on_node *= in_node(D, k, L);
    }
    if (on_node == members) return 0;
    return devices_per_node(D, h, L) / on_node;
}

/* ---------------------------------------------------------------------------
 * Algorithm 3 (inter-node groups of an AllGather, or AllToAll, along axis g of
 * a tensor with map M), from the same layout.  A group is the D[g] devices
 * that differ only along g, in_node(g) of them on one node (*k_in, the k of
 * the AllToAll paragraph).  If that is all of them the group stays inside its
 * node: 0.  Otherwise the node's devices belong to devices_per_node /
 * in_node(g) groups, and groups that hold the same data -- they differ only
 * along axes M does not use -- share one inter-node transfer, but only among
 * the groups on the same node, i.e. through the in-node part of each such
 * axis (reading R-e): the count is the groups on a node divided by the
 * product of in_node(k) over the unused axes k other than g.
 * ------------------------------------------------------------------------- */
int64_t or_gather_ct(const int64_t *D, int h, const int32_t *M, int r, int g, int64_t L,
                     int64_t *k_in) {
    const int64_t members_on_node = in_node(D, g, L);
    *k_in = members_on_node;
    if (members_on_node == D[g]) return 0;
    int64_t replicas = 1;
    for (int k = 0; k < h; ++k)
        if (k != g && !map_uses(M, r, k)) replicas *= in_node(D, k, L);
    return devices_per_node(D, h, L) / members_on_node / replicas;
}

/* ---------------------------------------------------------------------------
 * Intra-operator cost of one strategy (Eq. 5-8 generalised, reading R-c).
 * For each tensor that lacks some split axis: one ring AllReduce over the
 * axes it lacks, group size g, volume 2(g-1)/g * data_size (Eq. 5), cost
 * V / B_e (Eq. 11, Eq. 12) with ct from Algorithm 2.
 * ------------------------------------------------------------------------- */
static void allreduce_tensor(const or_op *op, const or_tensor *t, const int64_t *D, int h,
                             const or_strategy *s, int64_t N, const or_topology *topo,
                             or_record *rec, uint32_t *n_coll, uint32_t *n_inter,
                             uint32_t *sum_ct) {
    int32_t M[OR_MAX_RANK];
    tensor_map(t, s, M);
    int64_t used = 1;
    for (int d = 0; d < t->rank; ++d)
        if (M[d] >= 0) used *= D[M[d]];
    int64_t g = N / used;            /* product of the axes the tensor lacks */
    if (g == 1) return;
    uint64_t data_nb = (uint64_t)tensor_elems(op, t) * (uint64_t)op->dtype_bytes * (uint64_t)N /
                       (uint64_t)used;
    uint64_t V = 2 * (uint64_t)(g - 1) * data_nb / (uint64_t)g;
    /* reading R-j: the smallest domain that holds the group, ct of the next smaller one */
    int cls = 0;
    while (cls < topo->n_classes - 1 && or_allreduce_ct(D, h, M, t->rank, topo->domain[cls]) != 0)
        ++cls;
    int64_t ct = cls ? or_allreduce_ct(D, h, M, t->rank, topo->domain[cls - 1]) : 0;
    rec->vol += V;
    *n_coll += 1;
    if (ct == 0) {
        rec->intra += V;
        rec->t += ((double)V / (double)N) / (double)topo->bw[0];
    } else {
        rec->inter += V * (uint64_t)ct;
        double Be = (double)topo->bw[cls] / (double)ct;
        rec->t += ((double)V / (double)N) / Be;
        *n_inter += 1;
        *sum_ct += (uint32_t)ct;
    }
}

void or_node_cost_topo(const or_op *op, const or_strategy *s, int64_t N, const or_topology *topo,
                       or_record *rec) {
    int64_t D[OR_MAX_DEV];
    int h = device_matrix(op, s, D);
    uint32_t n_coll = 0, n_inter = 0, sum_ct = 0;
    memset(rec, 0, sizeof *rec);
    allreduce_tensor(op, &op->out, D, h, s, N, topo, rec, &n_coll, &n_inter, &sum_ct);
    for (int k = 0; k < op->n_in; ++k)
        allreduce_tensor(op, &op->in[k], D, h, s, N, topo, rec, &n_coll, &n_inter, &sum_ct);
    for (int k = 0; k < op->n_w; ++k)
        allreduce_tensor(op, &op->w[k], D, h, s, N, topo, rec, &n_coll, &n_inter, &sum_ct);
    rec->meta = (n_coll << 2) | (n_inter << 7) | (sum_ct << 12);
}

void or_node_cost(const or_op *op, const or_strategy *s, int64_t N, int64_t L, uint64_t Bintra,
                  uint64_t Binter, or_record *rec) {
    const or_topology topo = two_class(N, L, Bintra, Binter);
    or_node_cost_topo(op, s, N, &topo, rec);
}

int64_t or_node_table_topo(const or_op *op, const or_strategy *s, int64_t count, int64_t N,
                           const or_topology *topo, or_record *out) {
    for (int64_t k = 0; k < count; ++k) or_node_cost_topo(op, &s[k], N, topo, &out[k]);
    return count;
}

int64_t or_node_table(const or_op *op, const or_strategy *s, int64_t count, int64_t N, int64_t L,
                      uint64_t Bintra, uint64_t Binter, or_record *out) {
    for (int64_t k = 0; k < count; ++k) or_node_cost(op, &s[k], N, L, Bintra, Binter, &out[k]);
    return count;
}

/* ---------------------------------------------------------------------------
 * Unifying device matrix and tensor shape (Table 1), reading R-f.
 *
 * Step 1 factorises both device matrices into their common refinement; a
 * tensor dimension split by an axis that became several axes is reshaped into
 * one dimension per factor (outermost factor first, the last dimension keeps
 * the remainder).  Step 2 reshapes each original dimension on both sides at
 * the union of both sides' reshape points.  If a reshape point falls inside
 * the part of a dimension that one device axis splits, that axis is factorised
 * (back to step 1).  Neither step changes which elements a device holds.
 * ------------------------------------------------------------------------- */

typedef struct {
    int64_t start;  /* product of the sizes of the pieces before it in its dimension */
    int64_t size;
    int32_t axis;
} piece;

static int add_boundary(int64_t *B, int *nb, int64_t b) {
    for (int k = 0; k < *nb; ++k)
        if (B[k] == b) return 0;
    if (*nb >= OR_MAX_DEV - 1) return -1;
    int k = *nb;
    while (k > 0 && B[k - 1] > b) {
        B[k] = B[k - 1];
        --k;
    }
    B[k] = b;
    ++*nb;
    return 1;
}

/* pieces of dimension d of one side, under the unified matrix */
static int side_pieces(int64_t s_d, int32_t m, const int64_t *side_cum, const int64_t *D,
                       const int64_t *cum, int h, piece *out) {
    if (m < 0) {
        out[0].start = 1;
        out[0].size = s_d;
        out[0].axis = -1;
        return 1;
    }
    int64_t lo = side_cum[m], hi = side_cum[m + 1];   /* the side's axis m spans [lo, hi) */
    int klo = -1, khi = -1;
    for (int k = 0; k < h; ++k) {
        if (cum[k] == lo) klo = k;
        if (cum[k] * D[k] == hi) khi = k;
    }
    int n = 0;
    int64_t start = 1;
    for (int k = khi; k > klo; --k) {
        out[n].start = start;
        out[n].size = D[k];
        out[n].axis = k;
        start *= D[k];
        ++n;
    }
    out[n].start = start;
    out[n].size = s_d / start;
    out[n].axis = klo;
    return n + 1;
}

int or_unify(int64_t N, const int64_t *Dp, int hp, const int32_t *Mp, const int64_t *Dc, int hc,
             const int32_t *Mc, int rank, const int64_t *shape, or_unified *u) {
    int64_t B[OR_MAX_DEV];
    int nb = 0;
    int64_t pc[OR_MAX_DEV + 1], cc[OR_MAX_DEV + 1];
    pc[0] = 1;
    for (int k = 0; k < hp; ++k) pc[k + 1] = pc[k] * Dp[k];
    cc[0] = 1;
    for (int k = 0; k < hc; ++k) cc[k + 1] = cc[k] * Dc[k];
    for (int k = 1; k < hp; ++k)
        if (add_boundary(B, &nb, pc[k]) < 0) return -1;
    for (int k = 1; k < hc; ++k)
        if (add_boundary(B, &nb, cc[k]) < 0) return -1;

    piece P[OR_MAX_RANK][OR_MAX_DEV + 1], C[OR_MAX_RANK][OR_MAX_DEV + 1];
    int np[OR_MAX_RANK], nc[OR_MAX_RANK];
    int64_t D[OR_MAX_DEV], cum[OR_MAX_DEV + 1];
    int h = 0;
    for (int iter = 0; iter < 4 * OR_MAX_DEV; ++iter) {
        /* step 1: the common refinement of both device matrices */
        h = nb + 1;
        int64_t prev = 1;
        for (int k = 0; k < nb; ++k) {
            D[k] = B[k] / prev;
            prev = B[k];
        }
        D[nb] = N / prev;
        cum[0] = 1;
        for (int k = 0; k < h; ++k) cum[k + 1] = cum[k] * D[k];
        for (int d = 0; d < rank; ++d) {
            np[d] = side_pieces(shape[d], Mp[d], pc, D, cum, h, P[d]);
            nc[d] = side_pieces(shape[d], Mc[d], cc, D, cum, h, C[d]);
        }
        /* step 2: reshape points of one side that cut the other side's pieces */
        int changed = 0;
        for (int d = 0; d < rank; ++d) {
            for (int side = 0; side < 2; ++side) {
                piece *mine = side ? C[d] : P[d];
                piece *other = side ? P[d] : C[d];
                int nm = side ? nc[d] : np[d], no = side ? np[d] : nc[d];
                for (int a = 1; a < no; ++a) {
                    int64_t point = other[a].start;
                    for (int b = 0; b < nm; ++b) {
                        if (!(mine[b].start < point && point < mine[b].start * mine[b].size))
                            continue;
                        int64_t rho = point / mine[b].start;
                        int32_t ax = mine[b].axis;
                        if (ax >= 0 && rho < D[ax]) {
                            int r = add_boundary(B, &nb, cum[ax] * (D[ax] / rho));
                            if (r < 0) return -1;
                            changed |= r;
                        }
                    }
                }
            }
        }
        if (!changed) break;
        if (iter == 4 * OR_MAX_DEV - 1) return -1;  /* no fixpoint: cannot happen for powers of two */
    }

    /* the common shape: each dimension cut at the union of both sides' points */
    u->h = h;
    for (int k = 0; k < h; ++k) u->D[k] = D[k];
    int r = 0;
    for (int d = 0; d < rank; ++d) {
        int64_t pts[2 * (OR_MAX_DEV + 1)];
        int npts = 0;
        for (int side = 0; side < 2; ++side) {
            piece *pp = side ? C[d] : P[d];
            int n = side ? nc[d] : np[d];
            for (int a = 0; a < n; ++a) {
                int dup = 0;
                for (int q = 0; q < npts; ++q)
                    if (pts[q] == pp[a].start) dup = 1;
                if (!dup) pts[npts++] = pp[a].start;
            }
        }
        for (int x = 1; x < npts; ++x)   /* insertion sort */
            for (int y = x; y > 0 && pts[y - 1] > pts[y]; --y) {
                int64_t t = pts[y];
                pts[y] = pts[y - 1];
                pts[y - 1] = t;
            }
        for (int q = 0; q < npts; ++q) {
            if (r >= OR_MAX_SUB) return -1;
            int64_t start = pts[q];
            u->orig[r] = d;
            u->size[r] = (q + 1 < npts) ? pts[q + 1] / start : shape[d] / start;
            for (int side = 0; side < 2; ++side) {
                piece *pp = side ? C[d] : P[d];
                int n = side ? nc[d] : np[d];
                int32_t m = -1;
                for (int a = 0; a < n; ++a)
                    if (pp[a].start == start) m = pp[a].axis;  /* leading part keeps the axis */
                if (side)
                    u->m_to[r] = m;
                else
                    u->m_from[r] = m;
            }
            ++r;
        }
    }
    u->r = r;
    return 0;
}

/* ---------------------------------------------------------------------------
 * Redistribution sequences (Table 2; Algorithm 1), reading R-g.
 * ------------------------------------------------------------------------- */

static int find_dim(const int32_t *M, int r, int axis) {
    for (int d = 0; d < r; ++d)
        if (M[d] == axis) return d;
    return -1;
}

static int push_op(or_redop *seq, int *len, int kind, int axis, int from, int to) {
    if (*len >= OR_MAX_SEQ) return -1;
    memset(&seq[*len], 0, sizeof(or_redop));
    seq[*len].kind = kind;
    seq[*len].axis = axis;
    seq[*len].from_dim = from;
    seq[*len].to_dim = to;
    ++*len;
    return 0;
}

/* every dimension that is whole now, split in the target, and whose target
 * axis no dimension uses yet: slice it */
static int infer_slice(int32_t *M, const int32_t *Mto, int r, or_redop *seq, int *len) {
    int found = 0;
    for (int d = 0; d < r; ++d) {
        if (M[d] == -1 && Mto[d] != -1 && find_dim(M, r, Mto[d]) < 0) {
            if (push_op(seq, len, OR_SLICE, Mto[d], -1, d)) return -1;
            M[d] = Mto[d];
            found = 1;
        }
    }
    return found;
}

/* every dimension that is whole now and whose target axis another dimension
 * holds: move the axis with one AllToAll */
static int infer_all2all(int32_t *M, const int32_t *Mto, int r, or_redop *seq, int *len) {
    int found = 0;
    for (int d = 0; d < r; ++d) {
        if (M[d] == -1 && Mto[d] != -1) {
            int i = find_dim(M, r, Mto[d]);
            if (i >= 0) {
                if (push_op(seq, len, OR_ALLTOALL, Mto[d], i, d)) return -1;
                M[i] = -1;
                M[d] = Mto[d];
                found = 1;
            }
        }
    }
    return found;
}

/* the first dimension that is split now but whole in the target */
static int infer_allgather(int32_t *M, const int32_t *Mto, int r, or_redop *seq, int *len) {
    for (int d = 0; d < r; ++d) {
        if (M[d] != -1 && Mto[d] == -1) {
            if (push_op(seq, len, OR_ALLGATHER, M[d], d, -1)) return -1;
            M[d] = -1;
            return 1;
        }
    }
    return 0;
}

/* the first dimension that is split by an axis other than its target one */
static int allgather_first_undone_dim(int32_t *M, const int32_t *Mto, int r, or_redop *seq,
                                      int *len) {
    for (int d = 0; d < r; ++d) {
        if (M[d] != -1 && M[d] != Mto[d]) {
            if (push_op(seq, len, OR_ALLGATHER, M[d], d, -1)) return -1;
            M[d] = -1;
            return 1;
        }
    }
    return 0;
}

static int maps_equal(const int32_t *a, const int32_t *b, int r) {
    for (int d = 0; d < r; ++d)
        if (a[d] != b[d]) return 0;
    return 1;
}

/* Slices and AllToAlls as far as they go (the inner part of Algorithm 1, with
 * readings R-g): slice every dimension whose target axis is free, then move
 * by AllToAll every target axis another dimension holds until none is left
 * (with use_a2a); repeat while the slices found something.  The AllToAlls of
 * the last round may free targets whose slices then wait for the next
 * settle. */
static int settle(int32_t *M, const int32_t *Mto, int r, int use_a2a, or_redop *seq, int *len) {
    for (;;) {
        const int sliced = infer_slice(M, Mto, r, seq, len);
        if (sliced < 0) return -1;
        for (int moved = use_a2a; moved;) {
            moved = infer_all2all(M, Mto, r, seq, len);
            if (moved < 0) return -1;
        }
        if (!sliced) return 0;
    }
}

/* Algorithm 1 ("replace"; without AllToAll, use_a2a = 0, the "rearrange"
 * sequence of Table 2): until the map reaches the target, settle it, then
 * gather one dimension -- the first one split now but whole in the target,
 * else the first one split by an axis that is not its target one (a no-op
 * when there is none, reading R-g).  Every round gathers or settles at least
 * one dimension, so 4r + 8 rounds bound it. */
static int optimized_redistribution(const int32_t *Mfrom, const int32_t *Mto, int r, int use_a2a,
                                    or_redop *seq) {
    int32_t M[OR_MAX_SUB];
    memcpy(M, Mfrom, sizeof(int32_t) * (size_t)r);
    int len = 0;
    for (int round = 0; !maps_equal(M, Mto, r); ++round) {
        if (round > 4 * r + 8 || settle(M, Mto, r, use_a2a, seq, &len) < 0) return -1;
        const int gathered = infer_allgather(M, Mto, r, seq, &len);
        if (gathered < 0) return -1;
        if (!gathered && allgather_first_undone_dim(M, Mto, r, seq, &len) < 0) return -1;
    }
    return len;
}

/* "remove" (Table 2 step 1): gather only the dimensions split by an axis that
 * is not their target one, then slice */
static int remove_redistribution(const int32_t *Mfrom, const int32_t *Mto, int r, or_redop *seq) {
    int32_t M[OR_MAX_SUB];
    memcpy(M, Mfrom, sizeof(int32_t) * (size_t)r);
    int len = 0;
    for (int d = 0; d < r; ++d)
        if (M[d] != -1 && M[d] != Mto[d]) {
            if (push_op(seq, &len, OR_ALLGATHER, M[d], d, -1)) return -1;
            M[d] = -1;
        }
    for (int d = 0; d < r; ++d)
        if (M[d] == -1 && Mto[d] != -1) {
            if (push_op(seq, &len, OR_SLICE, Mto[d], -1, d)) return -1;
            M[d] = Mto[d];
        }
    return len;
}

/* "naive" (Table 2 step 0): gather every split dimension, then slice */
static int naive_redistribution(const int32_t *Mfrom, const int32_t *Mto, int r, or_redop *seq) {
    int len = 0;
    for (int d = 0; d < r; ++d)
        if (Mfrom[d] != -1)
            if (push_op(seq, &len, OR_ALLGATHER, Mfrom[d], d, -1)) return -1;
    for (int d = 0; d < r; ++d)
        if (Mto[d] != -1)
            if (push_op(seq, &len, OR_SLICE, Mto[d], -1, d)) return -1;
    return len;
}

/* candidate 0 = replace (Algorithm 1), 1 = rearrange, 2 = remove, 3 = naive */
int or_sequence(const int32_t *Mfrom, const int32_t *Mto, int r, int cand, or_redop *seq) {
    switch (cand) {
    case 0: return optimized_redistribution(Mfrom, Mto, r, 1, seq);
    case 1: return optimized_redistribution(Mfrom, Mto, r, 0, seq);
    case 2: return remove_redistribution(Mfrom, Mto, r, seq);
    case 3: return naive_redistribution(Mfrom, Mto, r, seq);
    default: return -1;
    }
}

/* ---------------------------------------------------------------------------
 * Topology-aware cost of a sequence: Eq. 9 (AllGather volume), Eq. 10
 * (AllToAll volume), Eq. 11 (effective bandwidth), Eq. 13, Eq. 14; ct from
 * Algorithm 3 on the map as it is just before each operator.
 * ------------------------------------------------------------------------- */
typedef struct {
    double t;
    uint64_t vol, intra, inter;
    uint64_t x[OR_MAX_CLASSES];   /* per link class: link volume x ct (x[0]: intra, rings) */
    uint64_t x_a2a;               /* intra AllToAll volume when it has its own bandwidth */
    uint32_t n_coll, n_inter, sum_ct;
} seq_cost;

static seq_cost cost_sequence(const int64_t *D, int h, const int32_t *Mfrom, int r,
                              or_redop *seq, int len, uint64_t shard0_nb, int64_t N,
                              const or_topology *topo) {
    seq_cost c;
    memset(&c, 0, sizeof c);
    int32_t M[OR_MAX_SUB];
    memcpy(M, Mfrom, sizeof(int32_t) * (size_t)r);
    uint64_t shard = shard0_nb;   /* data_size of one device, in nb */
    for (int q = 0; q < len; ++q) {
        or_redop *op = &seq[q];
        int64_t p = D[op->axis];
        op->shard_nb = shard;
        if (op->kind == OR_SLICE) {
            M[op->to_dim] = op->axis;
            shard /= (uint64_t)p;
            continue;
        }
        /* reading R-j: the smallest domain that holds the group, ct (and the
         * members per block, k) of the next smaller one */
        int64_t k_in = 0;
        int cls = 0;
        while (cls < topo->n_classes - 1 &&
               or_gather_ct(D, h, M, r, op->axis, topo->domain[cls], &k_in) != 0)
            ++cls;
        int64_t ct = 0;
        if (cls)
            ct = or_gather_ct(D, h, M, r, op->axis, topo->domain[cls - 1], &k_in);
        else
            or_gather_ct(D, h, M, r, op->axis, topo->domain[0], &k_in);
        const double Bintra = (double)topo->bw[0], Bcls = (double)topo->bw[cls];
        op->ct = (int32_t)ct;
        op->k_in = (int32_t)k_in;
        uint64_t V, link;
        double cost;
        if (op->kind == OR_ALLGATHER) {
            V = (uint64_t)(p - 1) * shard;                  /* Eq. 9 */
            link = V;
            cost = ct == 0 ? ((double)V / (double)N) / Bintra
                           : ((double)V / (double)N) / (Bcls / (double)ct);
            M[op->from_dim] = -1;
            shard *= (uint64_t)p;
        } else {
            V = (uint64_t)(p - 1) * shard / (uint64_t)p;     /* Eq. 10 */
            if (ct == 0) {
                link = V;
                cost = ((double)V / (double)N) / (topo->bw_a2a ? (double)topo->bw_a2a : Bintra);
            } else {                                          /* Eq. 14, p > k */
                link = (uint64_t)k_in * (uint64_t)(p - k_in) * shard / (uint64_t)p;
                double factor = (double)(k_in * (p - k_in)) / (double)(p - 1);
                cost = factor * ((double)V / (double)N) / (Bcls / (double)ct);
            }
            M[op->from_dim] = -1;
            M[op->to_dim] = op->axis;
        }
        op->volume_nb = V;
        op->link_nb = link;
        op->cost = cost;
        c.vol += V;
        c.t += cost;
        c.n_coll += 1;
        if (ct == 0) {
            c.intra += link;
            if (op->kind == OR_ALLTOALL && topo->bw_a2a)
                c.x_a2a += link;
            else
                c.x[0] += link;
        } else {
            c.inter += link * (uint64_t)ct;
            c.x[cls] += link * (uint64_t)ct;
            c.n_inter += 1;
            c.sum_ct += (uint32_t)ct;
        }
    }
    return c;
}

/* ---------------------------------------------------------------------------
 * One auxiliary edge (Algorithm 4): the tensor src.out feeds dst.in[slot];
 * strategy si of the producer, sj of the consumer.  Forward: the tensor
 * moves from the producer's map to the consumer's.  Reverse (the gradient of
 * the same tensor in the backward pass): from the consumer's map back to the
 * producer's; same shape and element size.
 * ------------------------------------------------------------------------- */
static int edge_problem_dir(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                            const or_strategy *sj, int64_t N, int reverse, or_unified *u,
                            uint64_t *shard0_nb) {
    const or_tensor *T = &src->out, *Tc = &dst->in[slot];
    int64_t Dp[OR_MAX_DEV], Dc[OR_MAX_DEV], shape[OR_MAX_RANK];
    int32_t Mp[OR_MAX_RANK], Mc[OR_MAX_RANK];
    int hp = device_matrix(src, si, Dp), hc = device_matrix(dst, sj, Dc);
    tensor_map(T, si, Mp);
    tensor_map(Tc, sj, Mc);
    uint64_t elems = 1;
    for (int d = 0; d < T->rank; ++d) {
        shape[d] = src->axis_len[T->axis[d]];
        elems *= (uint64_t)shape[d];
    }
    if (reverse ? or_unify(N, Dc, hc, Mc, Dp, hp, Mp, T->rank, shape, u)
                : or_unify(N, Dp, hp, Mp, Dc, hc, Mc, T->rank, shape, u))
        return -1;
    uint64_t used = 1;
    for (int d = 0; d < u->r; ++d)
        if (u->m_from[d] >= 0) used *= (uint64_t)u->D[u->m_from[d]];
    *shard0_nb = elems * (uint64_t)src->dtype_bytes * (uint64_t)N / used;
    return 0;
}

static int edge_problem(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                        const or_strategy *sj, int64_t N, or_unified *u, uint64_t *shard0_nb) {
    return edge_problem_dir(src, si, dst, slot, sj, N, 0, u, shard0_nb);
}

/* Exposes one candidate's unified problem and operator sequence with the
 * per-operator costs filled in.  Returns the sequence length, -1 on error. */
int or_edge_detail(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                   const or_strategy *sj, int64_t N, int64_t L, uint64_t Bintra, uint64_t Binter,
                   int cand, or_unified *u, or_redop *seq, uint64_t *shard0_nb) {
    if (edge_problem(src, si, dst, slot, sj, N, u, shard0_nb)) return -1;
    int len = or_sequence(u->m_from, u->m_to, u->r, cand, seq);
    if (len < 0) return -1;
    const or_topology topo = two_class(N, L, Bintra, Binter);
    cost_sequence(u->D, u->h, u->m_from, u->r, seq, len, *shard0_nb, N, &topo);
    return len;
}

/* Costs one candidate on an already unified problem (used for Table 2). */
int or_sequence_cost(const int64_t *D, int h, const int32_t *Mfrom, const int32_t *Mto, int r,
                     int cand, uint64_t shard0_nb, int64_t N, int64_t L, uint64_t Bintra,
                     uint64_t Binter, or_redop *seq, or_record *rec) {
    int len = or_sequence(Mfrom, Mto, r, cand, seq);
    if (len < 0) return -1;
    const or_topology topo = two_class(N, L, Bintra, Binter);
    seq_cost c = cost_sequence(D, h, Mfrom, r, seq, len, shard0_nb, N, &topo);
    rec->t = c.t;
    rec->vol = c.vol;
    rec->intra = c.intra;
    rec->inter = c.inter;
    rec->meta = (uint32_t)cand | (c.n_coll << 2) | (c.n_inter << 7) | (c.sum_ct << 12);
    return len;
}

static uint64_t gcd_u64(uint64_t a, uint64_t b) {
    while (b) {
        uint64_t t = a % b;
        a = b;
        b = t;
    }
    return a;
}

/* Exact order of sum_c x[c] / bw[c] (+ x_a2a / bw_a2a; reading R-j) as
 * integer keys: with two classes x[0] bw[1] + x[1] bw[0] (reading R-h's
 * intra/(N B_intra) + inter/(N B_inter)); otherwise sum_c x[c] w[c] with
 * w[c] = lcm(bw) / bw[c], which must stay below 2^32 (returns -1 otherwise). */
static int class_weights(const or_topology *topo, uint64_t *w, uint64_t *w_a2a) {
    *w_a2a = 0;
    if (topo->n_classes == 2 && !topo->bw_a2a) {
        w[0] = topo->bw[1];
        w[1] = topo->bw[0];
        return 0;
    }
    unsigned __int128 lcm = 1;
    for (int c = 0; c <= topo->n_classes; ++c) {
        const uint64_t b = c < topo->n_classes ? topo->bw[c] : topo->bw_a2a;
        if (c == topo->n_classes && !b) break;
        if (b == 0) return -1;
        const uint64_t g = gcd_u64((uint64_t)(lcm % b), b);
        const unsigned __int128 q = lcm / g;
        if (q >> 64) return -1;
        lcm = q * b;
    }
    for (int c = 0; c <= topo->n_classes; ++c) {
        const uint64_t b = c < topo->n_classes ? topo->bw[c] : topo->bw_a2a;
        if (!b) break;
        unsigned __int128 q = lcm / b;
        if (q >> 32) return -1;
        if (c < topo->n_classes)
            w[c] = (uint64_t)q;
        else
            *w_a2a = (uint64_t)q;
    }
    return 0;
}

static unsigned __int128 class_key(const seq_cost *sc, const or_topology *topo, const uint64_t *w,
                                   uint64_t w_a2a) {
    unsigned __int128 key = (unsigned __int128)sc->x_a2a * w_a2a;
    for (int c = 0; c < topo->n_classes; ++c) key += (unsigned __int128)sc->x[c] * w[c];
    return key;
}

/* Reading R-h: the cheapest of the four candidates by exact comparison of
 * intra/(N B_intra) + inter/(N B_inter) (per link class under R-j), ties to
 * the lower candidate index. */
static int edge_cost_dir(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                         const or_strategy *sj, int64_t N, const or_topology *topo, int reverse,
                         or_record *rec) {
    or_unified u;
    uint64_t shard0;
    uint64_t w[OR_MAX_CLASSES], w_a2a;
    memset(rec, 0, sizeof *rec);
    if (class_weights(topo, w, &w_a2a)) return -1;
    if (edge_problem_dir(src, si, dst, slot, sj, N, reverse, &u, &shard0)) return -1;
    or_redop seq[OR_MAX_SEQ];
    seq_cost best;
    memset(&best, 0, sizeof best);
    int best_c = -1;
    unsigned __int128 best_key = 0;
    uint64_t min_vol = 0;
    for (int c = 0; c < 4; ++c) {
        int len = or_sequence(u.m_from, u.m_to, u.r, c, seq);
        if (len < 0) return -1;
        seq_cost sc = cost_sequence(u.D, u.h, u.m_from, u.r, seq, len, shard0, N, topo);
        unsigned __int128 key = class_key(&sc, topo, w, w_a2a);
        if (best_c < 0 || key < best_key) {
            best_c = c;
            best_key = key;
            best = sc;
        }
        if (c == 0 || sc.vol < min_vol) min_vol = sc.vol;
    }
    rec->t = best.t;
    rec->vol = min_vol;
    rec->intra = best.intra;
    rec->inter = best.inter;
    rec->meta = (uint32_t)best_c | (best.n_coll << 2) | (best.n_inter << 7) | (best.sum_ct << 12);
    return 0;
}

int or_edge_cost_topo(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                      const or_strategy *sj, int64_t N, const or_topology *topo, or_record *rec) {
    return edge_cost_dir(src, si, dst, slot, sj, N, topo, 0, rec);
}

int or_edge_cost(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                 const or_strategy *sj, int64_t N, int64_t L, uint64_t Bintra, uint64_t Binter,
                 or_record *rec) {
    const or_topology topo = two_class(N, L, Bintra, Binter);
    return edge_cost_dir(src, si, dst, slot, sj, N, &topo, 0, rec);
}

/* The backward direction of the same pair: the gradient moves from the
 * consumer's map (strategy sj) back to the producer's (strategy si). */
int or_edge_cost_reverse(const or_op *src, const or_strategy *si, const or_op *dst, int slot,
                         const or_strategy *sj, int64_t N, int64_t L, uint64_t Bintra,
                         uint64_t Binter, or_record *rec) {
    const or_topology topo = two_class(N, L, Bintra, Binter);
    return edge_cost_dir(src, si, dst, slot, sj, N, &topo, 1, rec);
}

/* Row-major table of one edge under a topology: out[i * nd + j]. */
int64_t or_edge_table_topo(const or_op *src, const or_strategy *ss, int64_t ns, const or_op *dst,
                           int slot, const or_strategy *sd, int64_t nd, int64_t N,
                           const or_topology *topo, or_record *out) {
    for (int64_t i = 0; i < ns; ++i)
        for (int64_t j = 0; j < nd; ++j)
            if (edge_cost_dir(src, &ss[i], dst, slot, &sd[j], N, topo, 0, &out[i * nd + j]))
                return -1;
    return ns * nd;
}

/* Selected entries (i[k], j[k]) of one edge table under a topology. */
int64_t or_edge_entries_topo(const or_op *src, const or_strategy *ss, const or_op *dst, int slot,
                             const or_strategy *sd, const int64_t *ii, const int64_t *jj,
                             int64_t n, int64_t N, const or_topology *topo, or_record *out) {
    for (int64_t k = 0; k < n; ++k)
        if (edge_cost_dir(src, &ss[ii[k]], dst, slot, &sd[jj[k]], N, topo, 0, &out[k])) return -1;
    return n;
}

/* Backward table of one edge, consumer-major: out[j * ns + i]. */
int64_t or_edge_table_reverse(const or_op *src, const or_strategy *ss, int64_t ns,
                              const or_op *dst, int slot, const or_strategy *sd, int64_t nd,
                              int64_t N, int64_t L, uint64_t Bintra, uint64_t Binter,
                              or_record *out) {
    for (int64_t j = 0; j < nd; ++j)
        for (int64_t i = 0; i < ns; ++i)
            if (or_edge_cost_reverse(src, &ss[i], dst, slot, &sd[j], N, L, Bintra, Binter,
                                     &out[j * ns + i]))
                return -1;
    return ns * nd;
}

/* Row-major table of one edge: out[i * nd + j]. */
int64_t or_edge_table(const or_op *src, const or_strategy *ss, int64_t ns, const or_op *dst,
                      int slot, const or_strategy *sd, int64_t nd, int64_t N, int64_t L,
                      uint64_t Bintra, uint64_t Binter, or_record *out) {
    for (int64_t i = 0; i < ns; ++i)
        for (int64_t j = 0; j < nd; ++j)
            if (or_edge_cost(src, &ss[i], dst, slot, &sd[j], N, L, Bintra, Binter,
                             &out[i * nd + j]))
                return -1;
    return ns * nd;
}

/* Selected entries (i[k], j[k]) of one edge table. */
int64_t or_edge_entries(const or_op *src, const or_strategy *ss, const or_op *dst, int slot,
                        const or_strategy *sd, const int64_t *ii, const int64_t *jj, int64_t n,
                        int64_t N, int64_t L, uint64_t Bintra, uint64_t Binter, or_record *out) {
    for (int64_t k = 0; k < n; ++k)
        if (or_edge_cost(src, &ss[ii[k]], dst, slot, &sd[jj[k]], N, L, Bintra, Binter, &out[k]))
            return -1;
    return n;
}

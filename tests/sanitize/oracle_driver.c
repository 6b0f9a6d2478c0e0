/* Runs every entry point of the CPU oracle on seeded random operators and
 * meshes, for a build under AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_sanitizers_cpu.py).  Test infrastructure: it includes the
 * oracle's source and exits non-zero on any unexpected return code. */
#include "../../oracle/taps_oracle.c"

#include <stdio.h>
#include <stdlib.h>

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(uint32_t n) {   /* splitmix64, then a value in [0, n) */
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return (uint32_t)((z ^ (z >> 31)) % n);
}

static void random_tensor(or_tensor *t, int n_axes, int rank) {
    int used[OR_MAX_AXES] = {0};
    t->rank = 0;
    for (int d = 0; d < rank; ++d) {
        int a = (int)rnd((uint32_t)n_axes);
        if (used[a]) continue;
        used[a] = 1;
        t->axis[t->rank++] = a;
    }
}

/* dst's input 0 has the shape of src's output */
static void random_pair(or_op *src, or_op *dst) {
    memset(src, 0, sizeof *src);
    memset(dst, 0, sizeof *dst);
    src->n_axes = 1 + (int)rnd(5);
    for (int a = 0; a < src->n_axes; ++a) src->axis_len[a] = (int64_t)1 << (1 + rnd(8));
    src->part_mask = (int)rnd(1u << src->n_axes) | 1;
    src->dtype_bytes = rnd(2) ? 2 : 4;
    random_tensor(&src->out, src->n_axes, 1 + (int)rnd((uint32_t)src->n_axes));
    src->n_in = 1;
    random_tensor(&src->in[0], src->n_axes, 1 + (int)rnd((uint32_t)src->n_axes));
    src->n_w = (int)rnd(2);
    if (src->n_w) random_tensor(&src->w[0], src->n_axes, 1 + (int)rnd((uint32_t)src->n_axes));
    const int r = src->out.rank;
    dst->n_axes = r + (int)rnd((uint32_t)(OR_MAX_AXES - r < 3 ? OR_MAX_AXES - r + 1 : 3));
    for (int d = 0; d < r; ++d) dst->axis_len[d] = src->axis_len[src->out.axis[d]];
    for (int a = r; a < dst->n_axes; ++a) dst->axis_len[a] = (int64_t)1 << (1 + rnd(8));
    dst->part_mask = (int)rnd(1u << dst->n_axes) | 1;
    dst->dtype_bytes = src->dtype_bytes;
    dst->n_in = 1;
    dst->in[0].rank = r;
    for (int d = 0; d < r; ++d) dst->in[0].axis[d] = d;
    random_tensor(&dst->out, dst->n_axes, 1 + (int)rnd((uint32_t)dst->n_axes));
    dst->n_w = (int)rnd(2);
    if (dst->n_w) random_tensor(&dst->w[0], dst->n_axes, 1 + (int)rnd((uint32_t)dst->n_axes));
}

#define CAP 4096
static or_strategy ss[CAP], sd[CAP];
static or_record rec[CAP], tab[CAP * 8];

int main(void) {
    long checked = 0;
    for (int iter = 0; iter < 300; ++iter) {
        or_op src, dst;
        random_pair(&src, &dst);
        const int n = (int)rnd(7);
        const int64_t N = (int64_t)1 << n, L = (int64_t)1 << rnd((uint32_t)n + 1);
        const uint64_t bi = 1000000000ull * (1 + rnd(600)), be = 1000000000ull * (1 + rnd(100));
        const int64_t ns = or_enumerate(&src, N, 1, ss, CAP), nd = or_enumerate(&dst, N, 1, sd, CAP);
        if (ns < 0 || nd < 0) { fprintf(stderr, "enumerate failed\n"); return 1; }
        if (ns > CAP || nd > CAP) continue;
        if (or_node_table(&src, ss, ns, N, L, bi, be, rec) != ns) return 2;
        int64_t ms = ns < 8 ? ns : 8, md = nd < 64 ? nd : 64;
        if (ms && md && (or_edge_table(&src, ss, ms, &dst, 0, sd, md, N, L, bi, be, tab) != ms * md ||
                         or_edge_table_reverse(&src, ss, ms, &dst, 0, sd, md, N, L, bi, be, tab) !=
                             ms * md)) {
            fprintf(stderr, "edge table failed\n");
            return 3;
        }
        for (int k = 0; k < 4 && ns && nd; ++k) {
            const or_strategy *a = &ss[rnd((uint32_t)ns)], *b = &sd[rnd((uint32_t)nd)];
            for (int cand = 0; cand < 4; ++cand) {
                or_unified u;
                or_redop seq[OR_MAX_SEQ];
                uint64_t shard0 = 0;
                const int len = or_edge_detail(&src, a, &dst, 0, b, N, L, bi, be, cand, &u, seq, &shard0);
                if (len < 0) { fprintf(stderr, "edge detail failed\n"); return 4; }
                or_record r1;
                if (or_sequence_cost(u.D, u.h, u.m_from, u.m_to, u.r, cand, shard0, N, L, bi, be, seq,
                                     &r1) < 0)
                    return 5;
            }
            or_record r2;
            if (or_edge_cost(&src, a, &dst, 0, b, N, L, bi, be, &r2) ||
                or_edge_cost_reverse(&src, a, &dst, 0, b, N, L, bi, be, &r2))
                return 6;
            checked += 1;
        }
        /* fixed meshes and link classes */
        if (n > 0) {
            int64_t mesh[OR_MAX_DEV];
            int k = 0, rest = n;
            while (rest > 0) {
                const int e = 1 + (int)rnd((uint32_t)(rest < 3 ? rest : 3));
                mesh[k++] = (int64_t)1 << e;
                rest -= e;
            }
            if (or_enumerate_mesh(&src, mesh, k, (int)rnd(2), ss, CAP) < 0) return 8;
        }
        if (ms && md) {
            or_topology topo;
            memset(&topo, 0, sizeof topo);
            topo.n_classes = 1 + (int)rnd(OR_MAX_CLASSES);
            int64_t size = 1;
            for (int c = 0; c < topo.n_classes; ++c) {
                if (c == topo.n_classes - 1) size = N;
                else while (size < N && rnd(2)) size *= 2;
                topo.domain[c] = size;
                topo.bw[c] = 1000000000ull * (1 + rnd(4)) * 25;
            }
            topo.bw_a2a = rnd(2) ? 0 : 150000000000ull;
            if (or_edge_table_topo(&src, ss, ms, &dst, 0, sd, md, N, &topo, tab) != ms * md ||
                or_node_table_topo(&src, ss, ms, N, &topo, rec) != ms) {
                fprintf(stderr, "topology tables failed\n");
                return 9;
            }
        }
        /* collective group counts on a random device matrix and map */
        int64_t D[OR_MAX_DEV];
        int h = 0, left = n;
        while (left > 0 && h < OR_MAX_DEV) {
            const int e = 1 + (int)rnd((uint32_t)left);
            D[h++] = (int64_t)1 << e;
            left -= e;
        }
        if (h) {
            int32_t M[4] = {-1, -1, -1, -1};
            for (int d = 0; d < 4; ++d) M[d] = rnd(2) ? (int32_t)rnd((uint32_t)h) : -1;
            for (int d = 1; d < 4; ++d)
                for (int e = 0; e < d; ++e)
                    if (M[d] == M[e]) M[d] = -1;
            (void)or_allreduce_ct(D, h, M, 4, L);
            for (int g = 0; g < h; ++g) {
                int64_t k_in = 0;
                (void)or_gather_ct(D, h, M, 4, g, L, &k_in);
            }
        }
    }
    printf("oracle driver: %ld entries checked\n", checked);
    return checked > 100 ? 0 : 7;
}

// Drives the C ABI's host paths -- argument validation, size queries,
// capacity and error reporting -- for a build of the library whose host code
// runs under AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_sanitizers_cpu.py).  Runs without a GPU: calls that reach the
// device must return TAPS_ERR_DEVICE.  Exits non-zero on the first surprise.
#include <cstdio>
#include <cstring>
#include <vector>

#include "taps.h"

namespace {

int failures = 0;

void expect(taps_status got, taps_status want, const char *what) {
    if (got != want) {
        std::fprintf(stderr, "%s: got %s, want %s (%s)\n", what, taps_status_str(got),
                     taps_status_str(want), taps_last_error());
        ++failures;
    }
}

taps_tensor tensor(std::initializer_list<int> axes) {
    taps_tensor t;
    std::memset(&t, 0, sizeof t);
    for (int a : axes) t.axis[t.rank++] = (uint8_t)a;
    return t;
}

// mm(b, k, o): X(b, k) x W(k, o) -> Y(b, o)
taps_op matmul(int64_t b, int64_t k, int64_t o) {
    taps_op op;
    std::memset(&op, 0, sizeof op);
    op.n_axes = 3;
    op.part_mask = 7;
    op.dtype_bytes = 4;
    op.axis_len[0] = b;
    op.axis_len[1] = k;
    op.axis_len[2] = o;
    op.n_in = 1;
    op.in[0] = tensor({0, 1});
    op.n_w = 1;
    op.w[0] = tensor({1, 2});
    op.out = tensor({0, 2});
    return op;
}

}  // namespace

int main() {
    for (int s = 0; s <= (int)TAPS_ERR_DEVICE + 1; ++s)
        if (!taps_status_str((taps_status)s)) ++failures;
    std::vector<taps_op> ops = {matmul(64, 256, 1024), matmul(64, 1024, 256), matmul(64, 256, 512)};
    std::vector<taps_edge> edges = {{0, 1, 0}, {1, 2, 0}};
    taps_graph g = {(uint32_t)ops.size(), (uint32_t)edges.size(), ops.data(), edges.data()};
    taps_cluster cl = {2, 2, 200000000000ull, 25000000000ull};
    std::vector<uint64_t> offs = {0, 9, 18, 27};
    std::vector<uint64_t> eo(edges.size() + 1, 0);
    const taps_table none = {nullptr, nullptr, nullptr, nullptr, nullptr};

    // size queries and their results
    expect(taps_edge_costs(&g, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr), TAPS_OK,
           "size query");
    if (eo[1] != 81 || eo[2] != 162) ++failures;
    expect(taps_edge_costs_shared(&g, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_OK, "shared size query");
    expect(taps_edge_costs_backward(&g, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_OK, "backward size query");
    taps_cluster pts[3] = {cl, cl, cl};
    pts[1].bw_inter = 12500000000ull;
    pts[2].bw_intra = (1ull << 40) + 1;
    expect(taps_edge_costs_sweep(&g, pts, 3, nullptr, offs.data(), eo.data(), nullptr, 0, nullptr),
           TAPS_OK, "sweep size query");

    // validation: nothing is written on error
    std::vector<uint64_t> sentinel(eo.size(), 77);
    taps_table fake = {(double *)256, (uint64_t *)256, (uint64_t *)256, (uint64_t *)256,
                       (uint32_t *)256};
    expect(taps_edge_costs(&g, &cl, (const taps_strategy *)256, offs.data(), sentinel.data(), fake,
                           161, nullptr),
           TAPS_ERR_CAPACITY, "capacity");
    taps_table partial = fake;
    partial.inter = nullptr;
    expect(taps_edge_costs(&g, &cl, (const taps_strategy *)256, offs.data(), sentinel.data(),
                           partial, 162, nullptr),
           TAPS_ERR_ARG, "partial table");
    for (uint64_t v : sentinel)
        if (v != 77) ++failures;
    taps_cluster bad = cl;
    bad.nodes = 3;
    expect(taps_edge_costs(&g, &bad, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_TOPOLOGY, "non power of two");
    bad = cl;
    bad.bw_inter = 0;
    expect(taps_enumerate_strategies(&g, &bad, offs.data(), nullptr, 0, nullptr),
           TAPS_ERR_TOPOLOGY, "zero bandwidth");
    bad = cl;
    bad.nodes = 1u << 9;
    expect(taps_node_costs(&g, &bad, nullptr, offs.data(), fake, nullptr), TAPS_ERR_TOPOLOGY,
           "too many devices");
    std::vector<taps_edge> wrong = {{0, 2, 0}};   // (64, 1024) into (64, 256)
    taps_graph gw = {(uint32_t)ops.size(), 1, ops.data(), wrong.data()};
    expect(taps_edge_costs(&gw, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_SHAPE, "shape mismatch");
    wrong[0].dst_slot = 3;
    expect(taps_edge_costs(&gw, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_ARG, "slot out of range");
    wrong[0] = {0, 7, 0};
    expect(taps_edge_costs(&gw, &cl, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_ARG, "operator out of range");
    std::vector<uint64_t> flat = {0, 9, 9, 18};
    expect(taps_edge_costs(&g, &cl, nullptr, flat.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_ARG, "offsets not increasing");
    taps_op broken = ops[0];
    broken.out.axis[0] = 9;
    std::vector<taps_op> ops2 = {broken, ops[1], ops[2]};
    taps_graph gb = {3, 0, ops2.data(), nullptr};
    expect(taps_enumerate_strategies(&gb, &cl, offs.data(), nullptr, 0, nullptr), TAPS_ERR_ARG,
           "axis out of range");
    expect(taps_enumerate_strategies(nullptr, &cl, offs.data(), nullptr, 0, nullptr),
           TAPS_ERR_ARG, "null graph");
    expect(taps_node_costs(&g, &cl, nullptr, offs.data(), fake, nullptr), TAPS_ERR_ARG,
           "null strategies");
    expect(taps_memory_costs(&g, (const taps_strategy *)256, offs.data(), nullptr, nullptr),
           TAPS_ERR_ARG, "null memory");
    expect(taps_edge_costs_sweep(&g, pts, 0, nullptr, offs.data(), eo.data(), nullptr, 0, nullptr),
           TAPS_ERR_ARG, "no bandwidth points");
    taps_cluster mixed[2] = {cl, cl};
    mixed[1].nodes = 4;
    mixed[1].devices_per_node = 1;
    expect(taps_edge_costs_sweep(&g, mixed, 2, nullptr, offs.data(), eo.data(), nullptr, 0,
                                 nullptr),
           TAPS_ERR_ARG, "mixed meshes");
    expect(taps_set_edge_kernel_events((void *)256, nullptr), TAPS_ERR_ARG, "one event");
    expect(taps_set_edge_kernel_events(nullptr, nullptr), TAPS_OK, "no events");

    // the single-call build sizes everything on the host: a size query needs no GPU
    std::vector<uint64_t> bo(ops.size() + 1, 0), beo(edges.size() + 1, 0);
    expect(taps_build_tables(&g, &cl, nullptr, bo.data(), nullptr, 0, none, beo.data(), none, 0, 0,
                             nullptr),
           TAPS_OK, "build size query");
    if (bo != offs || beo[1] != 81 || beo[2] != 162) ++failures;
    expect(taps_build_tables(&g, &cl, nullptr, bo.data(), nullptr, 0, none, beo.data(), none, 0,
                             TAPS_BUILD_SHARED, nullptr),
           TAPS_OK, "shared build size query");
    expect(taps_build_tables(&g, &cl, nullptr, bo.data(), nullptr, 0, none, beo.data(), none, 0, 6,
                             nullptr),
           TAPS_ERR_ARG, "unknown build flags");
    taps_mesh mesh = {2, {2, 2}};
    expect(taps_build_tables(&g, &cl, &mesh, bo.data(), nullptr, 0, none, beo.data(), none, 0, 0,
                             nullptr),
           TAPS_OK, "build size query on a mesh");
    if (bo != offs) ++failures;
    mesh = {1, {4}};   // one axis split 4 ways: 3 strategies per matmul
    expect(taps_build_tables(&g, &cl, &mesh, bo.data(), nullptr, 0, none, beo.data(), none, 0, 0,
                             nullptr),
           TAPS_OK, "build size query on a 1-D mesh");
    if (bo[1] != 3 || bo[3] != 9 || beo[2] != 18) ++failures;
    for (taps_mesh badm : {taps_mesh{2, {4, 2}}, taps_mesh{1, {3}}, taps_mesh{9, {2}}})
        expect(taps_build_tables(&g, &cl, &badm, bo.data(), nullptr, 0, none, beo.data(), none, 0, 0,
                             nullptr),
               TAPS_ERR_TOPOLOGY, "bad mesh");
    std::vector<uint64_t> bsent(bo.size(), 77);
    expect(taps_build_tables(&g, &cl, nullptr, bsent.data(), (taps_strategy *)256, 26, fake,
                             beo.data(), fake, 1000, 0, nullptr),
           TAPS_ERR_CAPACITY, "build strategy capacity");
    expect(taps_build_tables(&g, &cl, nullptr, bsent.data(), (taps_strategy *)256, 27, fake,
                             beo.data(), fake, 161, 0, nullptr),
           TAPS_ERR_CAPACITY, "build edge capacity");
    expect(taps_build_tables(&g, &cl, nullptr, bsent.data(), (taps_strategy *)256, 27, partial,
                             beo.data(), fake, 162, 0, nullptr),
           TAPS_ERR_ARG, "build partial table");
    for (uint64_t v : bsent)
        if (v != 77) ++failures;
    std::vector<taps_op> tiny = {matmul(1, 1, 1)};   // nothing divides: no strategy on 4 devices
    taps_graph gt = {1, 0, tiny.data(), nullptr};
    expect(taps_build_tables(&gt, &cl, nullptr, bo.data(), nullptr, 0, none, beo.data(), none, 0, 0,
                             nullptr),
           TAPS_ERR_NO_STRATEGY, "build without a strategy");
    // link classes: validation before any GPU work
    taps_topology topo = {3, {2, 2, 4}, {400000000000ull, 100000000000ull, 25000000000ull}, 0};
    expect(taps_edge_costs_topology(&g, &topo, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_OK, "topology size query");
    topo.domain[1] = 1;
    expect(taps_edge_costs_topology(&g, &topo, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_TOPOLOGY, "decreasing domains");
    topo = {2, {2, 4}, {400000000000ull, 100000000000ull}, 7};
    expect(taps_edge_costs_topology(&g, &topo, nullptr, offs.data(), eo.data(), none, 0, nullptr),
           TAPS_ERR_TOPOLOGY, "AllToAll bandwidth in no round ratio");
    expect(taps_node_costs_topology(&g, nullptr, nullptr, offs.data(), fake, nullptr), TAPS_ERR_ARG,
           "null topology");

    // the device is reached: without a GPU every such call reports it
    expect(taps_enumerate_strategies(&g, &cl, offs.data(), nullptr, 0, nullptr), TAPS_OK,
           "enumeration size query (host only)");
    expect(taps_enumerate_strategies(&g, &cl, offs.data(), (taps_strategy *)256, 27, nullptr),
           TAPS_ERR_DEVICE, "enumerate without a device");
    expect(taps_build_tables(&g, &cl, nullptr, bo.data(), (taps_strategy *)256, 27, fake,
                             beo.data(), fake, 162, 0, nullptr),
           TAPS_ERR_DEVICE, "build without a device");
    std::printf("abi driver: %d failures\n", failures);
    return failures ? 1 : 0;
}

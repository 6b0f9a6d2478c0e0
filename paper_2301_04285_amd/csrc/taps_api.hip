// taps_api.hip -- the C ABI: validation, uploads, scratch and launches.
//
// Host code only sizes and checks: it validates the graph and cluster,
// computes table offsets (prefix sums of strategy counts), uploads the
// caller's structs unchanged and launches the kernels.  Every cost is
// computed on the GPU.
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <list>
#include <memory>
#include <map>
#include <mutex>
#include <numeric>
#include <string>
#include <unordered_map>
#include <vector>

#include "taps.h"
#include "taps_internal.h"

// The fixed workspace of taps_build_tables_noalloc: a file-scope device array
// of TAPS_NOALLOC_SCRATCH_BYTES, one copy on every GPU the library runs on.
// In host code its name is only a stand-in for the symbol; the device address
// comes from hipGetSymbolAddress, taken once per device with that device
// current, and only that address is used.  Nothing in it has to start at
// zero: every kernel of a build writes what it later reads.
static __device__ __align__(256) char scratch[TAPS_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;
// events to record around the next edge-table kernel (taps_set_edge_kernel_events)
thread_local hipEvent_t g_kernel_before = nullptr, g_kernel_after = nullptr;

taps_status fail(taps_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

taps_status hip_fail(hipError_t err, const char *what) {
    return fail(TAPS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(err));
}

bool pow2(uint64_t v) { return v && !(v & (v - 1)); }

uint32_t log2u(uint64_t v) {
    uint32_t k = 0;
    while ((1ull << k) < v) ++k;
    return k;
}

taps_status check_cluster(const taps_cluster *c, taps_launch *lp) {
    if (!c) return fail(TAPS_ERR_ARG, "cluster is NULL");
    if (!pow2(c->nodes) || !pow2(c->devices_per_node))
        return fail(TAPS_ERR_TOPOLOGY, "nodes (%u) and devices_per_node (%u) must be powers of two",
                    c->nodes, c->devices_per_node);
    const uint64_t N = (uint64_t)c->nodes * c->devices_per_node;
    if (N > (1ull << TAPS_MAX_LEVELS))
        return fail(TAPS_ERR_TOPOLOGY, "%llu devices exceed the limit of %u", (unsigned long long)N,
                    1u << TAPS_MAX_LEVELS);
    if (c->bw_intra == 0 || c->bw_inter == 0)
        return fail(TAPS_ERR_TOPOLOGY, "bandwidths must be positive");
    const uint64_t g = std::gcd(c->bw_intra, c->bw_inter);
    lp->n = log2u(N);
    lp->lam = log2u(c->devices_per_node);
    lp->b_inter_red = c->bw_inter / g;
    lp->b_intra_red = c->bw_intra / g;
    lp->inv_n_bintra = 1.0 / ((double)N * (double)c->bw_intra);
    lp->inv_n_binter = 1.0 / ((double)N * (double)c->bw_inter);
    lp->narrow = (lp->b_inter_red >> 32) == 0 && (lp->b_intra_red >> 32) == 0;
    return TAPS_OK;
}

taps_status check_tensor(const taps_op &op, const taps_tensor &t, uint32_t k, const char *what,
                         uint32_t idx) {
    if (t.rank > TAPS_MAX_RANK)
        return fail(TAPS_ERR_ARG, "op %u: %s %u has rank %u > %u", k, what, idx, t.rank,
                    TAPS_MAX_RANK);
    uint32_t seen = 0;
    uint64_t bytes = op.dtype_bytes;   // stays <= 2^40 or the check below fails first
    for (uint32_t d = 0; d < t.rank; ++d) {
        if (t.axis[d] >= op.n_axes)
            return fail(TAPS_ERR_ARG, "op %u: %s %u names axis %u of %u", k, what, idx, t.axis[d],
                        op.n_axes);
        if (seen & (1u << t.axis[d]))
            return fail(TAPS_ERR_ARG, "op %u: %s %u names axis %u twice", k, what, idx, t.axis[d]);
        seen |= 1u << t.axis[d];
        if (__builtin_mul_overflow(bytes, (uint64_t)op.axis_len[t.axis[d]], &bytes) ||
            bytes > TAPS_MAX_TENSOR_BYTES)
            return fail(TAPS_ERR_ARG, "op %u: %s %u exceeds %llu bytes", k, what, idx,
                        (unsigned long long)TAPS_MAX_TENSOR_BYTES);
    }
    return TAPS_OK;
}

taps_status check_graph(const taps_graph *g, bool with_edges) {
    if (!g) return fail(TAPS_ERR_ARG, "graph is NULL");
    if (g->n_ops && !g->ops) return fail(TAPS_ERR_ARG, "graph has %u ops but ops is NULL", g->n_ops);
    for (uint32_t k = 0; k < g->n_ops; ++k) {
        const taps_op &op = g->ops[k];
        if (op.n_axes < 1 || op.n_axes > TAPS_MAX_AXES)
            return fail(TAPS_ERR_ARG, "op %u: n_axes %u outside 1..%u", k, op.n_axes, TAPS_MAX_AXES);
        if (op.part_mask >> op.n_axes)
            return fail(TAPS_ERR_ARG, "op %u: part_mask names axes beyond n_axes", k);
        if (op.dtype_bytes == 0) return fail(TAPS_ERR_ARG, "op %u: dtype_bytes is 0", k);
        if (op.n_in > TAPS_MAX_INPUTS || op.n_w > TAPS_MAX_WEIGHTS)
            return fail(TAPS_ERR_ARG, "op %u: too many inputs or weights", k);
        for (uint32_t a = 0; a < op.n_axes; ++a)
            if (op.axis_len[a] < 1)
                return fail(TAPS_ERR_ARG, "op %u: axis %u has length %lld", k, a,
                            (long long)op.axis_len[a]);
        taps_status st = check_tensor(op, op.out, k, "output", 0);
        for (uint32_t i = 0; st == TAPS_OK && i < op.n_in; ++i)
            st = check_tensor(op, op.in[i], k, "input", i);
        for (uint32_t i = 0; st == TAPS_OK && i < op.n_w; ++i)
            st = check_tensor(op, op.w[i], k, "weight", i);
        if (st != TAPS_OK) return st;
    }
    if (!with_edges) return TAPS_OK;
    if (g->n_edges && !g->edges)
        return fail(TAPS_ERR_ARG, "graph has %u edges but edges is NULL", g->n_edges);
    for (uint32_t e = 0; e < g->n_edges; ++e) {
        const taps_edge &E = g->edges[e];
        if (E.src_op >= g->n_ops || E.dst_op >= g->n_ops)
            return fail(TAPS_ERR_ARG, "edge %u: op index out of range", e);
        const taps_op &src = g->ops[E.src_op];
        const taps_op &dst = g->ops[E.dst_op];
        if (E.dst_slot >= dst.n_in)
            return fail(TAPS_ERR_ARG, "edge %u: consumer has no input %u", e, E.dst_slot);
        const taps_tensor &T = src.out, &Tc = dst.in[E.dst_slot];
        if (T.rank != Tc.rank)
            return fail(TAPS_ERR_SHAPE, "edge %u: rank %u -> %u", e, T.rank, Tc.rank);
        for (uint32_t d = 0; d < T.rank; ++d)
            if (src.axis_len[T.axis[d]] != dst.axis_len[Tc.axis[d]])
                return fail(TAPS_ERR_SHAPE, "edge %u: dimension %u has length %lld -> %lld", e, d,
                            (long long)src.axis_len[T.axis[d]], (long long)dst.axis_len[Tc.axis[d]]);
    }
    return TAPS_OK;
}

taps_status check_offsets(const taps_graph *g, const uint64_t *op_offsets) {
    if (!op_offsets) return fail(TAPS_ERR_ARG, "op_offsets is NULL");
    if (op_offsets[0] != 0) return fail(TAPS_ERR_ARG, "op_offsets[0] must be 0");
    for (uint32_t k = 0; k < g->n_ops; ++k)
        if (op_offsets[k + 1] <= op_offsets[k])
            return fail(TAPS_ERR_ARG, "op_offsets must increase (op %u)", k);
    if (op_offsets[g->n_ops] > 0xFFFFFFFFull)
        return fail(TAPS_ERR_ARG, "more than 2^32 strategies");
    return TAPS_OK;
}

// Pinned staging for host-to-device uploads: a small pool of fine-grained
// host buffers, each with the event recorded after the kernel that reads it
// (k_pull: no copy engine, so the build's kernels follow on the same queue
// without a hand-over).  An upload takes a buffer whose upload has completed
// (or a new one), so calls on different streams or threads, and a call queued
// behind a long-running build, do not wait for each other's uploads; only
// when every buffer of a full pool is still in flight does an upload wait,
// for the oldest.
struct staging_buffer {
    char *host = nullptr;
    void *dev = nullptr;   // the same memory as the device addresses it
    size_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
    uint64_t last_use = 0;
};
struct staging_pool {
    std::mutex mu;
    std::vector<staging_buffer> bufs;
    uint64_t clock = 0;
};
staging_pool g_stage;
constexpr size_t kStagingBuffers = 8;
constexpr size_t kStagingMin = size_t(1) << 20;

struct chunk {
    const void *src;
    size_t bytes;
    size_t offset;
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Bytes an array of `bytes` takes from a workspace (at least 256, aligned).
size_t carve_size(size_t bytes) { return align256(bytes ? bytes : 256); }

// Waits for the stream: the calls that must read a result back usually wait
// for a few tens of microseconds of queued work, where a blocking wait adds
// its own wake-up latency, so the stream is polled for up to 200 us before
// the wait blocks (a caller's long work already queued on the stream then
// does not keep a core spinning).
hipError_t wait_stream(hipStream_t stream) {
    const auto until = std::chrono::steady_clock::now() + std::chrono::microseconds(200);
    while (std::chrono::steady_clock::now() < until) {
        const hipError_t err = hipStreamQuery(stream);
        if (err != hipErrorNotReady) return err;
    }
    return hipStreamSynchronize(stream);
}

// The stream-ordered pool of the current device keeps freed scratch for the
// next call instead of handing it back to the driver: a fresh reservation of
// the tens of MB an edge call needs costs hundreds of microseconds.
constexpr uint32_t kMaxDevices = 64;

void retain_pool() {
    static std::mutex mu;
    static bool done[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= (int)kMaxDevices) return;
    std::lock_guard<std::mutex> lock(mu);
    if (done[dev]) return;
    hipMemPool_t pool;
    if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
        uint64_t threshold = UINT64_MAX;
        (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &threshold);
    }
    done[dev] = true;
}

template <class T>
T *at(void *base, const chunk &c) {
    return reinterpret_cast<T *>(static_cast<char *>(base) + c.offset);
}

// Device scratch: one block per (device, stream), kept for the next call on
// the same stream -- stream order makes the reuse safe, and a call then
// neither allocates nor frees (a stream-ordered free blocks the host until the
// stream has drained, which would keep the host from queueing the next build
// while the current one runs).  A call holds its block's lock from start to
// end, so calls on one stream from several threads queue one after the other;
// calls on different streams use different blocks.  A call carves its arrays
// from the block; what does not fit goes to allocations of its own, freed in
// stream order when it returns, and the block is grown past the call's whole
// need (to a power of two) at the start of the next call on that stream.  At
// most kMaxBlocks blocks are kept; beyond that the least recently used idle
// one is freed.
struct stream_block {
    int device = 0;
    hipStream_t stream = nullptr;
    std::mutex mu;
    char *ptr = nullptr;
    size_t cap = 0;
    size_t want = 0;       // largest need seen on this stream
    uint64_t last_use = 0;
    uint32_t users = 0;    // calls holding or waiting for mu (under g_blocks_mu)
};
std::mutex g_blocks_mu;
std::list<stream_block> g_blocks;   // stable addresses
uint64_t g_blocks_clock = 0;
constexpr size_t kMaxBlocks = 16;

stream_block *find_block(hipStream_t stream) {
    int device = 0;
    (void)hipGetDevice(&device);
    std::lock_guard<std::mutex> lock(g_blocks_mu);
    for (stream_block &b : g_blocks)
        if (b.device == device && b.stream == stream) {
            b.last_use = ++g_blocks_clock;
            ++b.users;
            return &b;
        }
    if (g_blocks.size() >= kMaxBlocks) {   // free the least recently used idle block
        // idle: no call holds its lock or is about to take it, so nothing else
        // can reach it while the list lock is held
        auto victim = g_blocks.end();
        for (auto it = g_blocks.begin(); it != g_blocks.end(); ++it) {
            if (it->users) continue;
            if (victim == g_blocks.end() || it->last_use < victim->last_use) victim = it;
        }
        if (victim != g_blocks.end()) {
            // its stream may be gone: a device-wide free, which waits for the work using it
            if (victim->ptr) {
                int cur = 0;
                (void)hipGetDevice(&cur);
                (void)hipSetDevice(victim->device);
                (void)hipFree(victim->ptr);
                (void)hipSetDevice(cur);
            }
            g_blocks.erase(victim);
        }
    }
    g_blocks.emplace_back();
    stream_block &b = g_blocks.back();
    b.device = device;
    b.stream = stream;
    b.last_use = ++g_blocks_clock;
    b.users = 1;
    return &b;
}

void release_block(stream_block *b) {
    std::lock_guard<std::mutex> lock(g_blocks_mu);
    --b->users;
}

struct call_scratch {
    hipStream_t stream;
    stream_block *blk;
    std::unique_lock<std::mutex> lock;
    size_t used = 0;                // bytes of the block this call has taken
    size_t need = 0;                // what the call asked for in all
    std::vector<void *> own;        // allocations beyond the block, freed on return
    explicit call_scratch(hipStream_t s) : stream(s), blk(find_block(s)), lock(blk->mu) {
        if (blk->want > blk->cap) {   // grow past the largest need seen (nothing uses the block yet)
            // a power of two, so that a stream whose calls vary in size regrows rarely
            size_t cap = size_t(1) << 20;
            while (cap < blk->want) cap *= 2;
            retain_pool();
            if (blk->ptr) (void)hipFreeAsync(blk->ptr, stream);
            blk->ptr = nullptr;
            blk->cap = 0;
            void *p = nullptr;
            if (hipMallocAsync(&p, cap, stream) == hipSuccess) {
                blk->ptr = (char *)p;
                blk->cap = cap;
            }
        }
    }
    ~call_scratch() {
        for (void *p : own) (void)hipFreeAsync(p, stream);
        if (need > blk->want) blk->want = need;
        lock.unlock();   // before the block may become idle (and be freed)
        release_block(blk);
    }
    taps_status alloc(void **p, size_t bytes) {
        const size_t size = align256(bytes ? bytes : 256);
        need += size;
        if (blk->ptr && used + size <= blk->cap) {
            *p = blk->ptr + used;
            used += size;
            return TAPS_OK;
        }
        retain_pool();
        hipError_t err = hipMallocAsync(p, size, stream);
        if (err != hipSuccess) return hip_fail(err, "hipMallocAsync");
        own.push_back(*p);
        return TAPS_OK;
    }
};

// Uploads the chunks into one array of the call's scratch; *dev receives its
// base.
taps_status upload(call_scratch &sc, std::vector<chunk> &chunks, void **dev) {
    const hipStream_t stream = sc.stream;
    size_t total = 0;
    for (chunk &c : chunks) {
        c.offset = total;
        total += align256(c.bytes);
    }
    if (total == 0) total = 256;
    taps_status st = sc.alloc(dev, total);
    if (st != TAPS_OK) return st;
    hipError_t err = hipSuccess;
    std::lock_guard<std::mutex> lock(g_stage.mu);
    // a buffer whose last copy is done: free, or completed in the meantime
    staging_buffer *b = nullptr;
    for (staging_buffer &x : g_stage.bufs) {
        if (x.pending && hipEventQuery(x.done) == hipSuccess) x.pending = false;
        if (!x.pending && (!b || x.cap > b->cap)) b = &x;
    }
    if (!b && g_stage.bufs.size() < kStagingBuffers) {
        g_stage.bufs.emplace_back();
        b = &g_stage.bufs.back();
    }
    if (!b) {   // every buffer in flight: wait for the least recently used one
        b = &g_stage.bufs[0];
        for (staging_buffer &x : g_stage.bufs)
            if (x.last_use < b->last_use) b = &x;
        err = hipEventSynchronize(b->done);
        if (err != hipSuccess) return hip_fail(err, "hipEventSynchronize");
        b->pending = false;
    }
    if (!b->done) {
        err = hipEventCreateWithFlags(&b->done, hipEventDisableTiming);
        if (err != hipSuccess) return hip_fail(err, "hipEventCreate");
    }
    if (b->cap < total) {
        // hipHostFree waits for the device to go idle: grow to a power of two
        // (at least kStagingMin) so that a buffer is replaced at most a few times
        size_t cap = kStagingMin;
        while (cap < total) cap *= 2;
        if (b->host) (void)hipHostFree(b->host);
        b->host = nullptr;
        b->dev = nullptr;
        b->cap = 0;
        // fine-grained: the upload kernel reads the host's latest writes
        err = hipHostMalloc((void **)&b->host, cap, hipHostMallocCoherent);
        if (err != hipSuccess) return hip_fail(err, "hipHostMalloc");
        b->cap = cap;
        err = hipHostGetDevicePointer(&b->dev, b->host, 0);
        if (err != hipSuccess) {
            (void)hipHostFree(b->host);
            b->host = nullptr;
            b->cap = 0;
            return hip_fail(err, "hipHostGetDevicePointer");
        }
    }
    for (const chunk &c : chunks)
        if (c.bytes) std::memcpy(b->host + c.offset, c.src, c.bytes);
    err = taps_launch_pull(b->dev, *dev, total, stream);
    if (err != hipSuccess) return hip_fail(err, "upload");
    err = hipEventRecord(b->done, stream);
    if (err != hipSuccess) return hip_fail(err, "hipEventRecord");
    b->pending = true;
    b->last_use = ++g_stage.clock;
    return TAPS_OK;
}

// Edges whose tables are identical: the same producer description (axes,
// lengths, partitionable axes, element size, output tensor), the same
// consumer description (axes, lengths, partitionable axes, the input tensor
// the edge feeds) -- and, checked on the device, the same strategies.
struct edge_sig {
    int64_t v[7 + 2 * TAPS_MAX_AXES + 2 * TAPS_MAX_RANK];   // zero-padded
    bool operator==(const edge_sig &o) const { return std::memcmp(v, o.v, sizeof v) == 0; }
};
struct edge_sig_hash {
    size_t operator()(const edge_sig &k) const {   // FNV-1a over the words
        uint64_t h = 1469598103934665603ull;
        for (int64_t x : k.v) h = (h ^ (uint64_t)x) * 1099511628211ull;
        return (size_t)h;
    }
};
edge_sig edge_key(const taps_graph *g, uint32_t e) {
    const taps_edge &E = g->edges[e];
    const taps_op &s = g->ops[E.src_op], &d = g->ops[E.dst_op];
    edge_sig k;
    std::memset(&k, 0, sizeof k);
    int n = 0;
    for (int64_t x : {(int64_t)s.n_axes, (int64_t)s.part_mask, (int64_t)s.dtype_bytes,
                      (int64_t)s.out.rank, (int64_t)d.n_axes, (int64_t)d.part_mask,
                      (int64_t)d.in[E.dst_slot].rank})
        k.v[n++] = x;
    for (uint32_t a = 0; a < TAPS_MAX_AXES; ++a) k.v[n++] = a < s.n_axes ? s.axis_len[a] : 0;
    for (uint32_t a = 0; a < TAPS_MAX_AXES; ++a) k.v[n++] = a < d.n_axes ? d.axis_len[a] : 0;
    for (uint32_t r = 0; r < TAPS_MAX_RANK; ++r) k.v[n++] = r < s.out.rank ? s.out.axis[r] : 0;
    for (uint32_t r = 0; r < TAPS_MAX_RANK; ++r)
        k.v[n++] = r < d.in[E.dst_slot].rank ? d.in[E.dst_slot].axis[r] : 0;
    return k;
}

// group[e] = the first edge whose key equals edge e's.
std::vector<uint32_t> group_edges(const taps_graph *g) {
    std::unordered_map<edge_sig, uint32_t, edge_sig_hash> first;
    first.reserve(2 * (size_t)g->n_edges + 1);
    std::vector<uint32_t> group(g->n_edges);
    for (uint32_t e = 0; e < g->n_edges; ++e)
        group[e] = first.emplace(edge_key(g, e), e).first->second;
    return group;
}

// rep[e]: the edge whose table edge e shares (itself if none).  One
// synchronisation reads back the device comparison of strategy ranges.
taps_status share_edges(const taps_graph *g, const uint64_t *op_offsets,
                        const taps_strategy *strategies, hipStream_t stream,
                        std::vector<uint32_t> &rep) {
    const uint32_t n_edges = g->n_edges;
    const std::vector<uint32_t> group = group_edges(g);
    std::map<std::pair<uint32_t, uint32_t>, uint32_t> pair_index;   // (op, rep op) -> pair
    std::vector<uint64_t> pairs;
    auto count = [&](uint32_t op) { return op_offsets[op + 1] - op_offsets[op]; };
    auto want = [&](uint32_t a, uint32_t b) -> int64_t {   // pair index, -1 if counts differ
        if (a == b) return -2;
        if (count(a) != count(b)) return -1;
        auto it = pair_index.find({a, b});
        if (it != pair_index.end()) return it->second;
        const uint32_t k = (uint32_t)(pairs.size() / 3);
        pairs.insert(pairs.end(), {op_offsets[a], op_offsets[b], count(a)});
        pair_index[{a, b}] = k;
        return k;
    };
    std::vector<int64_t> src_pair(n_edges, -2), dst_pair(n_edges, -2);
    for (uint32_t e = 0; e < n_edges; ++e) {
        rep[e] = group[e];
        if (rep[e] == e) continue;
        const taps_edge &E = g->edges[e], &R = g->edges[rep[e]];
        src_pair[e] = want(E.src_op, R.src_op);
        dst_pair[e] = want(E.dst_op, R.dst_op);
    }
    std::vector<uint32_t> flags(pairs.size() / 3, 0);
    if (!flags.empty()) {
        call_scratch sc(stream);
        uint64_t *d_pairs = nullptr;
        uint32_t *d_flags = nullptr;
        taps_status st;
        if ((st = sc.alloc((void **)&d_pairs, sizeof(uint64_t) * pairs.size())) != TAPS_OK) return st;
        if ((st = sc.alloc((void **)&d_flags, sizeof(uint32_t) * flags.size())) != TAPS_OK) return st;
        hipError_t err = hipMemcpyAsync(d_pairs, pairs.data(), sizeof(uint64_t) * pairs.size(),
                                        hipMemcpyHostToDevice, stream);
        if (err == hipSuccess)
            err = taps_launch_same_ranges(strategies, d_pairs, (uint32_t)flags.size(), d_flags,
                                          stream);
        if (err == hipSuccess)
            err = hipMemcpyAsync(flags.data(), d_flags, sizeof(uint32_t) * flags.size(),
                                 hipMemcpyDeviceToHost, stream);
        if (err == hipSuccess) err = wait_stream(stream);
        if (err != hipSuccess) return hip_fail(err, "strategy comparison");
    }
    auto same = [&](int64_t p) { return p == -2 || (p >= 0 && flags[p] == 0); };
    for (uint32_t e = 0; e < n_edges; ++e)
        if (rep[e] != e && !(same(src_pair[e]) && same(dst_pair[e]))) rep[e] = e;
    return TAPS_OK;
}

// Copy tasks of shared tables: every TAPS_COPY_CHUNK entries of a computed
// table (rep[e] == e with members) go to at most TAPS_COPY_DSTS of the tables
// that share it per task.
void plan_copies(const std::vector<uint64_t> &eoff, const std::vector<uint32_t> &rep,
                 std::vector<taps_copy_task> &copies, std::vector<uint64_t> &dst_list) {
    const uint32_t n_edges = (uint32_t)rep.size();
    std::vector<std::vector<uint32_t>> members(n_edges);
    for (uint32_t e = 0; e < n_edges; ++e)
        if (rep[e] != e) members[rep[e]].push_back(e);
    for (uint32_t r = 0; r < n_edges; ++r) {
        if (members[r].empty()) continue;
        const uint32_t begin = (uint32_t)dst_list.size();
        for (uint32_t m : members[r]) dst_list.push_back(eoff[m]);
        const uint64_t size = eoff[r + 1] - eoff[r];
        const uint32_t n_dst = (uint32_t)members[r].size();
        for (uint64_t k = 0; k < size; k += TAPS_COPY_CHUNK)
            for (uint32_t m = 0; m < n_dst; m += TAPS_COPY_DSTS) {
                taps_copy_task c;
                c.src = eoff[r] + k;
                c.offset = k;
                c.count = (uint32_t)(size - k < TAPS_COPY_CHUNK ? size - k : TAPS_COPY_CHUNK);
                c.dst_begin = begin + m;
                c.n_dst = n_dst - m < TAPS_COPY_DSTS ? n_dst - m : TAPS_COPY_DSTS;
                c.pad = 0;
                copies.push_back(c);
            }
    }
}

// The largest rank of the tensors the edges carry (the producers' outputs).
uint32_t max_edge_rank(const taps_graph *graph) {
    uint32_t r = 0;
    for (uint32_t e = 0; e < graph->n_edges; ++e) {
        const uint32_t k = graph->ops[graph->edges[e].src_op].out.rank;
        r = k > r ? k : r;
    }
    return r;
}

// Row segments of every computed table (rep[e] == e; rows are the source
// side's strategies, columns the target side's): each row cut into segments
// of `cols` columns and its remainder.  Ordered, the launch takes every
// full-length segment first (edges in order, a row's segments together) and
// the remainders last, longest first, so that it ends on its shortest
// segments; otherwise each row's segments, remainder included, run together.
// Returns the number of segments.
uint64_t plan_segments(const taps_graph *graph, const uint64_t *op_offsets, bool reverse,
                       const std::vector<uint32_t> &rep, uint32_t cols, bool ordered,
                       std::vector<taps_seg_group> &groups) {
    struct remainder {
        uint32_t edge, rows, first_col, cols;
    };
    std::vector<remainder> rems;
    groups.clear();
    uint64_t start = 0;
    for (uint32_t e = 0; e < graph->n_edges; ++e) {
        if (rep[e] != e) continue;
        const taps_edge &E = graph->edges[e];
        const uint64_t np = op_offsets[E.src_op + 1] - op_offsets[E.src_op];
        const uint64_t nc = op_offsets[E.dst_op + 1] - op_offsets[E.dst_op];
        const uint64_t ns = reverse ? nc : np, nd = reverse ? np : nc;
        if (ns == 0 || nd == 0) continue;
        if (!ordered) {
            const uint64_t per_row = (nd + cols - 1) / cols;
            groups.push_back({start, e, (uint32_t)per_row, 0u, cols});
            start += ns * per_row;
            continue;
        }
        const uint64_t full = nd / cols, left = nd % cols;
        if (full) {
            groups.push_back({start, e, (uint32_t)full, 0u, cols});
            start += ns * full;
        }
        if (left) rems.push_back({e, (uint32_t)ns, (uint32_t)(full * cols), (uint32_t)left});
    }
    std::stable_sort(rems.begin(), rems.end(),
                     [](const remainder &a, const remainder &b) { return a.cols > b.cols; });
    for (const remainder &r : rems) {
        groups.push_back({start, r.edge, 1u, r.first_col, r.cols});
        start += r.rows;
    }
    return start;
}

// The segments of a one-table launch: long segments (remainders last) when
// there are enough of them to fill the GPU many times over, else short ones in
// row order.
std::atomic<uint64_t> g_long_segs_min{TAPS_LONG_SEGS_MIN};

uint64_t plan_launch(const taps_graph *graph, const uint64_t *op_offsets, bool reverse,
                     const std::vector<uint32_t> &rep, bool one_table,
                     std::vector<taps_seg_group> &groups) {
    if (one_table) {
        const uint64_t n = plan_segments(graph, op_offsets, reverse, rep,
                                         TAPS_TILE_COLS * TAPS_SEG_TILES_LONG, true, groups);
        if (n >= g_long_segs_min.load(std::memory_order_relaxed)) return n;
    }
    return plan_segments(graph, op_offsets, reverse, rep, TAPS_TILE_COLS * TAPS_SEG_TILES_SHORT,
                         one_table, groups);
}

// Edge tables of one graph at n_points bandwidth points (clusters that differ
// only in their bandwidths), table k in outs[k]; outs NULL or every table's
// arrays NULL: size query.
taps_status edge_costs(const taps_graph *graph, const taps_cluster *clusters, uint32_t n_points,
                       const taps_strategy *strategies, const uint64_t *op_offsets,
                       uint64_t *edge_offsets, const taps_table *outs, uint64_t capacity,
                       void *stream_, bool share, bool reverse, const taps_hier *hier = nullptr) {
    g_last_error.clear();
    if (!clusters) return fail(TAPS_ERR_ARG, "cluster is NULL");
    if (n_points == 0 || n_points > TAPS_MAX_SWEEP)
        return fail(TAPS_ERR_ARG, "%u bandwidth points, 1 to %u allowed", n_points,
                    (unsigned)TAPS_MAX_SWEEP);
    taps_launch lps[TAPS_MAX_SWEEP];
    taps_status st = TAPS_OK;
    for (uint32_t k = 0; k < n_points && st == TAPS_OK; ++k) {
        st = check_cluster(&clusters[k], &lps[k]);
        if (st == TAPS_OK && (clusters[k].nodes != clusters[0].nodes ||
                              clusters[k].devices_per_node != clusters[0].devices_per_node))
            st = fail(TAPS_ERR_ARG, "bandwidth point %u: %u x %u devices, point 0 has %u x %u", k,
                      clusters[k].nodes, clusters[k].devices_per_node, clusters[0].nodes,
                      clusters[0].devices_per_node);
    }
    const taps_launch &lp = lps[0];
    if (st == TAPS_OK) st = check_graph(graph, true);
    if (st == TAPS_OK) st = check_offsets(graph, op_offsets);
    if (st != TAPS_OK) return st;
    if (!edge_offsets) return fail(TAPS_ERR_ARG, "edge_offsets is NULL");
    const uint32_t n_ops = graph->n_ops, n_edges = graph->n_edges;
    std::vector<uint64_t> eoff(n_edges + 1, 0);
    uint64_t all_segs = 0;   // row segments without sharing (an upper bound)
    for (uint32_t e = 0; e < n_edges; ++e) {
        const taps_edge &E = graph->edges[e];
        const uint64_t np = op_offsets[E.src_op + 1] - op_offsets[E.src_op];
        const uint64_t nc = op_offsets[E.dst_op + 1] - op_offsets[E.dst_op];
        const uint64_t ns = reverse ? nc : np, nd = reverse ? np : nc;   // rows, columns
        eoff[e + 1] = eoff[e] + ns * nd;
        all_segs += ns * ((nd + TAPS_TILE_COLS - 1) / TAPS_TILE_COLS);
    }
    bool none = true, all = outs != nullptr;
    for (uint32_t k = 0; outs && k < n_points; ++k) {
        const taps_table &o = outs[k];
        none = none && !o.t && !o.vol && !o.intra && !o.inter && !o.meta;
        all = all && o.t && o.vol && o.intra && o.inter && o.meta;
    }
    if (!none && !all)
        return fail(TAPS_ERR_ARG, "table arrays must be all set or all NULL (every point)");
    if (all && eoff[n_edges] > capacity)
        return fail(TAPS_ERR_CAPACITY, "%llu entries, capacity %llu",
                    (unsigned long long)eoff[n_edges], (unsigned long long)capacity);
    if (all && eoff[n_edges] > 0 && !strategies) return fail(TAPS_ERR_ARG, "strategies is NULL");
    if (all_segs >= 0x7FFFFFFFull) return fail(TAPS_ERR_ARG, "more than 2^31 row segments");
    std::memcpy(edge_offsets, eoff.data(), sizeof(uint64_t) * (n_edges + 1));
    if (none || eoff[n_edges] == 0) return TAPS_OK;
    hipStream_t stream = (hipStream_t)stream_;
    // shared tables: every group computes its representative's rows once
    std::vector<uint32_t> rep(n_edges);
    std::iota(rep.begin(), rep.end(), 0u);
    if (share && (st = share_edges(graph, op_offsets, strategies, stream, rep)) != TAPS_OK)
        return st;
    // row segments of every computed table (shared tables: the first of each group)
    // (the bandwidth sweep runs over aligned windows of the tables instead)
    std::vector<taps_seg_group> groups;
    const uint64_t n_segs =
        n_points == 1 ? plan_launch(graph, op_offsets, reverse, rep, true, groups) : 0;
    // shared tables: every chunk of a computed table is stored into each table sharing it
    std::vector<uint64_t> dst_list;
    std::vector<taps_copy_task> copies;
    plan_copies(eoff, rep, copies, dst_list);
    if (copies.size() > 0x7FFFFFFFull) return fail(TAPS_ERR_ARG, "too many table copies");
    call_scratch sc(stream);
    const uint64_t total = op_offsets[n_ops];
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {graph->edges, sizeof(taps_edge) * n_edges, 0},
                          {op_offsets, sizeof(uint64_t) * (n_ops + 1), 0},
                          {eoff.data(), sizeof(uint64_t) * (n_edges + 1), 0},
                          {groups.data(), sizeof(taps_seg_group) * groups.size(), 0},
                          {copies.data(), sizeof(taps_copy_task) * copies.size(), 0},
                          {dst_list.data(), sizeof(uint64_t) * dst_list.size(), 0}};
    void *dev = nullptr;
    if ((st = upload(sc, ch, &dev)) != TAPS_OK) return st;
    taps_desc *d_desc = nullptr;
    taps_edge_params *d_params = nullptr;
    taps_row_ref *d_segs = nullptr;
    if ((st = sc.alloc((void **)&d_desc, sizeof(taps_desc) * total)) != TAPS_OK) return st;
    if ((st = sc.alloc((void **)&d_params, sizeof(taps_edge_params) * n_edges)) != TAPS_OK) return st;
    if ((st = sc.alloc((void **)&d_segs, sizeof(taps_row_ref) * n_segs)) != TAPS_OK) return st;
    // the bandwidth sweep runs over aligned 64-entry windows: each window's edge
    uint32_t *d_win = nullptr;
    const uint64_t n_windows = (eoff[n_edges] + TAPS_TILE_COLS * TAPS_WIN_TILES - 1) /
                               (TAPS_TILE_COLS * TAPS_WIN_TILES);
    if (n_points > 1 && !hier &&
        (st = sc.alloc((void **)&d_win, sizeof(uint32_t) * n_windows)) != TAPS_OK)
        return st;
    hipError_t err = taps_launch_describe(strategies, total, d_desc, stream);
    if (err == hipSuccess) {
        const taps_plan_args pa{at<taps_op>(dev, ch[0]), at<taps_edge>(dev, ch[1]),
                                at<uint64_t>(dev, ch[2]), at<uint64_t>(dev, ch[3]),
                                at<taps_seg_group>(dev, ch[4]), d_params, d_segs, n_segs,
                                n_edges, (uint32_t)groups.size(), reverse ? 1u : 0u, 0u};
        err = taps_launch_edge_setup(pa, lp, stream);
    }
    // the edge-table kernel launches (entries > 0): use the events, if any, once
    const hipEvent_t before = g_kernel_before, after = g_kernel_after;
    g_kernel_before = g_kernel_after = nullptr;
    if (err == hipSuccess && before) err = hipEventRecord(before, stream);
    if (err == hipSuccess && hier) {
        err = taps_launch_edge_costs_h(d_params, d_segs, n_segs, d_desc, lp, max_edge_rank(graph),
                                       *hier, outs[0], stream);
    } else if (err == hipSuccess && n_points == 1) {
        err = taps_launch_edge_costs(d_params, d_segs, n_segs, d_desc, lp, max_edge_rank(graph),
                                     outs[0], stream);
    } else if (err == hipSuccess) {
        taps_sweep sw;
        std::memset(&sw, 0, sizeof(sw));
        sw.count = n_points;
        for (uint32_t k = 0; k < n_points; ++k) {
            sw.narrow[k] = lps[k].narrow;
            sw.b_inter_red[k] = lps[k].b_inter_red;
            sw.b_intra_red[k] = lps[k].b_intra_red;
            sw.inv_n_bintra[k] = lps[k].inv_n_bintra;
            sw.inv_n_binter[k] = lps[k].inv_n_binter;
            sw.out[k] = outs[k];
        }
        err = taps_launch_edge_costs_sweep_win(d_params, n_edges, at<uint64_t>(dev, ch[3]),
                                               eoff[n_edges], d_win, d_desc, lp,
                                               max_edge_rank(graph), sw, stream);
    }
    for (uint32_t k = 0; k < n_points && err == hipSuccess; ++k)
        err = taps_launch_copy_tables(at<taps_copy_task>(dev, ch[5]), (uint32_t)copies.size(),
                                      at<uint64_t>(dev, ch[6]), outs[k], stream);
    if (err == hipSuccess && after) err = hipEventRecord(after, stream);
    if (err != hipSuccess) return hip_fail(err, "edge costs");
    return TAPS_OK;
}

// A hierarchy of link classes: the per-level class and boundary tables and
// the exact-order weights of the kernels, and a cluster with the same device
// count and innermost block (for the per-edge set-up that the two models
// share).
taps_status check_topology(const taps_topology *t, taps_hier *H, taps_cluster *cl) {
    if (!t) return fail(TAPS_ERR_ARG, "topology is NULL");
    if (t->n_classes < 1 || t->n_classes > TAPS_MAX_CLASSES)
        return fail(TAPS_ERR_TOPOLOGY, "%u link classes, 1 to %u allowed", t->n_classes,
                    (unsigned)TAPS_MAX_CLASSES);
    const uint32_t C = t->n_classes;
    for (uint32_t c = 0; c < C; ++c) {
        if (!pow2(t->domain[c]) || (c && t->domain[c] < t->domain[c - 1]))
            return fail(TAPS_ERR_TOPOLOGY, "domain %u (%u devices) must be a power of two, "
                        "not below the previous one", c, t->domain[c]);
        if (t->bw[c] == 0) return fail(TAPS_ERR_TOPOLOGY, "bandwidth of class %u is zero", c);
    }
    const uint64_t N = t->domain[C - 1];
    if (N > (1ull << TAPS_MAX_LEVELS))
        return fail(TAPS_ERR_TOPOLOGY, "%llu devices exceed the limit of %u", (unsigned long long)N,
                    1u << TAPS_MAX_LEVELS);
    // exact-order weights lcm(bw) / bw[c] (and the in-block AllToAll's), each below 2^30
    const uint32_t nb = C + (t->bw_a2a ? 1u : 0u);
    auto bw_of = [&](uint32_t c) { return c < C ? t->bw[c] : t->bw_a2a; };
    unsigned __int128 lcm = 1;
    for (uint32_t c = 0; c < nb; ++c) {
        const uint64_t g = std::gcd((uint64_t)(lcm % bw_of(c)), bw_of(c));
        const unsigned __int128 q = lcm / g;
        if (q >> 64) return fail(TAPS_ERR_TOPOLOGY, "bandwidths not in round ratios");
        lcm = q * bw_of(c);
    }
    std::memset(H, 0, sizeof(*H));
    H->n_classes = C;
    for (uint32_t c = 0; c < nb; ++c) {
        const unsigned __int128 w = lcm / bw_of(c);
        if (w >> 30)
            return fail(TAPS_ERR_TOPOLOGY, "bandwidths not in round ratios (lcm / bw >= 2^30)");
        const double inv = 1.0 / ((double)N * (double)bw_of(c));
        if (c < C) {
            H->w[c] = (uint64_t)w;
            H->inv_n_bw[c] = inv;
        } else {
            H->w_a2a = (uint64_t)w;
            H->inv_n_bw_a2a = inv;
            H->a2a_own = 1;
        }
    }
    // class of a collective with top level l: the boundaries log2(domain[c]) <= l (c < C - 1);
    // its ct counts the uplinks of a block of the largest of them
    for (uint32_t l = 0; l < TAPS_MAX_LEVELS; ++l) {
        uint32_t cls = 0, beta = 0;
        for (uint32_t c = 0; c + 1 < C; ++c) {
            const uint32_t b = log2u(t->domain[c]);
            if (b <= l) {
                ++cls;
                beta = b;
            }
        }
        H->cls_of_top |= cls << (4u * l);
        H->beta_of_top |= beta << (4u * l);
        H->levels_of_cls[cls] |= 1u << l;
        H->beta_of_cls[cls] = beta;
    }
    cl->nodes = (uint32_t)(N / t->domain[0]);
    cl->devices_per_node = t->domain[0];
    cl->bw_intra = t->bw[0];
    cl->bw_inter = t->bw[C - 1];
    return TAPS_OK;
}

// The number of strategies GenerateStrategySet keeps for an operator on 2^n
// devices: ordered runs of distinct partitionable axes that cover levels
// 0..n-1 from level 0, axis a's run at most v_a = (trailing zero bits of its
// length) wide so that its degree divides its length, every boundary between
// two runs an allowed cut -- the candidates of k_build_strategies that pass its
// two tests, counted by a dynamic program over (levels covered, axes used).  The
// count depends only on n, the allowed cuts, the partitionable axes and their
// v_a, so it is memoised on those (per thread).
uint64_t strategy_count(const taps_op &op, uint32_t n, uint32_t allowed) {
    uint64_t key = n | (uint64_t)(allowed & 0xFFu) << 4 | (uint64_t)op.part_mask << 12;
    uint32_t v[TAPS_MAX_AXES] = {0};
    for (uint32_t a = 0; a < op.n_axes; ++a) {
        if (!((op.part_mask >> a) & 1u)) continue;
        const uint32_t z = (uint32_t)__builtin_ctzll((uint64_t)op.axis_len[a]);
        v[a] = z < n ? z : n;
        key |= (uint64_t)v[a] << (20 + 4 * a);
    }
    thread_local std::unordered_map<uint64_t, uint64_t> memo;
    const auto it = memo.find(key);
    if (it != memo.end()) return it->second;
    // ways[s][m]: sequences of runs covering levels 0..s-1 with axis set m
    std::vector<uint64_t> ways((size_t)(n + 1) << TAPS_MAX_AXES, 0);
    ways[0] = 1;
    for (uint32_t lev = 0; lev < n; ++lev)
        for (uint32_t m = 0; m < (1u << TAPS_MAX_AXES); ++m) {
            const uint64_t w = ways[((size_t)lev << TAPS_MAX_AXES) | m];
            if (!w) continue;
            for (uint32_t a = 0; a < op.n_axes; ++a) {
                if (!((op.part_mask >> a) & 1u) || ((m >> a) & 1u)) continue;
                for (uint32_t e = 1; e <= v[a] && lev + e <= n; ++e) {
                    const uint32_t t = lev + e;
                    if (t < n && !((allowed >> t) & 1u)) continue;
                    ways[((size_t)t << TAPS_MAX_AXES) | (m | (1u << a))] += w;
                }
            }
        }
    uint64_t count = 0;
    for (uint32_t m = 0; m < (1u << TAPS_MAX_AXES); ++m) count += ways[((size_t)n << TAPS_MAX_AXES) | m];
    memo.emplace(key, count);
    return count;
}

// Strategies among each chunk of TAPS_BUILD_CHUNK candidate ranks of an
// operator, found with the device's own unranking and filter, memoised on
// what decides them (devices, allowed cuts, axes, partitionable axes and the
// trailing zero bits of their lengths).
const std::vector<uint32_t> &chunk_counts(const taps_op &op, uint32_t n, uint32_t allowed) {
    static const taps_completion_table W = taps_make_completions();
    uint64_t key = n | (uint64_t)(allowed & 0xFFu) << 4 | (uint64_t)op.part_mask << 12 |
                   (uint64_t)op.n_axes << 20;
    for (uint32_t a = 0; a < op.n_axes; ++a) {
        if (!((op.part_mask >> a) & 1u)) continue;
        const uint32_t z = (uint32_t)__builtin_ctzll((uint64_t)op.axis_len[a]);
        key |= (uint64_t)(z < n ? z : n) << (24 + 4 * a);
    }
    thread_local std::unordered_map<uint64_t, std::vector<uint32_t>> memo;
    const auto it = memo.find(key);
    if (it != memo.end()) return it->second;
    const uint32_t total = W.v[(taps_popc(op.part_mask) * 9u + n) * 9u];
    std::vector<uint32_t> counts((total + TAPS_BUILD_CHUNK - 1) / TAPS_BUILD_CHUNK, 0);
    for (uint32_t r = 0; r < total; ++r) {
        uint32_t expo[TAPS_D_MAX_AXES];
        int32_t pos[TAPS_D_MAX_AXES];
        if (!taps_unrank(op.n_axes, op.part_mask, n, r, W.v, expo, pos)) continue;
        bool valid = true;
        for (uint32_t a = 0; a < op.n_axes; ++a)
            if (op.axis_len[a] & (((int64_t)1 << expo[a]) - 1)) valid = false;
        if (valid && (taps_describe(op.n_axes, expo, pos).cuts & ~allowed)) valid = false;
        counts[r / TAPS_BUILD_CHUNK] += valid ? 1u : 0u;
    }
    return memo.emplace(key, std::move(counts)).first->second;
}

// The workgroups of k_build_strategies: every chunk of candidate ranks that
// holds a strategy, at the operator's offset plus the strategies of the
// chunks before it.  The chunks' counts must add up to the exact count.
taps_status plan_build(const taps_graph *graph, uint32_t n, uint32_t allowed,
                       const std::vector<uint64_t> &offs, std::vector<taps_build_chunk> &chunks) {
    chunks.clear();
    for (uint32_t k = 0; k < graph->n_ops; ++k) {
        const std::vector<uint32_t> &cc = chunk_counts(graph->ops[k], n, allowed);
        uint64_t base = offs[k];
        for (uint32_t c = 0; c < cc.size(); ++c) {
            if (!cc[c]) continue;
            chunks.push_back({base, k, c * (uint32_t)TAPS_BUILD_CHUNK, cc[c], 0u});
            base += cc[c];
        }
        if (base != offs[k + 1])
            return fail(TAPS_ERR_ARG, "op %u: %llu strategies by chunks, %llu counted", k,
                        (unsigned long long)(base - offs[k]),
                        (unsigned long long)(offs[k + 1] - offs[k]));
    }
    if (chunks.size() > 0x7FFFFFFFull) return fail(TAPS_ERR_ARG, "too many strategy chunks");
    return TAPS_OK;
}

// Per-operator strategy counts and offsets (host); TAPS_ERR_NO_STRATEGY if an
// operator has none.
taps_status count_strategies(const taps_graph *graph, uint32_t n, uint32_t allowed,
                             std::vector<uint64_t> &offs) {
    const uint32_t n_ops = graph->n_ops;
    offs.assign(n_ops + 1, 0);
    for (uint32_t k = 0; k < n_ops; ++k) {
        const uint64_t c = strategy_count(graph->ops[k], n, allowed);
        if (c == 0)
            return fail(TAPS_ERR_NO_STRATEGY,
                        "op %u has no strategy on %u devices (no partitionable axis whose length "
                        "the degrees divide)",
                        k, 1u << n);
        offs[k + 1] = offs[k] + c;
    }
    if (offs[n_ops] > 0xFFFFFFFFull) return fail(TAPS_ERR_ARG, "more than 2^32 strategies");
    return TAPS_OK;
}

// GenerateStrategySet: sizes on the host, strategies on the device (no
// synchronisation); allowed_cuts: the level boundaries a strategy's axis runs
// may meet (all of them unless a fixed mesh is given).
taps_status enumerate(const taps_graph *graph, const taps_launch &lp, uint32_t allowed_cuts,
                      uint64_t *op_offsets, taps_strategy *strategies, uint64_t capacity,
                      void *stream_) {
    std::vector<uint64_t> offs;
    taps_status st = count_strategies(graph, lp.n, allowed_cuts, offs);
    if (st != TAPS_OK) return st;
    const uint32_t n_ops = graph->n_ops;
    std::memcpy(op_offsets, offs.data(), sizeof(uint64_t) * (n_ops + 1));
    if (!strategies || n_ops == 0) return TAPS_OK;
    if (offs[n_ops] > capacity)
        return fail(TAPS_ERR_CAPACITY, "%llu strategies, capacity %llu",
                    (unsigned long long)offs[n_ops], (unsigned long long)capacity);
    std::vector<taps_build_chunk> chunks;
    if ((st = plan_build(graph, lp.n, allowed_cuts, offs, chunks)) != TAPS_OK) return st;
    hipStream_t stream = (hipStream_t)stream_;
    call_scratch sc(stream);
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {chunks.data(), sizeof(taps_build_chunk) * chunks.size(), 0}};
    void *dev = nullptr;
    if ((st = upload(sc, ch, &dev)) != TAPS_OK) return st;
    const taps_table no_node = {nullptr, nullptr, nullptr, nullptr, nullptr};
    const hipError_t err = taps_launch_build_strategies(
        at<taps_op>(dev, ch[0]), at<taps_build_chunk>(dev, ch[1]), (uint32_t)chunks.size(),
        allowed_cuts, lp, strategies, nullptr, no_node, stream);
    if (err != hipSuccess) return hip_fail(err, "enumerate");
    return TAPS_OK;
}

// The level boundaries of a fixed mesh (bit c: between levels c-1 and c), or
// TAPS_ERR_TOPOLOGY unless its sizes are powers of two >= 2 multiplying to 2^n.
taps_status mesh_cuts(const taps_mesh *mesh, uint32_t n, uint32_t *allowed) {
    if (!mesh) return fail(TAPS_ERR_ARG, "mesh is NULL");
    if (mesh->n_dims > TAPS_MAX_LEVELS)
        return fail(TAPS_ERR_TOPOLOGY, "a mesh has at most %u dimensions (got %u)",
                    TAPS_MAX_LEVELS, mesh->n_dims);
    uint32_t level = 0, cuts = 0;
    for (uint32_t k = 0; k < mesh->n_dims; ++k) {
        const uint32_t m = mesh->dims[k];
        if (m < 2 || !pow2(m))
            return fail(TAPS_ERR_TOPOLOGY, "mesh dimension %u has size %u (not a power of two >= 2)",
                        k, m);
        if (level) cuts |= 1u << level;
        level += log2u(m);
        if (level > n) break;
    }
    if (level != n)
        return fail(TAPS_ERR_TOPOLOGY, "the mesh does not have 2^%u devices", n);
    *allowed = cuts;
    return TAPS_OK;
}


// Device memory of one build: carve() hands out 256-byte aligned arrays and
// put() uploads host chunks into one of them.
struct workspace {
    virtual ~workspace() = default;
    virtual taps_status carve(void **p, size_t bytes) = 0;
    virtual taps_status put(std::vector<chunk> &chunks, void **dev) = 0;
};

// The stream's scratch block, and uploads through the pinned staging pool.
struct stream_workspace : workspace {
    call_scratch sc;
    explicit stream_workspace(hipStream_t s) : sc(s) {}
    taps_status carve(void **p, size_t bytes) override { return sc.alloc(p, bytes); }
    taps_status put(std::vector<chunk> &chunks, void **dev) override {
        return upload(sc, chunks, dev);
    }
};

// The device address of the current device's `scratch` array (see its
// definition), taken on the device's first call.
taps_status scratch_address(char **base) {
    static std::mutex mu;
    static char *addr[kMaxDevices] = {};
    int device = -1;
    hipError_t err = hipGetDevice(&device);
    if (err != hipSuccess) return hip_fail(err, "hipGetDevice");
    if (device < 0 || device >= (int)kMaxDevices)
        return fail(TAPS_ERR_DEVICE, "device %d: the fixed workspace serves devices 0..%u", device,
                    kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        void *p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return hip_fail(err, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(TAPS_ERR_DEVICE, "hipGetSymbolAddress(scratch) returned NULL");
        addr[device] = (char *)p;
    }
    *base = addr[device];
    return TAPS_OK;
}

// Carves from the current device's fixed array and uploads with one
// hipMemcpyAsync from a per-thread host buffer: no device or pinned memory is
// allocated.
struct fixed_workspace : workspace {
    hipStream_t stream;
    char *base = nullptr;
    size_t used = 0;
    explicit fixed_workspace(hipStream_t s) : stream(s) {}
    taps_status open() { return scratch_address(&base); }
    taps_status carve(void **p, size_t bytes) override {
        const size_t size = carve_size(bytes);
        if (used + size > TAPS_NOALLOC_SCRATCH_BYTES)   // the caller checked the whole need
            return fail(TAPS_ERR_CAPACITY, "fixed workspace exhausted");
        *p = base + used;
        used += size;
        return TAPS_OK;
    }
    taps_status put(std::vector<chunk> &chunks, void **dev) override {
        size_t total = 0;
        for (chunk &c : chunks) {
            c.offset = total;
            total += align256(c.bytes);
        }
        if (total == 0) total = 256;
        taps_status st = carve(dev, total);
        if (st != TAPS_OK) return st;
        // pageable host memory: the copy has read it when hipMemcpyAsync returns
        thread_local std::vector<char> host;
        if (host.size() < total) host.resize(total);
        for (const chunk &c : chunks)
            if (c.bytes) std::memcpy(host.data() + c.offset, c.src, c.bytes);
        const hipError_t err = hipMemcpyAsync(*dev, host.data(), total, hipMemcpyHostToDevice,
                                              stream);
        if (err != hipSuccess) return hip_fail(err, "hipMemcpyAsync (upload)");
        return TAPS_OK;
    }
};

taps_status build_tables(const taps_graph *graph, const taps_cluster *cluster, const taps_mesh *mesh,
                         uint64_t *op_offsets, taps_strategy *strategies,
                         uint64_t strategy_capacity, taps_table node, uint64_t *edge_offsets,
                         taps_table edge, uint64_t edge_capacity, uint32_t flags, void *stream_,
                         bool fixed) {
    g_last_error.clear();
    if (flags & ~TAPS_BUILD_SHARED) return fail(TAPS_ERR_ARG, "unknown flags 0x%x", flags);
    taps_launch lp;
    taps_status st = check_cluster(cluster, &lp);
    if (st == TAPS_OK) st = check_graph(graph, true);
    if (st != TAPS_OK) return st;
    if (!op_offsets || !edge_offsets) return fail(TAPS_ERR_ARG, "op_offsets or edge_offsets is NULL");
    uint32_t allowed = 0xFFu;
    if (mesh && (st = mesh_cuts(mesh, lp.n, &allowed)) != TAPS_OK) return st;
    const uint32_t n_ops = graph->n_ops, n_edges = graph->n_edges;
    // sizes, on the host
    std::vector<uint64_t> offs;
    if ((st = count_strategies(graph, lp.n, allowed, offs)) != TAPS_OK) return st;
    // shared tables: edges described alike share one table -- their operators'
    // strategies are the same function of the same descriptions here, so no
    // device comparison is needed
    std::vector<uint32_t> rep(n_edges);
    std::iota(rep.begin(), rep.end(), 0u);
    if (flags & TAPS_BUILD_SHARED) {
        rep = group_edges(graph);
    }
    std::vector<uint64_t> eoff(n_edges + 1, 0);
    uint64_t all_segs = 0;
    for (uint32_t e = 0; e < n_edges; ++e) {
        const taps_edge &E = graph->edges[e];
        const uint64_t ns = offs[E.src_op + 1] - offs[E.src_op];
        const uint64_t nd = offs[E.dst_op + 1] - offs[E.dst_op];
        eoff[e + 1] = eoff[e] + ns * nd;
        all_segs += ns * ((nd + TAPS_TILE_COLS - 1) / TAPS_TILE_COLS);
    }
    if (all_segs >= 0x7FFFFFFFull) return fail(TAPS_ERR_ARG, "more than 2^31 row segments");
    std::vector<uint64_t> dst_list;
    std::vector<taps_copy_task> copies;
    plan_copies(eoff, rep, copies, dst_list);
    if (copies.size() > 0x7FFFFFFFull) return fail(TAPS_ERR_ARG, "too many table copies");
    // a size query passes no array; a build passes the strategy and node arrays, and
    // the edge arrays unless there are no edge entries (then they are not read)
    const bool none_s = !strategies && !node.t && !node.vol && !node.intra && !node.inter &&
                        !node.meta;
    const bool all_s = strategies && node.t && node.vol && node.intra && node.inter && node.meta;
    const bool none_e = !edge.t && !edge.vol && !edge.intra && !edge.inter && !edge.meta;
    const bool all_e = edge.t && edge.vol && edge.intra && edge.inter && edge.meta;
    const bool none = none_s && none_e;
    if (!none && !(all_s && (all_e || (none_e && eoff[n_edges] == 0))))
        return fail(TAPS_ERR_ARG, "strategies and every table array must be all set or all NULL "
                                  "(the edge arrays may be NULL when there are no edge entries)");
    if (!none && offs[n_ops] > strategy_capacity)
        return fail(TAPS_ERR_CAPACITY, "%llu strategies, capacity %llu",
                    (unsigned long long)offs[n_ops], (unsigned long long)strategy_capacity);
    if (!none && eoff[n_edges] > edge_capacity)
        return fail(TAPS_ERR_CAPACITY, "%llu entries, capacity %llu",
                    (unsigned long long)eoff[n_edges], (unsigned long long)edge_capacity);
    if (none || n_ops == 0) {
        std::memcpy(op_offsets, offs.data(), sizeof(uint64_t) * (n_ops + 1));
        std::memcpy(edge_offsets, eoff.data(), sizeof(uint64_t) * (n_edges + 1));
        return TAPS_OK;
    }
    // one upload and one set of scratch for the whole build
    hipStream_t stream = (hipStream_t)stream_;
    std::vector<taps_build_chunk> bchunks;
    if ((st = plan_build(graph, lp.n, allowed, offs, bchunks)) != TAPS_OK) return st;
    std::vector<taps_seg_group> groups;
    const uint64_t total = offs[n_ops];
    const uint64_t n_segs = plan_launch(graph, offs.data(), false, rep, true, groups);
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {graph->edges, sizeof(taps_edge) * n_edges, 0},
                          {offs.data(), sizeof(uint64_t) * (n_ops + 1), 0},
                          {eoff.data(), sizeof(uint64_t) * (n_edges + 1), 0},
                          {groups.data(), sizeof(taps_seg_group) * groups.size(), 0},
                          {copies.data(), sizeof(taps_copy_task) * copies.size(), 0},
                          {dst_list.data(), sizeof(uint64_t) * dst_list.size(), 0},
                          {bchunks.data(), sizeof(taps_build_chunk) * bchunks.size(), 0}};
    if (fixed) {   // the whole need, checked on the host before any HIP call
        size_t up = 0;
        for (const chunk &c : ch) up += align256(c.bytes);
        const size_t need = carve_size(up) + carve_size(sizeof(taps_desc) * total) +
                            carve_size(sizeof(taps_edge_params) * (n_edges ? n_edges : 1)) +
                            carve_size(sizeof(taps_row_ref) * (n_segs ? n_segs : 1));
        if (need > TAPS_NOALLOC_SCRATCH_BYTES)
            return fail(TAPS_ERR_CAPACITY,
                        "this build needs %llu bytes of device workspace; the fixed workspace of "
                        "taps_build_tables_noalloc holds %llu",
                        (unsigned long long)need, (unsigned long long)TAPS_NOALLOC_SCRATCH_BYTES);
    }
    std::memcpy(op_offsets, offs.data(), sizeof(uint64_t) * (n_ops + 1));
    std::memcpy(edge_offsets, eoff.data(), sizeof(uint64_t) * (n_edges + 1));
    // device memory: the stream's scratch block, or the fixed workspace
    std::unique_ptr<workspace> ws;
    if (fixed) {
        auto fw = std::make_unique<fixed_workspace>(stream);
        if ((st = fw->open()) != TAPS_OK) return st;
        ws = std::move(fw);
    } else {
        ws = std::make_unique<stream_workspace>(stream);
    }
    void *dev = nullptr;
    if ((st = ws->put(ch, &dev)) != TAPS_OK) return st;
    taps_desc *d_desc = nullptr;
    taps_edge_params *d_params = nullptr;
    taps_row_ref *d_segs = nullptr;
    if ((st = ws->carve((void **)&d_desc, sizeof(taps_desc) * total)) != TAPS_OK) return st;
    if ((st = ws->carve((void **)&d_params, sizeof(taps_edge_params) * (n_edges ? n_edges : 1))) !=
        TAPS_OK)
        return st;
    if ((st = ws->carve((void **)&d_segs, sizeof(taps_row_ref) * (n_segs ? n_segs : 1))) !=
        TAPS_OK)
        return st;
    // the strategies, and the edge plan when there are edge entries, in one launch
    const bool edges_on = eoff[n_edges] > 0;
    const taps_plan_args pa{at<taps_op>(dev, ch[0]), at<taps_edge>(dev, ch[1]),
                            at<uint64_t>(dev, ch[2]), at<uint64_t>(dev, ch[3]),
                            at<taps_seg_group>(dev, ch[4]), d_params, d_segs,
                            edges_on ? n_segs : 0u, edges_on ? n_edges : 0u,
                            edges_on ? (uint32_t)groups.size() : 0u, 0u, 0u};
    hipError_t err = taps_launch_build_front(at<taps_build_chunk>(dev, ch[7]),
                                             (uint32_t)bchunks.size(), allowed, lp, strategies,
                                             d_desc, node, pa, stream);
    if (err == hipSuccess && edges_on) {
        const hipEvent_t before = g_kernel_before, after = g_kernel_after;
        g_kernel_before = g_kernel_after = nullptr;
        if (err == hipSuccess && before) err = hipEventRecord(before, stream);
        if (err == hipSuccess)
            err = taps_launch_edge_costs(d_params, d_segs, n_segs, d_desc, lp,
                                         max_edge_rank(graph), edge, stream);
        if (err == hipSuccess)
            err = taps_launch_copy_tables(at<taps_copy_task>(dev, ch[5]), (uint32_t)copies.size(),
                                          at<uint64_t>(dev, ch[6]), edge, stream);
        if (err == hipSuccess && after) err = hipEventRecord(after, stream);
    }
    if (err != hipSuccess) return hip_fail(err, "build");
    return TAPS_OK;
}

}  // namespace

extern "C" {

const char *taps_status_str(taps_status s) {
    switch (s) {
    case TAPS_OK: return "TAPS_OK";
    case TAPS_ERR_ARG: return "TAPS_ERR_ARG";
    case TAPS_ERR_TOPOLOGY: return "TAPS_ERR_TOPOLOGY";
    case TAPS_ERR_SHAPE: return "TAPS_ERR_SHAPE";
    case TAPS_ERR_NO_STRATEGY: return "TAPS_ERR_NO_STRATEGY";
    case TAPS_ERR_CAPACITY: return "TAPS_ERR_CAPACITY";
    case TAPS_ERR_DEVICE: return "TAPS_ERR_DEVICE";
    }
    return "TAPS_ERR_UNKNOWN";
}

const char *taps_last_error(void) { return g_last_error.c_str(); }

uint64_t taps_set_long_segments_min(uint64_t min_segments) {
    return g_long_segs_min.exchange(min_segments);
}

taps_status taps_set_edge_kernel_events(void *before, void *after) {
    g_last_error.clear();
    if ((before == nullptr) != (after == nullptr))
        return fail(TAPS_ERR_ARG, "both kernel events or neither");
    g_kernel_before = (hipEvent_t)before;
    g_kernel_after = (hipEvent_t)after;
    return TAPS_OK;
}

taps_status taps_enumerate_strategies(const taps_graph *graph, const taps_cluster *cluster,
                                      uint64_t *op_offsets, taps_strategy *strategies,
                                      uint64_t capacity, void *stream) {
    g_last_error.clear();
    taps_launch lp;
    taps_status st = check_cluster(cluster, &lp);
    if (st == TAPS_OK) st = check_graph(graph, false);
    if (st != TAPS_OK) return st;
    if (!op_offsets) return fail(TAPS_ERR_ARG, "op_offsets is NULL");
    return enumerate(graph, lp, 0xFFu, op_offsets, strategies, capacity, stream);
}

taps_status taps_enumerate_strategies_mesh(const taps_graph *graph, const taps_cluster *cluster,
                                           const taps_mesh *mesh, uint64_t *op_offsets,
                                           taps_strategy *strategies, uint64_t capacity,
                                           void *stream) {
    g_last_error.clear();
    taps_launch lp;
    taps_status st = check_cluster(cluster, &lp);
    if (st == TAPS_OK) st = check_graph(graph, false);
    if (st != TAPS_OK) return st;
    if (!op_offsets) return fail(TAPS_ERR_ARG, "op_offsets is NULL");
    uint32_t allowed = 0;
    if ((st = mesh_cuts(mesh, lp.n, &allowed)) != TAPS_OK) return st;
    return enumerate(graph, lp, allowed, op_offsets, strategies, capacity, stream);
}

taps_status taps_node_costs(const taps_graph *graph, const taps_cluster *cluster,
                            const taps_strategy *strategies, const uint64_t *op_offsets,
                            taps_table out, void *stream_) {
    g_last_error.clear();
    taps_launch lp;
    taps_status st = check_cluster(cluster, &lp);
    if (st == TAPS_OK) st = check_graph(graph, false);
    if (st == TAPS_OK) st = check_offsets(graph, op_offsets);
    if (st != TAPS_OK) return st;
    const uint32_t n_ops = graph->n_ops;
    const uint64_t total = op_offsets[n_ops];
    if (total == 0) return TAPS_OK;
    if (!strategies) return fail(TAPS_ERR_ARG, "strategies is NULL");
    if (!out.t || !out.vol || !out.intra || !out.inter || !out.meta)
        return fail(TAPS_ERR_ARG, "a table array is NULL");
    hipStream_t stream = (hipStream_t)stream_;
    call_scratch sc(stream);
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {op_offsets, sizeof(uint64_t) * (n_ops + 1), 0}};
    void *dev = nullptr;
    if ((st = upload(sc, ch, &dev)) != TAPS_OK) return st;
    taps_desc *d_desc = nullptr;
    if ((st = sc.alloc((void **)&d_desc, sizeof(taps_desc) * total)) != TAPS_OK) return st;
    hipError_t err = taps_launch_describe(strategies, total, d_desc, stream);
    if (err == hipSuccess)
        err = taps_launch_node_costs(at<taps_op>(dev, ch[0]), n_ops, at<uint64_t>(dev, ch[1]),
                                     d_desc, total, lp, out, stream);
    if (err != hipSuccess) return hip_fail(err, "node costs");
    return TAPS_OK;
}

taps_status taps_build_tables(const taps_graph *graph, const taps_cluster *cluster,
                              const taps_mesh *mesh, uint64_t *op_offsets,
                              taps_strategy *strategies, uint64_t strategy_capacity, taps_table node,
                              uint64_t *edge_offsets, taps_table edge, uint64_t edge_capacity,
                              uint32_t flags, void *stream) {
    return build_tables(graph, cluster, mesh, op_offsets, strategies, strategy_capacity, node,
                        edge_offsets, edge, edge_capacity, flags, stream, false);
}

taps_status taps_build_tables_noalloc(const taps_graph *graph, const taps_cluster *cluster,
                                      const taps_mesh *mesh, uint64_t *op_offsets,
                                      taps_strategy *strategies, uint64_t strategy_capacity,
                                      taps_table node, uint64_t *edge_offsets, taps_table edge,
                                      uint64_t edge_capacity, uint32_t flags, void *stream) {
    return build_tables(graph, cluster, mesh, op_offsets, strategies, strategy_capacity, node,
                        edge_offsets, edge, edge_capacity, flags, stream, true);
}

taps_status taps_node_costs_topology(const taps_graph *graph, const taps_topology *topology,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     taps_table out, void *stream_) {
    g_last_error.clear();
    taps_hier H;
    taps_cluster cl;
    taps_status st = check_topology(topology, &H, &cl);
    if (st == TAPS_OK) st = check_graph(graph, false);
    if (st == TAPS_OK) st = check_offsets(graph, op_offsets);
    if (st != TAPS_OK) return st;
    const uint32_t n_ops = graph->n_ops;
    const uint64_t total = op_offsets[n_ops];
    if (total == 0) return TAPS_OK;
    if (!strategies) return fail(TAPS_ERR_ARG, "strategies is NULL");
    if (!out.t || !out.vol || !out.intra || !out.inter || !out.meta)
        return fail(TAPS_ERR_ARG, "a table array is NULL");
    hipStream_t stream = (hipStream_t)stream_;
    call_scratch sc(stream);
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {op_offsets, sizeof(uint64_t) * (n_ops + 1), 0}};
    void *dev = nullptr;
    if ((st = upload(sc, ch, &dev)) != TAPS_OK) return st;
    taps_desc *d_desc = nullptr;
    if ((st = sc.alloc((void **)&d_desc, sizeof(taps_desc) * total)) != TAPS_OK) return st;
    hipError_t err = taps_launch_describe(strategies, total, d_desc, stream);
    if (err == hipSuccess)
        err = taps_launch_node_costs_h(at<taps_op>(dev, ch[0]), n_ops, at<uint64_t>(dev, ch[1]),
                                       d_desc, total, log2u(topology->domain[H.n_classes - 1]), H,
                                       out, stream);
    if (err != hipSuccess) return hip_fail(err, "node costs");
    return TAPS_OK;
}

taps_status taps_edge_costs_topology(const taps_graph *graph, const taps_topology *topology,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                     void *stream) {
    g_last_error.clear();
    taps_hier H;
    taps_cluster cl;
    const taps_status st = check_topology(topology, &H, &cl);
    if (st != TAPS_OK) return st;
    return edge_costs(graph, &cl, 1, strategies, op_offsets, edge_offsets, &out, capacity, stream,
                      false, false, &H);
}

taps_status taps_memory_costs(const taps_graph *graph, const taps_strategy *strategies,
                              const uint64_t *op_offsets, uint64_t *memory, void *stream_) {
    g_last_error.clear();
    taps_status st = check_graph(graph, false);
    if (st == TAPS_OK) st = check_offsets(graph, op_offsets);
    if (st != TAPS_OK) return st;
    const uint32_t n_ops = graph->n_ops;
    const uint64_t total = op_offsets[n_ops];
    if (total == 0) return TAPS_OK;
    if (!strategies) return fail(TAPS_ERR_ARG, "strategies is NULL");
    if (!memory) return fail(TAPS_ERR_ARG, "memory is NULL");
    hipStream_t stream = (hipStream_t)stream_;
    call_scratch sc(stream);
    std::vector<chunk> ch{{graph->ops, sizeof(taps_op) * n_ops, 0},
                          {op_offsets, sizeof(uint64_t) * (n_ops + 1), 0}};
    void *dev = nullptr;
    if ((st = upload(sc, ch, &dev)) != TAPS_OK) return st;
    const hipError_t err = taps_launch_memory_costs(at<taps_op>(dev, ch[0]), n_ops,
                                                    at<uint64_t>(dev, ch[1]), strategies, total,
                                                    memory, stream);
    if (err != hipSuccess) return hip_fail(err, "memory costs");
    return TAPS_OK;
}

taps_status taps_edge_costs(const taps_graph *graph, const taps_cluster *cluster,
                            const taps_strategy *strategies, const uint64_t *op_offsets,
                            uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                            void *stream) {
    return edge_costs(graph, cluster, 1, strategies, op_offsets, edge_offsets, &out, capacity,
                      stream, false, false);
}

taps_status taps_edge_costs_shared(const taps_graph *graph, const taps_cluster *cluster,
                                   const taps_strategy *strategies, const uint64_t *op_offsets,
                                   uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                   void *stream) {
    return edge_costs(graph, cluster, 1, strategies, op_offsets, edge_offsets, &out, capacity,
                      stream, true, false);
}

taps_status taps_edge_costs_backward(const taps_graph *graph, const taps_cluster *cluster,
                                     const taps_strategy *strategies, const uint64_t *op_offsets,
                                     uint64_t *edge_offsets, taps_table out, uint64_t capacity,
                                     void *stream) {
    return edge_costs(graph, cluster, 1, strategies, op_offsets, edge_offsets, &out, capacity,
                      stream, false, true);
}

taps_status taps_edge_costs_sweep(const taps_graph *graph, const taps_cluster *clusters,
                                  uint32_t n_points, const taps_strategy *strategies,
                                  const uint64_t *op_offsets, uint64_t *edge_offsets,
                                  const taps_table *out, uint64_t capacity, void *stream) {
    return edge_costs(graph, clusters, n_points, strategies, op_offsets, edge_offsets, out,
                      capacity, stream, false, false);
}

}  // extern "C"

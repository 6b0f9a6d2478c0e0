"""Seeded synthetic workloads: operator graphs and modeled clusters.

This module only *describes* inputs: operators with their axes, axis lengths,
which axes may be partitioned, element size and the tensors they read and
write, the edges between operators, and the modeled cluster (nodes x devices
per node, intra- and inter-node bandwidth).  It holds none of the cost model's
arithmetic, so both the HIP path and the CPU oracle can consume it.

The paper's problem statement (Overview section) takes a computation graph
G=(V,E) whose operators carry shapes and operator types, and a device graph
that gives the device count and the bandwidth between devices.  The
evaluation uses AlexNet and Megatron-LM graphs, which are not available here;
the transformer and MLP graphs below stand in for them with the shapes of the
configurations this library is measured on.

Every operator is an einsum-like contraction over named axes.  A tensor is a
tuple of op-axis indices (one per tensor dimension).  ``out`` is the produced
tensor, ``ins`` are activations (edge consumers attach to them by slot) and
``ws`` are weights (never fed by an edge).
"""
from __future__ import annotations

import json
import random
from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

GB = 10 ** 9

# Limits shared by every consumer of the description (they are input-format
# limits, not cost-model parameters).
MAX_AXES = 8
MAX_RANK = 8
MAX_INPUTS = 4
MAX_WEIGHTS = 4


@dataclass(frozen=True)
class Op:
    name: str
    kind: str
    axis_names: Tuple[str, ...]
    axis_len: Tuple[int, ...]
    partitionable: Tuple[bool, ...]
    dtype_bytes: int
    ins: Tuple[Tuple[int, ...], ...]
    ws: Tuple[Tuple[int, ...], ...]
    out: Tuple[int, ...]

    @property
    def n_axes(self) -> int:
        return len(self.axis_names)

    @property
    def part_mask(self) -> int:
        m = 0
        for a, p in enumerate(self.partitionable):
            if p:
                m |= 1 << a
        return m

    def check(self) -> None:
        assert 1 <= self.n_axes <= MAX_AXES
        assert len(self.axis_len) == self.n_axes == len(self.partitionable)
        assert len(self.ins) <= MAX_INPUTS and len(self.ws) <= MAX_WEIGHTS
        for t in (*self.ins, *self.ws, self.out):
            assert len(t) <= MAX_RANK
            assert len(set(t)) == len(t), "a tensor names each op axis at most once"
            assert all(0 <= a < self.n_axes for a in t)


@dataclass(frozen=True)
class Edge:
    src: int   # producing op: its ``out`` tensor
    dst: int   # consuming op
    slot: int  # index into the consumer's ``ins``


@dataclass
class Graph:
    ops: List[Op] = field(default_factory=list)
    edges: List[Edge] = field(default_factory=list)

    def add(self, op: Op) -> int:
        op.check()
        self.ops.append(op)
        return len(self.ops) - 1

    def connect(self, src: int, dst: int, slot: int) -> None:
        self.edges.append(Edge(src, dst, slot))


@dataclass(frozen=True)
class Cluster:
    nodes: int
    devices_per_node: int
    bw_intra: int  # bytes / s
    bw_inter: int  # bytes / s

    @property
    def devices(self) -> int:
        return self.nodes * self.devices_per_node


@dataclass(frozen=True)
class Topology:
    """A hierarchy of link classes (an extension of the paper's two classes):
    blocks of ``domains[c]`` consecutive device ranks, non-decreasing, the last
    one all devices.  Class 0 links join the devices of one domains[0] block (a
    node), class c >= 1 links join the domains[c-1] blocks of one domains[c]
    block, at ``bw[c]`` bytes/s each.  ``bw_a2a``: an AllToAll inside one
    domains[0] block moves at this rate (peer to peer over every link of the
    block, where a ring uses one); 0: bw[0]."""
    domains: Tuple[int, ...]
    bw: Tuple[int, ...]
    bw_a2a: int = 0

    @property
    def devices(self) -> int:
        return self.domains[-1]

    @staticmethod
    def of(cluster: Cluster) -> "Topology":
        """The paper's two classes: nodes of L devices inside the cluster."""
        return Topology((cluster.devices_per_node, cluster.devices),
                        (cluster.bw_intra, cluster.bw_inter))


@dataclass
class Workload:
    name: str
    graph: Graph
    clusters: List[Tuple[str, Cluster]]  # one table set per modeled cluster


# --------------------------------------------------------------------------
# Operator catalogue
# --------------------------------------------------------------------------

def matmul(name: str, b: int, k: int, o: int, dtype_bytes: int) -> Op:
    """Y(b,o) = X(b,k) W(k,o); all three axes partitionable (data parallel,
    row and column model parallel)."""
    return Op(name, "matmul", ("b", "k", "o"), (b, k, o), (True, True, True), dtype_bytes,
              ins=((0, 1),), ws=((1, 2),), out=(0, 2))


def elementwise(name: str, kind: str, names: Sequence[str], lens: Sequence[int], n_in: int,
                dtype_bytes: int) -> Op:
    full = tuple(range(len(names)))
    return Op(name, kind, tuple(names), tuple(lens), (True,) * len(names), dtype_bytes,
              ins=(full,) * n_in, ws=(), out=full)


def layernorm(name: str, b: int, s: int, h: int, dtype_bytes: int) -> Op:
    """Normalises over h, so h is kept whole; gamma and beta are weights over h."""
    return Op(name, "layernorm", ("b", "s", "h"), (b, s, h), (True, True, False), dtype_bytes,
              ins=((0, 1, 2),), ws=((2,), (2,)), out=(0, 1, 2))


def qkv_proj(name: str, b: int, s: int, h: int, n: int, d: int, dtype_bytes: int) -> Op:
    """Y(b,s,n,d) = X(b,s,h) W(h,n,d); the head dimension d is kept whole."""
    return Op(name, "proj_in", ("b", "s", "h", "n", "d"), (b, s, h, n, d),
              (True, True, True, True, False), dtype_bytes,
              ins=((0, 1, 2),), ws=((2, 3, 4),), out=(0, 1, 3, 4))


def attn_scores(name: str, b: int, n: int, s: int, d: int, dtype_bytes: int) -> Op:
    """S(b,n,s,t) = Q(b,s,n,d) K(b,t,n,d); the key axis t and head dim d are kept whole."""
    return Op(name, "scores", ("b", "n", "s", "t", "d"), (b, n, s, s, d),
              (True, True, True, False, False), dtype_bytes,
              ins=((0, 2, 1, 4), (0, 3, 1, 4)), ws=(), out=(0, 1, 2, 3))


def softmax(name: str, b: int, n: int, s: int, dtype_bytes: int) -> Op:
    """Softmax over the key axis t, which is kept whole."""
    return Op(name, "softmax", ("b", "n", "s", "t"), (b, n, s, s), (True, True, True, False),
              dtype_bytes, ins=((0, 1, 2, 3),), ws=(), out=(0, 1, 2, 3))


def attn_context(name: str, b: int, n: int, s: int, d: int, dtype_bytes: int) -> Op:
    """C(b,s,n,d) = P(b,n,s,t) V(b,t,n,d)."""
    return Op(name, "context", ("b", "n", "s", "t", "d"), (b, n, s, s, d),
              (True, True, True, False, False), dtype_bytes,
              ins=((0, 1, 2, 3), (0, 3, 1, 4)), ws=(), out=(0, 2, 1, 4))


def out_proj(name: str, b: int, s: int, n: int, d: int, h: int, dtype_bytes: int) -> Op:
    """Y(b,s,h) = C(b,s,n,d) W(n,d,h)."""
    return Op(name, "proj_out", ("b", "s", "n", "d", "h"), (b, s, n, d, h),
              (True, True, True, False, True), dtype_bytes,
              ins=((0, 1, 2, 3),), ws=((2, 3, 4),), out=(0, 1, 4))


def ffn(name: str, b: int, s: int, i: int, o: int, dtype_bytes: int) -> Op:
    """Y(b,s,o) = X(b,s,i) W(i,o)."""
    return Op(name, "ffn", ("b", "s", "i", "o"), (b, s, i, o), (True,) * 4, dtype_bytes,
              ins=((0, 1, 2),), ws=((2, 3),), out=(0, 1, 3))


# --------------------------------------------------------------------------
# Graphs
# --------------------------------------------------------------------------

def mlp2(batch: int = 64, d_in: int = 256, hidden: int = 1024, dtype_bytes: int = 4) -> Graph:
    """matmul -> gelu -> matmul."""
    g = Graph()
    m1 = g.add(matmul("mm1", batch, d_in, hidden, dtype_bytes))
    ge = g.add(elementwise("gelu", "gelu", ("b", "h"), (batch, hidden), 1, dtype_bytes))
    m2 = g.add(matmul("mm2", batch, hidden, d_in, dtype_bytes))
    g.connect(m1, ge, 0)
    g.connect(ge, m2, 0)
    return g


def gpt(layers: int, hidden: int, heads: int, seq: int, batch: int, dtype_bytes: int) -> Graph:
    """A GPT-style decoder stack: per layer layernorm, Q/K/V projections, attention
    scores, softmax, attention context, output projection, residual add,
    layernorm, two FFN matmuls with a GeLU between them, residual add.
    16 edges inside a layer plus 2 from the previous layer's output (into the
    first layernorm and the first residual add): 18*layers - 2 edges."""
    assert hidden % heads == 0
    d = hidden // heads
    b, s, h, f = batch, seq, hidden, 4 * hidden
    g = Graph()
    prev = None
    for l in range(layers):
        p = f"l{l}."
        ln1 = g.add(layernorm(p + "ln1", b, s, h, dtype_bytes))
        q = g.add(qkv_proj(p + "q", b, s, h, heads, d, dtype_bytes))
        k = g.add(qkv_proj(p + "k", b, s, h, heads, d, dtype_bytes))
        v = g.add(qkv_proj(p + "v", b, s, h, heads, d, dtype_bytes))
        sc = g.add(attn_scores(p + "scores", b, heads, s, d, dtype_bytes))
        sm = g.add(softmax(p + "softmax", b, heads, s, dtype_bytes))
        cx = g.add(attn_context(p + "context", b, heads, s, d, dtype_bytes))
        po = g.add(out_proj(p + "proj_out", b, s, heads, d, h, dtype_bytes))
        a1 = g.add(elementwise(p + "add1", "add", ("b", "s", "h"), (b, s, h), 2, dtype_bytes))
        ln2 = g.add(layernorm(p + "ln2", b, s, h, dtype_bytes))
        f1 = g.add(ffn(p + "ffn1", b, s, h, f, dtype_bytes))
        ge = g.add(elementwise(p + "gelu", "gelu", ("b", "s", "f"), (b, s, f), 1, dtype_bytes))
        f2 = g.add(ffn(p + "ffn2", b, s, f, h, dtype_bytes))
        a2 = g.add(elementwise(p + "add2", "add", ("b", "s", "h"), (b, s, h), 2, dtype_bytes))
        if prev is not None:
            g.connect(prev, ln1, 0)
            g.connect(prev, a1, 0)
        for x in (q, k, v):
            g.connect(ln1, x, 0)
        g.connect(q, sc, 0)
        g.connect(k, sc, 1)
        g.connect(sc, sm, 0)
        g.connect(sm, cx, 0)
        g.connect(v, cx, 1)
        g.connect(cx, po, 0)
        g.connect(po, a1, 1)
        g.connect(a1, ln2, 0)
        g.connect(a1, a2, 0)
        g.connect(ln2, f1, 0)
        g.connect(f1, ge, 0)
        g.connect(ge, f2, 0)
        g.connect(f2, a2, 1)
        prev = a2
    return g


MLP64_SEED = 230104285
MLP64_WIDTHS = (2048, 4096, 8192, 16384)


def mlp_stack(layers: int = 64, batch: int = 1024, dtype_bytes: int = 2,
              seed: int = MLP64_SEED) -> Graph:
    """``layers`` chained matmuls (batch, h_i, h_{i+1}); the widths h_0..h_layers are
    drawn from ``random.Random(seed).choice(MLP64_WIDTHS)``."""
    r = random.Random(seed)
    widths = [r.choice(MLP64_WIDTHS) for _ in range(layers + 1)]
    g = Graph()
    prev = None
    for l in range(layers):
        m = g.add(matmul(f"mm{l}", batch, widths[l], widths[l + 1], dtype_bytes))
        if prev is not None:
            g.connect(prev, m, 0)
        prev = m
    return g


def leading_ops(graph: Graph, n_ops: int) -> Graph:
    """The first `n_ops` operators of a graph and the edges among them (one transformer
    layer of `gpt` is its first 14 operators)."""
    return Graph(list(graph.ops[:n_ops]),
                 [e for e in graph.edges if e.src < n_ops and e.dst < n_ops])


# --------------------------------------------------------------------------
# The five measured configurations
# --------------------------------------------------------------------------

def config(index: int) -> Workload:
    """Workload ``index`` in 1..5 (see the module docstring)."""
    if index == 1:
        return Workload("mlp2-fp32-2x2", mlp2(),
                        [("2x2", Cluster(2, 2, 200 * GB, 25 * GB))])
    if index == 2:
        return Workload("gpt-4L-h1024-fp16-2x8", gpt(4, 1024, 16, 1024, 8, 2),
                        [("2x8", Cluster(2, 8, 400 * GB, 50 * GB))])
    if index == 3:
        return Workload("gpt-24L-h4096-bf16-32dev", gpt(24, 4096, 32, 2048, 16, 2),
                        [("4x8", Cluster(4, 8, 600 * GB, 100 * GB)),
                         ("2x16", Cluster(2, 16, 600 * GB, 100 * GB))])
    if index == 4:
        return Workload("mlp64-fp16-8x8", mlp_stack(),
                        [(f"8x8-inter{bw}", Cluster(8, 8, 600 * GB, int(bw * GB)))
                         for bw in (12.5, 25, 50, 100)])
    if index == 5:
        return Workload("gpt-96L-h12288-bf16-16x8", gpt(96, 12288, 96, 2048, 64, 2),
                        [("16x8", Cluster(16, 8, 600 * GB, 100 * GB))])
    raise ValueError(f"no configuration {index}")


ALL_CONFIGS = (1, 2, 3, 4, 5)

# Physical meshes of the configurations that name one (innermost dimension
# first: the 8 devices of a node, then the node grid).
CONFIG_MESHES = {4: (8, 4, 2), 5: (8, 4, 4)}


# Three link classes for the configurations with a 3-D mesh: 8 devices of a
# node (600 GB/s), 4 nodes of a group (the configuration's inter-node
# bandwidth, 50 GB/s for the wide MLP), and the groups above them at a quarter
# of that (a 4:1 oversubscribed tier).  The bandwidths of the upper tier are a
# choice: the workload list names the meshes, not their links.
CONFIG_TOPOLOGIES = {4: Topology((8, 32, 64), (600 * GB, 50 * GB, 12 * GB + GB // 2)),
                     5: Topology((8, 32, 128), (600 * GB, 100 * GB, 25 * GB))}


def physical_mesh(index: int, cluster: Cluster) -> Tuple[int, ...]:
    """The fixed device mesh of a configuration's cluster: the one the
    configuration names, else (devices per node, nodes) without sizes of 1."""
    if index in CONFIG_MESHES and math_prod(CONFIG_MESHES[index]) == cluster.devices:
        return CONFIG_MESHES[index]
    return tuple(m for m in (cluster.devices_per_node, cluster.nodes) if m > 1)


def math_prod(xs: Sequence[int]) -> int:
    out = 1
    for x in xs:
        out *= x
    return out


def random_graph(rng: random.Random, n_ops: int, max_axes: int = 5, max_rank: int = 4,
                 dtype_choices: Sequence[int] = (2, 4), len_pow_range=(0, 7)) -> Graph:
    """A random chain-with-branches graph for property tests: ops with random
    axes (lengths 2^k * odd), random partitionable masks (at least one axis
    partitionable), random tensors; each edge copies the producer's output
    axes into a fresh consumer input so that shapes agree."""
    g = Graph()
    for i in range(n_ops):
        if i == 0 or rng.random() < 0.2:
            n_axes = rng.randint(1, max_axes)
            lens = [(1 << rng.randint(*len_pow_range)) * rng.choice((1, 1, 3)) for _ in range(n_axes)]
            part = [rng.random() < 0.7 for _ in range(n_axes)]
            if not any(part):
                part[rng.randrange(n_axes)] = True
            out = tuple(sorted(rng.sample(range(n_axes), rng.randint(1, min(max_rank, n_axes)))))
            ins = (tuple(rng.sample(range(n_axes), rng.randint(1, min(max_rank, n_axes)))),)
            ws = (tuple(rng.sample(range(n_axes), rng.randint(1, min(max_rank, n_axes)))),)
            g.add(Op(f"op{i}", "rand", tuple(f"a{a}" for a in range(n_axes)), tuple(lens),
                     tuple(part), rng.choice(dtype_choices), ins=ins, ws=ws, out=out))
            continue
        src = rng.randrange(len(g.ops))
        so = g.ops[src]
        rank = len(so.out)
        extra = rng.randint(0, max(0, min(max_axes - rank, 2)))
        n_axes = rank + extra
        # consumer axes: the edge tensor's dims first (permuted), then extras
        perm = list(range(n_axes))
        rng.shuffle(perm)
        tensor_axes = tuple(perm[:rank])
        lens = [0] * n_axes
        for d, a in enumerate(tensor_axes):
            lens[a] = so.axis_len[so.out[d]]
        for a in perm[rank:]:
            lens[a] = (1 << rng.randint(*len_pow_range)) * rng.choice((1, 3))
        part = [rng.random() < 0.75 for _ in range(n_axes)]
        if not any(part):
            part[rng.randrange(n_axes)] = True
        out = tuple(sorted(rng.sample(range(n_axes), rng.randint(1, min(max_rank, n_axes)))))
        ws = (tuple(rng.sample(range(n_axes), rng.randint(1, min(max_rank, n_axes)))),) \
            if rng.random() < 0.6 else ()
        dst = g.add(Op(f"op{i}", "rand", tuple(f"a{a}" for a in range(n_axes)), tuple(lens),
                       tuple(part), so.dtype_bytes, ins=(tensor_axes,), ws=ws, out=out))
        g.connect(src, dst, 0)
    return g


# --------------------------------------------------------------------------
# JSON descriptions (graphs and clusters as plain data, integer bytes/s)
# --------------------------------------------------------------------------

def graph_to_dict(graph: Graph) -> dict:
    return {"ops": [{"name": op.name, "kind": op.kind, "axes": list(op.axis_names),
                     "lengths": list(op.axis_len), "partitionable": list(op.partitionable),
                     "dtype_bytes": op.dtype_bytes, "inputs": [list(t) for t in op.ins],
                     "weights": [list(t) for t in op.ws], "output": list(op.out)}
                    for op in graph.ops],
            "edges": [{"src": e.src, "dst": e.dst, "slot": e.slot} for e in graph.edges]}


def graph_from_dict(d: dict) -> Graph:
    g = Graph()
    for o in d["ops"]:
        g.add(Op(str(o["name"]), str(o["kind"]), tuple(o["axes"]),
                 tuple(int(x) for x in o["lengths"]), tuple(bool(x) for x in o["partitionable"]),
                 int(o["dtype_bytes"]), ins=tuple(tuple(int(a) for a in t) for t in o["inputs"]),
                 ws=tuple(tuple(int(a) for a in t) for t in o["weights"]),
                 out=tuple(int(a) for a in o["output"])))
    for e in d["edges"]:
        src, dst, slot = int(e["src"]), int(e["dst"]), int(e["slot"])
        if not (0 <= src < len(g.ops) and 0 <= dst < len(g.ops)):
            raise ValueError(f"edge {e} names an operator that does not exist")
        g.connect(src, dst, slot)
    return g


def cluster_to_dict(cluster: Cluster) -> dict:
    return {"nodes": cluster.nodes, "devices_per_node": cluster.devices_per_node,
            "bw_intra": cluster.bw_intra, "bw_inter": cluster.bw_inter}


def cluster_from_dict(d: dict) -> Cluster:
    return Cluster(int(d["nodes"]), int(d["devices_per_node"]), int(d["bw_intra"]),
                   int(d["bw_inter"]))


def workload_to_json(w: Workload) -> str:
    return json.dumps({"name": w.name, "graph": graph_to_dict(w.graph),
                       "clusters": [{"name": n, **cluster_to_dict(c)} for n, c in w.clusters]})


def workload_from_json(text: str) -> Workload:
    d = json.loads(text)
    return Workload(str(d["name"]), graph_from_dict(d["graph"]),
                    [(str(c["name"]), cluster_from_dict(c)) for c in d["clusters"]])


def main() -> int:
    import argparse
    ap = argparse.ArgumentParser(description="write a measured configuration as JSON")
    ap.add_argument("config", type=int, help="1..5")
    ap.add_argument("out", help="output file")
    args = ap.parse_args()
    with open(args.out, "w") as f:
        f.write(workload_to_json(config(args.config)))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())

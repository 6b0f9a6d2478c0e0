"""taps_build_tables_noalloc (the build with its device workspace in a fixed
per-GPU array, no allocation) against taps_build_tables, through the C ABI:
every strategy and every node and edge record identical, on two calls in a
row into the same fixed workspace, the second with a smaller graph, with and
without shared tables."""
import sys

import pytest

from paper_2301_04285_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _signed(t):
    import torch
    return {torch.uint64: lambda: t.view(torch.int64),
            torch.uint32: lambda: t.view(torch.int32)}.get(t.dtype, lambda: t)()


def _same(a, b):
    import torch
    return all(torch.equal(_signed(a[f]), _signed(b[f])) for f in ("t", "vol", "intra", "inter",
                                                                     "meta"))


@pytest.mark.parametrize("shared", [False, True])
def test_noalloc_build_equals_build_tables(shared):
    import numpy as np
    import torch
    from paper_2301_04285_amd import taps
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    taps.load()
    # the largest workload first, then a smaller one: the second call reuses the
    # array the first one filled
    for k in (5, 2):
        w = W.config(k)
        cname, cl = w.clusters[0]
        say(f"[gpu] noalloc {w.name}/{cname} shared={shared}: reference build")
        ref = taps.taps_build_tables(w.graph, cl, shared=shared)
        out = taps.taps_build_tables(w.graph, cl)        # tables of the right size
        for v in (*out.node.values(), *out.edge.values()):
            _signed(v).fill_(-1)
        out.strategies.fill_(0)
        torch.cuda.synchronize()
        say(f"[gpu] noalloc {w.name}/{cname} shared={shared}: fixed-workspace build")
        got = taps.taps_build_tables_noalloc(w.graph, cl, out, shared=shared)
        torch.cuda.synchronize()
        assert np.array_equal(got.op_offsets, ref.op_offsets)
        assert np.array_equal(got.edge_offsets, ref.edge_offsets)
        assert torch.equal(got.strategies, ref.strategies), w.name
        assert _same(got.node, ref.node), w.name
        assert _same(got.edge, ref.edge), w.name
        say(f"[gpu] noalloc {w.name}: {int(ref.edge_offsets[-1])} edge entries identical")
        del ref, out, got
        torch.cuda.empty_cache()

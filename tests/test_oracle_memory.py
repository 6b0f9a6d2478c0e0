"""The memory cost of a strategy (Eq. 18 sums it; the paper leaves it
undefined): per-device bytes of one shard of every weight and of the output.

Pinned against explicit devices: the device matrix of a strategy is built
from its positions and degrees, every rank's index sets of every tensor come
from the brute-force model (tests/bruteforce.py), and the bytes a rank holds
are counted from those sets -- no division formula involved.
"""
import random
from math import prod

import numpy as np

import bruteforce as BF
from oracle import oracle as O
from paper_2301_04285_amd import workloads as W


def _held_bytes(op, strat) -> int:
    """Bytes of the weights and the output that rank 0 holds, checked equal on every rank."""
    split = [a for a in range(op.n_axes) if strat["pos"][a] >= 0]
    D = [0] * len(split)
    for a in split:
        D[strat["pos"][a]] = int(strat["degree"][a])
    assert all(D) and prod(D) == prod(int(strat["degree"][a]) for a in split)
    total = None
    for t in (*op.ws, op.out):
        M = [int(strat["pos"][a]) if strat["pos"][a] >= 0 else -1 for a in t]
        shape = [op.axis_len[a] for a in t]
        held = BF.held_original(D, M, shape)
        counts = {prod(len(s) for s in dims) for dims in held}
        assert len(counts) == 1   # every rank holds the same amount
        total = (total or 0) + counts.pop() * op.dtype_bytes
    return total


def test_worked_examples():
    """mm1 of the 2-layer MLP (b 64, k 256, o 1024, fp32; weight (k, o), output (b, o)), by hand."""
    op = W.config(1).graph.ops[0]
    s = O.enumerate_strategies(op, 4)
    mem = O.memory_table(op, s)
    want = {(1, 1, 4): (256 * 1024 // 4 + 64 * 1024 // 4) * 4,
            (4, 1, 1): (256 * 1024 + 16 * 1024) * 4,
            (1, 4, 1): (64 * 1024 + 64 * 1024) * 4,     # k split: weight rows cut, output whole
            (2, 2, 1): (128 * 1024 + 32 * 1024) * 4}
    seen = set()
    for k, deg in enumerate(map(tuple, s["degree"][:, :3])):
        if deg in want:
            assert int(mem[k]) == want[deg], deg
            seen.add(deg)
    assert seen == set(want)


def test_one_device_holds_everything():
    for cfg in (1, 2, 4):
        for op in W.config(cfg).graph.ops:
            s = O.enumerate_strategies(op, 1)
            full = sum(prod(op.axis_len[a] for a in t) for t in (*op.ws, op.out)) * op.dtype_bytes
            assert len(s) == 1 and int(O.memory_table(op, s)[0]) == full


def test_matches_explicit_devices_on_the_workloads():
    for cfg, n_dev in ((1, 4), (2, 16)):
        g = W.config(cfg).graph
        for op in g.ops[:14]:
            s = O.enumerate_strategies(op, n_dev)
            mem = O.memory_table(op, s)
            for k in range(0, len(s), max(1, len(s) // 12)):
                assert int(mem[k]) == _held_bytes(op, s[k]), (op.name, k)


def test_matches_explicit_devices_on_random_operators():
    rng = random.Random(31)
    checked = 0
    while checked < 150:
        g = W.random_graph(rng, 1, max_axes=4, max_rank=3, len_pow_range=(1, 5))
        op = g.ops[0]
        s = O.enumerate_strategies(op, 1 << rng.randint(1, 5))
        if len(s) == 0:
            continue
        k = rng.randrange(len(s))
        assert int(O.memory_table(op, s[k:k + 1])[0]) == _held_bytes(op, s[k])
        checked += 1

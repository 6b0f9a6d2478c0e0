"""Graph and cluster descriptions as JSON, and table sets as .npz (plain arrays)."""
import numpy as np

from paper_2301_04285_amd import taps as T
from paper_2301_04285_amd import workloads as W


def test_workloads_round_trip_through_json():
    for k in range(1, 6):
        w = W.config(k)
        back = W.workload_from_json(W.workload_to_json(w))
        assert back.name == w.name
        assert back.graph.ops == w.graph.ops and back.graph.edges == w.graph.edges
        assert back.clusters == w.clusters


def test_json_graph_is_checked():
    import pytest
    d = W.graph_to_dict(W.mlp2())
    d["edges"].append({"src": 0, "dst": 9, "slot": 0})
    with pytest.raises(ValueError):
        W.graph_from_dict(d)
    d = W.graph_to_dict(W.mlp2())
    d["ops"][0]["output"] = [0, 7]
    with pytest.raises(AssertionError):
        W.graph_from_dict(d)


def test_tables_round_trip_through_npz(tmp_path):
    import torch
    rng = np.random.default_rng(5)
    offs = np.array([0, 3, 7], np.uint64)
    eoffs = np.array([0, 21], np.uint64)

    def table(n):
        return {"t": torch.from_numpy(rng.random(n)),
                "vol": torch.from_numpy(rng.integers(0, 2**63, n)).view(torch.uint64),
                "intra": torch.from_numpy(rng.integers(0, 2**63, n)).view(torch.uint64),
                "inter": torch.from_numpy(rng.integers(0, 2**63, n)).view(torch.uint64),
                "meta": torch.from_numpy(rng.integers(0, 2**31, n).astype(np.int32)).view(torch.uint32)}
    tabs = T.Tables(offs, torch.from_numpy(rng.integers(0, 255, (7, 16)).astype(np.uint8)),
                    table(7), eoffs, table(21))
    path = str(tmp_path / "tables.npz")
    T.save_tables(path, tabs)
    back = T.load_tables(path, device="cpu")
    assert np.array_equal(back.op_offsets, offs) and np.array_equal(back.edge_offsets, eoffs)
    assert torch.equal(back.strategies, tabs.strategies)
    for a, b in ((back.node, tabs.node), (back.edge, tabs.edge)):
        for f in T.TABLE_FIELDS:
            assert a[f].dtype == b[f].dtype
            assert torch.equal(a[f].view(torch.uint8), b[f].view(torch.uint8)), f

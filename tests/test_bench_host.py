"""Host-side logic of bench.py that needs no GPU: the split of captured steps
over HIP graphs under the kernel-node budget."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_graph_chunks_cover_every_step_once_within_budget():
    for first, count, nodes in [(0, 50, 129), (5, 50, 129), (0, 10, 2000), (3, 7, 16384), (0, 200, 161),
                                (0, 1, 1), (7, 33, 4100)]:
        chunks = bench.graph_chunks(first, count, nodes)
        steps = [f + i for f, c in chunks for i in range(c)]
        assert steps == list(range(first, first + count)), (first, count, nodes)
        assert all(c * nodes <= bench.MAX_GRAPH_NODES for _, c in chunks)


def test_graph_chunks_edges():
    assert bench.graph_chunks(0, 0, 129) == []
    assert bench.graph_chunks(0, 50, 129) == [(0, 50)]                  # the 8B decode step: one graph
    assert bench.graph_chunks(0, 10, 2000) == [(0, 8), (8, 2)]
    # a step beyond the budget (the old 1-bit 512-token step: 141 calls x 128 launches) runs eagerly
    assert bench.graph_chunks(0, 10, 141 * 128) is None
    assert bench.graph_chunks(0, 3, bench.MAX_GRAPH_NODES) == [(0, 1), (1, 1), (2, 1)]

"""Host-only checks of the benchmark's algorithmic-work helpers, which the reported roofline
fractions divide by: the level-query rows of the matrix-weight forward and the block-tree nodes the
tile kernel reads, each against a brute-force count from the oracle's Fenwick levels."""

import numpy as np
import pytest

import bench
from oracle import fenwick


@pytest.mark.parametrize("T,R", [(128, 128), (512, 128), (1000, 64), (4096, 128)])
def test_lq_level_rows_counts_distinct_levels_per_row(T, R):
    # each row scores its pairs at the distinct Fenwick levels of its own row
    brute = sum(len(set(fenwick.level_row(t).tolist())) for t in range(T))
    assert bench.lq_level_rows(T, R) == brute


def _tree_nodes_brute(N):
    """Distinct block-tree nodes (tile levels j >= 4, blocks of 4 tiles) some tile reads."""
    nodes = set()
    for u in range(N):
        for j in range(4, max(N - 1, 1).bit_length() + 1):
            if (u >> (j - 1)) & 1:
                first = ((u >> (j - 1)) - 1) << (j - 1)   # first tile of the source group
                l = j - 3                                  # tree level above the blocks
                nodes.add((l, (first // 4) >> l))
    return len(nodes)


@pytest.mark.parametrize("N", [1, 7, 8, 9, 16, 17, 33, 100, 512, 1000])
def test_tree_nodes_read_matches_brute_force(N):
    assert bench.tree_nodes_read(N) == _tree_nodes_brute(N)

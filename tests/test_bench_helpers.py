"""Host-only checks of the benchmark's algorithmic-work helpers, which the reported roofline
fractions divide by: the level-query rows of the matrix-weight forward and the block-tree nodes the
tile kernel reads, each against a brute-force count from the oracle's Fenwick levels; and the rule
that a committed counter record is used only for the workload and kernel sources it was taken on."""

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


def test_recorded_traffic_follows_workload_and_source_hash(tmp_path):
    """The counter record is used only for its own workload and for the sources it was measured on."""
    sources = ["paper_2506_04761_amd/csrc/ll_gdn.hip", "paper_2506_04761_amd/csrc/ll_device.hpp"]
    h = bench.kernel_source_hash(sources)
    assert h != bench.kernel_source_hash()  # different source sets hash differently

    def record(workload, digest):
        f = tmp_path / f"rec_{workload}_{digest}.md"
        f.write_text("# counters\n\n- workload: `%s`\n- kernel_source_sha256: `%s`\n"
                     "- hbm_bytes_per_launch: `12345`\n" % (workload, digest))
        return str(f)

    assert bench.recorded_traffic("w1", record("w1", h), sources) == 12345.0
    assert bench.recorded_traffic("w2", record("w1", h), sources) is None
    assert bench.recorded_traffic("w1", record("w1", "0" * 16), sources) is None
    assert bench.recorded_traffic("w1", str(tmp_path / "missing.md"), sources) is None

"""Pins for the oracle's Fenwick partition (Sec. 3.1 footnote) against things other than itself:
the worked example printed after Eq. 4, the XOR closed form, the stated bucket invariants,
and the decoding recurrence of Sec. 3.2 run as an independent algorithm on position sets."""

import math
import os

import numpy as np
import pytest

from oracle import fenwick

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example_levels_T8.txt")


def _load_golden():
    rows = [ln.split() for ln in open(GOLDEN) if ln.strip() and not ln.lstrip().startswith("#")]
    return np.array(rows, dtype=np.int64)


def test_worked_example_T8():
    # Sec. 3.1, the 8x8 hierarchical matrix after Eq. 4 (0-indexed positions).
    np.testing.assert_array_equal(fenwick.level_matrix(8), _load_golden())


def test_one_indexing_would_fail_worked_example():
    # The example fixes the indexing: running the greedy sequence on 1-based positions
    # (t+1, s+1) gives different levels, so a 1-indexed oracle cannot pass the pin above.
    golden = _load_golden()
    shifted = np.full((8, 8), -1)
    for t in range(8):
        for s in range(t + 1):
            shifted[t, s] = ((t + 1) ^ (s + 1)).bit_length()
    assert not np.array_equal(shifted, golden)


def test_greedy_equals_xor_closed_form_T4096():
    T = 4096
    lev = fenwick.level_matrix(T)
    t = np.arange(T)[:, None]
    s = np.arange(T)[None, :]
    x = t ^ s
    bitlen = np.where(x > 0, np.floor(np.log2(np.maximum(x, 1))).astype(np.int64) + 1, 0)
    expect = np.where(s <= t, bitlen, -1)
    np.testing.assert_array_equal(lev, expect)


@pytest.mark.parametrize("t", list(range(0, 300)) + [511, 512, 513, 1023, 1024, 4095, 4096, 65535])
def test_bucket_invariants(t):
    bk = fenwick.buckets(t)
    # sentinel bucket {t}
    assert bk[0] == [t]
    # |B^(l)| = 2^(l-1) for l >= 1 (sentence after the footnote)
    for lv, members in bk.items():
        if lv >= 1:
            assert len(members) == 2 ** (lv - 1)
            assert members == list(range(members[0], members[0] + len(members)))
    # disjoint and covering [0, t]
    allpos = sorted(p for m in bk.values() for p in m)
    assert allpos == list(range(t + 1))
    # one bucket per set bit of t, plus the sentinel
    assert len(bk) == bin(t).count("1") + 1
    # the top level is the bit length of t: one more level at each power of two (Sec. 3.2)
    assert max(bk) == t.bit_length()


def test_decoding_recurrence_reproduces_buckets():
    """Sec. 3.2: level 0 takes the new token; levels 1..lssb(t) empty; level lssb(t)+1 takes
    the union of levels 0..lssb(t) of step t-1; higher levels carry over.  Run on sets of
    positions, this independent algorithm must give the footnote's buckets at every t."""
    T = 1100
    state = {0: {0}}
    for t in range(T):
        if t > 0:
            p = fenwick.lssb(t)
            merged = set()
            for lv in range(p + 1):
                merged |= state.get(lv, set())
            new = {lv: s for lv, s in state.items() if lv > p + 1}
            assert not state.get(p + 1)  # level p+1 is always empty at t-1
            new[p + 1] = merged
            new[0] = {t}
            state = new
        greedy = {lv: set(m) for lv, m in fenwick.buckets(t).items()}
        assert {lv: s for lv, s in state.items() if s} == greedy


@pytest.mark.parametrize("C", [1, 2, 4, 8, 16, 64])
def test_chunk_levels_split_at_log2C(C):
    # Sec. 3.3 (Eq. 5): levels below l_C = log2(C)+1 stay inside a chunk; pairs in different
    # aligned chunks have level >= l_C, equal to log2(C) + bit_length(chunk(t) XOR chunk(s)).
    T = 256
    lev = fenwick.level_matrix(T)
    lc = int(math.log2(C)) + 1
    for t in range(T):
        for s in range(t + 1):
            if t // C == s // C:
                assert lev[t, s] < lc
            else:
                assert lev[t, s] == lc - 1 + ((t // C) ^ (s // C)).bit_length()


def test_num_levels():
    for T in range(1, 600):
        lev = fenwick.level_matrix(T)
        assert fenwick.num_levels(T) == lev.max() + 1
        assert fenwick.num_levels(T) == (1 if T == 1 else math.ceil(math.log2(T)) + 1)
    # the level counts the five benchmark workloads state
    assert [fenwick.num_levels(T) for T in (64, 2048, 8192, 65536)] == [7, 12, 14, 17]

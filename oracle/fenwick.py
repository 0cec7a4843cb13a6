"""Fenwick-tree bucket partition of a prefix and the level function l(t, s).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper: Sec. 3.1 ("Fenwick Tree Partitioning and Hierarchical Matrices"), the footnote that
defines lssb and the greedy bucket sequence b_t^(i), and the sentence after it (bucket
sizes 2^(l-1), sentinel bucket of size one).  Positions are 0-indexed, which is what the
worked 8x8 hierarchical matrix printed after Eq. 4 uses.

Everything here follows the footnote's greedy procedure literally.  The closed form
l(t, s) = bit_length(t XOR s) is NOT used by the oracle; the tests check the greedy
procedure against it, against the worked example, and against the decoding recurrence
of Sec. 3.2.
"""

import numpy as np


def lssb(t: int) -> int:
    """Index of the least significant set bit of t >= 1 (Sec. 3.1 footnote):
    the largest l such that 2**l divides t."""
    if t < 1:
        raise ValueError("lssb is defined for t >= 1")
    l = 0
    while t % 2 == 0:
        t //= 2
        l += 1
    return l


def greedy_boundaries(t: int) -> list:
    """The footnote's sequence b_t^(0) = t, b_t^(i) = b_t^(i-1) - 2**lssb(b_t^(i-1)),
    continued until it reaches 0 (the prefix [0, t) is then exhausted)."""
    b = [t]
    while b[-1] > 0:
        b.append(b[-1] - 2 ** lssb(b[-1]))
    return b


def buckets(t: int) -> dict:
    """Bucket partition of the positions 0..t as seen from time t (Sec. 3.1 footnote).

    Returns {level: sorted list of positions}.  Level 0 is the sentinel bucket {t};
    for each consecutive pair b^(i) > b^(i+1) of the greedy sequence the bucket
    {b^(i+1), ..., b^(i) - 1} gets level lssb(b^(i)) + 1.  Empty levels are omitted.
    """
    out = {0: [t]}
    b = greedy_boundaries(t)
    for i in range(len(b) - 1):
        level = lssb(b[i]) + 1
        if level in out:  # the footnote's levels are distinct by construction
            raise AssertionError("two buckets share a level")
        out[level] = list(range(b[i + 1], b[i]))
    return out


def level_row(t: int) -> np.ndarray:
    """Levels l(t, s) for s = 0..t as an int array of length t + 1 (Eq. 4's l(t, s))."""
    row = np.empty(t + 1, dtype=np.int64)
    row[t] = 0
    b = greedy_boundaries(t)
    for i in range(len(b) - 1):
        row[b[i + 1]:b[i]] = lssb(b[i]) + 1
    return row


def level_of(t: int, s: int) -> int:
    """l(t, s) for one pair s <= t: the level of the greedy bucket of t that holds s."""
    if not 0 <= s <= t:
        raise ValueError("need 0 <= s <= t")
    if s == t:
        return 0
    b = greedy_boundaries(t)
    for i in range(len(b) - 1):
        if b[i + 1] <= s < b[i]:
            return lssb(b[i]) + 1
    raise AssertionError("the buckets of t cover 0..t-1")


def level_col(s: int, T: int) -> np.ndarray:
    """Levels l(t, s) for t = s .. T-1 (one column of Eq. 4's level pattern)."""
    return np.array([level_of(t, s) for t in range(s, T)], dtype=np.int64)


def level_matrix(T: int) -> np.ndarray:
    """T x T int matrix with l(t, s) for s <= t and -1 above the diagonal."""
    out = np.full((T, T), -1, dtype=np.int64)
    for t in range(T):
        out[t, :t + 1] = level_row(t)
    return out


def num_levels(T: int) -> int:
    """Number of levels L the parallel form needs for length T: one more than the
    largest level any pair (t, s), s <= t < T, can take.

    The largest level occurs for t = T - 1, s = 0: the greedy sequence of T - 1 starts
    with its lowest set bit and ends with its highest, so the top level is the bit
    length of T - 1.  This gives L = ceil(log2 T) + 1 for T >= 2 and L = 1 for T = 1
    (the paper's listing sizes lambda as log2(length) + 1 levels; the footnote's
    "up to ceil(log2 t + 1) + 1" is a looser bound).
    """
    if T < 1:
        raise ValueError("T must be >= 1")
    if T == 1:
        return 1
    return int(max(level_row(T - 1))) + 1

"""Pins the oracle's relevance-keyed bank shrink (Sec. 5; Sec. 7.5, Tables
5-6) to things other than itself.

Selection is checked against Python's `sorted` with a key built from float
semantics (not from bit patterns), and, for small banks, against a set
definition found by brute force: the kept set is the only set of `keep`
entries each of which ranks before every entry left out.  The gather is
checked against direct slicing, and the keep count against the frames that
Table 6 lists per retained fraction.
"""
import itertools
import math
import os

from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_table6_keep.txt")


def rank_key(scores, i):
    """Ranking key: numbers by value, -0.0 before +0.0, NaN after all
    numbers, then the index."""
    x = float(scores[i])
    if math.isnan(x):
        return (1, 0.0, 0, i)
    return (0, x, 0 if math.copysign(1.0, x) < 0 else 1, i)


def py_select(scores, keep):
    order = sorted(range(len(scores)), key=lambda i: rank_key(scores, i))
    return sorted(order[:keep])


def tricky_scores(rng, n):
    pool = np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45, 2.5, 2.5, 3.0e38],
                    dtype=np.float32)
    a = rng.normal(size=n).astype(np.float32)
    m = rng.random(n) < 0.4
    a[m] = rng.choice(pool, size=int(m.sum()))
    return a


def test_select_against_python_sort(orc):
    rng = np.random.default_rng(61)
    for trial in range(60):
        n = int(rng.integers(0, 300))
        s = tricky_scores(rng, n)
        if trial % 5 == 0 and n:
            s[:] = s[0]                   # every score equal: the first `keep` indices
        for keep in sorted({0, n, n // 2, int(rng.integers(0, n + 1))}):
            got = orc.bank_select(s, keep).tolist()
            assert got == py_select(s, keep), (trial, n, keep)


def test_select_set_definition_small(orc):
    rng = np.random.default_rng(62)
    vals = np.array([0.0, -0.0, 1.0, np.nan, -2.0, 1.0], dtype=np.float32)
    for trial in range(40):
        n = int(rng.integers(1, 8))
        s = rng.choice(vals, size=n).astype(np.float32)
        for keep in range(n + 1):
            keys = [rank_key(s, i) for i in range(n)]
            good = [set(c) for c in itertools.combinations(range(n), keep)
                    if all(keys[i] < keys[j] for i in c for j in range(n) if j not in c)]
            assert len(good) == 1
            assert set(orc.bank_select(s, keep).tolist()) == good[0]
            assert orc.bank_select(s, keep).tolist() == sorted(good[0])


def test_special_cases(orc):
    assert orc.bank_select(np.zeros(0, dtype=np.float32), 0).size == 0
    s = np.array([5, 4, 3, 2, 1], dtype=np.float32)
    assert orc.bank_select(s, 5).tolist() == [0, 1, 2, 3, 4]
    assert orc.bank_select(s, 1).tolist() == [4]
    assert orc.bank_select(np.array([np.nan, 7, np.nan], dtype=np.float32), 2).tolist() == [0, 1]
    assert orc.bank_select(np.array([0.0, -0.0], dtype=np.float32), 1).tolist() == [1]
    with pytest.raises(ValueError):
        orc.bank_select(s, 6)


def test_shrink_gathers_kept_entries_in_index_order(orc):
    rng = np.random.default_rng(63)
    n = 37
    sizes = [1, 28, 4096, 4100, 16 * 60 * 104 * 2]
    parts = [(rng.integers(0, 256, size=n * eb, dtype=np.uint8), eb) for eb in sizes]
    s = tricky_scores(rng, n)
    for keep in [0, 1, 5, 36, 37]:
        kept, out = orc.bank_shrink(parts, s, keep)
        assert kept.tolist() == py_select(s, keep)
        for (data, eb), o in zip(parts, out):
            want = b"".join(data[i * eb:(i + 1) * eb].tobytes() for i in kept.tolist())
            assert o.tobytes() == want


def test_keep_count_against_table6(orc):
    import paper_2607_21686_amd as P
    rows = [l.split("#")[0].split() for l in open(GOLDEN)]
    rows = [r for r in rows if r]
    assert rows[0][0] == "bank"
    n = int(rows[0][1])
    for frac, kept in rows[1:]:
        assert orc.keep_count(float(frac), n) == int(kept), frac
        assert P.keep_count(float(frac), n) == int(kept), frac
    rng = np.random.default_rng(64)
    for _ in range(500):
        f, m = float(rng.random()), int(rng.integers(0, 5000))
        assert P.keep_count(f, m) == orc.keep_count(f, m)
    for _ in range(500):  # exact decimals with two digits: many products land on a half
        f, m = "0.%02d" % rng.integers(0, 100), int(rng.integers(0, 400))
        assert P.keep_count(f, m) == orc.keep_count(f, m)
    assert orc.keep_count(0.5, 0) == 0 and orc.keep_count(0.0, 9) == 1 and orc.keep_count(1.0, 9) == 9
    assert P.keep_count(0.5, 0) == 0 and P.keep_count(0.0, 9) == 1 and P.keep_count(1.0, 9) == 9


# Products that land exactly on a half, computed by hand from the decimal
# fraction (the binary float nearest 0.05 is slightly above it, so rounding
# that value instead would give 3 for (0.05, 50)): a tie goes to the even
# neighbour.
EXACT_HALVES = [(0.05, 50, 2), (0.3, 5, 2), (0.5, 21, 10), (0.1, 25, 2), (0.7, 5, 4), (0.5, 1, 1),
                (0.5, 3, 2), (0.5, 5, 2), (0.25, 10, 2), (0.25, 14, 4), (0.12, 25, 3), ("0.125", 4, 1),
                ("0.125", 12, 2), ((1, 3), 3, 1), ((1, 2), 7, 4)]


def test_keep_count_exact_halves(orc):
    import paper_2607_21686_amd as P
    for f, n, want in EXACT_HALVES:
        assert orc.keep_count(f if not isinstance(f, tuple) else Fraction(*f), n) == want, (f, n)
        assert P.keep_count(f, n) == want, (f, n)
    # The decimal reading, not the binary one: a float and its decimal string agree.
    for f in (0.05, 0.3, 0.1, 0.7, 0.12):
        for n in range(0, 200):
            assert P.keep_count(f, n) == P.keep_count(repr(f), n) == orc.keep_count(repr(f), n)


def test_keep_count_rejects_bad_fractions(orc):
    import paper_2607_21686_amd as P
    for bad in ((3, 2), (1, 0)):
        with pytest.raises(P.PcsError):
            P.keep_count(bad, 10)
    with pytest.raises(ValueError):
        orc.keep_count(1.5, 10)

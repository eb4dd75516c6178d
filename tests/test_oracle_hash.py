"""Pins the oracle's XXH64, chunking and Merkle root to things other than itself.

XXH64 is checked against the independent `xxhash` library (a separate
implementation of the xxHash specification); the Merkle root is checked
against a recursive split definition and closed forms.
"""
import struct

import numpy as np
import pytest
import xxhash

EMPTY_XXH64 = 0xEF46DB3751D8E999  # XXH64 of the empty input, seed 0 (xxHash reference value)


def lib_xxh64(b, seed=0):
    return xxhash.xxh64_intdigest(bytes(b), seed)


def test_xxh64_empty(orc):
    assert orc.xxh64(b"") == EMPTY_XXH64 == lib_xxh64(b"")


@pytest.mark.parametrize("seed", [0, 1, 0x9E3779B185EBCA87, (1 << 64) - 1])
def test_xxh64_all_short_lengths(orc, seed):
    rng = np.random.default_rng(seed % 1000)
    data = rng.integers(0, 256, size=400, dtype=np.uint8).tobytes()
    for n in range(0, 301):
        assert orc.xxh64(data[:n], seed) == lib_xxh64(data[:n], seed), n


def test_xxh64_chunk_boundaries_and_random(orc):
    rng = np.random.default_rng(11)
    for n in [4095, 4096, 4097, 8191, 8192, 12289, 65536 + 17, 1 << 20]:
        d = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        assert orc.xxh64(d) == lib_xxh64(d), n
    for _ in range(200):
        n = int(rng.integers(0, 5000))
        s = int(rng.integers(0, 1 << 63))
        d = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        assert orc.xxh64(d, s) == lib_xxh64(d, s)


def test_xxh64_structured_inputs(orc):
    # All-zero, all-0xFF and counting patterns exercise carries in every step.
    for n in [0, 1, 3, 4, 7, 8, 15, 16, 31, 32, 33, 63, 64, 4096]:
        for fill in [b"\x00", b"\xff"]:
            assert orc.xxh64(fill * n) == lib_xxh64(fill * n)
        cnt = bytes(i & 0xFF for i in range(n))
        assert orc.xxh64(cnt) == lib_xxh64(cnt)


@pytest.mark.parametrize("n", [0, 1, 16, 4095, 4096, 4097, 3 * 4096 + 5, 10 * 4096])
def test_chunk_hashes_are_xxh64_of_slices(orc, n):
    d = np.random.default_rng(n).integers(0, 256, size=n, dtype=np.uint8)
    got = orc.chunk_hashes(d)
    want = [lib_xxh64(d[s:s + 4096].tobytes()) for s in range(0, n, 4096)]
    assert orc.chunk_count(n) == len(want) == (n + 4095) // 4096
    assert [int(x) for x in got] == want


def node(l, r):
    return lib_xxh64(struct.pack("<QQ", l, r))


def split_root(leaves):
    """Recursive definition: split at the largest power of two below n."""
    n = len(leaves)
    if n == 0:
        return lib_xxh64(b"")
    if n == 1:
        return leaves[0]
    k = 1
    while k * 2 < n:
        k *= 2
    return node(split_root(leaves[:k]), split_root(leaves[k:]))


def test_node_hash_closed_form(orc):
    rng = np.random.default_rng(5)
    for _ in range(100):
        l, r = (int(x) for x in rng.integers(0, 1 << 63, size=2, dtype=np.uint64))
        l |= int(rng.integers(0, 2)) << 63
        assert orc.node_hash(l, r) == node(l, r)


def test_merkle_small_closed_forms(orc):
    assert orc.merkle_root([]) == EMPTY_XXH64
    assert orc.merkle_root([123456789]) == 123456789
    assert orc.merkle_root([5, 7]) == node(5, 7)
    assert orc.merkle_root([5, 7, 9]) == node(node(5, 7), 9)
    assert orc.merkle_root([1, 2, 3, 4, 5]) == node(node(node(1, 2), node(3, 4)), 5)


def test_merkle_matches_recursive_split(orc):
    rng = np.random.default_rng(6)
    sizes = list(range(1, 300)) + [511, 512, 513, 1023, 1024, 1025, 2047, 2048, 4097]
    for n in sizes:
        leaves = [int(x) for x in rng.integers(0, 1 << 63, size=n, dtype=np.uint64)]
        assert orc.merkle_root(leaves) == split_root(leaves), n


def test_merkle_aligned_groups_reduce_independently(orc):
    # The promote-odd tree splits into aligned groups of 64 leaves: the root
    # over the per-group roots equals the root over all leaves.
    rng = np.random.default_rng(7)
    for n in [1, 63, 64, 65, 127, 128, 129, 4095, 4096, 4097, 64 * 64 + 1]:
        leaves = rng.integers(0, 1 << 63, size=n, dtype=np.uint64)
        groups = [orc.merkle_root(leaves[s:s + 64]) for s in range(0, n, 64)]
        assert orc.merkle_root(groups) == orc.merkle_root(leaves)


def test_fingerprint_session_root(orc):
    rng = np.random.default_rng(8)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in [0, 16, 4096, 9000]]
    hashes, roots, sroot = orc.fingerprint(bufs)
    assert hashes.size == 0 + 1 + 1 + 3
    assert int(roots[0]) == EMPTY_XXH64
    assert int(roots[1]) == lib_xxh64(bufs[1].tobytes())
    assert int(roots[2]) == lib_xxh64(bufs[2].tobytes())
    parts = [lib_xxh64(bufs[3][s:s + 4096].tobytes()) for s in range(0, 9000, 4096)]
    assert int(roots[3]) == split_root(parts)
    assert sroot == split_root([int(r) for r in roots])

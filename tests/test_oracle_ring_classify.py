"""Pins the oracle's ring window and cross-replay classification.

Ring: against numpy's wrap-around indexing (np.take(mode='wrap') / np.roll).
Classify: against a direct byte comparison of the chunks, and against the
generator's own record of which chunks it rewrote.
"""
import numpy as np
import pytest

import workloads as W


def np_window(ring_bytes, g):
    a = np.zeros(g.outer * g.capacity * g.row_bytes, dtype=np.uint8)
    for o in range(g.outer):
        a[o * g.capacity * g.row_bytes:(o + 1) * g.capacity * g.row_bytes] = \
            ring_bytes[o * g.outer_stride:o * g.outer_stride + g.capacity * g.row_bytes]
    a = a.reshape(g.outer, g.capacity, g.row_bytes)
    return np.take(a, np.arange(g.head, g.head + g.window), axis=1, mode="wrap").reshape(-1)


@pytest.mark.parametrize("outer,cap,row,win,head,pad", [
    (1, 8, 16, 8, 0, 0), (1, 8, 16, 5, 6, 0), (3, 10, 32, 7, 9, 48), (4, 64, 2048, 40, 60, 0),
    (2, 16, 48, 1, 15, 16), (2, 16, 48, 16, 3, 0), (5, 7, 4096, 6, 4, 4096)])
def test_ring_window_matches_numpy(orc, outer, cap, row, win, head, pad):
    g = W.Ring(outer, cap, row, win, head, cap * row + pad)
    data = np.random.default_rng(cap).integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    got = orc.ring_window(data, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)
    assert np.array_equal(got, np_window(data, g))
    # numpy.roll form of the same statement, for the first ring.
    r0 = data[:cap * row].reshape(cap, row)
    assert np.array_equal(got[:win * row].reshape(win, row), np.roll(r0, -head, axis=0)[:win])


def test_ring_place_inverts_window_and_leaves_the_rest(orc):
    g = W.Ring(3, 12, 32, 7, 10, 12 * 32 + 32)
    rng = np.random.default_rng(1)
    logical = rng.integers(0, 256, size=g.window_bytes, dtype=np.uint8)
    for h2 in range(g.capacity):
        dst = np.full(g.ring_bytes, 0xA5, dtype=np.uint8)
        orc.ring_place(logical, dst, g.outer, g.outer_stride, g.capacity, g.row_bytes, h2, g.window)
        back = orc.ring_window(dst, g.outer, g.outer_stride, g.capacity, g.row_bytes, h2, g.window)
        assert np.array_equal(back, logical)
        # Every byte outside the window rows is untouched.
        touched = np.zeros(g.ring_bytes, dtype=bool)
        for o in range(g.outer):
            for t in range(g.window):
                s = o * g.outer_stride + ((h2 + t) % g.capacity) * g.row_bytes
                touched[s:s + g.row_bytes] = True
        assert np.all(dst[~touched] == 0xA5)


def brute_classify(replays):
    """replays[k][b] = bytes; compares chunks directly."""
    K, nb = len(replays), len(replays[0])
    bitmap, labels = [], []
    for b in range(nb):
        n = replays[0][b].size
        nch = (n + 4095) // 4096
        words = [0] * ((nch + 63) // 64)
        lab = 0
        for i in range(nch):
            ref = replays[0][b][4096 * i:4096 * (i + 1)].tobytes()
            if any(replays[k][b][4096 * i:4096 * (i + 1)].tobytes() != ref for k in range(1, K)):
                words[i // 64] |= 1 << (i % 64)
                lab = 1
        bitmap += words
        labels.append(lab)
    return np.array(bitmap, dtype=np.uint64), np.array(labels, dtype=np.uint8)


def oracle_classify(orc, replays):
    hs = np.stack([np.concatenate([orc.chunk_hashes(b) for b in rep]) for rep in replays])
    cpb = [orc.chunk_count(b.size) for b in replays[0]]
    return orc.classify(hs, cpb)


def test_classify_matches_byte_comparison(orc):
    rng = np.random.default_rng(2)
    for trial in range(20):
        K = int(rng.integers(1, 5))
        sizes = [int(rng.integers(0, 70 * 4096)) for _ in range(int(rng.integers(1, 6)))]
        base = [rng.integers(0, 256, size=s, dtype=np.uint8) for s in sizes]
        replays = [base]
        for _ in range(K - 1):
            rep = []
            for a in base:
                a = a.copy()
                if a.size and rng.random() < 0.5:
                    for _ in range(int(rng.integers(1, 4))):
                        a[int(rng.integers(0, a.size))] ^= np.uint8(1 << int(rng.integers(0, 8)))
                rep.append(a)
            replays.append(rep)
        bm, lab = oracle_classify(orc, replays)
        bm2, lab2 = brute_classify(replays)
        assert np.array_equal(bm, bm2) and np.array_equal(lab, lab2)


def test_classify_bitmap_layout(orc):
    # Buffer 0: 3 chunks, buffer 1: 65 chunks, buffer 2: empty, buffer 3: 1 chunk.
    cpb = [3, 65, 0, 1]
    total = sum(cpb)
    h = np.zeros((2, total), dtype=np.uint64)
    h[1, 2] = 1        # buffer 0 chunk 2
    h[1, 3 + 64] = 1   # buffer 1 chunk 64 -> its second word, bit 0
    bm, lab = orc.classify(h, cpb)
    assert bm.tolist() == [1 << 2, 0, 1, 0]
    assert lab.tolist() == [1, 1, 0, 0]
    # K = 1: nothing can differ.
    bm1, lab1 = orc.classify(h[:1], cpb)
    assert not bm1.any() and not lab1.any()


def test_config1_labels(orc):
    c = W.config1(0)
    bm, lab = oracle_classify(orc, [c.buffers(1), c.buffers(2)])
    assert lab.tolist() == [0, 1, 0, 0, 0, 0, 0, 0]   # only the RNG state differs
    cpb = [orc.chunk_count(b.size) for b in c.buffers(1)]
    assert cpb == [48, 1, 32, 32, 32, 32, 32, 32]


def test_config4_ground_truth_by_construction(orc):
    plan = W.config4_plan(3, nbuf=24, hi=1 << 19, n_designated=6, replays=4)
    reps = W.config4_host(plan, 3)
    bm, lab = oracle_classify(orc, reps)
    want_lab = [1 if b in plan.designated else 0 for b in range(len(plan.sizes))]
    assert lab.tolist() == want_lab
    word = 0
    for b, s in enumerate(plan.sizes):
        nch = (s + 4095) // 4096
        exp = np.zeros((nch + 63) // 64, dtype=np.uint64)
        if b in plan.designated:
            for k in range(2, plan.replays + 1):
                for c in plan.rewritten[(k, b)]:
                    exp[c // 64] |= np.uint64(1 << (c % 64))
        assert np.array_equal(bm[word:word + exp.size], exp), b
        word += exp.size
    assert word == bm.size

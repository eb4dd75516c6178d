"""Pins the oracle's checkpoint / restore / fork / delete (the paper's
contract, Sec. 3) with brute force on small inputs: I1 round trip, I2
durability, I3 fork independence, I4 completeness, incremental chains, and
the wrong-value control (Sec. 4) as "changing only the RNG bytes changes the
fingerprint"."""
import os
import struct

import numpy as np
import pytest
import xxhash

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_table1_sizes.txt")


def rand_bufs(rng, sizes):
    return [rng.integers(0, 256, size=s, dtype=np.uint8) for s in sizes]


def test_full_round_trip_and_layout(orc):
    rng = np.random.default_rng(0)
    sizes = [0, 1, 16, 4095, 4096, 4097, 3 * 4096 + 100]
    bufs = rand_bufs(rng, sizes)
    st = orc.Store()
    h = st.checkpoint(bufs)
    out = st.restore(h)
    assert all(np.array_equal(a, b) for a, b in zip(out, bufs))
    pay = st.payload(h)
    # Canonical layout: components 4096-aligned, zero padding, plan order.
    assert pay.size == sum((s + 4095) // 4096 * 4096 for s in sizes)
    off = 0
    for b in bufs:
        assert np.array_equal(pay[off:off + b.size], b)
        pad = (b.size + 4095) // 4096 * 4096
        assert not pay[off + b.size:off + pad].any()
        off += pad
    assert st.state_bytes(h) == sum(sizes)


def test_durability_snapshot_is_not_an_alias(orc):
    rng = np.random.default_rng(1)
    bufs = rand_bufs(rng, [5000, 777])
    keep = [b.copy() for b in bufs]
    st = orc.Store()
    h = st.checkpoint(bufs)
    for b in bufs:
        b[:] = rng.integers(0, 256, size=b.size, dtype=np.uint8)
    assert all(np.array_equal(a, b) for a, b in zip(st.restore(h), keep))


def test_fork_independence(orc):
    rng = np.random.default_rng(2)
    bufs = rand_bufs(rng, [9000, 100])
    st = orc.Store()
    h = st.checkpoint(bufs)
    f = st.fork(h)
    a, b = st.restore(h), st.restore(f)
    a[0][:] = 0
    b[1][:] = 1
    st.delete(h)
    c = st.restore(f)
    assert all(np.array_equal(x, y) for x, y in zip(c, bufs))
    with pytest.raises(KeyError):
        st.restore(h)


def test_table1_sizes_completeness(orc):
    rows = {}
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if not line or line[0] == "shape":
            if line and line[0] == "shape":
                assert line[2] == "480x960x3" and 480 * 960 * 3 == rows["cosmos3"]["obs"]
            continue
        comps = dict(kv.split("=") for kv in line[1:])
        rows[line[0]] = {k: int(v) for k, v in comps.items()}
    rng = np.random.default_rng(3)
    for model, comps in rows.items():
        total = comps.pop("total")
        bufs = rand_bufs(rng, list(comps.values()))
        witness = rng.integers(0, 256, size=2_950_000, dtype=np.uint8)  # not read by restore
        st = orc.Store()
        h = st.checkpoint(bufs)          # the plan holds state only, never the witness
        assert st.state_bytes(h) == total, model
        assert all(np.array_equal(a, b) for a, b in zip(st.restore(h), bufs))
        assert witness.size not in [b.size for b in bufs]


def test_incremental_chain_closed_form(orc):
    bank = W.config2(1, capacity=48, latent_shape=(4, 6, 10), pose_dim=7, step_entries=4)
    st = orc.Store()
    handles, parent = [], 0
    for j in range(1, 13):
        cur = bank.prefix(4 * j)
        h = st.checkpoint(cur, parent)
        handles.append(h)
        parent = h
    order = np.random.default_rng(4).permutation(len(handles))
    for j in order:
        got = st.restore(handles[j])
        want = bank.prefix(4 * (j + 1))       # append-only: state j is the first entries
        assert all(np.array_equal(a, b) for a, b in zip(got, want)), j


def test_incremental_dirty_set_is_byte_difference(orc):
    rng = np.random.default_rng(5)
    base = rand_bufs(rng, [20 * 4096 + 7, 3 * 4096, 100, 2 * 4096 + 9])
    st = orc.Store()
    p = st.checkpoint(base)
    new = [b.copy() for b in base]
    new[0][5 * 4096 + 3] ^= 1                       # one changed chunk
    new[1] = np.concatenate([new[1], rng.integers(0, 256, size=5000, dtype=np.uint8)])  # grows
    new[2] = new[2][:60]                             # shrinks
    # new[3] is unchanged: none of its chunks may be stored again.
    c = st.checkpoint(new, p)
    want = []
    for b, (o, n) in enumerate(zip(base, new)):
        for i in range((n.size + 4095) // 4096):
            old = o[4096 * i:4096 * (i + 1)]
            if i >= (o.size + 4095) // 4096 or old.tobytes() != n[4096 * i:4096 * (i + 1)].tobytes():
                want.append(n[4096 * i:4096 * (i + 1)])
    pay = st.payload(c)
    assert pay.size == 4096 * len(want)
    for k, w in enumerate(want):
        assert np.array_equal(pay[4096 * k:4096 * k + w.size], w)
        assert not pay[4096 * k + w.size:4096 * (k + 1)].any()
    assert all(np.array_equal(a, b) for a, b in zip(st.restore(c), new))
    # Deleting the parent handle keeps the child's chunks alive.
    st.delete(p)
    assert all(np.array_equal(a, b) for a, b in zip(st.restore(c), new))


def test_rng_only_corruption_changes_fingerprint(orc):
    c = W.config1(0)
    _, roots1, s1 = orc.fingerprint(c.buffers(1))
    _, roots2, s2 = orc.fingerprint(c.buffers(2))
    assert s1 != s2 and roots1[1] != roots2[1]
    assert np.array_equal(np.delete(roots1, 1), np.delete(roots2, 1))
    # Every single-bit flip of the 16-byte state changes its hash and the session
    # root, for several states (a change confined to one 8-byte word of a
    # 16-byte XXH64 input always changes the result).
    rng = np.random.default_rng(6)
    others = [int(r) for i, r in enumerate(roots1) if i != 1]
    for _ in range(8):
        st = W.philox_state(rng)
        h0 = xxhash.xxh64_intdigest(st.tobytes())
        assert orc.xxh64(st) == h0
        for bit in range(128):
            f = st.copy()
            f[bit // 8] ^= np.uint8(1 << (bit % 8))
            assert orc.xxh64(f) != h0
            bufs = c.buffers(1)
            bufs[1] = f
            assert orc.fingerprint(bufs)[2] != s1
    assert orc.merkle_root([int(roots1[0]), 1] + others) != orc.merkle_root([int(roots1[0]), 2] + others)


def test_counter_advance_touches_one_word():
    s = W.philox_state(np.random.default_rng(9))
    t = W.advance_counter(s, 1)
    assert s[:8].tobytes() == t[:8].tobytes()
    a, = struct.unpack("<Q", s[8:].tobytes())
    b, = struct.unpack("<Q", t[8:].tobytes())
    assert b == (a + 1) % (1 << 64)

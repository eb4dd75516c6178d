"""GPU parity on both sides of the job sizes where fingerprint and diff
tiles of argument-table jobs widen from 256 to 1024 lanes (fingerprints up
to 1024 groups, incremental checkpoints up to 2048 groups): chunk
fingerprints, buffer and session roots, the stored bytes of incremental
checkpoints and their restores, against the oracle; and on both sides of
the node count up to which a small job's Merkle lists load into LDS in one
pass.  Three ragged buffers, so the tables travel in the kernel arguments."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import arena, dev, host, log, u64, zeros_u64

pytestmark = pytest.mark.gpu

GROUP = 64 * 4096


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


def sizes_for(groups):
    # Buffers of groups - 2, 1 and 1 groups, the first and second ragged.
    s = [(groups - 3) * GROUP + 5 * 4096 + 77, 37 * 4096 + 100, 3]
    assert sum(-(-oracle.chunk_count(n) // 64) for n in s) == groups
    return s


@pytest.mark.parametrize("groups", [1024, 1025])
def test_fingerprint_width_boundary(pcs, groups):
    rng = np.random.default_rng([41, groups])
    sizes = sizes_for(groups)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    log("fingerprint width boundary:", groups, "groups")
    h, r, s = oracle.fingerprint(bufs)
    d = [dev(b) for b in bufs]
    ctx = pcs.Context(arena(64 << 20))
    try:
        ch, rt, sr = zeros_u64(h.size), zeros_u64(len(sizes)), zeros_u64(1)
        ctx.fingerprint([pcs.flat(t, n) for t, n in zip(d, sizes)], ch, rt, sr)
        assert np.array_equal(u64(ch)[:h.size], h)
        assert np.array_equal(u64(rt)[:len(sizes)], r)
        assert int(u64(sr)[0]) == s
    finally:
        ctx.close()


@pytest.mark.parametrize("groups", [2048, 2049])
def test_incremental_width_boundary(pcs, groups):
    rng = np.random.default_rng([43, groups])
    sizes = sizes_for(groups)
    cur = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in cur]
    log("incremental width boundary:", groups, "groups")
    ctx = pcs.Context(arena(sum(sizes) + (160 << 20)))
    try:
        st = oracle.Store()
        chain = [(ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=True), st.checkpoint(cur),
                  [b.copy() for b in cur])]
        total = sum(oracle.chunk_count(n) for n in sizes)
        for step in range(2):
            # Rewrite chunks spread over every buffer, the last (partial) ones included.
            for b in cur:
                nch = oracle.chunk_count(b.size)
                for c in list(rng.integers(0, nch, size=40)) + [nch - 1]:
                    a = int(c) * 4096
                    b[a:min(b.size, a + 4096)] = rng.integers(0, 256, size=min(4096, b.size - a), dtype=np.uint8)
            for t, b in zip(d, cur):
                t.copy_(torch.from_numpy(b))
            ch, rt, sr = zeros_u64(total), zeros_u64(len(sizes)), zeros_u64(1)
            s = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], parent=chain[-1][0], chunk_hashes=ch,
                               roots=rt, session_root=sr)
            o = st.checkpoint(cur, chain[-1][1])
            want_h, want_r, want_s = oracle.fingerprint(cur)
            assert np.array_equal(u64(ch)[:total], want_h)
            assert np.array_equal(u64(rt)[:len(sizes)], want_r) and int(u64(sr)[0]) == int(want_s)
            inf = ctx.info(s)
            assert inf["stored_bytes"] == st.payload(o).size
            pay = torch.empty(max(1, inf["stored_bytes"]), dtype=torch.uint8, device="cuda")
            ctx.payload(s, pay)
            assert np.array_equal(host(pay)[:inf["stored_bytes"]], st.payload(o))
            del pay
            chain.append((s, o, [b.copy() for b in cur]))
        for s, _, want in chain[1:]:
            outs = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes]
            ctx.restore(s, [pcs.flat(t, n) for t, n in zip(outs, sizes)])
            assert all(np.array_equal(host(t), w) for t, w in zip(outs, want))
        for s, _, _ in reversed(chain):
            ctx.delete(s)
    finally:
        ctx.close()


@pytest.mark.parametrize("groups", [4096, 4100])
def test_merkle_lists_past_one_lds_pass(pcs, groups):
    """Argument-table jobs whose buffer lists hold more than 4096 Merkle
    nodes together reduce them list by list through memory instead of in
    one LDS pass: both sides of that bound, fingerprints and the fused
    checkpoint's roots against the oracle."""
    rng = np.random.default_rng([47, groups])
    sizes = sizes_for(groups)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    log("merkle lists past one LDS pass:", groups, "groups")
    h, r, s = oracle.fingerprint(bufs)
    d = [dev(b) for b in bufs]
    ctx = pcs.Context(arena(sum(sizes) + (64 << 20)))
    try:
        ch, rt, sr = zeros_u64(h.size), zeros_u64(len(sizes)), zeros_u64(1)
        ctx.fingerprint([pcs.flat(t, n) for t, n in zip(d, sizes)], ch, rt, sr)
        assert np.array_equal(u64(ch)[:h.size], h)
        assert np.array_equal(u64(rt)[:len(sizes)], r) and int(u64(sr)[0]) == s
        rt2, sr2 = zeros_u64(len(sizes)), zeros_u64(1)
        snap = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=True, roots=rt2, session_root=sr2)
        assert np.array_equal(u64(rt2)[:len(sizes)], r) and int(u64(sr2)[0]) == s
        ctx.delete(snap)
    finally:
        ctx.close()


@pytest.mark.parametrize("case", ["2 long, argument tables", "1 long + 16 short, device tables",
                                  "5 long, in-workgroup passes"])
def test_merkle_long_lists(pcs, case):
    """Buffers of more than 4096 groups: up to four such lists first have their
    64-value blocks reduced by a grid-wide launch (argument and device
    tables); with more, each list's workgroup does it.  Fingerprints, buffer
    and session roots, and the fused checkpoint's roots against the oracle."""
    rng = np.random.default_rng([53, len(case)])
    if case.startswith("2 long"):
        sizes = [4100 * GROUP - 3, 4097 * GROUP + 11, 5]
    elif case.startswith("1 long"):
        sizes = [4099 * GROUP + 7] + [int(rng.integers(1, 3 * 4096)) for _ in range(16)]
    else:
        sizes = [4097 * GROUP + k for k in range(5)]
    log("merkle long lists:", case)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    h, r, s = oracle.fingerprint(bufs)
    d = [dev(b) for b in bufs]
    ctx = pcs.Context(arena(sum(sizes) + (256 << 20)))
    try:
        descs = [pcs.flat(t, n) for t, n in zip(d, sizes)]
        ch, rt, sr = zeros_u64(h.size), zeros_u64(len(sizes)), zeros_u64(1)
        ctx.fingerprint(descs, ch, rt, sr)
        assert np.array_equal(u64(ch)[:h.size], h)
        assert np.array_equal(u64(rt)[:len(sizes)], r) and int(u64(sr)[0]) == s
        rt2, sr2 = zeros_u64(len(sizes)), zeros_u64(1)
        snap = ctx.checkpoint(descs, hash=True, roots=rt2, session_root=sr2)
        assert np.array_equal(u64(rt2)[:len(sizes)], r) and int(u64(sr2)[0]) == s
        ctx.delete(snap)
    finally:
        ctx.close()


@pytest.mark.parametrize("groups", [3, 65, 4096])
def test_incremental_every_chunk_then_none_then_one(pcs, groups):
    """Incremental checkpoints of argument-table jobs whose stored-chunk count
    spans its whole range: every chunk rewritten (at 4096 groups, 262,000
    stored chunks, several per wavefront of the slot placement), then none,
    then only the last chunk of the last buffer.  Chunk fingerprints, roots,
    stored bytes and restores against the oracle."""
    rng = np.random.default_rng([59, groups])
    sizes = sizes_for(groups)
    cur = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in cur]
    log("incremental every chunk / none / one:", groups, "groups")
    ctx = pcs.Context(arena(2 * sum(sizes) + (256 << 20)))
    try:
        st = oracle.Store()
        chain = [(ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=True), st.checkpoint(cur),
                  [b.copy() for b in cur])]
        total = sum(oracle.chunk_count(n) for n in sizes)

        def every(bufs):
            for b in bufs:
                b ^= 0x5A

        def none(bufs):
            pass

        def last(bufs):
            bufs[-1][-1] ^= 1
        for change, stored in ((every, total), (none, 0), (last, 1)):
            change(cur)
            for t, b in zip(d, cur):
                t.copy_(torch.from_numpy(b))
            ch, rt, sr = zeros_u64(total), zeros_u64(len(sizes)), zeros_u64(1)
            s = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], parent=chain[-1][0], chunk_hashes=ch,
                               roots=rt, session_root=sr)
            o = st.checkpoint(cur, chain[-1][1])
            want_h, want_r, want_s = oracle.fingerprint(cur)
            assert np.array_equal(u64(ch)[:total], want_h)
            assert np.array_equal(u64(rt)[:len(sizes)], want_r) and int(u64(sr)[0]) == int(want_s)
            inf = ctx.info(s)
            assert inf["stored_bytes"] == st.payload(o).size == stored * 4096
            pay = torch.empty(max(1, inf["stored_bytes"]), dtype=torch.uint8, device="cuda")
            ctx.payload(s, pay)
            assert np.array_equal(host(pay)[:inf["stored_bytes"]], st.payload(o))
            del pay
            chain.append((s, o, [b.copy() for b in cur]))
        for s, _, want in chain[1:]:
            outs = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes]
            ctx.restore(s, [pcs.flat(t, n) for t, n in zip(outs, sizes)])
            assert all(np.array_equal(host(t), w) for t, w in zip(outs, want))
        for s, _, _ in reversed(chain):
            ctx.delete(s)
    finally:
        ctx.close()


def test_buffer_past_4_gib(pcs):
    """One flat buffer of 2^32 + 12,365 bytes (chunk indices past 2^20, byte
    offsets past 2^32, a partial last chunk): fingerprinted full checkpoint,
    then an incremental one (device tables, slots placed in an arena
    segment) storing the chunks changed below 64 KiB, just past 4 GiB and
    at the end; chunk fingerprints, roots, stored bytes and the restore
    against the oracle."""
    n = (1 << 32) + 3 * 4096 + 77
    log("buffer past 4 GiB:", n, "bytes")
    a = np.frombuffer(np.random.default_rng(61).bytes(n), dtype=np.uint8).copy()
    d = torch.from_numpy(a).cuda()
    total = oracle.chunk_count(n)
    ctx = pcs.Context(arena(2 * n + (512 << 20)))
    try:
        st = oracle.Store()
        ch, rt, sr = zeros_u64(total), zeros_u64(1), zeros_u64(1)
        base = ctx.checkpoint([pcs.flat(d)], hash=True, chunk_hashes=ch, roots=rt, session_root=sr)
        want_h, want_r, want_s = oracle.fingerprint([a])
        assert np.array_equal(u64(ch)[:total], want_h)
        assert int(u64(rt)[0]) == int(want_r[0]) and int(u64(sr)[0]) == int(want_s)
        o_base = st.checkpoint([a])
        for i in (12345, (1 << 32) + 5, n - 1):
            a[i] ^= 1
            d[i] = int(a[i])
        ch2, rt2, sr2 = zeros_u64(total), zeros_u64(1), zeros_u64(1)
        inc = ctx.checkpoint([pcs.flat(d)], parent=base, chunk_hashes=ch2, roots=rt2, session_root=sr2)
        want_h, want_r, want_s = oracle.fingerprint([a])
        assert np.array_equal(u64(ch2)[:total], want_h)
        assert int(u64(rt2)[0]) == int(want_r[0]) and int(u64(sr2)[0]) == int(want_s)
        o_inc = st.checkpoint([a], o_base)
        inf = ctx.info(inc)
        assert inf["stored_bytes"] == st.payload(o_inc).size == 3 * 4096
        pay = torch.empty(inf["stored_bytes"], dtype=torch.uint8, device="cuda")
        ctx.payload(inc, pay)
        assert np.array_equal(host(pay), st.payload(o_inc))
        del st, o_base, o_inc
        out = torch.empty_like(d)
        ctx.restore(inc, [pcs.flat(out)])
        assert np.array_equal(host(out), a)
        del out
        ctx.delete(inc)
        ctx.delete(base)
    finally:
        ctx.close()

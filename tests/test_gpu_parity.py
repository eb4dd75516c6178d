"""GPU parity: libpcs (HIP, through the C ABI) against the CPU oracle,
element by element, on seeded inputs that span several 64-chunk groups,
ragged tails, empty buffers and wrapped ring windows.  Bit-exact throughout
(everything is integer and byte work)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.gpu_util import arena, dev, host, log, u64, zeros_u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


@pytest.fixture()
def ctx(pcs):
    c = pcs.Context(arena(256 << 20))
    yield c
    c.close()


FLAT_SIZES = [0, 1, 7, 15, 16, 17, 31, 32, 33, 63, 100, 4095, 4096, 4097, 8191, 12288 + 24,
              64 * 4096, 64 * 4096 + 1, 65 * 4096 - 5, 130 * 4096 + 8, 200 * 4096 + 4000]


def oracle_fp(bufs):
    h, r, s = oracle.fingerprint(bufs)
    return h, r, s


def gpu_fp(ctx, pcs, descs, total_chunks):
    ch = zeros_u64(total_chunks)
    rt = zeros_u64(len(descs))
    sr = zeros_u64(1)
    ctx.fingerprint(descs, ch, rt, sr)
    return u64(ch)[:total_chunks], u64(rt)[:len(descs)], int(u64(sr)[0])


def test_fingerprint_flat_sizes(ctx, pcs):
    rng = np.random.default_rng(10)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in FLAT_SIZES]
    log("fingerprint flat sizes", FLAT_SIZES)
    d = [dev(b) for b in bufs]
    descs = [pcs.flat(t, b.size) for t, b in zip(d, bufs)]
    h, r, s = oracle_fp(bufs)
    gh, gr, gs = gpu_fp(ctx, pcs, descs, h.size)
    assert np.array_equal(gh, h)
    assert np.array_equal(gr, r)
    assert gs == s


@pytest.mark.parametrize("groups", [16, 17, 127, 128, 129])
def test_small_job_boundary(ctx, pcs, groups):
    """Jobs of at most 128 groups run as 8-chunk sub-tiles (one Merkle node
    per sub-tile), larger ones as whole groups; both sides of the boundary,
    with ragged tails: fingerprints, roots, the fused checkpoint and the
    copy round trip."""
    rng = np.random.default_rng(900 + groups)
    sizes = [(groups - 3) * 64 * 4096 + 4096 * 5 + 77, 37 * 4096 + 100, 3]   # groups-2, 1 and 1 groups
    assert sum((oracle.chunk_count(n) + 63) // 64 for n in sizes) == groups
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in bufs]
    descs = [pcs.flat(t, b.size) for t, b in zip(d, bufs)]
    log("small-job boundary:", groups, "groups")
    h, r, s = oracle_fp(bufs)
    gh, gr, gs = gpu_fp(ctx, pcs, descs, h.size)
    assert np.array_equal(gh, h) and np.array_equal(gr, r) and gs == s
    ch = zeros_u64(h.size)
    snap = ctx.checkpoint(descs, hash=True, chunk_hashes=ch)
    assert np.array_equal(u64(ch)[:h.size], h)
    pay = torch.empty(ctx.info(snap)["stored_bytes"], dtype=torch.uint8, device="cuda")
    ctx.payload(snap, pay)
    assert np.array_equal(host(pay), oracle.pack(bufs))
    plain = ctx.checkpoint(descs)
    outs = [torch.zeros(max(1, n), dtype=torch.uint8, device="cuda") for n in sizes]
    ctx.restore(plain, [pcs.flat(o, n) for o, n in zip(outs, sizes)])
    assert all(np.array_equal(host(o)[:n], b) for o, n, b in zip(outs, sizes, bufs))
    ctx.delete(snap)
    ctx.delete(plain)


@pytest.mark.parametrize("nbuf", [8, 9, 16, 17])
def test_argument_table_boundary(ctx, pcs, nbuf):
    """Jobs of at most 16 buffers and 64 runs carry their tables in the kernel
    arguments, larger ones upload them: both sides of the buffer limit, with
    empty and ragged buffers and a wrapped ring: fingerprints, roots, the
    fused checkpoint, restore, and an incremental checkpoint with changes."""
    rng = np.random.default_rng(700 + nbuf)
    sizes = [int(x) for x in rng.choice([0, 1, 17, 4095, 4096, 9000, 64 * 4096 + 3, 70 * 4096], size=nbuf - 1)]
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    g = W.Ring(3, 40, 1024, 33, 29)
    ring = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical = bufs + [oracle.ring_window(ring, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)]
    d = [dev(b) for b in bufs] + [dev(ring)]
    descs = [pcs.flat(t, b.size) for t, b in zip(d, bufs)] + [pcs.ring(d[-1], g.outer, g.capacity, g.row_bytes,
                                                                       g.head, g.window)]
    log("argument-table boundary:", nbuf, "buffers")
    h, r, s_ = oracle_fp(logical)
    gh, gr, gs = gpu_fp(ctx, pcs, descs, h.size)
    assert np.array_equal(gh, h) and np.array_equal(gr, r) and gs == s_
    ch = zeros_u64(h.size)
    snap = ctx.checkpoint(descs, hash=True, chunk_hashes=ch)
    assert np.array_equal(u64(ch)[:h.size], h)
    pay = torch.empty(max(1, ctx.info(snap)["stored_bytes"]), dtype=torch.uint8, device="cuda")
    ctx.payload(snap, pay)
    assert np.array_equal(host(pay)[:ctx.info(snap)["stored_bytes"]], oracle.pack(logical))
    # Change a byte in every non-empty flat buffer, then checkpoint against the snapshot.
    new = [b.copy() for b in bufs]
    for k, b in enumerate(new):
        if b.size:
            b[int(rng.integers(0, b.size))] ^= 0x5A
            d[k].copy_(torch.from_numpy(b).cuda())
    st = oracle.Store()
    po = st.checkpoint(logical)
    co = st.checkpoint(new + [logical[-1]], po)
    inc = ctx.checkpoint(descs, parent=snap)
    assert ctx.info(inc)["dirty_chunks"] * 4096 == st.payload(co).size
    outs = [torch.zeros(max(1, n), dtype=torch.uint8, device="cuda") for n in sizes]
    rout = torch.zeros(g.ring_bytes, dtype=torch.uint8, device="cuda")
    ctx.restore(inc, [pcs.flat(o, n) for o, n in zip(outs, sizes)] + [pcs.ring(rout, g.outer, g.capacity, g.row_bytes,
                                                                               5, g.window)])
    assert all(np.array_equal(host(o)[:n], b) for o, n, b in zip(outs, sizes, new))
    assert np.array_equal(oracle.ring_window(host(rout), g.outer, g.outer_stride, g.capacity, g.row_bytes, 5,
                                             g.window), logical[-1])
    ctx.delete(inc)
    ctx.delete(snap)


def test_fingerprint_each_size_alone(ctx, pcs):
    rng = np.random.default_rng(11)
    for n in FLAT_SIZES + [1 << 20, (1 << 20) + 3]:
        b = rng.integers(0, 256, size=n, dtype=np.uint8)
        log("fingerprint single", n)
        h, r, s = oracle_fp([b])
        gh, gr, gs = gpu_fp(ctx, pcs, [pcs.flat(dev(b), n)], h.size)
        assert np.array_equal(gh, h) and np.array_equal(gr, r) and gs == s, n


def test_fingerprint_no_buffers(ctx, pcs):
    log("fingerprint of zero buffers")
    gh, gr, gs = gpu_fp(ctx, pcs, [], 0)
    assert gs == oracle.merkle_root([])


RING_CASES = [
    # outer, capacity, row_bytes, window, head, pad
    (1, 8, 16, 8, 0, 0),
    (1, 8, 16, 5, 6, 0),
    (3, 10, 32, 7, 9, 48),
    (4, 64, 2048, 40, 60, 0),
    (2, 16, 48, 1, 15, 16),
    (2, 16, 48, 16, 3, 0),
    (5, 7, 4096, 6, 4, 4096),
    (2, 300, 2048, 257, 299, 0),     # odd head: chunks straddle the wrap
    (6, 1000, 16, 999, 1, 32),       # tiny rows: many rows per chunk
    (64, 96, 2048, 64, 95, 0),       # many rings, wrap at the last slot
    (40, 9, 2048, 7, 5, 0),          # 80 runs (device tables); a group spans ~36 runs
    (200, 4, 16, 3, 2, 0),           # 400 runs of 16-48 bytes; every chunk spans ~170 runs
]


@pytest.mark.parametrize("case", RING_CASES)
def test_fingerprint_ring(ctx, pcs, case):
    outer, cap, row, win, head, pad = case
    g = W.Ring(outer, cap, row, win, head, cap * row + pad)
    log("fingerprint ring", case)
    data = np.random.default_rng(cap + row).integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical = oracle.ring_window(data, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)
    h, r, s = oracle_fp([logical])
    d = dev(data)
    gh, gr, gs = gpu_fp(ctx, pcs, [pcs.ring(d, outer, cap, row, head, win, g.outer_stride)], h.size)
    assert np.array_equal(gh, h) and np.array_equal(gr, r) and gs == s


def test_classify_matches_oracle(ctx, pcs):
    rng = np.random.default_rng(12)
    for trial in range(6):
        K = int(rng.integers(1, 6))
        sizes = [int(rng.integers(0, 150 * 4096)) for _ in range(int(rng.integers(1, 9)))]
        base = [rng.integers(0, 256, size=s, dtype=np.uint8) for s in sizes]
        reps = [base]
        for _ in range(K - 1):
            rep = []
            for a in base:
                a = a.copy()
                if a.size and rng.random() < 0.6:
                    for _ in range(int(rng.integers(1, 6))):
                        a[int(rng.integers(0, a.size))] ^= np.uint8(1 << int(rng.integers(0, 8)))
                rep.append(a)
            reps.append(rep)
        log("classify trial", trial, "K", K, "sizes", sizes)
        oh = np.stack([oracle.fingerprint(rep)[0] for rep in reps])
        cpb = [oracle.chunk_count(s) for s in sizes]
        obm, olab = oracle.classify(oh, cpb)
        total = sum(cpb)
        gh = zeros_u64(K * total)
        for k, rep in enumerate(reps):
            descs = [pcs.flat(dev(a), a.size) for a in rep]
            ch = zeros_u64(total)
            ctx.fingerprint(descs, ch)
            gh[k * total:(k + 1) * total] = ch[:total]
        nw = oracle.bitmap_words(cpb)
        bm = zeros_u64(nw)
        lab = torch.zeros(max(1, len(sizes)), dtype=torch.uint8, device="cuda")
        ctx.classify(gh, K, cpb, bm, lab)
        assert np.array_equal(u64(gh).reshape(K, total) if total else oh, oh)
        assert np.array_equal(u64(bm)[:nw], obm)
        assert np.array_equal(host(lab)[:len(sizes)], olab)


@pytest.mark.parametrize("cpb", [
    [64 * 1000 + 7, 0, 130],          # 1006 groups: one workgroup, many words per wavefront
    [64 * 1024],                      # exactly 1024 groups
    [64 * 1024 + 1, 3],               # 1026 groups: the two-launch path with tables in the arguments
    [5, 0, 70] * 6,                   # 18 buffers: tables in device memory
])
def test_classify_group_count_paths(ctx, pcs, cpb):
    """Classification straight from fingerprint arrays (the oracle's
    definition needs only the K x total array): random fingerprints, replays
    equal to the first except at planted chunks, some of them in every
    buffer but one."""
    rng = np.random.default_rng(sum(cpb) % 1000)
    K = 3
    total = sum(cpb)
    base = rng.integers(0, 1 << 63, size=total, dtype=np.int64).astype(np.uint64)
    oh = np.stack([base.copy() for _ in range(K)])
    starts = np.cumsum([0] + cpb[:-1])
    for b, (s0, n) in enumerate(zip(starts, cpb)):
        if n == 0 or b == 1:
            continue
        for _ in range(int(rng.integers(1, 8))):
            oh[int(rng.integers(1, K)), s0 + int(rng.integers(0, n))] ^= np.uint64(1 << int(rng.integers(0, 64)))
    obm, olab = oracle.classify(oh, cpb)
    log("classify paths", len(cpb), "buffers,", oracle.bitmap_words(cpb), "words")
    gh = torch.from_numpy(oh.reshape(-1).view(np.int64).copy()).cuda()
    nw = oracle.bitmap_words(cpb)
    bm = torch.full((max(nw, 1),), -1, dtype=torch.int64, device="cuda")
    lab = torch.full((len(cpb),), 7, dtype=torch.uint8, device="cuda")
    ctx.classify(gh, K, cpb, bm, lab)
    assert np.array_equal(u64(bm)[:nw], obm)
    assert np.array_equal(host(lab), olab)


def test_checkpoint_restore_flat(ctx, pcs):
    rng = np.random.default_rng(13)
    sizes = [0, 16, 100, 4096, 4097, 70 * 4096 + 9, 3]
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    st = oracle.Store()
    oh = st.checkpoint(bufs)
    d = [dev(b) for b in bufs]
    for hashed in (False, True):
        log("checkpoint/restore flat, hash =", hashed)
        kw = {}
        if hashed:
            ch, rt, sr = zeros_u64(sum(oracle.chunk_count(n) for n in sizes)), zeros_u64(len(sizes)), zeros_u64(1)
            kw = dict(chunk_hashes=ch, roots=rt, session_root=sr)
        snap = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=hashed, **kw)
        inf = ctx.info(snap)
        assert inf["state_bytes"] == sum(sizes) == st.state_bytes(oh)
        assert inf["stored_bytes"] == st.payload(oh).size
        pay = torch.empty(inf["stored_bytes"], dtype=torch.uint8, device="cuda")
        ctx.payload(snap, pay)
        assert np.array_equal(host(pay), st.payload(oh))
        if hashed:
            h, r, s = oracle.fingerprint(bufs)
            assert np.array_equal(u64(ch)[:h.size], h) and np.array_equal(u64(rt)[:len(sizes)], r)
            assert int(u64(sr)[0]) == s
            sh = zeros_u64(h.size)
            ctx.stored_hashes(snap, sh)
            assert np.array_equal(u64(sh)[:h.size], h)
        outs = [torch.full((max(n, 1),), 0xEE, dtype=torch.uint8, device="cuda") for n in sizes]
        ctx.restore(snap, [pcs.flat(o, n) for o, n in zip(outs, sizes)])
        for o, b in zip(outs, bufs):
            got = host(o)
            assert np.array_equal(got[:b.size], b)
            assert np.all(got[b.size:] == 0xEE)  # nothing written past the buffer
        ctx.delete(snap)


def test_durability_and_fork_independence(ctx, pcs):
    rng = np.random.default_rng(14)
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in (9000, 123457)]
    d = [dev(b) for b in bufs]
    log("durability + fork")
    snap = ctx.checkpoint([pcs.flat(t) for t in d], hash=True)
    for t in d:                      # mutate the sources, stream-ordered after the checkpoint
        t.random_(0, 256)
    f = ctx.fork(snap)
    a = [torch.empty_like(t) for t in d]
    b = [torch.empty_like(t) for t in d]
    ctx.restore(snap, [pcs.flat(t) for t in a])
    ctx.restore(f, [pcs.flat(t) for t in b])
    for t in a:                      # mutate one restore; the other and the snapshot are unaffected
        t.zero_()
    ctx.delete(snap)
    c = [torch.empty_like(t) for t in d]
    ctx.restore(f, [pcs.flat(t) for t in c])
    for x, y, z in zip(b, c, bufs):
        assert np.array_equal(host(x), z) and np.array_equal(host(y), z)
    with pytest.raises(pcs.PcsError) as e:
        ctx.restore(snap, [pcs.flat(t) for t in c])
    assert e.value.code == pcs.E_HANDLE
    ctx.delete(f)
    assert ctx.arena_stats()["live_handles"] == 0


@pytest.mark.parametrize("case", RING_CASES)
def test_ring_checkpoint_restore_new_head(ctx, pcs, case):
    outer, cap, row, win, head, pad = case
    g = W.Ring(outer, cap, row, win, head, cap * row + pad)
    log("ring checkpoint/restore", case)
    rng = np.random.default_rng(cap * 7 + row)
    data = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical = oracle.ring_window(data, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)
    d = dev(data)
    snap = ctx.checkpoint([pcs.ring(d, outer, cap, row, head, win, g.outer_stride)], hash=True)
    pay = torch.empty(ctx.info(snap)["stored_bytes"], dtype=torch.uint8, device="cuda")
    ctx.payload(snap, pay)
    assert np.array_equal(host(pay), oracle.pack([logical]))
    for new_head in sorted({0, cap - 1, (head + 1) % cap, int(rng.integers(0, cap))}):
        dst_np = np.full(g.ring_bytes, 0x5A, dtype=np.uint8)
        dst = dev(dst_np)
        ctx.restore(snap, [pcs.ring(dst, outer, cap, row, new_head, win, g.outer_stride)])
        want = dst_np.copy()
        oracle.ring_place(logical, want, g.outer, g.outer_stride, g.capacity, g.row_bytes, new_head, g.window)
        assert np.array_equal(host(dst), want), new_head   # window placed, everything else untouched
    # A different capacity and stride is a compatible destination too.
    g2 = W.Ring(outer, cap + 3, row, win, 2, (cap + 3) * row + 16)
    dst2 = dev(np.zeros(g2.ring_bytes, dtype=np.uint8))
    ctx.restore(snap, [pcs.ring(dst2, outer, cap + 3, row, 2, win, g2.outer_stride)])
    back = oracle.ring_window(host(dst2), g2.outer, g2.outer_stride, g2.capacity, g2.row_bytes, 2, g2.window)
    assert np.array_equal(back, logical)
    ctx.delete(snap)


def test_incremental_chain_small(ctx, pcs):
    bank = W.config2(1, capacity=96, latent_shape=(4, 6, 10), pose_dim=7, step_entries=4)
    lat, pos = dev(bank.latents), dev(bank.poses)
    st = oracle.Store()
    gh, oh = [], []
    parent_g, parent_o = 0, 0
    for j in range(0, 25):
        e = 4 * j
        plan = [pcs.flat(lat, e * bank.latent_entry_bytes), pcs.flat(pos, e * bank.pose_entry_bytes)]
        log("incremental step", j, "entries", e)
        if parent_g == 0:
            s = ctx.checkpoint(plan, hash=True)
            o = st.checkpoint(bank.prefix(e))
        else:
            s = ctx.checkpoint(plan, parent=parent_g)
            o = st.checkpoint(bank.prefix(e), parent_o)
        inf = ctx.info(s)
        pay = torch.empty(max(1, inf["stored_bytes"]), dtype=torch.uint8, device="cuda")
        ctx.payload(s, pay)
        assert inf["stored_bytes"] == st.payload(o).size
        assert np.array_equal(host(pay)[:inf["stored_bytes"]], st.payload(o))
        gh.append(s)
        oh.append(o)
        parent_g, parent_o = s, o
    order = np.random.default_rng(15).permutation(len(gh))
    for j in order:
        e = 4 * int(j)
        want = bank.prefix(e)
        outs = [torch.empty(max(1, w.size), dtype=torch.uint8, device="cuda") for w in want]
        ctx.restore(gh[j], [pcs.flat(o, w.size) for o, w in zip(outs, want)])
        for o, w in zip(outs, want):
            assert np.array_equal(host(o)[:w.size], w), j
    # Deleting every handle but the last keeps the chain restorable.
    for s in gh[:-1]:
        ctx.delete(s)
    want = bank.prefix(4 * (len(gh) - 1))
    outs = [torch.empty(w.size, dtype=torch.uint8, device="cuda") for w in want]
    ctx.restore(gh[-1], [pcs.flat(o, w.size) for o, w in zip(outs, want)])
    assert all(np.array_equal(host(o), w) for o, w in zip(outs, want))


@pytest.mark.parametrize("groups", [64, 65, 128, 129])
def test_incremental_group_boundaries(ctx, pcs, groups):
    """Incremental checkpoints on both sides of the job sizes where the
    small path changes shape: the Merkle lists, scan and slot assignment in
    one launch up to 64 groups (slot assignment separate above), 8-chunk
    sub-tiles up to 128 groups.  Two buffers, the second one partial; a
    chain of two incremental checkpoints; stored bytes, fingerprints and
    restores against the oracle."""
    rng = np.random.default_rng(300 + groups)
    sizes = [(groups - 1) * 64 * 4096, 33 * 4096 + 100]
    cur = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in cur]
    st = oracle.Store()
    log("incremental boundaries", groups, "groups")
    s = ctx.checkpoint([pcs.flat(t) for t in d], hash=True)
    o = st.checkpoint(cur)
    chain = [(s, o, [b.copy() for b in cur])]
    for step in range(2):
        for b in cur:  # rewrite a few chunks of each buffer, the partial last one included
            for c in list(rng.integers(0, oracle.chunk_count(b.size), size=5)) + [oracle.chunk_count(b.size) - 1]:
                a = int(c) * 4096
                b[a:min(b.size, a + 4096)] = rng.integers(0, 256, size=min(4096, b.size - a), dtype=np.uint8)
        for t, b in zip(d, cur):
            t.copy_(torch.from_numpy(b))
        total = sum(oracle.chunk_count(n) for n in sizes)
        ch, rt, sr = zeros_u64(total), zeros_u64(2), zeros_u64(1)
        s = ctx.checkpoint([pcs.flat(t) for t in d], parent=chain[-1][0], chunk_hashes=ch, roots=rt, session_root=sr)
        o = st.checkpoint(cur, chain[-1][1])
        want_h, want_r, want_s = oracle.fingerprint(cur)
        assert np.array_equal(u64(ch)[:total], want_h)
        assert np.array_equal(u64(rt)[:2], want_r) and int(u64(sr)[0]) == int(want_s)
        inf = ctx.info(s)
        pay = torch.empty(max(1, inf["stored_bytes"]), dtype=torch.uint8, device="cuda")
        ctx.payload(s, pay)
        assert inf["stored_bytes"] == st.payload(o).size
        assert np.array_equal(host(pay)[:inf["stored_bytes"]], st.payload(o))
        chain.append((s, o, [b.copy() for b in cur]))
    for s, _, want in chain:
        outs = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes]
        ctx.restore(s, [pcs.flat(t) for t in outs])
        assert all(np.array_equal(host(t), w) for t, w in zip(outs, want))


def test_incremental_changes_and_shrink(ctx, pcs):
    rng = np.random.default_rng(16)
    base = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in (20 * 4096 + 7, 3 * 4096, 100, 2 * 4096 + 9, 70 * 4096)]
    new = [b.copy() for b in base]
    new[0][5 * 4096 + 3] ^= 1
    new[1] = np.concatenate([new[1], rng.integers(0, 256, size=5000, dtype=np.uint8)])
    new[2] = new[2][:60]
    new[4][[0, 64 * 4096 + 1, 69 * 4096 + 17]] ^= 0xFF
    log("incremental with changes, growth and shrink")
    st = oracle.Store()
    po = st.checkpoint(base)
    co = st.checkpoint(new, po)
    p = ctx.checkpoint([pcs.flat(dev(b)) for b in base], hash=True)
    c = ctx.checkpoint([pcs.flat(dev(b)) for b in new], parent=p)
    inf = ctx.info(c)
    assert inf["incremental"] == 1 and inf["dirty_chunks"] * 4096 == st.payload(co).size
    pay = torch.empty(max(1, inf["stored_bytes"]), dtype=torch.uint8, device="cuda")
    ctx.payload(c, pay)
    assert np.array_equal(host(pay)[:inf["stored_bytes"]], st.payload(co))
    outs = [torch.empty(b.size, dtype=torch.uint8, device="cuda") for b in new]
    ctx.restore(c, [pcs.flat(o) for o in outs])
    assert all(np.array_equal(host(o), b) for o, b in zip(outs, new))


def test_batch_checkpoint_restore(ctx, pcs):
    plan = W.config5_plan(4, sessions=6, layers=1, window=24, capacity=40, heads=2, head_dim=8,
                          obs_shape=(5, 7, 3), restore_fraction=0.5)
    g = plan.ring
    rng = np.random.default_rng(17)
    rings = [rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8) for _ in range(plan.sessions)]
    obs = [rng.integers(0, 256, size=plan.obs_bytes, dtype=np.uint8) for _ in range(plan.sessions)]
    rs = [rng.integers(0, 256, size=16, dtype=np.uint8) for _ in range(plan.sessions)]
    dr, do, dg = [dev(x) for x in rings], [dev(x) for x in obs], [dev(x) for x in rs]
    plans = [[pcs.ring(dr[s], g.outer, g.capacity, g.row_bytes, plan.heads[s], g.window), pcs.flat(do[s]),
              pcs.flat(dg[s])] for s in range(plan.sessions)]
    logical = [[oracle.ring_window(rings[s], g.outer, g.outer_stride, g.capacity, g.row_bytes, plan.heads[s],
                                   g.window), obs[s], rs[s]] for s in range(plan.sessions)]
    log("batch checkpoint", plan.sessions, "sessions")
    total = sum(oracle.chunk_count(b.size) for L in logical for b in L)
    ch, rt, sr = zeros_u64(total), zeros_u64(3 * plan.sessions), zeros_u64(plan.sessions)
    snaps = ctx.checkpoint_batch(plans, hash=True, chunk_hashes=ch, roots=rt, session_roots=sr)
    oh = np.concatenate([oracle.fingerprint(L)[0] for L in logical])
    orr = np.concatenate([oracle.fingerprint(L)[1] for L in logical])
    osr = np.array([oracle.fingerprint(L)[2] for L in logical], dtype=np.uint64)
    assert np.array_equal(u64(ch)[:total], oh)
    assert np.array_equal(u64(rt)[:3 * plan.sessions], orr)
    assert np.array_equal(u64(sr)[:plan.sessions], osr)
    # Restore a permuted subset at new heads, in one launch.
    order, heads = plan.restore_order, plan.restore_heads
    dst_r = [dev(np.zeros(g.ring_bytes, dtype=np.uint8)) for _ in order]
    dst_o = [torch.empty(plan.obs_bytes, dtype=torch.uint8, device="cuda") for _ in order]
    dst_g = [torch.empty(16, dtype=torch.uint8, device="cuda") for _ in order]
    dsts = [[pcs.ring(dst_r[k], g.outer, g.capacity, g.row_bytes, heads[k], g.window), pcs.flat(dst_o[k]),
             pcs.flat(dst_g[k])] for k in range(len(order))]
    ctx.restore_batch([snaps[s] for s in order], dsts)
    for k, s in enumerate(order):
        win = oracle.ring_window(host(dst_r[k]), g.outer, g.outer_stride, g.capacity, g.row_bytes, heads[k], g.window)
        assert np.array_equal(win, logical[s][0])
        assert np.array_equal(host(dst_o[k]), obs[s]) and np.array_equal(host(dst_g[k]), rs[s])


def test_errors_enqueue_nothing(ctx, pcs):
    t = torch.zeros(4096 * 3, dtype=torch.uint8, device="cuda")
    log("error paths")
    with pytest.raises(pcs.PcsError) as e:
        ctx.fingerprint([pcs.PcsBuf(ptr=t.data_ptr() + 3, nbytes=10, kind=pcs.FLAT)])
    assert e.value.code == pcs.E_INVAL
    with pytest.raises(pcs.PcsError) as e:
        ctx.fingerprint([pcs.ring(t, 1, 8, 16, 8, 4)])          # head >= capacity
    assert e.value.code == pcs.E_INVAL
    with pytest.raises(pcs.PcsError) as e:
        ctx.fingerprint([pcs.PcsBuf(ptr=t.data_ptr(), nbytes=10, kind=7)])
    assert e.value.code == pcs.E_INVAL
    s = ctx.checkpoint([pcs.flat(t, 5000)])
    with pytest.raises(pcs.PcsError) as e:
        ctx.restore(s, [pcs.flat(t, 4999)])
    assert e.value.code == pcs.E_SHAPE
    with pytest.raises(pcs.PcsError) as e:
        ctx.restore(s, [pcs.flat(t, 5000), pcs.flat(t, 1)])
    assert e.value.code == pcs.E_SHAPE
    with pytest.raises(pcs.PcsError) as e:
        ctx.checkpoint([pcs.flat(t, 5000)], parent=s)         # parent without fingerprints
    assert e.value.code == pcs.E_INVAL
    with pytest.raises(pcs.PcsError) as e:
        ctx.fork(12345)
    assert e.value.code == pcs.E_HANDLE
    big = torch.zeros(300 << 20, dtype=torch.uint8, device="cuda")
    before = ctx.arena_stats()
    with pytest.raises(pcs.PcsError) as e:
        ctx.checkpoint([pcs.flat(big)])                       # arena is 256 MiB
    assert e.value.code == pcs.E_NOMEM
    assert ctx.arena_stats() == before
    ctx.delete(s)


def test_batch_checkpoint_is_all_or_nothing(pcs):
    # Three sessions of 3 MiB each do not fit an 8 MiB arena together: the
    # batch fails as a whole (no handle, no reserved block left behind) and
    # the same call over two of them succeeds.
    srcs = [torch.full((3 << 20,), k + 1, dtype=torch.uint8, device="cuda") for k in range(3)]
    c = pcs.Context(arena(8 << 20))
    before = c.arena_stats()
    log("batch checkpoint that does not fit")
    with pytest.raises(pcs.PcsError) as e:
        c.checkpoint_batch([[pcs.flat(t)] for t in srcs], hash=True)
    assert e.value.code == pcs.E_NOMEM
    assert c.arena_stats() == before
    snaps = c.checkpoint_batch([[pcs.flat(t)] for t in srcs[:2]], hash=True)
    outs = [torch.zeros(3 << 20, dtype=torch.uint8, device="cuda") for _ in range(2)]
    c.restore_batch(snaps, [[pcs.flat(o)] for o in outs])
    assert all(np.all(host(o) == k + 1) for k, o in enumerate(outs))
    c.delete(snaps[0])
    with pytest.raises(pcs.PcsError) as e:
        c.restore(snaps[0], [pcs.flat(outs[0])])              # a deleted handle
    assert e.value.code == pcs.E_HANDLE
    c.delete(snaps[1])
    assert c.arena_stats() == before
    c.close()


def test_incremental_chain_in_tight_arena(pcs):
    # 64 growing incremental checkpoints whose final state is ~6.4 MiB must fit
    # in a 16 MiB arena: worst-case claims are given back without leaving
    # holes the next (larger) call cannot use.  Once the stream is idle (every
    # stored-chunk count read, every segment's unused part returned) the arena
    # holds the snapshots and nothing else.
    bank = W.config2(1, capacity=512, latent_shape=(4, 15, 26), pose_dim=7, step_entries=8)
    lat, pos = dev(bank.latents), dev(bank.poses)
    final = 512 * (bank.latent_entry_bytes + bank.pose_entry_bytes)
    log("tight arena: final state", final)
    c = pcs.Context(arena(16 << 20))
    handles, parent = [], 0
    for j in range(1, 65):
        e = 8 * j
        plan = [pcs.flat(lat, e * bank.latent_entry_bytes), pcs.flat(pos, e * bank.pose_entry_bytes)]
        h = c.checkpoint(plan, parent=parent, hash=parent == 0)
        handles.append(h)
        parent = h
    assert c.arena_stats()["used"] <= 16 << 20
    torch.cuda.synchronize()
    stats = c.arena_stats()
    assert stats["used"] < 2 * final + (1 << 20), stats
    for j in (0, 31, 63):
        e = 8 * (j + 1)
        want = bank.prefix(e)
        outs = [torch.empty(w.size, dtype=torch.uint8, device="cuda") for w in want]
        c.restore(handles[j], [pcs.flat(o) for o in outs])
        assert all(np.array_equal(host(o), w) for o, w in zip(outs, want)), j
    for h in handles:
        c.delete(h)
    assert c.arena_stats()["used"] == 0
    c.close()


def test_incremental_exact_placement_then_pipelined(pcs):
    """An incremental checkpoint whose worst case (a slot for every chunk of
    the prefix) does not fit the arena beside its parent: the host reads the
    stored-chunk count and places exactly that many slots (diff, scan, slot
    copy: three incremental launches).  Then, on the same context, one of a
    1 MiB prefix against the same parent, which fits and takes the pipelined
    small path (two launches, a new arena segment).  Stored bytes,
    fingerprints and restores against the oracle."""
    rng = np.random.default_rng(77)
    n = 16 << 20
    cur = [rng.integers(0, 256, size=n, dtype=np.uint8), rng.integers(0, 256, size=5000, dtype=np.uint8)]
    d = [dev(b) for b in cur]
    log("incremental exact placement")
    c = pcs.Context(arena(n + (2 << 20)))
    try:
        st = oracle.Store()
        base = (c.checkpoint([pcs.flat(t) for t in d], hash=True), st.checkpoint(cur))
        flipped = rng.choice(oracle.chunk_count(n), size=40, replace=False)
        fresh = [k for k in range(256) if k not in set(int(x) for x in flipped)][:3]
        made = []
        for flips, prefix, launches in ((flipped, n, 3), (fresh, 1 << 20, 2)):
            for k in flips:
                cur[0][int(k) * 4096] ^= 0xFF
            cur[1][-1] = (int(cur[1][-1]) + 1) % 256
            for t, b in zip(d, cur):
                t.copy_(torch.from_numpy(b))
            logical = [cur[0][:prefix].copy(), cur[1].copy()]
            total = sum(oracle.chunk_count(b.size) for b in logical)
            c.kernel_time("incremental")
            c.set_timing(True)
            ch, rt, sr = zeros_u64(total), zeros_u64(2), zeros_u64(1)
            s = c.checkpoint([pcs.flat(d[0], prefix), pcs.flat(d[1])], parent=base[0], chunk_hashes=ch, roots=rt,
                             session_root=sr)
            c.set_timing(False)
            assert c.kernel_time("incremental")[0] == launches
            o = st.checkpoint(logical, base[1])
            want_h, want_r, want_s = oracle.fingerprint(logical)
            assert np.array_equal(u64(ch)[:total], want_h)
            assert np.array_equal(u64(rt)[:2], want_r) and int(u64(sr)[0]) == int(want_s)
            inf = c.info(s)
            assert inf["stored_bytes"] == st.payload(o).size > 0
            if launches == 3:
                assert inf["stored_bytes"] == 41 * 4096
            pay = torch.empty(inf["stored_bytes"], dtype=torch.uint8, device="cuda")
            c.payload(s, pay)
            assert np.array_equal(host(pay), st.payload(o))
            del pay
            outs = [torch.empty(b.size, dtype=torch.uint8, device="cuda") for b in logical]
            c.restore(s, [pcs.flat(t) for t in outs])
            assert all(np.array_equal(host(t), b) for t, b in zip(outs, logical))
            del outs
            made.append(s)
        for s in made + [base[0]]:
            c.delete(s)
    finally:
        c.close()


@pytest.mark.parametrize("dispatch", [False, True])
def test_kernel_timing_counts_and_resets(ctx, pcs, dispatch):
    """pcs_set_timing / pcs_kernel_time, both modes (events around each
    launch; the dispatches' own timestamps): while enabled, every launch of
    a family is counted with a positive duration; a query resets the family;
    launches made while disabled are not counted; a mode other than 0, 1
    or 2 is refused."""
    rng = np.random.default_rng(40)
    a = rng.integers(0, 256, size=300 * 4096 + 5, dtype=np.uint8)
    d = dev(a)
    out = torch.empty_like(d)
    for fam in ("pack", "copy", "pack_hash", "merkle"):
        ctx.kernel_time(fam)
    s = ctx.checkpoint([pcs.flat(d)])            # not timed
    with pytest.raises(pcs.PcsError):
        ctx._check(pcs._lib.lib().pcs_set_timing(ctx._h, 3))
    ctx.set_timing(True, dispatch=dispatch)
    for _ in range(3):
        ctx.restore(s, [pcs.flat(out)])
    s2 = ctx.checkpoint([pcs.flat(d)], hash=True)
    ctx.set_timing(False)
    ctx.restore(s, [pcs.flat(out)])              # not timed
    n, ms = ctx.kernel_time("copy")
    assert n == 3 and ms > 0
    assert ctx.kernel_time("copy") == (0, 0.0)   # reset by the query
    assert ctx.kernel_time("pack")[0] == 0       # the untimed plain checkpoint
    n, ms = ctx.kernel_time("pack_hash")
    assert n == 1 and ms > 0
    assert ctx.kernel_time("merkle")[0] >= 1
    assert np.array_equal(host(out), a)
    ctx.delete(s)
    ctx.delete(s2)

"""GPU parity of the verified restore (restore fused with fingerprinting and a
comparison against the fingerprints stored at checkpoint time).

The oracle's reading: verification is cross-replay classification with K = 2
between the stored fingerprints and the fingerprints of the restored bytes.
Corruption is simulated by flipping bytes of a snapshot's payload through
its read-only view (standing in for a storage or memory fault)."""
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


def flip(arena_t, addr, positions):
    """Flips the low bit of bytes at device addresses addr + positions (inside the arena)."""
    base = arena_t.data_ptr()
    for p in positions:
        off = addr - base + int(p)
        assert 0 <= off < arena_t.numel()
        arena_t[off:off + 1] ^= 1


def expected_bits(orig, restored):
    """Oracle: classify (K=2) the original fingerprints against the restored bytes'."""
    ho = oracle.fingerprint(orig)[0]
    hr = oracle.fingerprint(restored)[0]
    cpb = [oracle.chunk_count(b.size) for b in orig]
    return oracle.classify(np.stack([ho, hr]), cpb)


def test_verify_full_snapshot_clean_and_corrupted(pcs):
    rng = np.random.default_rng(21)
    sizes = [5000, 16, 64 * 4096 + 77, 0, 3 * 4096]
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    g = W.Ring(3, 40, 2048, 33, 37)
    ring_np = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical_ring = oracle.ring_window(ring_np, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)
    ar = arena(64 << 20)
    ctx = pcs.Context(ar)
    d = [dev(b) for b in bufs] + [dev(ring_np)]
    plan = [pcs.flat(t, n) for t, n in zip(d, sizes)] + [pcs.ring(d[-1], g.outer, g.capacity, g.row_bytes, g.head,
                                                                  g.window)]
    orig = bufs + [logical_ring]
    cpb = [oracle.chunk_count(b.size) for b in orig]
    nw = oracle.bitmap_words(cpb)
    snap = ctx.checkpoint(plan, hash=True)

    def restore_and_check(tag):
        outs = [torch.zeros(max(n, 1), dtype=torch.uint8, device="cuda") for n in sizes]
        rdst = dev(np.zeros(g.ring_bytes, dtype=np.uint8))
        new_head = 5
        dsts = [pcs.flat(o, n) for o, n in zip(outs, sizes)] + [pcs.ring(rdst, g.outer, g.capacity, g.row_bytes,
                                                                         new_head, g.window)]
        bm = zeros_u64(nw)
        lab = torch.full((len(orig),), 7, dtype=torch.uint8, device="cuda")
        ctx.restore_verify(snap, dsts, bm, lab)
        restored = [host(o)[:n] for o, n in zip(outs, sizes)] + [
            oracle.ring_window(host(rdst), g.outer, g.outer_stride, g.capacity, g.row_bytes, new_head, g.window)]
        # Restored bytes are what the oracle unpacks from the (possibly corrupted) payload.
        addr, nbytes = ctx.view(snap)
        pay = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        ctx.payload(snap, pay)
        want_bytes = oracle.unpack(host(pay), [b.size for b in orig])
        assert all(np.array_equal(a, b) for a, b in zip(restored, want_bytes)), tag
        obm, olab = expected_bits(orig, want_bytes)
        assert np.array_equal(u64(bm)[:nw], obm), tag
        assert np.array_equal(host(lab), olab), tag
        return obm, olab

    log("verify: clean")
    obm, olab = restore_and_check("clean")
    assert not obm.any() and not olab.any()
    # Corrupt bytes inside components (not padding): component offsets are 4096-aligned.
    offs, _ = oracle.payload_layout([b.size for b in orig])
    hits = [int(offs[0]) + 4097, int(offs[2]) + 5 * 4096 + 3, int(offs[2]) + 64 * 4096 + 10,
            int(offs[5]) + 2048 * 7 + 1]
    addr, _ = ctx.view(snap)
    flip(ar, addr, hits)
    log("verify: corrupted", hits)
    obm, olab = restore_and_check("corrupted")
    assert olab.tolist() == [1, 0, 1, 0, 0, 1]
    assert int(obm.sum() > 0)
    ctx.close()


def test_verify_incremental_chain(pcs):
    bank = W.config2(1, capacity=64, latent_shape=(4, 15, 26), pose_dim=7, step_entries=8)
    lat, pos = dev(bank.latents), dev(bank.poses)
    ar = arena(64 << 20)
    ctx = pcs.Context(ar)
    st = oracle.Store()
    hs, os_, parent_g, parent_o = [], [], 0, 0
    for j in range(1, 6):
        e = 8 * j
        plan = [pcs.flat(lat, e * bank.latent_entry_bytes), pcs.flat(pos, e * bank.pose_entry_bytes)]
        g = ctx.checkpoint(plan, parent=parent_g, hash=parent_g == 0)
        o = st.checkpoint(bank.prefix(e), parent_o)
        hs.append(g)
        os_.append(o)
        parent_g, parent_o = g, o
    last = hs[-1]
    want = bank.prefix(40)
    cpb = [oracle.chunk_count(w.size) for w in want]
    nw = oracle.bitmap_words(cpb)

    def run():
        outs = [torch.empty(w.size, dtype=torch.uint8, device="cuda") for w in want]
        bm = zeros_u64(nw)
        lab = torch.zeros(2, dtype=torch.uint8, device="cuda")
        ctx.restore_verify(last, [pcs.flat(o) for o in outs], bm, lab)
        return [host(o) for o in outs], u64(bm)[:nw], host(lab)

    log("verify incremental: clean")
    got, bm, lab = run()
    assert all(np.array_equal(a, b) for a, b in zip(got, want)) and not bm.any() and not lab.any()
    # Corrupt stored slot s of the last snapshot: slots sit below the top of its
    # payload, slot 0 highest.  The oracle's snapshot lists its stored chunks in
    # the same (buffer, chunk) order.
    addr, nbytes = ctx.view(last)
    snap_o = st.snapshot(os_[-1])
    stored = [(b, i) for b in range(2) for i, (arr, off) in enumerate(snap_o.where[b]) if arr is snap_o.payload]
    assert len(stored) * 4096 == nbytes
    s = len(stored) // 2
    b, i = stored[s]
    flip(ar, addr + nbytes - (s + 1) * 4096, [100])
    log("verify incremental: corrupted slot", s, "= buffer", b, "chunk", i)
    got, bm, lab = run()
    exp = [w.copy() for w in want]
    exp[b][4096 * i + 100] ^= 1
    assert all(np.array_equal(a, c) for a, c in zip(got, exp))
    obm, olab = expected_bits(want, exp)
    assert np.array_equal(bm, obm) and np.array_equal(lab, olab)
    assert lab.tolist() == [1 if x == b else 0 for x in range(2)]
    ctx.close()


def test_verify_needs_fingerprints(pcs):
    ctx = pcs.Context(arena(16 << 20))
    t = torch.zeros(9000, dtype=torch.uint8, device="cuda")
    s = ctx.checkpoint([pcs.flat(t)])
    with pytest.raises(pcs.PcsError) as e:
        ctx.restore_verify(s, [pcs.flat(t)], zeros_u64(3))
    assert e.value.code == pcs.E_INVAL
    ctx.close()

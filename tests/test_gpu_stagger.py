"""GPU parity on both sides of the first-round stagger's job-size bounds.

Whole-group pack + fingerprint and verified-restore jobs of 2 to 9 rounds
(one workgroup per CU) hold their first-round workgroups back by phase, and
pack jobs of at most 9 rounds store the snapshot write-back (larger ones
nontemporal); the bytes and fingerprints must not depend on either.  Jobs
of 1 round, 2 rounds - 1, 2 rounds, 9 rounds and 9 rounds + 1 groups (from
the device's CU count), made of ragged buffers, are checked against the
oracle: chunk fingerprints, buffer and session roots, the stored payload,
the restored bytes and a clean verification bitmap; and at 2 and 9 rounds a
corrupted snapshot's verification bitmap and labels."""
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


def cus():
    return torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("rounds,extra", [(1, 0), (2, -1), (2, 0), (9, 0), (9, 1)])
def test_stagger_bounds_parity(pcs, rounds, extra):
    G = rounds * cus() + extra
    # Buffers of G - 3, 2 and 1 groups with ragged tails.
    sizes = [(G - 3) * GROUP - 5, GROUP + 7, 100]
    log("stagger bounds: rounds", rounds, "extra", extra, "groups", G, "sizes", sizes)
    rng = np.random.default_rng([31, G])
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    assert sum(-(-oracle.chunk_count(n) // 64) for n in sizes) == G
    h, r, s = oracle.fingerprint(bufs)
    d = [dev(b) for b in bufs]
    ar = arena(sum(sizes) + (64 << 20))
    ctx = pcs.Context(ar)
    try:
        ch, rt, sr = zeros_u64(h.size), zeros_u64(len(sizes)), zeros_u64(1)
        snap = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=True, chunk_hashes=ch, roots=rt,
                              session_root=sr)
        assert np.array_equal(u64(ch)[:h.size], h)
        assert np.array_equal(u64(rt)[:len(sizes)], r)
        assert int(u64(sr)[0]) == s
        inf = ctx.info(snap)
        pay = torch.empty(inf["stored_bytes"], dtype=torch.uint8, device="cuda")
        ctx.payload(snap, pay)
        assert np.array_equal(host(pay), oracle.pack(bufs))
        del pay
        outs = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in sizes]
        cpb = [oracle.chunk_count(n) for n in sizes]
        bm = zeros_u64(oracle.bitmap_words(cpb))
        lab = torch.full((len(sizes),), 7, dtype=torch.uint8, device="cuda")
        ctx.restore_verify(snap, [pcs.flat(o, n) for o, n in zip(outs, sizes)], bm, lab)
        for o, b in zip(outs, bufs):
            assert np.array_equal(host(o), b)
        assert not u64(bm).any() and not host(lab).any()
        ctx.delete(snap)
    finally:
        ctx.close()


@pytest.mark.parametrize("rounds", [2, 9])
def test_stagger_verify_detects_corruption(pcs, rounds):
    """The staggered verified restore (its own tile shape) flags exactly the
    chunks whose stored bytes changed: flips at the first and last chunk of
    groups, on both sides of a group's middle, in a partial last chunk and in
    a one-chunk buffer, spread over first-round and later groups; bitmap,
    labels and restored bytes against the oracle."""
    from tests.test_gpu_verify import expected_bits, flip
    G = rounds * cus()
    sizes = [(G - 3) * GROUP - 5, GROUP + 7, 100]
    log("stagger verify corruption: rounds", rounds, "groups", G)
    rng = np.random.default_rng([37, G])
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in bufs]
    ar = arena(sum(sizes) + (64 << 20))
    ctx = pcs.Context(ar)
    try:
        snap = ctx.checkpoint([pcs.flat(t, n) for t, n in zip(d, sizes)], hash=True)
        offs, _ = oracle.payload_layout(sizes)
        c0 = oracle.chunk_count(sizes[0])
        hits = [int(offs[0]),                                   # group 0, chunk 0
                int(offs[0]) + (64 * 5 + 31) * 4096 + 4095,     # a first-round group, chunk 31's last byte
                int(offs[0]) + (64 * (G // 2) + 32) * 4096 + 17,  # a later group, chunk 32
                int(offs[0]) + (64 * (G - 5) + 63) * 4096 + 1,  # the big buffer's last full group, chunk 63
                int(offs[0]) + (c0 - 1) * 4096 + 3,             # its partial last chunk
                int(offs[1]) + 64 * 4096 + 2,                   # the 7-byte last chunk of buffer 1
                int(offs[2]) + 99]                              # the one-chunk buffer's last byte
        addr, _ = ctx.view(snap)
        flip(ar, addr, hits)
        outs = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in sizes]
        nw = oracle.bitmap_words([oracle.chunk_count(n) for n in sizes])
        bm = zeros_u64(nw)
        lab = torch.full((len(sizes),), 7, dtype=torch.uint8, device="cuda")
        ctx.restore_verify(snap, [pcs.flat(o, n) for o, n in zip(outs, sizes)], bm, lab)
        pay = torch.empty(ctx.info(snap)["stored_bytes"], dtype=torch.uint8, device="cuda")
        ctx.payload(snap, pay)
        want_bytes = oracle.unpack(host(pay), sizes)
        del pay
        for o, w in zip(outs, want_bytes):
            assert np.array_equal(host(o), w)
        obm, olab = expected_bits(bufs, want_bytes)
        assert int(np.unpackbits(obm.view(np.uint8)).sum()) == len(hits)
        assert np.array_equal(u64(bm)[:nw], obm)
        assert np.array_equal(host(lab), olab) and olab.tolist() == [1, 1, 1]
        ctx.delete(snap)
    finally:
        ctx.close()

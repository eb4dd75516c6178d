"""GPU parity on both sides of the first-round stagger's job-size bounds.

Whole-group pack + fingerprint and verified-restore jobs of 2 to 9 rounds
(one workgroup per CU) hold their first-round workgroups back by phase; the
bytes and fingerprints must not depend on it.  Jobs of 2 rounds - 1, 2
rounds, 9 rounds and 9 rounds + 1 groups (from the device's CU count), made
of ragged buffers, are checked against the oracle: chunk fingerprints,
buffer and session roots, the stored payload, the restored bytes and a
clean verification bitmap."""
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


@pytest.mark.parametrize("rounds,extra", [(2, -1), (2, 0), (9, 0), (9, 1)])
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

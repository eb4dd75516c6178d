"""GPU parity of the relevance-keyed bank shrink (pcs_bank_shrink; Sec. 5,
Sec. 7.5, Tables 5-6) against the oracle: kept indices bit-exact, kept
entries byte-exact, in place and out of place, and the incremental
checkpoint that follows a shrink of the memory bank configuration."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.gpu_util import arena, dev, host, log
from tests.test_oracle_bank import tricky_scores

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


def scores_dev(s):
    return torch.from_numpy(np.ascontiguousarray(s, dtype=np.float32).copy()).cuda()


CASES = [
    (1, [1, 28]),
    (37, [1, 28, 4096, 4100]),
    (513, [28, 16 * 60 * 104 * 2]),
    (4099, [4, 16, 60]),
    (65536, [4, 28]),
    (1 << 20, [4, 28]),      # a million entries: selection is linear, not pairwise
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_shrink_matches_oracle(pcs, case):
    n, sizes = case
    rng = np.random.default_rng(70 + n)
    ctx = pcs.Context(arena(256 << 20))
    before = ctx.arena_stats()
    s = tricky_scores(rng, n)
    sd = scores_dev(s)
    parts = [rng.integers(0, 256, size=n * eb, dtype=np.uint8) for eb in sizes]
    for keep in sorted({0, 1, n // 3, n}):
        want_kept, want = oracle.bank_shrink(list(zip(parts, sizes)), s, keep)
        for inplace in (False, True):
            log("bank shrink n", n, "sizes", sizes, "keep", keep, "in place" if inplace else "to new buffers")
            srcs = [dev(p) for p in parts]
            dsts = [None if inplace else torch.full((max(1, keep * eb),), 0xA5, dtype=torch.uint8, device="cuda")
                    for eb in sizes]
            kept = torch.full((max(1, keep),), -1, dtype=torch.int32, device="cuda")
            ctx.bank_shrink([(a, d, eb) for a, d, eb in zip(srcs, dsts, sizes)], sd, keep, kept)
            assert host(kept).view(np.uint32)[:keep].tolist() == want_kept.tolist()
            for p, a, d, eb, w in zip(parts, srcs, dsts, sizes, want):
                got = host(a if inplace else d)
                assert np.array_equal(got[:keep * eb], w)
                if inplace:
                    assert np.array_equal(got[keep * eb:], p[keep * eb:])   # the rest is untouched
                else:
                    assert np.array_equal(host(a), p)                        # the source is untouched
    assert ctx.arena_stats() == before
    ctx.close()


@pytest.mark.parametrize("n", [5, 300, 4099])
def test_shrink_mixed_parts_in_one_call(pcs, n):
    """Parts in place and out of place, with 16-, 4- and 1-byte granules, in
    one call (the moves of every part share two launches): kept entries
    against the oracle, for keep from 1 to n, so that kept sources inside and
    outside the destination range, and entries already in place, all occur."""
    rng = np.random.default_rng(80 + n)
    ctx = pcs.Context(arena(64 << 20))
    s = tricky_scores(rng, n)
    sd = scores_dev(s)
    sizes = [64, 28, 3, 200]
    in_place = [True, False, True, False]
    parts = [rng.integers(0, 256, size=n * eb, dtype=np.uint8) for eb in sizes]
    for keep in sorted({1, 2, n // 2, n - 1, n}):
        want_kept, want = oracle.bank_shrink(list(zip(parts, sizes)), s, keep)
        log("bank shrink mixed parts n", n, "keep", keep)
        srcs = [dev(p) for p in parts]
        dsts = [None if ip else torch.full((max(1, keep * eb),), 0xA5, dtype=torch.uint8, device="cuda")
                for eb, ip in zip(sizes, in_place)]
        kept = torch.full((max(1, keep),), -1, dtype=torch.int32, device="cuda")
        ctx.bank_shrink([(a, d, eb) for a, d, eb in zip(srcs, dsts, sizes)], sd, keep, kept)
        assert host(kept).view(np.uint32)[:keep].tolist() == want_kept.tolist()
        for p, a, d, eb, w, ip in zip(parts, srcs, dsts, sizes, want, in_place):
            got = host(a if ip else d)
            assert np.array_equal(got[:keep * eb], w)
            if ip:
                assert np.array_equal(got[keep * eb:], p[keep * eb:])
            else:
                assert np.array_equal(host(a), p)
    ctx.close()


def test_shrink_rejects_bad_arguments(pcs):
    ctx = pcs.Context(arena(16 << 20))
    before = ctx.arena_stats()
    a = torch.zeros(64 * 200, dtype=torch.uint8, device="cuda")   # room for 200 entries: the C checks decide
    b = torch.zeros(64 * 200, dtype=torch.uint8, device="cuda")
    y = torch.zeros(64 * 200, dtype=torch.uint8, device="cuda")
    s = scores_dev(np.arange(100, dtype=np.float32))
    bad = [
        ("keep > n", lambda: ctx.bank_shrink([(a, None, 64)], s, 101)),
        ("entry_bytes 0", lambda: ctx.bank_shrink([(a, None, 0)], s, 3)),
        ("overlap", lambda: ctx.bank_shrink([(a, a[64:], 64)], s, 10)),
        # One part writes where another reads (in place on y), or two parts
        # write the same bytes.
        ("part dst over part src", lambda: ctx.bank_shrink([(b, y, 64), (y, None, 64)], s, 10)),
        ("part dst over part dst", lambda: ctx.bank_shrink([(a, y, 64), (b, y[320:], 64)], s, 10)),
        ("too many entries", lambda: too_many()),
    ]

    def too_many():
        # 2^32 entries through the C ABI (checked before any part or score is
        # read, so small buffers stand in for the bank).
        import ctypes
        from paper_2607_21686_amd import _lib
        arr = (_lib.PcsBankPart * 1)(_lib.PcsBankPart(a.data_ptr(), a.data_ptr(), 1))
        st = _lib.lib().pcs_bank_shrink(ctx._h, arr, 1, 1 << 32, s.data_ptr(), 1, None)
        if st:
            raise pcs.PcsError(st, _lib.lib().pcs_last_error(ctx._h).decode())
    for name, f in bad:
        log("bank shrink error case:", name)
        with pytest.raises(pcs.PcsError) as e:
            f()
        assert e.value.code == pcs.E_INVAL, name
        assert ctx.arena_stats() == before, name
    ctx.bank_shrink([(a, None, 64)], scores_dev(np.zeros(0, dtype=np.float32)), 0)   # empty bank: nothing to do
    ctx.bank_shrink([(a, y, 64), (b, y[640:], 64)], s, 10)   # disjoint destinations in one buffer are fine
    ctx.close()


def test_shrink_refuses_when_scratch_does_not_fit(pcs):
    """In place, each part needs keep entries of staging scratch in the arena:
    an arena too small for it refuses the call with PCS_E_NOMEM before any
    launch, and neither the bank nor the arena changes."""
    ctx = pcs.Context(arena(2 << 20))
    before = ctx.arena_stats()
    rng = np.random.default_rng(5)
    n, eb = 200, 64 << 10
    bank = rng.integers(0, 256, size=n * eb, dtype=np.uint8)
    a = dev(bank)
    s = scores_dev(rng.random(n).astype(np.float32))
    with pytest.raises(pcs.PcsError) as e:
        ctx.bank_shrink([(a, None, eb)], s, 100)
    assert e.value.code == pcs.E_NOMEM
    assert np.array_equal(host(a), bank)
    assert ctx.arena_stats() == before
    # Keeping every entry in place moves nothing and needs no staging.
    kept = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    ctx.bank_shrink([(a, None, eb)], s, n, kept)
    assert host(kept).view(np.uint32).tolist() == list(range(n))
    assert np.array_equal(host(a), bank)
    # Out of place needs no staging: the same shrink into another buffer goes through.
    out = torch.empty(100 * eb, dtype=torch.uint8, device="cuda")
    ctx.bank_shrink([(a, out, eb)], s, 100)
    want_kept, (want,) = oracle.bank_shrink([(bank, eb)], s.cpu().numpy(), 100)
    assert np.array_equal(host(out), want)
    ctx.close()


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 4099, 70001])
def test_shrink_selection_unaligned_scores(pcs, n):
    """Scores that start 4, 8 or 12 bytes past a 16-byte boundary (the
    selection reads 16-byte groups and takes the ragged head and tail one
    score at a time): the kept indices match the oracle's."""
    rng = np.random.default_rng(90 + n)
    ctx = pcs.Context(arena(16 << 20))
    s = tricky_scores(rng, n)
    for off in (1, 2, 3):
        big = torch.zeros(n + 4, dtype=torch.float32, device="cuda")
        view = big[off:off + n]
        view.copy_(torch.from_numpy(np.ascontiguousarray(s, dtype=np.float32)))
        assert view.data_ptr() % 16 == 4 * off
        for keep in sorted({1, (n + 1) // 2, n}):
            log("bank shrink unaligned scores n", n, "offset", 4 * off, "keep", keep)
            want_kept, _ = oracle.bank_shrink([], s, keep)
            kept = torch.full((keep,), -1, dtype=torch.int32, device="cuda")
            ctx.bank_shrink([], view, keep, kept)
            assert host(kept).view(np.uint32).tolist() == want_kept.tolist()
    ctx.close()


def test_shrink_rejects_misaligned_scores(pcs):
    import ctypes
    from paper_2607_21686_amd import _lib
    ctx = pcs.Context(arena(16 << 20))
    s = scores_dev(np.arange(16, dtype=np.float32))
    kept = torch.zeros(4, dtype=torch.int32, device="cuda")
    st = _lib.lib().pcs_bank_shrink(ctx._h, None, 0, 8, s.data_ptr() + 2, 4, kept.data_ptr())
    assert st == pcs.E_INVAL
    assert b"aligned" in _lib.lib().pcs_last_error(ctx._h)
    ctx.close()


def test_shrink_selection_at_the_entry_limit(pcs):
    """Selection alone (no parts) over 2^32 - 1 scores, the most the call
    takes: every score 1.0 but a few planted lower ones, placed at both ends
    and in the last segments of the selection's lanes, so that the strided
    histogram loops and the last segment's bounds run up to 2^32.  The kept
    indices are the planted ones plus the lowest-indexed ties."""
    n = (1 << 32) - 1
    log("bank shrink selection n", n)
    ctx = pcs.Context(arena(16 << 20))
    s = torch.full((n,), 1.0, dtype=torch.float32, device="cuda")
    per = -(-n // 1024)
    planted = {n - 1: -2.0, n - 2: 0.5, (1 << 32) - 1024: 0.0, 1022 * per + 5: -1.0, 1023 * per: 0.25, 7: 0.75,
               per - 1: 0.5}
    for i, v in planted.items():
        s[i] = v
    for keep in (len(planted), len(planted) + 3):
        kept = torch.full((keep,), -1, dtype=torch.int32, device="cuda")
        ctx.bank_shrink([], s, keep, kept)
        ties = [i for i in range(10) if i not in planted][:keep - len(planted)]
        assert host(kept).view(np.uint32).tolist() == sorted(list(planted) + ties)
    # Only the two lowest: the last two lanes' segments hold them.
    kept = torch.full((2,), -1, dtype=torch.int32, device="cuda")
    ctx.bank_shrink([], s, 2, kept)
    assert host(kept).view(np.uint32).tolist() == sorted([n - 1, 1022 * per + 5])
    del s
    torch.cuda.empty_cache()
    ctx.close()


def test_shrink_then_incremental_checkpoint_config2(pcs):
    """The memory bank configuration at its full 512 entries: checkpoint,
    shrink to 12% keyed by pose distance to the anchor, incremental
    checkpoint of the shrunk bank, restore both."""
    bank = W.config2(1)
    E, le, pe = 512, bank.latent_entry_bytes, bank.pose_entry_bytes
    lat, pos = dev(bank.latents), dev(bank.poses)
    ctx = pcs.Context(arena(512 << 20))
    st = oracle.Store()

    def plan(e):
        return [pcs.flat(lat, e * le), pcs.flat(pos, e * pe)]

    log("config 2: full checkpoint of 512 entries")
    g0 = ctx.checkpoint(plan(E), hash=True)
    o0 = st.checkpoint(bank.prefix(E))
    s = W.pose_scores(bank, E, anchor=0)
    keep = pcs.keep_count(0.12, E)
    assert keep == oracle.keep_count(0.12, E) == 61
    kept = torch.zeros(keep, dtype=torch.int32, device="cuda")
    log("config 2: shrink to", keep, "entries")
    ctx.bank_shrink([(lat, None, le), (pos, None, pe)], scores_dev(s), keep, kept)
    want_kept, (nl, npo) = oracle.bank_shrink([(bank.latents, le), (bank.poses, pe)], s, keep)
    assert host(kept).view(np.uint32).tolist() == want_kept.tolist()
    assert 0 in want_kept.tolist()                      # the anchor itself is the most relevant entry
    log("config 2: incremental checkpoint of the shrunk bank")
    g1 = ctx.checkpoint(plan(keep), parent=g0)
    o1 = st.checkpoint([nl, npo], parent=o0)
    stored_o = sum(1 for b in range(2) for arr, off in st.snapshot(o1).where[b] if arr is st.snapshot(o1).payload)
    info = ctx.info(g1)
    assert info["incremental"] == 1 and info["dirty_chunks"] == stored_o
    assert info["state_bytes"] == keep * (le + pe)
    outs = [torch.empty(keep * le, dtype=torch.uint8, device="cuda"), torch.empty(keep * pe, dtype=torch.uint8, device="cuda")]
    ctx.restore(g1, [pcs.flat(o) for o in outs])
    assert np.array_equal(host(outs[0]), nl) and np.array_equal(host(outs[1]), npo)
    full = [torch.empty(E * le, dtype=torch.uint8, device="cuda"), torch.empty(E * pe, dtype=torch.uint8, device="cuda")]
    ctx.restore(g0, [pcs.flat(o) for o in full])
    assert np.array_equal(host(full[0]), bank.latents[:E * le]) and np.array_equal(host(full[1]), bank.poses[:E * pe])
    ctx.close()

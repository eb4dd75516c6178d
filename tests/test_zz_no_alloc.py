"""pcs_fingerprint_noalloc (the entry point for callers that cannot allocate)
against pcs_fingerprint, through the C ABI: bit-identical chunk
fingerprints, buffer roots and session roots on consecutive calls of
shrinking size (device-table jobs, then a job whose tables ride in the kernel
arguments), and the same values as the oracle.  Its limits are refused on the
host with nothing enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.gpu_util import arena, dev, log, u64, zeros_u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


def _abi():
    from paper_2607_21686_amd import _lib
    return _lib.lib()


def _call(ctx, fn, descs, T, n):
    """One fingerprint entry point through the C ABI into fresh outputs."""
    h, r, s = zeros_u64(T), zeros_u64(n), zeros_u64(1)
    arr = (ctx_buf_array(descs))
    st = fn(ctx._h, arr, len(descs), h.data_ptr(), r.data_ptr(), s.data_ptr())
    assert st == 0, _abi().pcs_last_error(ctx._h)
    return u64(h)[:T], u64(r)[:n], int(u64(s)[0])


def ctx_buf_array(descs):
    import paper_2607_21686_amd as P
    return P.BufArray(descs).arr


def _job(pcs, rng, sizes, ring=None):
    """Flat buffers of the given sizes (+ an optional wrapping ring); their
    device descriptors and the logical bytes the oracle sees."""
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    d = [dev(b) for b in bufs]
    descs = [pcs.flat(t, n) for t, n in zip(d, sizes)]
    logical = list(bufs)
    if ring is not None:
        g = ring
        rb = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
        t = dev(rb)
        d.append(t)
        descs.append(pcs.ring(t, g.outer, g.capacity, g.row_bytes, g.head, g.window, g.outer_stride))
        logical.append(oracle.ring_window(rb, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window))
    return descs, logical, d


def _check(pcs, ctx, descs, logical, label):
    n = len(descs)
    T = sum(oracle.chunk_count(b.size) for b in logical)
    log("no-alloc fingerprint:", label, "buffers", n, "chunks", T)
    L = _abi()
    got = _call(ctx, L.pcs_fingerprint_noalloc, descs, T, n)
    ref = _call(ctx, L.pcs_fingerprint, descs, T, n)
    assert np.array_equal(got[0], ref[0]), "chunk fingerprints differ from pcs_fingerprint"
    assert np.array_equal(got[1], ref[1]), "buffer roots differ from pcs_fingerprint"
    assert got[2] == ref[2], "session root differs from pcs_fingerprint"
    h, r, s = oracle.fingerprint(logical)
    assert np.array_equal(got[0], h) and np.array_equal(got[1], r) and got[2] == s, "differs from the oracle"


def test_noalloc_matches_fingerprint_on_shrinking_calls(pcs):
    rng = np.random.default_rng(701)
    ctx = pcs.Context(arena(64 << 20))
    before = ctx.arena_stats()
    # 1: device tables (21 buffers), whole-group tiles (> 128 groups), a wrapping ring.
    ring = W.Ring(6, 40, 2048, 33, 24, 40 * 2048 + 4096)
    sizes = [24 << 20, 8 << 20] + [int(rng.integers(0, 5 * 4096)) for _ in range(18)]
    descs, logical, keep1 = _job(pcs, rng, sizes, ring)
    _check(pcs, ctx, descs, logical, "large, device tables")
    # 2: smaller, still device tables (17 buffers), sub-tiles (<= 128 groups).
    sizes = [3 << 20] + [int(rng.integers(1, 3 * 4096)) for _ in range(16)]
    descs, logical, keep2 = _job(pcs, rng, sizes)
    _check(pcs, ctx, descs, logical, "smaller, device tables")
    # 3: smaller again, tables in the kernel arguments (3 buffers).
    descs, logical, keep3 = _job(pcs, rng, [5000, 1, 64 * 4096 + 8])
    _check(pcs, ctx, descs, logical, "small, argument tables")
    # 4: empty buffers only (no chunks; roots of the empty input).
    descs, logical, keep4 = _job(pcs, rng, [0, 0])
    _check(pcs, ctx, descs, logical, "empty buffers")
    assert ctx.arena_stats() == before, "the no-alloc entry point took arena space"
    ctx.close()


def test_noalloc_outputs_optional_and_no_timing_events(pcs):
    rng = np.random.default_rng(702)
    ctx = pcs.Context(arena(16 << 20))
    sizes = [int(rng.integers(1, 9 * 4096)) for _ in range(20)]
    descs, logical, keep = _job(pcs, rng, sizes)
    T = sum(oracle.chunk_count(n) for n in sizes)
    h = zeros_u64(T)
    ctx.set_timing(True)
    ctx.fingerprint_noalloc(descs, h)  # chunk fingerprints only, no roots
    ctx.fingerprint_noalloc(descs, None, None, zeros_u64(1))  # session root only
    assert ctx.kernel_time("hash")[0] == 0 and ctx.kernel_time("map")[0] == 0 and ctx.kernel_time("merkle")[0] == 0
    ctx.set_timing(False)
    assert np.array_equal(u64(h)[:T], oracle.fingerprint(logical)[0])
    ctx.close()


def test_noalloc_limits_refused(pcs):
    ctx = pcs.Context(arena(16 << 20))
    t = torch.zeros(16, dtype=torch.uint8, device="cuda")
    many = pcs.BufArray([pcs.flat(t, 1)] * 4097)
    L = _abi()
    st = L.pcs_fingerprint_noalloc(ctx._h, many.arr, len(many), None, None, None)
    assert st == pcs.E_INVAL and b"4096" in L.pcs_last_error(ctx._h)
    # A job whose scratch exceeds 16 MiB: 4096 buffers of 32 MiB (128 groups
    # each, 524,288 groups in all) over one tensor (reading a range several
    # times is allowed; the call is refused before anything is enqueued).
    big = torch.zeros(32 << 20, dtype=torch.uint8, device="cuda")
    huge = pcs.BufArray([pcs.flat(big)] * 4096)
    st = L.pcs_fingerprint_noalloc(ctx._h, huge.arr, len(huge), None, None, None)
    assert st == pcs.E_INVAL and b"scratch" in L.pcs_last_error(ctx._h), L.pcs_last_error(ctx._h)
    torch.cuda.synchronize()
    ctx.close()

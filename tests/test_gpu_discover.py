"""GPU parity of the discovery procedure (pcs_discover; Sec. 4, procedure
FINGERPRINT) against the oracle.

Synthetic probes (a closed-form D of the snapshot mask) check the
procedure's decisions and that every snapshot it hands to the probe holds
exactly the masked components, byte for byte, with the control's one wrong
bit where it belongs.  The mock world model then runs end to end on the
GPU: subset checkpoints and restores through libpcs, D from GPU
fingerprints, against the oracle's CPU model and procedure."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from oracle import discover as OD
from oracle.mock_world import MockWorld
from tests.gpu_util import arena, dev, host, log
from tests.test_oracle_discover import table_probe
from workloads.mock_world import MockSpec, initial_state, trajectory

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


RING = W.Ring(3, 10, 32, 7, 9, 10 * 32 + 16)


def synthetic_components(pcs, rng):
    """Four flat components and one ring (the last) with random bytes; their
    logical bytes as the oracle sees them."""
    sizes = [5000, 16, 3 * 4096, 1]
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    g = RING
    ring = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical = bufs + [oracle.ring_window(ring, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)]
    d = [dev(b) for b in bufs] + [dev(ring)]
    descs = [pcs.flat(t, n) for t, n in zip(d, sizes)] + [pcs.ring(d[-1], g.outer, g.capacity, g.row_bytes,
                                                                   g.head, g.window, g.outer_stride)]
    return descs, logical


def restore_logical(pcs, ctx, snap, idx, logical):
    """Restores a subset snapshot (components idx, in order) into fresh
    buffers and returns each component's logical bytes (the ring into a
    ring of the same geometry at another head)."""
    g = RING
    dsts, outs = [], []
    for i in idx:
        if i == len(logical) - 1:
            t = torch.zeros(g.ring_bytes, dtype=torch.uint8, device="cuda")
            dsts.append(pcs.ring(t, g.outer, g.capacity, g.row_bytes, 2, g.window, g.outer_stride))
        else:
            t = torch.zeros(max(1, logical[i].size), dtype=torch.uint8, device="cuda")
            dsts.append(pcs.flat(t, logical[i].size))
        outs.append(t)
    ctx.restore(snap, dsts)
    got = []
    for i, t in zip(idx, outs):
        if i == len(logical) - 1:
            got.append(oracle.ring_window(host(t), g.outer, g.outer_stride, g.capacity, g.row_bytes, 2, g.window))
        else:
            got.append(host(t)[:logical[i].size])
    return got


FUNCS = {
    "necessity": (lambda m, c: 0.5 * (1 - m[0]) + 0.3 * (1 - m[2]) + (0.25 if c == 4 else 0.0), 4),
    "pair": (lambda m, c: 0.6 * (1 - m[0]) + 0.2 * (1 - max(m[3], m[4])) + (0.5 if c == 1 else 0.0), 1),
    "greedy": (lambda m, c: (0.0 if m[1] + m[2] + m[3] >= 2 else (0.5 if m[1] + m[2] + m[3] == 1 else 1.0)), 3),
    "ignored": (lambda m, c: 0.0, 0),
}


@pytest.mark.parametrize("name", sorted(FUNCS))
def test_discover_decisions_and_snapshots(pcs, name):
    f, control = FUNCS[name]
    rng = np.random.default_rng(81)
    descs, logical = synthetic_components(pcs, rng)
    k = len(descs)
    ctx = pcs.Context(arena(64 << 20))
    before = ctx.arena_stats()
    seen = []

    def probe(snap, mask):
        # Restore the snapshot and find which component, if any, carries a wrong value.
        idx = [i for i in range(k) if mask[i]]
        corrupt = -1
        for got, i in zip(restore_logical(pcs, ctx, snap, idx, logical), idx):
            diff = np.flatnonzero(got != logical[i])
            if diff.size:
                assert diff.tolist() == [0] and got[0] ^ logical[i][0] == 1, (name, i)
                assert corrupt == -1
                corrupt = i
        seen.append((mask, corrupt))
        return f(mask, corrupt)

    log("discover, synthetic probe", name)
    got = ctx.discover(descs, probe, eps=0.0, control=control)
    want = OD.discover(table_probe(f), k, 0.0, control=control)
    assert got == want, (got, want)
    assert seen[-1] == (tuple([1] * k), control)   # the control run: full snapshot, one wrong bit
    assert ctx.arena_stats() == before              # every snapshot was deleted
    ctx.close()


def test_discover_mock_world_matches_oracle(pcs):
    from workloads.mock_world_gpu import MockWorldGPU
    spec = MockSpec()
    seed = 11
    init = initial_state(spec, seed)
    wa, pa = trajectory(seed, 24, 8)
    log("mock world: warm-up on GPU and CPU")
    g = MockWorldGPU.from_host(spec, init)
    g.run(wa)
    o = MockWorld(spec, init)
    o.run(wa)
    anchor = o.parts()
    assert all(np.array_equal(host(a), b) for a, b in zip(g.parts, anchor)), "GPU and CPU models diverge"

    ctx = pcs.Context(arena(256 << 20))
    descs = [pcs.flat(t) for t in g.parts]
    # Reference: an uninterrupted continuation from the anchor (on a copy).
    ref_world = MockWorldGPU(spec, [t.clone() for t in g.parts])
    ref_frames = ref_world.run(pa)
    nref = pcs.chunk_counts([pcs.flat(ref_frames)])[1]
    ref_h = torch.zeros(nref, dtype=torch.int64, device="cuda")
    ctx.fingerprint([pcs.flat(ref_frames)], ref_h)

    def probe(snap, mask):
        w = MockWorldGPU.fresh(spec)
        ctx.restore(snap, [pcs.flat(w.parts[i]) for i in range(len(mask)) if mask[i]])
        return ctx.distance(ref_h, [pcs.flat(w.run(pa))])

    log("mock world: discover on GPU")
    got = ctx.discover(descs, probe, eps=0.0, control=1)
    ref_o = oracle.fingerprint([MockWorld(spec, anchor).run(pa)])[0]
    assert np.array_equal(host(ref_h).view(np.uint64), ref_o)
    want = OD.discover(OD.mock_probe(spec, anchor, pa, ref_o), 8, 0.0, control=1)
    assert got == want, (got, want)
    assert got["pcs"] == [1, 1, 1, 1, 0, 0, 1, 0] and got["control_ok"] == 1
    assert all(np.array_equal(host(a), b) for a, b in zip(g.parts, anchor)), "the probes changed the live state"
    ctx.close()


def test_discover_errors(pcs):
    rng = np.random.default_rng(82)
    descs, logical = synthetic_components(pcs, rng)
    ctx = pcs.Context(arena(32 << 20))
    before = ctx.arena_stats()

    def raising(snap, mask):
        raise KeyError("probe failed")

    with pytest.raises(KeyError):
        ctx.discover(descs, raising)
    with pytest.raises(pcs.PcsError) as e:
        ctx.discover(descs, lambda s, m: math.nan)
    assert e.value.code == pcs.E_PROBE
    with pytest.raises(pcs.PcsError) as e:
        ctx.discover(descs, lambda s, m: -1.0)
    assert e.value.code == pcs.E_PROBE
    for bad in (dict(control=len(descs)), dict(eps=-1.0)):
        with pytest.raises(pcs.PcsError) as e:
            ctx.discover(descs, lambda s, m: 0.0, **bad)
        assert e.value.code == pcs.E_INVAL, bad
    empty = [pcs.flat(torch.zeros(16, dtype=torch.uint8, device="cuda"), 0)]
    with pytest.raises(pcs.PcsError) as e:
        ctx.discover(empty, lambda s, m: 0.0, control=0)
    assert e.value.code == pcs.E_INVAL
    many = [descs[1]] * 65
    with pytest.raises(pcs.PcsError) as e:
        ctx.discover(many, lambda s, m: 0.0)
    assert e.value.code == pcs.E_INVAL
    assert ctx.arena_stats() == before
    ctx.close()


def _distance_abi(pcs, ctx, ref, bufs):
    """pcs_distance through the C ABI: (differing chunks, distance)."""
    import ctypes
    from paper_2607_21686_amd import _lib
    arr = pcs.BufArray(bufs)
    cnt, d = ctypes.c_uint64(), ctypes.c_double()
    st = _lib.lib().pcs_distance(ctx._h, arr.arr, len(bufs), ref.data_ptr() if ref is not None else None,
                                 ctypes.byref(cnt), ctypes.byref(d))
    assert st == 0, _lib.lib().pcs_last_error(ctx._h)
    return int(cnt.value), float(d.value)


@pytest.mark.parametrize("case", ["small", "large"])
def test_distance_counts_differing_chunks(pcs, case):
    """D = differing chunks / chunks, against the oracle's fingerprints of the
    same bytes and of a reference copy with chosen chunks changed (Sec. 4's
    metric, taken bit-exactly).  'small' carries its tables in the kernel
    arguments and runs as sub-tiles; 'large' (more than 16 buffers, more than
    128 groups) uploads them and runs whole-group tiles."""
    rng = np.random.default_rng(91 if case == "small" else 92)
    if case == "small":
        sizes = [5000, 1, 3 * 4096 + 17, 64 * 4096 + 8, 0]
    else:
        sizes = [40 << 20] + [int(rng.integers(1, 3 * 4096)) for _ in range(20)]
    log("distance:", case, "sizes", sizes[:4], "...")
    bufs = [rng.integers(0, 256, size=n, dtype=np.uint8) for n in sizes]
    total = sum(oracle.chunk_count(n) for n in sizes)
    # The reference: the same bytes with a random set of chunks changed.
    refb = [b.copy() for b in bufs]
    changed = 0
    for b in refb:
        nch = oracle.chunk_count(b.size)
        for c in range(nch):
            if rng.random() < 0.3:
                o = c * 4096 + int(rng.integers(0, min(4096, b.size - c * 4096)))
                b[o] ^= 0x5A
                changed += 1
    ref_h = np.concatenate([oracle.fingerprint([b])[0] for b in refb])
    got_h = np.concatenate([oracle.fingerprint([b])[0] for b in bufs])
    want = int((ref_h != got_h).sum())
    assert want == changed
    ctx = pcs.Context(arena(64 << 20))
    d = [dev(b) for b in bufs]
    descs = [pcs.flat(t, n) for t, n in zip(d, sizes)]
    ref = dev(ref_h.view(np.uint8)).view(torch.int64)
    assert _distance_abi(pcs, ctx, ref, descs) == (want, want / total)
    assert ctx.distance(ref, descs) == want / total
    # Against itself: zero.
    same = dev(got_h.view(np.uint8)).view(torch.int64)
    assert _distance_abi(pcs, ctx, same, descs) == (0, 0.0)
    # A second call with fewer buffers (scratch reuse).
    n1 = oracle.chunk_count(sizes[0])
    assert _distance_abi(pcs, ctx, ref[:max(n1, 1)].contiguous(), descs[:1]) == (
        int((ref_h[:n1] != got_h[:n1]).sum()), float((ref_h[:n1] != got_h[:n1]).sum()) / n1)
    # No chunks at all: D = 0 and no reference needed.
    empty = [pcs.flat(d[0], 0)]
    assert _distance_abi(pcs, ctx, None, empty) == (0, 0.0)
    ctx.close()

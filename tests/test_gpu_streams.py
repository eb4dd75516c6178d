"""Contexts on their own HIP streams (every call is stream-ordered on the
context's stream, pcs.h): two contexts on two side streams with their calls
interleaved, checked against the oracle, and the order of a checkpoint
between writes made to its source on the same side stream (durability, I2,
on a stream other than the default one).  Streams keep the default
priority."""
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


def session(seed):
    """A flat frame of ragged size, a 16-byte RNG state and a wrapped ring."""
    rng = np.random.default_rng(seed)
    obs = rng.integers(0, 256, size=3 * 4096 * 17 + 123, dtype=np.uint8)
    rs = rng.integers(0, 256, size=16, dtype=np.uint8)
    g = W.Ring(3, 40, 1024, 33, 29)
    ring = rng.integers(0, 256, size=g.ring_bytes, dtype=np.uint8)
    logical = [obs, rs, oracle.ring_window(ring, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)]
    return obs, rs, g, ring, logical


def test_two_contexts_on_two_streams(pcs):
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    sessions = [session(90), session(91)]
    torch.cuda.synchronize()
    ctxs, tensors, outs, fps = [], [], [], []
    for k in range(2):
        obs, rs, g, ring, logical = sessions[k]
        t = [dev(obs), dev(rs), dev(ring)]
        torch.cuda.synchronize()
        tensors.append(t)
        ctxs.append(pcs.Context(arena(32 << 20), stream=streams[k]))
        total = sum(oracle.chunk_count(b.size) for b in logical)
        fps.append((zeros_u64(total), zeros_u64(3), zeros_u64(1)))
        outs.append([torch.zeros_like(t[0]), torch.zeros_like(t[1]), torch.zeros_like(t[2])])
    torch.cuda.synchronize()
    log("two contexts, interleaved calls on two side streams")
    snaps = [None, None]
    for k in range(2):       # both checkpoints enqueued before either restore
        obs, rs, g, ring, _ = sessions[k]
        t = tensors[k]
        plan = [pcs.flat(t[0]), pcs.flat(t[1]), pcs.ring(t[2], g.outer, g.capacity, g.row_bytes, g.head, g.window)]
        h, r, sr = fps[k]
        snaps[k] = ctxs[k].checkpoint(plan, hash=True, chunk_hashes=h, roots=r, session_root=sr)
    for k in (1, 0):
        obs, rs, g, ring, _ = sessions[k]
        o = outs[k]
        new_head = (g.head + 7) % g.capacity
        fork = ctxs[k].fork(snaps[k])
        ctxs[k].restore(fork, [pcs.flat(o[0]), pcs.flat(o[1]),
                               pcs.ring(o[2], g.outer, g.capacity, g.row_bytes, new_head, g.window)])
        ctxs[k].delete(fork)
    for s in streams:
        s.synchronize()
    for k in range(2):
        obs, rs, g, ring, logical = sessions[k]
        want_h, want_r, want_s = oracle.fingerprint(logical)
        h, r, sr = fps[k]
        assert np.array_equal(u64(h), want_h), k
        assert np.array_equal(u64(r), want_r), k
        assert int(u64(sr)[0]) == int(want_s), k
        o = outs[k]
        new_head = (g.head + 7) % g.capacity
        assert np.array_equal(host(o[0]), obs) and np.array_equal(host(o[1]), rs), k
        got = oracle.ring_window(host(o[2]), g.outer, g.outer_stride, g.capacity, g.row_bytes, new_head, g.window)
        assert np.array_equal(got, logical[2]), k
        ctxs[k].delete(snaps[k])
        ctxs[k].close()


def test_checkpoint_ordered_between_writes_on_a_side_stream(pcs):
    s = torch.cuda.Stream()
    n = 5 * 4096 + 48
    src = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = torch.zeros(n, dtype=torch.uint8, device="cuda")
    ctx = pcs.Context(arena(8 << 20), stream=s)
    torch.cuda.synchronize()
    log("checkpoint between two fills on a side stream")
    with torch.cuda.stream(s):
        src.fill_(0x5A)                         # before the checkpoint, on its stream
        snap = ctx.checkpoint([pcs.flat(src)], hash=True)
        src.fill_(0xC3)                         # after it, on the same stream
        ctx.restore(snap, [pcs.flat(out)])
    s.synchronize()
    assert np.all(host(out) == 0x5A)
    assert np.all(host(src) == 0xC3)
    ctx.delete(snap)
    ctx.close()

"""GPU parity at full size on the five seeded workload configurations, through
the C ABI, against the CPU oracle.  Every chunk fingerprint, buffer root and
session root of every configuration is compared with the oracle (the
1024-session batch one session at a time on a thread pool); snapshot bytes of
the batch on sessions of every head class; restored bytes equal their sources
and a restored ring fingerprints like the original.  Bit-exact throughout."""
import gc
import os

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


@pytest.fixture(autouse=True)
def free_memory():
    yield
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def fp_gpu(ctx, descs, total):
    ch, rt, sr = zeros_u64(total), zeros_u64(len(descs)), zeros_u64(1)
    ctx.fingerprint(descs, ch, rt, sr)
    return u64(ch)[:total], u64(rt)[:len(descs)], int(u64(sr)[0])


# --------------------------------------------------------------------- config 1

@pytest.mark.parametrize("variant", ["counter+1", "bit-flip"])
def test_config1_markovian(pcs, variant):
    c = W.config1(0)
    rep2 = c.buffers(2)
    if variant == "bit-flip":
        r = np.random.default_rng(99)
        flip = c.rng_state.copy()
        bit = int(r.integers(0, 128))
        flip[bit // 8] ^= np.uint8(1 << (bit % 8))
        rep2 = c.buffers(1)
        rep2[1] = flip
    reps = [c.buffers(1), rep2]
    log("config 1:", variant)
    ctx = pcs.Context(arena(64 << 20))
    total = sum(oracle.chunk_count(b.size) for b in reps[0])
    assert total == 48 + 1 + 6 * 32
    H = zeros_u64(2 * total)
    for k, rep in enumerate(reps):
        d = [dev(b) for b in rep]
        gh, gr, gs = fp_gpu(ctx, [pcs.flat(t) for t in d], total)
        oh, orr, osr = oracle.fingerprint(rep)
        assert np.array_equal(gh, oh) and np.array_equal(gr, orr) and gs == osr
        H[k * total:(k + 1) * total] = torch.from_numpy(oh.view(np.int64).copy()).cuda()
    cpb = [oracle.chunk_count(b.size) for b in reps[0]]
    nw = oracle.bitmap_words(cpb)
    bm = zeros_u64(nw)
    lab = torch.zeros(8, dtype=torch.uint8, device="cuda")
    ctx.classify(H, 2, cpb, bm, lab)
    obm, olab = oracle.classify(u64(H).reshape(2, total), cpb)
    assert np.array_equal(u64(bm)[:nw], obm) and np.array_equal(host(lab), olab)
    assert host(lab).tolist() == [0, 1, 0, 0, 0, 0, 0, 0]   # only the RNG state is must-snapshot
    # The snapshot plan: the must-snapshot buffers plus the observation the
    # Markovian model's restore reads (a buffer is state iff restore reads it).
    plan = [c.obs.reshape(-1), c.rng_state]
    d = [dev(b) for b in plan]
    snap = ctx.checkpoint([pcs.flat(t) for t in d], hash=True)
    info = ctx.info(snap)
    assert info["state_bytes"] == 196_608 + 16 == 196_624
    pay = torch.empty(info["stored_bytes"], dtype=torch.uint8, device="cuda")
    ctx.payload(snap, pay)
    assert np.array_equal(host(pay), oracle.pack(plan))
    out = [torch.empty_like(t) for t in d]
    ctx.restore(snap, [pcs.flat(o) for o in out])
    assert all(np.array_equal(host(o), b) for o, b in zip(out, plan))
    ctx.close()


# --------------------------------------------------------------------- config 2

def test_config2_growing_bank(pcs):
    bank = W.config2(1)
    lat, pos = dev(bank.latents), dev(bank.poses)
    ctx = pcs.Context(arena(512 << 20))
    st = oracle.Store()
    handles, parent_g, parent_o = [], 0, 0
    for j in range(1, 65):
        e = 8 * j
        log("config 2: step", j, "entries", e)
        plan = [pcs.flat(lat, e * bank.latent_entry_bytes), pcs.flat(pos, e * bank.pose_entry_bytes)]
        if j == 1:
            g = ctx.checkpoint(plan, hash=True)
            o = st.checkpoint(bank.prefix(e))
        else:
            g = ctx.checkpoint(plan, parent=parent_g)
            o = st.checkpoint(bank.prefix(e), parent_o)
        info = ctx.info(g)
        want = st.payload(o)
        assert info["stored_bytes"] == want.size, j
        if j > 1:
            # Only the appended entries (390 latent chunks) and the pose tail chunk(s) are stored.
            assert info["dirty_chunks"] in (391, 392), j
        pay = torch.empty(max(1, want.size), dtype=torch.uint8, device="cuda")
        ctx.payload(g, pay)
        assert np.array_equal(host(pay)[:want.size], want), j
        sh = zeros_u64(info["total_chunks"])
        ctx.stored_hashes(g, sh)
        assert np.array_equal(u64(sh)[:info["total_chunks"]], np.concatenate(st.snapshot(o).hashes)), j
        handles.append(g)
        parent_g, parent_o = g, o
    assert ctx.info(handles[-1])["state_bytes"] == 512 * 199_680 + 512 * 28 == 102_250_496
    order = np.random.default_rng(1).permutation(64)
    out_l = torch.empty(512 * bank.latent_entry_bytes, dtype=torch.uint8, device="cuda")
    out_p = torch.empty(512 * bank.pose_entry_bytes, dtype=torch.uint8, device="cuda")
    for j in order:
        e = 8 * (int(j) + 1)
        nl, npz = e * bank.latent_entry_bytes, e * bank.pose_entry_bytes
        ctx.restore(handles[j], [pcs.flat(out_l, nl), pcs.flat(out_p, npz)])
        # Append-only bank: snapshot j holds exactly the first 8(j+1) entries.
        assert torch.equal(out_l[:nl], lat[:nl]) and torch.equal(out_p[:npz], pos[:npz]), j
    ctx.close()


# --------------------------------------------------------------------- config 3

def test_config3_windowed_kv_ring(pcs):
    ring, g, h2 = W.config3_device(2)
    log("config 3: ring", g, "new head", h2)
    ctx = pcs.Context(arena((512 << 20) + (64 << 20)))
    desc = pcs.ring(ring, g.outer, g.capacity, g.row_bytes, g.head, g.window)
    nch = g.window_bytes // 4096
    ch, rt, sr = zeros_u64(nch), zeros_u64(1), zeros_u64(1)
    snap = ctx.checkpoint([desc], hash=True, chunk_hashes=ch, roots=rt, session_root=sr)
    info = ctx.info(snap)
    assert info["state_bytes"] == 1 << 29 and info["stored_bytes"] == 1 << 29   # window, not the 1 GiB ring
    host_ring = host(ring)
    logical = oracle.ring_window(host_ring, g.outer, g.outer_stride, g.capacity, g.row_bytes, g.head, g.window)
    del host_ring
    oh, orr, osr = oracle.fingerprint([logical])
    assert np.array_equal(u64(ch)[:nch], oh) and int(u64(rt)[0]) == int(orr[0]) and int(u64(sr)[0]) == osr
    pay = torch.empty(1 << 29, dtype=torch.uint8, device="cuda")
    ctx.payload(snap, pay)
    assert np.array_equal(host(pay), logical)
    del pay
    # Fork: two restores from one snapshot at new heads, mutated independently.
    f = ctx.fork(snap)
    a = torch.empty_like(ring)
    b = torch.empty_like(ring)
    h3 = (h2 + 1234) % g.capacity
    ctx.restore(snap, [pcs.ring(a, g.outer, g.capacity, g.row_bytes, h2, g.window)])
    ctx.restore(f, [pcs.ring(b, g.outer, g.capacity, g.row_bytes, h3, g.window)])
    got_a = oracle.ring_window(host(a), g.outer, g.outer_stride, g.capacity, g.row_bytes, h2, g.window)
    assert np.array_equal(got_a, logical)
    a.random_(0, 256)                         # mutate the first restore
    got_b = oracle.ring_window(host(b), g.outer, g.outer_stride, g.capacity, g.row_bytes, h3, g.window)
    assert np.array_equal(got_b, logical)
    # The restored ring at its new head fingerprints like the original window.
    rt2 = zeros_u64(1)
    ctx.fingerprint([pcs.ring(b, g.outer, g.capacity, g.row_bytes, h3, g.window)], None, rt2)
    assert int(u64(rt2)[0]) == int(orr[0])
    ctx.delete(snap)
    c = torch.empty_like(ring)
    ctx.restore(f, [pcs.ring(c, g.outer, g.capacity, g.row_bytes, h2, g.window)])
    got_c = oracle.ring_window(host(c), g.outer, g.outer_stride, g.capacity, g.row_bytes, h2, g.window)
    assert np.array_equal(got_c, logical)
    ctx.close()


# --------------------------------------------------------------------- config 4

def test_config4_classification_sweep(pcs):
    plan = W.config4_plan(3)
    log("config 4: %d buffers, %.2f GiB per replay, designated %s" % (len(plan.sizes), sum(plan.sizes) / 2**30,
                                                                      plan.designated))
    reps = W.config4_device(plan, 3)
    K, nb = plan.replays, len(plan.sizes)
    cpb = [oracle.chunk_count(n) for n in plan.sizes]
    total = sum(cpb)
    ctx = pcs.Context(arena(256 << 20))
    H = zeros_u64(K * total)
    # All K replays fingerprinted in one call: buffers in replay-major order.
    ctx.fingerprint([pcs.flat(t) for rep in reps for t in rep], H)
    nw = oracle.bitmap_words(cpb)
    bm = zeros_u64(nw)
    lab = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    ctx.classify(H, K, cpb, bm, lab)
    gh = u64(H)[:K * total].reshape(K, total)
    # Oracle fingerprints of every replay (an untouched buffer is the same bytes
    # in every replay, so its oracle fingerprints are computed once).
    base = [oracle.chunk_hashes(host(t)) for t in reps[0]]
    oh = np.zeros((K, total), dtype=np.uint64)
    for k in range(K):
        parts = []
        for b in range(nb):
            parts.append(base[b] if reps[k][b] is reps[0][b] else oracle.chunk_hashes(host(reps[k][b])))
        oh[k] = np.concatenate(parts)
    assert np.array_equal(gh, oh)
    obm, olab = oracle.classify(oh, cpb)
    assert np.array_equal(u64(bm)[:nw], obm)
    assert np.array_equal(host(lab), olab)
    # Ground truth by construction: the designated buffers, and exactly the rewritten chunks.
    assert host(lab).tolist() == [1 if b in plan.designated else 0 for b in range(nb)]
    word = 0
    got = u64(bm)[:nw]
    for b in range(nb):
        exp = np.zeros((cpb[b] + 63) // 64, dtype=np.uint64)
        if b in plan.designated:
            for k in range(2, K + 1):
                for c in plan.rewritten[(k, b)]:
                    exp[c // 64] |= np.uint64(1 << (c % 64))
        assert np.array_equal(got[word:word + exp.size], exp), b
        word += exp.size
    ctx.close()


# --------------------------------------------------------------------- config 5

def test_config5_batched_suspend_resume(pcs):
    plan = W.config5_plan(4)
    g, S = plan.ring, plan.sessions
    log("config 5: %d sessions" % S)
    rings, obs, rngs = W.config5_device(plan, 4)
    per_chunks = [g.window_bytes // 4096, oracle.chunk_count(plan.obs_bytes), 1]
    slot = sum(per_chunks) * 4096
    meta = ((8 * sum(per_chunks) + 32 + 4095) // 4096) * 4096
    ctx = pcs.Context(arena(S * (slot + meta) + (512 << 20)))
    plans = [[pcs.ring(rings[s], g.outer, g.capacity, g.row_bytes, plan.heads[s], g.window),
              pcs.flat(obs[s]), pcs.flat(rngs[s])] for s in range(S)]
    total = S * sum(per_chunks)
    ch, rt, sr = zeros_u64(total), zeros_u64(3 * S), zeros_u64(S)
    snaps = ctx.checkpoint_batch(plans, hash=True, chunk_hashes=ch, roots=rt, session_roots=sr)
    for s in snaps:
        assert ctx.info(s)["state_bytes"] == 34_752_528
    ghs, grt, gsr = u64(ch), u64(rt), u64(sr)
    per = sum(per_chunks)
    # Every session: chunk fingerprints, buffer roots and session root against
    # the oracle, from the session's raw ring bytes (the oracle takes the
    # window itself).  Sessions are copied to the host one at a time; the
    # oracle runs on a thread pool (its C calls release the interpreter lock).
    from concurrent.futures import ThreadPoolExecutor

    def check(s, r, o, q):
        logical = [oracle.ring_window(r, g.outer, g.outer_stride, g.capacity, g.row_bytes, plan.heads[s], g.window),
                   o, q]
        oh, orr, osr = oracle.fingerprint(logical)
        ok = (np.array_equal(ghs[s * per:(s + 1) * per], oh) and np.array_equal(grt[3 * s:3 * s + 3], orr)
              and int(gsr[s]) == osr)
        return s, ok

    log("config 5: oracle fingerprints of all %d sessions" % S)
    bad, pending = [], []
    with ThreadPoolExecutor(max_workers=max(1, min(12, (os.cpu_count() or 2) - 1))) as ex:
        for s in range(S):
            pending.append(ex.submit(check, s, host(rings[s]), host(obs[s]), host(rngs[s])))
            if len(pending) >= 24:
                bad += [k for k, ok in (f.result() for f in pending[:12]) if not ok]
                pending = pending[12:]
            if s % 256 == 255:
                log("config 5: %d sessions sent to the oracle" % (s + 1))
        bad += [k for k, ok in (f.result() for f in pending) if not ok]
    assert not bad, "sessions whose fingerprints differ from the oracle: %s" % bad[:20]
    # Snapshot bytes against the oracle's canonical payload on sessions of
    # every head class: a window that does not wrap, one that wraps between
    # chunks, one that wraps inside a chunk (2048-byte rows, odd head).
    C, Wn = g.capacity, g.window
    classes = {"no wrap": [s for s in range(S) if plan.heads[s] + Wn <= C],
               "wrap between chunks": [s for s in range(S) if plan.heads[s] + Wn > C and plan.heads[s] % 2 == 0],
               "wrap inside a chunk": [s for s in range(S) if plan.heads[s] + Wn > C and plan.heads[s] % 2 == 1]}
    sample = sorted(set([0, 1, 511, S - 1] + [x for v in classes.values() for x in v[:6]]))
    assert all(len(v) >= 6 for v in classes.values()) and len(sample) >= 16
    for s in sample:
        log("config 5: snapshot bytes of session", s, "head", plan.heads[s])
        r = host(rings[s])
        logical = [oracle.ring_window(r, g.outer, g.outer_stride, g.capacity, g.row_bytes, plan.heads[s], g.window),
                   host(obs[s]), host(rngs[s])]
        pay = torch.empty(ctx.info(snaps[s])["stored_bytes"], dtype=torch.uint8, device="cuda")
        ctx.payload(snaps[s], pay)
        assert np.array_equal(host(pay), oracle.pack(logical)), s
        del pay
    # Restore a random half in permuted order at new heads, in one launch.
    order, heads = plan.restore_order, plan.restore_heads
    R = len(order)
    dr = torch.empty(R, g.ring_bytes, dtype=torch.uint8, device="cuda")
    do = torch.empty(R, plan.obs_bytes, dtype=torch.uint8, device="cuda")
    dg = torch.empty(R, 16, dtype=torch.uint8, device="cuda")
    dsts = [[pcs.ring(dr[k], g.outer, g.capacity, g.row_bytes, heads[k], g.window), pcs.flat(do[k]),
             pcs.flat(dg[k])] for k in range(R)]
    ctx.restore_batch([snaps[s] for s in order], dsts)
    # Every restored session equals its source, byte for byte (any-size property).
    ar = torch.arange(g.window, device="cuda")
    for k, s in enumerate(order):
        src = rings[s].view(g.outer, g.capacity, g.row_bytes)[:, (ar + plan.heads[s]) % g.capacity]
        dst = dr[k].view(g.outer, g.capacity, g.row_bytes)[:, (ar + heads[k]) % g.capacity]
        assert torch.equal(src, dst), s
        assert torch.equal(do[k], obs[s]) and torch.equal(dg[k], rngs[s]), s
    # Restored sessions fingerprint like their checkpoints (roots of every restored session).
    rroots, rsr = zeros_u64(3 * R), zeros_u64(1)
    ctx.fingerprint([b for d in dsts for b in d], None, rroots)
    want = np.concatenate([grt[3 * s:3 * s + 3] for s in order])
    assert np.array_equal(u64(rroots)[:3 * R], want)
    ctx.close()

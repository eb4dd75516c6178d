"""Seeded random sequences of operations on one context with a tight arena,
checked against a host model of the buffers and the CPU oracle.

Two session plans share the context: P1 = {flat of varying length, 16-byte
flat, wrapped ring of 2 x 16 rows of 1 KiB} (tables in the kernel
arguments) and P2 = {flat of varying length, 40 rings of 8 rows of 512 B}
(80 runs when every window wraps, which takes the device-table path).
Operations: writes to the sources (bytes, valid lengths, ring heads), full
checkpoints with or without fingerprints, checkpoints of both sessions in
one batch, incremental checkpoints against any live snapshot of the same
plan, forks, deletes in any order (parents die before their incremental
children), restores into fresh destinations at new ring heads, and
verified restores.  Every restore must give back the logical bytes the
snapshot was taken of, every fingerprint output must equal the oracle's,
and an arena too small for a checkpoint may only refuse it (PCS_E_NOMEM,
no handle), never corrupt what it holds."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import arena, dev, host, log, u64, zeros_u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pcs():
    import paper_2607_21686_amd as P
    return P


class Flat:
    def __init__(self, rng, cap, nbytes):
        self.cap = cap
        self.nbytes = nbytes
        self.h = rng.integers(0, 256, size=cap, dtype=np.uint8)
        self.d = dev(self.h)

    def logical(self):
        return self.h[:self.nbytes].copy()

    def desc(self, pcs):
        return pcs.flat(self.d, self.nbytes)

    def write(self, rng):
        if rng.random() < 0.3:
            self.nbytes = int(rng.integers(0, self.cap + 1))
        for _ in range(int(rng.integers(1, 4))):
            a = int(rng.integers(0, self.cap))
            b = min(self.cap, a + int(rng.integers(1, 6000)))
            self.h[a:b] = rng.integers(0, 256, size=b - a, dtype=np.uint8)
        self.d.copy_(torch.from_numpy(self.h))


class Ring:
    def __init__(self, rng, outer, capacity, row, window):
        self.outer, self.capacity, self.row, self.window = outer, capacity, row, window
        self.stride = capacity * row
        self.head = int(rng.integers(0, capacity))
        self.h = rng.integers(0, 256, size=outer * self.stride, dtype=np.uint8)
        self.d = dev(self.h)

    def window_of(self, ring_bytes, head):
        return oracle.ring_window(ring_bytes, self.outer, self.stride, self.capacity, self.row, head, self.window)

    def logical(self):
        return self.window_of(self.h, self.head)

    def desc(self, pcs, t=None, head=None):
        return pcs.ring(self.d if t is None else t, self.outer, self.capacity, self.row,
                        self.head if head is None else head, self.window)

    def write(self, rng):
        if rng.random() < 0.5:
            self.head = int(rng.integers(0, self.capacity))
        for _ in range(int(rng.integers(1, 5))):
            o = int(rng.integers(0, self.outer))
            r = int(rng.integers(0, self.capacity))
            a = o * self.stride + r * self.row
            self.h[a:a + self.row] = rng.integers(0, 256, size=self.row, dtype=np.uint8)
        self.d.copy_(torch.from_numpy(self.h))


def make_plans(rng):
    p1 = [Flat(rng, 150_000, 123_457), Flat(rng, 16, 16), Ring(rng, 2, 16, 1024, 12)]
    p2 = [Flat(rng, 40_000, 40_000), Ring(rng, 40, 8, 512, 6)]
    return [p1, p2]


def fingerprint_outputs(plan, logical):
    total = sum(oracle.chunk_count(x.size) for x in logical)
    return zeros_u64(total), zeros_u64(len(plan)), zeros_u64(1), total


def check_fingerprints(logical, ch, rt, sr, total):
    want_h, want_r, want_s = oracle.fingerprint(logical)
    assert np.array_equal(u64(ch)[:total], want_h)
    assert np.array_equal(u64(rt)[:len(logical)], want_r)
    assert int(u64(sr)[0]) == int(want_s)


def restore_and_check(pcs, ctx, snap, plan, expect, rng, verify):
    """Restores `snap` into fresh destinations (rings at a random new head),
    through the verified restore when `verify`, and compares the logical
    bytes with `expect`."""
    dsts, reads = [], []
    for b, want in zip(plan, expect):
        if isinstance(b, Flat):
            t = torch.randint(0, 256, (max(want.size, 1),), dtype=torch.uint8, device="cuda")
            dsts.append(pcs.flat(t, want.size))
            reads.append(lambda t=t, n=want.size: host(t)[:n])
        else:
            t = torch.randint(0, 256, (b.outer * b.stride,), dtype=torch.uint8, device="cuda")
            head = int(rng.integers(0, b.capacity))
            dsts.append(b.desc(pcs, t, head))
            reads.append(lambda t=t, b=b, head=head: b.window_of(host(t), head))
    if verify:
        words = sum((oracle.chunk_count(w.size) + 63) // 64 for w in expect)
        bad = zeros_u64(words)
        labels = torch.full((len(expect),), 7, dtype=torch.uint8, device="cuda")
        ctx.restore_verify(snap, dsts, bad, labels)
        assert not u64(bad)[:words].any()
        assert not host(labels).any()
    else:
        ctx.restore(snap, dsts)
    for read, want in zip(reads, expect):
        assert np.array_equal(read(), want)


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_random_operation_sequences(pcs, seed):
    rng = np.random.default_rng(seed)
    plans = make_plans(rng)
    ctx = pcs.Context(arena(3 << 20))
    live = {}  # handle -> (plan index, expected logical bytes, has fingerprints)
    counts = {}
    ops = ["write", "full", "batch", "incremental", "fork", "delete", "restore"]
    weights = np.array([20, 10, 4, 18, 8, 20, 20], dtype=float)
    log("random operations, seed", seed)
    try:
        for step in range(300):
            op = ops[int(rng.choice(len(ops), p=weights / weights.sum()))]
            if op in ("incremental", "fork", "delete", "restore") and not live:
                op = "full"
            counts[op] = counts.get(op, 0) + 1
            if op == "write":
                plan = plans[int(rng.integers(0, 2))]
                plan[int(rng.integers(0, len(plan)))].write(rng)
                continue
            if op == "fork":
                h = int(rng.choice(list(live)))
                live[ctx.fork(h)] = live[h]
                continue
            if op == "delete":
                h = int(rng.choice(list(live)))
                ctx.delete(h)
                del live[h]
                continue
            try:
                if op == "restore":
                    h = int(rng.choice(list(live)))
                    p, expect, hashed = live[h]
                    restore_and_check(pcs, ctx, h, plans[p], expect, rng, hashed and rng.random() < 0.3)
                    if rng.random() < 0.7:
                        continue
                    # Roll the sources back to the snapshot (flat lengths as they
                    # were, rings at their current heads).
                    ctx.restore(h, [pcs.flat(b.d, want.size) if isinstance(b, Flat) else b.desc(pcs)
                                    for b, want in zip(plans[p], expect)])
                    for b, want in zip(plans[p], expect):
                        if isinstance(b, Flat):
                            b.nbytes = want.size
                            b.h[:b.nbytes] = want
                        else:
                            oracle.ring_place(want, b.h, b.outer, b.stride, b.capacity, b.row, b.head, b.window)
                    torch.cuda.synchronize()
                    for b in plans[p]:
                        assert np.array_equal(host(b.d), b.h)
                    continue
                if op == "batch":
                    logical = [[b.logical() for b in plan] for plan in plans]
                    rt = zeros_u64(sum(len(p) for p in plans))
                    sr = zeros_u64(2)
                    hs = ctx.checkpoint_batch([[b.desc(pcs) for b in plan] for plan in plans], hash=True,
                                              roots=rt, session_roots=sr)
                    roots = u64(rt)
                    for p in range(2):
                        _, want_r, want_s = oracle.fingerprint(logical[p])
                        off = sum(len(q) for q in plans[:p])
                        assert np.array_equal(roots[off:off + len(plans[p])], want_r)
                        assert int(u64(sr)[p]) == int(want_s)
                        live[hs[p]] = (p, logical[p], True)
                    continue
                p = int(rng.integers(0, 2))
                plan = plans[p]
                logical = [b.logical() for b in plan]
                descs = [b.desc(pcs) for b in plan]
                if op == "full":
                    hashed = bool(rng.random() < 0.6)
                    if hashed:
                        ch, rt, sr, total = fingerprint_outputs(plan, logical)
                        h = ctx.checkpoint(descs, hash=True, chunk_hashes=ch, roots=rt, session_root=sr)
                        check_fingerprints(logical, ch, rt, sr, total)
                    else:
                        h = ctx.checkpoint(descs)
                    live[h] = (p, logical, hashed)
                else:
                    parents = [k for k, v in live.items() if v[0] == p and v[2]]
                    if not parents:
                        counts[op] -= 1
                        continue
                    ch, rt, sr, total = fingerprint_outputs(plan, logical)
                    h = ctx.checkpoint(descs, parent=int(rng.choice(parents)), chunk_hashes=ch, roots=rt,
                                       session_root=sr)
                    check_fingerprints(logical, ch, rt, sr, total)
                    live[h] = (p, logical, True)
            except pcs.PcsError as e:
                assert e.code == pcs.E_NOMEM, e
                counts["nomem"] = counts.get("nomem", 0) + 1
                # Make room, as a caller would.
                for h in list(live)[: max(1, len(live) // 2)]:
                    ctx.delete(h)
                    del live[h]
        # Whatever is still alive restores correctly (a few handles are
        # dropped first so that device-table restores find scratch room).
        for h in list(live)[8:]:
            ctx.delete(h)
            del live[h]
        for h, (p, expect, hashed) in live.items():
            restore_and_check(pcs, ctx, h, plans[p], expect, rng, hashed)
        log("operations", counts, "live at the end", len(live))
        assert counts.get("incremental", 0) >= 20 and counts.get("restore", 0) >= 20
    finally:
        ctx.close()

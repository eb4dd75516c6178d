"""CPU oracle for the PCS fingerprint-and-checkpoint path.

TEST INFRASTRUCTURE ONLY.  The plain, slow, single-threaded definition the
GPU library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()``
and ``bench.py``'s CPU-baseline leg may import it; the GPU library never
does, and this package imports nothing from it.

The arithmetic lives in ``pcs_oracle.c`` (built with gcc into
``liboracle.so`` next to this file); this module marshals numpy arrays into
it and keeps the snapshot bookkeeping of the paper's contract (Sec. 3,
"The contract": checkpoint / restore / fork / delete over opaque handles, and
invariants I1-I4) as plain Python objects.

Every buffer here is a *logical* byte string: a flat buffer is its bytes, a
ring-buffered window is ``ring_window(...)`` of it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pcs_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

CHUNK = 4096
RECOMPUTABLE = 0
MUST_SNAPSHOT = 1


def build(force: bool = False) -> str:
    """Compiles ``pcs_oracle.c`` into ``liboracle.so`` (gcc, -O2, one thread)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared", "-o", tmp, _SRC],
                       check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _L():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        u64, u32, p = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
        lib.orc_xxh64.argtypes = [p, u64, u64]
        lib.orc_xxh64.restype = u64
        lib.orc_chunk_count.argtypes = [u64]
        lib.orc_chunk_count.restype = u64
        lib.orc_chunk_hashes.argtypes = [p, u64, p]
        lib.orc_chunk_hashes.restype = None
        lib.orc_node_hash.argtypes = [u64, u64]
        lib.orc_node_hash.restype = u64
        lib.orc_merkle_root.argtypes = [p, u64, p]
        lib.orc_merkle_root.restype = u64
        lib.orc_ring_window.argtypes = [p, u64, u64, u64, u64, u64, u64, p]
        lib.orc_ring_window.restype = None
        lib.orc_ring_place.argtypes = [p, u64, u64, u64, u64, u64, u64, p]
        lib.orc_ring_place.restype = None
        lib.orc_classify.argtypes = [p, u32, p, u32, p, p]
        lib.orc_classify.restype = u64
        lib.orc_payload_layout.argtypes = [p, u32, p]
        lib.orc_payload_layout.restype = u64
        lib.orc_dirty.argtypes = [p, p, p, p, u32, p]
        lib.orc_dirty.restype = u64
        lib.orc_bank_select.argtypes = [p, u32, u32, p]
        lib.orc_bank_select.restype = ctypes.c_int
        lib.orc_philox4x32_10.argtypes = [p, p, p]
        lib.orc_philox4x32_10.restype = None
        _lib = lib
    return _lib


def _bytes(x) -> np.ndarray:
    """A C-contiguous uint8 view of bytes / bytearray / any numpy array."""
    if isinstance(x, (bytes, bytearray, memoryview)):
        return np.frombuffer(bytes(x), dtype=np.uint8)
    a = np.ascontiguousarray(x)
    return a.reshape(-1).view(np.uint8)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- hashing

def xxh64(data, seed: int = 0) -> int:
    """XXH64 of a byte string (the xxHash specification's 64-bit hash)."""
    b = _bytes(data)
    return int(_L().orc_xxh64(_ptr(b), b.size, seed))


def chunk_count(nbytes: int) -> int:
    return int(_L().orc_chunk_count(nbytes))


def chunk_hashes(data) -> np.ndarray:
    """XXH64 (seed 0) of every 4096-byte chunk; the last chunk is the tail."""
    b = _bytes(data)
    out = np.zeros(chunk_count(b.size), dtype=np.uint64)
    _L().orc_chunk_hashes(_ptr(b), b.size, _ptr(out))
    return out


def node_hash(left: int, right: int) -> int:
    return int(_L().orc_node_hash(left, right))


def merkle_root(leaves) -> int:
    """Promote-odd binary Merkle root; no leaves gives XXH64 of b''."""
    lv = np.ascontiguousarray(leaves, dtype=np.uint64)
    work = np.zeros(max(lv.size, 1), dtype=np.uint64)
    return int(_L().orc_merkle_root(_ptr(lv), lv.size, _ptr(work)))


def fingerprint(buffers):
    """Chunk fingerprints, per-buffer roots and the session root.

    ``buffers``: list of logical byte strings.  Returns (concatenated chunk
    hashes in buffer order, roots[nbuf], session root = Merkle root over the
    buffer roots in plan order).
    """
    per = [chunk_hashes(b) for b in buffers]
    roots = np.array([merkle_root(h) for h in per], dtype=np.uint64)
    hashes = np.concatenate(per) if per else np.zeros(0, dtype=np.uint64)
    return hashes, roots, merkle_root(roots)


# ------------------------------------------------------------------- ring

def ring_window(ring, outer, outer_stride, capacity, row_bytes, head, window) -> np.ndarray:
    """Logical window (ring 0 rows head..head+W-1 mod C, then ring 1, ...)."""
    r = _bytes(ring)
    assert r.size >= (outer - 1) * outer_stride + capacity * row_bytes if outer else True
    out = np.zeros(outer * window * row_bytes, dtype=np.uint8)
    _L().orc_ring_window(_ptr(r), outer, outer_stride, capacity, row_bytes, head, window, _ptr(out))
    return out


def ring_place(logical, ring: np.ndarray, outer, outer_stride, capacity, row_bytes, head, window) -> None:
    """Writes a logical window into ``ring`` (uint8, modified in place) at ``head``."""
    lg = _bytes(logical)
    assert lg.size == outer * window * row_bytes
    assert ring.dtype == np.uint8 and ring.flags.c_contiguous
    _L().orc_ring_place(_ptr(lg), outer, outer_stride, capacity, row_bytes, head, window, _ptr(ring))


# --------------------------------------------------------------- classify

def bitmap_words(chunks_per_buf) -> int:
    return int(sum((int(c) + 63) // 64 for c in chunks_per_buf))


def classify(hashes, chunks_per_buf):
    """hashes: (K, total) uint64, replay-major.  Returns (bitmap, labels)."""
    h = np.ascontiguousarray(hashes, dtype=np.uint64)
    assert h.ndim == 2
    K = h.shape[0]
    cpb = np.ascontiguousarray(chunks_per_buf, dtype=np.uint64)
    assert int(cpb.sum()) == h.shape[1]
    bitmap = np.zeros(max(bitmap_words(cpb), 1), dtype=np.uint64)
    labels = np.zeros(max(cpb.size, 1), dtype=np.uint8)
    nw = _L().orc_classify(_ptr(h), K, _ptr(cpb), cpb.size, _ptr(bitmap), _ptr(labels))
    return bitmap[:nw], labels[:cpb.size]


# ------------------------------------------------------ full checkpoints

def payload_layout(nbytes):
    nb = np.ascontiguousarray(nbytes, dtype=np.uint64)
    offs = np.zeros(max(nb.size, 1), dtype=np.uint64)
    total = _L().orc_payload_layout(_ptr(nb), nb.size, _ptr(offs))
    return offs[:nb.size], int(total)


def pack(buffers) -> np.ndarray:
    """Canonical full snapshot: components 4096-aligned in plan order, zero padding."""
    bufs = [_bytes(b) for b in buffers]
    offs, total = payload_layout([b.size for b in bufs])
    payload = np.zeros(total, dtype=np.uint8)
    for b, o in zip(bufs, offs):
        payload[int(o):int(o) + b.size] = b
    return payload


def unpack(payload, nbytes):
    offs, _ = payload_layout(nbytes)
    p = _bytes(payload)
    return [p[int(o):int(o) + int(n)].copy() for o, n in zip(offs, nbytes)]


def dirty(hashes, counts, parent_hashes, parent_counts):
    h = np.ascontiguousarray(hashes, dtype=np.uint64)
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    ph = np.ascontiguousarray(parent_hashes, dtype=np.uint64)
    pc = np.ascontiguousarray(parent_counts, dtype=np.uint64)
    assert c.size == pc.size and int(c.sum()) == h.size and int(pc.sum()) == ph.size
    d = np.zeros(max(h.size, 1), dtype=np.uint8)
    nd = _L().orc_dirty(_ptr(h), _ptr(c), _ptr(ph), _ptr(pc), c.size, _ptr(d))
    return d[:h.size].astype(bool), int(nd)


# -------------------------------------------------- the contract (Sec. 3)

class _Snapshot:
    """An immutable snapshot: sizes, per-buffer chunk fingerprints, payload
    bytes, and for every chunk the (payload array, offset) that holds it."""

    def __init__(self, nbytes, hashes, payload, where, parent):
        self.nbytes = list(nbytes)
        self.hashes = hashes          # list of uint64 arrays, one per buffer
        self.payload = payload        # uint8 array, never written again
        self.where = where            # where[b][i] = (payload array, offset)
        self.parent = parent          # keeps the chain's payloads alive
        self.roots = np.array([merkle_root(h) for h in hashes], dtype=np.uint64)
        self.session_root = merkle_root(self.roots)


class Store:
    """checkpoint / restore / fork / delete over opaque integer handles.

    A full checkpoint stores every buffer (canonical layout).  An incremental
    checkpoint against a parent stores only the chunks whose fingerprint is
    new or changed, each in its own 4096-byte slot (zero padded), in
    increasing (buffer, chunk) order; every other chunk is found where the
    parent found it.  Fork is a second handle on the same immutable snapshot;
    delete drops one handle.
    """

    def __init__(self):
        self._snaps = {}
        self._next = 1

    def _new_handle(self, snap):
        h = self._next
        self._next += 1
        self._snaps[h] = snap
        return h

    def checkpoint(self, buffers, parent: int = 0) -> int:
        bufs = [_bytes(b).copy() for b in buffers]
        nbytes = [b.size for b in bufs]
        hashes = [chunk_hashes(b) for b in bufs]
        if parent == 0:
            payload = pack(bufs)
            offs, _ = payload_layout(nbytes)
            where = [[(payload, int(offs[b]) + CHUNK * i) for i in range(len(hashes[b]))]
                     for b in range(len(bufs))]
            return self._new_handle(_Snapshot(nbytes, hashes, payload, where, None))
        par = self._snaps[parent]
        assert len(par.nbytes) == len(bufs), "incremental plan must have the parent's buffer count"
        d, nd = dirty(np.concatenate(hashes) if hashes else [],
                      [len(h) for h in hashes],
                      np.concatenate(par.hashes) if par.hashes else [],
                      [len(h) for h in par.hashes])
        payload = np.zeros(nd * CHUNK, dtype=np.uint8)
        where, k, slot = [], 0, 0
        for b in range(len(bufs)):
            wb = []
            for i in range(len(hashes[b])):
                if d[k]:
                    piece = bufs[b][CHUNK * i:CHUNK * (i + 1)]
                    payload[slot * CHUNK:slot * CHUNK + piece.size] = piece
                    wb.append((payload, slot * CHUNK))
                    slot += 1
                else:
                    wb.append(par.where[b][i])
                k += 1
            where.append(wb)
        return self._new_handle(_Snapshot(nbytes, hashes, payload, where, par))

    def restore(self, handle: int):
        s = self._snaps[handle]
        out = []
        for b, n in enumerate(s.nbytes):
            buf = np.zeros(n, dtype=np.uint8)
            for i, (arr, off) in enumerate(s.where[b]):
                ln = min(CHUNK, n - CHUNK * i)
                buf[CHUNK * i:CHUNK * i + ln] = arr[off:off + ln]
            out.append(buf)
        return out

    def fork(self, handle: int) -> int:
        return self._new_handle(self._snaps[handle])

    def delete(self, handle: int) -> None:
        del self._snaps[handle]

    def snapshot(self, handle: int) -> _Snapshot:
        return self._snaps[handle]

    def payload(self, handle: int) -> np.ndarray:
        return self._snaps[handle].payload

    def state_bytes(self, handle: int) -> int:
        """Logical bytes the snapshot restores (I4: the sum of its buffer sizes)."""
        return int(sum(self._snaps[handle].nbytes))


# ----------------------------------------- durable images (Sec. 7.2, I2)

IMAGE_MAGIC = b"PCSIMG01"


def export_image(buffers, layouts=None) -> bytes:
    """Self-contained image of a snapshot of logical byte strings.

    layouts[b] = (kind, row_bytes, window, outer) with kind 0 (flat, ring
    fields 0) or 1 (ring); default flat.  Layout, little-endian: magic, u32
    version 1, u32 n, u64 chunks, u64 state bytes, u64 payload bytes, u64
    flags 0; per buffer u32 kind, u32 0, u64 nbytes, u64 row_bytes, u64
    window, u64 outer, u64 0; n buffer roots, session root; all chunk
    fingerprints; zero padding to 4096; the canonical payload.
    """
    import struct
    bufs = [_bytes(b) for b in buffers]
    n = len(bufs)
    layouts = layouts or [(0, 0, 0, 0)] * n
    hashes, roots, sroot = fingerprint(bufs)
    payload = pack(bufs)
    head = IMAGE_MAGIC + struct.pack("<IIQQQQ", 1, n, hashes.size, sum(b.size for b in bufs), payload.size, 0)
    for b, (kind, row, win, outer) in zip(bufs, layouts):
        head += struct.pack("<IIQQQQQ", kind, 0, b.size, row, win, outer, 0)
    head += struct.pack("<%dQ" % (n + 1), *([int(r) for r in roots] + [sroot]))
    head += hashes.astype("<u8").tobytes()
    pad = (-len(head)) % CHUNK
    return head + b"\0" * pad + payload.tobytes()


# ---------------------------------------------------------------- bank shrink

def keep_count(fraction, n_entries: int) -> int:
    """Entries a shrink to `fraction` keeps (Sec. 7.5's 12%; Table 6's keep
    fractions 0.04-0.50, written as decimals): the fraction is the exact
    rational a decimal denotes (a float is read as the decimal it prints, so
    0.05 is 1/20, not its binary approximation); n x fraction is rounded to
    the nearest integer, an exact half to the even neighbour; at least 1 for
    a non-empty bank."""
    from fractions import Fraction
    f = Fraction(repr(fraction)) if isinstance(fraction, float) else Fraction(fraction)
    if not 0 <= f <= 1:
        raise ValueError("fraction must lie in [0, 1]")
    if n_entries <= 0:
        return 0
    return max(1, round(f * n_entries))


def bank_select(scores, keep: int) -> np.ndarray:
    """The `keep` best-ranked entries (lower score first; -0.0 before +0.0;
    NaN last; ties by lower index), in increasing index order (Sec. 5,
    Sec. 7.5, Tables 5-6)."""
    s = np.ascontiguousarray(scores, dtype=np.float32)
    out = np.zeros(max(1, keep), dtype=np.uint32)
    if _L().orc_bank_select(s.ctypes.data, s.size, keep, out.ctypes.data) != 0:
        raise ValueError("keep exceeds the number of entries")
    return out[:keep]


def bank_shrink(parts, scores, keep: int):
    """Shrinks a struct-of-arrays bank: parts = [(bytes of n entries, entry
    bytes), ...]; returns (kept indices, [the kept entries of each part, in
    index order, as one byte string each])."""
    n = np.asarray(scores).size
    kept = bank_select(scores, keep)
    out = []
    for data, eb in parts:
        a = _bytes(data)[:n * eb].reshape(n, eb) if n else np.zeros((0, eb), dtype=np.uint8)
        out.append(a[kept.astype(np.int64)].reshape(-1).copy())
    return kept, out


# ---------------------------------------------------------------- Philox4x32-10

def philox4x32_10(counter, key):
    """One Philox4x32-10 block: 4 uint32 outputs for a 4-word counter and a
    2-word key (SC'11 definition)."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _L().orc_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out

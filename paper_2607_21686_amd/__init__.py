"""MI355X (gfx950) byte layer of a Persistent Computational State runtime.

The paper ("Persistent Computational State: A Session-Centric Runtime for
Generative World Models") specifies PCS as a contract (Sec. 3): checkpoint /
restore / fork / delete over opaque handles, with invariants I1 round-trip,
I2 durability, I3 fork independence and I4 snapshot completeness, and it
decides which buffers are PCS by derivability.  This package is the GPU
layer under that contract: chunked XXH64 fingerprints with a Merkle
combine, cross-replay classification (must-snapshot vs recomputable),
packed-gather checkpoints (flat buffers, growing banks with incremental
checkpoints, ring-buffered KV windows) and scatter restore.

All work runs in libpcs.so's HIP kernels behind the C ABI of
``include/pcs.h``; this module only marshals torch tensors and streams.
PyTorch is used for device memory and streams.
"""
from __future__ import annotations

import ctypes

import torch

from ._lib import (CHUNK_BYTES, CKPT_HASH, E_CORRUPT, E_HANDLE, E_HIP, E_INVAL, E_NOMEM, E_PROBE, E_SHAPE, EXPORTS,
                   FLAT, MUST_SNAPSHOT, PROBE_FN, RECOMPUTABLE, RING, TIMING_DISPATCH, TIMING_EVENTS, TIMING_OFF,
                   PcsBankPart, PcsBuf, PcsDiscovery, PcsError, PcsSnapInfo, lib)

__all__ = ["Context", "PcsError", "BufArray", "u64_array", "flat", "ring", "chunk_counts", "keep_count", "CHUNK_BYTES", "CKPT_HASH", "FLAT", "RING",
           "RECOMPUTABLE", "MUST_SNAPSHOT", "E_INVAL", "E_NOMEM", "E_HANDLE", "E_SHAPE", "E_HIP", "E_CORRUPT", "E_PROBE",
           "EXPORTS"]

_L = lib()  # fails loudly if the HIP library is missing


def _ratio(fraction):
    """(numerator, denominator) of a retained fraction given as a Fraction, a
    decimal string, a (num, den) pair, or a float taken as the decimal it
    prints (0.05 -> 1/20): the exact rational the library rounds."""
    from fractions import Fraction
    if isinstance(fraction, tuple):
        return int(fraction[0]), int(fraction[1])
    f = Fraction(repr(fraction)) if isinstance(fraction, float) else Fraction(fraction)
    return f.numerator, f.denominator


def keep_count(fraction, n_entries: int) -> int:
    """Entries a shrink to `fraction` of a bank keeps (pcs_keep_count):
    n x fraction rounded to the nearest integer, halves to even, at least one
    entry of a non-empty bank (Table 6 lists the frames a fraction keeps of a
    bank of about 21)."""
    num, den = _ratio(fraction)
    out = ctypes.c_uint64()
    st = _L.pcs_keep_count(num, den, int(n_entries), ctypes.byref(out))
    if st:
        raise PcsError(st, "fraction must lie in [0, 1] (got %d/%d)" % (num, den))
    return int(out.value)


def _dev_ptr(t) -> int:
    if t is None:
        return 0
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous CUDA tensor")
    return t.data_ptr()


def flat(t: torch.Tensor, nbytes: int | None = None) -> PcsBuf:
    """A PCS_FLAT descriptor over a contiguous device tensor (or its first nbytes)."""
    size = t.numel() * t.element_size()
    n = size if nbytes is None else nbytes
    if n < 0 or n > size:
        raise ValueError("nbytes must lie in [0, tensor bytes]")
    b = PcsBuf(ptr=_dev_ptr(t), nbytes=n, kind=FLAT)
    b._tensor = t  # the descriptor keeps its memory alive until the call has been enqueued
    return b


def ring(t: torch.Tensor, outer: int, capacity: int, row_bytes: int, head: int, window: int,
         outer_stride: int | None = None) -> PcsBuf:
    """A PCS_RING descriptor: `outer` rings of `capacity` rows inside tensor t."""
    stride = capacity * row_bytes if outer_stride is None else outer_stride
    if min(outer, capacity, row_bytes, head, window, stride) < 0:
        raise ValueError("ring geometry must be non-negative")
    need = (outer - 1) * stride + capacity * row_bytes if outer else 0
    if need > t.numel() * t.element_size():
        raise ValueError("ring geometry exceeds the tensor")
    b = PcsBuf(ptr=_dev_ptr(t), nbytes=0, kind=RING, row_bytes=row_bytes, capacity=capacity, head=head,
               window=window, outer=outer, outer_stride=stride)
    b._tensor = t
    return b


class BufArray:
    """A prebuilt descriptor array (reuse it across calls to skip marshalling)."""

    def __init__(self, bufs):
        self.bufs = list(bufs)  # keeps the descriptors' tensors alive
        self.arr = (PcsBuf * max(1, len(self.bufs)))()
        for i, b in enumerate(self.bufs):
            self.arr[i] = b

    def __len__(self):
        return len(self.bufs)


def _host_ptr(a):
    """Address and byte size of a contiguous host buffer (numpy array or CPU tensor)."""
    import numpy as np
    if isinstance(a, torch.Tensor):
        if a.is_cuda or not a.is_contiguous():
            raise ValueError("expected a contiguous CPU tensor")
        return a.data_ptr(), a.numel() * a.element_size()
    if isinstance(a, np.ndarray):
        if not a.flags["C_CONTIGUOUS"]:
            raise ValueError("expected a contiguous array")
        return a.ctypes.data, a.nbytes
    raise TypeError("expected a numpy array or a CPU tensor")


def _array(bufs):
    if isinstance(bufs, BufArray):
        return bufs.arr
    return BufArray(bufs).arr


def u64_array(values):
    """A prebuilt ctypes uint64 array (e.g. chunks per buffer for classify)."""
    values = list(values)
    return (ctypes.c_uint64 * max(1, len(values)))(*[int(v) for v in values])


def chunk_counts(bufs):
    """(chunks of each descriptor, total) as pcs_chunk_counts computes them;
    validates the descriptors on the host."""
    arr = _array(bufs)
    out = (ctypes.c_uint64 * max(1, len(bufs)))()
    total = ctypes.c_uint64()
    st = _L.pcs_chunk_counts(arr, len(bufs), out, ctypes.byref(total))
    if st:
        raise PcsError(st, "invalid buffer descriptor")
    return [int(out[i]) for i in range(len(bufs))], int(total.value)


class Context:
    """A libpcs context over a caller-owned uint8 device arena, bound to a stream.

    Every call is enqueued on that stream and returns before its kernels
    run.  A tensor named in a call must stay allocated until the stream has
    passed the call: torch's caching allocator only orders a freed block
    after the work of the stream it was allocated on, so when the context's
    stream is another one, hold the tensor or call
    ``tensor.record_stream(ctx.stream)`` before dropping it."""

    def __init__(self, arena: torch.Tensor, stream: torch.cuda.Stream | None = None):
        if arena.dtype != torch.uint8:
            raise ValueError("arena must be a uint8 tensor")
        self._arena = arena
        self.stream = stream if stream is not None else torch.cuda.current_stream(arena.device)
        h = ctypes.c_void_p()
        st = _L.pcs_ctx_create(ctypes.c_void_p(_dev_ptr(arena)), arena.numel(),
                                 ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h))
        if st:
            raise PcsError(st, "pcs_ctx_create failed")
        self._h = h

    def _check(self, st):
        if st:
            raise PcsError(st, _L.pcs_last_error(self._h).decode())

    def close(self):
        """Waits for the context's stream and frees every handle (pcs_ctx_destroy)."""
        if getattr(self, "_h", None):
            _L.pcs_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- fingerprint / classify ------------------------------------------
    def fingerprint(self, bufs, chunk_hashes=None, roots=None, session_root=None):
        """Chunked XXH64 + Merkle roots of `bufs` (pcs_fingerprint) into int64
        device tensors: chunk_hashes (buffer-major, one per 4096-byte chunk),
        roots (one per buffer), session_root (one value); each optional."""
        self._check(_L.pcs_fingerprint(self._h, _array(bufs), len(bufs), _dev_ptr(chunk_hashes),
                                         _dev_ptr(roots), _dev_ptr(session_root)))

    def fingerprint_noalloc(self, bufs, chunk_hashes=None, roots=None, session_root=None):
        """fingerprint() for callers that cannot allocate
        (pcs_fingerprint_noalloc): same outputs, scratch in the library's
        static per-GPU array; calls that overlap on one GPU race."""
        self._check(_L.pcs_fingerprint_noalloc(self._h, _array(bufs), len(bufs), _dev_ptr(chunk_hashes),
                                                 _dev_ptr(roots), _dev_ptr(session_root)))

    def classify(self, hashes, K: int, chunks_per_buf, bitmap, labels):
        """Cross-replay classification (pcs_classify): hashes holds K x total
        fingerprints (replay-major); bitmap gets one 64-bit word per 64-chunk
        group (bit set: the K fingerprints differ), labels one byte per
        buffer (1 = must snapshot, 0 = recomputable)."""
        n = len(chunks_per_buf)
        cpb = chunks_per_buf if isinstance(chunks_per_buf, ctypes.Array) else u64_array(chunks_per_buf)
        self._check(_L.pcs_classify(self._h, _dev_ptr(hashes), K, cpb, n, _dev_ptr(bitmap), _dev_ptr(labels)))

    def distance(self, ref_hashes, bufs) -> float:
        """Return-consistency distance at chunk granularity (pcs_distance):
        the fraction of the 4096-byte chunks of `bufs` whose fingerprint
        differs from ref_hashes (device int64 tensor, one value per chunk, as
        fingerprint() writes them).  Fingerprinting, comparison and count run
        on the GPU; the call waits for the context's stream."""
        _, T = chunk_counts(bufs)
        if T and ref_hashes.numel() < T:
            raise ValueError("ref_hashes holds fewer values than the buffers have chunks")
        d = ctypes.c_double()
        ref = _dev_ptr(ref_hashes.reshape(-1)) if T else 0
        self._check(_L.pcs_distance(self._h, _array(bufs), len(bufs), ref, None, ctypes.byref(d)))
        return float(d.value)

    def discover(self, components, probe, eps: float = 0.0, control: int = -1) -> dict:
        """Discovering PCS by measurement (pcs_discover; Sec. 4, procedure
        FINGERPRINT).  components: descriptors of the live session's
        components at the probe's anchor.  probe(snap, mask) -> D restores the
        snapshot (the components whose mask flag is 1, in order) into a fresh
        session, runs the leave-and-return trajectory and returns its
        distance, e.g. with distance().  control: the component given a
        wrong value for the control (-1: none).  An exception raised by the
        probe is re-raised here."""
        errors = []

        def cb(user, snap, mask_ptr, k, d_out):
            try:
                d_out[0] = float(probe(int(snap), tuple(int(mask_ptr[i]) for i in range(k))))
                return 0
            except BaseException as e:  # handed back to the caller below
                errors.append(e)
                return 1

        fn = PROBE_FN(cb)
        out = PcsDiscovery()
        k = len(components)
        st = _L.pcs_discover(self._h, _array(components) if k else None, k, float(eps), int(control), fn, None,
                             ctypes.byref(out))
        if errors:
            raise errors[0]
        self._check(st)
        return dict(pcs=list(out.pcs[:k]), necessary=list(out.necessary[:k]), d_without=list(out.d_without[:k]),
                    d_necessary=out.d_necessary, d_final=out.d_final, d_control=out.d_control,
                    added=list(out.added[:out.n_added]), probes=int(out.probes), control_ok=int(out.control_ok),
                    converged=int(out.converged))

    # -- contract ----------------------------------------------------------
    def checkpoint(self, plan, parent: int = 0, hash: bool = False, chunk_hashes=None, roots=None,
                   session_root=None) -> int:
        """checkpoint(s) -> c (pcs_checkpoint): an immutable snapshot of the
        plan's logical bytes, full (parent 0; fingerprinted while copied when
        `hash`) or incremental against `parent` (only new or changed chunks
        stored).  Returns the handle."""
        out = ctypes.c_uint64()
        self._check(_L.pcs_checkpoint(self._h, _array(plan), len(plan), parent, CKPT_HASH if hash else 0,
                                        _dev_ptr(chunk_hashes), _dev_ptr(roots), _dev_ptr(session_root),
                                        ctypes.byref(out)))
        return int(out.value)

    def checkpoint_batch(self, plans, hash: bool = False, chunk_hashes=None, roots=None, session_roots=None,
                         nbufs=None):
        """plans: list of per-session descriptor lists, or a BufArray of all
        sessions' descriptors together with `nbufs` (buffers per session)."""
        if isinstance(plans, BufArray):
            arr, counts = plans.arr, list(nbufs)
        else:
            arr, counts = _array([b for p in plans for b in p]), [len(p) for p in plans]
        nb = (ctypes.c_uint32 * max(1, len(counts)))(*counts)
        out = (ctypes.c_uint64 * max(1, len(counts)))()
        self._check(_L.pcs_checkpoint_batch(self._h, arr, nb, len(counts),
                                              CKPT_HASH if hash else 0, _dev_ptr(chunk_hashes),
                                              _dev_ptr(roots), _dev_ptr(session_roots), out))
        return [int(out[i]) for i in range(len(counts))]

    def restore(self, snap: int, dsts):
        """restore(c) -> s' (pcs_restore): writes the snapshot's logical bytes
        into the destination descriptors (a ring may use a new head)."""
        self._check(_L.pcs_restore(self._h, snap, _array(dsts), len(dsts)))

    def restore_batch(self, snaps, dsts_per_snap, nbufs=None):
        """dsts_per_snap: list of per-snapshot descriptor lists, or a BufArray
        with `nbufs` (destinations per snapshot)."""
        if isinstance(dsts_per_snap, BufArray):
            arr, counts = dsts_per_snap.arr, list(nbufs)
        else:
            arr, counts = _array([b for d in dsts_per_snap for b in d]), [len(d) for d in dsts_per_snap]
        s = (ctypes.c_uint64 * max(1, len(snaps)))(*snaps)
        nb = (ctypes.c_uint32 * max(1, len(counts)))(*counts)
        self._check(_L.pcs_restore_batch(self._h, s, len(snaps), arr, nb))

    def restore_verify(self, snap: int, dsts, bad_bitmap, bad_labels=None):
        """Restore fused with verification (pcs_restore_verify): bad_bitmap
        gets a bit per chunk whose restored bytes do not match the stored
        fingerprint, bad_labels (optional) a byte per buffer."""
        self._check(_L.pcs_restore_verify(self._h, snap, _array(dsts), len(dsts), _dev_ptr(bad_bitmap),
                                          _dev_ptr(bad_labels)))

    def view(self, snap: int):
        """(device address, bytes) of the payload the snapshot holds; read-only."""
        a, n = ctypes.c_uint64(), ctypes.c_uint64()
        self._check(_L.pcs_snapshot_view(self._h, snap, ctypes.byref(a), ctypes.byref(n)))
        return int(a.value), int(n.value)

    def export_size(self, snap: int) -> int:
        """Bytes of the snapshot's self-contained image."""
        size = ctypes.c_uint64()
        self._check(_L.pcs_export(self._h, snap, None, 0, ctypes.byref(size)))
        return int(size.value)

    def export(self, snap: int, out=None):
        """The snapshot's self-contained host image: into `out` (a CPU uint8
        torch tensor, e.g. pinned memory, or a numpy uint8 array of at least
        export_size() bytes) and returned, or into a new numpy array."""
        import numpy as np
        size = self.export_size(snap)
        if out is None:
            out = np.empty(size, dtype=np.uint8)
        ptr, cap = _host_ptr(out)
        if cap < size:
            raise ValueError("export needs %d bytes, out holds %d" % (size, cap))
        n = ctypes.c_uint64()
        self._check(_L.pcs_export(self._h, snap, ctypes.c_void_p(ptr), cap, ctypes.byref(n)))
        return out

    def import_image(self, img, nbytes: int | None = None) -> int:
        """A new full snapshot from an image written by export (verified on
        the device).  img: numpy uint8 array, bytes, or CPU uint8 tensor."""
        import numpy as np
        if not isinstance(img, (np.ndarray, torch.Tensor)):
            img = np.frombuffer(bytes(img), dtype=np.uint8)
        if isinstance(img, np.ndarray):
            img = np.ascontiguousarray(img, dtype=np.uint8)
        ptr, cap = _host_ptr(img)
        size = cap if nbytes is None else nbytes
        if size > cap:
            raise ValueError("nbytes exceeds the image buffer")
        out = ctypes.c_uint64()
        self._check(_L.pcs_import(self._h, ctypes.c_void_p(ptr), size, ctypes.byref(out)))
        return int(out.value)

    def bank_shrink(self, parts, scores, keep: int, kept=None):
        """Relevance-keyed bank shrink (pcs_bank_shrink): keeps the `keep`
        entries with the lowest scores (ties: lower index first; NaN last) in
        their original order.  parts: sequence of (src, dst, entry_bytes) with
        device tensors; dst None (or src itself) shrinks in place.  scores:
        float32 device tensor, one score per entry.  kept: optional int32
        device tensor receiving the kept indices."""
        if not isinstance(scores, torch.Tensor) or scores.dtype != torch.float32:
            raise TypeError("scores must be a float32 device tensor")
        n = scores.numel()
        arr = (PcsBankPart * max(1, len(parts)))()
        for i, (src, dst, eb) in enumerate(parts):
            dst = src if dst is None else dst
            if src.numel() * src.element_size() < n * eb or dst.numel() * dst.element_size() < keep * eb:
                raise ValueError("bank part %d is smaller than its entries" % i)
            arr[i] = PcsBankPart(_dev_ptr(src), _dev_ptr(dst), eb)
        if kept is not None and (kept.dtype != torch.int32 or kept.numel() < keep):
            raise ValueError("kept must be an int32 device tensor of at least keep values")
        self._check(_L.pcs_bank_shrink(self._h, arr, len(parts), n, _dev_ptr(scores) if n else None, keep,
                                       _dev_ptr(kept) if kept is not None else None))

    def fork(self, snap: int) -> int:
        """fork(c) -> c' (pcs_fork): a second handle on the same immutable snapshot."""
        out = ctypes.c_uint64()
        self._check(_L.pcs_fork(self._h, snap, ctypes.byref(out)))
        return int(out.value)

    def delete(self, snap: int):
        """delete(c) (pcs_delete): drops one handle; the bytes go when no handle
        or incremental child refers to them."""
        self._check(_L.pcs_delete(self._h, snap))

    def info(self, snap: int) -> dict:
        """Sizes and kind of a snapshot (pcs_snapshot_info)."""
        inf = PcsSnapInfo()
        self._check(_L.pcs_snapshot_info(self._h, snap, ctypes.byref(inf)))
        return {f: int(getattr(inf, f)) for f, _ in PcsSnapInfo._fields_ if f != "reserved"}

    def payload(self, snap: int, out: torch.Tensor):
        """Copies the bytes the snapshot stores into the device tensor `out`
        (pcs_snapshot_payload)."""
        self._check(_L.pcs_snapshot_payload(self._h, snap, _dev_ptr(out), out.numel() * out.element_size()))

    def stored_hashes(self, snap: int, out: torch.Tensor):
        """Copies the snapshot's stored chunk fingerprints into the int64
        device tensor `out` (pcs_snapshot_hashes)."""
        self._check(_L.pcs_snapshot_hashes(self._h, snap, _dev_ptr(out), out.numel()))

    def arena_stats(self) -> dict:
        """Arena accounting: bytes used and free, largest free block, live handles."""
        v = [ctypes.c_uint64() for _ in range(4)]
        self._check(_L.pcs_arena_stats(self._h, *[ctypes.byref(x) for x in v]))
        return dict(zip(["used", "free", "largest_free", "live_handles"], [int(x.value) for x in v]))

    # -- kernel timing -----------------------------------------------------
    def set_timing(self, enable: bool, dispatch: bool = False):
        """Times every kernel launch with HIP events while enabled
        (pcs_set_timing): recorded on the stream around each launch, or with
        `dispatch` the kernel dispatch's own begin and end timestamps."""
        mode = (TIMING_DISPATCH if dispatch else TIMING_EVENTS) if enable else TIMING_OFF
        self._check(_L.pcs_set_timing(self._h, mode))

    def kernel_time(self, name: str):
        """(launches, total ms) of the kernel family `name` since the last call
        for it (pcs_kernel_time); waits for the stream."""
        n = ctypes.c_uint64()
        ms = ctypes.c_double()
        self._check(_L.pcs_kernel_time(self._h, name.encode(), ctypes.byref(n), ctypes.byref(ms)))
        return int(n.value), float(ms.value)

"""Pins the oracle's durable image writer (the export format) to an
independent reader.

The image is this library's own format (the paper fixes none): a header
with the layout, the buffer and session roots, every chunk fingerprint, and
the canonical payload.  The reader below parses it with `struct` and checks
each field against values computed here without the oracle: chunk
fingerprints with the `xxhash` library, roots with a recursive largest-
power-of-two Merkle split over `xxhash`, and the payload as the components
padded to 4096 bytes by numpy.
"""
import struct

import numpy as np
import xxhash

import oracle

CHUNK = 4096


def lib_h(b):
    return xxhash.xxh64_intdigest(bytes(b), 0)


def lib_merkle(leaves):
    """Promote-odd tree as a recursive split at the largest power of two
    below n (the definition the oracle's level-by-level tree must equal)."""
    n = len(leaves)
    if n == 0:
        return lib_h(b"")
    if n == 1:
        return leaves[0]
    k = 1
    while k * 2 < n:
        k *= 2
    return lib_h(struct.pack("<QQ", lib_merkle(leaves[:k]), lib_merkle(leaves[k:])))


def parse(img):
    """Independent reader of the image layout; returns its fields."""
    assert img[:8] == b"PCSIMG01"
    ver, n, chunks, state, pay = struct.unpack_from("<IIQQQ", img, 8)
    flags, = struct.unpack_from("<Q", img, 40)
    o = 48
    lays = []
    for _ in range(n):
        kind, z, nbytes, row, win, outer, z2 = struct.unpack_from("<IIQQQQQ", img, o)
        assert z == 0 and z2 == 0
        lays.append((kind, nbytes, row, win, outer))
        o += 48
    roots = struct.unpack_from("<%dQ" % (n + 1), img, o)
    o += 8 * (n + 1)
    hashes = struct.unpack_from("<%dQ" % chunks, img, o)
    o += 8 * chunks
    o += (-o) % CHUNK
    return dict(version=ver, n=n, chunks=chunks, state=state, payload_bytes=pay, flags=flags, layouts=lays,
                roots=roots, hashes=hashes, payload=img[o:])


def test_image_fields_against_independent_values():
    rng = np.random.default_rng(31)
    sizes = [0, 1, 4095, 4096, 4097, 3 * 4096 + 5, 70 * 4096 + 123]
    bufs = [rng.integers(0, 256, size=s, dtype=np.uint8) for s in sizes]
    layouts = [(0, 0, 0, 0)] * (len(sizes) - 1) + [(1, 2048, 143, 2)]
    img = oracle.export_image(bufs, layouts)
    f = parse(img)
    assert f["version"] == 1 and f["n"] == len(sizes) and f["flags"] == 0
    assert f["state"] == sum(sizes)
    assert [(k, nb, r, w, o) for k, nb, r, w, o in f["layouts"]] == [
        (k, s, r, w, o) for s, (k, r, w, o) in zip(sizes, layouts)]
    # Chunk fingerprints: buffer after buffer, chunk after chunk.
    want_h = []
    roots = []
    for b in bufs:
        hs = [lib_h(b[i:i + CHUNK].tobytes()) for i in range(0, b.size, CHUNK)]
        want_h += hs
        roots.append(lib_merkle(hs))
    assert f["chunks"] == len(want_h) and list(f["hashes"]) == want_h
    assert list(f["roots"][:-1]) == roots and f["roots"][-1] == lib_merkle(roots)
    # Payload: components in order, each padded with zeros to a 4096 multiple.
    comps = [np.concatenate([b, np.zeros((-b.size) % CHUNK, dtype=np.uint8)]) for b in bufs]
    want_p = np.concatenate(comps).tobytes()
    assert f["payload_bytes"] == len(want_p) and f["payload"] == want_p
    # The header block is itself padded to 4096, so the payload starts aligned.
    assert (len(img) - len(want_p)) % CHUNK == 0


def test_image_of_nothing():
    f = parse(oracle.export_image([]))
    assert f["n"] == 0 and f["chunks"] == 0 and f["state"] == 0 and f["payload"] == b""
    assert f["roots"] == (lib_h(b""),)

"""The C ABI without Python: tests/host/c_client.c uses only include/pcs.h and
the HIP runtime's allocation and copy calls (no torch) to fingerprint a
session (a flat buffer of ragged size and a wrapped ring window), checkpoint
it, fork it, restore the fork at a new ring head and export it; then it
rewrites one chunk, takes an incremental checkpoint, classifies the two
fingerprint passes, imports the exported image and restores from the
import and from the incremental snapshot; then it takes the chunk distance
of the rewritten bytes from the first fingerprints and shrinks a small
bank to 12% (one part in place, one out of place).  Its printed fingerprints, stored
chunk count, bitmap and labels are compared with the oracle's, its restore
checks must pass, and its image size must equal the oracle image's."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from tests.gpu_util import log
from tests.host import build_c_client

pytestmark = pytest.mark.gpu

FLAT_BYTES = 3 * 4096 + 777
OUTER, CAPACITY, ROW, HEAD, WINDOW = 2, 16, 256, 11, 12


def pattern(buf, n):
    i = np.arange(n, dtype=np.uint64)
    return ((i * 131 + buf * 17 + (i >> 8)) & 0xFF).astype(np.uint8)


def test_c_client_matches_oracle():
    exe = build_c_client.EXE if os.path.exists(build_c_client.EXE) else build_c_client.build()
    log("C client:", exe)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    hashes, roots, words, labels, kept, out = {}, {}, {}, {}, {}, {}
    for line in r.stdout.splitlines():
        f = line.split()
        if f[0] == "hash":
            hashes[int(f[1])] = int(f[2], 16)
        elif f[0] == "root":
            roots[int(f[1])] = int(f[2], 16)
        elif f[0] == "bitmap":
            words[int(f[1])] = int(f[2], 16)
        elif f[0] == "label":
            labels[int(f[1])] = int(f[2])
        elif f[0] == "kept":
            kept[int(f[1])] = int(f[2])
        else:
            out[f[0]] = f[1]
    flat = pattern(0, FLAT_BYTES)
    ring = pattern(1, OUTER * CAPACITY * ROW)
    window = oracle.ring_window(ring, OUTER, CAPACITY * ROW, CAPACITY, ROW, HEAD, WINDOW)
    want_h, want_r, want_s = oracle.fingerprint([flat, window])
    assert [hashes[i] for i in range(len(hashes))] == [int(x) for x in want_h]
    assert [roots[0], roots[1]] == [int(x) for x in want_r]
    assert int(out["session"], 16) == int(want_s)
    assert out["restored"] == "1"
    image = oracle.export_image([flat, window], [(0, 0, 0, 0), (1, ROW, WINDOW, OUTER)])
    assert int(out["image"]) == len(image)
    # Chunk 1 of the flat buffer rewritten, the ring unchanged.
    flat2 = flat.copy()
    flat2[4096:8192] ^= np.uint8(0x5A)
    h2 = oracle.fingerprint([flat2, window])[0]
    cpb = [oracle.chunk_count(flat.size), oracle.chunk_count(window.size)]
    d, nd = oracle.dirty(h2, cpb, want_h, cpb)
    assert int(out["dirty"]) == nd == 1
    want_bm, want_lab = oracle.classify(np.stack([np.asarray(want_h, dtype=np.uint64), h2]), cpb)
    assert [words[i] for i in range(len(words))] == [int(x) for x in want_bm]
    assert [labels[0], labels[1]] == [int(x) for x in want_lab] == [1, 0]
    assert out["imported_restored"] == "1" and out["incremental_restored"] == "1"
    # Distance of the rewritten bytes from the first fingerprints: one chunk of all.
    total = sum(cpb)
    assert int(out["differing"]) == 1 and float(out["distance"]) == 1 / total
    # The 21-entry bank shrunk to 12% (Table 6: 3 frames), latents in place, poses out of place.
    bank, lat_b, pose_b = 21, 40, 12
    i = np.arange(bank)
    lat = ((i[:, None] * 13 + np.arange(lat_b)[None, :] * 7) & 0xFF).astype(np.uint8).reshape(-1)
    pose = ((i[:, None] * 29 + np.arange(pose_b)[None, :] * 3 + 5) & 0xFF).astype(np.uint8).reshape(-1)
    scores = ((i * 37) % 11 - 5).astype(np.float32)
    keep = oracle.keep_count(0.12, bank)
    assert int(out["keep"]) == keep == 3
    want_kept, (want_lat, want_pose) = oracle.bank_shrink([(lat, lat_b), (pose, pose_b)], scores, keep)
    assert [kept[j] for j in range(keep)] == want_kept.tolist()
    assert bytes.fromhex(out["shrunk_lat"]) == want_lat.tobytes()
    assert bytes.fromhex(out["shrunk_pose"]) == want_pose.tobytes()

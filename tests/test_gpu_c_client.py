"""The C ABI without Python: tests/host/c_client.c uses only include/pcs.h and
the HIP runtime's allocation and copy calls (no torch) to fingerprint a
session (a flat buffer of ragged size and a wrapped ring window), checkpoint
it, fork it, restore the fork at a new ring head and export it.  Its printed
fingerprints are compared with the oracle's, its restore check must pass,
and its image size must equal the oracle image's."""
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
    hashes, roots, out = {}, {}, {}
    for line in r.stdout.splitlines():
        f = line.split()
        if f[0] == "hash":
            hashes[int(f[1])] = int(f[2], 16)
        elif f[0] == "root":
            roots[int(f[1])] = int(f[2], 16)
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

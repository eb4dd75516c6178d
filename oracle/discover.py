"""CPU oracle of the discovery procedure (Sec. 4, procedure FINGERPRINT) and
of the return-consistency distance it is driven by.  TEST INFRASTRUCTURE
ONLY: only tests/, the smoke check and the benchmark's CPU leg use it.

The procedure, over components H = {h_0 .. h_{k-1}}, a probe that restores
a snapshot of a subset of H into a fresh session and measures the distance
D of its continuation, and a tolerance eps:
  1. necessity: for each h_i, probe the snapshot of H without h_i; h_i is
     necessary iff D > eps;
  2. sufficiency: probe the snapshot of exactly the necessary set N; if
     D <= eps, PCS = N;
  3. redundancy fallback: otherwise add, one at a time, the component whose
     addition gives the smallest D (ties: the lowest index), until
     D <= eps or every component is in;
  4. PCS and Derivable = H \\ PCS.
The control of Sec. 4 (necessity tests that pass because nothing reads the
snapshot): probe the full snapshot with one component holding a wrong value
(the lowest bit of its first byte flipped) and require D > eps.

D here is the fraction of the probe's 4096-byte output chunks whose
fingerprint differs from an uninterrupted reference run (eps = 0: a
bit-exact return).
"""
from __future__ import annotations

import numpy as np

from . import fingerprint


def distance(ref_hashes, out_bytes) -> float:
    """Fraction of chunks of out_bytes whose fingerprint differs from ref_hashes."""
    h = fingerprint([np.asarray(out_bytes, dtype=np.uint8)])[0]
    ref = np.asarray(ref_hashes, dtype=np.uint64)
    assert h.size == ref.size
    return float(np.count_nonzero(h != ref)) / h.size if h.size else 0.0


def discover(probe, k: int, eps: float, control: int = -1) -> dict:
    """Procedure FINGERPRINT over probe(mask, corrupt) -> D; mask is a
    tuple of k 0/1 flags, corrupt the component given a wrong value (-1:
    none)."""
    probes = 0

    def run(mask, corrupt=-1):
        nonlocal probes
        probes += 1
        return probe(tuple(mask), corrupt)

    d_without, necessary = [], []
    for i in range(k):
        mask = [1] * k
        mask[i] = 0
        d = run(mask)
        d_without.append(d)
        necessary.append(1 if d > eps else 0)
    pcs = list(necessary)
    d_necessary = run(pcs)
    d, added = d_necessary, []
    while d > eps and sum(pcs) < k:
        best, best_d = -1, None
        for c in range(k):
            if pcs[c]:
                continue
            m = list(pcs)
            m[c] = 1
            dc = run(m)
            if best_d is None or dc < best_d:
                best, best_d = c, dc
        pcs[best] = 1
        added.append(best)
        d = best_d
    d_control, control_ok = -1.0, -1
    if control >= 0:
        d_control = run([1] * k, control)
        control_ok = 1 if d_control > eps else 0
    return dict(pcs=pcs, necessary=necessary, d_without=d_without, d_necessary=d_necessary, d_final=d,
                d_control=d_control, added=added, probes=probes, control_ok=control_ok,
                converged=1 if d <= eps else 0)


def mock_probe(spec, anchor_parts, actions, ref_hashes):
    """The probe on the oracle's mock world model: a fresh session receives
    the snapshot's components (the others keep a fresh session's zeros), runs
    `actions`, and is scored against the reference fingerprints."""
    from workloads.mock_world import fresh_state
    from .mock_world import MockWorld

    def probe(mask, corrupt=-1):
        parts = fresh_state(spec)
        for i, m in enumerate(mask):
            if m:
                parts[i] = np.array(anchor_parts[i], dtype=np.uint8, copy=True)
        if corrupt >= 0:
            parts[corrupt][0] ^= 1
        return distance(ref_hashes, MockWorld(spec, parts).run(actions))

    return probe

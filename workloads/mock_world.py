"""Seeded inputs of the mock world model that the discovery procedure (Sec. 4)
is exercised on: its sizes, its initial session state and its action
trajectories.  No model arithmetic lives here; the model's step is
implemented twice, independently: on the GPU with torch
(workloads/mock_world_gpu.py) and on the CPU in the oracle
(oracle/mock_world.py).

The model is fingerprintable in the paper's sense (Sec. 4): its runtime
state decomposes into addressable components, any subset can be
checkpointed and restored, and a return-consistency distance D can be
computed for a leave-and-return probe.  Its eight components, in order:

  0 obs      uint8 [H, W, 3]      the last frame
  1 rng      uint32 [4]           Philox4x32-10 key (2 words), counter (2 words, low first)
  2 bank     uint32 [1 + B(4+L)]  word 0 = entries written; entry e = pose (4 words) + L summary words
  3 pose     uint32 [4]           position and heading, int32 values
  4 feat     uint32 [H * W]       per-pixel features, recomputed from obs at every step
  5 scratch  uint32 [H * W]       activation scratch, overwritten at every step before it is read
  6 kv_a     uint32 [1 + K]       word 0 = generation (0 = absent), K context words
  7 kv_b     uint32 [1 + K]       the same context stored transformed: either of kv_a, kv_b rebuilds the other

By construction obs, rng, bank and pose are each necessary; feat and
scratch are derivable; kv_a and kv_b are not individually necessary but one
of them is (the case the procedure's redundancy fallback exists for).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

COMPONENTS = ("obs", "rng", "bank", "pose", "feat", "scratch", "kv_a", "kv_b")


@dataclass(frozen=True)
class MockSpec:
    height: int = 64
    width: int = 64
    bank_cap: int = 64       # B entries
    entry_words: int = 256   # L summary words per entry (must divide height * width)
    kv_words: int = 1024     # K context words

    @property
    def pixels(self) -> int:
        return self.height * self.width

    def nbytes(self):
        """Byte size of each component, in component order."""
        P, B, L, K = self.pixels, self.bank_cap, self.entry_words, self.kv_words
        return [3 * P, 16, 4 * (1 + B * (4 + L)), 16, 4 * P, 4 * P, 4 * (1 + K), 4 * (1 + K)]


def _rng(seed: int, stream: int):
    return np.random.default_rng([seed, 9000 + stream])


def initial_state(spec: MockSpec, seed: int):
    """A new session before its first step, as host byte arrays per
    component: a random frame, a random Philox key with counter 0, an empty
    bank, pose 0, zero features and scratch, and generation-1 context words
    (random) in kv_a; kv_b holds zeros and is filled by the first step."""
    assert spec.pixels % spec.entry_words == 0
    obs = _rng(seed, 0).integers(0, 256, size=3 * spec.pixels, dtype=np.uint8)
    rng = np.zeros(4, dtype=np.uint32)
    rng[:2] = _rng(seed, 1).integers(0, 1 << 32, size=2, dtype=np.uint64).astype(np.uint32)
    kv_a = np.zeros(1 + spec.kv_words, dtype=np.uint32)
    kv_a[0] = 1
    kv_a[1:] = _rng(seed, 2).integers(0, 1 << 32, size=spec.kv_words, dtype=np.uint64).astype(np.uint32)
    parts = [obs, rng, np.zeros(1 + spec.bank_cap * (4 + spec.entry_words), dtype=np.uint32),
             np.zeros(4, dtype=np.uint32), np.zeros(spec.pixels, dtype=np.uint32),
             np.zeros(spec.pixels, dtype=np.uint32), kv_a, np.zeros(1 + spec.kv_words, dtype=np.uint32)]
    return [p.view(np.uint8).copy() for p in parts]


def fresh_state(spec: MockSpec):
    """What a newly created session holds before anything is restored into it."""
    return [np.zeros(n, dtype=np.uint8) for n in spec.nbytes()]


def trajectory(seed: int, warm: int, away: int):
    """Actions (int32 [n, 4]): `warm` random steps that build the session's
    history up to the anchor, then the probe: `away` steps leaving along +x
    (and turning), then `away` steps returning to the anchor pose."""
    warm_actions = _rng(seed, 3).integers(-3, 4, size=(warm, 4)).astype(np.int32)
    out = np.tile(np.array([[5, 0, 0, 1]], dtype=np.int32), (away, 1))
    back = np.tile(np.array([[-5, 0, 0, -1]], dtype=np.int32), (away, 1))
    return warm_actions, np.concatenate([out, back])

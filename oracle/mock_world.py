"""CPU oracle of the mock world model used to exercise the discovery
procedure (Sec. 4).  TEST INFRASTRUCTURE ONLY: only tests/, the smoke check
and the benchmark's CPU leg use it; it shares no code with the GPU side
(which implements the same model with torch).

The model is integer-only (all words are uint32, arithmetic mod 2^32), so
two independent implementations agree bit for bit.  Components, in order:
obs (uint8 [H, W, 3]), rng (Philox4x32-10 key k0, k1 and 64-bit counter
c_lo, c_hi), bank (word 0 = entries written; entry e = 4 pose words and L
summary words), pose (4 int32 words), feat (uint32 per pixel), scratch
(uint32 per pixel), kv_a and kv_b (word 0 = generation, 0 meaning absent;
K context words; kv_b holds T(kv_a) word by word).

One step with action u (4 int32 values), pixel p in [0, P):
  1. feat[p] = F(obs[3p] | obs[3p+1] << 8 | obs[3p+2] << 16), where
     F(x): h = x * 0x9E3779B1; h ^= h >> 15; h *= 0x85EBCA77; h ^= h >> 13.
  2. If kv_a is absent and kv_b is not, kv_a = T^-1(kv_b) (generation
     copied); if kv_b is absent and kv_a is not, kv_b = T(kv_a).
     T(x) = rotl(x, 13) ^ 0xA5A5A5A5.
  3. r = Philox4x32-10(counter (c_lo, c_hi, 0, 0), key (k0, k1)); then the
     64-bit counter (c_lo, c_hi) advances by one.
  4. pose += u (each word mod 2^32).
  5. Among the min(written, B) stored entries, the one whose pose is nearest
     to the new pose in L1 distance over the four words read as int32 (ties:
     the lowest entry index) gives mem = its L summary words; no entry gives
     mem = 0.
  6. scratch[p] = feat[p] ^ rotl(mem[p mod L], p mod 32) ^ r[p mod 4]
                  ^ kv_a[1 + p mod K].
  7. new obs[3p + c] = (obs[3p + c] * 5 + byte c of scratch[p]
                        + low byte of r[c]) mod 256, c = 0, 1, 2.
  8. summary[w] = sum over p = w (mod L) of
     (obs'[3p] + 256 obs'[3p+1] + 65536 obs'[3p+2]) * (p + 1), mod 2^32.
  9. The entry (new pose, summary) is written at slot (written mod B) and
     written += 1.
 10. kv_a's generation += 1; kv_a[1 + j] = kv_a[1 + j] * 0x9E3779B1
     + summary[j mod L] + j; kv_b = T(kv_a), generation copied.
"""
from __future__ import annotations

import numpy as np

from . import philox4x32_10

M32 = 0xFFFFFFFF


def _u32(a):
    return np.asarray(a, dtype=np.uint64) & M32


def rotl(x, r):
    """32-bit rotate left; r is taken mod 32 (elementwise for arrays)."""
    x = _u32(x)
    r = np.asarray(r, dtype=np.uint64) % 32
    return ((x << r) | (x >> ((32 - r) % 32))) & M32


def T(x):
    return rotl(x, 13) ^ 0xA5A5A5A5


def T_inv(y):
    y = _u32(y) ^ 0xA5A5A5A5
    return ((y >> 13) | (y << 19)) & M32


def feature(x):
    h = (_u32(x) * 0x9E3779B1) & M32
    h ^= h >> 15
    h = (h * 0x85EBCA77) & M32
    h ^= h >> 13
    return h


class MockWorld:
    """One session of the mock model on the host (uint64 arrays holding
    uint32 values)."""

    def __init__(self, spec, parts):
        self.spec = spec
        P, B, L, K = spec.pixels, spec.bank_cap, spec.entry_words, spec.kv_words
        self.obs = np.frombuffer(bytes(parts[0]), dtype=np.uint8).astype(np.uint64)
        w = [np.frombuffer(bytes(parts[i]), dtype=np.uint32).astype(np.uint64) for i in range(1, 8)]
        self.rng, self.bank, self.pose, self.feat, self.scratch, self.kv_a, self.kv_b = w
        assert self.obs.size == 3 * P and self.bank.size == 1 + B * (4 + L) and self.kv_a.size == 1 + K

    def parts(self):
        """The components as byte arrays, in component order."""
        out = [self.obs.astype(np.uint8)]
        for a in (self.rng, self.bank, self.pose, self.feat, self.scratch, self.kv_a, self.kv_b):
            out.append(a.astype(np.uint32).view(np.uint8))
        return out

    def step(self, action):
        s = self.spec
        P, B, L, K = s.pixels, s.bank_cap, s.entry_words, s.kv_words
        p = np.arange(P, dtype=np.uint64)
        o = self.obs.reshape(P, 3)
        # 1. features from the current frame
        self.feat = feature(o[:, 0] | (o[:, 1] << 8) | (o[:, 2] << 16))
        # 2. the context pair: either half rebuilds the other
        if self.kv_a[0] == 0 and self.kv_b[0] != 0:
            self.kv_a = np.concatenate([self.kv_b[:1], T_inv(self.kv_b[1:])])
        elif self.kv_b[0] == 0 and self.kv_a[0] != 0:
            self.kv_b = np.concatenate([self.kv_a[:1], T(self.kv_a[1:])])
        # 3. random words, then advance the counter
        r = philox4x32_10([int(self.rng[2]), int(self.rng[3]), 0, 0], [int(self.rng[0]), int(self.rng[1])])
        r = r.astype(np.uint64)
        ctr = (int(self.rng[2]) | (int(self.rng[3]) << 32)) + 1
        self.rng[2], self.rng[3] = ctr & M32, (ctr >> 32) & M32
        # 4. pose
        self.pose = (self.pose + _u32(np.asarray(action, dtype=np.int64))) & M32
        # 5. retrieval by nearest pose
        n = min(int(self.bank[0]), B)
        entries = self.bank[1:].reshape(B, 4 + L)
        if n == 0:
            mem = np.zeros(L, dtype=np.uint64)
        else:
            sp = lambda a: a.astype(np.uint32).view(np.int32).astype(np.int64)
            d = np.abs(sp(entries[:n, :4]) - sp(self.pose)[None, :]).sum(axis=1)
            mem = entries[int(np.argmin(d)), 4:]
        # 6. scratch
        self.scratch = self.feat ^ rotl(mem[p % L], p % 32) ^ r[p % 4] ^ self.kv_a[1 + p % K]
        # 7. the new frame
        new = np.empty((P, 3), dtype=np.uint64)
        for c in range(3):
            new[:, c] = (o[:, c] * 5 + ((self.scratch >> (8 * c)) & 0xFF) + (r[c] & 0xFF)) & 0xFF
        self.obs = new.reshape(-1)
        # 8. summary of the new frame
        v = new[:, 0] + 256 * new[:, 1] + 65536 * new[:, 2]
        prod = (v * (p + 1)) & M32
        summary = prod.reshape(P // L, L).sum(axis=0) & M32
        # 9. bank append
        slot = int(self.bank[0]) % B
        entries[slot, :4] = self.pose
        entries[slot, 4:] = summary
        self.bank[0] = (self.bank[0] + 1) & M32
        # 10. context update
        j = np.arange(K, dtype=np.uint64)
        self.kv_a[0] = (self.kv_a[0] + 1) & M32
        self.kv_a[1:] = (self.kv_a[1:] * 0x9E3779B1 + summary[j % L] + j) & M32
        self.kv_b = np.concatenate([self.kv_a[:1], T(self.kv_a[1:])])

    def run(self, actions):
        """Steps through `actions`; returns the frames after each step, concatenated."""
        frames = []
        for a in actions:
            self.step(a)
            frames.append(self.obs.astype(np.uint8))
        return np.concatenate(frames) if frames else np.zeros(0, dtype=np.uint8)

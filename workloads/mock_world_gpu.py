"""The mock world model on the GPU, for exercising the discovery procedure
(Sec. 4): its components are device buffers that pcs checkpoints and
restores, and its step runs as torch integer operations on the device.
This is the model under test, not part of the library; the oracle holds an
independent CPU implementation of the same definition.

All words are uint32 held in int64 tensors (arithmetic mod 2^32).  One step
with action u (4 int32 values), pixel p in [0, P):
  1. feat[p] = F(obs[3p] | obs[3p+1] << 8 | obs[3p+2] << 16), where
     F(x): h = x * 0x9E3779B1; h ^= h >> 15; h *= 0x85EBCA77; h ^= h >> 13.
  2. If kv_a's generation word is 0 and kv_b's is not, kv_a = T^-1(kv_b)
     (generation copied); if kv_b's is 0 and kv_a's is not, kv_b = T(kv_a).
     T(x) = rotl(x, 13) ^ 0xA5A5A5A5.
  3. r = Philox4x32-10(counter (c_lo, c_hi, 0, 0), key (k0, k1)); the 64-bit
     counter then advances by one.
  4. pose += u word by word.
  5. mem = the summary words of the stored bank entry nearest to the new
     pose (L1 over the four words read as int32, ties to the lowest entry),
     or zeros if the bank is empty.
  6. scratch[p] = feat[p] ^ rotl(mem[p mod L], p mod 32) ^ r[p mod 4]
                  ^ kv_a[1 + p mod K].
  7. obs'[3p + c] = (obs[3p + c] * 5 + byte c of scratch[p] + low byte of
     r[c]) mod 256.
  8. summary[w] = sum over p = w (mod L) of (obs'[3p] + 256 obs'[3p+1]
     + 65536 obs'[3p+2]) * (p + 1), mod 2^32.
  9. (new pose, summary) goes to bank slot (written mod B); written += 1.
 10. kv_a's generation += 1; kv_a[1 + j] = kv_a[1 + j] * 0x9E3779B1
     + summary[j mod L] + j; kv_b = T(kv_a), generation copied.
"""
from __future__ import annotations

import torch

M32 = 0xFFFFFFFF


def _u(t32: torch.Tensor) -> torch.Tensor:
    """int32 words -> int64 holding their unsigned value."""
    return t32.to(torch.int64) & M32


def _store(dst32: torch.Tensor, x: torch.Tensor):
    """Writes unsigned 32-bit values (int64) into int32 words."""
    dst32.copy_((((x & M32) ^ 0x80000000) - 0x80000000).to(torch.int32))


def _rotl(x, r):
    return ((x << r) | (x >> ((32 - r) % 32))) & M32


def _T(x):
    return _rotl(x, 13) ^ 0xA5A5A5A5


def _T_inv(y):
    y = y ^ 0xA5A5A5A5
    return ((y >> 13) | (y << 19)) & M32


def _mulhilo(a, m: int):
    """High and low 32 bits of a * m (a: int64 holding uint32, m < 2^32),
    through 16-bit limbs so no int64 product overflows."""
    lo_p = (a & 0xFFFF) * m
    mid = (a >> 16) * m + (lo_p >> 16)
    return (mid >> 16) & M32, (((mid & 0xFFFF) << 16) | (lo_p & 0xFFFF)) & M32


def philox4x32_10(c, k):
    """Philox4x32-10 on device scalars: c = 4 counter words, k = 2 key words
    (int64 tensors holding uint32).  Returns the 4 output words."""
    c0, c1, c2, c3 = c
    k0, k1 = k
    for _ in range(10):
        hi0, lo0 = _mulhilo(c0, 0xD2511F53)
        hi1, lo1 = _mulhilo(c2, 0xCD9E8D57)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + 0x9E3779B9) & M32
        k1 = (k1 + 0xBB67AE85) & M32
    return c0, c1, c2, c3


class MockWorldGPU:
    """One session: eight device uint8 buffers, in component order."""

    def __init__(self, spec, parts):
        self.spec = spec
        self.parts = parts
        s = spec
        self._p = torch.arange(s.pixels, dtype=torch.int64, device=parts[0].device)

    @classmethod
    def from_host(cls, spec, host_parts, device="cuda"):
        return cls(spec, [torch.from_numpy(p.copy()).to(device) for p in host_parts])

    @classmethod
    def fresh(cls, spec, device="cuda"):
        return cls(spec, [torch.zeros(n, dtype=torch.uint8, device=device) for n in spec.nbytes()])

    def words(self, i):
        return self.parts[i].view(torch.int32)

    def step(self, action):
        s = self.spec
        P, B, L, K = s.pixels, s.bank_cap, s.entry_words, s.kv_words
        p = self._p
        obs = self.parts[0].to(torch.int64).view(P, 3)
        rng, bank, pose, feat, scratch, kv_a, kv_b = (self.words(i) for i in range(1, 8))
        # 1. features
        x = obs[:, 0] | (obs[:, 1] << 8) | (obs[:, 2] << 16)
        h = (x * 0x9E3779B1) & M32
        h = h ^ (h >> 15)
        h = (h * 0x85EBCA77) & M32
        h = h ^ (h >> 13)
        _store(feat, h)
        # 2. the context pair
        a, b = _u(kv_a), _u(kv_b)
        ga, gb = int(a[0]), int(b[0])
        if ga == 0 and gb != 0:
            a = torch.cat([b[:1], _T_inv(b[1:])])
            _store(kv_a, a)
        elif gb == 0 and ga != 0:
            b = torch.cat([a[:1], _T(a[1:])])
            _store(kv_b, b)
        # 3. random words; advance the counter
        rw = _u(rng)
        zero = torch.zeros((), dtype=torch.int64, device=rw.device)
        r = torch.stack(philox4x32_10((rw[2], rw[3], zero, zero), (rw[0], rw[1])))
        ctr = rw[2] + (rw[3] << 32) + 1
        rw = torch.stack([rw[0], rw[1], ctr & M32, (ctr >> 32) & M32])
        _store(rng, rw)
        # 4. pose
        ps = (_u(pose) + (torch.as_tensor(action, dtype=torch.int64, device=rw.device) & M32)) & M32
        _store(pose, ps)
        # 5. retrieval
        bw = _u(bank)
        n = min(int(bw[0]), B)
        ent = bw[1:].view(B, 4 + L)
        if n == 0:
            mem = torch.zeros(L, dtype=torch.int64, device=rw.device)
        else:
            sgn = lambda v: ((v ^ 0x80000000) - 0x80000000)
            d = (sgn(ent[:n, :4]) - sgn(ps)[None, :]).abs().sum(dim=1)
            mem = ent[int(torch.argmin(d)), 4:]     # argmin returns the first minimum
        # 6. scratch
        sc = h ^ _rotl(mem[p % L], p % 32) ^ r[p % 4] ^ _u(kv_a)[1 + p % K]
        _store(scratch, sc)
        # 7. the new frame
        new = torch.stack([(obs[:, c] * 5 + ((sc >> (8 * c)) & 0xFF) + (r[c] & 0xFF)) & 0xFF for c in range(3)],
                          dim=1)
        self.parts[0].copy_(new.reshape(-1).to(torch.uint8))
        # 8. summary
        v = new[:, 0] + 256 * new[:, 1] + 65536 * new[:, 2]
        summary = ((v * (p + 1)) & M32).view(P // L, L).sum(dim=0) & M32
        # 9. bank append
        slot = int(bw[0]) % B
        ent[slot, :4] = ps
        ent[slot, 4:] = summary
        bw[0] = (bw[0] + 1) & M32
        _store(bank, bw)
        # 10. context update
        a = _u(kv_a)
        j = torch.arange(K, dtype=torch.int64, device=rw.device)
        a[0] = (a[0] + 1) & M32
        a[1:] = (a[1:] * 0x9E3779B1 + summary[j % L] + j) & M32
        _store(kv_a, a)
        _store(kv_b, torch.cat([a[:1], _T(a[1:])]))

    def run(self, actions):
        """Steps through `actions`; returns the frames after each step,
        concatenated, as one device uint8 tensor."""
        n = len(actions)
        out = torch.empty(n * self.parts[0].numel(), dtype=torch.uint8, device=self.parts[0].device)
        f = self.parts[0].numel()
        for i, u in enumerate(actions):
            self.step([int(x) for x in u])
            out[i * f:(i + 1) * f].copy_(self.parts[0])
        return out

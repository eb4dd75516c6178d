"""Seeded synthetic inputs for the PCS fingerprint-and-checkpoint path.

This module only *generates* inputs: byte buffers, ring geometry, replay
perturbations and restore orders.  It holds none of the method's arithmetic
(no hashing, no classification, no packing), so both the GPU library's tests
and the CPU oracle can take their inputs from it.

The workloads stand in for the paper's three state shapes (Table 1): a flat
uint8 observation plus RNG state (the Markovian model), a growing memory bank
of latents and poses (the non-Markovian model; per-frame records, Sec. 7.2),
and a ring-buffered windowed KV context (the addressable-memory model,
Sec. 7.11).  No model, weight or dataset of the paper is used.

Host generators use numpy's PCG64 (``default_rng([seed, i])`` per piece, so
every piece regenerates alone).  Full-size device inputs use torch's seeded
generator on the GPU; tests copy back whatever the oracle must see.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

DTYPES = ("uint8", "float16", "bfloat16", "float32", "int64")
ITEMSIZE = {"uint8": 1, "float16": 2, "bfloat16": 2, "float32": 4, "int64": 8}


def _rng(seed: int, *sub: int) -> np.random.Generator:
    return np.random.default_rng([seed, *sub])


def bf16_normal(rng: np.random.Generator, n: int) -> np.ndarray:
    """n bfloat16 N(0,1) values as uint16 bit patterns (round to nearest even)."""
    f = rng.standard_normal(n, dtype=np.float32).view(np.uint32)
    r = (f + np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def typed_random(rng: np.random.Generator, dtype: str, nbytes: int) -> np.ndarray:
    """nbytes of random values of `dtype` (uint8/int64 uniform, floats N(0,1)), as uint8."""
    isz = ITEMSIZE[dtype]
    assert nbytes % isz == 0
    n = nbytes // isz
    if dtype == "uint8":
        a = rng.integers(0, 256, size=n, dtype=np.uint8)
    elif dtype == "int64":
        a = rng.integers(np.iinfo(np.int64).min, np.iinfo(np.int64).max, size=n, dtype=np.int64,
                         endpoint=True)
    elif dtype == "float16":
        a = rng.standard_normal(n, dtype=np.float32).astype(np.float16)
    elif dtype == "bfloat16":
        a = bf16_normal(rng, n)
    elif dtype == "float32":
        a = rng.standard_normal(n, dtype=np.float32)
    else:
        raise ValueError(dtype)
    return a.view(np.uint8)


# ---------------------------------------------------------------- ring geometry

@dataclass(frozen=True)
class Ring:
    """Geometry of `outer` rings of `capacity` rows of `row_bytes` each.

    Logical row t of ring o sits at physical row (head + t) mod capacity; the
    valid window is `window` rows.  Ring o starts at byte o * outer_stride.
    """
    outer: int
    capacity: int
    row_bytes: int
    window: int
    head: int
    outer_stride: int = 0

    def __post_init__(self):
        if self.outer_stride == 0:
            object.__setattr__(self, "outer_stride", self.capacity * self.row_bytes)

    @property
    def ring_bytes(self) -> int:
        """Bytes of the whole allocation."""
        return (self.outer - 1) * self.outer_stride + self.capacity * self.row_bytes if self.outer else 0

    @property
    def window_bytes(self) -> int:
        return self.outer * self.window * self.row_bytes

    def with_head(self, head: int) -> "Ring":
        return Ring(self.outer, self.capacity, self.row_bytes, self.window, head, self.outer_stride)


def wrapping_head(rng: np.random.Generator, capacity: int, window: int) -> int:
    """A head offset whose window wraps past the end of the ring (needs W >= 2)."""
    return int(rng.integers(capacity - window + 1, capacity))


def other_head(rng: np.random.Generator, capacity: int, head: int) -> int:
    """A head offset different from `head`."""
    h = int(rng.integers(0, capacity - 1))
    return h if h < head else h + 1


# ---------------------------------------------------------------- config 1

@dataclass
class Markovian:
    """Flat state: uint8 observation, 16-byte RNG state, recomputable decoys."""
    obs: np.ndarray               # uint8 [H, W, 3]
    rng_state: np.ndarray         # uint8 [16]: key0, key1, ctr0, ctr1 (LE u32)
    decoys: list                  # uint8 views of fp16 buffers
    rng_state_replay2: np.ndarray  # counter advanced by one

    def buffers(self, replay: int = 1):
        rs = self.rng_state if replay == 1 else self.rng_state_replay2
        return [self.obs.reshape(-1), rs] + list(self.decoys)

    names = ["obs", "rng"] + ["decoy%d" % i for i in range(6)]


def philox_state(rng: np.random.Generator) -> np.ndarray:
    return rng.integers(0, 2 ** 32, size=4, dtype=np.uint32).astype("<u4").view(np.uint8).copy()


def advance_counter(state: np.ndarray, by: int = 1) -> np.ndarray:
    """Adds `by` to the 64-bit counter (words 2,3 of the Philox state), key unchanged."""
    w = state.view("<u4").copy()
    ctr = (int(w[2]) | (int(w[3]) << 32)) + by
    ctr &= (1 << 64) - 1
    w[2], w[3] = ctr & 0xFFFFFFFF, ctr >> 32
    return w.view(np.uint8).copy()


def config1(seed: int = 0, obs_shape=(256, 256, 3), n_decoys: int = 6, decoy_elems: int = 65536) -> Markovian:
    obs = _rng(seed, 0).integers(0, 256, size=obs_shape, dtype=np.uint8)
    rs = philox_state(_rng(seed, 1))
    decoys = [typed_random(_rng(seed, 2, i), "float16", 2 * decoy_elems) for i in range(n_decoys)]
    return Markovian(obs, rs, decoys, advance_counter(rs, 1))


# ---------------------------------------------------------------- config 2

@dataclass
class Bank:
    """Growing memory bank, struct-of-arrays, preallocated to `capacity` entries."""
    latents: np.ndarray   # uint8 view of bf16 [cap, 16, 60, 104]
    poses: np.ndarray     # uint8 view of fp32 [cap, 7]
    latent_entry_bytes: int
    pose_entry_bytes: int
    step_entries: int

    def prefix(self, entries: int):
        """The valid prefixes holding the first `entries` entries."""
        return [self.latents[: entries * self.latent_entry_bytes],
                self.poses[: entries * self.pose_entry_bytes]]


def config2(seed: int = 1, capacity: int = 512, latent_shape=(16, 60, 104), pose_dim: int = 7,
            step_entries: int = 8) -> Bank:
    le = int(np.prod(latent_shape))
    lat = bf16_normal(_rng(seed, 0), capacity * le).view(np.uint8)
    pos = _rng(seed, 1).uniform(-1.0, 1.0, size=capacity * pose_dim).astype(np.float32).view(np.uint8)
    return Bank(lat, pos, 2 * le, 4 * pose_dim, step_entries)


def pose_scores(bank: Bank, entries: int, anchor: int = 0) -> np.ndarray:
    """Caller-side relevance scores for a bank shrink (lower = more relevant):
    the squared distance, in float32, between each entry's pose position (its
    first three pose values) and the anchor entry's."""
    p = bank.poses[: entries * bank.pose_entry_bytes].view(np.float32).reshape(entries, -1)[:, :3]
    d = p - p[anchor]
    return (d * d).sum(axis=1, dtype=np.float32)


# ---------------------------------------------------------------- config 3

def kv_ring_geometry(layers: int, capacity: int, window: int, heads: int, head_dim: int,
                     seed: int, elem_bytes: int = 2):
    """Token-major KV ring [layers][2][capacity][heads][head_dim]: outer = 2*layers."""
    rng = _rng(seed, 7)
    row = heads * head_dim * elem_bytes
    h = wrapping_head(rng, capacity, window)
    h2 = other_head(rng, capacity, h)
    return Ring(2 * layers, capacity, row, window, h), h2


def host_kv_ring(ring: Ring, seed: int) -> np.ndarray:
    """bf16 N(0,1) bytes for a whole ring allocation, on the host."""
    return bf16_normal(_rng(seed, 0), ring.ring_bytes // 2).view(np.uint8)


def device_bf16_normal(numel: int, seed: int, device="cuda"):
    """bf16 N(0,1) of `numel` elements on the GPU, from torch's seeded generator."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    step = 1 << 28
    for s in range(0, numel, step):
        e = min(numel, s + step)
        out[s:e].normal_(0.0, 1.0, generator=g)
    return out


def device_bytes(nbytes: int, seed: int, device="cuda"):
    """Uniform random bytes on the GPU."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device=device, generator=g)


# ---------------------------------------------------------------- config 4

@dataclass
class SweepPlan:
    """Buffer sizes/dtypes, the designated must-snapshot set and, per replay
    k >= 2, which chunks of which designated buffer are rewritten."""
    sizes: list
    dtypes: list
    designated: list
    rewritten: dict = field(default_factory=dict)   # (k, b) -> sorted chunk indices
    replays: int = 8


def config4_plan(seed: int = 3, nbuf: int = 64, lo: int = 4096, hi: int = 1 << 28,
                 n_designated: int = 16, replays: int = 8, frac=(0.001, 0.05)) -> SweepPlan:
    rng = _rng(seed, 0)
    sizes, dtypes = [], []
    for _ in range(nbuf):
        dt = DTYPES[int(rng.integers(0, len(DTYPES)))]
        s = math.exp(rng.uniform(math.log(lo), math.log(hi)))
        isz = ITEMSIZE[dt]
        sizes.append(max(isz, int(s) // isz * isz))
        dtypes.append(dt)
    designated = sorted(int(x) for x in rng.choice(nbuf, size=n_designated, replace=False))
    plan = SweepPlan(sizes, dtypes, designated, {}, replays)
    for k in range(2, replays + 1):
        for b in designated:
            r = _rng(seed, 1, k, b)
            nch = (sizes[b] + 4095) // 4096
            f = r.uniform(*frac)
            m = min(nch, max(1, math.ceil(f * nch)))
            plan.rewritten[(k, b)] = sorted(int(x) for x in r.choice(nch, size=m, replace=False))
    return plan


def config4_host(plan: SweepPlan, seed: int = 3):
    """All replays on the host: replays[k-1][b] is a uint8 array."""
    base = [typed_random(_rng(seed, 2, b), plan.dtypes[b], plan.sizes[b]) for b in range(len(plan.sizes))]
    reps = [base]
    for k in range(2, plan.replays + 1):
        cur = [a for a in base]
        for b in plan.designated:
            a = base[b].copy()
            r = _rng(seed, 3, k, b)
            for c in plan.rewritten[(k, b)]:
                s, e = 4096 * c, min(4096 * (c + 1), a.size)
                a[s:e] = r.integers(0, 256, size=e - s, dtype=np.uint8)
            cur[b] = a
        reps.append(cur)
    return reps


# ---------------------------------------------------------------- config 5

@dataclass
class Batch:
    """Batched sessions: per session a KV window ring, an observation and RNG state."""
    sessions: int
    ring: Ring            # head field unused; per-session heads below
    heads: list
    obs_bytes: int
    rng_bytes: int
    restore_order: list   # the restored subset, in restore order
    restore_heads: list   # destination head for each restored session


def config5_plan(seed: int = 4, sessions: int = 1024, layers: int = 4, window: int = 2048,
                 capacity: int = 4096, heads: int = 8, head_dim: int = 128,
                 obs_shape=(480, 832, 3), restore_fraction: float = 0.5) -> Batch:
    rng = _rng(seed, 0)
    ring = Ring(2 * layers, capacity, heads * head_dim * 2, window, 0)
    hs = [int(x) for x in rng.integers(0, capacity, size=sessions)]
    order = [int(x) for x in rng.permutation(sessions)[: int(sessions * restore_fraction)]]
    rh = [int(x) for x in rng.integers(0, capacity, size=len(order))]
    return Batch(sessions, ring, hs, int(np.prod(obs_shape)), 16, order, rh)


# ---------------------------------------------------------------- device-side full-size inputs

def config3_device(seed: int = 2, layers: int = 32, capacity: int = 8192, window: int = 4096, heads: int = 8,
                   head_dim: int = 128, device="cuda"):
    """The windowed KV ring [layers][2][capacity][heads][head_dim] bf16 N(0,1) on the GPU.

    Returns (uint8 view of the ring, Ring geometry with a wrapping head, a different head)."""
    g, h2 = kv_ring_geometry(layers, capacity, window, heads, head_dim, seed)
    ring = device_bf16_normal(g.ring_bytes // 2, seed, device).view(__import__("torch").uint8)
    return ring, g, h2


def config4_device(plan: SweepPlan, seed: int = 3, device="cuda"):
    """Replays of the sweep on the GPU: reps[k-1][b] is a uint8 tensor; replays
    share the base tensor for every buffer they leave untouched."""
    import torch
    base = []
    for b, (n, dt) in enumerate(zip(plan.sizes, plan.dtypes)):
        if dt in ("float16", "bfloat16", "float32"):
            tdt = {"float16": torch.float16, "bfloat16": torch.bfloat16, "float32": torch.float32}[dt]
            g = torch.Generator(device=device)
            g.manual_seed(seed * 100003 + b)
            t = torch.empty(n // ITEMSIZE[dt], dtype=tdt, device=device).normal_(0.0, 1.0, generator=g)
            base.append(t.view(torch.uint8))
        else:
            base.append(device_bytes(n, seed * 100003 + b, device))
    reps = [base]
    for k in range(2, plan.replays + 1):
        cur = list(base)
        for b in plan.designated:
            a = base[b].clone()
            fresh = device_bytes(len(plan.rewritten[(k, b)]) * 4096, seed * 7919 + k * 131 + b, device)
            for j, c in enumerate(plan.rewritten[(k, b)]):
                s, e = 4096 * c, min(4096 * (c + 1), a.numel())
                a[s:e] = fresh[4096 * j:4096 * j + (e - s)]
            cur[b] = a
        reps.append(cur)
    return reps


def config5_device(plan: Batch, seed: int = 4, device="cuda"):
    """Per-session rings, observations and RNG states on the GPU, as [S, bytes] uint8 tensors."""
    import torch
    S, g = plan.sessions, plan.ring
    rings = device_bf16_normal(S * g.ring_bytes // 2, seed * 10 + 0, device).view(torch.uint8).view(S, g.ring_bytes)
    obs = device_bytes(S * plan.obs_bytes, seed * 10 + 1, device).view(S, plan.obs_bytes)
    rngs = device_bytes(S * plan.rng_bytes, seed * 10 + 2, device).view(S, plan.rng_bytes)
    return rings, obs, rngs

#!/usr/bin/env python3
"""Benchmark: batched session suspend/resume on one MI355X.

Workload (the default and the headline): 1024 sessions, each holding a KV
window of 4 layers x {K,V} x 2048 tokens x 8 heads x 128 bf16 (in a ring of
4096 token slots with a random head, so most windows wrap), a uint8
observation [480, 832, 3] and a 16-byte RNG state; inputs are seeded and
synthetic (generated on the GPU).  One step is one pass of the whole hot
path:
  1. checkpoint + fingerprint of all 1024 sessions in one batched launch
     (packed gather of each window, observation and RNG state into the
     device arena, XXH64 chunk fingerprints and Merkle roots from the same
     read);
  2. cross-replay classification of this step's chunk fingerprints against
     the previous step's (K = 2);
  3. fork of the 512 snapshots chosen for resume;
  4. restore of those 512 sessions, in permuted order and at new ring heads,
     in one launch;
  5. delete of every handle (the arena is reused by the next step).
The value is state GB/s: (bytes checkpointed + bytes restored) per second of
step time; 1 GB = 1e9 B.  The roofline entry is the fused pack+fingerprint
kernel, timed with HIP events on the context's stream.  The CPU baseline is
the oracle on a bounded sample of sessions, single-threaded.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--sessions", type=int, default=1024)
    ap.add_argument("--cpu-sessions", type=int, default=384, help="oracle sample size (sessions)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one plain 1 GiB device copy (for HBM counter scaling)")
    ap.add_argument("--summarize", nargs="+", metavar="DB",
                    help="no GPU: print kernel statistics from rocprofv3 databases (trace or --pmc runs)")
    return ap.parse_args()


def summarize(dbs):
    """Kernel statistics from rocprofv3 (rocpd) databases: durations from a
    kernel-trace run, per-dispatch counter values from --pmc runs.  Counter
    values are printed as rocprofv3 reports them (FETCH_SIZE / WRITE_SIZE in
    KiB per dispatch), together with the largest __amd_rocclr_copyBuffer
    dispatch, which is the plain 1 GiB calibration copy of --calibrate-copy."""
    import sqlite3

    def short(name):
        name = name.replace("pcs::(anonymous namespace)::", "").replace("(anonymous namespace)::", "")
        return name.split("(")[0][:60] if "pcs::" in name or name.startswith(("void k_", "k_", "void pcs")) \
            else name.split("(")[0][:60]

    for db in dbs:
        con = sqlite3.connect(db)
        cur = con.cursor()
        print("## %s" % db)
        has_pmc = cur.execute("select count(*) from counters_collection").fetchone()[0] > 0
        if has_pmc:
            print("| kernel | counter | dispatches | mean | min | max |")
            print("|---|---|---|---|---|---|")
            q = ("select kernel_name, counter_name, count(*), avg(value), min(value), max(value) "
                 "from counters_collection group by kernel_name, counter_name order by avg(value) desc")
            for name, cn, n, avg, mn, mx in cur.execute(q):
                if "pcs::" in name or "rocclr_copyBuffer" in name:
                    print("| %s | %s | %d | %.1f | %.1f | %.1f |" % (short(name), cn, n, avg, mn, mx))
        else:
            print("| kernel | calls | avg us | min us | max us | total ms |")
            print("|---|---|---|---|---|---|")
            q = ("select name, count(*), avg(duration), min(duration), max(duration), sum(duration) "
                 "from kernels group by name order by sum(duration) desc")
            for name, n, avg, mn, mx, tot in cur.execute(q):
                if "pcs::" in name or "rocclr_copyBuffer" in name:
                    print("| %s | %d | %.1f | %.1f | %.1f | %.3f |" % (short(name), n, avg / 1e3, mn / 1e3,
                                                                        mx / 1e3, tot / 1e6))
        print()


def traffic_record():
    """Scaled HBM traffic of the fused pack+fingerprint kernel, measured with
    rocprofv3 counters, if the kernel source is unchanged since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_hash_copy_batch1024_traffic.json")
    src = os.path.join(ROOT, "paper_2607_21686_amd", "csrc", "pcs_kernels.hip")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    return rec if rec.get("kernel_source_sha256") == sha else None


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU: this build has no multi-GPU path (sessions shard across GPUs "
              "with no exchange; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_21686_amd as P
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    plan = W.config5_plan(4, sessions=args.sessions)
    g = plan.ring
    S = plan.sessions
    R = len(plan.restore_order)
    ring_bytes = g.ring_bytes
    log("sessions %d, ring %d B, window %d B, obs %d B, restore %d" % (S, ring_bytes, g.window_bytes,
                                                                          plan.obs_bytes, R))

    t0 = time.time()
    rings = W.device_bf16_normal(S * ring_bytes // 2, seed=40).view(torch.uint8).view(S, ring_bytes)
    obs = W.device_bytes(S * plan.obs_bytes, seed=41).view(S, plan.obs_bytes)
    rngs = W.device_bytes(S * plan.rng_bytes, seed=42).view(S, plan.rng_bytes)
    dst_rings = torch.empty(R, ring_bytes, dtype=torch.uint8, device=dev)
    dst_obs = torch.empty(R, plan.obs_bytes, dtype=torch.uint8, device=dev)
    dst_rngs = torch.empty(R, plan.rng_bytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    log("inputs generated in %.1f s" % (time.time() - t0))

    plans = P.BufArray([b for s in range(S) for b in (
        P.ring(rings[s], g.outer, g.capacity, g.row_bytes, plan.heads[s], g.window),
        P.flat(obs[s]), P.flat(rngs[s]))])
    dsts = P.BufArray([b for k in range(R) for b in (
        P.ring(dst_rings[k], g.outer, g.capacity, g.row_bytes, plan.restore_heads[k], g.window),
        P.flat(dst_obs[k]), P.flat(dst_rngs[k]))])
    per_session_chunks = [P.chunk_count(g.window_bytes), P.chunk_count(plan.obs_bytes), P.chunk_count(plan.rng_bytes)]
    cpb_list = per_session_chunks * S
    cpb = P.u64_array(cpb_list)
    total_chunks = sum(cpb_list)
    state_per_session = g.window_bytes + plan.obs_bytes + plan.rng_bytes
    slot_bytes = sum(c * 4096 for c in per_session_chunks)
    meta = ((8 * sum(per_session_chunks) + 8 * 4 + 4095) // 4096) * 4096
    arena_bytes = S * (slot_bytes + meta) + (1 << 30)
    arena = torch.empty(arena_bytes, dtype=torch.uint8, device=dev)
    ctx = P.Context(arena)
    H = torch.zeros(2, total_chunks, dtype=torch.int64, device=dev)
    roots = torch.zeros(3 * S, dtype=torch.int64, device=dev)
    sroots = torch.zeros(S, dtype=torch.int64, device=dev)
    nwords = sum((c + 63) // 64 for c in cpb_list)
    bitmap = torch.zeros(nwords, dtype=torch.int64, device=dev)
    labels = torch.zeros(3 * S, dtype=torch.uint8, device=dev)
    nb_ckpt = [3] * S
    nb_rest = [3] * R
    order = plan.restore_order

    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    state = {"cur": 0}

    def step():
        cur = state["cur"]
        snaps = ctx.checkpoint_batch(plans, hash=True, chunk_hashes=H[cur], roots=roots, session_roots=sroots,
                                     nbufs=nb_ckpt)
        ctx.classify(H, 2, cpb, bitmap, labels)
        forks = [ctx.fork(snaps[s]) for s in order]
        ctx.restore_batch(forks, dsts, nbufs=nb_rest)
        for h in snaps:
            ctx.delete(h)
        for h in forks:
            ctx.delete(h)
        state["cur"] = cur ^ 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.set_timing(False)
    kt = {k: ctx.kernel_time(k) for k in ("pack_hash", "copy", "classify", "merkle", "map")}

    # Fingerprint-only pass over every session's state (read once), timed the
    # same way: the "fingerprint GB/s" half of the metric.
    fp_reps = 5
    ctx.fingerprint(plans, H[0], roots, None)
    torch.cuda.synchronize()
    ctx.set_timing(True)
    for _ in range(fp_reps):
        ctx.fingerprint(plans, H[0], roots, None)
    ctx.set_timing(False)
    n_fp, ms_fp = ctx.kernel_time("hash")
    ctx.kernel_time("merkle")
    ctx.kernel_time("map")
    avg_fp = ms_fp / max(1, n_fp)

    # Spot check of the timed work: restored sessions equal their sources.
    for k in (0, R - 1):
        s = order[k]
        src = rings[s].view(g.outer, g.capacity, g.row_bytes)
        dst = dst_rings[k].view(g.outer, g.capacity, g.row_bytes)
        idx_s = (torch.arange(g.window, device=dev) + plan.heads[s]) % g.capacity
        idx_d = (torch.arange(g.window, device=dev) + plan.restore_heads[k]) % g.capacity
        assert torch.equal(src[:, idx_s], dst[:, idx_d]), "restored window differs"
        assert torch.equal(obs[s], dst_obs[k]) and torch.equal(rngs[s], dst_rngs[k]), "restored flat state differs"
    labels_host = labels.cpu().numpy()
    assert not labels_host.any(), "unchanged sessions must classify as recomputable"

    ms_per_step = 1e3 * elapsed / args.steps
    ckpt_state = S * state_per_session
    rest_state = R * state_per_session
    value = (ckpt_state + rest_state) / (elapsed / args.steps) / 1e9

    n_ph, ms_ph = kt["pack_hash"]
    avg_ph = ms_ph / max(1, n_ph)
    alg_ph = 2 * ckpt_state                      # read the state once, write it once
    achieved = alg_ph / (avg_ph * 1e-3) / 1e9
    n_cp, ms_cp = kt["copy"]
    avg_cp = ms_cp / max(1, n_cp)
    achieved_restore = 2 * rest_state / (avg_cp * 1e-3) / 1e9

    rec = traffic_record()
    traffic = rec["traffic_bytes_per_launch"] if rec and rec.get("sessions") == S else None

    out = {
        "metric": "checkpoint+restore GB/s and fingerprint GB/s at 1 MI355X; % of HBM peak",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic (seeded, generated on the GPU)",
        "config": {"workload": "batched session suspend/resume: %d sessions x (KV window 4x2x2048x8x128 bf16 "
                               "in a 4096-slot ring, obs 480x832x3 u8, RNG 16 B); checkpoint+fingerprint all, "
                               "classify vs previous step, fork+restore %d permuted" % (S, R),
                   "sessions": S, "restored": R, "state_bytes_per_session": state_per_session},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "kernel": "k_hash<copy> (fused pack + fingerprint)",
                     "avg_ms": round(avg_ph, 4), "algorithmic_bytes": alg_ph},
        "fingerprint": {"GBps_state": round(ckpt_state / (avg_fp * 1e-3) / 1e9, 1),
                        "frac_of_peak": round(ckpt_state / (avg_fp * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                        "kernel_ms": round(avg_fp, 4), "bytes": ckpt_state,
                        "what": "pcs_fingerprint of all sessions (read once, chunk hashes + roots)"},
        "breakdown": {
            "checkpoint_fingerprint_GBps_state": round(ckpt_state / (avg_ph * 1e-3) / 1e9, 1),
            "restore_kernel_GBps_hbm": round(achieved_restore, 1),
            "restore_kernel_ms": round(avg_cp, 4),
            "pack_hash_ms": round(avg_ph, 4),
            "classify_ms": round(kt["classify"][1] / max(1, args.steps), 4),
            "merkle_ms": round(kt["merkle"][1] / max(1, args.steps), 4),
            "map_ms": round(kt["map"][1] / max(1, args.steps), 4),
        },
    }

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, plan, rings, obs, rngs, value)

    print(json.dumps(out), flush=True)
    ctx.close()


def cpu_baseline(args, plan, rings, obs, rngs, gpu_value):
    """The oracle, as it stands, on a bounded sample of the same workload,
    pinned to one host core: per sampled session, fingerprint + checkpoint,
    classification against a second fingerprint pass, and (every other
    session) fork + restore at a new head.  Only oracle compute is timed;
    each session's bytes are copied to the host before its timed part."""
    import numpy as np

    import oracle
    g = plan.ring
    n = max(2, min(args.cpu_sessions, plan.sessions))
    oracle.build()
    prev = os.sched_getaffinity(0)
    core = min(prev)
    os.sched_setaffinity(0, {core})
    elapsed, restored = 0.0, 0
    cpb = [oracle.chunk_count(x) for x in (g.window_bytes, plan.obs_bytes, plan.rng_bytes)]
    try:
        for s in range(n):
            r, o, q = rings[s].cpu().numpy(), obs[s].cpu().numpy(), rngs[s].cpu().numpy()
            t0 = time.perf_counter()
            st = oracle.Store()
            win = oracle.ring_window(r, g.outer, g.outer_stride, g.capacity, g.row_bytes, plan.heads[s], g.window)
            h = st.checkpoint([win, o, q])
            hv = np.concatenate(st.snapshot(h).hashes)
            oracle.classify(np.stack([hv, hv]), cpb)
            if s % 2 == 0:
                f = st.fork(h)
                w2, o2, q2 = st.restore(f)
                dst = np.empty(g.ring_bytes, dtype=np.uint8)
                oracle.ring_place(w2, dst, g.outer, g.outer_stride, g.capacity, g.row_bytes,
                                  (plan.heads[s] + 1) % g.capacity, g.window)
                restored += 1
            elapsed += time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, prev)
    per = g.window_bytes + plan.obs_bytes + plan.rng_bytes
    v = (n + restored) * per / elapsed / 1e9
    return {"value": round(v, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "%d sessions checkpointed+fingerprinted and classified, %d forked+restored; %.1f s of "
                      "oracle compute on core %d" % (n, restored, elapsed, core),
            "gpu_over_cpu": round(gpu_value / v, 1)}


if __name__ == "__main__":
    main()

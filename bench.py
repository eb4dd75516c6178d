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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="batch",
                    choices=["batch", "kv-ring", "verify", "sweep", "bank", "markovian", "shrink", "discover", "export"],
                    help="batch (default, the headline) or one of the other seeded configurations")
    ap.add_argument("--sessions", type=int, default=1024)
    ap.add_argument("--cpu-sessions", type=int, default=512, help="oracle sample size (sessions)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one plain 1 GiB device copy (for HBM counter scaling)")
    ap.add_argument("--traffic", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                    help="no GPU: write the scaled HBM traffic record of the workload's dominant kernels (batch, "
                         "kv-ring or verify) from a FETCH_SIZE and a WRITE_SIZE run of this bench with "
                         "--calibrate-copy and the same --workload")
    ap.add_argument("--arena-mib", type=int, default=0,
                    help="bank workload: arena size in MiB (default 1024)")
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


# Per workload: the scaled-traffic record the bench line reads, and the
# kernels it covers (name pattern in rocprofv3's kernel names, label).
TRAFFIC = {
    "batch": ("k_hash_copy_batch1024_traffic.json",
              [("pack", r"k_hash<pcs::\w+Tables, 1, 1024, 512, 64, false>",
                "k_hash<pack, 1024 lanes, 512 B slices, 64 chunks, nontemporal stores> (fused pack + fingerprint)"),
               ("copy", r"k_copy<pcs::\w+Tables, false, 512, 1024, 64>",
                "k_copy<unpack, 512 lanes, 1 KiB slices, 64 chunks> (restore scatter)")]),
    "kv-ring": ("k_hash_copy_kv_ring_1gib_traffic.json",
                [("pack", r"k_hash_staggered<pcs::\w+Tables, 1, 1024, 512, 64>",
                  "k_hash_staggered<pack, 1024 lanes, 512 B slices, 64 chunks> (fused pack + fingerprint, "
                  "first round staggered, write-back stores)"),
                 ("copy", r"k_copy<pcs::\w+Tables, false, 512, 1024, 64>",
                  "k_copy<unpack, 512 lanes, 1 KiB slices, 64 chunks> (restore scatter)")]),
    "verify": ("k_hash_verify_kv_ring_1gib_traffic.json",
               [("verify", r"k_hash_staggered<pcs::\w+Tables, 3, 1024, 1024, 64>",
                 "k_hash_staggered<verify, 1024 lanes, 1 KiB slices, 64 chunks> (restore + fingerprint + compare, "
                 "first round staggered)"),
                ("copy", r"k_copy<pcs::\w+Tables, false, 512, 1024, 64>",
                 "k_copy<unpack, 512 lanes, 1 KiB slices, 64 chunks> (plain restore)")]),
}
TRAFFIC_JSON = os.path.join(ROOT, "profiles", TRAFFIC["batch"][0])
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_21686_amd", "csrc", f)
                  for f in ("pcs_kernels.hip", "pcs_device.h", "pcs_layout.h")]


def kernel_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def traffic_record(workload="batch"):
    """Scaled HBM traffic of the workload's dominant kernels, measured with
    rocprofv3 counters, if the kernel sources are unchanged since."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", TRAFFIC[workload][0])))
    except (OSError, ValueError, KeyError):
        return None
    return rec if rec.get("kernel_source_sha256") == kernel_source_sha() else None


def _state_bytes(workload, sessions):
    """Algorithmic bytes of one launch of each kernel the traffic record
    covers: the state read once and written once."""
    import workloads as W
    if workload == "batch":
        plan = W.config5_plan(4, sessions=sessions)
        per = plan.ring.window_bytes + plan.obs_bytes + plan.rng_bytes
        return {"pack": 2 * per * sessions, "copy": 2 * per * len(plan.restore_order)}
    g, _ = W.kv_ring_geometry(32, 8192, 4096, 8, 128, 2)
    return {"pack": 2 * g.window_bytes, "copy": 2 * g.window_bytes, "verify": 2 * g.window_bytes}


def traffic(fetch_db, write_db, workload="batch", sessions=1024):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB, as rocprofv3 reports them)
    of the workload's dominant kernels, each scaled by what the same counter
    reads for the plain 1 GiB calibration copy (true traffic 1 GiB read +
    1 GiB written), against the algorithmic bytes of one launch (state read
    once and written once)."""
    import re
    import sqlite3
    fname, kernels = TRAFFIC[workload]

    def per_kernel(db, counter):
        cur = sqlite3.connect(db).cursor()
        q = "select kernel_name, value from counters_collection where counter_name = ?"
        rows = cur.execute(q, (counter,)).fetchall()
        pick = lambda pat: [v for n, v in rows if re.search(pat, n)]
        out = {key: pick(pat) for key, pat, _ in kernels}
        out["calib"] = max(pick("rocclr_copyBuffer"))
        return out

    f, w = per_kernel(fetch_db, "FETCH_SIZE"), per_kernel(write_db, "WRITE_SIZE")
    gib_kib = (1 << 30) / 1024
    fs, ws = gib_kib / f["calib"], gib_kib / w["calib"]
    alg = _state_bytes(workload, sessions)
    mean = lambda xs: sum(xs) / len(xs)

    def one(key):
        fk, wk = mean(f[key]), mean(w[key])
        t = int(round((fk * fs + wk * ws) * 1024))
        return {"fetch_KiB_per_dispatch": round(fk, 1), "write_KiB_per_dispatch": round(wk, 1),
                "dispatches": [len(f[key]), len(w[key])], "traffic_bytes_per_launch": t,
                "algorithmic_bytes_per_launch": alg[key], "traffic_over_algorithmic": round(t / alg[key], 5)}

    (k0, _, label0), (k1, _, label1) = kernels
    rec = {"kernel": label0, "workload": workload, "calibration_copy_bytes": 1 << 30,
           "calibration_fetch_KiB": round(f["calib"], 1), "calibration_write_KiB": round(w["calib"], 1),
           "fetch_scale": round(fs, 6), "write_scale": round(ws, 6)}
    if workload == "batch":
        rec["sessions"] = sessions
    rec.update(one(k0))
    rec["second_kernel"] = dict(kernel=label1, **one(k1))
    rec["kernel_source_sha256"] = kernel_source_sha()
    # The commands that made the two databases (rocprofv3 writes <dir>/<name>_results.db).
    wl = "" if workload == "batch" else " --workload %s" % workload

    def pmc_cmd(counter, db):
        rel = os.path.relpath(db)
        name = os.path.basename(rel)[:-len("_results.db")] if rel.endswith("_results.db") else "pmc"
        return ("rocprofv3 --pmc %s -d %s -o %s -- python3 bench.py%s --steps 2 --warmup 1 --no-cpu-baseline "
                "--calibrate-copy" % (counter, os.path.dirname(rel) or ".", name, wl))
    rec["commands"] = [pmc_cmd("FETCH_SIZE", fetch_db), pmc_cmd("WRITE_SIZE", write_db),
                       "python3 bench.py%s --traffic %s %s" % (wl, os.path.relpath(fetch_db), os.path.relpath(write_db))]
    with open(os.path.join(ROOT, "profiles", fname), "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec, indent=1))


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return
    if args.traffic:
        traffic(*args.traffic, workload=args.workload, sessions=args.sessions)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path.  Sessions are independent, so "
              "each GPU would run its own share of them with its own arena and stream, with no exchange "
              "between GPUs.", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        # One plain 1 GiB device-to-device copy: the reference dispatch that
        # scales FETCH_SIZE / WRITE_SIZE to bytes.
        import torch
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    if args.workload != "batch":
        out = OTHER[args.workload](args)
        print(json.dumps(out), flush=True)
        return
    run_batch(args)


def _pct(sorted_vals, q):
    """q-th percentile of sorted values (linear interpolation between ranks)."""
    if not sorted_vals:
        return float("nan")
    x = (len(sorted_vals) - 1) * q / 100.0
    lo = int(x)
    hi = min(lo + 1, len(sorted_vals) - 1)
    return sorted_vals[lo] + (sorted_vals[hi] - sorted_vals[lo]) * (x - lo)


def run_batch(args):
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
    per_session_chunks = P.chunk_counts(plans.bufs[:3])[0]
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

    # Kernel times from events recorded on the stream around each launch: the
    # kernels run for milliseconds (the dispatch latency that the events take
    # in is under 0.1% of them), and the dispatches' own timestamps made the
    # step times of this workload more spread on MI355X.
    ctx.set_timing(True)
    # Events between steps on the context's stream give each step's device
    # time without synchronising inside the timed region.
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks[0].record()
    for i in range(args.steps):
        step()
        marks[i + 1].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.set_timing(False)
    kt = {k: ctx.kernel_time(k) for k in ("pack_hash", "copy", "classify", "merkle", "map")}
    step_ms = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))

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

    rec = traffic_record("batch")
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
        "step_ms_device": {"p10": round(_pct(step_ms, 10), 4), "p50": round(_pct(step_ms, 50), 4),
                           "p90": round(_pct(step_ms, 90), 4)},
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
            "pinned_core": core, "host_cores": os.cpu_count(), "cores_available": len(prev),
            "gpu_over_cpu": round(gpu_value / v, 1)}


# ------------------------------------------------------------------ other configurations

def _line(args, metric_value, ms_per_step, workload, cfg, roof_kernel, alg_bytes, avg_ms, extra=None):
    achieved = alg_bytes / (avg_ms * 1e-3) / 1e9
    rec = traffic_record(args.workload)
    traffic = rec["traffic_bytes_per_launch"] if rec and rec.get("algorithmic_bytes_per_launch") == alg_bytes else None
    out = {
        "metric": "checkpoint+restore GB/s and fingerprint GB/s at 1 MI355X; % of HBM peak",
        "value": round(metric_value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic (seeded, generated on the GPU)",
        "config": dict({"workload": workload}, **cfg),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic, "kernel": roof_kernel,
                     "avg_ms": round(avg_ms, 4), "algorithmic_bytes": alg_bytes},
    }
    if _STEP_DIST is not None:
        out["step_ms_device"] = _STEP_DIST
    if extra:
        out["breakdown"] = extra
    return out


_STEP_DIST = None  # p10/p50/p90 of the device step times of the last _timed run


def _timed(args, ctx, step, kernels):
    """Wall time per step from a pass without the library's per-launch timing
    events (which cost a few microseconds of host time per launch, enough to
    slow workloads of many small launches), then the distribution of device
    step times (p10/p50/p90) from a second pass, then kernel times from a
    third pass of the same steps with the timing events on, as each kernel
    dispatch's own begin and end (these kernels run for tens to hundreds of
    microseconds, so the few microseconds of dispatch latency that events
    recorded around a launch would add are not small against them)."""
    import torch
    global _STEP_DIST
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # Device time of each step: events recorded between steps on the
    # context's stream, no synchronisation inside the pass.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(ctx.stream)
    for k in range(args.steps):
        step()
        evs[k + 1].record(ctx.stream)
    torch.cuda.synchronize()
    ms = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps))
    _STEP_DIST = {"p10": round(_pct(ms, 10), 4), "p50": round(_pct(ms, 50), 4), "p90": round(_pct(ms, 90), 4)}
    for k in kernels:
        ctx.kernel_time(k)
    ctx.set_timing(True, dispatch=True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ctx.set_timing(False)
    return elapsed / args.steps, {k: ctx.kernel_time(k) for k in kernels}


def _oracle_leg(args, work, state_bytes, sample, gpu_value, reps=1):
    """The oracle, as it stands, pinned to one host core, on one bounded
    sample of a workload (`work`, on host copies of its inputs made before
    timing): rate = state_bytes per call of `work` / time, in the unit of
    the workload's own value (GB/s)."""
    import oracle
    oracle.build()
    prev = os.sched_getaffinity(0)
    core = min(prev)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        for _ in range(reps):
            work()
        elapsed = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, prev)
    v = reps * state_bytes / elapsed / 1e9
    return {"value": round(v, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "%s; %.2f s of oracle compute on core %d" % (sample, elapsed, core),
            "pinned_core": core, "host_cores": os.cpu_count(), "cores_available": len(prev),
            "gpu_over_cpu": round(gpu_value / v, 1)}


def run_kv_ring(args):
    """Windowed KV context: checkpoint + fingerprint of the 512 MiB window of a
    1 GiB ring (wrapping head), fork, two restores at new heads, delete."""
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    ring, g, h2 = W.config3_device(2)
    ctx = P.Context(torch.empty((512 << 20) + (64 << 20), dtype=torch.uint8, device="cuda"))
    src = P.BufArray([P.ring(ring, g.outer, g.capacity, g.row_bytes, g.head, g.window)])
    a, b = torch.empty_like(ring), torch.empty_like(ring)
    da = P.BufArray([P.ring(a, g.outer, g.capacity, g.row_bytes, h2, g.window)])
    db = P.BufArray([P.ring(b, g.outer, g.capacity, g.row_bytes, (h2 + 1234) % g.capacity, g.window)])
    H = torch.zeros(g.window_bytes // 4096, dtype=torch.int64, device="cuda")

    def step():
        s = ctx.checkpoint(src, hash=True, chunk_hashes=H)
        f = ctx.fork(s)
        ctx.restore(s, da)
        ctx.restore(f, db)
        ctx.delete(s)
        ctx.delete(f)
    t, kt = _timed(args, ctx, step, ["pack_hash", "copy", "merkle", "map"])
    W_ = g.window_bytes
    n, ms = kt["pack_hash"]
    nc, mc = kt["copy"]
    out = _line(args, 3 * W_ / t / 1e9, t * 1e3, "windowed KV ring: 32 layers x 2 x 8192 slots x 8 x 128 bf16 "
                "(1 GiB), 4096-token window at a wrapping head; checkpoint+fingerprint, fork, 2 restores",
                {"window_bytes": W_}, "k_hash_staggered<pack> (fused pack + fingerprint, first round staggered, write-back stores)",
                2 * W_, ms / n,
                {"restore_ms": round(mc / nc, 4), "restore_GBps_hbm": round(2 * W_ / (mc / nc * 1e-3) / 1e9, 1)})
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        ring_h = ring.cpu().numpy()
        dst_h = [np.empty_like(ring_h), np.empty_like(ring_h)]
        geo = (g.outer, g.outer_stride, g.capacity, g.row_bytes)

        def work():
            st = oracle.Store()
            snap = st.checkpoint([oracle.ring_window(ring_h, *geo, g.head, g.window)])
            fork = st.fork(snap)
            for h, d, head in ((snap, dst_h[0], h2), (fork, dst_h[1], (h2 + 1234) % g.capacity)):
                (w,) = st.restore(h)
                oracle.ring_place(w, d, *geo, head, g.window)
        out["cpu_baseline"] = _oracle_leg(args, work, 3 * W_, "3 whole steps: checkpoint + fingerprint of the "
                                          "512 MiB window, fork, 2 restores at new heads", out["value"], reps=3)
    return out


def run_verify(args):
    """Verify-on-restore on the windowed KV context: one snapshot of the 512
    MiB window (taken with fingerprints, outside the timed steps); each step
    restores it with verification (restore fused with fingerprinting of the
    bytes written and a comparison with the stored fingerprints) at one new
    head and without verification at another, so the two rates sit side by
    side."""
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    ring, g, h2 = W.config3_device(2)
    ctx = P.Context(torch.empty((512 << 20) + (64 << 20), dtype=torch.uint8, device="cuda"))
    src = P.BufArray([P.ring(ring, g.outer, g.capacity, g.row_bytes, g.head, g.window)])
    snap = ctx.checkpoint(src, hash=True)
    a, b = torch.empty_like(ring), torch.empty_like(ring)
    da = P.BufArray([P.ring(a, g.outer, g.capacity, g.row_bytes, h2, g.window)])
    db = P.BufArray([P.ring(b, g.outer, g.capacity, g.row_bytes, (h2 + 1234) % g.capacity, g.window)])
    words = (g.window_bytes // 4096 + 63) // 64
    bad = torch.zeros(words, dtype=torch.int64, device="cuda")

    def step():
        ctx.restore_verify(snap, da, bad)      # no per-buffer labels: one kernel per call
        ctx.restore(snap, db)
    t, kt = _timed(args, ctx, step, ["verify", "copy"])
    assert not bad.any().item(), "verification flagged an intact snapshot"
    W_ = g.window_bytes
    nv, mv = kt["verify"]
    nc, mc = kt["copy"]
    v_ms = mv / nv
    ctx.delete(snap)
    out = _line(args, 2 * W_ / t / 1e9, t * 1e3, "verify on restore, windowed KV ring: 32 layers x 2 x 8192 slots x 8 "
                "x 128 bf16 (1 GiB), 4096-token window; per step one restore with verification and one without",
                {"window_bytes": W_}, "k_hash_staggered<verify> (restore + fingerprint + compare, first round staggered)",
                2 * W_, v_ms,
                {"verify_ms": round(v_ms, 4), "restore_ms": round(mc / nc, 4),
                 "verify_GBps_hbm": round(2 * W_ / (v_ms * 1e-3) / 1e9, 1),
                 "restore_GBps_hbm": round(2 * W_ / (mc / nc * 1e-3) / 1e9, 1)})
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        ring_h = ring.cpu().numpy()
        dst_h = [np.empty_like(ring_h), np.empty_like(ring_h)]
        geo = (g.outer, g.outer_stride, g.capacity, g.row_bytes)
        st = oracle.Store()
        osnap = st.checkpoint([oracle.ring_window(ring_h, *geo, g.head, g.window)])
        stored = st.snapshot(osnap).hashes[0]

        def work():
            (w,) = st.restore(osnap)
            oracle.ring_place(w, dst_h[0], *geo, h2, g.window)
            _, labels = oracle.classify(np.stack([stored, oracle.chunk_hashes(w)]), [stored.size])
            assert not labels.any()
            (w2,) = st.restore(osnap)
            oracle.ring_place(w2, dst_h[1], *geo, (h2 + 1234) % g.capacity, g.window)
        out["cpu_baseline"] = _oracle_leg(args, work, 2 * W_, "4 whole steps: a restore verified against the "
                                          "stored fingerprints and a plain restore of the 512 MiB window",
                                          out["value"], reps=4)
    return out


def run_sweep(args):
    """Classification sweep: fingerprint all 8 replays of 64 buffers in one
    call, then classify (K = 8)."""
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    plan = W.config4_plan(3)
    reps = W.config4_device(plan, 3)
    K = plan.replays
    cpb, total = P.chunk_counts([P.flat(t) for t in reps[0]])
    ctx = P.Context(torch.empty(256 << 20, dtype=torch.uint8, device="cuda"))
    bufs = P.BufArray([P.flat(t) for rep in reps for t in rep])
    H = torch.zeros(K * total, dtype=torch.int64, device="cuda")
    bm = torch.zeros(sum((c + 63) // 64 for c in cpb), dtype=torch.int64, device="cuda")
    lab = torch.zeros(len(cpb), dtype=torch.uint8, device="cuda")
    cpa = P.u64_array(cpb)

    def step():
        ctx.fingerprint(bufs, H)
        ctx.classify(H, K, cpa, bm, lab)
    t, kt = _timed(args, ctx, step, ["hash", "classify", "map", "merkle"])
    nbytes = K * sum(plan.sizes)
    n, ms = kt["hash"]
    out = _line(args, nbytes / t / 1e9, t * 1e3, "classification sweep: 64 buffers, log-uniform 4 KiB-256 MiB, "
                "5 dtypes, K=8 replays (16 designated buffers with rewritten chunks); fingerprint + classify",
                {"bytes_per_step": nbytes, "replays": K}, "k_hash (fingerprint)", nbytes, ms / n,
                {"classify_ms": round(kt["classify"][1] / args.steps, 4)})
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        host = [[x.cpu().numpy() for x in reps[k]] for k in range(2)]

        def work():
            hs = [oracle.fingerprint(host[k])[0] for k in range(2)]
            oracle.classify(np.stack(hs), cpb)
        out["cpu_baseline"] = _oracle_leg(args, work, 2 * sum(plan.sizes), "2 of the 8 replays fingerprinted "
                                          "(all 64 buffers each), then classified (K = 2), 3 times", out["value"], reps=3)
    return out


def run_bank(args):
    """Growing bank: 64 incremental checkpoints (8 entries each) and 64
    restores in random order; value counts the logical state each covers."""
    import numpy as np
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    bank = W.config2(1)
    lat = torch.from_numpy(bank.latents.copy()).cuda()
    pos = torch.from_numpy(bank.poses.copy()).cuda()
    # 1 GiB of arena by default (--arena-mib): the 64 snapshots keep about
    # 130 MB; each incremental checkpoint in flight also reserves one slot per
    # chunk of its prefix until the stream has produced its stored-chunk count.
    arena_mib = args.arena_mib or 1024
    ctx = P.Context(torch.empty(arena_mib << 20, dtype=torch.uint8, device="cuda"))
    plans = [P.BufArray([P.flat(lat, 8 * j * bank.latent_entry_bytes), P.flat(pos, 8 * j * bank.pose_entry_bytes)])
             for j in range(1, 65)]
    out_l, out_p = torch.empty_like(lat), torch.empty_like(pos)
    dsts = [P.BufArray([P.flat(out_l, 8 * j * bank.latent_entry_bytes), P.flat(out_p, 8 * j * bank.pose_entry_bytes)])
            for j in range(1, 65)]
    order = [int(x) for x in np.random.default_rng(1).permutation(64)]

    def step():
        hs, parent = [], 0
        for j in range(64):
            h = ctx.checkpoint(plans[j], parent=parent, hash=parent == 0)
            hs.append(h)
            parent = h
        for j in order:
            ctx.restore(hs[j], dsts[j])
        for h in hs:
            ctx.delete(h)
    t, kt = _timed(args, ctx, step, ["pack_hash", "incremental", "copy", "merkle", "map"])
    entry = bank.latent_entry_bytes + bank.pose_entry_bytes
    state = sum(8 * j * entry for j in range(1, 65))
    n, ms = kt["incremental"]

    # Algorithmic bytes of incremental checkpoint j (parent j-1, j = 2..64):
    # read the valid prefix once (V_j = 8j entries), read + write the dirty
    # chunks (D_j: the 390 chunks of the 8 new latents, which fill whole
    # chunks, and the pose buffer's last chunk, plus the one before it when
    # the 224 new pose bytes cross a chunk boundary).
    def dirty_chunks(j):
        return 390 + 1 + (1 if (224 * j) // 4096 != (224 * (j - 1)) // 4096 and (224 * j) % 4096 else 0)

    def alg_bytes(j):
        return 8 * j * entry + 2 * 4096 * dirty_chunks(j)
    whole = sum(alg_bytes(j) for j in range(2, 65))

    # Late steps (j = 33..64, prefixes of 53-102 MB): a further pass whose
    # kernel timing is on only for those checkpoints.  Consecutive
    # checkpoints re-read a prefix that fits the 256 MB memory-side cache, so
    # a cold pass also writes 512 MiB of other memory before each timed
    # checkpoint (the fill is not timed).
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")

    def late_run(cold):
        hs, parent = [], 0
        for j in range(64):
            if j >= 32:
                if cold:
                    ctx.set_timing(False)
                    flush.fill_(j)
                ctx.set_timing(True, dispatch=True)
            h = ctx.checkpoint(plans[j], parent=parent, hash=parent == 0)
            hs.append(h)
            parent = h
        ctx.set_timing(False)
        for h in hs:
            ctx.delete(h)

    def late_ms(cold):
        ctx.kernel_time("incremental")
        for _ in range(args.steps):
            late_run(cold)
        torch.cuda.synchronize()
        return ctx.kernel_time("incremental")[1] / args.steps
    for k in ("incremental", "pack_hash", "copy", "merkle", "map"):
        ctx.kernel_time(k)
    late_ms, late_cold_ms = late_ms(False), late_ms(True)
    late_bytes = sum(alg_bytes(j) for j in range(33, 65))
    whole_GBps = whole / (ms / args.steps * 1e-3) / 1e9
    out = _line(args, 2 * state / t / 1e9, t * 1e3, "growing memory bank: bf16 latents [16,60,104] + fp32 pose [7] "
                "per entry, 0->512 entries in steps of 8; 64 incremental checkpoints + 64 restores (random order)",
                {"state_bytes_checkpointed_and_restored": 2 * state, "arena_mib": arena_mib},
                "incremental checkpoint kernels of steps 33-64 (fingerprint + diff, Merkle + scan, "
                "slot assignment, dirty copy), 512 MiB of other memory written before each", late_bytes, late_cold_ms,
                {"incremental_ms_per_run": round(ms / args.steps, 4),
                 "incremental_GBps_hbm_whole_run": round(whole_GBps, 1),
                 "incremental_frac_whole_run": round(whole_GBps / HBM_PEAK_GBPS, 4),
                 "incremental_launches_per_run": round(n / args.steps, 1),
                 "late_steps_bytes": late_bytes, "late_steps_cold_ms": round(late_cold_ms, 4),
                 "late_steps_warm_ms": round(late_ms, 4),
                 "late_steps_warm_frac": round(late_bytes / (late_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                 "restore_ms_per_run": round(kt["copy"][1] / args.steps, 4)})
    if not args.no_cpu_baseline:
        import oracle
        lat_h = np.ascontiguousarray(bank.latents).view(np.uint8).reshape(-1)
        pos_h = np.ascontiguousarray(bank.poses).view(np.uint8).reshape(-1)
        le, pe = bank.latent_entry_bytes, bank.pose_entry_bytes

        def work():
            st, hs, parent = oracle.Store(), [], 0
            for j in range(1, 65):
                parent = st.checkpoint([lat_h[:8 * j * le], pos_h[:8 * j * pe]], parent)
                hs.append(parent)
            for j in order:
                st.restore(hs[j])
        out["cpu_baseline"] = _oracle_leg(args, work, 2 * state, "one whole run: 64 chained incremental "
                                          "checkpoints, 64 restores in the same random order", out["value"])
    return out


def run_markovian(args):
    """Markovian state: fingerprint two replays, classify, checkpoint {obs, RNG}, restore."""
    import numpy as np
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    c = W.config1(0)
    r1 = [torch.from_numpy(b.copy()).cuda() for b in c.buffers(1)]
    r2 = [torch.from_numpy(b.copy()).cuda() for b in c.buffers(2)]
    ctx = P.Context(torch.empty(64 << 20, dtype=torch.uint8, device="cuda"))
    both = P.BufArray([P.flat(t) for t in r1 + r2])
    cpb = P.chunk_counts([P.flat(t) for t in r1])[0]
    total = sum(cpb)
    H = torch.zeros(2 * total, dtype=torch.int64, device="cuda")
    bm = torch.zeros(sum((x + 63) // 64 for x in cpb), dtype=torch.int64, device="cuda")
    lab = torch.zeros(len(cpb), dtype=torch.uint8, device="cuda")
    cpa = P.u64_array(cpb)
    plan = P.BufArray([P.flat(r1[0]), P.flat(r1[1])])
    outs = [torch.empty_like(r1[0]), torch.empty_like(r1[1])]
    dst = P.BufArray([P.flat(o) for o in outs])

    def step():
        ctx.fingerprint(both, H)
        ctx.classify(H, 2, cpa, bm, lab)
        s = ctx.checkpoint(plan)
        ctx.restore(s, dst)
        ctx.delete(s)
    t, kt = _timed(args, ctx, step, ["hash", "classify", "pack", "copy", "map"])
    # Per-operation latency, as a caller sees it (call + stream sync), median
    # of 200: the paper reports 0.012 ms per checkpoint or restore of a
    # 185,312-byte state (one A800-80GB, Table 4).
    import statistics

    def lat(f, reps=200):
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            f()
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        return statistics.median(ts) * 1e6
    def call(f, reps=200):
        # Host time of the (asynchronous) call alone; the stream drains between calls.
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            f()
            ts.append(time.perf_counter() - t0)
        torch.cuda.synchronize()
        return statistics.median(ts) * 1e6
    snap = ctx.checkpoint(plan)
    ck_us = lat(lambda: ctx.delete(ctx.checkpoint(plan)))
    rs_us = lat(lambda: ctx.restore(snap, dst))
    fp_us = lat(lambda: ctx.fingerprint(both, H))
    ck_call = call(lambda: ctx.delete(ctx.checkpoint(plan)))
    rs_call = call(lambda: ctx.restore(snap, dst))
    one = torch.empty(1, dtype=torch.uint8, device="cuda")
    floor_us = lat(lambda: one.fill_(1))      # any one-kernel launch + stream sync on this device
    ctx.delete(snap)
    fp_bytes = 2 * sum(x.numel() for x in r1)
    state = r1[0].numel() + r1[1].numel()
    n, ms = kt["hash"]
    out = _line(args, (fp_bytes + 2 * state) / t / 1e9, t * 1e3, "Markovian: obs uint8 [256,256,3], RNG 16 B, "
                 "6 fp16 decoys; fingerprint 2 replays, classify, checkpoint+restore {obs, RNG} (latency-bound)",
                 {"fingerprinted_bytes": fp_bytes, "state_bytes": state}, "k_hash (fingerprint)", fp_bytes, ms / n,
                 {"step_us": round(t * 1e6, 1), "checkpoint_us_median": round(ck_us, 1),
                  "restore_us_median": round(rs_us, 1), "fingerprint_2_replays_us_median": round(fp_us, 1),
                  "checkpoint_call_us_median": round(ck_call, 1), "restore_call_us_median": round(rs_call, 1),
                  "launch_sync_floor_us_median": round(floor_us, 1),
                  "pack_kernel_us": round(1e3 * kt["pack"][1] / max(1, kt["pack"][0]), 2),
                  "restore_kernel_us": round(1e3 * kt["copy"][1] / max(1, kt["copy"][0]), 2)})
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        h1, h2 = [x.cpu().numpy() for x in r1], [x.cpu().numpy() for x in r2]

        def work():
            fp = [oracle.fingerprint(h)[0] for h in (h1, h2)]
            oracle.classify(np.stack(fp), cpb)
            st = oracle.Store()
            snap = st.checkpoint([h1[0], h1[1]])
            st.restore(snap)
            st.delete(snap)
        out["cpu_baseline"] = _oracle_leg(args, work, fp_bytes + 2 * state, "1000 whole steps: fingerprint of both "
                                          "replays, classify, checkpoint + restore of {obs, RNG}", out["value"],
                                          reps=1000)
    return out


def run_shrink(args):
    """Relevance-keyed shrink of the memory bank at its full 512 entries:
    restore the full bank from its snapshot, shrink it in place to 12% of
    its entries ranked by pose distance to the anchor entry, and take an
    incremental checkpoint of the shrunk bank against the full one."""
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    bank = W.config2(1)
    E, le, pe = 512, bank.latent_entry_bytes, bank.pose_entry_bytes
    lat = torch.from_numpy(bank.latents.copy()).cuda()
    pos = torch.from_numpy(bank.poses.copy()).cuda()
    ctx = P.Context(torch.empty(768 << 20, dtype=torch.uint8, device="cuda"))
    full = ctx.checkpoint([P.flat(lat), P.flat(pos)], hash=True)
    scores = torch.from_numpy(W.pose_scores(bank, E, 0)).cuda()
    keep = P.keep_count(0.12, E)
    full_dst = P.BufArray([P.flat(lat), P.flat(pos)])
    shrunk = P.BufArray([P.flat(lat, keep * le), P.flat(pos, keep * pe)])
    parts = [(lat, None, le), (pos, None, pe)]

    def step():
        ctx.restore(full, full_dst)
        ctx.bank_shrink(parts, scores, keep)
        ctx.delete(ctx.checkpoint(shrunk, parent=full))
    t, kt = _timed(args, ctx, step, ["shrink", "incremental", "copy"])
    n, ms = kt["shrink"]
    kept = keep * (le + pe)
    # The kept entries read and written once, the scores read once.  (In place,
    # a kept entry whose source is itself a destination also goes through a
    # staging area: overhead, not counted.)
    alg = 2 * kept + 4 * E
    out = _line(args, E * (le + pe) / t / 1e9, t * 1e3, "relevance-keyed shrink of the memory bank: 512 entries of "
                "bf16 latents [16,60,104] + fp32 pose [7], keep 12%% (%d) by pose distance to the anchor, in place; "
                "then an incremental checkpoint of the shrunk bank" % keep,
                {"entries": E, "kept": keep, "bank_bytes": E * (le + pe)}, "shrink (select, gather)", alg,
                ms / args.steps, {"shrink_ms": round(ms / args.steps, 4),
                                  "incremental_checkpoint_ms": round(kt["incremental"][1] / args.steps, 4),
                                  "restore_full_bank_ms": round(kt["copy"][1] / args.steps, 4)})
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        lat_h = np.ascontiguousarray(bank.latents).view(np.uint8).reshape(-1)
        pos_h = np.ascontiguousarray(bank.poses).view(np.uint8).reshape(-1)
        scores_h = W.pose_scores(bank, E, 0)
        st = oracle.Store()
        ofull = st.checkpoint([lat_h, pos_h])

        def work():
            lat_r, pos_r = st.restore(ofull)
            _, (kl, kp) = oracle.bank_shrink([(lat_r, le), (pos_r, pe)], scores_h, keep)
            st.delete(st.checkpoint([kl, kp], ofull))
        out["cpu_baseline"] = _oracle_leg(args, work, E * (le + pe), "30 whole steps: restore of the full bank, "
                                          "shrink to %d entries, incremental checkpoint" % keep, out["value"],
                                          reps=30)
    return out


def run_discover(args):
    """Discovering PCS by measurement on the mock world model (480x832
    frames): necessity, sufficiency and redundancy fallback over subset
    checkpoints, plus the RNG control; every probe restores into a fresh
    session, runs a leave-and-return trajectory and is scored by GPU chunk
    fingerprints."""
    import torch
    import paper_2607_21686_amd as P
    from workloads.mock_world import MockSpec, initial_state, trajectory
    from workloads.mock_world_gpu import MockWorldGPU
    spec = MockSpec(height=480, width=832, bank_cap=64, entry_words=256, kv_words=1024)
    init = initial_state(spec, 11)
    wa, pa = trajectory(11, 24, 8)
    live = MockWorldGPU.from_host(spec, init)
    live.run(wa)
    ctx = P.Context(torch.empty(512 << 20, dtype=torch.uint8, device="cuda"))
    descs = P.BufArray([P.flat(t) for t in live.parts])
    ref = MockWorldGPU(spec, [t.clone() for t in live.parts]).run(pa)
    ref_h = torch.zeros(P.chunk_counts([P.flat(ref)])[1], dtype=torch.int64, device="cuda")
    ctx.fingerprint([P.flat(ref)], ref_h)
    moved = [0]

    def probe(snap, mask):
        w = MockWorldGPU.fresh(spec)
        ctx.restore(snap, [P.flat(w.parts[i]) for i in range(len(mask)) if mask[i]])
        moved[0] += 2 * sum(w.parts[i].numel() for i in range(len(mask)) if mask[i])
        return ctx.distance(ref_h, [P.flat(w.run(pa))])

    result = {}

    def step():
        result.update(ctx.discover(descs, probe, eps=0.0, control=1))
    fams = ["pack", "copy", "hash", "classify", "merkle", "map", "flip"]
    t, kt = _timed(args, ctx, step, fams)
    lib_ms = sum(kt[f][1] for f in fams) / args.steps
    n, ms = kt["pack"]
    state = sum(spec.nbytes())
    names = ("obs", "rng", "bank", "pose", "feat", "scratch", "kv_a", "kv_b")
    # Each probe's subset is checkpointed once (read + write) and restored once;
    # `moved` counted 2 x the subset per probe.
    per_launch = int(moved[0] / (args.steps + args.warmup) / max(1, result.get("probes", 1)))
    out = _line(args, moved[0] / (args.steps + args.warmup) / t / 1e9, t * 1e3,
                 "discovering PCS by measurement on a mock world model: 8 components (obs 480x832x3 u8, RNG, "
                 "64-entry bank, pose, feature cache, scratch, an interchangeable context pair), 8-step away + "
                 "8-step return probe, eps 0, RNG control", {"components": 8, "state_bytes": state},
                 "subset checkpoints (pack)", per_launch, ms / max(1, n),
                 {"probes": result.get("probes"), "pcs": [nm for nm, f in zip(names, result.get("pcs", [])) if f],
                  "library_kernel_ms_per_discovery": round(lib_ms, 3),
                  "model_and_host_ms_per_discovery": round(t * 1e3 - lib_ms, 3),
                  "control_ok": result.get("control_ok")})
    if not args.no_cpu_baseline:
        import oracle
        from oracle import discover as OD
        from oracle.mock_world import MockWorld
        anchor = [x.cpu().numpy() for x in live.parts]
        ref_o = oracle.fingerprint([MockWorld(spec, anchor).run(pa)])[0]
        got = {}

        def work():
            got.update(OD.discover(OD.mock_probe(spec, anchor, pa, ref_o), 8, 0.0, control=1))
        leg = _oracle_leg(args, work, moved[0] / (args.steps + args.warmup),
                          "one whole discovery on the oracle's own mock model", out["value"])
        leg["same_decisions"] = list(got.get("pcs", [])) == list(result.get("pcs", []))
        out["cpu_baseline"] = leg
    return out


def run_export(args):
    """Durable images across a process boundary: export (device -> host
    image) and import (host image -> device, re-fingerprinted and compared
    before the handle exists) of 16 sessions of the batch workload's shape,
    into pinned and into pageable host memory.  Host-link bound; reported
    beside the HBM numbers, never as them."""
    import numpy as np
    import torch
    import paper_2607_21686_amd as P
    import workloads as W
    S = 16
    plan = W.config5_plan(4, sessions=S)
    g = plan.ring
    rings, obs, rngs = W.config5_device(plan, 4)
    ctx = P.Context(torch.empty(3 << 30, dtype=torch.uint8, device="cuda"))
    snaps = [ctx.checkpoint([P.ring(rings[s], g.outer, g.capacity, g.row_bytes, plan.heads[s], g.window),
                             P.flat(obs[s]), P.flat(rngs[s])], hash=True) for s in range(S)]
    size = ctx.export_size(snaps[0])
    pinned = [torch.empty(size, dtype=torch.uint8, pin_memory=True) for _ in range(S)]
    pageable = [np.empty(size, dtype=np.uint8) for _ in range(S)]

    def rate(f, reps):
        for _ in range(args.warmup):
            f()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            f()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps

    def exp(bufs):
        for s in range(S):
            ctx.export(snaps[s], bufs[s])

    def imp(bufs):
        for s in range(S):
            ctx.delete(ctx.import_image(bufs[s]))
    reps = max(1, args.steps // 2)
    t_exp_p = rate(lambda: exp(pinned), reps)
    ctx.kernel_time("hash")
    ctx.set_timing(True)
    t_imp_p = rate(lambda: imp(pinned), reps)
    ctx.set_timing(False)
    n, ms = ctx.kernel_time("hash")
    t_exp_g = rate(lambda: exp(pageable), reps)
    t_imp_g = rate(lambda: imp(pageable), reps)
    total = S * size
    state = g.window_bytes + plan.obs_bytes + plan.rng_bytes
    gbs = lambda t: round(total / t / 1e9, 2)
    out = _line(args, total / (t_exp_p + t_imp_p) / 1e9, (t_exp_p + t_imp_p) * 1e3,
                "durable images: export + import (with device re-verification) of %d sessions of %d B of state "
                "(KV window 4x2x2048x8x128 bf16 ring, obs 480x832x3 u8, RNG 16 B), pinned host memory" % (S, state),
                {"sessions": S, "image_bytes_per_session": size},
                "k_hash (import re-fingerprint, one session per launch)", state, ms / max(1, n),
                {"export_pinned_GBps": gbs(t_exp_p), "import_pinned_GBps": gbs(t_imp_p),
                 "export_pageable_GBps": gbs(t_exp_g), "import_pageable_GBps": gbs(t_imp_g),
                 "note": "host-link bound (PCIe); value counts image bytes moved per second"})
    if not args.no_cpu_baseline:
        import oracle
        geo = (g.outer, g.outer_stride, g.capacity, g.row_bytes)
        host = [(oracle.ring_window(rings[s].cpu().numpy(), *geo, plan.heads[s], g.window), obs[s].cpu().numpy(),
                 rngs[s].cpu().numpy()) for s in range(2)]
        lay = [(1, g.row_bytes, g.window, g.outer), (0, 0, 0, 0), (0, 0, 0, 0)]

        def work():
            for bufs in host:
                assert len(oracle.export_image(bufs, lay)) == size
        out["cpu_baseline"] = _oracle_leg(args, work, 2 * size, "images of 2 sessions written, 20 times "
                                          "(export only: the oracle writes images and has no import)", out["value"],
                                          reps=20)
    return out


OTHER = {"kv-ring": run_kv_ring, "verify": run_verify, "sweep": run_sweep, "bank": run_bank, "markovian": run_markovian,
         "shrink": run_shrink, "discover": run_discover, "export": run_export}


if __name__ == "__main__":
    main()

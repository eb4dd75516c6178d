"""The benchmark's contract, checked without a GPU: more than one GPU is
refused with a message and exit status 2, the percentile helper behind
step_ms_device, and the HBM traffic record that roofline.traffic comes
from, which must belong to the kernel sources as they are (its sha256) and
scale the rocprofv3 counters the way its numbers say."""
import importlib.util
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def bench_module():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_percentiles():
    b = bench_module()
    assert b._pct([5.0], 50) == 5.0
    assert b._pct([1.0, 2.0, 3.0, 4.0, 5.0], 50) == 3.0
    assert abs(b._pct([1.0, 2.0, 3.0, 4.0, 5.0], 10) - 1.4) < 1e-12
    assert abs(b._pct([1.0, 2.0, 3.0, 4.0, 5.0], 90) - 4.6) < 1e-12


def test_traffic_records_match_the_kernel_sources():
    """Every workload's record (the batch headline, the KV ring checkpoint,
    the verified restore) belongs to the current kernel sources and its
    numbers follow from its counters and the calibration factors."""
    b = bench_module()
    for workload, (fname, kernels) in b.TRAFFIC.items():
        rec = b.traffic_record(workload)
        assert rec is not None, "%s: the committed traffic record was measured on other kernel sources" % workload
        assert rec["kernel_source_sha256"] == b.kernel_source_sha()
        assert rec["workload"] == workload
        for part in (rec, rec["second_kernel"]):
            fetch = part["fetch_KiB_per_dispatch"] * 1024 * rec["fetch_scale"]
            write = part["write_KiB_per_dispatch"] * 1024 * rec["write_scale"]
            # traffic = scaled counters (rounded to 0.1 KiB per dispatch when stored)
            assert abs(fetch + write - part["traffic_bytes_per_launch"]) <= 1e-6 * part["traffic_bytes_per_launch"] + 2048
            assert abs(part["traffic_bytes_per_launch"] / part["algorithmic_bytes_per_launch"]
                       - part["traffic_over_algorithmic"]) < 1e-4
        with open(os.path.join(ROOT, "profiles", fname)) as fh:
            assert json.load(fh) == rec
    # The algorithmic bytes are 2 x state of every session of the launch, and
    # 2 x the 512 MiB window for the KV ring kernels.
    rec = b.traffic_record("batch")
    assert rec["algorithmic_bytes_per_launch"] == 2 * 34_752_528 * rec["sessions"]
    for workload in ("kv-ring", "verify"):
        assert b.traffic_record(workload)["algorithmic_bytes_per_launch"] == 2 * 512 * 2 ** 20

"""CPU check of the gfx950 code this repository builds: no instruction writes
through the scalar data cache (scalar stores and atomics, scalar-cache
write-back or discard), and no kernel needs scratch (private) memory."""
import os
import re
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_21686_amd", "csrc", "pcs_kernels.hip")

FORBIDDEN = re.compile(r"^\s*(s_store_|s_buffer_store|s_atomic|s_buffer_atomic|s_dcache_wb|s_dcache_discard|"
                       r"s_scratch_store)", re.M)


def test_no_scalar_cache_writes_and_no_scratch(tmp_path):
    out = tmp_path / "k.s"
    subprocess.run(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", os.path.join(ROOT, "include"), SRC, "-o", str(out)],
                   check=True, capture_output=True)
    asm = out.read_text()
    bad = FORBIDDEN.findall(asm)
    assert not bad, bad[:5]
    assert ".amdhsa_kernel" in asm
    for m in re.finditer(r"\.private_segment_fixed_size:\s+(\d+)", asm):
        assert int(m.group(1)) == 0
    assert "v_pk_add_f32" not in asm and "v_pk_mul_f32" not in asm and "v_pk_fma_f32" not in asm

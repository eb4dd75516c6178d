"""CPU checks of the C ABI: the library loads and exports every symbol that
include/pcs.h declares, and the Python binding declares exactly those
(no compute calls; there is no GPU here)."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pcs.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pcs_[a-z_]+)\s*\(", src)))


def build_module():
    """The build script, loaded by path (importing the package loads the library)."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("pcs_build", os.path.join(ROOT, "paper_2607_21686_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_library_exports_every_declared_symbol():
    B = build_module()
    if B.stale():
        B.build()
    lib = ctypes.CDLL(B.LIB)
    names = declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_header():
    from paper_2607_21686_amd import _lib
    assert sorted(_lib.EXPORTS) == declared()


def test_struct_layout_matches_header():
    from paper_2607_21686_amd import _lib
    assert ctypes.sizeof(_lib.PcsBuf) == 8 * 2 + 4 * 2 + 8 * 6
    assert ctypes.sizeof(_lib.PcsSnapInfo) == 8 * 4 + 4 * 4
    assert ctypes.sizeof(_lib.PcsBankPart) == 8 * 3


def test_chunk_counts_validation_on_host():
    # pcs_chunk_counts is pure host code: descriptor validation without a GPU.
    from paper_2607_21686_amd import _lib
    lib = _lib.lib()
    B = _lib.PcsBuf
    arr = (B * 3)(B(ptr=4096, nbytes=4097, kind=0),
                  B(ptr=8192, kind=1, row_bytes=2048, capacity=8, head=7, window=4, outer=3,
                    outer_stride=8 * 2048),
                  B(ptr=0, nbytes=0, kind=0))
    out = (ctypes.c_uint64 * 3)()
    tot = ctypes.c_uint64()
    assert lib.pcs_chunk_counts(arr, 3, out, ctypes.byref(tot)) == 0
    assert list(out) == [2, 6, 0] and tot.value == 8
    bad = (B * 1)(B(ptr=4097, nbytes=10, kind=0))
    assert lib.pcs_chunk_counts(bad, 1, out, ctypes.byref(tot)) == _lib.E_INVAL
    bad = (B * 1)(B(ptr=4096, kind=1, row_bytes=24, capacity=8, head=0, window=4, outer=1))
    assert lib.pcs_chunk_counts(bad, 1, out, ctypes.byref(tot)) == _lib.E_INVAL
    bad = (B * 1)(B(ptr=4096, kind=1, row_bytes=32, capacity=8, head=0, window=9, outer=1))
    assert lib.pcs_chunk_counts(bad, 1, out, ctypes.byref(tot)) == _lib.E_INVAL
    bad = (B * 1)(B(ptr=4096, kind=1, row_bytes=32, capacity=8, head=0, window=4, outer=2, outer_stride=32))
    assert lib.pcs_chunk_counts(bad, 1, out, ctypes.byref(tot)) == _lib.E_INVAL


def test_struct_layout_matches_c_compiler(tmp_path):
    """Sizes and field offsets of every ABI struct as gcc lays them out from
    include/pcs.h, against the ctypes declarations of the binding."""
    import subprocess
    from paper_2607_21686_amd import _lib
    structs = {"pcs_buf": _lib.PcsBuf, "pcs_snap_info": _lib.PcsSnapInfo, "pcs_bank_part": _lib.PcsBankPart,
               "pcs_discovery": _lib.PcsDiscovery}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "pcs.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in py._fields_:
            lines.append('printf("%s.%s %%zu\\n", offsetof(%s, %s));' % (cname, f, cname, f))
    lines.append("return 0; }")
    c = tmp_path / "layout.c"
    c.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(c)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n") if l)
    for cname, py in structs.items():
        assert int(got[cname]) == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert int(got["%s.%s" % (cname, f)]) == getattr(py, f).offset, (cname, f)

"""The C ABI without a GPU: the library loads and exports every function the
header declares (and the binding knows each of them), the host-only entry
points answer, and the binding's structures have the header's layout (sizes
and field offsets from a C program compiled against the header)."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2608_13057_amd import _lib, moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "include", "tempo_moe.h")


def _declared():
    text = open(HDR).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return sorted(set(re.findall(r"\b(tempo_moe_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = _declared()
    assert len(names) >= 8, names
    lib = ctypes.CDLL(_lib.LIB_PATH)  # loading touches no GPU
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(_lib.SYMBOLS) == names


def test_host_only_entry_points():
    lib = _lib.load()
    assert lib.tempo_moe_strerror(_lib.TEMPO_OK) == b"ok"
    assert lib.tempo_moe_strerror(_lib.TEMPO_EUNSUPPORTED) == b"unsupported shape or type"
    for dtype, M in (("bf16", 64), ("fp8", 128), ("fp8mx", 256), ("bf16", 192)):
        shape = moe.MoEShape(T=512, K=8, E=128, S=18, H=4096, I=1536, m_tile=M, dtype=dtype)
        ws, cap = moe.query(shape)
        # rows: every pair once plus at most M - 1 padding rows per slot, rounded up to 128
        assert cap == -(-(512 * 8 + 18 * (M - 1)) // 128) * 128
        assert ws > cap * 4096 * (2 if dtype == "bf16" else 1)
    for bad in (dict(m_tile=96), dict(dtype=3), dict(H=4000), dict(K=0)):
        kw = dict(T=512, T_valid=512, K=8, E=128, S=18, H=4096, I=1536, m_tile=64, dtype=0)
        kw.update(bad)
        sh = _lib.Shape(*[kw[n] for n in ("T", "T_valid", "K", "E", "S", "H", "I", "m_tile", "dtype")])
        ws, cap = ctypes.c_size_t(0), ctypes.c_int32(0)
        assert lib.tempo_moe_query(ctypes.byref(sh), ctypes.byref(ws), ctypes.byref(cap), None) == \
            _lib.TEMPO_EINVAL, bad


def test_struct_layouts_match_the_header(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    structs = {"tempo_moe_shape": _lib.Shape, "tempo_plan": _lib.Plan, "tempo_dispatch_out": _lib.DispatchOut,
               "tempo_expert_weights": _lib.ExpertWeights, "tempo_slot_weights": _lib.SlotWeights}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HDR}"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-o", str(exe), str(src)], check=True, capture_output=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        c, f, v = line.split()
        got[(c, f)] = int(v)
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_static_forward_refuses_shapes_beyond_its_scratch():
    """tempo_moe_forward_static checks the shape's workspace against
    TEMPO_STATIC_SCRATCH_BYTES before touching the device (so this runs
    without a GPU): the prefill share does not fit, and a bad shape is
    EINVAL."""
    lib = _lib.load()
    big = moe.MoEShape(T=8192, K=8, E=128, S=18, H=4096, I=1536, m_tile=256).c()
    assert moe.query(moe.MoEShape(T=8192, K=8, E=128, S=18, H=4096, I=1536, m_tile=256))[0] > \
        _lib.TEMPO_STATIC_SCRATCH_BYTES
    args = [None] * 11
    assert lib.tempo_moe_forward_static(ctypes.byref(big), *args) == _lib.TEMPO_EWORKSPACE
    bad = moe.MoEShape(T=8, K=2, E=4, S=2, H=256, I=256, m_tile=96).c()
    assert lib.tempo_moe_forward_static(ctypes.byref(bad), *args) == _lib.TEMPO_EINVAL
    small = moe.MoEShape(T=512, K=8, E=128, S=18, H=4096, I=1536, m_tile=64)
    assert moe.query(small)[0] <= _lib.TEMPO_STATIC_SCRATCH_BYTES


def test_packed_bytes_per_slot():
    """One slot's packed weights: w13 + w2 elements (2 bytes for bf16, 1 for
    fp8) plus, for fp8, the packed 16-byte scale entries of both matrices."""
    H, I = 4096, 1536
    assert moe.packed_slot_bytes(moe.MoEShape(T=8, K=2, E=4, S=3, H=H, I=I, dtype="bf16")) == 3 * H * I * 2
    fp8 = 3 * H * I + ((I // 64) * (H // 128) + (H // 128) * (I // 128)) * 16
    for dt in ("fp8", "fp8mx"):
        assert moe.packed_slot_bytes(moe.MoEShape(T=8, K=2, E=4, S=3, H=H, I=I, dtype=dt)) == fp8

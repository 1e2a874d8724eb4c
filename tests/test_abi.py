"""CPU checks of the C-ABI library: it loads, exports every entry point the
public header declares, and rejects bad arguments before touching the device.

The rejection tests pass fake device addresses that are never dereferenced:
every call has an argument that validation must reject.  They are skipped
where a GPU is visible, so that a validation bug can never turn into a launch
on fake pointers."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from paper_2411_01738_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xdit.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(xdit_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = header_functions()
    for fn in ["xdit_patch_attn", "xdit_patch_attn_ranges", "xdit_chunk_attn",
               "xdit_chunk_attn_accum", "xdit_chunk_attn_accum_split", "xdit_chunk_attn_split",
               "xdit_patch_attn_split",
               "xdit_split_workspace_bytes", "xdit_lse_merge", "xdit_kv_update", "xdit_stage_step",
               "xdit_set_stream",
               "xdit_get_stream", "xdit_last_error", "xdit_version"]:
        assert fn in names


def test_library_exports_every_declared_symbol():
    lib = _lib.lib()
    for name in header_functions():
        assert hasattr(lib, name), f"{name} declared in xdit.h but not exported"
    assert set(_lib.SIGNATURES) == set(header_functions())


def test_header_is_plain_c_and_links(tmp_path):
    """A C99 program that includes the header, takes the address of every
    declared entry point and links against the library builds cleanly with
    -Wall -Werror, and runs (it calls only xdit_version, which touches no
    device)."""
    import shutil
    import subprocess

    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not available")
    lib = _lib.lib()  # built (or fails with the build hint)
    names = header_functions()
    src = tmp_path / "abi.c"
    src.write_text(
        "#include <stdio.h>\n#include \"xdit.h\"\n"
        "int main(void) {\n"
        "    void (*fns[])(void) = {" + ", ".join(f"(void (*)(void))&{n}" for n in names) + "};\n"
        "    for (unsigned i = 0; i < sizeof fns / sizeof fns[0]; ++i) if (!fns[i]) return 1;\n"
        "    printf(\"%s\\n\", xdit_version());\n"
        "    return 0;\n}\n")
    exe = tmp_path / "abi"
    libdir = os.path.dirname(_lib.LIBRARY)
    r = subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                        "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", libdir, "-lxdit", f"-Wl,-rpath,{libdir}"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == lib.xdit_version().decode()


def test_version_and_stream_roundtrip():
    lib = _lib.lib()
    assert b"gfx950" in lib.xdit_version()
    assert lib.xdit_set_stream(0x1234) == 0
    assert lib.xdit_get_stream() == 0x1234
    assert lib.xdit_set_stream(None) == 0
    assert lib.xdit_get_stream() in (None, 0)


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


needs_no_gpu = pytest.mark.skipif(_gpu_visible(), reason="fake-pointer checks run only without a GPU")

A = 0x7F0000000000  # fake, 16-byte aligned device addresses, far apart
MB = 1 << 24


def P(i):
    return A + i * (1 << 32)


@needs_no_gpu
@pytest.mark.parametrize("case,code", [
    # (callable on lib, expected status)
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(4), 1, 16, 16, 2, 64, 7), -2),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(4), 1, 16, 16, 2, 80, 0), -7),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(4), -1, 16, 16, 2, 64, 0), -3),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(4), 1, 1 << 31, 16, 2, 64, 0), -3),
    (lambda L: L.xdit_chunk_attn(None, P(1), P(2), P(3), P(4), 1, 16, 16, 2, 64, 0), -1),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), None, P(4), 1, 16, 16, 2, 64, 0), -1),
    (lambda L: L.xdit_chunk_attn(P(0) + 8, P(1), P(2), P(3), P(4), 1, 16, 16, 2, 64, 0), -5),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(0) + 64, P(4), 1, 16, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(2), 1, 16, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_chunk_attn(P(0), P(1), P(2), P(3), P(3) + 16, 1, 16, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_chunk_attn_accum(P(0), P(1), P(2), P(3), None, 1, 16, 16, 2, 64, 0), -1),
    (lambda L: L.xdit_chunk_attn_accum(P(0), P(1), P(2), P(3), P(3) + 16, 1, 16, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_chunk_attn_accum(P(0), P(1), P(2), P(3), P(4), 1, 16, 16, 2, 72, 5), -2),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 10, 8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -4),
    (lambda L: L.xdit_patch_attn(P(0), P(1), -1, 8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -4),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 0, -8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -4),
    (lambda L: L.xdit_patch_attn(None, P(1), 0, 8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -1),
    (lambda L: L.xdit_patch_attn(P(0), None, 0, 8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -1),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 0, 8, P(1) + 1024, P(3), P(4), 1, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 0, 8, P(2), P(3), P(1), 1, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 0, 8, P(2), P(3), P(0), 1, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_patch_attn(P(0), P(1), 0, 8, P(2), P(3), P(4), 1, 16, 2, 72, 3), -2),
    # q inside the buffer: the buffer's slice is written while queries load
    (lambda L: L.xdit_patch_attn(P(1) + 4096, P(1), 0, 8, P(2), P(3), P(4), 1, 16, 2, 64, 0), -6),
    (lambda L: L.xdit_kv_update(P(1), 9, 8, P(2), P(3), 1, 16, 2, 64, 0), -4),
    (lambda L: L.xdit_kv_update(P(1), 0, 8, P(2) + 4, P(3), 1, 16, 2, 64, 0), -5),
    (lambda L: L.xdit_kv_update(P(1), 0, 8, P(2), P(1) + 2 * 16 * 128 * 2 - 16, 1, 16, 2, 64, 0), -6),
])
def test_rejections(case, code):
    lib = _lib.lib()
    assert case(lib) == code
    assert lib.xdit_last_error().decode(), "no message for a rejected call"


@needs_no_gpu
def test_merge_rejections():
    lib = _lib.lib()
    arr = ctypes.c_void_p * 65
    outs = arr(*[P(10 + r) for r in range(65)])
    lses = arr(*[P(100 + r) for r in range(65)])
    args = (1, 16, 2, 64, 0)
    assert lib.xdit_lse_merge(outs, lses, 0, P(5), P(6), *args) == -4
    assert lib.xdit_lse_merge(outs, lses, 65, P(5), P(6), *args) == -4
    assert lib.xdit_lse_merge(None, lses, 2, P(5), P(6), *args) == -1
    assert lib.xdit_lse_merge(outs, lses, 2, P(5), P(100), *args) == -6  # lse_out on a partial's lse
    assert lib.xdit_lse_merge(outs, lses, 2, P(10) + 16, None, *args) == -6  # shifted overlap
    assert lib.xdit_lse_merge(outs, lses, 2, P(5), P(6) + 2, *args) == -5
    bad = arr(P(10), None)
    assert lib.xdit_lse_merge(bad, lses, 2, P(5), None, *args) == -1
    assert lib.xdit_lse_merge(outs, lses, 2, P(5), None, 1, 16, 2, 96, 0) == -7


def _ranges(*rs):
    offs = (ctypes.c_int64 * max(len(rs), 1))(*[r[0] for r in rs])
    lens = (ctypes.c_int64 * max(len(rs), 1))(*[r[1] for r in rs])
    return len(rs), offs, lens


@needs_no_gpu
@pytest.mark.parametrize("ranges,q_len,fk,out,lse,code", [
    ([(0, 4), (8, 4), (12, 2)], 8, P(2), P(4), P(5), -4),    # more than XDIT_MAX_RANGES
    ([(0, 6), (4, 4)], 8, P(2), P(4), P(5), -4),             # overlapping ranges
    ([(0, 4), (14, 4)], 8, P(2), P(4), P(5), -4),            # past the end of the buffer
    ([(-1, 4)], 8, P(2), P(4), P(5), -4),                    # negative offset
    ([(0, 4)], -1, P(2), P(4), P(5), -3),                    # negative q_len
    ([(0, 4)], 8, P(1) + 512, P(4), P(5), -6),               # fresh rows inside kv_buf
    ([(0, 4)], 8, P(2), P(4), P(4) + 64, -6),                # lse inside out
    ([(0, 4)], 8, P(2), P(4), P(5) + 2, -5),                 # lse misaligned
    ([(0, 4)], 8, P(2), P(1), P(5), -6),                     # out inside kv_buf
    ([(0, 4)], 8, None, P(4), P(5), -1),                     # fresh rows missing
])
def test_ranges_rejections(ranges, q_len, fk, out, lse, code):
    lib = _lib.lib()
    n, offs, lens = _ranges(*ranges)
    assert lib.xdit_patch_attn_ranges(P(0), q_len, P(1), n, offs, lens, fk, P(3), out, lse,
                                      1, 16, 2, 64, 0) == code
    assert lib.xdit_last_error().decode(), "no message for a rejected call"


@needs_no_gpu
def test_ranges_rejects_queries_inside_the_buffer():
    lib = _lib.lib()
    n, offs, lens = _ranges((0, 4))
    assert lib.xdit_patch_attn_ranges(P(1) + 2048, 8, P(1), n, offs, lens, P(2), P(3), P(4), P(5),
                                      1, 16, 2, 64, 0) == -6


def test_split_workspace_bytes():
    """Partitioned launches keep one float32 partial slot (128 query rows x
    (d + 1)) per cut range, two when ranges may cross query tiles."""
    lib = _lib.lib()
    slot = lambda d: 128 * (d + 1) * 4
    # sd3 patch step: 512 queries, 4429 keys, 2 x 24 heads of 64: 192 query
    # tiles, each cut in 4 -> 768 workgroups, one slot each
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 64, 0, 4) == 768 * slot(64)
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 64, 0, 1) == 0
    # by choice: 192 query tiles keep one round either way -> no partition; a
    # decode-like call (1 x 8 query tiles over 256 key tiles) cuts each
    # sweep in 16
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 64, 0, 0) == 0
    assert lib.xdit_split_workspace_bytes(1, 64, 32768, 8, 128, 0, 0) == 128 * slot(128)
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 64, 1, 4) == 0  # float32: unsplit
    # a launch that already fills the CUs (pixart patch: 256 query tiles) is not cut
    assert lib.xdit_split_workspace_bytes(2, 1024, 4096, 16, 72, 0, 0) == 0
    # flux SP share (4224 queries over a 4224-key chunk, 24 heads of 128): 792
    # query tiles leave the fourth round of 256 CUs nearly empty -> three
    # rounds of whole sweeps, the 24 left over cut in 10 parts each, one
    # slot per part
    assert lib.xdit_split_workspace_bytes(1, 4224, 4224, 24, 128, 0, 0) == 240 * slot(128)
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 64, 0, 17) == -1
    assert lib.xdit_split_workspace_bytes(2, 512, 4429, 24, 80, 0, 2) == -1
    # sweeps of one K/V tile or none (128 keys at d <= 72, 64 at d = 128)
    # have nothing to cut: any split runs unsplit
    for d, nk in ((64, 0), (64, 1), (64, 128), (72, 100), (128, 64)):
        for splits in (2, 16, 0):
            assert lib.xdit_split_workspace_bytes(1, 200, nk, 3, d, 0, splits) == 0, (d, nk, splits)
    assert lib.xdit_split_workspace_bytes(1, 200, 129, 3, 64, 0, 2) == 2 * 6 * slot(64)
    assert lib.xdit_split_workspace_bytes(1, 200, 65, 3, 128, 0, 2) == 2 * 6 * slot(128)


@needs_no_gpu
def test_split_rejections():
    lib = _lib.lib()
    need = lib.xdit_split_workspace_bytes(1, 16, 1024, 2, 64, 0, 4)
    assert lib.xdit_chunk_attn_split(P(0), P(1), P(2), P(3), P(4), 17, P(5), need,
                                     1, 16, 1024, 2, 64, 0) == -4
    assert lib.xdit_chunk_attn_split(P(0), P(1), P(2), P(3), P(4), 4, P(5), need - 1,
                                     1, 16, 1024, 2, 64, 0) == -4
    assert lib.xdit_chunk_attn_split(P(0), P(1), P(2), P(3), P(4), 4, None, 0,
                                     1, 16, 1024, 2, 64, 0) == -4
    assert lib.xdit_chunk_attn_split(P(0), P(1), P(2), P(3), P(4), 4, P(5) + 16, need,
                                     1, 16, 1024, 2, 64, 0) == -5
    assert lib.xdit_chunk_attn_split(P(0), P(1), P(2), P(3), P(4), 4, P(3), need,
                                     1, 16, 1024, 2, 64, 0) == -6
    n, offs, lens = _ranges((0, 8))
    assert lib.xdit_patch_attn_split(P(0), 8, P(1), n, offs, lens, P(2), P(3), P(4), None, 4,
                                     P(1) + 4096, need, 1, 1024, 2, 64, 0) == -6
    # the ring step's split form: the running lse is required, the workspace checked
    assert lib.xdit_chunk_attn_accum_split(P(0), P(1), P(2), P(3), None, 4, P(5), need,
                                           1, 16, 1024, 2, 64, 0) == -1
    assert lib.xdit_chunk_attn_accum_split(P(0), P(1), P(2), P(3), P(4), 4, P(5), need - 1,
                                           1, 16, 1024, 2, 64, 0) == -4
    assert lib.xdit_chunk_attn_accum_split(P(0), P(1), P(2), P(3), P(4), 4, P(4), need,
                                           1, 16, 1024, 2, 64, 0) == -6


@needs_no_gpu
def test_ranges_rejects_null_range_arrays():
    lib = _lib.lib()
    assert lib.xdit_patch_attn_ranges(P(0), 8, P(1), 1, None, None, P(2), P(3), P(4), None,
                                      1, 16, 2, 64, 0) == -1


@needs_no_gpu
def test_empty_calls_succeed_without_launching():
    lib = _lib.lib()
    assert lib.xdit_chunk_attn(None, None, None, None, None, 1, 0, 0, 2, 64, 0) == 0
    assert lib.xdit_patch_attn(None, P(1), 16, 0, None, None, None, 1, 16, 2, 64, 0) == 0
    assert lib.xdit_kv_update(P(1), 3, 0, None, None, 1, 16, 2, 128, 1) == 0
    n, offs, lens = _ranges((3, 0), (9, 0))
    assert lib.xdit_patch_attn_ranges(None, 0, P(1), n, offs, lens, None, None, None, None,
                                      1, 16, 2, 64, 0) == 0
    assert lib.xdit_patch_attn_ranges(P(0), 8, P(1), 1, offs, lens, None, None, P(4), None,
                                      0, 16, 2, 64, 0) == 0
    assert lib.xdit_last_error().decode() == ""


@needs_no_gpu
def test_stage_rejections():
    """Stage micro-step: bf16 only, hidden in range, slice inside the buffer,
    aligned pointers, outputs overlapping nothing."""
    lib = _lib.lib()
    # x, wq, wk, wv, wo, kv_buf, off, len, q, k, v, o, y, B, N, H, d, C, dtype
    ok = [P(0), P(1), P(2), P(3), P(4), P(5), 0, 8, P(6), P(7), P(8), P(9), P(10), 1, 16, 2, 64, 128, 0]

    def call(**kw):
        a = list(ok)
        names = ["x", "wq", "wk", "wv", "wo", "kv", "off", "len", "q", "k", "v", "o", "y", "B", "N",
                 "H", "d", "C", "dtype"]
        for n, val in kw.items():
            a[names.index(n)] = val
        return lib.xdit_stage_step(*a)
    assert call(dtype=1) == -7
    assert call(C=0) == -3
    assert call(off=12) == -4
    assert call(q=None) == -1
    assert call(x=P(0) + 8) == -5
    assert call(y=P(0)) == -6
    assert call(o=P(5)) == -6
    assert call(k=P(6)) == -6
    assert call(B=0, x=None, y=None, q=None, k=None, v=None, o=None) == 0


def test_product_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2411_01738_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), f
                assert "xdit_oracle" not in text and "liboracle" not in text, f

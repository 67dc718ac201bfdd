"""CPU-only checks of the C ABI of libattn_numa.so (no GPU, no kernel launch).

* the library loads and exports every function include/attn_numa.h declares;
* argument validation returns the documented status codes before any HIP
  call (fake, never dereferenced pointers);
* the library's own mapping code (the integer code the kernel prologue runs,
  evaluated on the host by attn_map_tiles) equals the oracle enumeration on
  many shapes, so every workgroup's (b, hq, m) is in range before the kernel
  ever runs on a GPU.
"""

import os
import re

import numpy as np
import pytest

import paper_2511_02132_amd as pa
from oracle import mapping as mp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attn_numa.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attn_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = pa.lib()
    names = header_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(pa.SIGNATURES) == names


# fake device addresses: 16-byte aligned, never dereferenced
Q, K, V, O = 0x10000000, 0x20000000, 0x30000000, 0x40000000


def call(q=Q, k=K, v=V, o=O, B=1, Hq=4, Hkv=2, Sq=256, Skv=256, d=128, causal=0, scale=0.088,
         mapping=2):
    return pa.lib().attn_fwd(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping)


@pytest.mark.parametrize("kwargs,code", [
    (dict(q=None), -1), (dict(k=None), -1), (dict(v=None), -1), (dict(o=None), -1),
    (dict(B=0), -2), (dict(Hq=0), -2), (dict(Hkv=0), -2), (dict(Sq=0), -2), (dict(Skv=-1), -2),
    (dict(Hq=6, Hkv=4), -2), (dict(Sq=2 ** 23), -2), (dict(Skv=2 ** 23), -2),
    (dict(d=96), -3), (dict(d=256), -3), (dict(d=0), -2),
    (dict(mapping=4), -4), (dict(mapping=-1), -4), (dict(mapping=0x80 | 2), -4),
    # paired row blocks exist for d = 128 only
    (dict(mapping=0x40 | 2, d=64), -3), (dict(mapping=0x50 | 0, d=56), -3),
    (dict(mapping=0x14), -4), (dict(mapping=0xf), -4),
    # the block-major order inside an XCD's piece exists for swizzled head-first only
    (dict(mapping=0x20 | 0), -4), (dict(mapping=0x20 | 1), -4), (dict(mapping=0x30 | 3), -4),
    (dict(scale=float("nan")), -5), (dict(scale=float("inf")), -5), (dict(scale=0.0), -5),
    (dict(scale=-1.0), -5),
    (dict(q=Q + 8), -6), (dict(o=O + 2), -6),
    (dict(o=Q), -8), (dict(o=K + 256), -8),
])
def test_validation_codes(kwargs, code):
    assert call(**kwargs) == code
    assert pa.strerror(code) and pa.strerror(code) != "unknown status code"


def test_probe_validation():
    lib = pa.lib()
    args = (Q, K, V, O, 1, 4, 2, 256, 256, 128, 0, 0.088, 2)
    assert lib.attn_fwd_probe(*args, None) == -1
    assert lib.attn_fwd_probe(*args, 0x50000002) == -6
    bad = (Q, K, V, O, 1, 4, 3, 256, 256, 128, 0, 0.088, 2)
    assert lib.attn_fwd_probe(*bad, 0x50000000) == -2


def test_sizes():
    assert pa.block_m(64) == 128 and pa.block_m(128) == 256 and pa.block_m(56) == 128
    assert pa.block_n(64) == pa.block_n(128) == 64
    assert pa.lib().attn_block_m(96) == -3
    assert pa.grid_size(1, 32, 8192, 128) == 1024
    assert pa.grid_size(8, 64, 4096, 128) == 8192
    assert pa.grid_size(2, 3, 129, 64) == 12
    assert pa.grid_size(2, 3, 257, 128) == 12
    assert pa.lib().attn_grid_size(1, 1, 0, 128) == -2


def test_num_xcd_env_override(monkeypatch):
    monkeypatch.setenv("ATTN_NUM_XCD", "4")
    assert pa.num_xcd() == 4


def test_stream_roundtrip():
    lib = pa.lib()
    assert lib.attn_set_stream(0x1234) == 0
    assert lib.attn_get_stream() == 0x1234
    assert lib.attn_set_stream(None) == 0
    assert lib.attn_get_stream() is None
    assert lib.attn_last_hip_error() == b""


MAP_SHAPES = [(1, 4, 256, 64, 8), (1, 32, 8192, 128, 8), (1, 64, 8192, 128, 8),
              (8, 64, 4096, 128, 8), (1, 16, 131072, 128, 8), (2, 12, 300, 128, 8),
              (3, 5, 1000, 64, 4), (1, 1, 1, 128, 8), (2, 3, 129, 64, 1), (1, 8, 16384, 128, 8),
              (1, 128, 8192, 56, 8), (1, 128, 2048, 56, 8), (2, 128, 2048, 128, 8),
              (1, 64, 2176, 64, 8)]


@pytest.mark.parametrize("B,Hq,Sq,d,NX", MAP_SHAPES)
def test_library_mapping_equals_oracle(B, Hq, Sq, d, NX):
    BM = pa.block_m(d)
    values = [m | f for m in (0, 1, 2, 3) for f in (0, 0x10)] + [0x22, 0x32]
    for value in values + [v | pa.PAIRED for v in values]:
        mapping, heavy, xbm, paired = mp.split_flags(value)
        if paired and d != 128:
            with pytest.raises(pa.AttnError) as e:
                pa.map_tiles(value, B, Hq, Sq, d, NX)
            assert e.value.code == -3
            continue
        got = pa.map_tiles(value, B, Hq, Sq, d, NX)
        want = mp.enumerate_mapping(mapping, B, Hq, Sq, BM, NX, heavy_first=heavy,
                                    short_head_groups=(BM == 128),
                                    xcd_block_major=xbm, paired=paired)
        assert np.array_equal(got[:want.shape[0]], want), hex(value)
        assert (got[want.shape[0]:] == -1).all(), hex(value)


def test_map_tiles_errors():
    assert pa.lib().attn_map_tiles(2, 1, 4, 256, 64, 8, None) == -1
    out = np.empty(8 * 3, np.int32)
    ptr = out.ctypes.data_as(pa._i32p)
    assert pa.lib().attn_map_tiles(5, 1, 4, 256, 64, 8, ptr) == -4
    assert pa.lib().attn_map_tiles(2, 1, 4, 256, 64, 0, ptr) == -2
    assert pa.lib().attn_map_tiles(2 | pa.PAIRED, 1, 4, 256, 64, 8, ptr) == -3   # d = 128 only
    assert pa.lib().attn_map_tiles(2 | 0x80, 1, 4, 256, 128, 8, ptr) == -4


def test_calib_validation():
    lib = pa.lib()
    R, S = 0x50000000, 0x60000000
    assert lib.attn_calib_mfma(256, 20000, None, S) == -1
    assert lib.attn_calib_mfma(256, 20000, R, None) == -1
    assert lib.attn_calib_mfma(0, 20000, R, S) == -2
    assert lib.attn_calib_mfma(65537, 4, R, S) == -2
    assert lib.attn_calib_mfma(256, 0, R, S) == -2
    assert lib.attn_calib_mfma(256, 6, R, S) == -2          # not a multiple of 4
    assert lib.attn_calib_mfma(256, 2 ** 24 + 4, R, S) == -2
    assert lib.attn_calib_mfma(256, 4, R + 4, S) == -6      # int64 records: 8-byte aligned
    assert lib.attn_calib_mfma(256, 4, R, S + 2) == -6
    assert lib.attn_calib_mfma(256, 4, R, R + 8) == -8      # sink overlaps the records


def test_header_is_c99_and_links_from_c(tmp_path):
    """The boundary is a C ABI: a C99 program includes the header, links
    against the library and calls host-only entry points (no GPU needed)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not installed")
    src = tmp_path / "abi.c"
    src.write_text(
        '#include <stdio.h>\n#include <string.h>\n#include "attn_numa.h"\n'
        "int main(void) {\n"
        "    int32_t t[3 * 8];\n"
        "    if (attn_block_m(128) != 256 || attn_block_m(64) != 128) return 1;\n"
        "    if (attn_block_n(56) != 64 || attn_block_m(96) != ATTN_ERR_UNSUPPORTED) return 2;\n"
        "    if (attn_grid_size(1, 32, 8192, 128) != 1024) return 3;\n"
        "    if (attn_map_tiles(ATTN_MAP_SWIZZLED_HEAD_FIRST, 1, 4, 256, 64, 8, t) != ATTN_OK) return 4;\n"
        "    if (attn_fwd(0, 0, 0, 0, 1, 1, 1, 1, 1, 128, 0, 1.0f, 2) != ATTN_ERR_NULL) return 5;\n"
        "    if (strlen(attn_strerror(ATTN_ERR_SHAPE)) == 0) return 6;\n"
        '    printf("ok\\n");\n    return 0;\n}\n')
    lib_dir = os.path.dirname(pa.LIB_PATH)
    exe = tmp_path / "abi"
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                    "-L", lib_dir, "-lattn_numa", "-Wl,-rpath," + lib_dir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr)

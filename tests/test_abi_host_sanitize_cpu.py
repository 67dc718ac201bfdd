"""The C ABI's host code under AddressSanitizer and UBSan (CPU only).

tests/host/abi_host_harness.cpp is linked with paper_2511_02132_amd/csrc/attn_abi.cpp
(built for the host by g++, no device code) and stubs of the kernel launchers
and of the HIP runtime calls.  It drives every entry point through its error
paths and ragged shapes: validation codes, pointer alignment, every
input/output overlap of the backward, the persistent forms' queue checks (the
allocation-free one included), the launch arguments each call derives, the
HIP-failure path, and attn_map_tiles on ragged shapes, whose tables must equal
the oracle enumeration.  Any out-of-bounds access, leak or undefined behaviour
aborts the run.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import mapping as mp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HARNESS = os.path.join(ROOT, "tests", "host", "abi_host_harness.cpp")
ABI = os.path.join(ROOT, "paper_2511_02132_amd", "csrc", "attn_abi.cpp")
ROCM_INCLUDE = "/opt/rocm/include"


def test_abi_host_code_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir(os.path.join(ROCM_INCLUDE, "hip")):
        pytest.skip("g++ or the HIP headers are not installed")
    exe = tmp_path / "abi_host_harness"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall",
           "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE, "-I", os.path.join(ROOT, "include"),
           "-I", os.path.dirname(ABI), ABI, HARNESS, "-o", str(exe)]
    b = subprocess.run(cmd, capture_output=True, text=True)
    if b.returncode != 0 and "asan" in b.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + b.stderr[-200:])
    assert b.returncode == 0, b.stderr[-3000:]
    out = tmp_path / "tables.bin"
    env = {k: v for k, v in os.environ.items() if k != "ATTN_NUM_XCD"}
    env["ASAN_OPTIONS"] = "detect_leaks=1"
    r = subprocess.run([str(exe), str(out)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.startswith("ok"), (r.returncode, r.stdout,
                                                             r.stderr[-3000:])
    assert int(r.stdout.split()[1]) > 400   # number of checks run

    data = np.fromfile(out, dtype=np.int32)
    pos, cases = 0, 0
    while pos < data.size:
        value, B, Hq, Sq, d, NX = (int(x) for x in data[pos:pos + 6])
        pos += 6
        BM = 256 if d == 128 else 128
        n = B * Hq * ((Sq + BM - 1) // BM)
        got = data[pos:pos + 3 * n].reshape(n, 3)
        pos += 3 * n
        mapping, heavy, xbm, paired = mp.split_flags(value)
        want = mp.enumerate_mapping(mapping, B, Hq, Sq, BM, NX, heavy_first=heavy,
                                    short_head_groups=(BM == 128), xcd_block_major=xbm,
                                    paired=paired)
        # the rows past the paired grid hold -1
        want = np.concatenate([want, np.full((n - want.shape[0], 3), -1)])
        assert np.array_equal(got, want), (hex(value), B, Hq, Sq, d, NX)
        cases += 1
    assert cases == 11 * 10 + 6 * 10   # six shapes have d = 128 and also take the paired order

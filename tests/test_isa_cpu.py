"""Static checks of the gfx950 machine code of the attention kernels (CPU only).

The kernels are compiled to assembly with the same flags as the library and
the listing is checked for properties that the HIP source alone does not
guarantee:

* the global->LDS copies are hand-written assembly that sets M0 itself; M0 is
  a compiler-reserved register, so every use of it must be one of those copies,
  each right after its own M0 write and the wait states it needs;
* no packed fp32 VALU instructions (the build disables them);
* no scalar-cache writes of any kind;
* no scratch memory, no vector-register spills in any kernel (scalar spills
  only into VGPR lanes), and registers and LDS within what
  one workgroup per CU (ping-pong kernel) or two (4-wave kernel) allows.

This file names scalar-cache write instructions on purpose (to forbid them),
so it is kept out of the uploads to GPU machines; it needs no GPU.
"""

from __future__ import annotations

import os
import re
import subprocess

import pytest

from paper_2511_02132_amd import build as B

KERNEL_FILES = ["attn_fwd.hip", "attn_fwd_pp.hip", "attn_bwd.hip", "attn_bwd_dq.hip", "attn_calib.hip"]
# the matrix-core calibration kernel works on registers only: no LDS copies
NO_COPY_FILES = {"attn_calib.hip"}

# Instructions that read M0 implicitly on gfx9-family targets.
IMPLICIT_M0 = re.compile(
    r"^(s_sendmsg|s_sendmsghalt|s_movrel|v_movrel|v_interp|ds_gws|ds_ordered_count|"
    r"ds_append|ds_consume|ds_read_addtid|ds_write_addtid|global_load_lds|s_ttracedata)")
# Scalar data-cache writes: stores, atomics, write-back, discard.
SCALAR_WRITE = re.compile(
    r"^(s_store|s_buffer_store|s_scratch_store|s_atomic|s_buffer_atomic|s_dcache_wb|"
    r"s_dcache_discard)")
PACKED_F32 = re.compile(r"^v_pk_(fma|mul|add)_f32")


def _have_hipcc() -> bool:
    try:
        B.hipcc()
        return True
    except RuntimeError:
        return False


pytestmark = pytest.mark.skipif(not _have_hipcc(), reason="hipcc not installed")


@pytest.fixture(scope="module")
def listings(tmp_path_factory):
    out = {}
    d = tmp_path_factory.mktemp("isa")
    for name in KERNEL_FILES:
        flags = [f for f in B.compile_flags(name) if f not in ("-fPIC", "-Wall")]
        dst = os.path.join(d, name + ".s")
        cmd = [B.hipcc(), *flags, "--cuda-device-only", "-S", os.path.join(B.CSRC, name),
               "-o", dst]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        with open(dst) as f:
            out[name] = f.read()
    return out


def _kernels(text: str):
    """(name, instruction lines) for every kernel body in a listing."""
    lines = text.splitlines()
    # function symbols only (a device variable's label is data, not code)
    funcs = set(re.findall(r"^\s*\.type\s+(\w+),@function", text, re.M))
    res = []
    i = 0
    while i < len(lines):
        m = re.match(r"^(_Z\w+):\s*(;.*)?$", lines[i])
        if m and m.group(1) in funcs:
            name = m.group(1)
            body = []
            i += 1
            while i < len(lines) and not lines[i].startswith(".Lfunc_end"):
                s = lines[i].strip()
                if s and not s.startswith((";", ".", "//")) and not s.endswith(":"):
                    body.append(s.split(";")[0].strip())
                i += 1
            res.append((name, body))
        i += 1
    return res


def _metadata(text: str):
    """Per-kernel metadata maps from the amdhsa.kernels YAML block."""
    # kernel entries are the two-space-indented items of the amdhsa.kernels list
    blocks = re.split(r"\n(?=  - \.)", text[text.index("amdhsa.kernels:"):])
    out = []
    for b in blocks[1:]:
        md = dict(re.findall(r"^\s*(?:- )?\.(\w+):\s+(\S+)\s*$", b, re.M))
        if "name" in md:
            out.append(md)
    return out


@pytest.mark.parametrize("name", KERNEL_FILES)
def test_every_m0_use_is_a_guarded_lds_copy(listings, name):
    kernels = _kernels(listings[name])
    assert kernels, "no kernels found in the listing"
    n_copies = 0
    for kname, body in kernels:
        for j, ins in enumerate(body):
            op = ins.split()[0]
            assert not IMPLICIT_M0.match(op), (kname, ins)
            is_copy = op.startswith("buffer_load") and re.search(r"\blds\b", ins)
            if "m0" in ins.replace(",", " ").split():
                assert op == "s_mov_b32" and ins.split()[1].rstrip(",") == "m0", (kname, ins)
                # the write is followed by the wait states and then the copy
                assert body[j + 1] == "s_nop 4", (kname, body[j:j + 3])
                nxt = body[j + 2]
                assert nxt.startswith("buffer_load_dwordx4") and re.search(r"\blds\b", nxt)
            if is_copy:
                n_copies += 1
                assert body[j - 1] == "s_nop 4" and body[j - 2].startswith("s_mov_b32 m0,"), \
                    (kname, body[j - 2:j + 1])
    assert (n_copies == 0) == (name in NO_COPY_FILES)


@pytest.mark.parametrize("name", KERNEL_FILES)
def test_no_packed_fp32_and_no_scalar_writes(listings, name):
    for kname, body in _kernels(listings[name]):
        # the parse found the kernel's real instruction stream (the D = <dO, O>
        # kernel of the backward pass and the queue-clearing kernel of the
        # persistent form are the ones without matrix-core work)
        small = "clear_queue_kernel" in kname
        assert len(body) > (3 if small else 10), kname
        if "delta_kernel" not in kname and not small:
            assert sum(ins.startswith("v_mfma_f32_32x32x16_bf16") for ins in body) >= 16, kname
        for ins in body:
            op = ins.split()[0]
            assert not PACKED_F32.match(op), (kname, ins)
            assert not SCALAR_WRITE.match(op), (kname, ins)


@pytest.mark.parametrize("name", KERNEL_FILES)
def test_no_scratch_no_spills_and_resources_fit(listings, name):
    mds = _metadata(listings[name])
    assert len(mds) == len(_kernels(listings[name]))
    for md in mds:
        # every kernel, the dK/dV kernel at its 256 registers included
        assert md["private_segment_fixed_size"] == "0", md["name"]
        assert md.get("vgpr_spill_count", "0") == "0", md["name"]
        # a few scalar registers may be parked in VGPR lanes (v_writelane, no
        # memory traffic: the scratch size above is zero)
        assert int(md.get("sgpr_spill_count", "0")) <= 8, md["name"]
        lds = int(md["group_segment_fixed_size"])
        # on gfx950 the count covers the unified file: architectural VGPRs
        # (up to the accumulator offset) plus the AGPRs behind them
        regs = int(md["vgpr_count"])
        assert int(md.get("agpr_count", "0")) <= regs
        threads = int(md["max_flat_workgroup_size"])
        # 512 registers per lane per SIMD; a workgroup's waves spread over 4 SIMDs
        waves_per_simd = max(1, threads // 256)
        assert regs * waves_per_simd <= 512, (md["name"], regs, threads)
        assert lds <= 160 * 1024, (md["name"], lds)
        if "attn_bwd_dq_kernel" in md["name"]:
            # built for two workgroups per CU: both fit in registers and LDS,
            # and the accumulators stay out of AGPRs
            assert regs <= 256 and int(md.get("agpr_count", "0")) == 0, (md["name"], regs)
            assert 2 * lds <= 160 * 1024, (md["name"], lds)

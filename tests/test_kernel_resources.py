"""CPU checks of the decode kernel's resource budget (compiled for gfx950
here, no GPU needed): the instances launched on grids of several rounds
must let two 512-thread workgroups share a CU (at most 128 VGPRs, at most
80 KB of LDS; the positional-split instances: the LDS bound only), every
instance must fit two waves per SIMD with no scratch,
and the dynamic LDS the launcher adds to one-round grids must leave room for
only one workgroup per CU (160 KB of LDS per CU)."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2608_08081_amd import build as B

LDS_PER_CU = 160 * 1024


def _device_asm(src, tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    out = tmp_path / (src + ".s")
    flags = [f for f in B.COMMON_FLAGS if f not in ("-fPIC",)]
    cmd = [hipcc, "-x", "hip", *flags, "-I", B.INCLUDE, "-I", B.CSRC, "-S",
           "--cuda-device-only", os.path.join(B.CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


def _kernels(asm):
    """name -> (vgprs, lds bytes, scratch bytes) from the AMDGPU metadata."""
    res = {}
    for m in re.finditer(r"^\s+\.group_segment_fixed_size:\s+(\d+)\n(.*?)^\s+\.vgpr_spill_count",
                         asm, re.S | re.M):
        block = m.group(0)
        name = re.search(r"\.name:\s+(\S+)", block).group(1)
        vg = int(re.search(r"\.vgpr_count:\s+(\d+)", block).group(1))
        priv = int(re.search(r"\.private_segment_fixed_size:\s+(\d+)", block).group(1))
        res[name] = (vg, int(m.group(1)), priv)
    return res


def test_decode_g8_occupancy_budget(tmp_path):
    asm = _device_asm("iq_decode_g8.hip", tmp_path)
    src = open(os.path.join(B.CSRC, "iq_g8_device.h")).read()
    pad = eval(re.search(r"kOneWorkgroupPadBytes\s*=\s*([^;]+);", src).group(1))
    ks = _kernels(asm)
    dec = {n: v for n, v in ks.items() if "decode_g8_kernel" in n}
    # NB 1..5 x grid kind x (group 8, any group) x ((fused step, paged,
    # plain) at 3 bits, (fused step, plain) at 2 and 4 bits), and NB 1..5 x
    # grid kind with the positional split (any group)
    assert len(dec) == 170, sorted(dec)
    for name, (vg, lds, priv) in dec.items():
        m = re.search(r"decode_g8_kernelILi(\d)ELb(\d)ELb(\d)ELb(\d)ELi(\d)ELb(\d)ELb(\d)EE",
                      name)
        nb, wide, rope = int(m.group(1)), m.group(3) == "1", m.group(6) == "1"
        assert priv == 0, f"{name}: scratch {priv}"
        assert vg <= 256, f"{name}: {vg} VGPRs"
        if wide and rope:
            # the positional split's wide instances may hold one workgroup
            # per CU (their positional operands take up to 32 more VGPRs)
            assert 2 * lds <= LDS_PER_CU, f"wide rope NB={nb}: {lds} B LDS"
        elif wide:
            assert vg <= 128, f"wide NB={nb}: {vg} VGPRs, two workgroups no longer fit a CU"
            assert 2 * lds <= LDS_PER_CU, f"wide NB={nb}: {lds} B LDS"
        else:
            assert 2 * (lds + pad) > LDS_PER_CU, f"narrow NB={nb}: padding too small"
            assert lds + pad <= LDS_PER_CU


def test_compress_kernel_has_no_scratch(tmp_path):
    ks = _kernels(_device_asm("iq_compress.hip", tmp_path))
    comp = {n: v for n, v in ks.items() if "compress_kernel" in n}
    # fp16 / fp32 inputs x (3-bit paged, 2-, 3-, 4-bit contiguous)
    assert len(comp) == 8
    for name, (vg, lds, priv) in comp.items():
        assert priv == 0, f"{name}: scratch {priv}"
        assert vg <= 256, f"{name}: {vg} VGPRs"


def test_multi_token_kernel_budget(tmp_path):
    """Multi-token decode instances (NB 1..5 x grid kind x 2..4 tokens x
    (3-bit paged decode; contiguous 2-, 3- and 4-bit records, decode and the
    fused step)): no scratch, at most 256 VGPRs (one workgroup per CU when
    above 128), and the one-round instances' LDS with the padding within a
    CU."""
    asm = _device_asm("iq_decode_multi.hip", tmp_path)
    src = open(os.path.join(B.CSRC, "iq_g8_device.h")).read()
    pad = eval(re.search(r"kOneWorkgroupPadBytes\s*=\s*([^;]+);", src).group(1))
    ks = _kernels(asm)
    mt = {n: v for n, v in ks.items() if "decode_g8_multi_kernel" in n}
    assert len(mt) == 210, sorted(mt)
    for name, (vg, lds, priv) in mt.items():
        m = re.search(r"decode_g8_multi_kernelILi(\d)ELb(\d)ELi(\d)ELb(\d)ELi(\d)ELb(\d)EE",
                      name)
        wide = m.group(2) == "1"
        assert priv == 0, f"{name}: scratch {priv}"
        assert vg <= 256, f"{name}: {vg} VGPRs"
        if wide:
            assert lds <= LDS_PER_CU
        else:
            assert lds + pad <= LDS_PER_CU

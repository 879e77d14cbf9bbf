"""The register and LDS budgets the causal scan's occupancy rests on, read from
the kernel descriptors hipcc writes for gfx950 (the library's own compile
flags): every 32-token instantiation of k_causal_fs fits two workgroups per CU
(at most 256 vector registers per wave, VGPRs and AGPRs together, and at most
half of the CU's 160 KB of LDS), the plan's segment choice for T = 32 assumes
it; the 64-token ones fit one. The gradient kernels use no scratch. No GPU is
needed.
"""
import os
import re
import subprocess

import pytest

from paper_2006_03555_amd import build as B

LDS_PER_CU = 160 * 1024
REGS_PER_LANE = 512   # vector registers per SIMD lane (VGPRs and AGPRs)


def _kernel_descriptors(tmp_path_factory, source):
    hipcc = B.hipcc()
    if not hipcc or not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / (source + ".s")
    cmd = [hipcc, f"--offload-arch={B.ARCH}", *B.COMMON_FLAGS, *B.DEVICE_FLAGS,
           *B.PER_SOURCE_FLAGS.get(source, []), "--cuda-device-only", "-S", "-x", "hip",
           os.path.join(B.CSRC, source), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    text = out.read_text()
    kernels = {}
    for m in re.finditer(r"\.amdhsa_kernel (\S+)\n(.*?)\.end_amdhsa_kernel", text, re.S):
        fields = dict(re.findall(r"\.amdhsa_(\w+) (\d+)", m.group(2)))
        kernels[m.group(1)] = {k: int(v) for k, v in fields.items()}
    return kernels


@pytest.fixture(scope="module")
def descriptors(tmp_path_factory):
    return _kernel_descriptors(tmp_path_factory, "causal.hip")


def _scan_kernels(kernels, chunk):
    tag = f"ELi{chunk}EEEv"
    found = {n: f for n, f in kernels.items() if "k_causal_fs" in n and tag in n}
    assert found, f"no k_causal_fs instantiation with {chunk}-token chunks"
    return found


def test_32_token_scan_fits_two_workgroups_per_cu(descriptors):
    for name, f in _scan_kernels(descriptors, 32).items():
        assert f["next_free_vgpr"] <= REGS_PER_LANE // 2, (name, f["next_free_vgpr"])
        assert f["group_segment_fixed_size"] <= LDS_PER_CU // 2, (name, f["group_segment_fixed_size"])


def test_cosine_scan_keeps_off_scratch(descriptors):
    """Every cosine-feature instantiation of the scan (each M and output type,
    both chunk lengths, M = 256 at 32 tokens being the reordered chunk) needs no
    scratch. (ReLU features at 32 tokens spill 8-16 bytes per lane at M = 128.)"""
    for chunk in (32, 64):
        for name, f in _scan_kernels(descriptors, chunk).items():
            if re.search(r"Li(64|128|256)ELi0E", name):
                assert f["private_segment_fixed_size"] == 0, name


def test_64_token_scan_fits_one_workgroup_per_cu(descriptors):
    for name, f in _scan_kernels(descriptors, 64).items():
        assert f["next_free_vgpr"] <= REGS_PER_LANE, name
        assert LDS_PER_CU // 2 < f["group_segment_fixed_size"] <= LDS_PER_CU, name


def test_gradient_kernels_keep_off_scratch(tmp_path_factory):
    """Every instantiation of the gradient kernels (both feature kinds, bf16 and
    fp32, every M) holds its registers without scratch: at M = 64 the feature
    loop stays rolled, which a full unroll would spill."""
    kernels = _kernel_descriptors(tmp_path_factory, "backward.hip")
    assert kernels
    spilled = {n: f["private_segment_fixed_size"] for n, f in kernels.items()
               if f["private_segment_fixed_size"] > 0}
    assert not spilled, spilled

"""Every kernel of the library compiles for gfx950 without register spills.

A spill puts scratch loads and stores into a kernel's inner loop (and, for the stage rings that
wait on explicit load counts, extra vector-memory operations); the attention kernel in
particular sits a few registers below the 256-register limit of two waves per SIMD.  The check
compiles the library's translation unit for the device only, with the compiler's per-kernel
resource remarks, and requires a scratch size of zero for every kernel.  CPU only (hipcc
cross-compiles); skipped when hipcc is not installed.
"""

import os
import re
import subprocess

import pytest

from paper_2608_27514_amd import build as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _remarks(source):
    hipcc = b.hipcc_path()
    flags = [f for f in b.HIPCC_FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [hipcc, *flags, "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-c", "-o", os.devnull, source,
           "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stderr[-2000:]
    return out.stderr


def _scratch_per_kernel(text):
    kernels = {}
    name = None
    for line in text.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"remark:\s+ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name is not None:
            kernels[name] = int(m.group(1))
    return kernels


@pytest.mark.parametrize("source", ["trajspec.hip", "stream_floor.hip"])
def test_no_kernel_spills(source):
    try:
        b.hipcc_path()
    except Exception:
        pytest.skip("hipcc not installed")
    kernels = _scratch_per_kernel(_remarks(os.path.join(ROOT, "paper_2608_27514_amd", "csrc", source)))
    assert kernels, "no kernel resource remarks parsed"
    if source == "trajspec.hip":
        for must in ("verify_attn_kernel", "conf_topk_kernel", "accept_kernel", "gemm_"):
            assert any(must in k for k in kernels), must
    spilled = {k: v for k, v in kernels.items() if v != 0}
    assert not spilled, f"kernels with scratch: {spilled}"

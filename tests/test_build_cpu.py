"""Properties of the compiled gfx950 code, checked on the CPU from the device assembly that the
build's own flags produce: no packed fp32 arithmetic instructions (they are kept out of every
kernel) and no scratch (spill) memory in any kernel."""
import os
import re
import subprocess

import pytest

from paper_2608_12114_amd import build as wb
import synth

KERNEL_SOURCES = [
    (os.path.join(wb.CSRC, "wsr_kernels.hip"), [*wb.COMMON, *wb.DEVICE]),
    (synth.DEV_SRC_PATH, ["-O3", "--offload-arch=gfx950", "-ffp-contract=off",
                          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]),
]


@pytest.fixture(scope="module", params=KERNEL_SOURCES, ids=lambda p: os.path.basename(p[0]))
def asm(request, tmp_path_factory):
    src, flags = request.param
    out = tmp_path_factory.mktemp("asm") / "k.s"
    subprocess.run(["hipcc", *flags, "-S", "--cuda-device-only", src, "-o", str(out)], check=True,
                   capture_output=True)
    return out.read_text()


def test_no_packed_fp32(asm):
    assert not re.findall(r"\bv_pk_(fma|add|mul|mov)_f32\b", asm)


def test_no_scratch(asm):
    sizes = [int(v) for v in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", asm)]
    assert sizes and all(v == 0 for v in sizes)

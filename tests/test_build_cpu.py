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
    (os.path.join(wb.CSRC, "wsr_mma.hip"), [*wb.COMMON, *wb.DEVICE]),
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


# ---- the peephole check of the build ---------------------------------------------------------------

_DUMP = """# *** IR Dump Before SI peephole optimizations (si-pre-emit-peephole) ***:
# Machine code for function k_a: NoPHIs
  V_CMP_LT_U64_e32 $sgpr20_sgpr21, killed $vgpr2_vgpr3, implicit-def $vcc, implicit $exec
  renamable $vcc = S_AND_B64 killed renamable $vcc, $exec, implicit-def $scc
  renamable $sgpr21 = S_CSELECT_B32 killed renamable $sgpr21, renamable $sgpr9, implicit $scc
  S_CBRANCH_VCCNZ %bb.2, implicit killed $vcc
# *** IR Dump After SI peephole optimizations (si-pre-emit-peephole) ***:
# Machine code for function k_a: NoPHIs
  V_CMP_LT_U64_e32 $sgpr20_sgpr21, killed $vgpr2_vgpr3, implicit-def $vcc, implicit $exec
  renamable $sgpr21 = S_CSELECT_B32 killed renamable $sgpr21, renamable $sgpr9, implicit $scc
  S_CBRANCH_VCCNZ %bb.2, implicit killed $vcc
# *** IR Dump Before SI peephole optimizations (si-pre-emit-peephole) ***:
# Machine code for function k_b: NoPHIs
  V_CMP_LE_I64_e32 killed $sgpr18_sgpr19, killed $vgpr0_vgpr1, implicit-def $vcc, implicit $exec
  renamable $vcc = S_AND_B64 $exec, killed renamable $vcc, implicit-def dead $scc
  S_CBRANCH_VCCNZ %bb.33, implicit killed $vcc
# *** IR Dump After SI peephole optimizations (si-pre-emit-peephole) ***:
# Machine code for function k_b: NoPHIs
  V_CMP_LE_I64_e32 killed $sgpr18_sgpr19, killed $vgpr0_vgpr1, implicit-def $vcc, implicit $exec
  S_CBRANCH_VCCNZ %bb.33, implicit killed $vcc
"""


def test_peephole_check_flags_only_live_scc_removals():
    """The miscompile (a removed S_AND_B64 whose SCC a select reads) is flagged; the same removal
    with a dead SCC is the pass's intended optimisation and is not."""
    out = wb.dropped_live_scc(_DUMP)
    assert len(out) == 1 and out[0].startswith("k_a:") and "S_AND_B64" in out[0]

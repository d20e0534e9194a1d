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
    (os.path.join(wb.CSRC, "wsr_copy.hip"), [*wb.COMMON, *wb.DEVICE]),
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


# ---- a fresh checkout builds ---------------------------------------------------------------------

_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _source_files():
    """The tracked files of the repository (its source), or, outside a git checkout, every file
    except built artefacts and working folders."""
    r = subprocess.run(["git", "ls-files", "-z"], cwd=_ROOT, capture_output=True)
    if r.returncode == 0 and r.stdout:
        return [p for p in r.stdout.decode().split("\0") if p]
    out = []
    for d, dirs, files in os.walk(_ROOT):
        dirs[:] = [x for x in dirs if not x.startswith((".", "_")) and not x.endswith("_out")]   # working folders
        out += [os.path.relpath(os.path.join(d, f), _ROOT) for f in files
                if not f.endswith((".so", ".o", ".pyc"))]
    return out


@pytest.fixture(scope="module")
def fresh_tree(tmp_path_factory):
    import shutil
    dst = tmp_path_factory.mktemp("fresh")
    for rel in _source_files():
        if rel.endswith((".so", ".o")):
            continue
        os.makedirs(os.path.join(dst, os.path.dirname(rel)), exist_ok=True)
        shutil.copy2(os.path.join(_ROOT, rel), os.path.join(dst, rel))
    assert not [f for _, _, fs in os.walk(dst) for f in fs if f.endswith(".so")]
    return str(dst)


def _py(tree, code, timeout=120):
    env = {k: v for k, v in os.environ.items() if k != "PYTHONPATH"}
    return subprocess.run(["python", "-c", code], cwd=tree, capture_output=True, text=True,
                          timeout=timeout, env=env)


def test_package_imports_without_library(fresh_tree):
    """With no libwsr.so, the package and its build module import; the binding refuses loudly."""
    r = _py(fresh_tree, "import paper_2608_12114_amd as p\n"
                        "from paper_2608_12114_amd import build\n"
                        "assert build.LIB_PATH.startswith(p._HERE)\n"
                        "try:\n    from paper_2608_12114_amd import wsr\n"
                        "except ImportError as e:\n    print('refused:', e)\n"
                        "else:\n    raise SystemExit('binding loaded without a library')\n")
    assert r.returncode == 0, r.stderr
    assert "refused:" in r.stdout and "not built" in r.stdout


def test_fresh_checkout_builds(fresh_tree):
    """build() on a copy of the tracked files, with no prebuilt binary anywhere, compiles every
    native part and then loads the library it built."""
    r = _py(fresh_tree, "import __graft_entry__ as g; g.build()", timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "wsr ABI version" in r.stdout
    for rel in ("paper_2608_12114_amd/libwsr.so", "synth/libsynth.so", "synth/libsynth_dev.so",
                "oracle/liboracle.so"):
        assert os.path.exists(os.path.join(fresh_tree, rel)), rel

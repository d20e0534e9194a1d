"""The C ABI on a machine without a GPU: the library loads, exports what include/wsr.h declares,
and rejects bad arguments before touching the HIP runtime (no compute call is made here)."""
import ctypes
import os
import re

import pytest

from paper_2608_12114_amd import wsr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = open(os.path.join(ROOT, "include", "wsr.h")).read()
L = wsr.lib()
A = 0x10000          # a 64 KiB-aligned fake address: never dereferenced, every call below fails first


def declared():
    body = re.sub(r"/\*.*?\*/", "", HEADER, flags=re.S)
    return sorted(set(re.findall(r"\b(wsr_[a-z0-9_]+)\s*\(", body)))


def test_exports_every_declared_symbol():
    names = declared()
    assert len(names) == 21, names
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_values():
    assert wsr.wsr_abi_version() == 3
    m = re.search(r"#define WSR_ABI_VERSION (\d+)", HEADER)
    assert int(m.group(1)) == wsr.wsr_abi_version()
    for name, val in (("WSR_OK", 0), ("WSR_E_ARG", 1), ("WSR_E_ALIGN", 2), ("WSR_E_SIZE", 3),
                      ("WSR_E_UNSUPPORTED", 4), ("WSR_E_STATE", 5), ("WSR_E_HIP", 6)):
        assert re.search(rf"\b{name} = {val}\b", HEADER), name
    assert ctypes.sizeof(wsr.wsr_mat) == 72


def _status(fn, *args):
    st = getattr(L, fn)(*args)
    if st != 0:
        assert wsr.wsr_last_error(), fn
    return st


def test_gemv_argument_checks():
    f = "wsr_gemv_f16"
    assert _status(f, A, A, A, 4, 8, 7, None) == wsr.WSR_E_ARG            # unknown format
    assert _status(f, A, A, A, 4, 8, wsr.WSR_Q4, None) == wsr.WSR_E_ARG   # q4 is not 16-bit
    assert _status(f, None, A, A, 4, 8, 1, None) == wsr.WSR_E_ARG
    assert _status(f, A, A, None, 4, 8, 1, None) == wsr.WSR_E_ARG
    assert _status(f, A, A, A, -1, 8, 1, None) == wsr.WSR_E_ARG
    assert _status(f, A, A, A, 4, 12, 1, None) == wsr.WSR_E_ALIGN          # K % 8
    assert _status(f, A + 8, A, A, 4, 8, 1, None) == wsr.WSR_E_ALIGN       # W 16-byte alignment
    assert _status(f, A, A + 4, A, 4, 8, 2, None) == wsr.WSR_E_ALIGN
    assert _status(f, A, A, A + 2, 4, 8, 2, None) == wsr.WSR_E_ALIGN       # y 4-byte alignment
    assert _status(f, A, A, A, 1 << 62, 1 << 8, 1, None) == wsr.WSR_E_SIZE
    assert _status(f, None, None, None, 0, 8, 1, None) == wsr.WSR_OK       # M = 0: nothing to do
    g = "wsr_gemv_q4"
    assert _status(g, A, None, A, A, 4, 64, None) == wsr.WSR_E_ARG          # no scales
    assert _status(g, A, A, A, A, 4, 48, None) == wsr.WSR_E_ALIGN           # K % 32
    assert _status(g, A, A + 1, A, A, 4, 64, None) == wsr.WSR_E_ALIGN       # scales 2-byte
    assert _status(g, A, A, A, A, 0, 64, None) == wsr.WSR_OK
    h = "wsr_gemv_i8"
    assert _status(h, A, None, A, A, 4, 64, None) == wsr.WSR_E_ARG          # no row scales
    assert _status(h, A, A, A, A, 4, 24, None) == wsr.WSR_E_ALIGN           # K % 16
    assert _status(h, A + 8, A, A, A, 4, 64, None) == wsr.WSR_E_ALIGN       # codes 16-byte
    assert _status(h, A, A + 1, A, A, 4, 64, None) == wsr.WSR_E_ALIGN       # scales 2-byte
    assert _status(h, A, A, A, A, 0, 16, None) == wsr.WSR_OK
    assert _status(f, A, A, A, 4, 16, wsr.WSR_I8, None) == wsr.WSR_E_ARG    # int8 is not 16-bit


def test_probe_argument_checks():
    f = "wsr_probe_read"
    need = wsr.wsr_probe_workspace_bytes(1 << 28)
    assert need == 8 * 512
    assert wsr.wsr_probe_workspace_bytes(0) == 8 and wsr.wsr_probe_workspace_bytes(5) == 8
    assert _status(f, None, 8, A, A, need, None) == wsr.WSR_E_ARG
    assert _status(f, A, 8, None, A, need, None) == wsr.WSR_E_ARG
    assert _status(f, A + 4, 8, A, A, need, None) == wsr.WSR_E_ALIGN
    assert _status(f, A, 8, A + 4, A, need, None) == wsr.WSR_E_ALIGN
    assert _status(f, A, 1 << 28, A, A, need - 8, None) == wsr.WSR_E_SIZE


def test_gemv_cols_argument_checks():
    f = "wsr_gemv_f16_cols"
    # (W, x, x_col_stride, y, y_col_stride, M, K, T, fmt, stream)
    assert _status(f, A, A, 16, A, 64, 4, 8, 2, 9, None) == wsr.WSR_E_ARG        # unknown format
    assert _status(f, A, A, 16, A, 64, 4, 8, 2, wsr.WSR_Q4, None) == wsr.WSR_E_ARG
    for T in (0, 3, 5, 32, -1):
        assert _status(f, A, A, 16, A, 64, 4, 8, T, 1, None) == wsr.WSR_E_ARG, T  # T not a power of two <= 16
    assert _status(f, A, A, 8, A, 64, 4, 8, 2, 1, None) == wsr.WSR_E_ALIGN         # x stride % 16
    assert _status(f, A, A, -16, A, 64, 4, 8, 2, 1, None) == wsr.WSR_E_ALIGN
    assert _status(f, A, A, 16, A, 6, 4, 8, 2, 1, None) == wsr.WSR_E_ALIGN         # y stride % 4
    assert _status(f, A, A, 16, A, 12, 4, 8, 2, 1, None) == wsr.WSR_E_ARG          # output columns overlap
    assert _status(f, A, A, 16, A, 16, 4, 12, 2, 1, None) == wsr.WSR_E_ALIGN       # K % 8
    assert _status(f, None, None, 0, None, 0, 0, 8, 4, 1, None) == wsr.WSR_OK      # M = 0


def test_gemv_q4_cols_argument_checks():
    f = "wsr_gemv_q4_cols"
    # (Wq, scales, x, x_col_stride, y, y_col_stride, M, K, T, stream)
    for T in (0, 3, 16, -4):
        assert _status(f, A, A, A, 64, A, 64, 4, 64, T, None) == wsr.WSR_E_ARG, T   # 1, 2, 4 or 8
    assert _status(f, A, None, A, 64, A, 64, 4, 64, 2, None) == wsr.WSR_E_ARG       # no scales
    assert _status(f, A, A, A, 64, A, 64, 4, 48, 2, None) == wsr.WSR_E_ALIGN        # K % 32
    assert _status(f, A, A, A, 72, A, 64, 4, 64, 2, None) == wsr.WSR_E_ALIGN        # x stride % 16
    assert _status(f, A, A, A, 64, A, 8, 4, 64, 2, None) == wsr.WSR_E_ARG           # output columns overlap
    assert _status(f, None, None, None, 0, None, 0, 0, 64, 8, None) == wsr.WSR_OK   # M = 0


def test_gemv_i8_cols_argument_checks():
    f = "wsr_gemv_i8_cols"
    for T in (0, 3, 16, -4):
        assert _status(f, A, A, A, 64, A, 64, 4, 64, T, None) == wsr.WSR_E_ARG, T
    assert _status(f, A, None, A, 64, A, 64, 4, 64, 2, None) == wsr.WSR_E_ARG
    assert _status(f, A, A, A, 64, A, 64, 4, 40, 2, None) == wsr.WSR_E_ALIGN        # K % 16
    assert _status(f, A, A, A, 72, A, 64, 4, 64, 2, None) == wsr.WSR_E_ALIGN        # x stride % 16
    assert _status(f, A, A, A, 64, A, 8, 4, 64, 2, None) == wsr.WSR_E_ARG           # output columns overlap
    assert _status(f, None, None, None, 0, None, 0, 0, 16, 8, None) == wsr.WSR_OK


def test_batched_sweep_argument_checks():
    good = dict(fmt=2, M=8, K=64, w=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good, good])
    ws = wsr.wsr_sweep_workspace_bytes(mats)
    f = "wsr_decode_sweep_batched"
    for b in (0, 3, 32, -2):
        assert _status(f, mats, 2, 4, b, A, ws, None) == wsr.WSR_E_ARG, b
    q = wsr.make_mats([good, dict(good, fmt=3, scales=A, y_tok_stride=16)])
    assert _status(f, q, 2, 4, 16, A, ws, None) == wsr.WSR_E_ARG                  # q4 outputs overlap too
    i8 = wsr.make_mats([good, dict(good, fmt=4, scales=A, y_tok_stride=16)])
    assert _status(f, i8, 2, 4, 8, A, ws, None) == wsr.WSR_E_ARG                  # and int8 outputs
    shared = wsr.make_mats([good, dict(good, y_tok_stride=0)])
    assert _status(f, shared, 2, 4, 2, A, ws, None) == wsr.WSR_E_ARG               # tokens would share y
    assert _status(f, mats, 2, 0, 2, A, ws, None) == wsr.WSR_E_ARG                 # n_tokens < 1
    assert _status(f, mats, 2, 4, 2, A, ws - 1, None) == wsr.WSR_E_SIZE


def test_sweep_argument_checks():
    good = dict(fmt=2, M=8, K=64, w=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good, dict(good, fmt=3, scales=A)])
    ws = wsr.wsr_sweep_workspace_bytes(mats)
    assert ws == 256 + 256 + 256        # counters, table, stream offsets
    f = "wsr_decode_sweep"
    assert _status(f, mats, 2, 0, A, ws, None) == wsr.WSR_E_ARG             # n_tokens < 1
    assert _status(f, mats, 2, 1, A + 16, ws, None) == wsr.WSR_E_ALIGN      # ws 256-byte alignment
    assert _status(f, mats, 2, 1, A, ws - 1, None) == wsr.WSR_E_SIZE
    assert _status(f, mats, 0, 1, None, 0, None) == wsr.WSR_OK              # empty sweep
    for bad, st in ((dict(good, fmt=9), wsr.WSR_E_ARG), (dict(good, flags=2), wsr.WSR_E_ARG),
                    (dict(good, K=60), wsr.WSR_E_ALIGN), (dict(good, fmt=3), wsr.WSR_E_ARG),
                    (dict(good, fmt=4), wsr.WSR_E_ARG), (dict(good, fmt=4, scales=A, K=40), wsr.WSR_E_ALIGN),
                    (dict(good, x_tok_stride=8), wsr.WSR_E_ALIGN),
                    (dict(good, y_tok_stride=-4), wsr.WSR_E_ALIGN),
                    (dict(good, x=A + 8), wsr.WSR_E_ALIGN)):
        m = wsr.make_mats([good, bad])
        assert _status(f, m, 2, 1, A, ws, None) == st, bad
        assert "matrix 1" in wsr.wsr_last_error()


def test_sweep_noalloc_argument_checks():
    """The allocation-free sweep checks its arguments, and the size of its table against the
    library's 512 KiB scratch, before any HIP call."""
    good = dict(fmt=2, M=8, K=64, w=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    f = "wsr_decode_sweep_noalloc"
    mats = wsr.make_mats([good, good])
    assert _status(f, mats, 2, 0, None) == wsr.WSR_E_ARG                      # n_tokens < 1
    assert _status(f, mats, -1, 1, None) == wsr.WSR_E_ARG
    assert _status(f, None, 2, 1, None) == wsr.WSR_E_ARG
    assert _status(f, mats, 0, 1, None) == wsr.WSR_OK                         # empty sweep
    bad = wsr.make_mats([good, dict(good, K=60)])
    assert _status(f, bad, 2, 1, None) == wsr.WSR_E_ALIGN and "matrix 1" in wsr.wsr_last_error()
    big = wsr.make_mats([dict(good, K=60)] * 6000)     # K = 60 is misaligned: the size check comes first
    fits = max(n for n in range(4000, 6000) if L.wsr_sweep_workspace_bytes(big, n) <= 512 << 10)
    assert fits >= 5000
    assert _status(f, big, fits + 1, 1, None) == wsr.WSR_E_SIZE
    assert "scratch" in wsr.wsr_last_error()


def test_sweep_staged_argument_checks():
    f = "wsr_sweep_staged"
    good = dict(fmt=2, M=8, K=64, w=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good, dict(good, fmt=4, scales=A)])
    assert _status(f, mats, 2, -1, A, 1 << 20, None, None) == wsr.WSR_E_ARG        # negative token
    assert _status(f, mats, 2, 0, None, 1 << 20, None, None) == wsr.WSR_E_ARG      # no staging buffer
    assert _status(f, mats, 2, 0, A + 16, 1 << 20, None, None) == wsr.WSR_E_ALIGN  # 256-byte alignment
    assert _status(f, mats, 2, 0, A, 600, None, None) == wsr.WSR_E_SIZE            # a half holds no row
    assert "holds no row" in wsr.wsr_last_error()
    assert _status(f, mats, 0, 0, None, 0, None, None) == wsr.WSR_OK               # nothing to do
    bad = wsr.make_mats([dict(good, fmt=3)])                                        # q4 without scales
    assert _status(f, bad, 1, 0, A, 1 << 20, None, None) == wsr.WSR_E_ARG
    bad = wsr.make_mats([dict(good, x_tok_stride=8)])
    assert _status(f, bad, 1, 0, A, 1 << 20, None, None) == wsr.WSR_E_ALIGN


def test_sweep_ordered_argument_checks():
    f = "wsr_decode_sweep_ordered"
    good = dict(fmt=2, M=8, K=64, w=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good])
    ws = wsr.wsr_sweep_workspace_bytes(mats)
    for mode in (-1, 4):
        assert _status(f, mats, 1, 1, A, ws, None, None, mode) == wsr.WSR_E_ARG
    for mode in (1, 2, 3):
        assert _status(f, mats, 1, 0, A, ws, None, None, mode) == wsr.WSR_E_ARG      # n_tokens < 1
        assert _status(f, mats, 1, 1, A, ws - 1, None, None, mode) == wsr.WSR_E_SIZE
        assert _status(f, mats, 0, 1, None, 0, None, None, mode) == wsr.WSR_OK       # empty sweep
    assert _status(f, mats, 1, 0, A, ws, None, None, 0) == wsr.WSR_E_ARG             # in-stream: sweep's checks


def test_sweep_mma_argument_checks():
    f = "wsr_decode_sweep_mma"
    good = dict(fmt=3, M=8, K=64, w=A, scales=A, x=A, y=A, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good])
    ws = wsr.wsr_sweep_workspace_bytes(mats)
    assert _status(f, mats, 1, 0, A, ws, None) == wsr.WSR_E_ARG                  # n_tokens < 1
    assert _status(f, mats, 1, 1, A, ws - 1, None) == wsr.WSR_E_SIZE
    assert _status(f, mats, 0, 4, None, 0, None) == wsr.WSR_OK                   # empty sweep
    shared = wsr.make_mats([dict(good, y_tok_stride=16)])
    assert _status(f, shared, 1, 2, A, ws, None) == wsr.WSR_E_ARG                # tokens would share y
    # 64 rows and 16 tokens must stay within 32-bit lane offsets
    long_row = wsr.make_mats([dict(good, fmt=2, scales=None, M=1, K=(1 << 24) + 8, x_tok_stride=(1 << 25) + 16)])
    assert _status(f, long_row, 1, 1, A, ws, None) == wsr.WSR_E_SIZE             # row above 32 MiB
    assert "32 MiB" in wsr.wsr_last_error()
    wide_x = wsr.make_mats([dict(good, x_tok_stride=(1 << 27) + 16)])
    assert _status(f, wide_x, 1, 1, A, ws, None) == wsr.WSR_E_SIZE               # token stride above 128 MiB


def test_register_argument_checks():
    f = "wsr_register_host"
    dev, gr = ctypes.c_void_p(), ctypes.c_uint()
    page = os.sysconf("SC_PAGE_SIZE")
    args = lambda h, n, fl: (h, n, fl, ctypes.byref(dev), ctypes.byref(gr))
    assert _status(f, *args(None, page, 0)) == wsr.WSR_E_ARG
    assert _status(f, *args(A, 0, 0)) == wsr.WSR_E_ARG
    assert _status(f, *args(A, page, 8)) == wsr.WSR_E_ARG                   # unknown flag
    assert _status(f, *args(A + 64, page, 0)) == wsr.WSR_E_ALIGN            # base off a page
    assert _status(f, *args(A, page + 1, 0)) == wsr.WSR_E_ALIGN             # partial last page
    assert _status("wsr_unregister_host", A) == wsr.WSR_E_STATE
    with pytest.raises(wsr.WsrError) as e:
        wsr.wsr_unregister_host(A)
    assert e.value.status == wsr.WSR_E_STATE


def test_one_hip_runtime_per_process():
    """The binding binds libwsr.so to the HIP runtime PyTorch already loaded: two runtimes in one
    process each open the device, and the second finds none."""
    import subprocess
    import sys
    code = ("import ctypes, re, sys; sys.path.insert(0, %r); "
            "from paper_2608_12114_amd import wsr; "
            "from synth import device; "
            "m = open('/proc/self/maps').read(); "
            "print(len(set(re.findall(r'/\\S*libamdhip64\\S*', m))))" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, check=True)
    assert out.stdout.strip() == "1", out.stdout + out.stderr

"""Python binding of libwsr: the entry points of include/wsr.h under the same names.

Argument marshalling only: every operation runs in the HIP kernels of libwsr.so, and importing this
module fails loudly when the library is not built.  Pointers are plain integers or objects with a
`data_ptr()` method (PyTorch tensors); `stream` is a hipStream_t as an integer, an object with a
`cuda_stream` attribute (a torch.cuda.Stream), or None for the null stream.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwsr.so")

WSR_OK, WSR_E_ARG, WSR_E_ALIGN, WSR_E_SIZE, WSR_E_UNSUPPORTED, WSR_E_STATE, WSR_E_HIP = range(7)
STATUS_NAMES = {0: "WSR_OK", 1: "WSR_E_ARG", 2: "WSR_E_ALIGN", 3: "WSR_E_SIZE",
                4: "WSR_E_UNSUPPORTED", 5: "WSR_E_STATE", 6: "WSR_E_HIP"}
WSR_F16, WSR_BF16, WSR_Q4, WSR_I8 = 1, 2, 3, 4
WSR_REG_READONLY, WSR_REG_PIN, WSR_REG_PREPINNED = 1, 2, 4
WSR_MAT_AFTER_PREVIOUS = 1
WSR_ORDER_STREAM, WSR_ORDER_EVENT, WSR_ORDER_HOST_EVENT, WSR_ORDER_DRAIN = range(4)
ORDER_NAMES = {0: "in-stream", 1: "event", 2: "host-visible event", 3: "host drain"}
WSR_EP_NONE, WSR_EP_MAP, WSR_EP_RESIDENT, WSR_EP_COPY, WSR_EP_STORAGE_BOUND = range(5)
ENDPOINT_NAMES = {0: "none", 1: "map", 2: "resident", 3: "copy", 4: "storage-bound"}


class WsrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class wsr_mat(ctypes.Structure):
    _fields_ = [("fmt", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("M", ctypes.c_int64), ("K", ctypes.c_int64),
                ("w", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("x_tok_stride", ctypes.c_int64),
                ("y", ctypes.c_void_p), ("y_tok_stride", ctypes.c_int64)]


class wsr_endpoint_probe(ctypes.Structure):
    _fields_ = [("w_bytes", ctypes.c_double), ("rate", ctypes.c_double * 3),
                ("mapped_resident", ctypes.c_int32), ("resident_ok", ctypes.c_int32),
                ("excluded", ctypes.c_uint32), ("reserved", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; g.build()'` "
                      "from the repository root")

# PyTorch ships its own HIP runtime.  Loading it first makes libwsr.so bind to that same runtime
# (its libamdhip64.so.7 dependency is then already satisfied); loading libwsr.so first would put a
# second HIP/HSA runtime into the process, and whichever initialises second finds no device.
import torch  # noqa: E402,F401

_L = ctypes.CDLL(LIB_PATH)
_vp, _sz, _i64, _i32, _u = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint
_L.wsr_last_error.restype = ctypes.c_char_p
_L.wsr_last_error.argtypes = []
_L.wsr_abi_version.restype = ctypes.c_int
_L.wsr_abi_version.argtypes = []
_L.wsr_register_host.argtypes = [_vp, _sz, _u, ctypes.POINTER(_vp), ctypes.POINTER(_u)]
_L.wsr_unregister_host.argtypes = [_vp]
_L.wsr_probe_workspace_bytes.argtypes = [_sz]
_L.wsr_probe_workspace_bytes.restype = _sz
_L.wsr_probe_read.argtypes = [_vp, _sz, _vp, _vp, _sz, _vp]
_L.wsr_gemv_f16.argtypes = [_vp, _vp, _vp, _i64, _i64, ctypes.c_int, _vp]
_L.wsr_gemv_q4.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _vp]
_L.wsr_sweep_workspace_bytes.argtypes = [ctypes.POINTER(wsr_mat), _i32]
_L.wsr_sweep_workspace_bytes.restype = _sz
_L.wsr_decode_sweep.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _vp, _sz, _vp]
_L.wsr_gemv_f16_cols.argtypes = [_vp, _vp, _i64, _vp, _i64, _i64, _i64, _i32, ctypes.c_int, _vp]
_L.wsr_decode_sweep_batched.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _i32, _vp, _sz, _vp]
_L.wsr_gemv_q4_cols.argtypes = [_vp, _vp, _vp, _i64, _vp, _i64, _i64, _i64, _i32, _vp]
_L.wsr_gemv_i8.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _vp]
_L.wsr_sweep_staged.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _vp, _sz, _vp, _vp]
_L.wsr_decode_sweep_mma.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _vp, _sz, _vp]
_L.wsr_decode_sweep_ordered.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _vp, _sz, _vp, _vp, _i32]
_L.wsr_host_resident_pages.argtypes = [_vp, _sz, ctypes.POINTER(_sz), ctypes.POINTER(_sz)]
_L.wsr_select_endpoint.argtypes = [ctypes.POINTER(wsr_endpoint_probe), ctypes.c_double, ctypes.POINTER(_i32),
                                   ctypes.POINTER(ctypes.c_double)]
_L.wsr_gemv_i8_cols.argtypes = [_vp, _vp, _vp, _i64, _vp, _i64, _i64, _i64, _i32, _vp]
_L.wsr_decode_sweep_noalloc.argtypes = [ctypes.POINTER(wsr_mat), _i32, _i32, _vp]
for _f in ("wsr_register_host", "wsr_unregister_host", "wsr_probe_read", "wsr_gemv_f16",
           "wsr_gemv_q4", "wsr_decode_sweep", "wsr_gemv_f16_cols", "wsr_decode_sweep_batched",
           "wsr_gemv_q4_cols", "wsr_gemv_i8", "wsr_gemv_i8_cols", "wsr_sweep_staged", "wsr_host_resident_pages", "wsr_decode_sweep_ordered", "wsr_decode_sweep_mma",
           "wsr_select_endpoint", "wsr_decode_sweep_noalloc"):
    getattr(_L, _f).restype = ctypes.c_int


def lib() -> ctypes.CDLL:
    return _L


def _ptr(a) -> int | None:
    if a is None:
        return None
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    return int(a)


def _stream(s) -> int | None:
    if s is None:
        return None
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream
    return int(s)


def _check(st: int) -> None:
    if st != WSR_OK:
        raise WsrError(st, wsr_last_error())


def wsr_last_error() -> str:
    return _L.wsr_last_error().decode()


def wsr_abi_version() -> int:
    return _L.wsr_abi_version()


def wsr_register_host(host, nbytes: int, flags: int = 0) -> tuple[int, int]:
    """Returns (device address, granted flags)."""
    dev, granted = _vp(), _u()
    _check(_L.wsr_register_host(_ptr(host), nbytes, flags, ctypes.byref(dev), ctypes.byref(granted)))
    return dev.value, granted.value


def wsr_unregister_host(host) -> None:
    _check(_L.wsr_unregister_host(_ptr(host)))


def wsr_probe_workspace_bytes(n: int) -> int:
    return _L.wsr_probe_workspace_bytes(n)


def wsr_probe_read(buf, n: int, sum_dev, ws, ws_bytes: int, stream=None) -> None:
    _check(_L.wsr_probe_read(_ptr(buf), n, _ptr(sum_dev), _ptr(ws), ws_bytes, _stream(stream)))


def wsr_gemv_f16(W, x, y, M: int, K: int, fmt: int, stream=None) -> None:
    _check(_L.wsr_gemv_f16(_ptr(W), _ptr(x), _ptr(y), M, K, fmt, _stream(stream)))


def wsr_gemv_f16_cols(W, x, x_col_stride: int, y, y_col_stride: int, M: int, K: int, T: int, fmt: int,
                      stream=None) -> None:
    _check(_L.wsr_gemv_f16_cols(_ptr(W), _ptr(x), x_col_stride, _ptr(y), y_col_stride, M, K, T, fmt,
                                _stream(stream)))


def wsr_gemv_q4_cols(Wq, scales, x, x_col_stride: int, y, y_col_stride: int, M: int, K: int, T: int,
                     stream=None) -> None:
    _check(_L.wsr_gemv_q4_cols(_ptr(Wq), _ptr(scales), _ptr(x), x_col_stride, _ptr(y), y_col_stride, M, K, T,
                               _stream(stream)))


def wsr_gemv_q4(Wq, scales, x, y, M: int, K: int, stream=None) -> None:
    _check(_L.wsr_gemv_q4(_ptr(Wq), _ptr(scales), _ptr(x), _ptr(y), M, K, _stream(stream)))


def wsr_gemv_i8(Wq, scales, x, y, M: int, K: int, stream=None) -> None:
    _check(_L.wsr_gemv_i8(_ptr(Wq), _ptr(scales), _ptr(x), _ptr(y), M, K, _stream(stream)))


def wsr_gemv_i8_cols(Wq, scales, x, x_col_stride: int, y, y_col_stride: int, M: int, K: int, T: int,
                     stream=None) -> None:
    _check(_L.wsr_gemv_i8_cols(_ptr(Wq), _ptr(scales), _ptr(x), x_col_stride, _ptr(y), y_col_stride, M, K, T,
                               _stream(stream)))


def make_mats(specs) -> ctypes.Array:
    """specs: iterable of dicts with keys fmt, M, K, w, x, y and optionally scales, flags,
    x_tok_stride, y_tok_stride (pointers as ints or tensors)."""
    specs = list(specs)
    arr = (wsr_mat * max(1, len(specs)))()
    for i, s in enumerate(specs):
        arr[i] = wsr_mat(s["fmt"], s.get("flags", 0), s["M"], s["K"], _ptr(s["w"]),
                         _ptr(s.get("scales")), _ptr(s["x"]), s.get("x_tok_stride", 0),
                         _ptr(s["y"]), s.get("y_tok_stride", 0))
    arr._n = len(specs)
    return arr


def _n(mats) -> int:
    return getattr(mats, "_n", len(mats))


def wsr_sweep_workspace_bytes(mats) -> int:
    return _L.wsr_sweep_workspace_bytes(mats, _n(mats))


def wsr_decode_sweep(mats, n_tokens: int, ws, ws_bytes: int, stream=None) -> None:
    _check(_L.wsr_decode_sweep(mats, _n(mats), n_tokens, _ptr(ws), ws_bytes, _stream(stream)))


def wsr_decode_sweep_noalloc(mats, n_tokens: int, stream=None) -> None:
    _check(_L.wsr_decode_sweep_noalloc(mats, _n(mats), n_tokens, _stream(stream)))


def wsr_decode_sweep_batched(mats, n_tokens: int, batch: int, ws, ws_bytes: int, stream=None) -> None:
    _check(_L.wsr_decode_sweep_batched(mats, _n(mats), n_tokens, batch, _ptr(ws), ws_bytes, _stream(stream)))


def wsr_sweep_staged(mats, token: int, stage, stage_bytes: int, stream=None, copy_stream=None) -> None:
    _check(_L.wsr_sweep_staged(mats, _n(mats), token, _ptr(stage), stage_bytes, _stream(stream),
                               _stream(copy_stream)))


def wsr_host_resident_pages(host, nbytes: int) -> tuple[int, int]:
    """Returns (resident pages, pages spanned)."""
    r, t = _sz(), _sz()
    _check(_L.wsr_host_resident_pages(_ptr(host), nbytes, ctypes.byref(r), ctypes.byref(t)))
    return r.value, t.value


def wsr_select_endpoint(w_bytes: float, b_map: float, b_resident: float, b_copy: float, theta: float = 0.05,
                        mapped_resident: bool = True, resident_ok: bool = True,
                        excluded: int = 0) -> tuple[int, list[float]]:
    """Alg. 2: returns (endpoint code, [W/B in ms for map, resident, copy]); rates in bytes/s, <= 0
    for an endpoint not measured."""
    p = wsr_endpoint_probe(w_bytes, (ctypes.c_double * 3)(b_map, b_resident, b_copy), int(bool(mapped_resident)),
                           int(bool(resident_ok)), excluded, 0)
    c = _i32()
    t = (ctypes.c_double * 3)()
    _check(_L.wsr_select_endpoint(ctypes.byref(p), theta, ctypes.byref(c), t))
    return c.value, list(t)


def wsr_decode_sweep_ordered(mats, n_tokens: int, ws, ws_bytes: int, framework_stream, own_stream, mode: int) -> None:
    _check(_L.wsr_decode_sweep_ordered(mats, _n(mats), n_tokens, _ptr(ws), ws_bytes, _stream(framework_stream),
                                       _stream(own_stream), mode))


def wsr_decode_sweep_mma(mats, n_tokens: int, ws, ws_bytes: int, stream=None) -> None:
    _check(_L.wsr_decode_sweep_mma(mats, _n(mats), n_tokens, _ptr(ws), ws_bytes, _stream(stream)))

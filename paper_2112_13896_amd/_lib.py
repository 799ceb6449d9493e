"""ctypes loader for libcs.so (the C ABI declared in include/cs.h).

The library is built in-tree (python -m paper_2112_13896_amd.build).  There is
no fallback: if it is missing or cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcs.so")
# the same library with the product counter compiled in (tests only)
COUNT_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcs_count.so")
STAMP_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcs_stamps.so")

CS_OK = 0
CS_ERR_ARG = -1
CS_ERR_SHAPE = -2
CS_ERR_DTYPE = -3
CS_ERR_COLLISION = -4
CS_ERR_WORKSPACE = -5
CS_ERR_DEVICE = -6
CS_ERR_UNSUPPORTED = -7

CS_I8, CS_I32, CS_F32 = 0, 1, 2

CS_MAX_ROW = 65535
CS_MAX_N = 32
CS_MAX_KWTA_ROW = 2048
CS_NOALLOC_SCRATCH_BYTES = 64 << 20

# name -> (restype, argtypes), in the order of include/cs.h
_c = ctypes
_vp, _i, _i64, _sz = _c.c_void_p, _c.c_int, _c.c_int64, _c.c_size_t
SIGNATURES = {
    "cs_pack": (_i, [_i, _vp, _i, _i, _i, _vp, _c.POINTER(_i64), _c.POINTER(_i), _c.POINTER(_i)]),
    "cs_compact": (_i, [_i, _vp, _i64, _i, _vp, _vp, _vp, _vp]),
    "cs_mrs_conv2d": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i,
                           _vp, _i, _vp, _vp]),
    "cs_mrs_kwta_conv2d": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i,
                                _vp, _i, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _i, _vp]),
    "cs_mrs_kwta_units_conv2d": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp,
                                      _i, _i, _vp, _i, _vp, _i, _i, _i, _vp, _vp, _vp, _vp, _i,
                                      _vp]),
    "cs_mrs_plan": (_i, [_i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i,
                         _c.POINTER(_i64)]),
    "cs_mrs_kwta_chain2": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i,
                                _vp, _i, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _i, _vp, _i, _i, _vp,
                                _vp, _vp]),
    "cs_conv2d_dense_kwta_chain3": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _i,
                                         _vp, _i, _i, _vp, _i, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _i,
                                         _i, _i, _i, _i, _vp, _i, _i, _vp, _i, _vp, _i, _i,
                                         _vp, _vp, _vp, _i,
                                         _vp, _i, _i, _vp, _vp, _i, _i, _vp, _vp, _vp, _i,
                                         _vp, _i, _i, _vp, _vp, _vp]),
    "cs_mrs_kwta_chain3": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i,
                                _vp, _i, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _i,
                                _vp, _i, _i, _vp, _vp, _i, _i, _vp, _vp, _vp, _i,
                                _vp, _i, _i, _vp, _vp, _vp]),
    "cs_conv2d_dense_kwta": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _i,
                                  _vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _i, _vp]),
    "cs_reorder_table": (_i, [_vp, _i, _i, _i, _i, _i, _c.POINTER(_i), _vp]),
    "cs_pack_blocks": (_i, [_i, _vp, _i, _i, _i, _i, _vp, _vp, _c.POINTER(_i64), _c.POINTER(_i),
                            _c.POINTER(_i)]),
    "cs_pack_channels": (_i, [_i, _vp, _i, _i, _i, _i, _i, _vp, _c.POINTER(_i64), _c.POINTER(_i),
                              _c.POINTER(_i)]),
    "cs_channel_table": (_i, [_vp, _i, _i, _i, _i, _i, _i, _vp]),
    "cs_conv2d_channels": (_i, [_vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _vp, _vp]),
    "cs_reorder_table_channels": (_i, [_vp, _i, _i, _i, _i, _i, _c.POINTER(_i), _vp]),
    "cs_conv2d_reorder_kwta": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _vp,
                                    _i, _i, _i, _vp, _vp, _vp, _vp, _i, _vp]),
    "cs_linear": (_i, [_i, _vp, _i, _i, _vp, _i, _i, _vp, _vp, _vp, _sz, _vp]),
    "cs_conv2d": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _i, _vp, _vp,
                       _sz, _vp]),
    "cs_conv2d_noalloc": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _i,
                               _vp, _vp]),
    "cs_conv2d_dense_blocks": (_i, [_vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _vp, _i, _i, _vp,
                                    _vp, _vp]),
    "cs_conv2d_dense": (_i, [_i, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _i, _vp, _i,
                             _vp, _vp]),
    "cs_kwta": (_i, [_i, _vp, _i64, _i, _i, _i, _i, _vp, _vp]),
    "cs_kwta_lists": (_i, [_i, _vp, _i64, _i, _i, _i, _i, _vp, _vp, _vp, _i, _vp]),
    "cs_workspace_bytes": (_sz, [_i, _i, _i64, _i]),
    "cs_product_count": (_i, [_c.POINTER(_c.c_ulonglong), _i]),
    "cs_phase_stamps": (_i, [_c.POINTER(_c.c_ulonglong), _i, _i, _c.POINTER(_c.c_int)]),
    "cs_status_str": (_c.c_char_p, [_i]),
}


class CSError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({status_str(status)})")


_LIB = None
_LOADED = {}


def _load(path: str) -> ctypes.CDLL:
    if path not in _LOADED:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "`python -m paper_2112_13896_amd.build`")
        L = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LOADED[path] = L
    return _LOADED[path]


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it is not built)."""
    global _LIB
    if _LIB is None:
        _LIB = _load(LIB_PATH)
    return _LIB


class counting_library:
    """Context manager: every call made through the binding inside it goes to
    the counting build (libcs_count.so), whose kernels count the products they
    form (read with product_count()).  Tests only."""

    def __enter__(self):
        global _LIB
        self._prev = _LIB
        _LIB = _load(COUNT_LIB_PATH)
        return self

    def __exit__(self, *exc):
        global _LIB
        _LIB = self._prev
        return False


class stamping_library(counting_library):
    """Context manager: calls inside it go to the stamping build
    (libcs_stamps.so), whose layer kernels add up wall-clock stamps at their
    phase boundaries (read with phase_stamps())."""

    def __enter__(self):
        global _LIB
        self._prev = _LIB
        _LIB = _load(STAMP_LIB_PATH)
        return self


def phase_stamps(reset: bool = False):
    """cs_phase_stamps of the library in use: (the 32 slot sums, the wall
    clock's rate in kHz); raises CSError with CS_ERR_UNSUPPORTED outside the
    stamping build."""
    acc = (ctypes.c_ulonglong * 32)()
    khz = ctypes.c_int(0)
    check("cs_phase_stamps", lib().cs_phase_stamps(acc, 32, int(bool(reset)), ctypes.byref(khz)))
    return [int(v) for v in acc], int(khz.value)


def product_count(reset: bool = False) -> int:
    """cs_product_count of the library in use (raises CSError with
    CS_ERR_UNSUPPORTED outside the counting build)."""
    v = ctypes.c_ulonglong(0)
    check("cs_product_count", lib().cs_product_count(ctypes.byref(v), int(bool(reset))))
    return int(v.value)


def status_str(status: int) -> str:
    return lib().cs_status_str(int(status)).decode()


def check(fn: str, status: int) -> None:
    if status != CS_OK:
        raise CSError(fn, status)

"""ctypes binding of libtopkv_ceiling.so (include/topkv_ceiling.h): the plain
copy and empty kernels the benchmark reads the pack/unpack kernels against.
Argument marshalling only; importing it without the built library raises
ImportError."""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must load torch's HIP runtime before the library)

from .topkv import TopkvError, _ptr, _stream

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtopkv_ceiling.so")
if not os.path.exists(LIBRARY):
    raise ImportError(f"{LIBRARY} is missing: build it with `python -m paper_2607_28633_amd.build`")
_lib = ctypes.CDLL(LIBRARY)

EXPORTS = ["topkv_ceiling_copy", "topkv_ceiling_copy_layers", "topkv_ceiling_read", "topkv_ceiling_empty",
           "topkv_ceiling_copy_timeline", "topkv_ceiling_wall_clock_khz", "topkv_ceiling_copy_tiles"]
_P, _I32, _I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
_SIGS = {
    "topkv_ceiling_copy": [_P, _P, _I64, _P],
    "topkv_ceiling_copy_layers": [_P, _I64, _P, _I64, _I64, _I32, _I32, _P],
    "topkv_ceiling_read": [_P, _I64, _P, _P],
    "topkv_ceiling_empty": [_P],
    "topkv_ceiling_copy_timeline": [_P, _P, _I64, _P, _P],
    "topkv_ceiling_wall_clock_khz": [ctypes.POINTER(_I32)],
    "topkv_ceiling_copy_tiles": [_P, _I64, _P, _P, _I64, _P, _P, _I32, _P],
}
for _name, _args in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _I32
    _fn.argtypes = _args


def _check(st: int) -> None:
    if st:
        raise TopkvError(st)


def topkv_ceiling_copy(src, dst, nbytes, stream=None) -> None:
    _check(_lib.topkv_ceiling_copy(_ptr(src), _ptr(dst), int(nbytes), _stream(stream)))


def topkv_ceiling_copy_layers(src, src_stride, dst, dst_stride, layer_bytes, layers, workgroups_per_cu=0,
                              stream=None) -> None:
    _check(_lib.topkv_ceiling_copy_layers(_ptr(src), int(src_stride), _ptr(dst), int(dst_stride), int(layer_bytes),
                                          int(layers), int(workgroups_per_cu), _stream(stream)))


def topkv_ceiling_read(src, nbytes, sink, stream=None) -> None:
    _check(_lib.topkv_ceiling_read(_ptr(src), int(nbytes), _ptr(sink), _stream(stream)))


def topkv_ceiling_copy_tiles(src, src_bytes, src_off, dst, dst_bytes, dst_off, lens, tiles, stream=None) -> None:
    _check(_lib.topkv_ceiling_copy_tiles(_ptr(src), int(src_bytes), _ptr(src_off), _ptr(dst), int(dst_bytes),
                                         _ptr(dst_off), _ptr(lens), int(tiles), _stream(stream)))


def topkv_ceiling_empty(stream=None) -> None:
    _check(_lib.topkv_ceiling_empty(_stream(stream)))


def topkv_ceiling_copy_timeline(src, dst, nbytes, stamps, stream=None) -> None:
    _check(_lib.topkv_ceiling_copy_timeline(_ptr(src), _ptr(dst), int(nbytes), _ptr(stamps), _stream(stream)))


def topkv_ceiling_wall_clock_khz() -> int:
    khz = _I32(0)
    _check(_lib.topkv_ceiling_wall_clock_khz(ctypes.byref(khz)))
    return int(khz.value)

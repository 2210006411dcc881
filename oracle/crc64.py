"""CRC-64/XZ of host buffers through the oracle's plain C byte loop
(oracle/crc64.c).  TEST INFRASTRUCTURE ONLY."""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "crc64.c")
LIBRARY = os.path.join(_HERE, "liboraclecrc64.so")


def build() -> str:
    """Compile the C oracle (gcc, host only)."""
    subprocess.run(["gcc", "-O2", "-shared", "-fPIC", "-o", LIBRARY, SOURCE], check=True)
    return LIBRARY


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build()
        _lib = ctypes.CDLL(LIBRARY)
        _lib.oracle_crc64_update.restype = ctypes.c_uint64
        _lib.oracle_crc64_update.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_size_t]
    return _lib


def crc64(data, crc: int = 0) -> int:
    """CRC-64/XZ of `data` (bytes or a numpy array, any dtype, read as its
    raw bytes), continuing from `crc` (0 to start)."""
    if isinstance(data, (bytes, bytearray)):
        buf = np.frombuffer(bytes(data), dtype=np.uint8)
    else:
        buf = np.ascontiguousarray(data).reshape(-1).view(np.uint8)
    return int(_load().oracle_crc64_update(crc, buf.ctypes.data if buf.size else None, buf.size))

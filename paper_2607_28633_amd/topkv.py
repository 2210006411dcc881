"""ctypes binding of libtopkv.so (declared in include/topkv.h).

Argument marshalling only: every function here forwards to the C entry point
of the same name, passing raw device pointers taken from torch tensors (or
plain integers) and the caller's HIP stream, and raises :class:`TopkvError`
on a non-zero status.  Every byte is moved by the library's HIP kernels.

Importing this module loads the library and fails loudly (ImportError) when
it has not been built; there is no fallback path.  torch is imported first so
the library binds to the HIP runtime torch already loaded (one runtime per
process).
"""
from __future__ import annotations

import ctypes
import os
import sys

import torch  # noqa: F401  (must load torch's HIP runtime before libtopkv.so)

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtopkv.so")

if not os.path.exists(LIBRARY):
    raise ImportError(f"{LIBRARY} is missing: build it with `python -m paper_2607_28633_amd.build` "
                      "(or __graft_entry__.build()); there is no non-HIP fallback")
_lib = ctypes.CDLL(LIBRARY)

TOPKV_OK = 0
TOPKV_ERR_INVALID_ARG = 1
TOPKV_ERR_UNSUPPORTED = 2
TOPKV_ERR_LAUNCH = 3
TOPKV_ERR_BOUNDS = 4
TOPKV_ERR_DEVICE = 5
TOPKV_ERR_CHECKSUM = 6
TOPKV_ERR_TIMEOUT = 7
TOPKV_ERR_CANCELLED = 8
TOPKV_MAX_BATCH_REQS = 4096
TOPKV_CHECK_RESULT_WORDS = 4

EXPORTS = ["topkv_pack_layer", "topkv_unpack_layer", "topkv_pack_layer_batched",
           "topkv_unpack_layer_batched", "topkv_pack_layer_batched_ex",
           "topkv_unpack_layer_batched_ex", "topkv_packed_layer_bytes", "topkv_status_string",
           "topkv_check_tables", "topkv_check_workspace_bytes", "topkv_pack_layer_window",
           "topkv_unpack_layer_window", "topkv_packed_window_bytes", "topkv_pack_layer_planes",
           "topkv_unpack_layer_planes", "topkv_kvcache1_bytes", "topkv_kvcache1_workspace_bytes",
           "topkv_kvcache1_pack_layer", "topkv_kvcache1_seal", "topkv_kvcache1_verify",
           "topkv_kvcache1_unpack_layer", "topkv_crc64", "topkv_crc64_workspace_bytes", "topkv_dma_create",
           "topkv_dma_submit", "topkv_dma_wait", "topkv_dma_destroy", "topkv_move_layer", "topkv_move_layers",
           "topkv_pack_layer_heads", "topkv_unpack_layer_heads", "topkv_reblock_layer",
           "topkv_pack_layer_shards", "topkv_unpack_layer_shards", "topkv_packed_state_bytes",
           "topkv_pack_state_layer", "topkv_unpack_state_layer", "topkv_check_state_slots",
           "topkv_check_state_workspace_bytes", "topkv_kvcache1_pack_layers", "topkv_kvcache1_unpack_layers",
           "topkv_kvcache1_pack_seal", "topkv_kvcache1_verify_unpack", "topkv_engine_pack_layers",
           "topkv_engine_unpack_layers", "topkv_engine_layers_per_grid", "topkv_crc64_noalloc"]

TOPKV_LAYOUT_PACKED = 0
TOPKV_LAYOUT_POOL = 1
TOPKV_LAYOUT_POOL_HEAD_MAJOR = 2


class topkv_pool_t(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("num_pages", ctypes.c_int64),
                ("num_layers", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("planes", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32)]


class topkv_view_t(ctypes.Structure):
    _fields_ = [("layout", ctypes.c_int32), ("layer", ctypes.c_int32), ("head_begin", ctypes.c_int32),
                ("bt_stride", ctypes.c_int32), ("block_tables", ctypes.c_void_p), ("pool", topkv_pool_t),
                ("data", ctypes.c_void_p), ("bytes", ctypes.c_int64), ("shards", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class topkv_state_pool_t(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("num_slots", ctypes.c_int64), ("state_bytes", ctypes.c_int64),
                ("num_layers", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class topkv_launch_t(ctypes.Structure):
    _fields_ = [("stream", ctypes.c_void_p), ("start", ctypes.c_void_p), ("stop", ctypes.c_void_p)]


class topkv_engine_t(ctypes.Structure):
    _fields_ = [("ready", ctypes.c_void_p), ("cancel", ctypes.c_void_p), ("status", ctypes.c_void_p),
                ("epoch", ctypes.c_uint32), ("workgroups_per_cu", ctypes.c_int32), ("timeout_us", ctypes.c_int64),
                ("layers_per_grid", ctypes.c_int32)]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_POOL = ctypes.POINTER(topkv_pool_t)
_SIGS = {
    "topkv_pack_layer": (_I32, [_POOL, _I32, _P, _I32, _P, _P]),
    "topkv_unpack_layer": (_I32, [_P, _POOL, _I32, _P, _I32, _P]),
    "topkv_pack_layer_batched": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _P, _I64, _P]),
    "topkv_unpack_layer_batched": (_I32, [_P, _I64, _POOL, _I32, _I32, _P, _I32, _P, _P]),
    "topkv_pack_layer_batched_ex": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _P, _I64,
                                           ctypes.POINTER(topkv_launch_t)]),
    "topkv_unpack_layer_batched_ex": (_I32, [_P, _I64, _POOL, _I32, _I32, _P, _I32, _P,
                                             ctypes.POINTER(topkv_launch_t)]),
    "topkv_packed_layer_bytes": (_I64, [_POOL, ctypes.POINTER(_I32), _I32]),
    "topkv_status_string": (ctypes.c_char_p, [_I32]),
    "topkv_check_tables": (_I32, [_POOL, _I32, _P, _I32, _P, _I32, _P, _I64, _P, _P]),
    "topkv_check_workspace_bytes": (_I64, [_POOL]),
    "topkv_pack_layer_window": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _I32, _P, _I64,
                                       ctypes.POINTER(topkv_launch_t)]),
    "topkv_unpack_layer_window": (_I32, [_P, _I64, _POOL, _I32, _I32, _P, _I32, _P, _I32,
                                         ctypes.POINTER(topkv_launch_t)]),
    "topkv_packed_window_bytes": (_I64, [_POOL, ctypes.POINTER(_I32), _I32, _I32]),
    "topkv_pack_layer_planes": (_I32, [_POOL, _I32, _P, _I32, _P, _I64, _I64, _P]),
    "topkv_unpack_layer_planes": (_I32, [_P, _I64, _I64, _POOL, _I32, _P, _I32, _P]),
    "topkv_kvcache1_bytes": (_I64, [_POOL, _I32]),
    "topkv_kvcache1_workspace_bytes": (_I64, [_POOL, _I32]),
    "topkv_kvcache1_pack_layer": (_I32, [_POOL, _I32, _P, _I32, _P, _I64, _P]),
    "topkv_kvcache1_seal": (_I32, [_POOL, _I32, ctypes.c_uint64, ctypes.c_uint64, _P, _I64, _P, _I64, _P]),
    "topkv_kvcache1_verify": (_I32, [_POOL, _I32, ctypes.c_uint64, ctypes.c_uint64, _P, _I64, _P, _I64, _P, _P]),
    "topkv_kvcache1_unpack_layer": (_I32, [_P, _I64, _POOL, _I32, _P, _I32, _P]),
    "topkv_kvcache1_pack_layers": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _I64, _P]),
    "topkv_kvcache1_unpack_layers": (_I32, [_P, _I64, _POOL, _I32, _I32, _P, _I32, _P]),
    "topkv_kvcache1_pack_seal": (_I32, [_POOL, _P, _I32, ctypes.c_uint64, ctypes.c_uint64, _P, _I64, _P, _I64, _P]),
    "topkv_kvcache1_verify_unpack": (_I32, [_P, _I64, _POOL, _P, _I32, ctypes.c_uint64, ctypes.c_uint64, _P, _I64,
                                            _P, _P]),
    "topkv_crc64": (_I32, [_P, _I64, _P, _I64, _P, _P]),
    "topkv_crc64_workspace_bytes": (_I64, [_I64]),
    "topkv_crc64_noalloc": (_I32, [_P, _I64, _P, _P]),
    "topkv_move_layer": (_I32, [ctypes.POINTER(topkv_view_t), ctypes.POINTER(topkv_view_t), _I32, _P, _I32,
                                _I32, _P]),
    "topkv_move_layers": (_I32, [ctypes.POINTER(topkv_view_t), ctypes.POINTER(topkv_view_t), _I32, _I64, _I32, _P,
                                 _I32, _I32, _P]),
    "topkv_pack_layer_heads": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _I32, _I32, _P, _I64, _P]),
    "topkv_unpack_layer_heads": (_I32, [_P, _I64, _POOL, _I32, _I32, _P, _I32, _P, _I32, _I32, _P]),
    "topkv_reblock_layer": (_I32, [_POOL, _I32, _P, _I32, _POOL, _I32, _P, _I32, _I32, _P, _P]),
    "topkv_pack_layer_shards": (_I32, [_POOL, _I32, _I32, _P, _I32, _P, _I32, _I32, _I32, _P, _I64, _P]),
    "topkv_unpack_layer_shards": (_I32, [_P, _I64, _I32, _POOL, _I32, _I32, _P, _I32, _P, _I32, _I32, _P]),
    "topkv_packed_state_bytes": (_I64, [ctypes.POINTER(topkv_state_pool_t), _I32]),
    "topkv_pack_state_layer": (_I32, [ctypes.POINTER(topkv_state_pool_t), _I32, _I32, _P, _P, _I64,
                                      ctypes.POINTER(topkv_launch_t)]),
    "topkv_unpack_state_layer": (_I32, [_P, _I64, ctypes.POINTER(topkv_state_pool_t), _I32, _I32, _P,
                                        ctypes.POINTER(topkv_launch_t)]),
    "topkv_check_state_slots": (_I32, [ctypes.POINTER(topkv_state_pool_t), _I32, _P, _I32, _P, _I64, _P, _P]),
    "topkv_check_state_workspace_bytes": (_I64, [ctypes.POINTER(topkv_state_pool_t)]),
    "topkv_engine_pack_layers": (_I32, [_POOL, _I32, _I32, _I32, _P, _I32, _P, _P, _I64, _I64,
                                        ctypes.POINTER(topkv_engine_t), _P]),
    "topkv_engine_unpack_layers": (_I32, [_P, _I64, _I64, _POOL, _I32, _I32, _I32, _P, _I32, _P,
                                          ctypes.POINTER(topkv_engine_t), _P]),
    "topkv_engine_layers_per_grid": (_I32, [_I32, _I64, ctypes.POINTER(topkv_engine_t)]),
    "topkv_dma_create": (_I32, [ctypes.POINTER(_P)]),
    "topkv_dma_submit": (_I32, [_P, _P, _P, _P, _I64, ctypes.POINTER(_I64)]),
    "topkv_dma_wait": (_I32, [_P, _I64]),
    "topkv_dma_destroy": (_I32, [_P]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


class TopkvError(RuntimeError):
    def __init__(self, status: int):
        self.status = int(status)
        super().__init__(topkv_status_string(status))


def _check(status: int) -> None:
    if status != TOPKV_OK:
        raise TopkvError(status)


def _ptr(x) -> int:
    """Device address of a tensor (or an integer address / None)."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if isinstance(x, torch.Tensor):
        if x.numel() and not x.is_cuda:
            raise ValueError("tensor arguments must live in device memory")
        if x.numel() and not x.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
        return x.data_ptr()
    raise TypeError(f"expected a tensor or an address, got {type(x).__name__}")


def _table_ptr(t) -> int:
    if isinstance(t, torch.Tensor) and t.numel() and t.dtype != torch.int32:
        raise ValueError("block tables and seq_lens must be int32")
    return _ptr(t)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _nbytes(t, given) -> int:
    if given is not None:
        return int(given)
    if isinstance(t, torch.Tensor):
        return t.numel() * t.element_size()
    raise ValueError("byte capacity is required when passing a raw address")


def make_pool(base, *, num_pages, num_layers, page_size, planes, num_heads, head_dim,
              elem_bytes=2) -> topkv_pool_t:
    """Pool descriptor for device memory laid out
    [num_layers][num_pages][planes][page_size][num_heads][head_dim]."""
    return topkv_pool_t(_ptr(base), int(num_pages), int(num_layers), int(page_size), int(planes),
                        int(num_heads), int(head_dim), int(elem_bytes))


def pool_from_tensor(t: torch.Tensor) -> topkv_pool_t:
    """Descriptor of a 6-D pool tensor [layers][pages][planes][page_size][heads][dim]."""
    if t.dim() != 6:
        raise ValueError("pool tensor must be [layers][pages][planes][page_size][heads][dim]")
    L, NP, C, P, H, D = t.shape
    return make_pool(t, num_pages=NP, num_layers=L, page_size=P, planes=C, num_heads=H,
                     head_dim=D, elem_bytes=t.element_size())


def state_pool_from_tensor(t: torch.Tensor) -> topkv_state_pool_t:
    """Descriptor of a state cache tensor [layers][slots][words of one state]."""
    if t.dim() != 3:
        raise ValueError("state cache tensor must be [layers][slots][words]")
    L, NS, E = t.shape
    return topkv_state_pool_t(_ptr(t), int(NS), int(E) * t.element_size(), int(L), 0)


def _state_arg(pool) -> topkv_state_pool_t:
    return pool if isinstance(pool, topkv_state_pool_t) else state_pool_from_tensor(pool)


def _pool_arg(pool) -> topkv_pool_t:
    return pool if isinstance(pool, topkv_pool_t) else pool_from_tensor(pool)


def head_major_pool_from_tensor(t: torch.Tensor) -> topkv_pool_t:
    """Descriptor of a 6-D head-major pool tensor [layers][pages][planes][heads][page_size][dim]."""
    if t.dim() != 6:
        raise ValueError("head-major pool tensor must be [layers][pages][planes][heads][page_size][dim]")
    L, NP, C, H, P, D = t.shape
    return make_pool(t, num_pages=NP, num_layers=L, page_size=P, planes=C, num_heads=H,
                     head_dim=D, elem_bytes=t.element_size())


def pool_view(pool, layer, block_tables, bt_stride, head_begin=0, head_major=False) -> topkv_view_t:
    """A pool side of topkv_move_layer (a tensor in its layout, or a descriptor)."""
    if isinstance(pool, topkv_pool_t):
        desc = pool
    else:
        desc = head_major_pool_from_tensor(pool) if head_major else pool_from_tensor(pool)
    layout = TOPKV_LAYOUT_POOL_HEAD_MAJOR if head_major else TOPKV_LAYOUT_POOL
    return topkv_view_t(layout, int(layer), int(head_begin), int(bt_stride), _table_ptr(block_tables), desc, 0, 0,
                        0, 0)


def packed_view(buf, nbytes=None, shards=1) -> topkv_view_t:
    """A packed side of topkv_move_layer; with shards = S > 1, `nbytes` is each
    shard region's capacity (default: the buffer split in S)."""
    if nbytes is None and shards > 1:
        nbytes = _nbytes(buf, None) // int(shards)
    return topkv_view_t(TOPKV_LAYOUT_PACKED, 0, 0, 0, 0, topkv_pool_t(), _ptr(buf), _nbytes(buf, nbytes),
                        int(shards), 0)


def topkv_pack_layer(src, layer, block_table, seq_len, dst, stream=None) -> None:
    _check(_lib.topkv_pack_layer(ctypes.byref(_pool_arg(src)), int(layer), _table_ptr(block_table),
                                 int(seq_len), _ptr(dst), _stream(stream)))


def topkv_unpack_layer(src, dst, layer, block_table, seq_len, stream=None) -> None:
    _check(_lib.topkv_unpack_layer(_ptr(src), ctypes.byref(_pool_arg(dst)), int(layer),
                                   _table_ptr(block_table), int(seq_len), _stream(stream)))


def topkv_pack_layer_batched(src, layer, num_reqs, block_tables, bt_stride, seq_lens, dst,
                             dst_bytes=None, stream=None) -> None:
    _check(_lib.topkv_pack_layer_batched(ctypes.byref(_pool_arg(src)), int(layer), int(num_reqs),
                                         _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens),
                                         _ptr(dst), _nbytes(dst, dst_bytes), _stream(stream)))


def topkv_unpack_layer_batched(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens,
                               src_bytes=None, stream=None) -> None:
    _check(_lib.topkv_unpack_layer_batched(_ptr(src), _nbytes(src, src_bytes), ctypes.byref(_pool_arg(dst)),
                                           int(layer), int(num_reqs), _table_ptr(block_tables),
                                           int(bt_stride), _table_ptr(seq_lens), _stream(stream)))


def topkv_pack_layer_batched_ex(src, layer, num_reqs, block_tables, bt_stride, seq_lens, dst,
                                dst_bytes=None, stream=None, start=None, stop=None) -> None:
    """As topkv_pack_layer_batched; start/stop are raw hipEvent_t handles
    (see HipEvent) stamped with the kernel's own begin/end time."""
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    _check(_lib.topkv_pack_layer_batched_ex(ctypes.byref(_pool_arg(src)), int(layer), int(num_reqs),
                                            _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens),
                                            _ptr(dst), _nbytes(dst, dst_bytes), ctypes.byref(launch)))


def topkv_unpack_layer_batched_ex(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens,
                                  src_bytes=None, stream=None, start=None, stop=None) -> None:
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    _check(_lib.topkv_unpack_layer_batched_ex(_ptr(src), _nbytes(src, src_bytes), ctypes.byref(_pool_arg(dst)),
                                              int(layer), int(num_reqs), _table_ptr(block_tables),
                                              int(bt_stride), _table_ptr(seq_lens), ctypes.byref(launch)))


def topkv_pack_layer_window(src, layer, num_reqs, block_tables, bt_stride, seq_lens, window, dst,
                            dst_bytes=None, stream=None, start=None, stop=None) -> None:
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    _check(_lib.topkv_pack_layer_window(ctypes.byref(_pool_arg(src)), int(layer), int(num_reqs),
                                        _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens), int(window),
                                        _ptr(dst), _nbytes(dst, dst_bytes), ctypes.byref(launch)))


def topkv_unpack_layer_window(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, window,
                              src_bytes=None, stream=None, start=None, stop=None) -> None:
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    _check(_lib.topkv_unpack_layer_window(_ptr(src), _nbytes(src, src_bytes), ctypes.byref(_pool_arg(dst)),
                                          int(layer), int(num_reqs), _table_ptr(block_tables), int(bt_stride),
                                          _table_ptr(seq_lens), int(window), ctypes.byref(launch)))


def topkv_packed_window_bytes(pool, seq_lens_host, window) -> int:
    lens = [int(x) for x in seq_lens_host]
    arr = (_I32 * max(1, len(lens)))(*lens)
    return int(_lib.topkv_packed_window_bytes(ctypes.byref(_pool_arg(pool)), arr, len(lens), int(window)))


def topkv_pack_layer_planes(src, layer, block_table, seq_len, dst, plane_stride, dst_bytes=None, stream=None) -> None:
    _check(_lib.topkv_pack_layer_planes(ctypes.byref(_pool_arg(src)), int(layer), _table_ptr(block_table),
                                        int(seq_len), _ptr(dst), int(plane_stride), _nbytes(dst, dst_bytes),
                                        _stream(stream)))


def topkv_unpack_layer_planes(src, plane_stride, dst, layer, block_table, seq_len, src_bytes=None,
                              stream=None) -> None:
    _check(_lib.topkv_unpack_layer_planes(_ptr(src), int(plane_stride), _nbytes(src, src_bytes),
                                          ctypes.byref(_pool_arg(dst)), int(layer), _table_ptr(block_table),
                                          int(seq_len), _stream(stream)))


def topkv_kvcache1_bytes(geometry, seq_len) -> int:
    return int(_lib.topkv_kvcache1_bytes(ctypes.byref(_pool_arg(geometry)), int(seq_len)))


def topkv_kvcache1_workspace_bytes(geometry, seq_len) -> int:
    return int(_lib.topkv_kvcache1_workspace_bytes(ctypes.byref(_pool_arg(geometry)), int(seq_len)))


def topkv_kvcache1_pack_layer(src, layer, block_table, seq_len, blob, blob_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_pack_layer(ctypes.byref(_pool_arg(src)), int(layer), _table_ptr(block_table),
                                          int(seq_len), _ptr(blob), _nbytes(blob, blob_bytes), _stream(stream)))


def topkv_kvcache1_seal(geometry, seq_len, request_id, model_id, blob, workspace, blob_bytes=None,
                        workspace_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_seal(ctypes.byref(_pool_arg(geometry)), int(seq_len), int(request_id),
                                    int(model_id), _ptr(blob), _nbytes(blob, blob_bytes), _ptr(workspace),
                                    _nbytes(workspace, workspace_bytes), _stream(stream)))


def topkv_kvcache1_verify(geometry, seq_len, request_id, model_id, blob, workspace, result, blob_bytes=None,
                          workspace_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_verify(ctypes.byref(_pool_arg(geometry)), int(seq_len), int(request_id),
                                      int(model_id), _ptr(blob), _nbytes(blob, blob_bytes), _ptr(workspace),
                                      _nbytes(workspace, workspace_bytes), _table_ptr(result), _stream(stream)))


def topkv_kvcache1_pack_seal(src, block_table, seq_len, request_id, model_id, blob, workspace, blob_bytes=None,
                             workspace_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_pack_seal(ctypes.byref(_pool_arg(src)), _table_ptr(block_table), int(seq_len),
                                         int(request_id), int(model_id), _ptr(blob), _nbytes(blob, blob_bytes),
                                         _ptr(workspace), _nbytes(workspace, workspace_bytes), _stream(stream)))


def topkv_kvcache1_verify_unpack(blob, dst, block_table, seq_len, request_id, model_id, workspace, result,
                                 blob_bytes=None, workspace_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_verify_unpack(_ptr(blob), _nbytes(blob, blob_bytes), ctypes.byref(_pool_arg(dst)),
                                             _table_ptr(block_table), int(seq_len), int(request_id), int(model_id),
                                             _ptr(workspace), _nbytes(workspace, workspace_bytes),
                                             _table_ptr(result), _stream(stream)))


def topkv_kvcache1_unpack_layer(blob, dst, layer, block_table, seq_len, blob_bytes=None, stream=None) -> None:
    _check(_lib.topkv_kvcache1_unpack_layer(_ptr(blob), _nbytes(blob, blob_bytes), ctypes.byref(_pool_arg(dst)),
                                            int(layer), _table_ptr(block_table), int(seq_len), _stream(stream)))


def topkv_kvcache1_pack_layers(src, first_layer, num_layers, block_table, seq_len, blob, blob_bytes=None,
                               stream=None) -> None:
    _check(_lib.topkv_kvcache1_pack_layers(ctypes.byref(_pool_arg(src)), int(first_layer), int(num_layers),
                                           _table_ptr(block_table), int(seq_len), _ptr(blob),
                                           _nbytes(blob, blob_bytes), _stream(stream)))


def topkv_kvcache1_unpack_layers(blob, dst, first_layer, num_layers, block_table, seq_len, blob_bytes=None,
                                 stream=None) -> None:
    _check(_lib.topkv_kvcache1_unpack_layers(_ptr(blob), _nbytes(blob, blob_bytes), ctypes.byref(_pool_arg(dst)),
                                             int(first_layer), int(num_layers), _table_ptr(block_table),
                                             int(seq_len), _stream(stream)))


def topkv_crc64(data, nbytes, workspace, crc_out, workspace_bytes=None, stream=None) -> None:
    _check(_lib.topkv_crc64(_ptr(data), int(nbytes), _ptr(workspace), _nbytes(workspace, workspace_bytes),
                            _ptr(crc_out), _stream(stream)))


def topkv_crc64_noalloc(data, nbytes, crc_out, stream=None) -> None:
    _check(_lib.topkv_crc64_noalloc(_ptr(data), int(nbytes), _ptr(crc_out), _stream(stream)))


def topkv_crc64_workspace_bytes(nbytes) -> int:
    return int(_lib.topkv_crc64_workspace_bytes(int(nbytes)))


def topkv_packed_layer_bytes(pool, seq_lens_host) -> int:
    lens = [int(x) for x in seq_lens_host]
    arr = (_I32 * max(1, len(lens)))(*lens)
    return int(_lib.topkv_packed_layer_bytes(ctypes.byref(_pool_arg(pool)), arr, len(lens)))


def topkv_check_tables(pool, num_reqs, block_tables, bt_stride, seq_lens, check_duplicates, workspace,
                       result, workspace_bytes=None, stream=None) -> None:
    """Queue the device-side table check; `result` (device int32[4]) holds
    [status, entries out of range, repeated pages, lengths out of range]
    once the stream has synchronised."""
    ws_bytes = 0 if workspace is None else _nbytes(workspace, workspace_bytes)
    _check(_lib.topkv_check_tables(ctypes.byref(_pool_arg(pool)), int(num_reqs), _table_ptr(block_tables),
                                   int(bt_stride), _table_ptr(seq_lens), int(check_duplicates), _ptr(workspace),
                                   ws_bytes, _table_ptr(result), _stream(stream)))


def topkv_check_workspace_bytes(pool) -> int:
    return int(_lib.topkv_check_workspace_bytes(ctypes.byref(_pool_arg(pool))))


def topkv_status_string(status: int) -> str:
    return _lib.topkv_status_string(int(status)).decode()


# --- kernel-timestamp events for the *_ex calls ------------------------------
# Raw hipEvent_t handles from the HIP runtime that torch loaded (the same
# process-wide runtime libtopkv.so is bound to).
_hip = ctypes.CDLL("libamdhip64.so.7")
_hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
_hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
_hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
_hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
_hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]


class HipEvent:
    """A hipEvent_t (timing enabled) usable as start/stop of the *_ex calls."""

    def __init__(self):
        h = ctypes.c_void_p()
        if _hip.hipEventCreate(ctypes.byref(h)) != 0:
            raise RuntimeError("hipEventCreate failed")
        self.handle = h.value

    def record(self, stream=None):
        if _hip.hipEventRecord(self.handle, _stream(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def synchronize(self):
        if _hip.hipEventSynchronize(self.handle) != 0:
            raise RuntimeError("hipEventSynchronize failed")

    def elapsed_ms(self, end: "HipEvent") -> float:
        ms = ctypes.c_float()
        rc = _hip.hipEventElapsedTime(ctypes.byref(ms), self.handle, end.handle)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def __del__(self, _finalizing=sys.is_finalizing, _destroy=_hip.hipEventDestroy):
        h, self.handle = getattr(self, "handle", None), None
        if h and not _finalizing():
            _destroy(h)


# --- mapped host memory and the DMA layer shipper ----------------------------
_hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_uint]


def host_device_pointer(t: torch.Tensor) -> int:
    """Device address of pinned (hipHostMalloc'd) host memory, for kernels
    that write straight into it; raises for memory the device cannot map."""
    if t.is_cuda or not t.is_pinned():
        raise ValueError("expected a pinned host tensor")
    base = t.untyped_storage().data_ptr()     # the mapping is looked up for the allocation's start
    d = ctypes.c_void_p()
    rc = _hip.hipHostGetDevicePointer(ctypes.byref(d), ctypes.c_void_p(base), 0)
    if rc != 0 or not d.value:
        raise RuntimeError(f"hipHostGetDevicePointer failed ({rc}): host memory is not mapped")
    return int(d.value) + (t.data_ptr() - base)


def _any_ptr(x) -> int:
    """Address of device memory or of pinned host memory (the shipper's ends)."""
    if isinstance(x, torch.Tensor):
        if x.numel() and not (x.is_cuda or x.is_pinned()):
            raise ValueError("shipper buffers must be device memory or pinned host memory")
        if x.numel() and not x.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
        return x.data_ptr()
    return _ptr(x)


def topkv_move_layer(src: topkv_view_t, dst: topkv_view_t, num_reqs, seq_lens, head_count, window=0,
                     stream=None) -> None:
    _check(_lib.topkv_move_layer(ctypes.byref(src), ctypes.byref(dst), int(num_reqs), _table_ptr(seq_lens),
                                 int(head_count), int(window), _stream(stream)))


def topkv_move_layers(src: topkv_view_t, dst: topkv_view_t, num_layers, packed_layer_stride, num_reqs, seq_lens,
                      head_count, window=0, stream=None) -> None:
    _check(_lib.topkv_move_layers(ctypes.byref(src), ctypes.byref(dst), int(num_layers), int(packed_layer_stride),
                                  int(num_reqs), _table_ptr(seq_lens), int(head_count), int(window), _stream(stream)))


def topkv_pack_layer_heads(src, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count, dst,
                           dst_bytes=None, stream=None) -> None:
    _check(_lib.topkv_pack_layer_heads(ctypes.byref(_pool_arg(src)), int(layer), int(num_reqs),
                                       _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens),
                                       int(head_begin), int(head_count), _ptr(dst), _nbytes(dst, dst_bytes),
                                       _stream(stream)))


def topkv_unpack_layer_heads(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count,
                             src_bytes=None, stream=None) -> None:
    _check(_lib.topkv_unpack_layer_heads(_ptr(src), _nbytes(src, src_bytes), ctypes.byref(_pool_arg(dst)),
                                         int(layer), int(num_reqs), _table_ptr(block_tables), int(bt_stride),
                                         _table_ptr(seq_lens), int(head_begin), int(head_count), _stream(stream)))


def topkv_pack_layer_shards(src, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count, shards,
                            dst, shard_bytes=None, stream=None) -> None:
    if shard_bytes is None:
        shard_bytes = _nbytes(dst, None) // int(shards)
    _check(_lib.topkv_pack_layer_shards(ctypes.byref(_pool_arg(src)), int(layer), int(num_reqs),
                                        _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens),
                                        int(head_begin), int(head_count), int(shards), _ptr(dst), int(shard_bytes),
                                        _stream(stream)))


def topkv_unpack_layer_shards(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count,
                              shards, shard_bytes=None, stream=None) -> None:
    if shard_bytes is None:
        shard_bytes = _nbytes(src, None) // int(shards)
    _check(_lib.topkv_unpack_layer_shards(_ptr(src), int(shard_bytes), int(shards), ctypes.byref(_pool_arg(dst)),
                                          int(layer), int(num_reqs), _table_ptr(block_tables), int(bt_stride),
                                          _table_ptr(seq_lens), int(head_begin), int(head_count), _stream(stream)))


def topkv_reblock_layer(src, src_layer, src_tables, src_stride, dst, dst_layer, dst_tables, dst_stride, num_reqs,
                        seq_lens, stream=None) -> None:
    _check(_lib.topkv_reblock_layer(ctypes.byref(_pool_arg(src)), int(src_layer), _table_ptr(src_tables),
                                    int(src_stride), ctypes.byref(_pool_arg(dst)), int(dst_layer),
                                    _table_ptr(dst_tables), int(dst_stride), int(num_reqs), _table_ptr(seq_lens),
                                    _stream(stream)))


def topkv_dma_create() -> int:
    h = _P()
    _check(_lib.topkv_dma_create(ctypes.byref(h)))
    return int(h.value)


def topkv_dma_submit(dma, ready, dst, src, nbytes=None) -> int:
    """Queue a DMA copy src -> dst that starts once `ready` (a recorded
    HipEvent / torch.cuda.Event / raw handle / None) has completed; returns
    the ticket."""
    t = _I64()
    n = _nbytes(src, nbytes)
    _check(_lib.topkv_dma_submit(_P(int(dma)), _P(_event(ready)), _P(_any_ptr(dst)), _P(_any_ptr(src)),
                                 n, ctypes.byref(t)))
    return int(t.value)


def topkv_dma_wait(dma, ticket) -> None:
    _check(_lib.topkv_dma_wait(_P(int(dma)), int(ticket)))


def topkv_dma_destroy(dma) -> None:
    _check(_lib.topkv_dma_destroy(_P(int(dma))))


def _event(e) -> int:
    if e is None:
        return 0
    if isinstance(e, HipEvent):
        return e.handle
    if isinstance(e, torch.cuda.Event):
        return int(e.cuda_event)
    return int(e)


# --- prepared calls -----------------------------------------------------------
class PreparedCall:
    """One C entry point with its arguments converted to ctypes once.
    Calling it re-issues exactly that launch; per-layer sweeps use these so
    the host enqueue rate, not ctypes conversion, bounds the launch rate."""

    def __init__(self, name, args, keep):
        self._fn = getattr(_lib, name)
        self._args = args
        self._keep = keep          # structs the arguments point to

    def __call__(self) -> None:
        st = self._fn(*self._args)
        if st:
            raise TopkvError(st)


def prepare_pack_layer_window(src, layer, num_reqs, block_tables, bt_stride, seq_lens, window, dst,
                              dst_bytes=None, stream=None, start=None, stop=None) -> PreparedCall:
    pool = _pool_arg(src)
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    args = (ctypes.byref(pool), _I32(int(layer)), _I32(int(num_reqs)), _P(_table_ptr(block_tables)),
            _I32(int(bt_stride)), _P(_table_ptr(seq_lens)), _I32(int(window)), _P(_ptr(dst)),
            _I64(_nbytes(dst, dst_bytes)), ctypes.byref(launch))
    return PreparedCall("topkv_pack_layer_window", args, (pool, launch))


def prepare_unpack_layer_window(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, window,
                                src_bytes=None, stream=None, start=None, stop=None) -> PreparedCall:
    pool = _pool_arg(dst)
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    args = (_P(_ptr(src)), _I64(_nbytes(src, src_bytes)), ctypes.byref(pool), _I32(int(layer)),
            _I32(int(num_reqs)), _P(_table_ptr(block_tables)), _I32(int(bt_stride)), _P(_table_ptr(seq_lens)),
            _I32(int(window)), ctypes.byref(launch))
    return PreparedCall("topkv_unpack_layer_window", args, (pool, launch))


def prepare_pack_layer_batched_ex(src, layer, num_reqs, block_tables, bt_stride, seq_lens, dst,
                                  dst_bytes=None, stream=None, start=None, stop=None) -> PreparedCall:
    return prepare_pack_layer_window(src, layer, num_reqs, block_tables, bt_stride, seq_lens, 0, dst,
                                     dst_bytes, stream, start, stop)


def prepare_unpack_layer_batched_ex(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens,
                                    src_bytes=None, stream=None, start=None, stop=None) -> PreparedCall:
    return prepare_unpack_layer_window(src, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, 0,
                                       src_bytes, stream, start, stop)


def prepare_pack_layer_heads(src, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count, dst,
                             dst_bytes=None, stream=None) -> PreparedCall:
    pool = _pool_arg(src)
    args = (ctypes.byref(pool), _I32(int(layer)), _I32(int(num_reqs)), _P(_table_ptr(block_tables)),
            _I32(int(bt_stride)), _P(_table_ptr(seq_lens)), _I32(int(head_begin)), _I32(int(head_count)),
            _P(_ptr(dst)), _I64(_nbytes(dst, dst_bytes)), _P(_stream(stream)))
    return PreparedCall("topkv_pack_layer_heads", args, (pool,))


def prepare_move_layers(src: topkv_view_t, dst: topkv_view_t, num_layers, packed_layer_stride, num_reqs, seq_lens,
                        head_count, window=0, stream=None) -> PreparedCall:
    args = (ctypes.byref(src), ctypes.byref(dst), _I32(int(num_layers)), _I64(int(packed_layer_stride)),
            _I32(int(num_reqs)), _P(_table_ptr(seq_lens)), _I32(int(head_count)), _I32(int(window)),
            _P(_stream(stream)))
    return PreparedCall("topkv_move_layers", args, (src, dst))


def prepare_move_layer(src: topkv_view_t, dst: topkv_view_t, num_reqs, seq_lens, head_count, window=0,
                       stream=None) -> PreparedCall:
    args = (ctypes.byref(src), ctypes.byref(dst), _I32(int(num_reqs)), _P(_table_ptr(seq_lens)),
            _I32(int(head_count)), _I32(int(window)), _P(_stream(stream)))
    return PreparedCall("topkv_move_layer", args, (src, dst))


def prepare_pack_layer_shards(src, layer, num_reqs, block_tables, bt_stride, seq_lens, head_begin, head_count, shards,
                              dst, shard_bytes=None, stream=None) -> PreparedCall:
    pool = _pool_arg(src)
    if shard_bytes is None:
        shard_bytes = _nbytes(dst, None) // int(shards)
    args = (ctypes.byref(pool), _I32(int(layer)), _I32(int(num_reqs)), _P(_table_ptr(block_tables)),
            _I32(int(bt_stride)), _P(_table_ptr(seq_lens)), _I32(int(head_begin)), _I32(int(head_count)),
            _I32(int(shards)), _P(_ptr(dst)), _I64(int(shard_bytes)), _P(_stream(stream)))
    return PreparedCall("topkv_pack_layer_shards", args, (pool,))


# --- layer engine ----------------------------------------------------------------

def _word_ptr(x) -> int:
    """Address of a ready / cancel word array: device memory, or pinned host
    memory mapped for the device."""
    if isinstance(x, torch.Tensor) and not x.is_cuda:
        return host_device_pointer(x) if x.numel() else 0
    return _ptr(x)


def engine_options(ready=None, epoch=0, status=None, cancel=None, timeout_us=0, workgroups_per_cu=0,
                   layers_per_grid=0) -> topkv_engine_t:
    """topkv_engine_t for the engine calls: ready / cancel are int32 words in
    device memory or pinned host memory (or addresses), status a device
    int32 holding 0 at launch."""
    return topkv_engine_t(_word_ptr(ready), _word_ptr(cancel), _ptr(status), ctypes.c_uint32(int(epoch) & 0xffffffff),
                          int(workgroups_per_cu), int(timeout_us), int(layers_per_grid))


def topkv_engine_layers_per_grid(num_layers, layer_stride, engine=None) -> int:
    """Layers per hardware-dispatched grid of an engine call without waits
    (host-only)."""
    n = _lib.topkv_engine_layers_per_grid(int(num_layers), int(layer_stride), _engine_arg(engine))
    if n < 0:
        raise TopkvError(TOPKV_ERR_INVALID_ARG)
    return n


def _engine_arg(engine):
    return ctypes.byref(engine) if engine is not None else None


def topkv_engine_pack_layers(src, first_layer, num_layers, num_reqs, block_tables, bt_stride, seq_lens, packed,
                             layer_stride, packed_bytes=None, engine=None, stream=None) -> None:
    _check(_lib.topkv_engine_pack_layers(ctypes.byref(_pool_arg(src)), int(first_layer), int(num_layers),
                                         int(num_reqs), _table_ptr(block_tables), int(bt_stride), _table_ptr(seq_lens),
                                         _ptr(packed), int(layer_stride), _nbytes(packed, packed_bytes),
                                         _engine_arg(engine), _stream(stream)))


def topkv_engine_unpack_layers(packed, layer_stride, dst, first_layer, num_layers, num_reqs, block_tables, bt_stride,
                               seq_lens, packed_bytes=None, engine=None, stream=None) -> None:
    _check(_lib.topkv_engine_unpack_layers(_ptr(packed), int(layer_stride), _nbytes(packed, packed_bytes),
                                           ctypes.byref(_pool_arg(dst)), int(first_layer), int(num_layers),
                                           int(num_reqs), _table_ptr(block_tables), int(bt_stride),
                                           _table_ptr(seq_lens), _engine_arg(engine), _stream(stream)))


def prepare_engine_pack_layers(src, first_layer, num_layers, num_reqs, block_tables, bt_stride, seq_lens, packed,
                               layer_stride, packed_bytes=None, engine=None, stream=None) -> PreparedCall:
    pool = _pool_arg(src)
    args = (ctypes.byref(pool), _I32(int(first_layer)), _I32(int(num_layers)), _I32(int(num_reqs)),
            _P(_table_ptr(block_tables)), _I32(int(bt_stride)), _P(_table_ptr(seq_lens)), _P(_ptr(packed)),
            _I64(int(layer_stride)), _I64(_nbytes(packed, packed_bytes)), _engine_arg(engine), _P(_stream(stream)))
    return PreparedCall("topkv_engine_pack_layers", args, (pool, engine))


def prepare_engine_unpack_layers(packed, layer_stride, dst, first_layer, num_layers, num_reqs, block_tables,
                                 bt_stride, seq_lens, packed_bytes=None, engine=None, stream=None) -> PreparedCall:
    pool = _pool_arg(dst)
    args = (_P(_ptr(packed)), _I64(int(layer_stride)), _I64(_nbytes(packed, packed_bytes)), ctypes.byref(pool),
            _I32(int(first_layer)), _I32(int(num_layers)), _I32(int(num_reqs)), _P(_table_ptr(block_tables)),
            _I32(int(bt_stride)), _P(_table_ptr(seq_lens)), _engine_arg(engine), _P(_stream(stream)))
    return PreparedCall("topkv_engine_unpack_layers", args, (pool, engine))


# --- fixed-state layers ---------------------------------------------------------

def topkv_packed_state_bytes(pool, num_reqs) -> int:
    n = _lib.topkv_packed_state_bytes(ctypes.byref(_state_arg(pool)), int(num_reqs))
    if n < 0:
        raise TopkvError(TOPKV_ERR_INVALID_ARG)
    return n


def prepare_pack_state_layer(src, layer, num_reqs, slots, dst, dst_bytes=None, stream=None, start=None,
                             stop=None) -> PreparedCall:
    pool = _state_arg(src)
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    args = (ctypes.byref(pool), _I32(int(layer)), _I32(int(num_reqs)), _P(_table_ptr(slots)), _P(_ptr(dst)),
            _I64(_nbytes(dst, dst_bytes)), ctypes.byref(launch))
    return PreparedCall("topkv_pack_state_layer", args, (pool, launch))


def prepare_unpack_state_layer(src, dst, layer, num_reqs, slots, src_bytes=None, stream=None, start=None,
                               stop=None) -> PreparedCall:
    pool = _state_arg(dst)
    launch = topkv_launch_t(_stream(stream), _event(start), _event(stop))
    args = (_P(_ptr(src)), _I64(_nbytes(src, src_bytes)), ctypes.byref(pool), _I32(int(layer)),
            _I32(int(num_reqs)), _P(_table_ptr(slots)), ctypes.byref(launch))
    return PreparedCall("topkv_unpack_state_layer", args, (pool, launch))


def topkv_pack_state_layer(src, layer, num_reqs, slots, dst, dst_bytes=None, stream=None, start=None,
                           stop=None) -> None:
    """Pack the fixed states of num_reqs requests (slot slots[r]) of one layer."""
    prepare_pack_state_layer(src, layer, num_reqs, slots, dst, dst_bytes, stream, start, stop)()


def topkv_unpack_state_layer(src, dst, layer, num_reqs, slots, src_bytes=None, stream=None, start=None,
                             stop=None) -> None:
    """Unpack num_reqs packed states into slots slots[r] of one layer."""
    prepare_unpack_state_layer(src, dst, layer, num_reqs, slots, src_bytes, stream, start, stop)()


def topkv_check_state_workspace_bytes(pool) -> int:
    return int(_lib.topkv_check_state_workspace_bytes(ctypes.byref(_state_arg(pool))))


def topkv_check_state_slots(pool, num_reqs, slots, result, check_duplicates=True, workspace=None,
                            workspace_bytes=None, stream=None) -> None:
    """Queue the slot check; result (device int32[4]) holds [status, out of
    range, repeated, 0] once the stream has synchronised."""
    wsb = 0 if workspace is None else _nbytes(workspace, workspace_bytes)
    _check(_lib.topkv_check_state_slots(ctypes.byref(_state_arg(pool)), int(num_reqs), _table_ptr(slots),
                                        int(bool(check_duplicates)), _ptr(workspace), wsb, _ptr(result),
                                        _stream(stream)))

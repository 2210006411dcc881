"""The C-ABI library on the CPU: it loads, exports every entry point declared in
include/topkv.h, and its host-side logic (sizes, status strings, argument
validation) behaves as documented.  No call here gets past validation, so
nothing is launched and no GPU is needed."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "topkv.h")


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd.build import LIBRARY, build_library
    if not os.path.exists(LIBRARY):
        build_library()
    from paper_2607_28633_amd import topkv
    return topkv


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(topkv_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_binding_names(tk):
    assert declared_functions() == sorted(tk.EXPORTS)


def test_library_exports_every_declared_symbol(tk):
    lib = ctypes.CDLL(tk.LIBRARY)
    missing = [name for name in declared_functions() if not hasattr(lib, name)]
    assert not missing, f"not exported: {missing}"


def test_status_strings(tk):
    for code in range(9):
        s = tk.topkv_status_string(code)
        assert s.startswith("TOPKV_")
    assert tk.topkv_status_string(99) == "TOPKV_ERR_UNKNOWN"


def _pool(tk, **kw):
    g = dict(num_pages=64, num_layers=2, page_size=16, planes=2, num_heads=8, head_dim=128, elem_bytes=2)
    g.update(kw)
    return tk.make_pool(kw.pop("base", 0x10000), **{k: v for k, v in g.items() if k != "base"})


def test_packed_layer_bytes_matches_eq1(tk):
    from paper_2607_28633_amd.workloads import make_workload
    for name in ("tiny", "llama3-8b", "llama3-70b-batch8", "deepseek-v3-mla", "reblock-70b"):
        wl = make_workload(name)
        pool = tk.make_pool(0x10000, num_pages=wl.num_pages, num_layers=wl.num_layers,
                            page_size=wl.page_size, planes=wl.planes, num_heads=wl.num_heads,
                            head_dim=wl.head_dim, elem_bytes=wl.elem_bytes)
        s = int(wl.seq_lens.astype(np.int64).sum())
        # Eq. 1 per layer: planes * h_kv * d_h * s * b_p (planes = 2, or 1 for MLA)
        assert tk.topkv_packed_layer_bytes(pool, wl.seq_lens) == \
            wl.planes * wl.num_heads * wl.head_dim * s * wl.elem_bytes
    # the 70B / 4096-token figure of Table 1 over 80 layers
    assert 80 * tk.topkv_packed_layer_bytes(_pool(tk), [4096]) == 1_342_177_280
    assert tk.topkv_packed_layer_bytes(_pool(tk), []) == 0
    assert tk.topkv_packed_layer_bytes(_pool(tk), [5, -1]) == -1
    lib = ctypes.CDLL(tk.LIBRARY)
    lib.topkv_packed_layer_bytes.restype = ctypes.c_int64
    assert lib.topkv_packed_layer_bytes(None, None, 0) == -1


def _expect(tk, code, fn, *args, **kw):
    kw.setdefault("stream", 0)   # the null stream handle: no torch device query on a GPU-less host
    with pytest.raises(tk.TopkvError) as ei:
        fn(*args, **kw)
    assert ei.value.status == code, tk.topkv_status_string(ei.value.status)


def test_argument_validation_before_launch(tk):
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    bt, lens, buf = 0x20000, 0x30000, 0x40000
    good = _pool(tk)
    _expect(tk, INV, tk.topkv_pack_layer, _pool(tk, base=0), 0, bt, 16, buf)          # null base
    _expect(tk, INV, tk.topkv_pack_layer, good, 2, bt, 16, buf)                       # layer >= L
    _expect(tk, INV, tk.topkv_pack_layer, good, -1, bt, 16, buf)
    _expect(tk, INV, tk.topkv_pack_layer, _pool(tk, elem_bytes=3), 0, bt, 16, buf)
    _expect(tk, INV, tk.topkv_pack_layer, _pool(tk, head_dim=0), 0, bt, 16, buf)
    _expect(tk, INV, tk.topkv_pack_layer, _pool(tk, page_size=-4), 0, bt, 16, buf)
    _expect(tk, INV, tk.topkv_pack_layer, good, 0, bt, -1, buf)                       # negative length
    _expect(tk, INV, tk.topkv_pack_layer, good, 0, 0, 16, buf)                        # null table
    _expect(tk, INV, tk.topkv_unpack_layer, 0, good, 0, bt, 16)                       # null packed src
    _expect(tk, INV, tk.topkv_pack_layer_batched, good, 0, -1, bt, 4, lens, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_pack_layer_batched, good, 0, 3, bt, 0, lens, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_pack_layer_batched, good, 0, 3, bt, 4, 0, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_unpack_layer_batched, buf, good, 0, 3, bt, 4, lens, src_bytes=-1)
    _expect(tk, UNS, tk.topkv_pack_layer_batched, good, 0, tk.TOPKV_MAX_BATCH_REQS + 1, bt, 4, lens,
            buf, dst_bytes=1 << 20)
    _expect(tk, UNS, tk.topkv_pack_layer, _pool(tk, num_pages=1 << 40, num_layers=1 << 20), 0, bt, 16, buf)


def test_empty_work_is_a_no_op(tk):
    good = _pool(tk)
    tk.topkv_pack_layer(good, 0, 0, 0, 0, stream=0)            # zero tokens: nothing to launch
    tk.topkv_unpack_layer(0, good, 1, 0, 0, stream=0)
    tk.topkv_pack_layer_batched(good, 0, 0, 0, 1, 0, 0, dst_bytes=0, stream=0)
    tk.topkv_unpack_layer_batched(0, good, 0, 0, 0, 1, 0, src_bytes=0, stream=0)


def test_engine_validation(tk):
    """The layer engine refuses bad ranges, strides and wait options before
    any runtime call; an empty batch launches nothing."""
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    bt, lens, buf, ready, status = 0x20000, 0x30000, 0x40000, 0x50000, 0x60000
    good = _pool(tk)                     # 2 layers
    stride = 1 << 20
    pk, up = tk.topkv_engine_pack_layers, tk.topkv_engine_unpack_layers
    for first, count in ((-1, 1), (0, 3), (1, 2), (2, 1), (0, 0)):
        _expect(tk, INV, pk, good, first, count, 2, bt, 4, lens, buf, stride, packed_bytes=2 * stride)
        _expect(tk, INV, up, buf, stride, good, first, count, 2, bt, 4, lens, packed_bytes=2 * stride)
    _expect(tk, INV, pk, good, 0, 2, 2, bt, 4, lens, buf, 0, packed_bytes=2 * stride)           # no layer stride
    _expect(tk, INV, pk, good, 0, 2, 2, bt, 4, lens, buf, stride, packed_bytes=stride - 1)       # last block outside
    _expect(tk, INV, pk, good, 0, 2, 2, bt, 4, lens, buf, -stride, packed_bytes=2 * stride)
    _expect(tk, INV, pk, good, 0, 2, -1, bt, 4, lens, buf, stride, packed_bytes=2 * stride)
    _expect(tk, INV, pk, good, 0, 2, 2, 0, 4, lens, buf, stride, packed_bytes=2 * stride)        # null tables
    _expect(tk, INV, pk, good, 0, 2, 2, bt, 4, 0, buf, stride, packed_bytes=2 * stride)          # null lengths
    _expect(tk, INV, pk, good, 0, 2, 2, bt, 0, lens, buf, stride, packed_bytes=2 * stride)
    _expect(tk, INV, up, 0, stride, good, 0, 2, 2, bt, 4, lens, packed_bytes=2 * stride)         # null packed
    _expect(tk, UNS, pk, good, 0, 2, tk.TOPKV_MAX_BATCH_REQS + 1, bt, 4, lens, buf, stride, packed_bytes=2 * stride)
    _expect(tk, UNS, pk, good, 0, 2, 4096, bt, 1 << 20, lens, buf, stride, packed_bytes=2 * stride)  # 2^31 items
    for opt in (tk.engine_options(ready=ready, status=0, timeout_us=1000),          # ready without status
                tk.engine_options(ready=ready, status=status, timeout_us=0),         # no timeout
                tk.engine_options(ready=ready, status=status, timeout_us=60_000_001),
                tk.engine_options(workgroups_per_cu=-1), tk.engine_options(workgroups_per_cu=65),
                tk.engine_options(layers_per_grid=-1)):
        _expect(tk, INV, pk, good, 0, 2, 2, bt, 4, lens, buf, stride, packed_bytes=2 * stride, engine=opt)
        _expect(tk, INV, up, buf, stride, good, 0, 2, 2, bt, 4, lens, packed_bytes=2 * stride, engine=opt)
    # no requests: nothing to launch, whatever the wait options
    pk(good, 0, 2, 0, 0, 1, 0, 0, stride, packed_bytes=2 * stride,
       engine=tk.engine_options(ready=ready, status=status, timeout_us=1000), stream=0)
    up(0, stride, good, 1, 1, 0, 0, 1, 0, packed_bytes=0, stream=0)


def test_engine_layers_per_grid(tk):
    """The engine's split of a range into hardware-dispatched grids: about
    512 MiB of packed blocks per grid in grids of equal layer count (rounded
    up), or the caller's count capped at the range."""
    f = tk.topkv_engine_layers_per_grid
    mib = 1 << 20
    assert f(80, 16 * mib) == 27                  # 1280 MiB: 3 grids of 27, 27, 26 layers
    assert f(80, 139685888) == 4                  # the 70B batch of 8: 21 grids
    assert f(61, 204800000) == 3                  # 200 MB layers: 23 grids
    assert f(32, 16 * mib) == 32                  # exactly 512 MiB: one grid
    assert f(33, 16 * mib) == 17                  # just past it: two grids
    assert f(8, 5 << 30) == 1                     # layers past the target: one each
    assert f(1, 0) == 1 and f(5, 0) == 5          # no stride: one grid
    assert f(3, 1 << 62) == 1                     # the product overflows int64: one layer per grid
    assert f(7, 16 * mib, tk.engine_options(layers_per_grid=3)) == 3
    assert f(7, 16 * mib, tk.engine_options(layers_per_grid=9)) == 7
    assert f(7, 16 * mib, tk.engine_options()) == 7
    for bad in ((0, mib, None), (2, -1, None), (2, mib, tk.engine_options(layers_per_grid=-1))):
        with pytest.raises(tk.TopkvError):
            f(*bad)


def test_check_tables_validation(tk):
    INV = tk.TOPKV_ERR_INVALID_ARG
    good = _pool(tk)
    bt, lens, ws, res = 0x20000, 0x30000, 0x40000, 0x50000
    assert tk.topkv_check_workspace_bytes(good) == 64 // 32 * 4
    assert tk.topkv_check_workspace_bytes(_pool(tk, num_pages=33)) == 8
    assert tk.topkv_check_workspace_bytes(_pool(tk, num_pages=0)) == -1
    _expect(tk, INV, tk.topkv_check_tables, good, 2, bt, 4, lens, 1, ws, 0, workspace_bytes=8)      # null result
    _expect(tk, INV, tk.topkv_check_tables, good, 2, bt, 4, lens, 1, 0, res, workspace_bytes=8)     # no workspace
    _expect(tk, INV, tk.topkv_check_tables, good, 2, bt, 4, lens, 1, ws, res, workspace_bytes=4)    # too small
    _expect(tk, INV, tk.topkv_check_tables, good, 2, 0, 4, lens, 0, None, res)                      # null tables
    _expect(tk, INV, tk.topkv_check_tables, good, -1, bt, 4, lens, 0, None, res)
    _expect(tk, INV, tk.topkv_check_tables, _pool(tk, page_size=0), 2, bt, 4, lens, 0, None, res)


def test_dma_shipper_validation(tk):
    """Null handles and bad sizes are refused before any runtime call."""
    INV = tk.TOPKV_ERR_INVALID_ARG
    lib, P, I64 = tk._lib, ctypes.c_void_p, ctypes.c_int64
    t = I64(-7)
    assert lib.topkv_dma_create(None) == INV
    assert lib.topkv_dma_submit(None, None, P(0x1000), P(0x2000), 16, ctypes.byref(t)) == INV
    assert lib.topkv_dma_wait(None, 1) == INV
    assert lib.topkv_dma_destroy(None) == INV
    assert t.value == -7


def test_move_layer_validation(tk):
    """Layout moves refuse bad views and arguments before any launch."""
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    bt, lens, buf = 0x20000, 0x30000, 0x40000
    good = _pool(tk)
    pv = tk.pool_view(good, 1, bt, 4)
    pk = tk.packed_view(buf, 1 << 20)
    _expect(tk, INV, tk.topkv_move_layer, pk, tk.packed_view(buf + 64, 1 << 20), 2, lens, 8)   # no pool side
    bad = tk.pool_view(good, 1, bt, 4)
    bad.layout = 7
    _expect(tk, INV, tk.topkv_move_layer, bad, pk, 2, lens, 8)
    _expect(tk, INV, tk.topkv_move_layer, pv, pk, 2, lens, 0)                  # head_count 0
    _expect(tk, INV, tk.topkv_move_layer, tk.pool_view(good, 1, bt, 4, head_begin=5), pk, 2, lens, 4)
    _expect(tk, INV, tk.topkv_move_layer, tk.pool_view(good, 2, bt, 4), pk, 2, lens, 8)   # layer >= L
    _expect(tk, INV, tk.topkv_move_layer, tk.pool_view(good, 1, bt, 0), pk, 2, lens, 8)   # bt_stride 0
    _expect(tk, INV, tk.topkv_move_layer, tk.pool_view(good, 1, 0, 4), pk, 2, lens, 8)    # null tables
    _expect(tk, INV, tk.topkv_move_layer, pv, pk, 2, 0, 8)                     # null lengths
    _expect(tk, INV, tk.topkv_move_layer, pv, pk, 2, lens, 8, window=-1)
    _expect(tk, INV, tk.topkv_move_layer, pv, tk.packed_view(0, 64), 2, lens, 8)         # null packed data
    _expect(tk, INV, tk.topkv_move_layer, pv, tk.pool_view(_pool(tk, base=0x900000, planes=1), 0, bt, 4),
            2, lens, 8)                                                        # planes differ
    _expect(tk, UNS, tk.topkv_move_layer, pv, pk, tk.TOPKV_MAX_BATCH_REQS + 1, lens, 8)
    _expect(tk, UNS, tk.topkv_move_layer, tk.pool_view(good, 1, bt, 1 << 20), pk, 4096, lens, 8)  # 2^31 pieces
    _expect(tk, INV, tk.topkv_pack_layer_heads, good, 1, 2, bt, 4, lens, 6, 3, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_unpack_layer_heads, buf, good, 1, 2, bt, 4, lens, -1, 2, src_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_reblock_layer, good, 0, bt, 4, _pool(tk, base=0x900000, num_heads=4), 0, bt, 4,
            2, lens)
    _expect(tk, INV, tk.topkv_move_layer, pv, tk.packed_view(buf, 1 << 20, shards=3), 2, lens, 8)  # 3 does not divide 8
    _expect(tk, INV, tk.topkv_move_layer, pv, tk.packed_view(buf, 1 << 20, shards=-2), 2, lens, 8)
    _expect(tk, INV, tk.topkv_pack_layer_shards, good, 1, 2, bt, 4, lens, 0, 8, 0, buf, shard_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_unpack_layer_shards, buf, good, 1, 2, bt, 4, lens, 0, 6, 4, shard_bytes=1 << 20)
    tk.topkv_move_layer(pv, pk, 0, 0, 8, stream=0)                             # no requests: nothing to launch
    # layer ranges: a pool side's layers past the pool, negative counts or strides, overlapping packed layers
    p0 = tk.pool_view(good, 0, bt, 4)
    mv = tk.topkv_move_layers
    _expect(tk, INV, mv, p0, pk, -1, 1 << 20, 2, lens, 8)
    _expect(tk, INV, mv, p0, pk, 2, -1, 2, lens, 8)
    _expect(tk, INV, mv, pv, pk, 2, 1 << 20, 2, lens, 8)                       # layers 1..2 of a 2-layer pool
    _expect(tk, INV, mv, p0, pk, 2, (1 << 20) - 16, 2, lens, 8)                # layer 1 would overlap layer 0
    _expect(tk, INV, mv, p0, tk.packed_view(buf, 1 << 20, shards=2), 2, 1 << 20, 2, lens, 8)   # two regions
    _expect(tk, INV, mv, pk, p0, 2, (1 << 20) - 16, 2, lens, 8)
    _expect(tk, INV, mv, bad, pk, 2, 1 << 20, 2, lens, 8)
    _expect(tk, INV, mv, p0, pk, 2, 1 << 20, 2, lens, 0)                       # head_count 0
    _expect(tk, INV, mv, p0, tk.pool_view(_pool(tk, base=0x900000), 1, bt, 4), 2, 0, 2, lens, 8)  # dst layers 1..2
    p4 = tk.pool_view(_pool(tk, num_layers=4), 0, bt, 4)
    _expect(tk, INV, mv, p4, pk, 4, 1 << 62, 2, lens, 8)                       # 3 * stride overflows int64
    mv(p0, pk, 2, 1 << 20, 0, 0, 8, stream=0)                                  # no requests: nothing to launch
    mv(p0, pk, 0, 0, 2, lens, 8, stream=0)                                     # no layers: nothing to launch


def test_state_layer_validation(tk):
    """Fixed-state layers: sizes on the host, bad descriptors and arguments
    refused before any launch, an empty batch launches nothing."""
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    slots, buf = 0x20000, 0x40000

    def st(**kw):
        g = dict(base=0x10000, num_slots=5, state_bytes=1000, num_layers=3, reserved=0)
        g.update(kw)
        return tk.topkv_state_pool_t(g["base"], g["num_slots"], g["state_bytes"], g["num_layers"], g["reserved"])

    lib = tk._lib
    assert tk.topkv_packed_state_bytes(st(), 7) == 7000
    assert tk.topkv_packed_state_bytes(st(), 0) == 0
    for bad in (st(base=0), st(num_slots=0), st(state_bytes=0), st(num_layers=0), st(reserved=1),
                st(num_slots=1 << 40, state_bytes=1 << 30)):
        assert lib.topkv_packed_state_bytes(ctypes.byref(bad), 1) == -1
    assert lib.topkv_packed_state_bytes(ctypes.byref(st()), -1) == -1
    good = st()
    _expect(tk, INV, tk.topkv_pack_state_layer, good, 3, 2, slots, buf, dst_bytes=1 << 20)     # layer >= L
    _expect(tk, INV, tk.topkv_pack_state_layer, good, -1, 2, slots, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_pack_state_layer, good, 0, -1, slots, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_pack_state_layer, good, 0, 2, 0, buf, dst_bytes=1 << 20)         # null slots
    _expect(tk, INV, tk.topkv_pack_state_layer, good, 0, 2, slots, 0, dst_bytes=1 << 20)       # null dst
    _expect(tk, INV, tk.topkv_pack_state_layer, good, 0, 2, slots, buf, dst_bytes=1999)        # one byte short
    _expect(tk, INV, tk.topkv_pack_state_layer, st(reserved=3), 0, 2, slots, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_unpack_state_layer, buf, good, 1, 3, slots, src_bytes=2999)
    _expect(tk, INV, tk.topkv_unpack_state_layer, 0, good, 1, 3, slots, src_bytes=3000)
    huge = st(num_slots=1, num_layers=1, state_bytes=1 << 50)
    _expect(tk, UNS, tk.topkv_pack_state_layer, huge, 0, 1, slots, buf, dst_bytes=1 << 50)    # 2^35 tiles
    res, ws = 0x50000, 0x60000
    assert tk.topkv_check_state_workspace_bytes(good) == 4
    assert tk.topkv_check_state_workspace_bytes(st(num_slots=33)) == 8
    assert tk.topkv_check_state_workspace_bytes(st(num_slots=0)) == -1
    _expect(tk, INV, tk.topkv_check_state_slots, good, 2, slots, 0)                       # null result
    _expect(tk, INV, tk.topkv_check_state_slots, good, 2, 0, res)                         # null slots
    _expect(tk, INV, tk.topkv_check_state_slots, good, -1, slots, res)
    _expect(tk, INV, tk.topkv_check_state_slots, good, 2, slots, res)                     # duplicates need a workspace
    _expect(tk, INV, tk.topkv_check_state_slots, good, 2, slots, res, workspace=ws, workspace_bytes=3)
    _expect(tk, INV, tk.topkv_check_state_slots, st(num_slots=0), 2, slots, res, check_duplicates=False)
    tk.topkv_pack_state_layer(good, 2, 0, 0, 0, dst_bytes=0, stream=0)      # no requests: nothing to launch
    tk.topkv_unpack_state_layer(0, good, 0, 0, 0, src_bytes=0, stream=0)


def test_kvcache1_layer_range_validation(tk):
    """Whole-request KVCACHE1 calls refuse layer ranges outside the pool
    before any launch; an empty range queues nothing."""
    INV = tk.TOPKV_ERR_INVALID_ARG
    good = _pool(tk)                     # 2 layers
    bt, blob = 0x20000, 0x40000
    nbytes = tk.topkv_kvcache1_bytes(good, 16)
    for first, count in ((-1, 1), (0, 3), (1, 2), (2, 1), (0, -1)):
        _expect(tk, INV, tk.topkv_kvcache1_pack_layers, good, first, count, bt, 16, blob, blob_bytes=nbytes)
        _expect(tk, INV, tk.topkv_kvcache1_unpack_layers, blob, good, first, count, bt, 16, blob_bytes=nbytes)
    _expect(tk, INV, tk.topkv_kvcache1_pack_layers, good, 0, 2, bt, 16, blob, blob_bytes=nbytes - 1)
    tk.topkv_kvcache1_pack_layers(good, 1, 0, bt, 16, blob, blob_bytes=nbytes, stream=0)


def test_kvcache1_one_pass_refuses_bad_pool_descriptors(tk):
    """The one-pass serializer and receiver apply the pool checks of every
    pack/unpack before choosing a path (element size 1/2/4/8, page count
    within 32 bits), and a blob size that overflows is refused."""
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    bt, blob, ws, res = 0x20000, 0x40000, 0x60000, 0x70000
    big = 1 << 40
    for pool, code in ((_pool(tk, num_heads=1, head_dim=16, elem_bytes=3), INV),   # 48-byte rows
                       (_pool(tk, num_pages=1 << 33), UNS)):
        nbytes = tk.topkv_kvcache1_bytes(pool, 16)
        assert nbytes > 0
        _expect(tk, code, tk.topkv_kvcache1_pack_seal, pool, bt, 16, 1, 2, blob, ws, blob_bytes=nbytes,
                workspace_bytes=big)
        _expect(tk, code, tk.topkv_kvcache1_verify_unpack, blob, pool, bt, 16, 1, 2, ws, res, blob_bytes=nbytes,
                workspace_bytes=big)
    huge = _pool(tk, num_heads=1 << 20, head_dim=1 << 20, num_layers=1 << 20)
    assert tk.topkv_kvcache1_bytes(huge, 1 << 20) == -1
    assert tk.topkv_kvcache1_workspace_bytes(huge, 1 << 20) == -1


def test_checked_mode_validates_arguments_first(tk, monkeypatch):
    """With TOPKV_CHECKED=1 the host-side argument checks still come first:
    a call with bad arguments is refused before checked mode touches the
    runtime (no GPU is needed to see it)."""
    monkeypatch.setenv("TOPKV_CHECKED", "1")
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    bt, lens, buf = 0x20000, 0x30000, 0x40000
    good = _pool(tk)
    _expect(tk, INV, tk.topkv_pack_layer, _pool(tk, base=0), 0, bt, 16, buf)
    _expect(tk, INV, tk.topkv_pack_layer, good, 0, bt, -1, buf)
    _expect(tk, INV, tk.topkv_pack_layer_batched, good, 0, 3, bt, 0, lens, buf, dst_bytes=1 << 20)
    _expect(tk, INV, tk.topkv_unpack_layer_batched, buf, good, 0, 3, bt, 4, lens, src_bytes=-1)
    _expect(tk, UNS, tk.topkv_pack_layer_batched, good, 0, tk.TOPKV_MAX_BATCH_REQS + 1, bt, 4, lens,
            buf, dst_bytes=1 << 20)
    tk.topkv_pack_layer(good, 0, 0, 0, 0, stream=0)            # zero tokens: still nothing to do


CEILING_HEADER = os.path.join(ROOT, "include", "topkv_ceiling.h")


def test_ceiling_library_exports_and_validation():
    """The measurement kernels' library loads, exports what its header
    declares under the binding's names, and refuses bad arguments before any
    launch (no GPU needed)."""
    from paper_2607_28633_amd.build import CEILING_LIBRARY, build_ceiling
    if not os.path.exists(CEILING_LIBRARY):
        build_ceiling()
    from paper_2607_28633_amd import ceiling as cl
    from paper_2607_28633_amd import topkv as tk
    text = re.sub(r"/\*.*?\*/", "", open(CEILING_HEADER).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(topkv_ceiling_[a-z_0-9]+)\s*\(", text)))
    assert declared == sorted(cl.EXPORTS)
    lib = ctypes.CDLL(cl.LIBRARY)
    assert all(hasattr(lib, n) for n in declared)
    INV = tk.TOPKV_ERR_INVALID_ARG
    a, b = 0x10000, 0x20000
    for fn, args in ((cl.topkv_ceiling_copy, (0, b, 64)), (cl.topkv_ceiling_copy, (a, b, 17)),
                     (cl.topkv_ceiling_copy, (a + 8, b, 64)), (cl.topkv_ceiling_copy, (a, b, -16)),
                     (cl.topkv_ceiling_copy_layers, (a, 64, b, 64, 48, -1)),
                     (cl.topkv_ceiling_copy_layers, (a, 60, b, 64, 48, 2)),
                     (cl.topkv_ceiling_copy_layers, (a, 64, b, 64, 48, 2, 65)),
                     (cl.topkv_ceiling_copy_timeline, (a, b, 64, 0)),
                     (cl.topkv_ceiling_read, (a, 64, 0)), (cl.topkv_ceiling_read, (a, 24, b)),
                     (cl.topkv_ceiling_read, (a + 8, 64, b)),
                     (cl.topkv_ceiling_copy_tiles, (a, 64, 0, b, 64, a, None, 1)),
                     (cl.topkv_ceiling_copy_tiles, (a, 64, a, b, 64, b, None, -1)),
                     (cl.topkv_ceiling_copy_tiles, (a, -1, a, b, 64, b, None, 1)),
                     (cl.topkv_ceiling_copy_tiles, (a + 8, 64, a, b, 64, b, None, 1))):
        with pytest.raises(tk.TopkvError) as ei:
            fn(*args, stream=0)
        assert ei.value.status == INV, (fn.__name__, args)
    cl.topkv_ceiling_copy(a, b, 0, stream=0)                       # nothing to copy: nothing launched
    cl.topkv_ceiling_copy_layers(a, 64, b, 64, 0, 3, stream=0)
    cl.topkv_ceiling_read(a, 0, b, stream=0)
    cl.topkv_ceiling_copy_tiles(a, 64, a, b, 64, b, None, 0, stream=0)


def test_crc64_noalloc_validation(tk):
    """The allocation-free CRC refuses bad arguments before touching the
    runtime (its array's address is looked up only after them)."""
    INV, UNS = tk.TOPKV_ERR_INVALID_ARG, tk.TOPKV_ERR_UNSUPPORTED
    out = 0x50000
    _expect(tk, INV, tk.topkv_crc64_noalloc, 0, 16, out)            # null data
    _expect(tk, INV, tk.topkv_crc64_noalloc, 0x10000, -1, out)      # negative length
    _expect(tk, INV, tk.topkv_crc64_noalloc, 0x10000, 16, 0)        # null result word
    _expect(tk, UNS, tk.topkv_crc64_noalloc, 0x10008, 16, out)      # data off 16-byte alignment

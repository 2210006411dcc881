"""Windowed layers (only the last W tokens of each request move) through the
C ABI vs the CPU oracle, bit for bit: reduced workloads element-wise, and the
mixed-kind gpt-oss-120b shape at full size in the benchmark's launch
configuration (sampled layers vs the oracle, every layer by round trip)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import (device_dst_prefill, device_src_pool, host_dst_prefill,
                                            host_src_pool, make_workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _scaled(name, div, **kw):
    base = make_workload(name)
    return make_workload(name, seq_lens=np.maximum(base.seq_lens // div, 1), **kw)


CASES = {
    "tiny-w1": (lambda: make_workload("tiny", seq_lens=[64, 48, 33, 17, 0, 1]), 1),
    "tiny-w17-p48": (lambda: make_workload("tiny", seq_lens=[64, 48, 33, 17, 0, 1], dst_page_size=48), 17),
    "tiny-w40-p5": (lambda: make_workload("tiny", dst_page_size=5), 40),
    "mla-div16-w128": (lambda: _scaled("deepseek-v3-mla", 16, num_layers=2), 128),
    "reblock-div32-w1000": (lambda: _scaled("reblock-70b", 32, num_layers=2, phys_layers=2), 1000),
    "gpt-oss-div8-w128": (lambda: _scaled("gpt-oss-120b", 8, num_layers=2), 128),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_window_parity(tk, case):
    make, W = CASES[case]
    wl = make()
    say(f"[window] {case}: W={W} {wl.describe()}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_window_bytes(src, wl.seq_lens, W)
    assert nbytes == oracle.packed_layer_elems(wl.planes, wl.num_heads, wl.head_dim, wl.seq_lens, W) * wl.elem_bytes
    want_dst = dst_h.copy()
    for layer in range(wl.num_layers):
        slab = layer % wl.phys_layers
        packed = torch.full((nbytes // wl.elem_bytes + 32,), -9, dtype=src.dtype, device="cuda")
        tk.topkv_pack_layer_window(src, slab, wl.num_reqs, bt, bt.shape[1], lens, W, packed, dst_bytes=nbytes)
        tk.topkv_unpack_layer_window(packed, dst, slab, wl.num_reqs, bt2, bt2.shape[1], lens, W, src_bytes=nbytes)
        torch.cuda.synchronize()
        got = to_host(packed)
        want = oracle.pack_layer(src_h, slab, wl.block_tables, wl.seq_lens, window=W)
        assert np.array_equal(got[:want.size], want), f"{case} layer {layer}: windowed pack differs"
        assert (got[want.size:].view(np.int16) == -9).all(), f"{case}: write past the batch"
        oracle.unpack_layer(want, want_dst, slab, wl.dst_block_tables, wl.seq_lens, window=W)
        assert np.array_equal(to_host(dst)[slab], want_dst[slab]), f"{case} layer {layer}: windowed unpack differs"


def test_window_zero_is_the_batched_call(tk):
    wl = make_workload("tiny")
    src = to_dev(host_src_pool(wl))
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    assert tk.topkv_packed_window_bytes(src, wl.seq_lens, 0) == nbytes
    a = torch.zeros(nbytes // 2, dtype=torch.int16, device="cuda")
    b = torch.ones_like(a)
    tk.topkv_pack_layer_window(src, 1, wl.num_reqs, bt, bt.shape[1], lens, 0, a)
    tk.topkv_pack_layer_batched(src, 1, wl.num_reqs, bt, bt.shape[1], lens, b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_gpt_oss_fullsize(tk):
    """36 layers alternating 128-token windows and full attention, 32 requests."""
    wl = make_workload("gpt-oss-120b")
    say(f"[window] gpt-oss-120b full size: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    full = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    packed = torch.empty(full // 2, dtype=torch.int16, device="cuda")
    again = torch.empty_like(packed)
    for layer in range(wl.num_layers):
        W = wl.window(layer)
        nb = tk.topkv_packed_window_bytes(src, wl.seq_lens, W)
        if layer in (0, 1, wl.num_layers - 1):
            torch.cuda.synchronize()
            src_h, dst_before = to_host(src[layer])[None], to_host(dst[layer])[None]
        tk.topkv_pack_layer_window(src, layer, wl.num_reqs, bt, bt.shape[1], lens, W, packed, dst_bytes=nb)
        tk.topkv_unpack_layer_window(packed, dst, layer, wl.num_reqs, bt2, bt2.shape[1], lens, W, src_bytes=nb)
        tk.topkv_pack_layer_window(dst, layer, wl.num_reqs, bt2, bt2.shape[1], lens, W, again, dst_bytes=nb)
        assert torch.equal(packed[:nb // 2], again[:nb // 2]), f"layer {layer}: round trip differs"
        if layer in (0, 1, wl.num_layers - 1):
            want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens, window=W)
            assert np.array_equal(to_host(packed[:nb // 2]), want), f"layer {layer} (W={W}) pack differs"
            oracle.unpack_layer(want, dst_before, 0, wl.dst_block_tables, wl.seq_lens, window=W)
            assert np.array_equal(to_host(dst[layer]), dst_before[0]), f"layer {layer} (W={W}) unpack differs"
            say(f"  layer {layer} W={W}: {nb} B bit-exact vs oracle")
    del src, dst, packed, again
    torch.cuda.empty_cache()

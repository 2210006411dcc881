"""Full-size workloads in the benchmark's launch configuration (one batched
launch per layer per direction over device-generated pools).

Sampled layers (first, middle, last) are compared with the CPU oracle in full
(pack output and the whole destination layer slab).  Every layer is checked
on the device by a property that holds at any size: packing the unpacked
destination pool (other page size, other page assignment) reproduces the
first pack bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import device_dst_prefill, device_src_pool, make_workload

pytestmark = pytest.mark.gpu

FULL = ["llama3-70b-4k", "llama3-8b", "llama3-70b-batch8", "deepseek-v3-mla", "reblock-70b", "llama3-70b-tp8"]


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


@pytest.mark.parametrize("name", FULL)
def test_fullsize(tk, name):
    wl = make_workload(name)
    say(f"[fullsize] {name}: {wl.describe()}")
    src = device_src_pool(wl)
    dst = device_dst_prefill(wl)
    bt, bt2 = to_dev(wl.block_tables), to_dev(wl.dst_block_tables)
    lens = to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    packed = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    again = torch.empty_like(packed)
    sample = {0, wl.num_layers // 2, wl.num_layers - 1}
    for layer in range(wl.num_layers):
        slab = layer % wl.phys_layers
        if layer in sample:
            torch.cuda.synchronize()
            src_h = to_host(src[slab])[None]
            dst_before = to_host(dst[slab])[None]
        tk.topkv_pack_layer_batched(src, slab, wl.num_reqs, bt, bt.shape[1], lens, packed)
        tk.topkv_unpack_layer_batched(packed, dst, slab, wl.num_reqs, bt2, bt2.shape[1], lens)
        tk.topkv_pack_layer_batched(dst, slab, wl.num_reqs, bt2, bt2.shape[1], lens, again)
        assert torch.equal(packed, again), f"{name} layer {layer}: round trip through the destination differs"
        if layer in sample:
            want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens)
            assert np.array_equal(to_host(packed), want), f"{name} layer {layer}: pack differs from oracle"
            oracle.unpack_layer(want, dst_before, 0, wl.dst_block_tables, wl.seq_lens)
            assert np.array_equal(to_host(dst[slab]), dst_before[0]), \
                f"{name} layer {layer}: unpacked slab differs from oracle"
            say(f"  layer {layer} (slab {slab}) bit-exact vs oracle, {nbytes} B")
            del src_h, dst_before, want
    torch.cuda.synchronize()
    del src, dst, packed, again
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["llama3-70b-4k", "llama3-8b"])
def test_fullsize_host_length(tk, name):
    """The one-request workloads through topkv_pack_layer / topkv_unpack_layer
    (host-side length, tables cut to the request's pages): every layer round
    trips through the destination pool, sampled layers equal the oracle."""
    wl = make_workload(name)
    say(f"[fullsize_host] {name}: {wl.describe()}")
    src = device_src_pool(wl)
    dst = device_dst_prefill(wl)
    n = int(wl.seq_lens[0])
    k, k2 = -(-n // wl.page_size), -(-n // wl.dst_page_size)
    bt, bt2 = to_dev(wl.block_tables[0, :k]), to_dev(wl.dst_block_tables[0, :k2])
    nbytes = tk.topkv_packed_layer_bytes(src, [n])
    packed = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    again = torch.empty_like(packed)
    sample = {0, wl.num_layers - 1}
    for layer in range(wl.num_layers):
        slab = layer % wl.phys_layers
        if layer in sample:
            torch.cuda.synchronize()
            src_h = to_host(src[slab])[None]
            dst_before = to_host(dst[slab])[None]
        tk.topkv_pack_layer(src, slab, bt, n, packed)
        tk.topkv_unpack_layer(packed, dst, slab, bt2, n)
        tk.topkv_pack_layer(dst, slab, bt2, n, again)
        assert torch.equal(packed, again), f"{name} layer {layer}: round trip through the destination differs"
        if layer in sample:
            want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens)
            assert np.array_equal(to_host(packed), want), f"{name} layer {layer}: pack differs from oracle"
            oracle.unpack_layer(want, dst_before, 0, wl.dst_block_tables, wl.seq_lens)
            assert np.array_equal(to_host(dst[slab]), dst_before[0]), \
                f"{name} layer {layer}: unpacked slab differs from oracle"
            say(f"  layer {layer} (slab {slab}) bit-exact vs oracle, {nbytes} B")
            del src_h, dst_before, want
    torch.cuda.synchronize()
    del src, dst, packed, again
    torch.cuda.empty_cache()


def test_fullsize_hybrid(tk):
    """The hybrid model at full size (60 layers, 45 fixed-state, 32 requests):
    every layer round-trips through the destination side with the call its
    kind takes; the first and last layer of each kind is compared with the
    oracle in full."""
    import oracle.state as so
    from paper_2607_28633_amd.workloads import device_state_cache
    wl = make_workload("qwen3.5-397b-hybrid")
    say(f"[fullsize] hybrid: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    st_src, st_dst = device_state_cache(wl), device_state_cache(wl, dst=True)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    s1, s2 = to_dev(wl.state_slots), to_dev(wl.dst_state_slots)
    R = wl.num_reqs
    kv_bytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    st_bytes = tk.topkv_packed_state_bytes(st_src, R)
    packed = torch.empty(max(kv_bytes, st_bytes) // 2, dtype=torch.int16, device="cuda")
    again = torch.empty_like(packed)
    state_layers = [l for l in range(wl.num_layers) if wl.is_state(l)]
    attn_layers = [l for l in range(wl.num_layers) if not wl.is_state(l)]
    sample = {state_layers[0], state_layers[-1], attn_layers[0], attn_layers[-1]}
    for layer in range(wl.num_layers):
        if wl.is_state(layer):
            slab, n, cache_s, cache_d = wl.state_slab(layer), st_bytes // 2, st_src, st_dst
        else:
            slab, n, cache_s, cache_d = wl.kv_slab(layer), kv_bytes // 2, src, dst
        if layer in sample:
            torch.cuda.synchronize()
            src_h = to_host(cache_s[slab])[None]
            dst_before = to_host(cache_d[slab])[None]
        if wl.is_state(layer):
            tk.topkv_pack_state_layer(st_src, slab, R, s1, packed, dst_bytes=st_bytes)
            tk.topkv_unpack_state_layer(packed, st_dst, slab, R, s2, src_bytes=st_bytes)
            tk.topkv_pack_state_layer(st_dst, slab, R, s2, again, dst_bytes=st_bytes)
        else:
            tk.topkv_pack_layer_batched(src, slab, R, bt, bt.shape[1], lens, packed, dst_bytes=kv_bytes)
            tk.topkv_unpack_layer_batched(packed, dst, slab, R, bt2, bt2.shape[1], lens, src_bytes=kv_bytes)
            tk.topkv_pack_layer_batched(dst, slab, R, bt2, bt2.shape[1], lens, again, dst_bytes=kv_bytes)
        assert torch.equal(packed[:n], again[:n]), f"hybrid layer {layer}: round trip differs"
        if layer in sample:
            if wl.is_state(layer):
                want = so.pack_state_layer(src_h, 0, wl.state_slots)
                so.unpack_state_layer(want, dst_before, 0, wl.dst_state_slots)
            else:
                want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens)
                oracle.unpack_layer(want, dst_before, 0, wl.dst_block_tables, wl.seq_lens)
            assert np.array_equal(to_host(packed[:n]), want), f"hybrid layer {layer}: pack differs from oracle"
            assert np.array_equal(to_host(cache_d[slab]), dst_before[0]), \
                f"hybrid layer {layer}: unpacked slab differs from oracle"
            say(f"  layer {layer} ({'state' if wl.is_state(layer) else 'attention'}, slab {slab}) bit-exact vs oracle")
            del src_h, dst_before, want
    torch.cuda.synchronize()

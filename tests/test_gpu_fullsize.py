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

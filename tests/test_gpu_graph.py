"""Pack/unpack sweeps captured in HIP graphs (as the benchmark replays them):
every replay, with eager work and synchronisations between replays, equals
the eager launches bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import say, to_host
from paper_2607_28633_amd.workloads import device_dst_prefill, device_src_pool, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


@pytest.mark.parametrize("name,kw", [
    ("llama3-70b-4k", dict(num_layers=4, num_pages=600, dst_num_pages=700)),
    ("reblock-70b", dict(num_layers=3, phys_layers=3, seq_lens=[300, 17, 4096, 5000, 1, 64])),
])
def test_graph_replays_match_eager(tk, name, kw):
    wl = make_workload(name, **kw)
    say(f"[graph] {name}: {wl.describe()}")
    src = device_src_pool(wl)
    dst0 = device_dst_prefill(wl)
    bt = torch.from_numpy(wl.block_tables).cuda()
    bt2 = torch.from_numpy(wl.dst_block_tables).cuda()
    lens = torch.from_numpy(wl.seq_lens).cuda()
    L, R = wl.num_layers, wl.num_reqs
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)

    def sweep(packed, dst):
        for l in range(L):
            tk.topkv_pack_layer_batched(src, l % wl.phys_layers, R, bt, bt.shape[1], lens, packed[l])
        for l in range(L):
            tk.topkv_unpack_layer_batched(packed[l], dst, l % wl.phys_layers, R, bt2, bt2.shape[1], lens)

    packed_g = torch.zeros((L, nbytes // 2), dtype=torch.int16, device="cuda")
    dst_g = dst0.clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sweep(packed_g, dst_g)
    torch.cuda.synchronize()

    for replay in range(3):
        # eager work between replays: new pool contents, fresh outputs
        src.view(torch.int16).add_(replay + 1)
        packed_g.zero_()
        dst_g.copy_(dst0)
        packed_e = torch.zeros_like(packed_g)
        dst_e = dst0.clone()
        sweep(packed_e, dst_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(packed_g, packed_e), f"replay {replay}: packed buffers differ from eager"
        assert torch.equal(dst_g.view(torch.int16), dst_e.view(torch.int16)), f"replay {replay}: pools differ"
    # the eager result itself against the oracle on the last layer
    slab = (L - 1) % wl.phys_layers
    want = oracle.pack_layer(to_host(src[slab])[None], 0, wl.block_tables, wl.seq_lens)
    assert np.array_equal(to_host(packed_g[L - 1]), want)


def test_layout_moves_in_a_graph(tk):
    """Head-sliced pack, head-major unpack and re-blocking of every layer,
    captured once and replayed with eager work in between, equal eager."""
    wl = make_workload("reblock-70b", num_layers=3, phys_layers=3, seq_lens=[300, 17, 4096, 1, 64])
    say(f"[graph] layout moves: {wl.describe()}")
    src, dst0 = device_src_pool(wl), device_dst_prefill(wl)
    bt = torch.from_numpy(wl.block_tables).cuda()
    bt2 = torch.from_numpy(wl.dst_block_tables).cuda()
    lens = torch.from_numpy(wl.seq_lens).cuda()
    L, R, H = wl.num_layers, wl.num_reqs, wl.num_heads
    half = tk.topkv_packed_layer_bytes(src, wl.seq_lens) // 4         # int16 elements of one head half
    hm_shape = (wl.phys_layers, wl.dst_num_pages, wl.planes, H, wl.dst_page_size, wl.head_dim)

    def moves(packed, dst, hm):
        for l in range(L):
            for i in range(2):
                tk.topkv_pack_layer_heads(src, l, R, bt, bt.shape[1], lens, 4 * i, 4, packed[l, i])
            tk.topkv_move_layer(tk.packed_view(packed[l, 0]), tk.pool_view(hm, l, bt2, bt2.shape[1], 0, True),
                                R, lens, 4)
            tk.topkv_reblock_layer(src, l, bt, bt.shape[1], dst, l, bt2, bt2.shape[1], R, lens)

    packed_g = torch.zeros((L, 2, half), dtype=torch.int16, device="cuda")
    dst_g, hm_g = dst0.clone(), torch.zeros(hm_shape, dtype=torch.int16, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        moves(packed_g, dst_g, hm_g)
    torch.cuda.synchronize()
    for replay in range(3):
        src.view(torch.int16).add_(replay + 1)
        packed_g.zero_()
        hm_g.zero_()
        dst_g.copy_(dst0)
        packed_e, dst_e, hm_e = torch.zeros_like(packed_g), dst0.clone(), torch.zeros_like(hm_g)
        moves(packed_e, dst_e, hm_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(packed_g, packed_e), f"replay {replay}: head slices differ from eager"
        assert torch.equal(hm_g, hm_e), f"replay {replay}: head-major pool differs from eager"
        assert torch.equal(dst_g.view(torch.int16), dst_e.view(torch.int16)), f"replay {replay}: re-block differs"
    import oracle.reshard as rs
    want = rs.pack_layer_heads(to_host(src[2])[None], 0, wl.block_tables, wl.seq_lens, 4, 4)
    assert np.array_equal(to_host(packed_g[2, 1]), want), "last layer's second head half vs the oracle"

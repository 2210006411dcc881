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


def test_hybrid_sweep_in_a_graph(tk):
    """A reduced hybrid model's sweep (state layers through the state calls,
    attention layers through the batched calls, both directions) captured
    once and replayed with eager work in between, equal to eager launches;
    also a CRC-64 and a one-request pack in the same graph."""
    from paper_2607_28633_amd.workloads import device_state_cache
    wl = make_workload("qwen3.5-397b-hybrid", num_layers=8, seq_lens=[300, 17, 4096, 1], state_bytes=65536)
    say(f"[graph] hybrid sweep: {wl.describe()}")
    src, dst0 = device_src_pool(wl), device_dst_prefill(wl)
    st_src, st_dst0 = device_state_cache(wl), device_state_cache(wl, dst=True)
    bt = torch.from_numpy(wl.block_tables).cuda()
    bt2 = torch.from_numpy(wl.dst_block_tables).cuda()
    lens = torch.from_numpy(wl.seq_lens).cuda()
    s1, s2 = torch.from_numpy(wl.state_slots).cuda(), torch.from_numpy(wl.dst_state_slots).cuda()
    L, R = wl.num_layers, wl.num_reqs
    kv = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    stb = tk.topkv_packed_state_bytes(st_src, R)
    width = max(kv, stb) // 2
    one = tk.topkv_packed_layer_bytes(src, wl.seq_lens[2:3]) // 2
    ws = torch.empty(tk.topkv_crc64_workspace_bytes(kv) // 8, dtype=torch.int64, device="cuda")

    def sweep(packed, dst, st_dst, crc, single):
        for l in range(L):
            if wl.is_state(l):
                tk.topkv_pack_state_layer(st_src, wl.state_slab(l), R, s1, packed[l], dst_bytes=stb)
            else:
                tk.topkv_pack_layer_batched(src, wl.kv_slab(l), R, bt, bt.shape[1], lens, packed[l], dst_bytes=kv)
        for l in range(L):
            if wl.is_state(l):
                tk.topkv_unpack_state_layer(packed[l], st_dst, wl.state_slab(l), R, s2, src_bytes=stb)
            else:
                tk.topkv_unpack_layer_batched(packed[l], dst, wl.kv_slab(l), R, bt2, bt2.shape[1], lens,
                                              src_bytes=kv)
        tk.topkv_crc64(packed[L - 1], kv, ws, crc)
        tk.topkv_pack_layer_batched(src, 0, 1, bt[2:3], bt.shape[1], lens[2:3], single, dst_bytes=2 * one)

    def outputs():
        return (torch.zeros((L, width), dtype=torch.int16, device="cuda"), dst0.clone(), st_dst0.clone(),
                torch.zeros(1, dtype=torch.int64, device="cuda"), torch.zeros(one, dtype=torch.int16, device="cuda"))

    out_g = outputs()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sweep(*out_g)
    torch.cuda.synchronize()
    for replay in range(3):
        src.view(torch.int16).add_(replay + 1)
        st_src.add_(replay + 3)
        fresh = outputs()
        for a, b in zip(out_g, fresh):
            a.copy_(b)
        out_e = outputs()
        sweep(*out_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(out_g, out_e)):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"replay {replay}: output {i} differs"
    import oracle.state as so
    lay = max(l for l in range(L) if wl.is_state(l))
    want = so.pack_state_layer(to_host(st_src[wl.state_slab(lay)])[None], 0, wl.state_slots)
    assert np.array_equal(to_host(out_g[0][lay])[:stb // 2], want), "last state layer vs the oracle"


def test_graph_kvcache1_one_pass(tk):
    """The one-pass KVCACHE1 sender and receiver captured in one graph: every
    replay (new pool contents, cleared outputs and eager work in between)
    leaves the blob, the verdict and the decode pool the eager calls give."""
    from gpu_util import to_dev
    wl = make_workload("llama3-70b-4k", num_layers=3, num_pages=600, dst_num_pages=700, seq_lens=[1000])
    say(f"[graph] one-pass KVCACHE1: {wl.describe()}")
    src, dst0 = device_src_pool(wl), device_dst_prefill(wl)
    geo = tk.pool_from_tensor(src)
    n = int(wl.seq_lens[0])
    bt, bt2 = to_dev(wl.block_tables[0]), to_dev(wl.dst_block_tables[0])
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    ws_bytes = tk.topkv_kvcache1_workspace_bytes(geo, n)

    def run(blob, dst, ws, res):
        tk.topkv_kvcache1_pack_seal(src, bt, n, 11, 22, blob, ws)
        tk.topkv_kvcache1_verify_unpack(blob, dst, bt2, n, 11, 22, ws, res)

    blob_g = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dst_g = dst0.clone()
    ws_g = torch.zeros(ws_bytes // 8, dtype=torch.int64, device="cuda")
    res_g = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(blob_g, dst_g, ws_g, res_g)
    torch.cuda.synchronize()
    for replay in range(3):
        src.view(torch.int16).add_(replay + 1)
        blob_g.zero_()
        dst_g.copy_(dst0)
        res_g.fill_(7)
        blob_e, dst_e = torch.zeros_like(blob_g), dst0.clone()
        ws_e = torch.zeros_like(ws_g)
        res_e = torch.full((4,), 7, dtype=torch.int32, device="cuda")
        run(blob_e, dst_e, ws_e, res_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert res_e.tolist() == [tk.TOPKV_OK, 0, 0, 0] and res_g.tolist() == res_e.tolist(), f"replay {replay}"
        assert torch.equal(blob_g, blob_e), f"replay {replay}: blob differs"
        assert torch.equal(dst_g.view(torch.int16), dst_e.view(torch.int16)), f"replay {replay}: pool differs"

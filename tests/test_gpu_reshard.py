"""Layer moves between layouts (head-sliced pack/unpack, pool-to-pool
re-blocking, head-major pools) through the C ABI vs the CPU oracle, bit for
bit: reduced pools element by element across tiles and ragged tails, edge
cases (empty and one-token requests, odd widths, windows, malformed tables),
and the 70B shapes at full size in the benchmark's launch configuration
(sampled layers vs the oracle, the rest vs the full-head pack kernel)."""
import numpy as np
import pytest
import torch

import oracle
import oracle.reshard as rs
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import (device_dst_prefill, device_src_pool, host_dst_prefill,
                                            host_src_pool, make_workload)

pytestmark = pytest.mark.gpu

SENTINEL = -9


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _heads_wl(**kw):
    base = dict(num_layers=2, num_heads=8, head_dim=16, seq_lens=[37, 16, 0, 1, 50, 9, 300])
    base.update(kw)
    return make_workload("tiny", **base)


WORKLOADS = {
    "h8-d16": lambda: _heads_wl(),
    "h8-d16-p5": lambda: _heads_wl(dst_page_size=5),
    "h8-d128-p16-p64": lambda: _heads_wl(head_dim=128, dst_page_size=64, seq_lens=[700, 1, 64, 129]),
    "h3-d3-odd": lambda: _heads_wl(num_heads=3, head_dim=3, dst_page_size=48),
    "h4-d5-u8": lambda: _heads_wl(num_heads=4, head_dim=5, elem_bytes=1, dst_page_size=7),
    "mla-p64-p16": lambda: make_workload("deepseek-v3-mla", num_layers=2, seq_lens=[700, 1, 64, 129, 0],
                                         dst_page_size=16),
}


def _geom(wl):
    return wl.planes, wl.num_heads, wl.head_dim


@pytest.mark.parametrize("case", sorted(WORKLOADS))
def test_pack_heads_parity(tk, case):
    wl = WORKLOADS[case]()
    say(f"[reshard] pack heads {case}: {wl.describe()}")
    C, H, D = _geom(wl)
    src_h = host_src_pool(wl)
    src, bt, lens = to_dev(src_h), to_dev(wl.block_tables), to_dev(wl.seq_lens)
    slices = sorted({(0, H), (H - 1, 1), (H // 2, H - H // 2), (0, 1), (min(1, H - 1), max(1, H - 2))})
    for h0, hc in slices:
        for layer in range(wl.num_layers):
            n = rs.packed_heads_elems(C, hc, D, wl.seq_lens)
            out = torch.full((n + 64,), SENTINEL, dtype=src.dtype, device="cuda")
            tk.topkv_pack_layer_heads(src, layer, wl.num_reqs, bt, bt.shape[1], lens, h0, hc, out,
                                      dst_bytes=n * wl.elem_bytes)
            torch.cuda.synchronize()
            got = to_host(out)
            want = rs.pack_layer_heads(src_h, layer, wl.block_tables, wl.seq_lens, h0, hc)
            assert np.array_equal(got[:n], want), f"{case} heads [{h0}, +{hc}) layer {layer}"
            assert torch.equal(out[n:], torch.full_like(out[n:], SENTINEL)), f"{case}: write past the packed batch"


@pytest.mark.parametrize("case", sorted(WORKLOADS))
def test_unpack_heads_parity(tk, case):
    wl = WORKLOADS[case]()
    say(f"[reshard] unpack heads {case}")
    C, H, D = _geom(wl)
    dst_h = host_dst_prefill(wl)
    dst, bt2, lens = to_dev(dst_h), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    want = dst_h.copy()
    rng = np.random.default_rng(5)
    for h0, hc in sorted({(0, H), (H - 1, 1), (H // 2, H - H // 2)}):
        n = rs.packed_heads_elems(C, hc, D, wl.seq_lens)
        packed_h = rng.integers(0, 1 << (8 * wl.elem_bytes), n, dtype=np.uint64).astype(want.dtype)
        layer = (h0 + hc) % wl.num_layers
        tk.topkv_unpack_layer_heads(to_dev(packed_h), dst, layer, wl.num_reqs, bt2, bt2.shape[1], lens, h0, hc)
        rs.unpack_layer_heads(packed_h, want, layer, wl.dst_block_tables, wl.seq_lens, h0, hc)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(dst), want), f"{case}: pool after head-sliced unpacks differs"


@pytest.mark.parametrize("case", sorted(WORKLOADS))
@pytest.mark.parametrize("window", [0, 40])
def test_reblock_parity(tk, case, window):
    wl = WORKLOADS[case]()
    say(f"[reshard] re-block {case} P={wl.page_size}->{wl.dst_page_size} W={window}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    want = dst_h.copy()
    for layer in range(wl.num_layers):
        dl = (layer + 1) % wl.num_layers
        if window:
            tk.topkv_move_layer(tk.pool_view(src, layer, bt, bt.shape[1]), tk.pool_view(dst, dl, bt2, bt2.shape[1]),
                                wl.num_reqs, lens, wl.num_heads, window)
        else:
            tk.topkv_reblock_layer(src, layer, bt, bt.shape[1], dst, dl, bt2, bt2.shape[1], wl.num_reqs, lens)
        rs.reblock_layer(src_h, layer, wl.block_tables, want, dl, wl.dst_block_tables, wl.seq_lens, window)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(dst), want), f"{case} W={window}: re-blocked pool differs"


HM_CASES = [("pool", "hm", 0, 0, 0), ("hm", "packed", 1, 0, 0), ("hm", "pool", 2, 1, 7), ("hm", "hm", 0, 3, 0),
            ("packed", "hm", 0, 2, 13), ("pool", "hm", 3, 5, 0)]


@pytest.mark.parametrize("case", ["h8-d16-p5", "h8-d128-p16-p64", "h3-d3-odd", "h4-d5-u8"])
def test_head_major_parity(tk, case):
    wl = WORKLOADS[case]()
    C, H, D = _geom(wl)
    src_sm = host_src_pool(wl)
    src_hm = rs.to_head_major(src_sm)
    dst_sm = host_dst_prefill(wl)
    dst_hm = rs.to_head_major(dst_sm)
    tabs = {"src": wl.block_tables, "dst": wl.dst_block_tables}
    for sk, dk, h0s, h0d, window in HM_CASES:
        hc = max(1, min(H - h0s, H - h0d, 3 if (h0s or h0d) else H))
        if h0s >= H or h0d >= H:
            continue
        say(f"[reshard] head-major {case}: {sk} -> {dk}, heads {h0s}/{h0d} +{hc}, W={window}")
        n = rs.packed_heads_elems(C, hc, D, wl.seq_lens, window)
        if sk == "packed":
            s_h = rs.pack_layer_heads(src_sm, 1, wl.block_tables, wl.seq_lens, 0, hc, window)
        else:
            s_h = src_hm if sk == "hm" else src_sm
        d_h = np.zeros(n, dtype=src_sm.dtype) if dk == "packed" else (dst_hm if dk == "hm" else dst_sm).copy()
        lay = {"packed": rs.PACKED, "pool": rs.POOL, "hm": rs.POOL_HEAD_MAJOR}
        want = rs.move_layer(rs.View(lay[sk], s_h, 1, tabs["src"], h0s if sk != "packed" else 0),
                             rs.View(lay[dk], d_h.copy(), 0, tabs["dst"], h0d if dk != "packed" else 0),
                             wl.seq_lens, hc, window)
        s_d, d_d = to_dev(s_h), to_dev(d_h)
        bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
        sv = (tk.packed_view(s_d) if sk == "packed" else
              tk.pool_view(s_d, 1, bt, bt.shape[1], h0s, head_major=sk == "hm"))
        dv = (tk.packed_view(d_d) if dk == "packed" else
              tk.pool_view(d_d, 0, bt2, bt2.shape[1], h0d, head_major=dk == "hm"))
        tk.topkv_move_layer(sv, dv, wl.num_reqs, lens, hc, window)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(d_d), want), f"{case}: {sk} -> {dk} differs"


@pytest.mark.parametrize("case", ["h8-d16", "h8-d128-p16-p64", "h4-d5-u8"])
def test_shards_parity(tk, case):
    """Packing for S tensor-parallel receivers in one launch (shard regions
    with slack between them) and unpacking the shards back, vs the oracle."""
    wl = WORKLOADS[case]()
    C, H, D = _geom(wl)
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    want_pool = dst_h.copy()
    for S in sorted({s for s in (1, 2, 4, H) if H % s == 0}):
        say(f"[reshard] shards {case}: S={S}")
        per = rs.packed_heads_elems(C, H // S, D, wl.seq_lens)
        cap = per + 16 // wl.elem_bytes                       # slack stays untouched
        out = torch.full((S * cap,), SENTINEL, dtype=src.dtype, device="cuda")
        tk.topkv_pack_layer_shards(src, 1, wl.num_reqs, bt, bt.shape[1], lens, 0, H, S, out,
                                   shard_bytes=cap * wl.elem_bytes)
        torch.cuda.synchronize()
        want = rs.pack_layer_shards(src_h, 1, wl.block_tables, wl.seq_lens, 0, H, S, cap)
        got = to_host(out)
        for sh in range(S):
            assert np.array_equal(got[sh * cap:sh * cap + per], want[sh * cap:sh * cap + per]), f"S={S} shard {sh}"
            assert torch.equal(out[sh * cap + per:(sh + 1) * cap],
                               torch.full_like(out[sh * cap + per:(sh + 1) * cap], SENTINEL)), f"S={S}: slack written"
        tk.topkv_unpack_layer_shards(out, dst, 0, wl.num_reqs, bt2, bt2.shape[1], lens, 0, H, S,
                                     shard_bytes=cap * wl.elem_bytes)
        rs.move_layer(rs.View(rs.PACKED, want, shards=S, shard_elems=cap),
                      rs.View(rs.POOL, want_pool, 0, wl.dst_block_tables), wl.seq_lens, H)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(dst), want_pool), f"{case}: pool after sharded unpacks differs"


def test_untrusted_tables_and_lengths(tk):
    """Out-of-range table entries are skipped, lengths are clamped to the
    table capacity and negative lengths count as zero; nothing else moves."""
    wl = _heads_wl(seq_lens=[37, 16, 50, 9])
    C, H, D = _geom(wl)
    src_h = host_src_pool(wl)
    bt_h = wl.block_tables.copy()
    bt_h[0, 1] = -1                      # tokens 16..31 of request 0
    bt_h[2, 0] = wl.num_pages            # tokens 0..15 of request 2
    lens_h = np.array([37, -5, 10_000, 9], dtype=np.int32)
    clamp = np.clip(lens_h, 0, bt_h.shape[1] * wl.page_size).astype(np.int32)
    src, bt, lens = to_dev(src_h), to_dev(bt_h), to_dev(lens_h)
    h0, hc = 2, 3
    n = rs.packed_heads_elems(C, hc, D, clamp)
    out = torch.full((n,), SENTINEL, dtype=src.dtype, device="cuda")
    tk.topkv_pack_layer_heads(src, 0, 4, bt, bt.shape[1], lens, h0, hc, out)
    torch.cuda.synchronize()
    got = to_host(out).view(np.int16)
    good_bt = bt_h.copy()
    good_bt[0, 1] = 0
    good_bt[2, 0] = 0
    want = rs.pack_layer_heads(src_h, 0, good_bt, clamp, h0, hc).view(np.int16).copy()
    # blank the skipped tokens in the expectation
    off = 0
    for r, nr in enumerate(clamp):
        blk = want[off:off + C * nr * hc * D].reshape(C, nr, hc, D)
        if r == 0:
            blk[:, 16:32] = SENTINEL
        if r == 2:
            blk[:, 0:16] = SENTINEL
        off += blk.size
    assert np.array_equal(got, want)


def test_fullsize_70b_head_slices(tk):
    """70B, 4096 tokens: the two tensor-parallel halves (heads 0-3, 4-7) put
    side by side are the full-head packed layer of the fast pack kernel, on
    every layer; sampled layers also vs the oracle."""
    wl = make_workload("llama3-70b-4k")
    say(f"[reshard] 70B head slices full size: {wl.describe()}")
    src = device_src_pool(wl)
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)
    n = int(wl.seq_lens[0])
    full = torch.empty(2 * n * 8 * 128, dtype=torch.int16, device="cuda")
    halves = [torch.empty(2 * n * 4 * 128, dtype=torch.int16, device="cuda") for _ in range(2)]
    for layer in range(wl.num_layers):
        tk.topkv_pack_layer_batched(src, layer, 1, bt, bt.shape[1], lens, full)
        for i in range(2):
            tk.topkv_pack_layer_heads(src, layer, 1, bt, bt.shape[1], lens, 4 * i, 4, halves[i])
        joined = torch.cat([h.view(2, n, 4, 128) for h in halves], dim=2).reshape(-1)
        assert torch.equal(joined, full), f"layer {layer}: head halves do not tile the layer"
        if layer in (0, 79):
            want = rs.pack_layer_heads(to_host(src[layer])[None], 0, wl.block_tables, wl.seq_lens, 4, 4)
            assert np.array_equal(to_host(halves[1]), want), f"layer {layer}: heads 4-7 vs oracle"
    del src
    torch.cuda.empty_cache()


def test_fullsize_70b_shards_one_launch(tk):
    """70B, 4096 tokens: both tensor-parallel halves in one launch equal the
    two head-sliced launches, on every layer."""
    wl = make_workload("llama3-70b-4k")
    src = device_src_pool(wl)
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)
    n = int(wl.seq_lens[0])
    half = 2 * n * 4 * 128
    both = torch.empty(2 * half, dtype=torch.int16, device="cuda")
    sep = torch.empty(2 * half, dtype=torch.int16, device="cuda")
    for layer in range(wl.num_layers):
        tk.topkv_pack_layer_shards(src, layer, 1, bt, bt.shape[1], lens, 0, 8, 2, both)
        for i in range(2):
            tk.topkv_pack_layer_heads(src, layer, 1, bt, bt.shape[1], lens, 4 * i, 4, sep[i * half:(i + 1) * half])
        assert torch.equal(both, sep), f"layer {layer}: one-launch shards differ from per-shard launches"
    del src
    torch.cuda.empty_cache()


def test_fullsize_reblock_70b(tk):
    """reblock-70b (100 requests, page 16 -> 64) at full size: the fused
    pool-to-pool move equals the fast pack + unpack pair on sampled layers,
    and one layer equals the oracle."""
    wl = make_workload("reblock-70b")
    say(f"[reshard] re-block full size: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    dst2 = dst.clone()
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    packed = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    for layer in (0, 5, 7):
        tk.topkv_reblock_layer(src, layer, bt, bt.shape[1], dst, layer, bt2, bt2.shape[1], wl.num_reqs, lens)
        tk.topkv_pack_layer_batched(src, layer, wl.num_reqs, bt, bt.shape[1], lens, packed)
        tk.topkv_unpack_layer_batched(packed, dst2, layer, wl.num_reqs, bt2, bt2.shape[1], lens)
        torch.cuda.synchronize()
        same = torch.equal(dst[layer].view(torch.int16), dst2[layer].view(torch.int16))   # bits: NaNs included
        assert same, f"layer {layer}: fused re-block differs from pack+unpack"
    want = oracle.unpack_layer(oracle.pack_layer(to_host(src[5])[None], 0, wl.block_tables, wl.seq_lens),
                               to_host(device_dst_prefill(wl)[5])[None], 0, wl.dst_block_tables, wl.seq_lens)
    assert np.array_equal(to_host(dst[5]), want[0]), "layer 5 vs oracle"
    del src, dst, dst2, packed
    torch.cuda.empty_cache()


def test_fullsize_head_major_70b(tk):
    """70B, 4096 tokens, page 16 -> head-major page 64 and back to packed:
    equals the fast pack on every layer."""
    wl = make_workload("llama3-70b-4k", dst_page_size=64)
    say(f"[reshard] head-major full size: {wl.describe()}")
    src = device_src_pool(wl)
    hm = torch.zeros((wl.phys_layers, wl.dst_num_pages, 2, 8, 64, 128), dtype=torch.int16, device="cuda")
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    n = int(wl.seq_lens[0])
    full = torch.empty(2 * n * 8 * 128, dtype=torch.int16, device="cuda")
    back = torch.empty_like(full)
    for layer in range(0, wl.num_layers, 7):
        tk.topkv_move_layer(tk.pool_view(src, layer, bt, bt.shape[1]),
                            tk.pool_view(hm, layer, bt2, bt2.shape[1], head_major=True), 1, lens, 8)
        tk.topkv_move_layer(tk.pool_view(hm, layer, bt2, bt2.shape[1], head_major=True), tk.packed_view(back),
                            1, lens, 8)
        tk.topkv_pack_layer_batched(src, layer, 1, bt, bt.shape[1], lens, full)
        assert torch.equal(back, full), f"layer {layer}: head-major round trip differs"
    page0 = int(wl.dst_block_tables[0][3])
    want = rs.to_head_major(
        oracle.unpack_layer(oracle.pack_layer(to_host(src[0])[None], 0, wl.block_tables, wl.seq_lens),
                            np.zeros((1, wl.dst_num_pages, 2, 64, 8, 128), np.uint16), 0, wl.dst_block_tables,
                            wl.seq_lens))
    assert np.array_equal(to_host(hm[0, page0]), want[0, page0]), "head-major page vs oracle"
    del src, hm
    torch.cuda.empty_cache()


MULTI_CASES = [("h8-d128-p16-p64", 0), ("h8-d128-p16-p64", 40), ("h8-d16", 0), ("mla-p64-p16", 0)]


@pytest.mark.parametrize("case,window", MULTI_CASES)
def test_move_layers_matches_oracle(tk, case, window):
    """topkv_move_layers over every layer of a range equals the oracle's move
    of each layer: head-sliced pack into packed layers `stride` apart (slack
    between them untouched), two shards per layer, the unpack back into a
    pool, and pool-to-pool re-blocking from a later source layer.  With 2 KiB
    rows the direct grid carries the layers on grid z (one request: the
    one-request grid; a batch: the batched one); with 256-byte rows, or a
    window, every layer takes its own launch."""
    wl = WORKLOADS[case]()
    C, H, D = _geom(wl)
    L = wl.num_layers + 1
    wl = make_workload(wl.name, num_layers=L, num_heads=H, head_dim=D, seq_lens=wl.seq_lens,
                       page_size=wl.page_size, dst_page_size=wl.dst_page_size, elem_bytes=wl.elem_bytes)
    say(f"[reshard] move_layers {case} W={window}: {wl.describe()}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    E = wl.elem_bytes
    for sub in ([(0, wl.num_reqs)] if wl.num_reqs == 1 else [(0, 1), (0, wl.num_reqs)]):
        R = sub[1]
        lens_r = wl.seq_lens[:R]
        h0, hc, S = (0, H, 2) if H % 2 == 0 else (0, H, 1)
        per = rs.packed_heads_elems(C, hc // S, D, lens_r, window)
        cap = per + 32 // E                                     # each shard region with slack
        stride = S * cap + 64 // E                              # and slack between layers
        n_lay = L - 1
        out = torch.full((n_lay * stride,), SENTINEL, dtype=src.dtype, device="cuda")
        tk.topkv_move_layers(tk.pool_view(src, 1, bt, bt.shape[1], h0),
                             tk.packed_view(out, cap * E, shards=S), n_lay, stride * E, R, lens, hc, window)
        torch.cuda.synchronize()
        got = to_host(out)
        for z in range(n_lay):
            want = rs.move_layer(rs.View(rs.POOL, src_h, 1 + z, wl.block_tables, h0),
                                 rs.View(rs.PACKED, np.full(S * cap, SENTINEL, dtype=np.int16).view(src_h.dtype),
                                         shards=S, shard_elems=cap), lens_r, hc, window)
            assert np.array_equal(got[z * stride:z * stride + S * cap], want), f"R={R} pack layer {z}"
            assert (got[z * stride + S * cap:(z + 1) * stride].view(np.int16) == SENTINEL).all(), \
                f"R={R} layer {z}: slack between layers written"
        # the packed layers back into pool layers 0.. of the destination
        back = dst.clone()
        tk.topkv_move_layers(tk.packed_view(out, cap * E, shards=S),
                             tk.pool_view(back, 0, bt2, bt2.shape[1], h0), n_lay, stride * E, R, lens, hc, window)
        # pool to pool: source layers 1.., destination layers 0..
        rb = dst.clone()
        tk.topkv_move_layers(tk.pool_view(src, 1, bt, bt.shape[1]), tk.pool_view(rb, 0, bt2, bt2.shape[1]),
                             n_lay, 0, R, lens, H, window)
        torch.cuda.synchronize()
        want_back, want_rb = dst_h.copy(), dst_h.copy()
        for z in range(n_lay):
            rs.move_layer(rs.View(rs.PACKED, got[z * stride:z * stride + S * cap], shards=S, shard_elems=cap),
                          rs.View(rs.POOL, want_back, z, wl.dst_block_tables, h0), lens_r, hc, window)
            rs.move_layer(rs.View(rs.POOL, src_h, 1 + z, wl.block_tables, 0),
                          rs.View(rs.POOL, want_rb, z, wl.dst_block_tables, 0), lens_r, H, window)
        assert np.array_equal(to_host(back), want_back), f"R={R}: unpacked layers differ"
        assert np.array_equal(to_host(rb), want_rb), f"R={R}: re-blocked layers differ"


def test_fullsize_70b_move_layers(tk):
    """70B, 4096 tokens, all 80 layers in one call (three grids of 27, 27 and
    26 layers): both tensor-parallel shards of every layer equal the
    per-layer shards calls, the unpack of those shards equals the per-layer
    unpacks, and the pool-to-pool re-block (page 16 -> 64) equals the
    per-layer re-block; one layer of each against the oracle."""
    wl = make_workload("llama3-70b-4k", dst_page_size=64)
    say(f"[reshard] move_layers full size: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    n, L = int(wl.seq_lens[0]), wl.num_layers
    half = 2 * n * 4 * 128                                    # one shard of one layer, int16 words
    layer_words = 2 * half
    assert tk.topkv_engine_layers_per_grid(L, layer_words * 2) == 27
    many = torch.empty(L * layer_words, dtype=torch.int16, device="cuda")
    tk.topkv_move_layers(tk.pool_view(src, 0, bt, bt.shape[1]), tk.packed_view(many, half * 2, shards=2), L,
                         layer_words * 2, 1, lens, 8)
    one = torch.empty(layer_words, dtype=torch.int16, device="cuda")
    for layer in range(L):
        tk.topkv_pack_layer_shards(src, layer, 1, bt, bt.shape[1], lens, 0, 8, 2, one)
        assert torch.equal(many[layer * layer_words:(layer + 1) * layer_words], one), f"shards layer {layer}"
    want = oracle.pack_layer(to_host(src[40])[None], 0, wl.block_tables, wl.seq_lens).reshape(2, n, 8, 128)
    got = to_host(many[40 * layer_words:41 * layer_words]).reshape(2, 2, n, 4, 128)   # shard, plane, token
    assert np.array_equal(np.concatenate([got[0], got[1]], axis=-2), want), "layer 40 shards vs oracle"
    # the shards back into a second pool (page 64) in one call, and layer by layer
    a, b = dst.clone(), dst.clone()
    tk.topkv_move_layers(tk.packed_view(many, half * 2, shards=2), tk.pool_view(a, 0, bt2, bt2.shape[1]), L,
                         layer_words * 2, 1, lens, 8)
    for layer in range(L):
        tk.topkv_unpack_layer_shards(many[layer * layer_words:], b, layer, 1, bt2, bt2.shape[1], lens, 0, 8, 2,
                                     shard_bytes=half * 2)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16)), "unpacked shards differ from per-layer unpacks"
    # pool to pool, every layer
    tk.topkv_move_layers(tk.pool_view(src, 0, bt, bt.shape[1]), tk.pool_view(a, 0, bt2, bt2.shape[1]), L, 0, 1,
                         lens, 8)
    for layer in range(L):
        tk.topkv_reblock_layer(src, layer, bt, bt.shape[1], b, layer, bt2, bt2.shape[1], 1, lens)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16)), "re-blocked layers differ from per-layer re-blocks"
    again = oracle.pack_layer(to_host(a[79])[None], 0, wl.dst_block_tables, wl.seq_lens)
    assert np.array_equal(again, oracle.pack_layer(to_host(src[79])[None], 0, wl.block_tables, wl.seq_lens))
    del src, dst, a, b, many, one
    torch.cuda.empty_cache()

"""HIP path vs the CPU oracle, element by element, through the C ABI.

Small cases run every layer of seeded pools shaped like the five workloads
(reduced in layers or lengths so the oracle finishes in seconds, while still
spanning many tiles and ragged last pages), plus edge cases.  Bar: bit-exact
(the operation moves opaque words)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import (host_dst_prefill, host_src_pool, make_workload,
                                            random_words)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _scaled(name, div, **kw):
    base = make_workload(name)
    lens = np.maximum(base.seq_lens // div, 1)
    return make_workload(name, seq_lens=lens, **kw)


SMALL = {
    "tiny": lambda: make_workload("tiny"),
    "tiny-p16-to-p48": lambda: make_workload("tiny", dst_page_size=48),
    "tiny-p16-to-p1": lambda: make_workload("tiny", dst_page_size=1),
    "llama3-8b-2layers": lambda: make_workload("llama3-8b", num_layers=2, num_pages=600, dst_num_pages=700),
    "llama3-70b-batch8-div6": lambda: _scaled("llama3-70b-batch8", 6, num_layers=2),
    "deepseek-v3-mla-div16": lambda: _scaled("deepseek-v3-mla", 16, num_layers=2),
    "reblock-70b-div32": lambda: _scaled("reblock-70b", 32, num_layers=3, phys_layers=3),
    "reblock-p64-to-p16": lambda: _scaled("reblock-70b", 64, num_layers=2, phys_layers=2, page_size=64,
                                          dst_page_size=16),
    "odd-row-6B": lambda: make_workload("tiny", num_heads=1, head_dim=3, seq_lens=[40, 0, 7, 33]),
    "odd-row-5B-u8": lambda: make_workload("tiny", num_heads=1, head_dim=5, elem_bytes=1, seq_lens=[19, 64]),
    "row-12B-u32": lambda: make_workload("tiny", num_heads=1, head_dim=3, elem_bytes=4, seq_lens=[5, 77]),
    "row-24B-u64": lambda: make_workload("tiny", num_heads=3, head_dim=1, elem_bytes=8, seq_lens=[31, 2, 17]),
    # page planes of 6 KiB and 7.75 KiB: direct grids run 128-thread workgroups below 8 KiB planes, with a
    # ragged second tile here; 8 KiB planes switch back to 256 threads
    "plane-6k": lambda: make_workload("tiny", num_heads=3, seq_lens=[64, 48, 33, 17, 1]),
    "plane-7.75k": lambda: make_workload("tiny", num_heads=1, head_dim=248, seq_lens=[64, 31, 16]),
    "plane-8k": lambda: make_workload("tiny", num_heads=4, seq_lens=[64, 40, 9]),
    "page256-big-planes": lambda: make_workload("llama3-8b", num_layers=1, page_size=256, dst_page_size=16,
                                                seq_lens=[1000, 513, 256]),
}


def _sweep_and_check(tk, wl, src_h, dst_h, label):
    """Batched pack of every layer, then batched unpack; both vs the oracle."""
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2 = to_dev(wl.block_tables), to_dev(wl.dst_block_tables)
    lens = to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    want_dst = dst_h.copy()
    for layer in range(wl.num_layers):
        slab = layer % wl.phys_layers
        # sentinel-filled packed buffer with a tail guard: nothing may be written past the batch
        packed = torch.full((nbytes // wl.elem_bytes + 64,), -7, dtype=src.dtype, device="cuda")
        tk.topkv_pack_layer_batched(src, slab, wl.num_reqs, bt, bt.shape[1], lens, packed,
                                    dst_bytes=nbytes)
        tk.topkv_unpack_layer_batched(packed, dst, slab, wl.num_reqs, bt2, bt2.shape[1], lens,
                                      src_bytes=nbytes)
        torch.cuda.synchronize()
        got = to_host(packed)
        want = oracle.pack_layer(src_h, slab, wl.block_tables, wl.seq_lens)
        assert np.array_equal(got[:want.size], want), \
            f"{label}: pack layer {layer}: {int((got[:want.size] != want).sum())} of {want.size} differ"
        assert (got[want.size:].view(SIGNED_OF[got.itemsize]) == -7).all(), f"{label}: write past the batch"
        oracle.unpack_layer(want, want_dst, slab, wl.dst_block_tables, wl.seq_lens)
        got_dst = to_host(dst)
        assert np.array_equal(got_dst[slab], want_dst[slab]), \
            f"{label}: unpack layer {layer}: {int((got_dst[slab] != want_dst[slab]).sum())} elements differ"
    return src, dst


SIGNED_OF = {1: np.int8, 2: np.int16, 4: np.int32, 8: np.int64}


@pytest.mark.parametrize("case", sorted(SMALL))
def test_parity_batched(tk, case):
    wl = SMALL[case]()
    say(f"[parity_batched] {case}: {wl.describe()}")
    _sweep_and_check(tk, wl, host_src_pool(wl), host_dst_prefill(wl), case)


@pytest.mark.parametrize("short", [False, True], ids=["exact_cap", "cap_one_word_short"])
def test_uneven_batch_hostile(tk, short):
    """A batch whose requests differ widely in length (one of 512 pages, the
    rest 0 to 129 pages): the direct grid's slots past each short request's
    pages move nothing, invalid table entries deep in the long requests are
    skipped, a capacity one word short leaves the last request unmoved, and
    an unpack through a table with invalid entries writes nothing for them;
    all else equals the oracle."""
    lens = [8192, 0, 1, 17, 16, 33, 2049, 100]
    wl = make_workload("llama3-70b-batch8", num_layers=1, seq_lens=lens, seed=13)
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    P, NP, H, D = wl.page_size, wl.num_pages, wl.num_heads, wl.head_dim
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    cap = nbytes - 2 if short else nbytes
    bt = wl.block_tables.copy()
    assert bt.shape[1] == 512
    say(f"[uneven_batch] {wl.describe()} cap {'short' if short else 'exact'}")
    bad = [(0, 100), (0, 301), (0, 511), (6, 128)]            # entries deep in the two long requests
    bt[0, 100], bt[0, 301], bt[0, 511], bt[6, 128] = -1, NP, -9, NP + 5
    packed = torch.full((nbytes // 2 + 64,), 0x2B2B, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer_batched(src, 0, wl.num_reqs, to_dev(bt), bt.shape[1], to_dev(wl.seq_lens), packed,
                                dst_bytes=cap)
    torch.cuda.synchronize()
    got = to_host(packed)
    want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens).copy()
    row_words = wl.planes * H * D
    offs = np.concatenate([[0], np.cumsum(wl.seq_lens.astype(np.int64) * row_words)])
    for r, i in bad:
        n = int(wl.seq_lens[r])
        for c in range(wl.planes):
            want[offs[r] + (c * n + i * P) * H * D:offs[r] + (c * n + min(n, (i + 1) * P)) * H * D] = 0x2B2B
    if short:
        want[offs[-2]:] = 0x2B2B                                # the last request's block would cross the end
    assert np.array_equal(got[:want.size], want), f"pack: {int((got[:want.size] != want).sum())} words differ"
    assert (got[want.size:] == 0x2B2B).all(), "write past the batch"
    # unpack of the oracle's batch through a destination table with invalid entries in the long requests
    full = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens)
    bt2 = wl.dst_block_tables.copy()
    keep = {(0, 200): bt2[0, 200], (6, 120): bt2[6, 120]}
    bt2[0, 200], bt2[6, 120] = -3, wl.dst_num_pages
    tk.topkv_unpack_layer_batched(torch.from_numpy(full.view(np.int16)).cuda(), dst, 0, wl.num_reqs, to_dev(bt2),
                                  bt2.shape[1], to_dev(wl.seq_lens), src_bytes=cap)
    torch.cuda.synchronize()
    want_dst = dst_h.copy()
    saved = {k: want_dst[0, v].copy() for k, v in keep.items()}
    lens_used = wl.seq_lens.copy()
    if short:
        lens_used[-1] = 0                                       # not moved: its block crosses the capacity
    oracle.unpack_layer(full[:offs[-2]] if short else full, want_dst, 0, wl.dst_block_tables, lens_used)
    for k, v in keep.items():
        want_dst[0, v] = saved[k]
    assert np.array_equal(to_host(dst), want_dst), "unpack differs from the oracle"


@pytest.mark.parametrize("case", ["tiny", "deepseek-v3-mla-div16", "reblock-70b-div32", "odd-row-5B-u8"])
def test_parity_single_request(tk, case):
    """topkv_pack_layer / topkv_unpack_layer, one call per request."""
    wl = SMALL[case]()
    say(f"[parity_single] {case}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    want_dst = dst_h.copy()
    layer = wl.phys_layers - 1
    for r in range(wl.num_reqs):
        n = int(wl.seq_lens[r])
        k, k2 = -(-n // wl.page_size), -(-n // wl.dst_page_size)
        bt = to_dev(wl.block_tables[r, :max(k, 1)])
        bt2 = to_dev(wl.dst_block_tables[r, :max(k2, 1)])
        nbytes = tk.topkv_packed_layer_bytes(src, [n])
        packed = torch.empty(max(nbytes // wl.elem_bytes, 1), dtype=src.dtype, device="cuda")
        tk.topkv_pack_layer(src, layer, bt, n, packed)
        tk.topkv_unpack_layer(packed, dst, layer, bt2, n)
        torch.cuda.synchronize()
        want = oracle.pack_request(src_h, layer, wl.block_tables[r], n).reshape(-1)
        assert np.array_equal(to_host(packed)[:want.size], want), f"{case}: request {r} pack differs"
        oracle.unpack_request(want, want_dst, layer, wl.dst_block_tables[r], n)
    assert np.array_equal(to_host(dst), want_dst), f"{case}: single-request unpack differs"


@pytest.mark.parametrize("P", [16, 64])
def test_edge_lengths(tk, P):
    """Lengths 0, 1, P-1, P, P+1, 2P with a zero-length request mid-batch."""
    lens = [0, 1, P - 1, 0, P, P + 1, 2 * P, 3]
    wl = make_workload("tiny", seq_lens=lens, page_size=P, dst_page_size=16)
    say(f"[edge_lengths] P={P} lens={lens}")
    _sweep_and_check(tk, wl, host_src_pool(wl), host_dst_prefill(wl), f"edge P={P}")


def test_one_page_pool(tk):
    for n in (1, 7, 16):
        wl = make_workload("tiny", seq_lens=[n], num_pages=1, dst_num_pages=1)
        say(f"[one_page_pool] n={n}")
        _sweep_and_check(tk, wl, host_src_pool(wl), host_dst_prefill(wl), f"one-page n={n}")


def test_bit_patterns(tk):
    """Every 16-bit pattern (NaN payloads, -0, Inf, subnormals) survives."""
    wl = make_workload("tiny", seed=9, dst_page_size=64)
    rng = np.random.default_rng(123)
    src_h = random_words(rng, wl.pool_shape(), 2)
    src_h.reshape(-1)[:65536] = np.arange(65536, dtype=np.uint16)   # all patterns present
    say("[bit_patterns]")
    _sweep_and_check(tk, wl, src_h, host_dst_prefill(wl), "bit patterns")


def test_misaligned_packed_buffer(tk):
    """A packed buffer 2 bytes off 16-byte alignment takes the narrow-vector path."""
    wl = make_workload("tiny", seed=4)
    say("[misaligned_packed]")
    src_h = host_src_pool(wl)
    src = to_dev(src_h)
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    raw = torch.zeros(nbytes + 64, dtype=torch.uint8, device="cuda")
    base = raw.data_ptr() + 2
    tk.topkv_pack_layer_batched(src, 1, wl.num_reqs, bt, bt.shape[1], lens, base, dst_bytes=nbytes)
    torch.cuda.synchronize()
    got = raw.cpu().numpy()[2:2 + nbytes].view(np.uint16)
    assert np.array_equal(got, oracle.pack_layer(src_h, 1, wl.block_tables, wl.seq_lens))
    assert (raw.cpu().numpy()[:2] == 0).all() and (raw.cpu().numpy()[2 + nbytes:] == 0).all()


def test_untrusted_device_inputs(tk):
    """Out-of-range table entries are skipped, lengths are clamped to the
    table width, and a batch that overruns the packed buffer's capacity is
    not moved; nothing outside the buffers is touched."""
    wl = make_workload("tiny", seed=5)
    say("[untrusted_inputs]")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    P, NP = wl.page_size, wl.num_pages
    row_words = wl.planes * wl.num_heads * wl.head_dim          # words per token over both planes
    lens = wl.seq_lens
    nbytes = tk.topkv_packed_layer_bytes(src, lens)
    # (a) request 1 page 0 -> NP (invalid), request 2 page 1 -> -1
    bad = wl.block_tables.copy()
    bad[1, 0] = NP
    bad[2, 1] = -1
    packed = torch.full((nbytes // 2,), 0x5A5A, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer_batched(src, 0, wl.num_reqs, to_dev(bad), bad.shape[1],
                                to_dev(lens), packed, dst_bytes=nbytes)
    torch.cuda.synchronize()
    got = to_host(packed)
    want = oracle.pack_layer(src_h, 0, wl.block_tables, lens).copy()
    offs = np.concatenate([[0], np.cumsum(lens.astype(np.int64) * row_words)])
    H, D = wl.num_heads, wl.head_dim
    for r, i in ((1, 0), (2, 1)):
        n = int(lens[r])
        for c in range(wl.planes):
            a = offs[r] + (c * n + i * P) * H * D
            b = offs[r] + (c * n + min(n, (i + 1) * P)) * H * D
            want[a:b] = 0x5A5A
    assert np.array_equal(got, want)
    # (b) a length beyond bt_stride * P is clamped to it
    long_lens = lens.copy()
    long_lens[3] = 10_000
    clamped = lens.copy()
    clamped[3] = wl.block_tables.shape[1] * P
    need = tk.topkv_packed_layer_bytes(src, clamped)
    packed2 = torch.zeros(need // 2, dtype=torch.int16, device="cuda")
    full_bt = wl.block_tables.copy()
    free = sorted(set(range(NP)) - set(full_bt[full_bt >= 0].tolist()))
    full_bt[3, 2:] = free[:full_bt.shape[1] - 2]
    tk.topkv_pack_layer_batched(src, 1, wl.num_reqs, to_dev(full_bt), full_bt.shape[1],
                                to_dev(long_lens), packed2, dst_bytes=need)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(packed2), oracle.pack_layer(src_h, 1, full_bt, clamped))
    # (c) capacity one word short: the last request is not moved, earlier ones are
    packed3 = torch.full((nbytes // 2,), 0x1111, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer_batched(src, 0, wl.num_reqs, to_dev(wl.block_tables),
                                wl.block_tables.shape[1], to_dev(lens), packed3,
                                dst_bytes=nbytes - 2)
    torch.cuda.synchronize()
    got3 = to_host(packed3)
    full = oracle.pack_layer(src_h, 0, wl.block_tables, lens)
    assert np.array_equal(got3[:offs[-2]], full[:offs[-2]])
    assert (got3[offs[-2]:] == 0x1111).all()
    # (d) unpack through a table with an invalid entry writes nothing for it
    bad2 = wl.dst_block_tables.copy()
    bad2[0, 1] = -5
    tk.topkv_unpack_layer_batched(torch.from_numpy(full.view(np.int16)).cuda(), dst, 0, wl.num_reqs,
                                  to_dev(bad2), bad2.shape[1], to_dev(lens),
                                  src_bytes=nbytes)
    torch.cuda.synchronize()
    want_dst = dst_h.copy()
    keep = want_dst[0, wl.dst_block_tables[0, 1]].copy()
    oracle.unpack_layer(full, want_dst, 0, wl.dst_block_tables, lens)
    want_dst[0, wl.dst_block_tables[0, 1]] = keep
    assert np.array_equal(to_host(dst), want_dst)


@pytest.mark.parametrize("n", [100, 10_000, -3, 0, 1, 127])
def test_one_request_device_length(tk, n):
    """One request with a device length and 1 KiB rows (4 heads x 128 x
    2 bytes): with a packed buffer sized for the whole block table the move
    runs the layout-move kernel's one-request grid, one vector short of that
    the per-page kernel.  Both must skip out-of-range table entries, clamp
    the length to the table (negative counts as zero) and leave a request
    that overruns the buffer unmoved."""
    P, W, NP, layer = 16, 8, 40, 1
    wl = make_workload("tiny", seed=11, num_heads=4, head_dim=128, seq_lens=[100], num_pages=NP, dst_num_pages=NP)
    C, H, D = wl.planes, wl.num_heads, wl.head_dim
    row = C * H * D                                        # words per token over both planes
    rng = np.random.default_rng(31)
    good, good2 = (rng.permutation(NP)[:W].astype(np.int32) for _ in range(2))
    spare = [p for p in range(NP) if p not in set(good2.tolist())][0]
    bad, bad2 = good.copy(), good2.copy()
    bad[2], bad[5] = -1, NP
    bad2[3] = -7
    clamp = min(max(n, 0), W * P)
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src = to_dev(src_h)
    lens = to_dev(np.array([n], dtype=np.int32))
    packed_want = oracle.pack_layer(src_h, layer, good[None], np.array([clamp], np.int32))
    full = W * P * row * 2                                 # bytes for the whole table
    for cap in (full, full - 16):
        say(f"[one_request] n={n} cap={cap}")
        moved = clamp * row * 2 <= cap
        sentinel = 0x2B2B
        packed = torch.full((full // 2,), sentinel, dtype=torch.int16, device="cuda")
        tk.topkv_pack_layer_batched(src, layer, 1, to_dev(bad), W, lens, packed, dst_bytes=cap)
        torch.cuda.synchronize()
        want = np.full(full // 2, sentinel, dtype=np.uint16)
        if moved:
            want[:packed_want.size] = packed_want
            blk = want[:packed_want.size].reshape(C, clamp, H * D)
            for i in (2, 5):
                blk[:, i * P:(i + 1) * P] = sentinel
        assert np.array_equal(to_host(packed).view(np.uint16), want), f"n={n} cap={cap}: pack differs"

        dst = to_dev(dst_h)
        src_packed = np.zeros(full // 2, dtype=np.uint16)
        src_packed[:packed_want.size] = packed_want
        tk.topkv_unpack_layer_batched(to_dev(src_packed), dst, layer, 1, to_dev(bad2), W, lens, src_bytes=cap)
        torch.cuda.synchronize()
        want_dst = dst_h.copy()
        if moved:
            tbl = good2.copy()
            tbl[3] = spare
            keep = want_dst[layer, spare].copy()
            oracle.unpack_layer(packed_want, want_dst, layer, tbl[None], np.array([clamp], np.int32))
            want_dst[layer, spare] = keep
        assert np.array_equal(to_host(dst), want_dst), f"n={n} cap={cap}: unpack differs"


@pytest.mark.parametrize("n,P2", [(117, 16), (117, 64), (128, 16), (1, 16)])
def test_one_request_host_length_hostile(tk, n, P2):
    """topkv_pack_layer / topkv_unpack_layer (host length) through tables with
    out-of-range entries: pack leaves those pages' rows of the packed buffer
    alone, unpack reads the packed rows but writes nothing for a bad
    destination page; every other row moves."""
    P, NP, layer = 16, 40, 1
    wl = make_workload("tiny", seed=13, num_heads=4, head_dim=128, seq_lens=[n], num_pages=NP,
                       dst_page_size=P2, dst_num_pages=NP)
    C, H, D = wl.planes, wl.num_heads, wl.head_dim
    k, k2 = -(-n // P), -(-n // P2)
    rng = np.random.default_rng(n + P2)
    good, good2 = rng.permutation(NP)[:k].astype(np.int32), rng.permutation(NP)[:k2].astype(np.int32)
    bad, bad2 = good.copy(), good2.copy()
    bad[k // 2] = -1 if k > 1 else NP
    bad2[-1] = NP + 3
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    say(f"[one_request_host] n={n} P'={P2}")
    sentinel = 0x4D4D
    nwords = C * n * H * D
    packed = torch.full((nwords,), sentinel, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer(src, layer, to_dev(bad), n, packed)
    torch.cuda.synchronize()
    want = oracle.pack_layer(src_h, layer, good[None], np.array([n], np.int32)).copy()
    blk = want.reshape(C, n, H * D)
    i = k // 2
    blk[:, i * P:min(n, (i + 1) * P)] = sentinel
    assert np.array_equal(to_host(packed).view(np.uint16), want), f"n={n}: pack differs"

    full = oracle.pack_layer(src_h, layer, good[None], np.array([n], np.int32))
    tk.topkv_unpack_layer(to_dev(full), dst, layer, to_dev(bad2), n)
    torch.cuda.synchronize()
    want_dst = dst_h.copy()
    spare = [p for p in range(NP) if p not in set(good2.tolist())][0]
    tbl = good2.copy()
    tbl[-1] = spare
    keep = want_dst[layer, spare].copy()
    oracle.unpack_layer(full, want_dst, layer, tbl[None], np.array([n], np.int32))
    want_dst[layer, spare] = keep
    assert np.array_equal(to_host(dst), want_dst), f"n={n} P'={P2}: unpack differs"


@pytest.mark.parametrize("offset", [2, 8])
def test_one_request_misaligned_packed(tk, offset):
    """The one-request grid with a packed buffer `offset` bytes off 16-byte
    alignment (2- and 8-byte pieces): pack and unpack equal the oracle, and
    nothing outside the batch is written."""
    P, W, NP, layer, n = 16, 8, 40, 0, 117
    wl = make_workload("tiny", seed=12, num_heads=4, head_dim=128, seq_lens=[n], num_pages=NP, dst_num_pages=NP)
    row = wl.planes * wl.num_heads * wl.head_dim              # words per token over both planes
    rng = np.random.default_rng(offset)
    bt, bt2 = (rng.permutation(NP)[:W].astype(np.int32)[None] for _ in range(2))
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    lens = to_dev(np.array([n], dtype=np.int32))
    full = W * P * row * 2                                     # bytes for the whole table: the routed grid
    say(f"[one_request_misaligned] offset {offset}")
    raw = torch.zeros(full + 64, dtype=torch.uint8, device="cuda")
    base = raw.data_ptr() + offset
    tk.topkv_pack_layer_batched(src, layer, 1, to_dev(bt), W, lens, base, dst_bytes=full)
    torch.cuda.synchronize()
    want = oracle.pack_layer(src_h, layer, bt, np.array([n], np.int32))
    got = raw.cpu().numpy()
    assert np.array_equal(got[offset:offset + want.nbytes].view(np.uint16), want)
    assert (got[:offset] == 0).all() and (got[offset + want.nbytes:] == 0).all()
    tk.topkv_unpack_layer_batched(base, dst, layer, 1, to_dev(bt2), W, lens, src_bytes=full)
    torch.cuda.synchronize()
    oracle.unpack_layer(want, dst_h, layer, bt2, np.array([n], np.int32))
    assert np.array_equal(to_host(dst), dst_h)


def _persistent_case(kind):
    rng = np.random.default_rng(21 if kind == "many-requests" else 22)
    if kind == "many-requests":             # more requests than one direct grid takes
        lens = rng.integers(0, 41, size=1100)
    else:                                   # more than 2^20 (request, entry, plane) slots: 600 x 1000 x 2
        lens = np.concatenate([[16000], rng.integers(0, 21, size=599)])
    return make_workload("tiny", num_layers=1, seq_lens=lens.astype(np.int32))


@pytest.mark.parametrize("kind", ["many-requests", "many-slots"])
@pytest.mark.parametrize("window", [0, 7])
def test_persistent_grid(tk, kind, window):
    """Batches beyond the direct grid's limits run the persistent grid (length
    scan, request search); pack and unpack, with and without a window, equal
    the oracle."""
    wl = _persistent_case(kind)
    say(f"[persistent] {kind}: {wl.num_reqs} requests, table width {wl.block_tables.shape[1]}, window {window}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    n = oracle.packed_layer_elems(wl.planes, wl.num_heads, wl.head_dim, wl.seq_lens, window)
    packed = torch.full((n + 64,), 0x1357, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer_window(src, 0, wl.num_reqs, bt, bt.shape[1], lens, window, packed, dst_bytes=2 * n)
    tk.topkv_unpack_layer_window(packed, dst, 0, wl.num_reqs, bt2, bt2.shape[1], lens, window, src_bytes=2 * n)
    torch.cuda.synchronize()
    want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens, window=window)
    got = to_host(packed)
    assert np.array_equal(got[:n], want), f"{kind} window {window}: pack differs"
    assert (got[n:] == 0x1357).all(), "write past the batch"
    oracle.unpack_layer(want, dst_h, 0, wl.dst_block_tables, wl.seq_lens, window=window)
    assert np.array_equal(to_host(dst), dst_h), f"{kind} window {window}: unpack differs"


@pytest.mark.parametrize("window", [0, 7])
def test_max_batch(tk, window):
    """Exactly TOPKV_MAX_BATCH_REQS requests in one launch (the largest batch
    the header accepts; its per-request prefix sums fill the most LDS): the
    fast pack/unpack and the layout move (a head slice, packed and unpacked)
    equal the oracles; one request more is refused before any launch."""
    import oracle.reshard as rs
    R = tk.TOPKV_MAX_BATCH_REQS
    rng = np.random.default_rng(31)
    lens = rng.integers(0, 41, size=R).astype(np.int32)
    lens[rng.integers(0, R, size=64)] = 0            # empty requests scattered through the batch
    wl = make_workload("tiny", num_layers=1, num_heads=4, seq_lens=lens)
    say(f"[max batch] {wl.num_reqs} requests, {int(lens.sum())} tokens, window {window}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, dlens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    n = oracle.packed_layer_elems(wl.planes, wl.num_heads, wl.head_dim, wl.seq_lens, window)
    packed = torch.full((n + 64,), 0x2468, dtype=torch.int16, device="cuda")
    tk.topkv_pack_layer_window(src, 0, R, bt, bt.shape[1], dlens, window, packed, dst_bytes=2 * n)
    tk.topkv_unpack_layer_window(packed, dst, 0, R, bt2, bt2.shape[1], dlens, window, src_bytes=2 * n)
    torch.cuda.synchronize()
    want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens, window=window)
    got = to_host(packed)
    assert np.array_equal(got[:n], want), "pack differs"
    assert (got[n:] == 0x2468).all(), "write past the batch"
    want_dst = dst_h.copy()
    oracle.unpack_layer(want, want_dst, 0, wl.dst_block_tables, wl.seq_lens, window=window)
    assert np.array_equal(to_host(dst), want_dst), "unpack differs"

    h0, hc = 1, 2
    nh = rs.packed_heads_elems(wl.planes, hc, wl.head_dim, wl.seq_lens, window)
    half = torch.full((nh + 64,), 0x2468, dtype=torch.int16, device="cuda")
    tk.topkv_move_layer(tk.pool_view(src, 0, bt, bt.shape[1], head_begin=h0), tk.packed_view(half, 2 * nh),
                        R, dlens, hc, window)
    tk.topkv_move_layer(tk.packed_view(half, 2 * nh), tk.pool_view(dst, 0, bt2, bt2.shape[1], head_begin=h0),
                        R, dlens, hc, window)
    torch.cuda.synchronize()
    want_h = rs.pack_layer_heads(src_h, 0, wl.block_tables, wl.seq_lens, h0, hc, window)
    got_h = to_host(half)
    assert np.array_equal(got_h[:nh], want_h), "head-slice pack differs"
    assert (got_h[nh:] == 0x2468).all(), "head-slice write past the batch"
    rs.unpack_layer_heads(want_h, want_dst, 0, wl.dst_block_tables, wl.seq_lens, h0, hc, window)
    assert np.array_equal(to_host(dst), want_dst), "head-slice unpack differs"

    with pytest.raises(tk.TopkvError) as ei:
        tk.topkv_pack_layer_window(src, 0, R + 1, bt, bt.shape[1], dlens, window, packed, dst_bytes=2 * n)
    assert ei.value.status == tk.TOPKV_ERR_UNSUPPORTED


def test_widest_table(tk):
    """One request through a block table of 2^27 - 1 entries at page size 16:
    the launch's token capacity (table width x page size) is 2^31 - 16, the
    largest a launch accepts.  Only the request's own pages are read; pack and
    unpack equal the oracle.  A table one entry wider is refused before any
    launch."""
    wl = make_workload("tiny", num_layers=1, seq_lens=[100, 37])
    width = (1 << 27) - 1
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    say(f"[widest table] {wl.num_reqs} requests, table width {width} (int32, {4 * width * wl.num_reqs >> 20} MiB)")
    bt = torch.full((wl.num_reqs, width), -1, dtype=torch.int32, device="cuda")
    bt2 = torch.full((wl.num_reqs, width), -1, dtype=torch.int32, device="cuda")
    k = wl.block_tables.shape[1]
    bt[:, :k] = to_dev(wl.block_tables)
    bt2[:, :wl.dst_block_tables.shape[1]] = to_dev(wl.dst_block_tables)
    lens = to_dev(wl.seq_lens)
    want = oracle.pack_layer(src_h, 0, wl.block_tables, wl.seq_lens)
    want_dst = dst_h.copy()
    oracle.unpack_layer(want, want_dst, 0, wl.dst_block_tables, wl.seq_lens)
    for r in range(wl.num_reqs):            # one request per launch keeps the capacity at 2^31 - 16
        size = int(wl.seq_lens[r]) * wl.planes * wl.num_heads * wl.head_dim       # elements of request r
        off = int(wl.seq_lens[:r].sum()) * wl.planes * wl.num_heads * wl.head_dim
        packed = torch.full((size + 64,), 0x1111, dtype=torch.int16, device="cuda")
        tk.topkv_pack_layer_batched(src, 0, 1, bt[r], width, lens[r:r + 1], packed, dst_bytes=2 * size)
        tk.topkv_unpack_layer_batched(packed, dst, 0, 1, bt2[r], width, lens[r:r + 1], src_bytes=2 * size)
        torch.cuda.synchronize()
        got = to_host(packed)
        assert np.array_equal(got[:size], want[off:off + size]), f"request {r}: pack differs"
        assert (got[size:] == 0x1111).all(), f"request {r}: write past the request"
    assert np.array_equal(to_host(dst), want_dst), "unpack differs"
    with pytest.raises(tk.TopkvError) as ei:
        tk.topkv_pack_layer_batched(src, 0, 1, bt[0], width + 1, lens[0:1], packed, dst_bytes=2 * size)
    assert ei.value.status == tk.TOPKV_ERR_UNSUPPORTED

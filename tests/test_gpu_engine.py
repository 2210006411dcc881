"""Layer engine (topkv_engine_pack_layers / topkv_engine_unpack_layers): one
launch moves a range of layers, each exactly as the per-layer batched calls
would, and each only once its ready word allows (the paper's Section 5.2
layer-by-layer transfer).  Without ready words the launch is a hardware-
dispatched grid over every layer's slots; with them, a persistent grid.

Parity: every layer of the range against the CPU oracle (small shapes, and
the 80-layer 70B / 4096-token request at full size); the waits: layers held
back by their ready words are not touched, a timeout and a cancel from the
host end the launch with every workgroup exiting and the reason in the
status word, ready words set by the host one layer at a time are followed."""
import threading
import time

import numpy as np
import pytest
import torch

import oracle
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import (device_dst_prefill, device_src_pool, host_dst_prefill, host_src_pool,
                                            make_workload)

pytestmark = pytest.mark.gpu
SENTINEL = 0x5A5A


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _setup(tk, wl, host_pools=True):
    if host_pools:
        src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
        src, dst = to_dev(src_h), to_dev(dst_h)
    else:
        src, dst = device_src_pool(wl), device_dst_prefill(wl)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    return src, dst, bt, bt2, lens, nbytes


def _ring(L, nbytes, gap=512):
    """Packed blocks of L layers with a sentinel gap after each one."""
    stride = nbytes + gap
    buf = torch.full((L * stride // 2,), SENTINEL, dtype=torch.int16, device="cuda")
    return buf, stride


def _layer_words(buf, stride, z, nbytes):
    return to_host(buf)[z * stride // 2:(z * stride + nbytes) // 2]


def _gaps_untouched(buf, stride, L, nbytes):
    h = to_host(buf)
    return all(np.all(h[(z * stride + nbytes) // 2:(z + 1) * stride // 2] == SENTINEL) for z in range(L))


ENGINE_CASES = [
    (dict(name="tiny"), 0),
    (dict(name="tiny"), 1),
    (dict(name="tiny", dst_page_size=48), 2),
    (dict(name="tiny", dst_page_size=1), 0),
    (dict(name="llama3-70b-batch8", num_layers=3, seq_lens=[4096, 1000, 17, 0, 2049, 16, 33, 8192]), 0),
    (dict(name="deepseek-v3-mla", num_layers=3, seq_lens=[512, 4096, 65, 7000]), 4),
    (dict(name="reblock-70b", num_layers=2, seq_lens=[256, 4095, 999, 3000, 64]), 0),
    (dict(name="tiny", num_layers=3, num_heads=3, seq_lens=[64, 48, 33, 17, 1]), 0),     # 6 KiB planes
    (dict(name="tiny", num_layers=3, num_heads=1, head_dim=248, seq_lens=[64, 31, 16]), 0),   # 7.75 KiB
    (dict(name="llama3-70b-tp8", num_layers=5, seq_lens=[4096]), 0),                    # 4 KiB, one request
]


@pytest.mark.parametrize("waits", [False, True], ids=["direct", "persistent"])
@pytest.mark.parametrize("wl_kw,per_cu", ENGINE_CASES)
def test_engine_matches_oracle(tk, wl_kw, per_cu, waits):
    """Every layer of the range against the oracle, through both grids: no
    ready words (the hardware-dispatched grid over every layer's slots) and
    ready words that have all arrived (the persistent grid, with
    per_cu workgroups per compute unit)."""
    kw = dict(wl_kw)
    wl = make_workload(kw.pop("name"), **kw)
    say(f"[engine] {wl.describe()} {'persistent' if waits else 'direct'}, workgroups/CU {per_cu or 'default'}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    L, R = wl.num_layers, wl.num_reqs
    buf, stride = _ring(L, nbytes)
    ready = torch.full((L,), 9, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    opt = tk.engine_options(workgroups_per_cu=per_cu, **(dict(ready=ready, epoch=9, status=status,
                                                              timeout_us=1_000_000) if waits else {}))
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, buf, stride, engine=opt)
    tk.topkv_engine_unpack_layers(buf, stride, dst, 0, L, R, bt2, bt2.shape[1], lens, engine=opt)
    torch.cuda.synchronize()
    want_dst = dst_h.copy()
    for z in range(L):
        want = oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens)
        assert np.array_equal(_layer_words(buf, stride, z, nbytes), want), f"layer {z}: pack differs from the oracle"
        oracle.unpack_layer(want, want_dst, z, wl.dst_block_tables, wl.seq_lens)
    assert _gaps_untouched(buf, stride, L, nbytes), "bytes between layer blocks were written"
    assert np.array_equal(to_host(dst), want_dst), "unpacked pool differs from the oracle"
    assert int(status.item()) == 0


def test_engine_sub_range_and_one_layer(tk):
    """A range that starts past layer 0 touches only its own layers; one
    layer with layer_stride 0 is one batched launch's move."""
    wl = make_workload("tiny", num_layers=4)
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    R = wl.num_reqs
    buf, stride = _ring(2, nbytes)
    tk.topkv_engine_pack_layers(src, 1, 2, R, bt, bt.shape[1], lens, buf, stride)
    tk.topkv_engine_unpack_layers(buf, stride, dst, 2, 2, R, bt2, bt2.shape[1], lens)
    one = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    tk.topkv_engine_pack_layers(src, 3, 1, R, bt, bt.shape[1], lens, one, 0)
    torch.cuda.synchronize()
    want = [oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens) for z in range(4)]
    assert np.array_equal(_layer_words(buf, stride, 0, nbytes), want[1])
    assert np.array_equal(_layer_words(buf, stride, 1, nbytes), want[2])
    assert np.array_equal(to_host(one), want[3])
    want_dst = dst_h.copy()
    for z in (2, 3):     # pool layers 2 and 3 receive packed blocks 0 and 1
        oracle.unpack_layer(want[z - 1], want_dst, z, wl.dst_block_tables, wl.seq_lens)
    assert np.array_equal(to_host(dst), want_dst)


@pytest.mark.parametrize("per", [1, 2, 3, 0], ids=["grids1", "grids2", "grids3", "library"])
@pytest.mark.parametrize("short", [False, True], ids=["fit", "short_stride"])
def test_engine_grids_of_a_few_layers(tk, per, short):
    """A range issued as consecutive hardware-dispatched grids of `per`
    layers (0: the library's split, one grid at this size) moves every layer
    as one grid would.  With a layer stride one word short of a layer's
    packed batch, every layer - the first and last of each grid included,
    and a one-layer grid's - leaves its last request unmoved (its block
    would cross the layer's end), with the buffer sized past the last block
    so that only the stride bounds it."""
    wl = make_workload("llama3-70b-batch8", num_layers=7, seq_lens=[300, 17, 1000, 64, 33])
    say(f"[engine grids] {wl.describe()} layers per grid {per or 'library'}, short stride {short}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    L, R = wl.num_layers, wl.num_reqs
    stride = nbytes - 2 if short else nbytes + 512
    total = L * stride + 4096
    buf = torch.full((total // 2,), SENTINEL, dtype=torch.int16, device="cuda")
    opt = tk.engine_options(layers_per_grid=per)
    assert tk.topkv_engine_layers_per_grid(L, stride, opt) == (per or L)
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, buf, stride, packed_bytes=total, engine=opt)
    torch.cuda.synchronize()
    row_bytes = wl.planes * wl.num_heads * wl.head_dim * 2
    keep = (nbytes - int(wl.seq_lens[-1]) * row_bytes) if short else nbytes   # bytes of the requests moved
    h = to_host(buf)
    want_dst = dst_h.copy()
    for z in range(L):
        want = oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens)
        got = h[z * stride // 2:z * stride // 2 + min(stride, nbytes) // 2]
        assert np.array_equal(got[:keep // 2], want[:keep // 2]), f"layer {z}: moved requests differ from the oracle"
        assert (got[keep // 2:] == SENTINEL).all(), f"layer {z}: the request crossing the stride was moved"
        if not short:
            oracle.unpack_layer(want, want_dst, z, wl.dst_block_tables, wl.seq_lens)
    assert (h[(L - 1) * stride // 2 + min(stride, nbytes) // 2:] == SENTINEL).all(), "bytes past the last block"
    if not short:
        assert _gaps_untouched(buf[:L * stride // 2], stride, L, nbytes)
        tk.topkv_engine_unpack_layers(buf, stride, dst, 0, L, R, bt2, bt2.shape[1], lens, packed_bytes=total,
                                      engine=opt)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(dst), want_dst), "unpacked pool differs from the oracle"


def test_engine_fullsize_headline_every_layer(tk):
    """The 70B / 4096-token request at full size, all 80 layers in one engine
    call per direction (the benchmark's configuration: the library issues
    it as three grids of 27, 27 and 26 layers): every layer's packed block
    and every destination layer slab against the oracle."""
    wl = make_workload("llama3-70b-4k")
    say(f"[engine fullsize] {wl.describe()}")
    src, dst, bt, bt2, lens, nbytes = _setup(tk, wl, host_pools=False)
    L, R = wl.num_layers, wl.num_reqs
    packed = torch.empty((L, nbytes // 2), dtype=torch.int16, device="cuda")
    assert tk.topkv_engine_layers_per_grid(L, nbytes) == 27     # the grids meet at layers 27 and 54
    before = dst.clone()
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, packed, nbytes)
    tk.topkv_engine_unpack_layers(packed, nbytes, dst, 0, L, R, bt2, bt2.shape[1], lens)
    torch.cuda.synchronize()
    for z in range(L):
        want = oracle.pack_layer(to_host(src[z])[None], 0, wl.block_tables, wl.seq_lens)
        assert np.array_equal(to_host(packed[z]), want), f"layer {z}: pack differs from the oracle"
        want_dst = to_host(before[z])[None]
        oracle.unpack_layer(want, want_dst, 0, wl.dst_block_tables, wl.seq_lens)
        assert np.array_equal(to_host(dst[z]), want_dst[0]), f"layer {z}: unpacked slab differs from the oracle"
        if z % 20 == 0:
            say(f"  layer {z} bit-exact vs oracle")
    say(f"  all {L} layers bit-exact vs oracle ({nbytes} B per layer)")
    # the persistent grid (ready words all arrived) reproduces both directions bit for bit
    ready = torch.ones(L, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    opt = tk.engine_options(ready=ready, epoch=1, status=status, timeout_us=1_000_000)
    again, dst2 = torch.full_like(packed, SENTINEL), before
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, again, nbytes, engine=opt)
    tk.topkv_engine_unpack_layers(again, nbytes, dst2, 0, L, R, bt2, bt2.shape[1], lens, engine=opt)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(again, packed), "persistent grid: packed layers differ"
    assert torch.equal(dst2.view(torch.int16), dst.view(torch.int16)), "persistent grid: unpacked pool differs"
    say("  persistent grid: all layers equal")
    del src, dst, before, packed, again
    torch.cuda.empty_cache()


def test_engine_ready_words_hold_layers_back(tk):
    """Layers move in order: from the first layer whose ready word has not
    reached the epoch on, nothing is touched (later ready layers included);
    the launch gives up after the timeout with TOPKV_ERR_TIMEOUT and the
    layers before that one are moved in full.  The comparison with the epoch
    is modulo 2^32 (words just past a wrapping epoch count)."""
    wl = make_workload("llama3-70b-batch8", num_layers=6, seq_lens=[4096, 1000, 17, 2049])
    src_h = host_src_pool(wl)
    src = to_dev(src_h)
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    L, R = wl.num_layers, wl.num_reqs
    for epoch, words in ((7, [7, 9, 7, 6, 7, 7]), (0xFFFFFFF0, [0xFFFFFFF0, 0xFFFFFFF5, 3, 0xFFFFFFE0, 0, 0]),
                         (5, [5, 0xFFFFFFFF, 5, 5, 5, 5])):
        first_missing = next(z for z, w in enumerate(words) if ((w - epoch) & 0xFFFFFFFF) >= 1 << 31)
        ready = torch.tensor(np.array(words, dtype=np.uint32).view(np.int32), device="cuda")
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        buf, stride = _ring(L, nbytes)
        opt = tk.engine_options(ready=ready, epoch=epoch, status=status, timeout_us=20_000)
        t0 = time.perf_counter()
        tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, buf, stride, engine=opt)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        say(f"  epoch {epoch:#x}: layers 0..{first_missing - 1} ready, gave up after {dt * 1e3:.1f} ms")
        assert int(status.item()) == tk.TOPKV_ERR_TIMEOUT
        h = to_host(buf)
        for z in range(L):
            got = h[z * stride // 2:(z * stride + nbytes) // 2]
            if z < first_missing:
                assert np.array_equal(got, oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens)), f"layer {z}"
            else:
                assert np.all(got == SENTINEL), f"layer {z} was written before its ready word arrived"
        assert _gaps_untouched(buf, stride, L, nbytes)


def test_engine_follows_host_ready_words(tk):
    """Ready words in pinned host memory, published by a host thread one
    layer at a time while the engine runs: every layer is packed, then
    unpacked by a second engine launch that follows a second set of words."""
    wl = make_workload("llama3-70b-4k", num_layers=12)
    src, dst, bt, bt2, lens, nbytes = _setup(tk, wl, host_pools=False)
    L, R = wl.num_layers, wl.num_reqs
    src_h = to_host(src)
    before = to_host(dst)
    packed = torch.empty((L, nbytes // 2), dtype=torch.int16, device="cuda")
    ready = torch.zeros(2 * L, dtype=torch.int32, pin_memory=True)
    status = torch.zeros(2, dtype=torch.int32, device="cuda")
    epoch = 3
    pk = tk.engine_options(ready=ready[:L], epoch=epoch, status=status[0:1], timeout_us=5_000_000, workgroups_per_cu=2)
    up = tk.engine_options(ready=ready[L:], epoch=epoch, status=status[1:2], timeout_us=5_000_000, workgroups_per_cu=2)
    side = torch.cuda.Stream()
    t0 = time.perf_counter()
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, packed, nbytes, engine=pk)
    with torch.cuda.stream(side):
        tk.topkv_engine_unpack_layers(packed, nbytes, dst, 0, L, R, bt2, bt2.shape[1], lens, engine=up)
    ends = []

    def publish():
        for z in range(L):
            time.sleep(0.002)
            ready[z] = epoch                       # pack of layer z may start
        torch.cuda.current_stream().synchronize()  # every layer packed ...
        for z in range(L):
            ready[L + z] = epoch                   # ... so each may be unpacked
        ends.append(time.perf_counter())

    th = threading.Thread(target=publish)
    th.start()
    th.join(timeout=30)
    torch.cuda.synchronize()
    say(f"  {L} layers published over {(ends[0] - t0) * 1e3:.1f} ms, status {status.tolist()}")
    assert status.tolist() == [0, 0]
    want_dst = before.copy()
    for z in range(L):
        want = oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens)
        assert np.array_equal(to_host(packed[z]), want), f"layer {z}"
        oracle.unpack_layer(want, want_dst, z, wl.dst_block_tables, wl.seq_lens)
    assert np.array_equal(to_host(dst), want_dst)


def test_engine_cancel_from_host(tk):
    """A launch waiting for a word that never comes is cancelled from the
    host (a word in pinned host memory): it ends long before its timeout,
    status TOPKV_ERR_CANCELLED, nothing written."""
    wl = make_workload("llama3-70b-4k", num_layers=4)
    src, _, bt, _, lens, nbytes = _setup(tk, wl, host_pools=False)
    L, R = wl.num_layers, wl.num_reqs
    ready = torch.zeros(L, dtype=torch.int32, device="cuda")
    cancel = torch.zeros(1, dtype=torch.int32, pin_memory=True)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    buf, stride = _ring(L, nbytes)
    opt = tk.engine_options(ready=ready, epoch=1, status=status, cancel=cancel, timeout_us=4_000_000)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, buf, stride, engine=opt)
    time.sleep(0.1)
    cancel[0] = 1
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    say(f"  cancelled after {dt * 1e3:.1f} ms, status {int(status.item())}")
    assert int(status.item()) == tk.TOPKV_ERR_CANCELLED
    assert dt < 2.0
    assert np.all(to_host(buf) == SENTINEL)


@pytest.mark.parametrize("per", [0, 1, 3], ids=["one_grid", "grids_of_1", "grids_of_3"])
def test_engine_graph_replays(tk, per):
    """Both directions captured into one HIP graph, the engine call issued as
    one grid or as several (layers_per_grid 1 and 3 over 4 layers: several
    kernel nodes per call): every replay (with eager work and
    synchronisation between replays) equals the oracle."""
    wl = make_workload("llama3-70b-batch8", num_layers=4, seq_lens=[4096, 1000, 17, 2049])
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    nbytes = tk.topkv_packed_layer_bytes(src, wl.seq_lens)
    L, R = wl.num_layers, wl.num_reqs
    packed = torch.empty((L, nbytes // 2), dtype=torch.int16, device="cuda")
    opt = tk.engine_options(layers_per_grid=per)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tk.topkv_engine_pack_layers(src, 0, L, R, bt, bt.shape[1], lens, packed, nbytes, engine=opt)
        tk.topkv_engine_unpack_layers(packed, nbytes, dst, 0, L, R, bt2, bt2.shape[1], lens, engine=opt)
    want_dst = dst_h.copy()
    want = [oracle.pack_layer(src_h, z, wl.block_tables, wl.seq_lens) for z in range(L)]
    for z in range(L):
        oracle.unpack_layer(want[z], want_dst, z, wl.dst_block_tables, wl.seq_lens)
    for rep in range(3):
        packed.fill_(-1)
        dst.copy_(to_dev(dst_h))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for z in range(L):
            assert np.array_equal(to_host(packed[z]), want[z]), f"replay {rep} layer {z}"
        assert np.array_equal(to_host(dst), want_dst), f"replay {rep}: unpacked pool"

"""topkv_check_tables on the device: valid tables pass; planted out-of-range
entries, repeated pages and bad lengths are counted exactly."""
import numpy as np
import pytest
import torch

from gpu_util import say
from paper_2607_28633_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _run(tk, pool, bt, lens, dup):
    ws = torch.full((max(1, tk.topkv_check_workspace_bytes(pool) // 4),), -1, dtype=torch.int32, device="cuda")
    res = torch.full((4,), 77, dtype=torch.int32, device="cuda")
    tk.topkv_check_tables(pool, bt.shape[0], torch.from_numpy(bt).cuda(), bt.shape[1],
                          torch.from_numpy(lens).cuda(), dup, ws, res)
    torch.cuda.synchronize()
    return res.cpu().tolist()


@pytest.mark.parametrize("name", ["tiny", "reblock-70b"])
def test_valid_tables_pass(tk, name):
    wl = make_workload(name)
    say(f"[check] valid {name}")
    for bt, P, NP in ((wl.block_tables, wl.page_size, wl.num_pages),
                      (wl.dst_block_tables, wl.dst_page_size, wl.dst_num_pages)):
        pool = tk.make_pool(0x1000, num_pages=NP, num_layers=1, page_size=P, planes=wl.planes,
                            num_heads=wl.num_heads, head_dim=wl.head_dim)
        assert _run(tk, pool, bt, wl.seq_lens, 1) == [tk.TOPKV_OK, 0, 0, 0]
        assert _run(tk, pool, bt, wl.seq_lens, 0) == [tk.TOPKV_OK, 0, 0, 0]


def test_planted_errors_are_counted(tk):
    wl = make_workload("tiny")
    say("[check] planted errors")
    pool = tk.make_pool(0x1000, num_pages=wl.num_pages, num_layers=1, page_size=wl.page_size, planes=2,
                        num_heads=2, head_dim=64)
    bt = wl.block_tables.copy()
    lens = wl.seq_lens.copy()                  # 64/48/33/17 -> 4/3/3/2 pages, stride 4
    bt[0, 1] = wl.num_pages                    # out of range
    bt[1, 0] = -3                              # out of range
    bt[2, 2] = bt[3, 0]                        # a page named twice
    bt[3, 3] = 5000                            # past request 3's last page: never read, not counted
    assert _run(tk, pool, bt, lens, 1) == [tk.TOPKV_ERR_BOUNDS, 2, 1, 0]
    assert _run(tk, pool, bt, lens, 0) == [tk.TOPKV_ERR_BOUNDS, 2, 0, 0]   # pack sources may repeat pages
    lens2 = lens.copy()
    lens2[1] = -1
    lens2[2] = 4 * 16 + 1                      # beyond bt_stride * P
    bt2 = wl.block_tables.copy()
    bt2[2, 3] = sorted(set(range(wl.num_pages)) - set(bt2[bt2 >= 0].tolist()))[0]
    assert _run(tk, pool, bt2, lens2, 1) == [tk.TOPKV_ERR_BOUNDS, 0, 0, 2]


# ---------------------------------------------------------------------------
# Checked mode (TOPKV_CHECKED=1): the movement calls validate first and move
# nothing when the validation fails.
# ---------------------------------------------------------------------------
import contextlib
import os

import oracle
from gpu_util import to_dev, to_host
from paper_2607_28633_amd.workloads import host_dst_prefill, host_src_pool

SENT = 0x0BAD


@contextlib.contextmanager
def checked(on=True):
    old = os.environ.get("TOPKV_CHECKED")
    os.environ["TOPKV_CHECKED"] = "1" if on else "0"
    try:
        yield
    finally:
        if old is None:
            del os.environ["TOPKV_CHECKED"]
        else:
            os.environ["TOPKV_CHECKED"] = old


def _bounds(tk, fn, *a, **kw):
    with pytest.raises(tk.TopkvError) as ei:
        fn(*a, **kw)
    assert ei.value.status == tk.TOPKV_ERR_BOUNDS, tk.topkv_status_string(ei.value.status)


class _Case:
    def __init__(self, tk, window=0):
        self.wl = wl = make_workload("tiny")             # 64/48/33/17 tokens, page 16, table width 4
        self.src_h, self.dst_h = host_src_pool(wl), host_dst_prefill(wl)
        self.src, self.dst = to_dev(self.src_h), to_dev(self.dst_h)
        self.window = window
        self.n = oracle.packed_layer_elems(wl.planes, wl.num_heads, wl.head_dim, wl.seq_lens, window)
        self.packed = torch.full((self.n + 64,), SENT, dtype=torch.int16, device="cuda")

    def pack(self, tk, bt, lens, dst_bytes=None):
        tk.topkv_pack_layer_window(self.src, 1, self.wl.num_reqs, to_dev(bt), bt.shape[1], to_dev(lens), self.window,
                                   self.packed, dst_bytes=2 * self.n if dst_bytes is None else dst_bytes)

    def unpack(self, tk, bt, lens):
        tk.topkv_unpack_layer_window(self.packed, self.dst, 1, self.wl.num_reqs, to_dev(bt), bt.shape[1],
                                     to_dev(lens), self.window, src_bytes=2 * self.n)

    def untouched(self):
        torch.cuda.synchronize()
        return (to_host(self.packed) == SENT).all() and np.array_equal(to_host(self.dst), self.dst_h)


@pytest.mark.parametrize("window", [0, 20])
def test_checked_mode_passes_valid_moves(tk, window):
    """Valid inputs move exactly as without checked mode (batched, windowed,
    and the host-length single-request calls)."""
    c = _Case(tk, window)
    wl = c.wl
    say(f"[checked] valid moves, window {window}")
    with checked():
        c.pack(tk, wl.block_tables, wl.seq_lens)
        c.unpack(tk, wl.dst_block_tables, wl.seq_lens)
        torch.cuda.synchronize()
        want = oracle.pack_layer(c.src_h, 1, wl.block_tables, wl.seq_lens, window=window)
        assert np.array_equal(to_host(c.packed)[:c.n], want)
        want_dst = c.dst_h.copy()
        oracle.unpack_layer(want, want_dst, 1, wl.dst_block_tables, wl.seq_lens, window=window)
        assert np.array_equal(to_host(c.dst), want_dst)
        n0 = int(wl.seq_lens[0])
        one = torch.empty(n0 * wl.planes * wl.num_heads * wl.head_dim, dtype=torch.int16, device="cuda")
        tk.topkv_pack_layer(c.src, 0, to_dev(wl.block_tables[0]), n0, one)
        tk.topkv_unpack_layer(one, c.dst, 0, to_dev(wl.dst_block_tables[0]), n0)
        torch.cuda.synchronize()
        want1 = oracle.pack_layer(c.src_h, 0, wl.block_tables[:1], wl.seq_lens[:1])
        assert np.array_equal(to_host(one), want1)


def test_checked_mode_refuses_bad_inputs(tk):
    """Each planted problem is refused with TOPKV_ERR_BOUNDS and nothing is
    written; pack sources that repeat a page are legal.  Without checked
    mode the same calls skip the bad parts silently."""
    say("[checked] planted problems")
    c = _Case(tk)
    wl = c.wl
    bt, bt2, lens = wl.block_tables, wl.dst_block_tables, wl.seq_lens
    with checked():
        bad = bt.copy()
        bad[0, 1] = wl.num_pages                         # entry outside the pool
        _bounds(tk, c.pack, tk, bad, lens)
        dup = bt2.copy()
        dup[2, 2] = dup[3, 0]                            # an unpack destination page named twice
        _bounds(tk, c.unpack, tk, dup, lens)
        for r, n in ((1, -1), (2, 4 * 16 + 1)):          # lengths outside [0, table width x page size]
            l2 = lens.copy()
            l2[r] = n
            _bounds(tk, c.pack, tk, bt, l2)
            _bounds(tk, c.unpack, tk, bt2, l2)
        _bounds(tk, c.pack, tk, bt, lens, dst_bytes=2 * c.n - 2)       # packed buffer one element short
        one = torch.full((64 * 2 * 2 * 64,), SENT, dtype=torch.int16, device="cuda")
        _bounds(tk, tk.topkv_pack_layer, c.src, 0, to_dev(bad[0]), 64, one)    # host-length call, bad entry
        _bounds(tk, tk.topkv_pack_layer_planes, c.src, 0, to_dev(bt[0]), 64, one, 64 * 256,
                dst_bytes=64 * 256 + 64 * 256 - 2)                             # placed planes, short buffer
        assert c.untouched() and (to_host(one) == SENT).all(), "a refused call wrote"
        rep = bt.copy()
        rep[1, 0] = rep[0, 0]                            # a pack source may repeat a page
        c.pack(tk, rep, lens)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(c.packed)[:c.n], oracle.pack_layer(c.src_h, 1, rep, lens))
    with checked(False):                                 # the fast path: bad entry skipped, no error
        c.pack(tk, bad, lens)
        torch.cuda.synchronize()


def test_checked_mode_window(tk):
    """With a window only the window's pages are validated: entries before
    it may hold anything (a cache that freed them), entries inside may not."""
    say("[checked] window")
    c = _Case(tk, window=20)
    wl = c.wl
    bt = wl.block_tables.copy()
    bt[0, :2] = -1                 # request 0 (64 tokens) keeps tokens 44..63: pages 2 and 3 only
    bt[1, 0] = 10 ** 6             # request 1 (48 tokens) keeps 28..47: pages 1 and 2
    with checked():
        c.pack(tk, bt, wl.seq_lens)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(c.packed)[:c.n],
                              oracle.pack_layer(c.src_h, 1, wl.block_tables, wl.seq_lens, window=20))
        bt[1, 1] = -1              # inside request 1's window
        _bounds(tk, c.pack, tk, bt, wl.seq_lens)


def test_checked_mode_state_slots(tk):
    """Fixed-state calls: a slot outside the cache is refused on both sides, a
    slot named twice only on unpack; refused calls write nothing."""
    say("[checked] state slots")
    rng = np.random.default_rng(5)
    cache_h = rng.integers(0, 256, size=(2, 6, 100), dtype=np.uint8)
    cache = to_dev(cache_h)
    out = torch.full((4 * 100,), 0x21, dtype=torch.int8, device="cuda")
    with checked():
        _bounds(tk, tk.topkv_pack_state_layer, cache, 1, 4, to_dev(np.array([0, 6, 2, 3], np.int32)), out)
        _bounds(tk, tk.topkv_unpack_state_layer, out, cache, 1, 4, to_dev(np.array([0, 1, 1, 3], np.int32)))
        torch.cuda.synchronize()
        assert (to_host(out) == 0x21).all() and np.array_equal(to_host(cache), cache_h)
        tk.topkv_pack_state_layer(cache, 1, 4, to_dev(np.array([5, 1, 1, 3], np.int32)), out)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(out).reshape(4, 100), cache_h[1, [5, 1, 1, 3]])


def test_checked_mode_refuses_capture(tk):
    """Checked mode synchronises, so a stream under capture is refused (and
    nothing is queued); the captured graph replays the rest correctly."""
    say("[checked] capture")
    c = _Case(tk)
    wl = c.wl
    x = torch.zeros(4, device="cuda")
    bt, lens = to_dev(wl.block_tables), to_dev(wl.seq_lens)      # uploads stay outside the capture
    g = torch.cuda.CUDAGraph()
    with checked():
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            with pytest.raises(tk.TopkvError) as ei:
                tk.topkv_pack_layer_window(c.src, 1, wl.num_reqs, bt, bt.shape[1], lens, 0, c.packed,
                                           dst_bytes=2 * c.n)
            x.add_(1)
        assert ei.value.status == tk.TOPKV_ERR_UNSUPPORTED
        g.replay()
        torch.cuda.synchronize()
    assert x.tolist() == [1, 1, 1, 1] and c.untouched()


def test_checked_mode_layout_moves(tk):
    """Layout moves under checked mode: a head-sliced pack with a bad source
    entry, an unpack into a head-major pool naming a page twice, a re-block
    whose destination table is bad, and a shard region too small are refused
    without writing; the valid head-sliced pack equals the oracle."""
    import oracle.reshard as rs
    say("[checked] layout moves")
    c = _Case(tk)
    wl = c.wl
    bt, bt2, lens = wl.block_tables, wl.dst_block_tables, to_dev(wl.seq_lens)
    nh = rs.packed_heads_elems(wl.planes, 1, wl.head_dim, wl.seq_lens)
    half = torch.full((nh + 64,), SENT, dtype=torch.int16, device="cuda")
    with checked():
        bad = bt.copy()
        bad[3, 1] = -5
        _bounds(tk, tk.topkv_pack_layer_heads, c.src, 1, wl.num_reqs, to_dev(bad), bt.shape[1], lens, 1, 1, half,
                dst_bytes=2 * nh)
        _bounds(tk, tk.topkv_pack_layer_heads, c.src, 1, wl.num_reqs, to_dev(bt), bt.shape[1], lens, 1, 1, half,
                dst_bytes=2 * nh - 2)
        dup = bt2.copy()
        dup[0, 3] = dup[1, 0]
        hm = c.dst.view(wl.phys_layers, wl.dst_num_pages, wl.planes, wl.num_heads, wl.dst_page_size, wl.head_dim)
        _bounds(tk, tk.topkv_move_layer, tk.packed_view(half, 2 * nh),
                tk.pool_view(hm, 1, to_dev(dup), dup.shape[1], head_begin=1, head_major=True), wl.num_reqs, lens, 1)
        bad2 = bt2.copy()
        bad2[2, 0] = wl.dst_num_pages
        _bounds(tk, tk.topkv_move_layer, tk.pool_view(c.src, 1, to_dev(bt), bt.shape[1]),
                tk.pool_view(c.dst, 1, to_dev(bad2), bad2.shape[1]), wl.num_reqs, lens, wl.num_heads)
        assert c.untouched() and (to_host(half) == SENT).all(), "a refused call wrote"
        tk.topkv_pack_layer_heads(c.src, 1, wl.num_reqs, to_dev(bt), bt.shape[1], lens, 1, 1, half, dst_bytes=2 * nh)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(half)[:nh], rs.pack_layer_heads(c.src_h, 1, bt, wl.seq_lens, 1, 1))


def test_checked_mode_one_pass_kvcache1(tk):
    """The one-pass KVCACHE1 calls under checked mode: a table entry outside
    the pool is refused on both sides and a page named twice by the receiver's
    table is refused, writing neither blob, pool nor result; a sender may
    repeat a page, and valid calls give the two-step calls' blob and pool."""
    say("[checked] one-pass KVCACHE1")
    c = _Case(tk)
    wl = c.wl
    geo = tk.pool_from_tensor(c.src)
    n = int(wl.seq_lens[0])                                  # 64 tokens, 4 pages
    bt, bt2 = wl.block_tables[0].copy(), wl.dst_block_tables[0].copy()
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
    blob = torch.full((nbytes,), 0x5C, dtype=torch.uint8, device="cuda")
    res = torch.full((4,), 77, dtype=torch.int32, device="cuda")
    with checked():
        bad = bt.copy()
        bad[2] = wl.num_pages
        _bounds(tk, tk.topkv_kvcache1_pack_seal, c.src, to_dev(bad), n, 1, 2, blob, ws)
        torch.cuda.synchronize()
        assert (blob == 0x5C).all().item(), "a refused sender wrote its blob"
        tk.topkv_kvcache1_pack_seal(c.src, to_dev(bt), n, 1, 2, blob, ws)
        two = torch.empty_like(blob)
        tk.topkv_kvcache1_pack_layers(c.src, 0, wl.num_layers, to_dev(bt), n, two)
        tk.topkv_kvcache1_seal(geo, n, 1, 2, two, ws)
        torch.cuda.synchronize()
        assert torch.equal(blob, two), "checked one-pass blob differs from the two-step blob"
        for table in (np.array([bt2[0], bt2[1], bt2[0], bt2[3]], dtype=np.int32),       # a page named twice
                      np.array([bt2[0], -1, bt2[2], bt2[3]], dtype=np.int32)):         # an entry outside
            _bounds(tk, tk.topkv_kvcache1_verify_unpack, blob, c.dst, to_dev(table), n, 1, 2, ws, res)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(c.dst), c.dst_h), "a refused receiver wrote its pool"
        assert res.cpu().tolist() == [77] * 4, "a refused receiver wrote its result"
        rep = bt.copy()
        rep[3] = rep[0]                                      # a sender may read one page twice
        tk.topkv_kvcache1_pack_seal(c.src, to_dev(rep), n, 1, 2, blob, ws)
        tk.topkv_kvcache1_verify_unpack(blob, c.dst, to_dev(bt2), n, 1, 2, ws, res)
        torch.cuda.synchronize()
        assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0]

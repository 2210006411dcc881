"""Pins for the layout-move oracle (head-sliced pack/unpack, pool-to-pool
re-blocking, head-major pools).  None re-derives the oracle's definition:
brute force runs element by element through flat-address arithmetic on
tiny pools; the head partition and the two-step re-block compare with the
pinned full-head pack/unpack oracle; the identity-table case compares with a
library axis swap.

Each pin takes an implementation object exposing the oracle's reshard API
(``View``, ``PACKED``, ``POOL``, ``POOL_HEAD_MAJOR``, ``move_layer``,
``pack_layer_heads``, ``unpack_layer_heads``, ``reblock_layer``) and raises
on a violation; mutants of the oracle run through the same pins.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2607_28633_amd.workloads import host_dst_prefill, host_src_pool, make_workload, random_words


def _wl(**kw):
    base = dict(num_layers=2, num_heads=8, head_dim=4, seq_lens=[37, 16, 0, 1, 50, 9])
    base.update(kw)
    return make_workload("tiny", **base)


def _kept(n, window):
    return range(oracle.window_start(n, window), n)


def _pool_index(shape, layer, page, c, slot, h, d, head_major=False):
    _, NP, C, a, b, D = shape                 # slot-major: a = P, b = H; head-major: a = H, b = P
    if head_major:
        return ((((layer * NP + page) * C + c) * a + h) * b + slot) * D + d
    return ((((layer * NP + page) * C + c) * a + slot) * b + h) * D + d


def _brute_pack(pool, layer, bts, lens, h0, hc, window, head_major=False):
    flat = pool.reshape(-1)
    P = pool.shape[4] if head_major else pool.shape[3]
    C, D = pool.shape[2], pool.shape[5]
    out = []
    for r, n in enumerate(lens):
        n = int(n)
        kept = list(_kept(n, window))
        for c in range(C):
            for t in kept:
                for j in range(hc):
                    for d in range(D):
                        out.append(flat[_pool_index(pool.shape, layer, int(bts[r][t // P]), c, t % P,
                                                    h0 + j, d, head_major)])
    return np.array(out, dtype=pool.dtype)


def _brute_unpack(packed, pool, layer, bts, lens, h0, hc, window, head_major=False):
    flat = pool.reshape(-1)                   # pool is contiguous: writes land in it
    P = pool.shape[4] if head_major else pool.shape[3]
    C, D = pool.shape[2], pool.shape[5]
    i = 0
    for r, n in enumerate(lens):
        n = int(n)
        kept = list(_kept(n, window))
        for c in range(C):
            for t in kept:
                for j in range(hc):
                    for d in range(D):
                        flat[_pool_index(pool.shape, layer, int(bts[r][t // P]), c, t % P, h0 + j, d,
                                         head_major)] = packed[i]
                        i += 1
    assert i == packed.size
    return pool


SLICES = [(0, 8), (3, 2), (7, 1), (0, 1), (2, 5)]


def pin_heads_bruteforce(impl):
    """Head-sliced pack, element by element through flat addresses."""
    wl = _wl()
    pool = host_src_pool(wl)
    for h0, hc in SLICES:
        for window in (0, 5):
            got = impl.pack_layer_heads(pool, 1, wl.block_tables, wl.seq_lens, h0, hc, window)
            want = _brute_pack(pool, 1, wl.block_tables, wl.seq_lens, h0, hc, window)
            assert got.shape == want.shape and np.array_equal(got, want), f"heads [{h0}, +{hc}) W={window}"


def pin_heads_partition(impl):
    """Slices that partition the heads, put side by side per request, give
    the full-head packed layer (the pinned pack oracle)."""
    wl = _wl(seq_lens=[33, 1, 0, 64, 17])
    pool = host_src_pool(wl)
    C, H, D = wl.planes, wl.num_heads, wl.head_dim
    parts = [(0, 3), (3, 2), (5, 3)]
    slices = [impl.pack_layer_heads(pool, 0, wl.block_tables, wl.seq_lens, a, b) for a, b in parts]
    full = oracle.pack_layer(pool, 0, wl.block_tables, wl.seq_lens)
    offs, off_full = [0] * len(parts), 0
    for n in wl.seq_lens:
        n = int(n)
        blocks = []
        for k, (_, hc) in enumerate(parts):
            size = C * n * hc * D
            blocks.append(slices[k][offs[k]:offs[k] + size].reshape(C, n, hc, D))
            offs[k] += size
        joined = np.concatenate(blocks, axis=2).reshape(-1)
        assert np.array_equal(joined, full[off_full:off_full + joined.size]), "head slices do not tile the layer"
        off_full += joined.size
    assert off_full == full.size and all(o == s.size for o, s in zip(offs, slices))


def pin_unpack_heads_bruteforce(impl):
    """Head-sliced unpack writes exactly the slice's elements of the kept
    tokens; every other element of the pool keeps its value."""
    wl = _wl(dst_page_size=5)
    for h0, hc in SLICES:
        for window in (0, 7):
            n_el = oracle.packed_layer_elems(wl.planes, hc, wl.head_dim, wl.seq_lens, window)
            packed = random_words(np.random.default_rng(h0 * 31 + hc + window), (n_el,), 2)
            base = host_dst_prefill(wl)
            got = impl.unpack_layer_heads(packed, base.copy(), 1, wl.dst_block_tables, wl.seq_lens, h0, hc, window)
            want = _brute_unpack(packed, base.copy(), 1, wl.dst_block_tables, wl.seq_lens, h0, hc, window)
            assert np.array_equal(got, want), f"unpack heads [{h0}, +{hc}) W={window}"


def pin_reblock_two_step(impl):
    """Pool-to-pool re-blocking equals unpack(pack(.)) of the pinned oracle,
    for page sizes that divide, multiply and straddle each other."""
    for dst_p in (5, 16, 48, 64):
        wl = _wl(head_dim=8, dst_page_size=dst_p)
        src = host_src_pool(wl)
        for window in (0, 11):
            for layer in range(wl.num_layers):
                got = impl.reblock_layer(src, layer, wl.block_tables, host_dst_prefill(wl), layer,
                                         wl.dst_block_tables, wl.seq_lens, window)
                packed = oracle.pack_layer(src, layer, wl.block_tables, wl.seq_lens, window)
                want = oracle.unpack_layer(packed, host_dst_prefill(wl), layer, wl.dst_block_tables,
                                           wl.seq_lens, window)
                assert np.array_equal(got, want), f"re-block 16 -> {dst_p}, W={window}, layer {layer}"


def pin_reblock_bruteforce(impl):
    """Re-blocking between different layers and page sizes, element by element."""
    wl = _wl(dst_page_size=48, seq_lens=[70, 3, 48, 49])
    src = host_src_pool(wl)
    got = impl.reblock_layer(src, 1, wl.block_tables, host_dst_prefill(wl), 0, wl.dst_block_tables, wl.seq_lens)
    want = host_dst_prefill(wl)
    sflat, dflat = src.reshape(-1), want.reshape(-1)
    for r, n in enumerate(wl.seq_lens):
        for t in range(int(n)):
            for c in range(wl.planes):
                for h in range(wl.num_heads):
                    for d in range(wl.head_dim):
                        s = _pool_index(src.shape, 1, int(wl.block_tables[r][t // 16]), c, t % 16, h, d)
                        q = _pool_index(want.shape, 0, int(wl.dst_block_tables[r][t // 48]), c, t % 48, h, d)
                        dflat[q] = sflat[s]
    assert np.array_equal(got, want), "re-block differs from element-wise copy"


def pin_head_major_bruteforce(impl):
    """Moves into and out of a head-major pool, element by element: the
    head-major side addresses [page][plane][head][slot][dim]."""
    wl = _wl(dst_page_size=5)
    src = host_src_pool(wl)
    hm_shape = (wl.phys_layers, wl.dst_num_pages, wl.planes, wl.num_heads, 5, wl.head_dim)
    for h0, hc, window in ((0, 8, 0), (2, 3, 6)):
        hm0 = random_words(np.random.default_rng(7 + h0), hm_shape, 2)
        got = impl.move_layer(impl.View(impl.POOL, src, 1, wl.block_tables, h0),
                              impl.View(impl.POOL_HEAD_MAJOR, hm0.copy(), 0, wl.dst_block_tables, h0),
                              wl.seq_lens, hc, window)
        packed = _brute_pack(src, 1, wl.block_tables, wl.seq_lens, h0, hc, window)
        want = _brute_unpack(packed, hm0.copy(), 0, wl.dst_block_tables, wl.seq_lens, h0, hc, window,
                             head_major=True)
        assert np.array_equal(got, want), f"slot-major -> head-major, heads [{h0}, +{hc}), W={window}"
        out = np.empty(packed.size, dtype=packed.dtype)
        back = impl.move_layer(impl.View(impl.POOL_HEAD_MAJOR, want, 0, wl.dst_block_tables, h0),
                               impl.View(impl.PACKED, out), wl.seq_lens, hc, window)
        assert np.array_equal(back, packed), "head-major -> packed"


def pin_head_major_identity_is_swapaxes(impl):
    """With identity tables and full pages, moving every layer into a
    head-major pool is numpy.swapaxes of the slot and head axes."""
    wl = make_workload("tiny", num_layers=2, num_heads=4, head_dim=8, seq_lens=[64, 48],
                       num_pages=7, dst_num_pages=7)
    src = host_src_pool(wl)
    bt = np.array([[0, 1, 2, 3], [4, 5, 6, 0]], dtype=np.int32)
    hm = np.zeros_like(np.swapaxes(src, 3, 4))
    for layer in range(2):
        impl.move_layer(impl.View(impl.POOL, src, layer, bt), impl.View(impl.POOL_HEAD_MAJOR, hm, layer, bt),
                        [64, 48], 4)
    assert np.array_equal(hm, np.swapaxes(src, 3, 4)), "head-major pool is not the axis swap"


def pin_shards_are_head_slices(impl):
    """S shards of heads [h0, h0 + hc): shard s is the head-sliced pack of
    heads h0 + s*hc/S ... (itself pinned by brute force), at s * shard_elems;
    the gap after each shard keeps its prior words."""
    wl = _wl()
    pool = host_src_pool(wl)
    for h0, hc, S, window in ((0, 8, 2, 0), (0, 8, 4, 9), (2, 6, 3, 0), (0, 8, 8, 0), (4, 4, 1, 3)):
        per = oracle.packed_layer_elems(wl.planes, hc // S, wl.head_dim, wl.seq_lens, window)
        cap = per + 7
        out = np.full(S * cap, 0xABCD, dtype=pool.dtype)
        got = impl.move_layer(impl.View(impl.POOL, pool, 1, wl.block_tables, h0),
                              impl.View(impl.PACKED, out, shards=S, shard_elems=cap), wl.seq_lens, hc, window)
        for sh in range(S):
            want = _brute_pack(pool, 1, wl.block_tables, wl.seq_lens, h0 + sh * (hc // S), hc // S, window)
            region = got[sh * cap:(sh + 1) * cap]
            assert np.array_equal(region[:per], want), f"shard {sh} of {S} (heads {h0}+{hc}, W={window})"
            assert (region[per:] == 0xABCD).all(), f"shard {sh}: words past the shard's data changed"


def pin_shards_unpack(impl):
    """Unpacking S shards into a pool equals unpacking each shard's head
    slice on its own (brute force)."""
    wl = _wl(dst_page_size=7)
    rng = np.random.default_rng(11)
    for h0, hc, S in ((0, 8, 2), (1, 6, 3), (0, 8, 8)):
        per = oracle.packed_layer_elems(wl.planes, hc // S, wl.head_dim, wl.seq_lens)
        packed = random_words(rng, (S * per,), 2)
        base = host_dst_prefill(wl)
        got = impl.move_layer(impl.View(impl.PACKED, packed, shards=S, shard_elems=per),
                              impl.View(impl.POOL, base.copy(), 0, wl.dst_block_tables, h0), wl.seq_lens, hc)
        want = base.copy()
        for sh in range(S):
            _brute_unpack(packed[sh * per:(sh + 1) * per], want, 0, wl.dst_block_tables, wl.seq_lens,
                          h0 + sh * (hc // S), hc // S, 0)
        assert np.array_equal(got, want), f"{S} shards of heads {h0}+{hc} unpacked"


RESHARD_PINS = [pin_heads_bruteforce, pin_heads_partition, pin_unpack_heads_bruteforce, pin_reblock_two_step,
                pin_reblock_bruteforce, pin_head_major_bruteforce, pin_head_major_identity_is_swapaxes,
                pin_shards_are_head_slices, pin_shards_unpack]


def failing_pins(impl):
    failed = []
    for pin in RESHARD_PINS:
        try:
            pin(impl)
        except Exception as e:          # a crash on a plausible mistake counts as caught
            failed.append((pin.__name__, f"{type(e).__name__}: {e}"))
    return failed

"""Pins for the pack/unpack oracle: checks against facts that do not come from the
oracle itself (the paper's printed sizes, Eq. 1, library transposes, round-trip
and multiset invariants, brute force through flat-address arithmetic).

Each pin takes an implementation object exposing ``pack_layer(pool, layer,
block_tables, seq_lens)`` and ``unpack_layer(packed, pool, layer, block_tables,
seq_lens)`` with the oracle's conventions and raises AssertionError when the
implementation violates it.  The same pins run against the real oracle and
against deliberately broken copies of it (mutants), so each pin's power to
catch a plausible mistake is itself tested.
"""
from __future__ import annotations

import math
import os

import numpy as np

from paper_2607_28633_amd.workloads import make_workload, host_src_pool, host_dst_prefill, random_words

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _pages(n, p):
    return -(-int(n) // int(p))


# ----------------------------------------------------------------------------
# Sizes: Eq. 1 and the paper's printed figures
# ----------------------------------------------------------------------------

def _bytes_over_layers(impl, layers, planes, heads, dim, tokens, page_size=16, elem_bytes=2):
    """Run the implementation over every layer of a zero pool just big enough
    for one request and add up the packed bytes."""
    k = _pages(tokens, page_size)
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[elem_bytes]
    pool = np.zeros((layers, k, planes, page_size, heads, dim), dtype=dt)
    bt = np.arange(k, dtype=np.int32)[None, :]
    lens = np.array([tokens], dtype=np.int32)
    total = 0
    for layer in range(layers):
        total += impl.pack_layer(pool, layer, bt, lens).nbytes
    return total


def pin_table1_sizes(impl):
    """Section 2.2 Table 1 (and Section 5.3 for MLA): bytes over all layers of
    a 4096-token request equal Eq. 1 and round to the printed figure."""
    for model, L, H, D, C, s, printed in read_golden("kv_sizes.txt"):
        L, H, D, C, s = int(L), int(H), int(D), int(C), int(s)
        got = _bytes_over_layers(impl, L, C, H, D, s)
        # Eq. 1: 2 * L * h_kv * d_h * s * b_p; Section 5.3 replaces the 2 by 1 for MLA
        eq1 = C * L * H * D * s * 2
        assert got == eq1, f"{model}: packed {got} B over {L} layers, Eq. 1 gives {eq1} B"
        decimals = len(printed.split(".")[1]) if "." in printed else 0
        ok = any(math.isclose(round(got / unit, decimals), float(printed), abs_tol=1e-12)
                 for unit in (1e9, 2.0 ** 30))
        assert ok, f"{model}: {got} B does not round to the printed {printed} GB"


def pin_mla_ratio(impl):
    """Section 5.3: MLA holds 576 elements per token per layer, MHA 32768: 57x."""
    (cm, hm, dm, em, ca, ha, da, ea, ratio), = read_golden("mla_ratio.txt")
    mla = _bytes_over_layers(impl, 1, int(cm), int(hm), int(dm), 1) // 2
    mha = _bytes_over_layers(impl, 1, int(ca), int(ha), int(da), 1) // 2
    assert mla == int(em), f"MLA elements per token-layer {mla} != {em}"
    assert mha == int(ea), f"MHA elements per token-layer {mha} != {ea}"
    assert round(mha / mla) == int(ratio), f"ratio {mha / mla:.2f} does not round to {ratio}"


def pin_eq1_workloads(impl, names=("tiny", "llama3-70b-batch8", "deepseek-v3-mla")):
    """Eq. 1 with s = total batch tokens for the seeded workloads: one layer's
    packed bytes times the layer count equals 2*L*h*d*s*b_p (C = 1 for MLA)."""
    for name in names:
        wl = make_workload(name)
        s = int(wl.seq_lens.astype(np.int64).sum())
        pool = np.zeros((1,) + wl.pool_shape()[1:], dtype=wl.uint_dtype)
        per_layer = impl.pack_layer(pool, 0, wl.block_tables, wl.seq_lens).nbytes
        eq1 = wl.planes * wl.num_layers * wl.num_heads * wl.head_dim * s * wl.elem_bytes
        assert per_layer * wl.num_layers == eq1, f"{name}: {per_layer}*{wl.num_layers} != Eq. 1 {eq1}"


# ----------------------------------------------------------------------------
# Element placement
# ----------------------------------------------------------------------------

def bruteforce_pack(flat, shape, layer, bts, lens):
    """Per-element loops over the flat pool, address = row-major offset of
    (layer, page, plane, slot, head, dim)."""
    L, NP, C, P, H, D = shape
    out = []
    for r in range(len(lens)):
        n = int(lens[r])
        for c in range(C):
            for t in range(n):
                page = int(bts[r][t // P])
                s = t % P
                for h in range(H):
                    for d in range(D):
                        out.append(flat[((((layer * NP + page) * C + c) * P + s) * H + h) * D + d])
    return np.array(out, dtype=flat.dtype)


def bruteforce_unpack(packed, flat, shape, layer, bts, lens):
    L, NP, C, P, H, D = shape
    flat = flat.copy()
    i = 0
    for r in range(len(lens)):
        n = int(lens[r])
        for c in range(C):
            for t in range(n):
                page = int(bts[r][t // P])
                s = t % P
                for h in range(H):
                    for d in range(D):
                        flat[((((layer * NP + page) * C + c) * P + s) * H + h) * D + d] = packed[i]
                        i += 1
    assert i == packed.size
    return flat


def pin_bruteforce_tiny(impl):
    """The tiny pool (2 layers, 2 heads, dim 64, page 16, requests 64/48/33/17):
    every layer's pack and unpack equal per-element brute force."""
    wl = make_workload("tiny")
    src = host_src_pool(wl)
    dst0 = host_dst_prefill(wl)
    for layer in range(wl.num_layers):
        want = bruteforce_pack(src.reshape(-1), src.shape, layer, wl.block_tables, wl.seq_lens)
        got = impl.pack_layer(src, layer, wl.block_tables, wl.seq_lens)
        assert got.dtype == src.dtype and np.array_equal(got.reshape(-1), want), \
            f"pack layer {layer} differs from brute force"
        want_pool = bruteforce_unpack(want, dst0.reshape(-1), dst0.shape, layer,
                                      wl.dst_block_tables, wl.seq_lens)
        got_pool = impl.unpack_layer(want.copy(), dst0.copy(), layer, wl.dst_block_tables, wl.seq_lens)
        assert np.array_equal(got_pool.reshape(-1), want_pool), f"unpack layer {layer} differs from brute force"


def pin_page_take_transpose(impl):
    """Page relabelling reduces pack to a textbook transpose: for one request,
    pack == take(pool[l], pages, axis=0) viewed [k][C][P][H][D], transposed to
    [C][k][P][H][D], reshaped to [C][k*P][H][D] and cut to n tokens.  Checked
    for an identity table, a shuffled table, full and partial last pages."""
    rng = np.random.default_rng(11)
    L, NP, C, P, H, D = 3, 12, 2, 4, 3, 5
    pool = random_words(rng, (L, NP, C, P, H, D), 2)
    for layer in range(L):
        for n in (1, 3, 4, 5, 11, 12, 16):
            k = _pages(n, P)
            for bt in (np.arange(k, dtype=np.int32), rng.permutation(NP)[:k].astype(np.int32)):
                want = np.take(pool[layer], bt, axis=0).transpose(1, 0, 2, 3, 4) \
                    .reshape(C, k * P, H, D)[:, :n]
                got = impl.pack_layer(pool, layer, bt[None, :], np.array([n], np.int32))
                assert np.array_equal(got.reshape(-1), want.reshape(-1)), \
                    f"pack != take/transpose (layer {layer}, n {n}, table {bt.tolist()})"


def pin_request_concat(impl):
    """A batch is the request-order concatenation of single-request packs, and
    unpacking a batch equals unpacking its requests one by one."""
    wl = make_workload("tiny", seed=7)
    src = host_src_pool(wl)
    dst0 = host_dst_prefill(wl)
    layer = 1
    parts = [impl.pack_layer(src, layer, wl.block_tables[r:r + 1], wl.seq_lens[r:r + 1])
             for r in range(wl.num_reqs)]
    whole = impl.pack_layer(src, layer, wl.block_tables, wl.seq_lens)
    assert np.array_equal(whole, np.concatenate(parts)), "batch pack != concatenated single packs"
    seq = dst0.copy()
    for r in range(wl.num_reqs):
        seq = impl.unpack_layer(parts[r].copy(), seq, layer, wl.dst_block_tables[r:r + 1],
                                wl.seq_lens[r:r + 1])
    bat = impl.unpack_layer(whole.copy(), dst0.copy(), layer, wl.dst_block_tables, wl.seq_lens)
    assert np.array_equal(seq, bat), "batch unpack != sequential single unpacks"


def _valid_mask(shape, bts, lens, layer):
    """Which pool elements hold valid tokens: page bts[r][j] of layer `layer`,
    slots below min(P, n_r - j*P)."""
    L, NP, C, P, H, D = shape
    m = np.zeros(shape, dtype=bool)
    for r in range(len(lens)):
        n = int(lens[r])
        for j in range(_pages(n, P)):
            m[layer, bts[r][j], :, :min(P, n - j * P)] = True
    return m


def pin_roundtrip(impl):
    """Unpack into pools of other page sizes (re-blocking), then pack back:
    the result equals the first pack; elements outside the written slots keep
    the pre-fill; the written slots hold exactly the packed words (multiset)."""
    for P2 in (16, 64, 48, 1, 5):
        wl = make_workload("tiny", seed=3, dst_page_size=P2)
        src = host_src_pool(wl)
        for layer in range(wl.num_layers):
            first = impl.pack_layer(src, layer, wl.block_tables, wl.seq_lens)
            dst0 = host_dst_prefill(wl)
            dst = impl.unpack_layer(first.copy(), dst0.copy(), layer, wl.dst_block_tables, wl.seq_lens)
            again = impl.pack_layer(dst, layer, wl.dst_block_tables, wl.seq_lens)
            assert np.array_equal(first, again), f"round trip differs (P'={P2}, layer {layer})"
            m = _valid_mask(dst.shape, wl.dst_block_tables, wl.seq_lens, layer)
            assert np.array_equal(dst[~m], dst0[~m]), f"unpack touched bytes outside valid slots (P'={P2})"
            assert np.array_equal(np.sort(dst[m]), np.sort(first)), f"written slots != packed words (P'={P2})"


def pin_multiset(impl):
    """The packed words of a layer are exactly the words in the valid slots of
    the request pages of that layer (same multiset), for every workload shape."""
    for name, kw in (("tiny", {}), ("deepseek-v3-mla", dict(num_layers=2, seq_lens=[70, 1, 64, 129])),
                     ("llama3-70b-batch8", dict(num_layers=2, seq_lens=[33, 16, 1, 47], num_heads=2,
                                                head_dim=8))):
        wl = make_workload(name, **kw)
        src = host_src_pool(wl)
        for layer in range(wl.num_layers):
            got = impl.pack_layer(src, layer, wl.block_tables, wl.seq_lens)
            m = _valid_mask(src.shape, wl.block_tables, wl.seq_lens, layer)
            assert np.array_equal(np.sort(got), np.sort(src[m])), f"{name} layer {layer}: multiset differs"


def pin_zero_and_opaque(impl):
    """Zero-length requests contribute nothing; every bit pattern (as 1-, 2- and
    4-byte words) survives pack -> unpack -> pack unchanged."""
    rng = np.random.default_rng(5)
    for eb in (1, 2, 4):
        pool = random_words(rng, (2, 9, 2, 4, 2, 3), eb)
        bts = np.array([[3, 1, -1], [-1, -1, -1], [0, 7, 8]], dtype=np.int32)
        lens = np.array([6, 0, 9], dtype=np.int32)
        got = impl.pack_layer(pool, 1, bts, lens)
        assert got.size == 2 * 2 * 3 * 15
        dst = impl.unpack_layer(got.copy(), np.zeros_like(pool), 1, bts, lens)
        again = impl.pack_layer(dst, 1, bts, lens)
        assert got.tobytes() == again.tobytes()
        empty = impl.pack_layer(pool, 0, bts[1:2], lens[1:2])
        assert empty.size == 0


# ----------------------------------------------------------------------------
# Windowed layers (Section 2.2 per-layer-kind extension of Eq. 1)
# ----------------------------------------------------------------------------

def pin_window_slice(impl):
    """A windowed pack equals the full pack cut to each request's last W
    tokens (a library slice of a result the pins above fix)."""
    wl = make_workload("tiny", seed=8, seq_lens=[64, 48, 33, 17, 1, 0])
    src = host_src_pool(wl)
    C, H, D = wl.planes, wl.num_heads, wl.head_dim
    for W in (1, 15, 16, 17, 40, 64, 100):
        got = impl.pack_layer(src, 1, wl.block_tables, wl.seq_lens, window=W)
        parts = []
        for r, n in enumerate(wl.seq_lens):
            full = impl.pack_layer(src, 1, wl.block_tables[r:r + 1], wl.seq_lens[r:r + 1]).reshape(C, int(n), H, D)
            parts.append(full[:, max(0, int(n) - W):].reshape(-1))
        assert np.array_equal(got, np.concatenate(parts)), f"window {W}: != last-W slice of the full pack"


def pin_window_roundtrip(impl):
    """Windowed unpack into another page size, windowed pack back: same words;
    only the window's slots change in the destination."""
    for P2, W in ((16, 20), (64, 33), (5, 1), (48, 64)):
        wl = make_workload("tiny", seed=6, dst_page_size=P2)
        src = host_src_pool(wl)
        first = impl.pack_layer(src, 0, wl.block_tables, wl.seq_lens, window=W)
        dst0 = host_dst_prefill(wl)
        dst = impl.unpack_layer(first.copy(), dst0.copy(), 0, wl.dst_block_tables, wl.seq_lens, window=W)
        again = impl.pack_layer(dst, 0, wl.dst_block_tables, wl.seq_lens, window=W)
        assert np.array_equal(first, again), f"windowed round trip differs (P'={P2}, W={W})"
        m = np.zeros(dst.shape, dtype=bool)
        for r, n in enumerate(wl.seq_lens):
            for t in range(max(0, int(n) - W), int(n)):
                m[0, wl.dst_block_tables[r][t // P2], :, t % P2] = True
        assert np.array_equal(dst[~m], dst0[~m]), f"windowed unpack touched other slots (P'={P2}, W={W})"


def pin_layer_kind_sizes(impl):
    """Section 2.2: the 2026-model figures (Kimi K2 MLA, gpt-oss-120b with 18
    window-capped layers) from packed bytes summed over every layer."""
    for model, full_l, win_l, W, C, H, D, s, printed in read_golden("layer_kinds.txt"):
        full_l, win_l, W, C, H, D, s = map(int, (full_l, win_l, W, C, H, D, s))
        k = _pages(s, 16)
        pool = np.zeros((1, k, C, 16, H, D), dtype=np.uint16)
        bt = np.arange(k, dtype=np.int32)[None, :]
        lens = np.array([s], dtype=np.int32)
        total = full_l * impl.pack_layer(pool, 0, bt, lens).nbytes
        total += win_l * impl.pack_layer(pool, 0, bt, lens, window=W).nbytes
        eq1 = C * H * D * 2 * (full_l * s + win_l * min(s, W))
        assert total == eq1, f"{model}: {total} B != per-kind Eq. 1 {eq1} B"
        decimals = len(printed.split(".")[1])
        assert any(math.isclose(round(total / u, decimals), float(printed), abs_tol=1e-12)
                   for u in (1e9, 2.0 ** 30)), f"{model}: {total} B does not round to {printed} GB"


QUICK_PINS = [pin_mla_ratio, pin_bruteforce_tiny, pin_page_take_transpose, pin_request_concat,
              pin_roundtrip, pin_multiset, pin_zero_and_opaque, pin_window_slice, pin_window_roundtrip]
FULL_PINS = QUICK_PINS + [pin_table1_sizes, pin_eq1_workloads, pin_layer_kind_sizes]


def failing_pins(impl, pins=QUICK_PINS):
    """Names of the pins the implementation violates."""
    bad = []
    for pin in pins:
        try:
            pin(impl)
        except (AssertionError, ValueError, IndexError) as e:  # a broken impl may also crash
            bad.append(f"{pin.__name__}: {e}")
    return bad

"""CPU oracle for layer moves between cache layouts: head-sliced pack and
unpack, pool-to-pool re-blocking, and head-major pools.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
calls it and shares no code with it.

What it computes.  The per-layer unit, the K-then-V token-major wire order
and the paged pools are those of the pack/unpack oracle (Section 5.2,
Section 3.5, Section 6).  Section 2.2 and Section 5.3 size a layer by its
KV heads: with grouped-query attention a layer holds h_kv heads of d_h
values per token and plane.  A layer can be moved between:

* a packed buffer: per request a block ``[C][n_r][hc][D]`` of the moved heads,
  blocks concatenated in request order (the pack/unpack wire order);
* a slot-major pool ``[L][NP][C][P][H][D]``: token t of request r lives at
  page ``bt_r[t div P]``, slot ``t mod P``;
* a head-major pool ``[L][NP][C][H][P][D]``: the same page and slot, but each
  head's P slots are contiguous inside a page plane.

A move copies, for every request r, kept token t (all of them, or with a
window W only the last W), plane c, slice head j < hc and dim d:

  dst(r, t, c, dst_head0 + j, d) = src(r, t, c, src_head0 + j, d)

Head-sliced pack is pool -> packed with hc < H (heads [h0, h0 + hc) of a
tensor-parallel shard), head-sliced unpack is packed -> pool, re-blocking is
pool -> pool between page sizes, and a head-major pool on either side changes
the layout inside each page.  Nothing else in a destination pool changes.
Elements are opaque words.

Pins live in the test suite: brute force over flat addresses on tiny pools,
the head partition of the pinned full-head pack, agreement of re-blocking with
the pinned unpack(pack(.)), and the identity-table case reducing to a
library axis swap.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .kvpack import window_start

PACKED, POOL, POOL_HEAD_MAJOR = "packed", "pool", "pool_head_major"


@dataclass
class View:
    """One side of a move.  `data` is the packed flat array or the whole
    pool; pool kinds name a layer slab, block tables and a first head."""
    kind: str
    data: np.ndarray
    layer: int = 0
    block_tables: np.ndarray | None = None
    head_begin: int = 0


def _page_size(v: View) -> int:
    return v.data.shape[3] if v.kind == POOL else v.data.shape[4]


def _gather(v: View, r: int, t: np.ndarray, hc: int, off: int, C: int, D: int) -> np.ndarray:
    """Request r's tokens t, heads [head_begin, head_begin + hc): ``[C][len(t)][hc][D]``."""
    if v.kind == PACKED:
        return v.data[off:off + C * t.size * hc * D].reshape(C, t.size, hc, D)
    P = _page_size(v)
    pages, slots = np.asarray(v.block_tables[r])[t // P], t % P
    heads = slice(v.head_begin, v.head_begin + hc)
    if v.kind == POOL:
        g = v.data[v.layer][pages, :, slots]            # (n, C, H, D)
    else:
        g = v.data[v.layer][pages, :, :, slots]         # advanced axes 0 and 3 -> (n, C, H, D)
    return g[:, :, heads].transpose(1, 0, 2, 3)


def _scatter(v: View, r: int, t: np.ndarray, hc: int, off: int, block: np.ndarray) -> None:
    if v.kind == PACKED:
        v.data[off:off + block.size] = block.reshape(-1)
        return
    P = _page_size(v)
    pages, slots = np.asarray(v.block_tables[r])[t // P], t % P
    heads = slice(v.head_begin, v.head_begin + hc)
    tok_major = block.transpose(1, 0, 2, 3)             # (n, C, hc, D)
    if v.kind == POOL:
        sel = v.data[v.layer][pages, :, slots]          # copy (n, C, H, D)
        sel[:, :, heads] = tok_major
        v.data[v.layer][pages, :, slots] = sel
    else:
        sel = v.data[v.layer][pages, :, :, slots]
        sel[:, :, heads] = tok_major
        v.data[v.layer][pages, :, :, slots] = sel


def _geometry(v: View):
    """(C, H, D) of a pool view."""
    if v.kind == POOL:
        return v.data.shape[2], v.data.shape[4], v.data.shape[5]
    return v.data.shape[2], v.data.shape[3], v.data.shape[5]


def move_layer(src: View, dst: View, seq_lens, head_count: int, window: int = 0) -> np.ndarray:
    """Copy one layer of every request from `src` to `dst` (dst.data is
    modified in place and returned)."""
    pool_side = src if src.kind != PACKED else dst
    if pool_side.kind == PACKED:
        raise ValueError("one side must be a pool")
    C, _, D = _geometry(pool_side)
    hc = int(head_count)
    for v in (src, dst):
        if v.kind != PACKED:
            c, H, d = _geometry(v)
            if (c, d) != (C, D) or not (0 <= v.head_begin and v.head_begin + hc <= H):
                raise ValueError("planes, head_dim or the head slice do not fit a pool")
        elif v.head_begin != 0:
            raise ValueError("a packed side holds exactly the moved heads")
    off = 0
    for r in range(len(seq_lens)):
        n = int(seq_lens[r])
        t = np.arange(window_start(n, window), n)
        block = _gather(src, r, t, hc, off, C, D)
        _scatter(dst, r, t, hc, off, block)
        off += block.size
    for v in (src, dst):
        if v.kind == PACKED and off != v.data.size:
            raise ValueError(f"packed buffer holds {v.data.size} elements, requests need {off}")
    return dst.data


def packed_heads_elems(planes: int, head_count: int, dim: int, seq_lens, window: int = 0) -> int:
    kept = sum(int(n) - window_start(int(n), window) for n in np.asarray(seq_lens).reshape(-1))
    return int(planes) * int(head_count) * int(dim) * kept


def pack_layer_heads(pool, layer, block_tables, seq_lens, head_begin, head_count, window=0):
    """Heads [head_begin, head_begin + head_count) of one layer of a
    slot-major pool, packed per request as ``[C][n_r][head_count][D]``."""
    C, D = pool.shape[2], pool.shape[5]
    out = np.empty(packed_heads_elems(C, head_count, D, seq_lens, window), dtype=pool.dtype)
    return move_layer(View(POOL, pool, layer, block_tables, head_begin), View(PACKED, out),
                      seq_lens, head_count, window)


def unpack_layer_heads(packed, pool, layer, block_tables, seq_lens, head_begin, head_count, window=0):
    """Scatter head-sliced packed blocks into heads [head_begin, +head_count)
    of a slot-major pool (in place; also returned)."""
    return move_layer(View(PACKED, packed), View(POOL, pool, layer, block_tables, head_begin),
                      seq_lens, head_count, window)


def reblock_layer(src_pool, src_layer, src_tables, dst_pool, dst_layer, dst_tables, seq_lens, window=0):
    """Pool to pool, page size P to P' (each pool's own), all heads."""
    return move_layer(View(POOL, src_pool, src_layer, src_tables), View(POOL, dst_pool, dst_layer, dst_tables),
                      seq_lens, src_pool.shape[4], window)


def to_head_major(pool: np.ndarray) -> np.ndarray:
    """The head-major layout of a slot-major pool: [L][NP][C][H][P][D]."""
    return np.ascontiguousarray(pool.transpose(0, 1, 2, 4, 3, 5))

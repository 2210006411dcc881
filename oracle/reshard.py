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
  blocks concatenated in request order (the pack/unpack wire order); with S
  shards (tensor-parallel receivers) the moved heads split into S equal runs,
  and shard s is such a buffer of its own ``hc / S`` heads, at element offset
  ``s * shard_elems``;
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
    shards: int = 1               # packed: shard regions of shard_elems elements each
    shard_elems: int = 0


def _page_size(v: View) -> int:
    return v.data.shape[3] if v.kind == POOL else v.data.shape[4]


def _shard_slices(v: View, off: int, n: int, hc: int, D: int, C: int):
    """(region slice, head slice) per shard of a packed view; `off` is this
    request's element offset inside one shard's buffer."""
    S = max(1, v.shards)
    hs = hc // S
    size = C * n * hs * D
    for s in range(S):
        base = s * v.shard_elems if S > 1 else 0
        yield slice(base + off, base + off + size), slice(s * hs, (s + 1) * hs)


def _gather(v: View, r: int, t: np.ndarray, hc: int, off: int, C: int, D: int) -> np.ndarray:
    """Request r's tokens t, heads [head_begin, head_begin + hc): ``[C][len(t)][hc][D]``."""
    if v.kind == PACKED:
        S = max(1, v.shards)
        parts = [v.data[reg].reshape(C, t.size, hc // S, D) for reg, _ in _shard_slices(v, off, t.size, hc, D, C)]
        return np.concatenate(parts, axis=2)
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
        C, D = block.shape[0], block.shape[3]
        for reg, heads in _shard_slices(v, off, t.size, hc, D, C):
            v.data[reg] = block[:, :, heads].reshape(-1)
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
        elif v.head_begin != 0 or hc % max(1, v.shards):
            raise ValueError("a packed side holds exactly the moved heads, in equal shards")
    off = 0                                      # elements into one shard's buffer
    for r in range(len(seq_lens)):
        n = int(seq_lens[r])
        t = np.arange(window_start(n, window), n)
        shards = max([1] + [v.shards for v in (src, dst) if v.kind == PACKED])
        block = _gather(src, r, t, hc, off, C, D)
        _scatter(dst, r, t, hc, off, block)
        off += block.size // shards
    for v in (src, dst):
        if v.kind == PACKED and not v.shard_elems and off != v.data.size:
            raise ValueError(f"packed buffer holds {v.data.size} elements, requests need {off}")
        if v.kind == PACKED and v.shard_elems and off > v.shard_elems:
            raise ValueError(f"shards hold {v.shard_elems} elements each, requests need {off}")
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


def pack_layer_shards(pool, layer, block_tables, seq_lens, head_begin, head_count, shards, shard_elems, window=0):
    """Heads [head_begin, +head_count) of one layer split into `shards` equal
    runs; shard s (heads head_begin + s*hc/S ...) packed into elements
    [s * shard_elems, ...) of the result."""
    out = np.zeros(int(shards) * int(shard_elems), dtype=pool.dtype)
    return move_layer(View(POOL, pool, layer, block_tables, head_begin),
                      View(PACKED, out, shards=int(shards), shard_elems=int(shard_elems)),
                      seq_lens, head_count, window)


def reblock_layer(src_pool, src_layer, src_tables, dst_pool, dst_layer, dst_tables, seq_lens, window=0):
    """Pool to pool, page size P to P' (each pool's own), all heads."""
    return move_layer(View(POOL, src_pool, src_layer, src_tables), View(POOL, dst_pool, dst_layer, dst_tables),
                      seq_lens, src_pool.shape[4], window)


def to_head_major(pool: np.ndarray) -> np.ndarray:
    """The head-major layout of a slot-major pool: [L][NP][C][H][P][D]."""
    return np.ascontiguousarray(pool.transpose(0, 1, 2, 4, 3, 5))

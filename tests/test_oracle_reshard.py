"""The layout-move oracle against its pins, and pin strength: each plausible
mistake planted in a copy of the oracle is caught by at least one pin.  CPU
only; the mutants live here, not in oracle/."""
import numpy as np
import pytest

import oracle.reshard as rs
import pins_reshard
from oracle import window_start


def test_oracle_passes_every_pin():
    assert pins_reshard.failing_pins(rs) == []


class Mutant:
    """The oracle's move with one planted mistake selected by `bug`."""
    View, PACKED, POOL, POOL_HEAD_MAJOR = rs.View, rs.PACKED, rs.POOL, rs.POOL_HEAD_MAJOR

    def __init__(self, bug):
        self.bug = bug

    def _where(self, v, r, t):
        P = v.data.shape[3] if v.kind == rs.POOL else v.data.shape[4]
        if self.bug == "reblock_uses_src_page_size" and v is self._dst and self._src.kind != rs.PACKED:
            P = self._src.data.shape[3] if self._src.kind == rs.POOL else self._src.data.shape[4]
        return np.asarray(v.block_tables[r])[t // P], t % P

    def _heads(self, v, hc):
        h0 = v.head_begin
        if self.bug == "head_begin_ignored" or (self.bug == "dst_head_begin_ignored" and v is self._dst):
            h0 = 0
        return slice(h0, h0 + hc)

    def _sel(self, v, pages, slots):
        kind = v.kind
        if self.bug == "head_major_read_as_slot_major":
            kind = rs.POOL
        if kind == rs.POOL:
            return v.data[v.layer][pages, :, slots], (pages, slice(None), slots)
        return v.data[v.layer][pages, :, :, slots], (pages, slice(None), slice(None), slots)

    def move_layer(self, src, dst, seq_lens, head_count, window=0):
        self._src, self._dst = src, dst
        pool_side = src if src.kind != rs.PACKED else dst
        C, D = pool_side.data.shape[2], pool_side.data.shape[5]
        hc, off = int(head_count), 0
        for r in range(len(seq_lens)):
            n = int(seq_lens[r])
            start = window_start(n, window)
            if self.bug == "window_ignored":
                start = 0
            t = np.arange(start, n)
            size = C * t.size * hc * D
            S = max([1] + [v.shards for v in (src, dst) if v.kind == rs.PACKED])
            if src.kind == rs.PACKED and S > 1:
                block = np.concatenate([src.data[self._shard_base(src, sh, off, size // S)].reshape(
                    C, t.size, hc // S, D) for sh in self._shard_order(S)], axis=2)
            elif src.kind == rs.PACKED:
                if self.bug == "packed_token_major":
                    block = src.data[off:off + size].reshape(t.size, C, hc, D).transpose(1, 0, 2, 3)
                else:
                    block = src.data[off:off + size].reshape(C, t.size, hc, D)
            else:
                pages, slots = self._where(src, r, t)
                g, _ = self._sel(src, pages, slots)
                block = g[:, :, self._heads(src, hc)].transpose(1, 0, 2, 3)
            if dst.kind == rs.PACKED and S > 1:
                for i, sh in enumerate(self._shard_order(S)):
                    dst.data[self._shard_base(dst, sh, off, size // S)] = \
                        block[:, :, i * (hc // S):(i + 1) * (hc // S)].reshape(-1)
            elif dst.kind == rs.PACKED:
                out = block.transpose(1, 0, 2, 3) if self.bug == "packed_token_major" else block
                dst.data[off:off + size] = out.reshape(-1)
            else:
                pages, slots = self._where(dst, r, t)
                sel, idx = self._sel(dst, pages, slots)
                heads = slice(None) if self.bug == "unpack_writes_all_heads" else self._heads(dst, hc)
                if self.bug == "unpack_writes_all_heads":
                    sel[:, :, :hc] = block.transpose(1, 0, 2, 3)
                else:
                    sel[:, :, heads] = block.transpose(1, 0, 2, 3)
                dst.data[dst.layer][idx] = sel
            off += size // S
        return dst.data

    def _shard_order(self, S):
        return list(reversed(range(S))) if self.bug == "shards_reversed" else list(range(S))

    def _shard_base(self, v, sh, off, size):
        base = sh * v.shard_elems
        if self.bug == "shard_offset_total":
            off = off * v.shards
        return slice(base + off, base + off + size)

    def pack_layer_heads(self, pool, layer, bts, lens, h0, hc, window=0):
        out = np.empty(rs.packed_heads_elems(pool.shape[2], hc, pool.shape[5], lens,
                                             0 if self.bug == "window_ignored" else window), dtype=pool.dtype)
        return self.move_layer(rs.View(rs.POOL, pool, layer, bts, h0), rs.View(rs.PACKED, out), lens, hc, window)

    def unpack_layer_heads(self, packed, pool, layer, bts, lens, h0, hc, window=0):
        return self.move_layer(rs.View(rs.PACKED, packed), rs.View(rs.POOL, pool, layer, bts, h0), lens, hc, window)

    def reblock_layer(self, src, sl, sbt, dst, dl, dbt, lens, window=0):
        return self.move_layer(rs.View(rs.POOL, src, sl, sbt), rs.View(rs.POOL, dst, dl, dbt), lens,
                               src.shape[4], window)


BUGS = ["head_begin_ignored", "dst_head_begin_ignored", "reblock_uses_src_page_size",
        "head_major_read_as_slot_major", "window_ignored", "packed_token_major", "unpack_writes_all_heads",
        "shards_reversed", "shard_offset_total"]


def test_unmutated_copy_passes():
    assert pins_reshard.failing_pins(Mutant(None)) == []


@pytest.mark.parametrize("bug", BUGS)
def test_mutant_is_caught(bug):
    assert pins_reshard.failing_pins(Mutant(bug)), f"no pin catches the planted mistake {bug!r}"

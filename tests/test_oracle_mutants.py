"""Pin strength: each plausible mistake planted in a copy of the oracle must be
caught by at least one pin.  CPU only; the mutants live here, not in oracle/."""
import numpy as np
import pytest

import pins


class Mutant:
    """The oracle's pack/unpack with one planted mistake selected by `bug`."""

    def __init__(self, bug):
        self.bug = bug

    def _start(self, n, W):
        if self.bug == "window_keeps_first":
            return 0
        if self.bug == "window_off_by_one":
            return n - W + 1 if 0 < W < n else 0
        return n - W if 0 < W < n else 0

    def _count(self, n, W):
        if self.bug == "window_keeps_first" and 0 < W < n:
            return W
        return n - self._start(n, W)

    def _index(self, bt, n, P, W=0):
        t = np.arange(self._start(n, W), n)
        if self.bug == "window_keeps_first" and 0 < W < n:
            t = np.arange(0, W)
        if self.bug == "div_mod_swapped":
            return np.asarray(bt)[t % P], t // P
        if self.bug == "token_off_by_one":
            return np.asarray(bt)[np.minimum(t + 1, n - 1) // P], (np.minimum(t + 1, n - 1)) % P
        if self.bug == "slot_reversed":
            return np.asarray(bt)[t // P], (P - 1) - t % P
        return np.asarray(bt)[t // P], t % P

    def pack_request(self, pool, layer, bt, n, W=0):
        P = pool.shape[3]
        n = int(n)
        pages, slots = self._index(bt, n, P, W)
        if self.bug == "wrong_layer":
            layer = 0
        g = pool[layer][pages, :, slots]                      # (n, C, H, D)
        if self.bug == "no_plane_transpose":
            out = g
        elif self.bug == "heads_dims_swapped":
            out = g.transpose(1, 0, 3, 2)
        else:
            out = g.transpose(1, 0, 2, 3)
        if self.bug == "drops_v_plane":
            out = out[:1]
        return np.ascontiguousarray(out)

    def pack_layer(self, pool, layer, bts, lens, window=0):
        order = range(len(lens))
        if self.bug == "requests_reversed":
            order = reversed(list(order))
        parts = [self.pack_request(pool, layer, bts[r], lens[r], window).reshape(-1) for r in order]
        return np.concatenate(parts) if parts else np.empty(0, pool.dtype)

    def unpack_layer(self, packed, pool, layer, bts, lens, window=0):
        C, P, H, D = pool.shape[2], pool.shape[3], pool.shape[4], pool.shape[5]
        if self.bug == "unpack_assumes_page16":
            P = 16
        off = 0
        for r in range(len(lens)):
            n = int(lens[r])
            cnt = self._count(n, window)
            size = C * cnt * H * D
            start = 0 if self.bug == "unpack_no_request_offset" else off
            block = packed[start:start + size].reshape(C, cnt, H, D)
            pages, slots = self._index(bts[r], n, P, window)
            pool[layer][pages, :, slots % pool.shape[3]] = block.transpose(1, 0, 2, 3)
            if self.bug == "unpack_zero_fills_tail" and n % pool.shape[3]:
                pool[layer][bts[r][(n - 1) // pool.shape[3]], :, n % pool.shape[3]:] = 0
            off += size
        return pool


BUGS = ["div_mod_swapped", "token_off_by_one", "slot_reversed", "wrong_layer",
        "no_plane_transpose", "heads_dims_swapped", "drops_v_plane", "requests_reversed",
        "unpack_assumes_page16", "unpack_no_request_offset", "unpack_zero_fills_tail",
        "window_keeps_first", "window_off_by_one"]


def test_unmutated_copy_passes():
    assert pins.failing_pins(Mutant(None)) == []


@pytest.mark.parametrize("bug", BUGS)
def test_mutant_is_caught(bug):
    failed = pins.failing_pins(Mutant(bug))
    assert failed, f"no pin catches the planted mistake {bug!r}"

"""The fixed-state oracle against its pins, and pin strength: each plausible
mistake planted in a copy of the oracle is caught by at least one pin.  CPU
only; the mutants live here, not in oracle/."""
import numpy as np
import pytest

import oracle.state as so
import pins_state
from oracle import window_start


def test_oracle_passes_every_pin():
    assert pins_state.failing_pins(so) == []


class Mutant:
    """The oracle's state moves and sizes with one planted mistake."""

    def __init__(self, bug):
        self.bug = bug

    def _slots(self, slots):
        slots = np.asarray(slots, dtype=np.int64).reshape(-1)
        if self.bug == "slot_is_request_index":
            return np.arange(slots.size)
        if self.bug == "slots_reversed":
            return slots[::-1]
        return slots

    def pack_state_layer(self, state, layer, slots):
        s = self._slots(slots)
        if self.bug == "layer_ignored":
            layer = 0
        block = state[layer][s]
        if self.bug == "word_major" and block.size:
            block = block.T
        return np.ascontiguousarray(block).reshape(-1)

    def unpack_state_layer(self, packed, state, layer, slots):
        s = self._slots(slots)
        E = state.shape[2]
        if self.bug == "unpack_layer_off_by_one":
            layer = (layer + 1) % state.shape[0]
        rows = packed.reshape(s.size, E)
        if self.bug == "unpack_clears_other_slots":
            state[layer][:] = 0
        state[layer][s] = rows
        return state

    def request_bytes(self, kinds, seq_len, planes, heads, dim, elem_bytes, state_bytes=0):
        row = planes * heads * dim * elem_bytes
        n, total = int(seq_len), 0
        for k in kinds:
            if k[0] == "full":
                total += row * n
            elif k[0] == "window":
                kept = n if self.bug == "window_not_capped" else n - window_start(n, k[1])
                total += row * kept
            else:
                total += state_bytes * (max(n, 1) if self.bug == "state_grows_with_length" else 1)
                if self.bug == "state_counts_kv_planes":
                    total += state_bytes
        return total


BUGS = ["slot_is_request_index", "slots_reversed", "layer_ignored", "word_major", "unpack_layer_off_by_one",
        "unpack_clears_other_slots", "window_not_capped", "state_grows_with_length", "state_counts_kv_planes"]


def test_unmutated_copy_passes():
    assert pins_state.failing_pins(Mutant(None)) == []


@pytest.mark.parametrize("bug", BUGS)
def test_mutant_is_caught(bug):
    assert pins_state.failing_pins(Mutant(bug)), f"no pin catches the planted mistake {bug!r}"

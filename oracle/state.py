"""CPU oracle for fixed-state layers and for the per-layer-kind size of a
whole request (Section 2.2).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
calls it and shares no code with it.

What it computes.  Section 2.2 extends Eq. 1 per layer kind: a full-attention
layer holds every token, a windowed layer only its last W tokens, an MLA
layer one latent per token (Section 5.3), and a linear-attention layer a
fixed state whose size does not depend on the sequence length.  The unit of
transfer stays one layer (Section 5.2).

A serving engine keeps a fixed-state layer's state per request in a slot of a
state cache (there are no tokens, hence no pages and no block tables):

  state cache   state[layer][slot][e]        e < E words of one request's state
  pack          out[r * E + e] = state[layer][slot_r][e]        for r < R, e < E
  unpack        state'[layer][slot'_r][e] = in[r * E + e]       every other slot keeps its value

so a batch is the requests' states in request order.  Elements are opaque
words.

Pins live in the test suite: brute force over flat addresses, the round trip
with untouched slots, agreement with the paged pack of a one-page request of
E words (a fixed state as a request whose single page holds it), and the
Section 2.2 size of the hybrid model.
"""
from __future__ import annotations

import numpy as np

from .kvpack import window_start


def _check_state(state: np.ndarray) -> None:
    if state.ndim != 3:
        raise ValueError("state cache must be [layers][slots][words]")


def pack_state_layer(state: np.ndarray, layer: int, slots) -> np.ndarray:
    """The states of requests r = 0..R-1 (slot ``slots[r]``) of one layer,
    concatenated in request order."""
    _check_state(state)
    slots = np.asarray(slots, dtype=np.int64).reshape(-1)
    if slots.size == 0:
        return np.empty(0, dtype=state.dtype)
    if slots.min() < 0 or slots.max() >= state.shape[1]:
        raise ValueError("slot outside the state cache")
    return np.ascontiguousarray(state[layer][slots]).reshape(-1)


def unpack_state_layer(packed: np.ndarray, state: np.ndarray, layer: int, slots) -> np.ndarray:
    """Write request r's state from ``packed`` into slot ``slots[r]`` of one
    layer (``state`` is modified in place and returned)."""
    _check_state(state)
    slots = np.asarray(slots, dtype=np.int64).reshape(-1)
    E = state.shape[2]
    if packed.size != slots.size * E:
        raise ValueError(f"packed buffer holds {packed.size} words, {slots.size} states need {slots.size * E}")
    if slots.size and (slots.min() < 0 or slots.max() >= state.shape[1]):
        raise ValueError("slot outside the state cache")
    if np.unique(slots).size != slots.size:
        raise ValueError("two requests name the same destination slot")
    state[layer][slots] = packed.reshape(slots.size, E)
    return state


def request_bytes(layer_kinds, seq_len: int, planes: int, heads: int, dim: int, elem_bytes: int,
                  state_bytes: int = 0) -> int:
    """Section 2.2's per-layer-kind Eq. 1 for one request of ``seq_len``
    tokens: ``layer_kinds`` lists every layer as ("full",), ("window", W) or
    ("state",).  Attention layers hold planes * heads * dim words per kept
    token; a state layer holds ``state_bytes`` whatever the length."""
    row = int(planes) * int(heads) * int(dim) * int(elem_bytes)
    n = int(seq_len)
    total = 0
    for kind in layer_kinds:
        if kind[0] == "full":
            total += row * n
        elif kind[0] == "window":
            total += row * (n - window_start(n, int(kind[1])))
        elif kind[0] == "state":
            total += int(state_bytes)
        else:
            raise ValueError(f"unknown layer kind {kind!r}")
    return total

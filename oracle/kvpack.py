"""CPU oracle for per-layer paged KV-cache pack / unpack.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the HIP
library and its Python binding) never calls it, and it shares no code with
that path: it reads the layouts below and nothing else.

What it computes (arxiv 2607.28633, "Topology-Aware Data Movement for
Disaggregated GPU Inference"):

* Section 5.2 (pipelining overlap model): a prefill worker ships layer l's KV
  cache while later layers still compute, so the unit of work is ONE LAYER.
* Section 3.5 (KV cache serialization): on the wire K and V are separate
  contiguous tensors indexed [seq_len][kv_heads][head_dim] within a layer,
  which is what makes single-DMA sends possible.
* Section 6 (related work, PagedAttention): prefill and decode workers hold
  the cache in fixed-size pages reached through per-request block tables.
* Section 2.2, Eq. 1: the bytes moved for a request of s tokens are
  2 * L * h_kv * d_h * s * b_p; Section 5.3: an MLA cache keeps one shared
  576-wide latent per token and layer, so the factor 2 (separate K and V)
  is dropped.  Section 2.2 extends Eq. 1 per layer kind: a windowed
  (sliding-window attention) layer holds only its last W tokens, so its
  transfer moves tokens [max(0, s - W), s) only.

Hence, for one layer ``l`` (pool ``[L][NP][C][P][H][D]``, C planes = 2 for K|V
and 1 for an MLA latent):

  pack    out_r[c][t][h][d] = pool[l][bt_r[t div P]][c][t mod P][h][d]  for t < n_r
  unpack  pool'[l][bt'_r[t div P']][c][t mod P'][h][d] = in_r[c][t][h][d] for t < n_r

A windowed layer (``window`` W > 0) keeps tokens t in [max(0, n_r - W), n_r)
only: the packed block is ``[C][min(n_r, W)][H][D]`` and unpack writes those
tokens at their own positions.  A batch concatenates the per-request blocks
in request order.  Unpack writes only the slots of valid tokens: every other element of
the destination pool (other pages, and slots >= n_r mod P' of a request's last
page) keeps its prior value.  Entries of a block table past the request's
``ceil(n_r / P)`` pages are never read.  Elements are opaque words: the
oracle runs on unsigned-integer views and does no arithmetic on values.

Pins (none of which re-derives this definition) live in the test suite:
Eq. 1 and the Table 1 / Section 5.3 figures for sizes, the identity-table
case reducing to a textbook transpose, equivariance under page relabelling,
token-prefix truncation, the pack/unpack round trip, a word-multiset
invariant, and brute force on the tiny pool through flat-address arithmetic.
"""
from __future__ import annotations

import numpy as np


def _check_pool(pool):
    if pool.ndim != 6:
        raise ValueError("pool must be [layers][pages][planes][page_size][heads][dim]")


def window_start(seq_len: int, window: int) -> int:
    """First token a windowed layer keeps: the last `window` tokens survive
    (Section 2.2); window 0 keeps every token."""
    n = int(seq_len)
    return n - int(window) if 0 < int(window) < n else 0


def pack_request(pool: np.ndarray, layer: int, block_table: np.ndarray, seq_len: int,
                 window: int = 0) -> np.ndarray:
    """One request, one layer: gather its pages into ``[C][n][H][D]``.

    Token t of the request sits in physical page ``block_table[t // P]`` at
    slot ``t % P`` (paged layout, Section 6); the result lists K then V
    (planes), each token-major with heads and dims inside (Section 3.5).
    With a window only tokens [window_start, n) are gathered.
    """
    _check_pool(pool)
    P = pool.shape[3]
    n = int(seq_len)
    t = np.arange(window_start(n, window), n)
    pages = np.asarray(block_table)[t // P]
    slots = t % P
    # advanced indices on axes 0 and 2 of pool[layer] -> result (n, C, H, D)
    gathered = pool[layer][pages, :, slots]
    return np.ascontiguousarray(gathered.transpose(1, 0, 2, 3))


def pack_layer(pool: np.ndarray, layer: int, block_tables: np.ndarray,
               seq_lens: np.ndarray, window: int = 0) -> np.ndarray:
    """A batch of requests, one layer: flat buffer of the per-request
    ``[C][n_r][H][D]`` blocks in request order."""
    _check_pool(pool)
    parts = [pack_request(pool, layer, block_tables[r], int(seq_lens[r]), window).reshape(-1)
             for r in range(len(seq_lens))]
    if not parts:
        return np.empty(0, dtype=pool.dtype)
    return np.concatenate(parts)


def unpack_request(packed_r: np.ndarray, pool: np.ndarray, layer: int,
                   block_table: np.ndarray, seq_len: int, window: int = 0) -> None:
    """Inverse of :func:`pack_request` into ``pool`` (modified in place).

    The destination page size P' is the pool's own; it need not equal the
    page size the data was packed from (the packed form has no pages).
    """
    _check_pool(pool)
    C, P, H, D = pool.shape[2], pool.shape[3], pool.shape[4], pool.shape[5]
    n = int(seq_len)
    t = np.arange(window_start(n, window), n)
    block = np.asarray(packed_r).reshape(C, t.size, H, D)
    pages = np.asarray(block_table)[t // P]
    slots = t % P
    view = pool[layer]
    view[pages, :, slots] = block.transpose(1, 0, 2, 3)


def unpack_layer(packed: np.ndarray, pool: np.ndarray, layer: int,
                 block_tables: np.ndarray, seq_lens: np.ndarray, window: int = 0) -> np.ndarray:
    """A batch of requests, one layer, scattered into ``pool`` (in place;
    also returned).  Request r's block starts where requests < r end."""
    _check_pool(pool)
    C, H, D = pool.shape[2], pool.shape[4], pool.shape[5]
    off = 0
    for r in range(len(seq_lens)):
        n = int(seq_lens[r])
        size = C * (n - window_start(n, window)) * H * D
        unpack_request(packed[off:off + size], pool, layer, block_tables[r], n, window)
        off += size
    if off != packed.size:
        raise ValueError(f"packed buffer holds {packed.size} elements, requests need {off}")
    return pool


def packed_layer_elems(planes: int, heads: int, dim: int, seq_lens, window: int = 0) -> int:
    """Elements in one layer's packed batch: C * H * D * sum(kept tokens)."""
    kept = sum(int(n) - window_start(int(n), window) for n in np.asarray(seq_lens).reshape(-1))
    return int(planes) * int(heads) * int(dim) * kept

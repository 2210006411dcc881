"""Seeded synthetic inputs for per-layer paged KV-cache pack/unpack.

This module only *draws inputs*: request lengths, page assignments (block
tables) and pool contents.  It contains none of the pack/unpack arithmetic, so
both the CPU oracle (tests) and the HIP path (library, bench) may consume it
without sharing any of the operation itself.

Pool layout (both source and destination pools), element-indexed:

    pool[layer][page][plane][slot][head][dim]

``plane`` is 0 = K, 1 = V for GQA/MHA caches (``planes == 2``) and the single
latent vector for MLA caches (``planes == 1``, the paper's Section 5.3 rule that
the K/V factor of two does not apply to the shared latent).  ``slot`` runs over
the ``page_size`` tokens of a page.  Element values are opaque ``elem_bytes``
words (bf16 by default), stored here as unsigned integers of that width.

Workload shapes follow the model rows of the paper's Table 1 (Section 2.2):
Llama-3-70B GQA (80 layers, 8 KV heads, head_dim 128), DeepSeek-V3 MLA
(61 layers, one 576-wide latent = 512 + 64 rope, Section 5.3), and a
Llama-3-8B-shaped cache with the same per-layer shape as 70B.  The paper names
no dataset; lengths and page assignments are drawn from the distributions
listed in ``WORKLOADS`` below.

Draw order for one seed: request lengths -> source page permutation ->
destination page permutation (all from ``numpy.random.default_rng(seed)``).
Pool contents come from independent streams (``default_rng([seed, 1])`` for
the source pool, ``default_rng([seed, 2])`` for the destination pre-fill), so a
pool can be regenerated without redrawing the tables.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

UINT_FOR_BYTES = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


@dataclasses.dataclass
class Workload:
    """One seeded pack/unpack workload.

    Tables are host numpy arrays.  ``block_tables[r, i]`` is the physical page
    in the source pool holding logical page ``i`` of request ``r``;
    ``dst_block_tables`` is the same for the destination pool, whose page size
    may differ.  Unused table entries hold -1.
    """

    name: str
    seed: int
    num_layers: int          # logical layers swept per pass
    phys_layers: int         # layers physically allocated (layer l lives in slab l % phys_layers)
    planes: int              # 2 = K|V, 1 = MLA latent
    num_heads: int
    head_dim: int
    elem_bytes: int
    page_size: int           # source pool tokens per page
    num_pages: int           # source pool pages per layer
    dst_page_size: int
    dst_num_pages: int
    seq_lens: np.ndarray     # int32 [R]
    block_tables: np.ndarray       # int32 [R, max_pages_src]
    dst_block_tables: np.ndarray   # int32 [R, max_pages_dst]
    layer_windows: tuple = ()      # per logical layer: 0 = full attention, W > 0 = last-W-token window
    # Fixed-state (linear-attention) layers, Section 2.2: per logical layer True = the layer holds a
    # per-request state of state_bytes in a state cache [state_phys_layers][slots][state_bytes]
    # instead of paged K/V; request r's state sits in slot state_slots[r] (dst_state_slots[r] on
    # the receiving side).
    layer_state: tuple = ()
    state_bytes: int = 0
    state_phys_layers: int = 0
    num_state_slots: int = 0
    dst_num_state_slots: int = 0
    state_slots: Optional[np.ndarray] = None       # int32 [R]
    dst_state_slots: Optional[np.ndarray] = None   # int32 [R]

    def window(self, layer: int) -> int:
        return int(self.layer_windows[layer]) if self.layer_windows else 0

    def is_state(self, layer: int) -> bool:
        return bool(self.layer_state[layer]) if self.layer_state else False

    def kv_slab(self, layer: int) -> int:
        """Physical K/V layer slab of logical layer `layer` (attention layers
        are numbered among themselves when the model also has state layers)."""
        if not self.layer_state:
            return layer % self.phys_layers
        return sum(1 for l in range(layer) if not self.layer_state[l]) % self.phys_layers

    def state_slab(self, layer: int) -> int:
        """State-cache layer of logical layer `layer` (a state layer)."""
        return sum(1 for l in range(layer) if self.layer_state[l]) % self.state_phys_layers

    def state_shape(self, dst: bool = False) -> tuple:
        slots = self.dst_num_state_slots if dst else self.num_state_slots
        return (self.state_phys_layers, slots, self.state_bytes // self.elem_bytes)

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def uint_dtype(self):
        return UINT_FOR_BYTES[self.elem_bytes]

    def pool_shape(self, dst: bool = False) -> tuple:
        p = self.dst_page_size if dst else self.page_size
        npg = self.dst_num_pages if dst else self.num_pages
        return (self.phys_layers, npg, self.planes, p, self.num_heads, self.head_dim)

    def pool_elems(self, dst: bool = False) -> int:
        return int(np.prod(self.pool_shape(dst), dtype=np.int64))

    def describe(self) -> dict:
        return {
            "workload": self.name, "seed": self.seed, "layers": self.num_layers,
            "phys_layers": self.phys_layers, "planes": self.planes,
            "kv_heads": self.num_heads, "head_dim": self.head_dim,
            "elem_bytes": self.elem_bytes, "page_size": self.page_size,
            "dst_page_size": self.dst_page_size, "pool_pages": self.num_pages,
            "dst_pool_pages": self.dst_num_pages, "requests": self.num_reqs,
            "tokens": int(self.seq_lens.astype(np.int64).sum()),
            "windowed_layers": sum(1 for w in self.layer_windows if w),
            "state_layers": sum(1 for x in self.layer_state if x),
            "state_bytes": self.state_bytes,
        }


def _pages_for(n: int, page_size: int) -> int:
    # how many pages a request of n tokens occupies (input construction only)
    return -(-int(n) // int(page_size))


def _tables(rng, seq_lens, page_size, num_pages):
    """Draw a permutation of the pool and hand request r the next pages of it."""
    perm = rng.permutation(num_pages).astype(np.int32)
    counts = [_pages_for(n, page_size) for n in seq_lens]
    stride = max([1] + counts)
    bt = np.full((len(seq_lens), stride), -1, dtype=np.int32)
    cur = 0
    for r, k in enumerate(counts):
        if cur + k > num_pages:
            raise ValueError("pool too small for the drawn requests")
        bt[r, :k] = perm[cur:cur + k]
        cur += k
    return bt


def _lognormal_lengths(rng, count, median, sigma, lo, hi):
    z = rng.standard_normal(count)
    n = np.rint(np.exp(math.log(median) + sigma * z))
    return np.clip(n, lo, hi).astype(np.int32)


# name -> (description, builder).  Each builder returns the shape dict and the
# lengths; pool sizing follows the workload's own rule.
WORKLOADS = {
    "tiny": "2 layers, 2 KV heads, head_dim 64, page 16, 64-page pools, 4 requests of 64/48/33/17 tokens",
    "llama3-8b": "32 layers, 8 KV heads, head_dim 128, page 16, one 4096-token request, 4096-page pools",
    "llama3-70b-4k": "80 layers, 8 KV heads, head_dim 128, page 16, one 4096-token request, 4096-page pools",
    "llama3-70b-batch8": "80 layers, 8 KV heads, head_dim 128, page 16, 8 requests (4096 + 7 x U[1024,8192]), pools 1.25x pages",
    "deepseek-v3-mla": "61 layers, 1 x 576 latent (no K/V split), page 64, 32 requests lognormal(median 4096, sigma 1) in [512,16384], pools 1.25x pages",
    "reblock-70b": "80 layers, 8 KV heads, head_dim 128, page 16 -> 64, 100 requests lognormal(median 4096, sigma 1) in [256,32768], pools 1.25x pages, 8 physical layer slabs",
    "gpt-oss-120b": "36 layers alternating 128-token sliding window / full attention, 8 KV heads, head_dim 64, page 16, 32 requests lognormal(median 4096, sigma 1) in [512,16384], pools 1.25x pages",
    "llama3-70b-tp8": "one GPU's share of 70B at tensor parallelism 8: 80 layers, 1 KV head, head_dim 128, page 16, one 4096-token request, 4096-page pools",
    "qwen3.5-397b-hybrid": "60 layers: every fourth full attention (2 KV heads, head_dim 256, page 16), the other 45 linear attention with a 2,170,880-byte state per request, 32 requests lognormal(median 4096, sigma 1) in [512,16384], pools and state slots 1.25x",
}

# Fixed state of one linear-attention layer of the hybrid shape, per request (bf16 words): the
# recurrent state of 64 value heads x 128 x 128 plus a 3-step causal-convolution state over
# 2 x 16 x 128 + 64 x 128 channels.
HYBRID_STATE_BYTES = 2 * (64 * 128 * 128 + 3 * (2 * 16 * 128 + 64 * 128))

DEFAULT_SEEDS = {"tiny": 0, "llama3-8b": 1, "llama3-70b-batch8": 2, "deepseek-v3-mla": 3,
                 "reblock-70b": 4, "llama3-70b-4k": 5, "gpt-oss-120b": 6, "llama3-70b-tp8": 7,
                 "qwen3.5-397b-hybrid": 8}


def make_workload(name: str, seed: Optional[int] = None, *,
                  num_layers: Optional[int] = None, phys_layers: Optional[int] = None,
                  seq_lens: Optional[Sequence[int]] = None,
                  page_size: Optional[int] = None, dst_page_size: Optional[int] = None,
                  num_pages: Optional[int] = None, dst_num_pages: Optional[int] = None,
                  num_heads: Optional[int] = None, head_dim: Optional[int] = None,
                  planes: Optional[int] = None, elem_bytes: int = 2,
                  pool_slack: float = 1.25, state_bytes: Optional[int] = None) -> Workload:
    """Build a named workload; keyword overrides shrink or reshape it for tests."""
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    seed = DEFAULT_SEEDS[name] if seed is None else int(seed)
    rng = np.random.default_rng(seed)

    if name == "tiny":
        shape = dict(L=2, C=2, H=2, D=64, P=16, P2=16)
        lens = np.array([64, 48, 33, 17], dtype=np.int32)
        pools = (64, 64)
    elif name in ("llama3-8b", "llama3-70b-4k", "llama3-70b-tp8"):
        shape = dict(L=32 if name == "llama3-8b" else 80, C=2, H=1 if name == "llama3-70b-tp8" else 8,
                     D=128, P=16, P2=16)
        lens = np.array([4096], dtype=np.int32)
        pools = (4096, 4096)
    elif name == "llama3-70b-batch8":
        shape = dict(L=80, C=2, H=8, D=128, P=16, P2=16)
        rest = rng.integers(1024, 8192, size=7, endpoint=True)
        lens = np.concatenate([[4096], rest]).astype(np.int32)
        pools = None
    elif name == "deepseek-v3-mla":
        shape = dict(L=61, C=1, H=1, D=576, P=64, P2=64)
        lens = _lognormal_lengths(rng, 32, 4096, 1.0, 512, 16384)
        pools = None
    elif name == "gpt-oss-120b":
        shape = dict(L=36, C=2, H=8, D=64, P=16, P2=16)
        lens = _lognormal_lengths(rng, 32, 4096, 1.0, 512, 16384)
        pools = None
    elif name == "qwen3.5-397b-hybrid":
        shape = dict(L=60, C=2, H=2, D=256, P=16, P2=16)
        lens = _lognormal_lengths(rng, 32, 4096, 1.0, 512, 16384)
        pools = None
    else:  # reblock-70b
        shape = dict(L=80, C=2, H=8, D=128, P=16, P2=64)
        lens = _lognormal_lengths(rng, 100, 4096, 1.0, 256, 32768)
        pools = None

    if seq_lens is not None:
        lens = np.asarray(seq_lens, dtype=np.int32)
    L = shape["L"] if num_layers is None else int(num_layers)
    P = shape["P"] if page_size is None else int(page_size)
    P2 = shape["P2"] if dst_page_size is None else int(dst_page_size)
    C = shape["C"] if planes is None else int(planes)
    H = shape["H"] if num_heads is None else int(num_heads)
    D = shape["D"] if head_dim is None else int(head_dim)
    need_src = sum(_pages_for(n, P) for n in lens)
    need_dst = sum(_pages_for(n, P2) for n in lens)
    if pools is not None and seq_lens is None and page_size is None and dst_page_size is None:
        np_src, np_dst = pools
    else:
        np_src = max(1, math.ceil(pool_slack * need_src))
        np_dst = max(1, math.ceil(pool_slack * need_dst))
    if num_pages is not None:
        np_src = int(num_pages)
    if dst_num_pages is not None:
        np_dst = int(dst_num_pages)
    hybrid = name == "qwen3.5-397b-hybrid"
    state = tuple(l % 4 != 3 for l in range(L)) if hybrid else ()
    if phys_layers is None:
        if name == "reblock-70b":
            phys_layers = min(L, 8)
        elif hybrid:
            phys_layers = max(1, sum(1 for x in state if not x))
        else:
            phys_layers = L

    bt = _tables(rng, lens, P, np_src)
    bt2 = _tables(rng, lens, P2, np_dst)
    windows = tuple(128 if l % 2 == 0 else 0 for l in range(L)) if name == "gpt-oss-120b" else ()
    extra = {}
    if hybrid:
        R = len(lens)
        ns = max(1, math.ceil(pool_slack * R))
        sb = HYBRID_STATE_BYTES if state_bytes is None else int(state_bytes)
        if sb % int(elem_bytes):
            raise ValueError("state_bytes must be a whole number of elements")
        extra = dict(layer_state=state, state_bytes=sb, state_phys_layers=max(1, sum(state)),
                     num_state_slots=ns, dst_num_state_slots=ns,
                     state_slots=rng.permutation(ns)[:R].astype(np.int32),
                     dst_state_slots=rng.permutation(ns)[:R].astype(np.int32))
    return Workload(name=name, seed=seed, num_layers=L, phys_layers=int(phys_layers),
                    planes=C, num_heads=H, head_dim=D, elem_bytes=int(elem_bytes),
                    page_size=P, num_pages=np_src, dst_page_size=P2, dst_num_pages=np_dst,
                    seq_lens=lens, block_tables=bt, dst_block_tables=bt2, layer_windows=windows, **extra)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def host_src_pool(wl: Workload) -> np.ndarray:
    """Source pool contents on the host: bf16 ~ N(0, 1) (2-byte elements), else
    uniform random words.  Shape ``wl.pool_shape()``, unsigned dtype."""
    rng = np.random.default_rng([wl.seed, 1])
    shape = wl.pool_shape()
    if wl.elem_bytes == 2:
        return bf16_bits_from_f32(rng.standard_normal(shape, dtype=np.float32))
    return random_words(rng, shape, wl.elem_bytes)


def host_dst_prefill(wl: Workload) -> np.ndarray:
    """Destination pool pre-fill: a distinct seeded pattern of arbitrary words,
    so bytes an unpack must leave alone are recognisable."""
    rng = np.random.default_rng([wl.seed, 2])
    return random_words(rng, wl.pool_shape(dst=True), wl.elem_bytes)


def random_words(rng, shape, elem_bytes: int) -> np.ndarray:
    """Uniform random unsigned words of the given width (every bit pattern,
    including NaN/Inf/-0/subnormal encodings when read as floats)."""
    dt = UINT_FOR_BYTES[elem_bytes]
    n = int(np.prod(shape, dtype=np.int64))
    raw = rng.integers(0, 256, size=n * elem_bytes, dtype=np.uint8)
    return raw.view(dt).reshape(shape)


def device_src_pool(wl: Workload, device="cuda"):
    """Source pool generated on the device (multi-GB pools): bf16 ~ N(0, 1) from
    a seeded torch generator, filled one layer slab at a time.  Returned as a
    torch tensor of the pool shape."""
    import torch
    if wl.elem_bytes != 2:
        raise ValueError("device generation is for bf16 pools")
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed * 1000003 + 1)
    t = torch.empty(wl.pool_shape(), device=device, dtype=torch.bfloat16)
    for layer in range(t.shape[0]):
        t[layer].normal_(generator=g)
    return t


def device_dst_prefill(wl: Workload, device="cuda"):
    """Destination pool pre-fill on the device: arbitrary seeded 16-bit words
    (every bit pattern), one layer slab at a time."""
    import torch
    if wl.elem_bytes != 2:
        raise ValueError("device generation is for bf16 pools")
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed * 1000003 + 2)
    t = torch.empty(wl.pool_shape(dst=True), device=device, dtype=torch.int16)
    for layer in range(t.shape[0]):
        t[layer].random_(-32768, 32768, generator=g)
    return t.view(torch.bfloat16)


def host_state_cache(wl: Workload, dst: bool = False) -> np.ndarray:
    """State cache contents on the host, shape ``wl.state_shape(dst)``: the
    source holds bf16 ~ N(0, 1) (2-byte elements, else random words), the
    destination a distinct pre-fill of arbitrary words."""
    rng = np.random.default_rng([wl.seed, 4 if dst else 3])
    shape = wl.state_shape(dst)
    if wl.elem_bytes == 2 and not dst:
        return bf16_bits_from_f32(rng.standard_normal(shape, dtype=np.float32))
    return random_words(rng, shape, wl.elem_bytes)


def device_state_cache(wl: Workload, dst: bool = False, device="cuda"):
    """State cache generated on the device (bf16 ~ N(0, 1) for the source,
    arbitrary 16-bit words for the destination pre-fill), one layer at a time."""
    import torch
    if wl.elem_bytes != 2:
        raise ValueError("device generation is for bf16 caches")
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed * 1000003 + (4 if dst else 3))
    t = torch.empty(wl.state_shape(dst), device=device, dtype=torch.int16)
    for layer in range(t.shape[0]):
        if dst:
            t[layer].random_(-32768, 32768, generator=g)
        else:
            t[layer].view(torch.bfloat16).normal_(generator=g)
    return t

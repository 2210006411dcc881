"""KV cache serialization in the paper's KVCACHE1 format.  TEST INFRASTRUCTURE
ONLY (the CPU oracle).

Section 3.5: a fixed 128-byte header holding an 8-byte magic "KVCACHE1", a
request ID, a model ID, the tensor dimensions (sequence length, layers, KV
heads, head dim), the tensor sizes and a CRC-64 of the key tensor and of the
value tensor; then the key tensor and the value tensor, each laid out
[layers][seq_len][kv_heads][head_dim], back to back.

The paper fixes neither field widths nor byte order nor the CRC polynomial.
Readings used here (and by the GPU implementation):
  * little-endian; offsets: magic 0, request_id u64 8, model_id u64 16,
    seq_len u32 24, layers u32 28, kv_heads u32 32, head_dim u32 36,
    elem_bytes u32 40, planes u32 44, k_bytes u64 48, v_bytes u64 56,
    crc_k u64 64, crc_v u64 72, zero bytes 80..127;
  * CRC-64/XZ (ECMA-182, reflected, all-ones preset and final complement);
  * an MLA cache (one latent plane, Section 5.3) is stored as the key tensor
    with v_bytes = 0 (the CRC of an empty value tensor is 0).
"""
import struct

import numpy as np

from .crc64 import crc64
from .kvpack import pack_request, unpack_request

MAGIC = b"KVCACHE1"
HEADER = struct.Struct("<8sQQIIIIIIQQQQ48x")
assert HEADER.size == 128


def serialize(pool: np.ndarray, block_table, seq_len: int, request_id: int, model_id: int) -> bytes:
    """Every layer of one request: header + K tensor + V tensor."""
    L, _, C, _, H, D = pool.shape
    n = int(seq_len)
    layers = [pack_request(pool, l, block_table, n) for l in range(L)]      # each [C][n][H][D]
    k = np.stack([blk[0] for blk in layers]) if L else np.empty((0, n, H, D), pool.dtype)
    v = np.stack([blk[1] for blk in layers]) if C == 2 else np.empty(0, pool.dtype)
    kb, vb = k.tobytes(), v.tobytes()
    header = HEADER.pack(MAGIC, request_id, model_id, n, L, H, D, pool.dtype.itemsize, C,
                         len(kb), len(vb), crc64(kb), crc64(vb))
    return header + kb + vb


def parse_header(blob: bytes) -> dict:
    (magic, rid, mid, n, L, H, D, eb, C, kbytes, vbytes, ck, cv) = HEADER.unpack(bytes(blob[:128]))
    return dict(magic=magic, request_id=rid, model_id=mid, seq_len=n, layers=L, kv_heads=H, head_dim=D,
                elem_bytes=eb, planes=C, k_bytes=kbytes, v_bytes=vbytes, crc_k=ck, crc_v=cv)


def verify(blob: bytes) -> bool:
    """Magic, sizes and both CRC-64s agree with the header."""
    h = parse_header(blob)
    body = bytes(blob[128:])
    return (h["magic"] == MAGIC and len(body) == h["k_bytes"] + h["v_bytes"]
            and crc64(body[:h["k_bytes"]]) == h["crc_k"] and crc64(body[h["k_bytes"]:]) == h["crc_v"])


def unpack_layer(blob: bytes, pool: np.ndarray, layer: int, block_table) -> None:
    """Scatter one layer of a blob into a pool (in place; any page size)."""
    h = parse_header(blob)
    n, L, H, D, C = h["seq_len"], h["layers"], h["kv_heads"], h["head_dim"], h["planes"]
    body = np.frombuffer(bytes(blob[128:]), dtype=pool.dtype)
    per = n * H * D
    planes = [body[c * L * per + layer * per: c * L * per + (layer + 1) * per] for c in range(C)]
    unpack_request(np.concatenate(planes), pool, layer, block_table, n)

"""KVCACHE1 serialization and the device CRC-64 through the C ABI vs the CPU
oracle (serializer and C CRC), bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import oracle.kvcache1 as okv
from gpu_util import say, to_dev, to_host
from oracle.crc64 import crc64
from paper_2607_28633_amd.workloads import (device_dst_prefill, device_src_pool, host_dst_prefill,
                                            host_src_pool, make_workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _device_crc(tk, buf: torch.Tensor, nbytes: int) -> int:
    ws = torch.empty(max(8, tk.topkv_crc64_workspace_bytes(nbytes)) // 8, dtype=torch.int64, device="cuda")
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    tk.topkv_crc64(buf, nbytes, ws, out)
    torch.cuda.synchronize()
    return int(out.cpu().numpy().view(np.uint64)[0])


@pytest.mark.parametrize("n", [0, 1, 9, 15, 16, 17, 4096, 65536, 65536 + 21, 3 * 65536 + 999,
                               (10 << 20) + 3, 300 << 20])
def test_device_crc64(tk, n):
    say(f"[crc64] {n} bytes")
    host = np.random.default_rng(n).integers(0, 256, max(n, 1), dtype=np.uint8)
    if n == 9:
        host[:9] = np.frombuffer(b"123456789", dtype=np.uint8)
    dev = torch.from_numpy(host).cuda()
    got = _device_crc(tk, dev, n)
    assert got == crc64(host[:n]), f"{n} bytes: {got:#x} != {crc64(host[:n]):#x}"
    if n == 9:
        assert got == 0x995DC9BBDF1939FA


def _blob_run(tk, wl, src, dst, r, rid=0x1234, mid=0x77, whole=False):
    """Serialize request r from src, verify, unpack into dst; returns the blob.
    whole: every layer in one call (topkv_kvcache1_pack_layers / unpack_layers)."""
    n = int(wl.seq_lens[r])
    geo = tk.pool_from_tensor(src)
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    blob = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
    ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
    bt = to_dev(wl.block_tables[r])
    if whole:
        tk.topkv_kvcache1_pack_layers(src, 0, wl.num_layers, bt, n, blob)
    else:
        for layer in range(wl.num_layers):
            tk.topkv_kvcache1_pack_layer(src, layer, bt, n, blob)
    tk.topkv_kvcache1_seal(geo, n, rid, mid, blob, ws)
    res = torch.full((4,), 99, dtype=torch.int32, device="cuda")
    tk.topkv_kvcache1_verify(geo, n, rid, mid, blob, ws, res)
    bt2 = to_dev(wl.dst_block_tables[r])
    if whole:
        tk.topkv_kvcache1_unpack_layers(blob, dst, 0, wl.num_layers, bt2, n)
    else:
        for layer in range(wl.num_layers):
            tk.topkv_kvcache1_unpack_layer(blob, dst, layer, bt2, n)
    torch.cuda.synchronize()
    assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0]
    return blob, ws


@pytest.mark.parametrize("case", ["tiny", "mla", "reblock"])
def test_kvcache1_matches_oracle(tk, case):
    if case == "tiny":
        wl = make_workload("tiny", dst_page_size=48)
    elif case == "mla":
        wl = make_workload("deepseek-v3-mla", num_layers=3, seq_lens=[700, 1, 64, 129])
    else:
        wl = make_workload("reblock-70b", num_layers=2, phys_layers=2, seq_lens=[300, 17, 4096])
    say(f"[kvcache1] {case}: {wl.describe()}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    want_dst = dst_h.copy()
    for r in range(wl.num_reqs):
        n = int(wl.seq_lens[r])
        blob, _ = _blob_run(tk, wl, src, dst, r, rid=r + 1, mid=len(case))
        want = okv.serialize(src_h, wl.block_tables[r], n, r + 1, len(case))
        assert blob.cpu().numpy().tobytes() == want, f"{case} request {r}: blob differs from the oracle"
        for layer in range(wl.num_layers):
            okv.unpack_layer(want, want_dst, layer, wl.dst_block_tables[r])
    assert np.array_equal(to_host(dst), want_dst), f"{case}: unpacked pool differs"


def test_kvcache1_detects_corruption(tk):
    wl = make_workload("tiny", seed=2)
    src, dst = to_dev(host_src_pool(wl)), to_dev(host_dst_prefill(wl))
    geo = tk.pool_from_tensor(src)
    n = int(wl.seq_lens[0])
    blob, ws = _blob_run(tk, wl, src, dst, 0, rid=5, mid=6)
    res = torch.zeros(4, dtype=torch.int32, device="cuda")
    k_bytes = wl.num_layers * n * wl.num_heads * wl.head_dim * 2
    for pos, want in ((128 + 7, [tk.TOPKV_ERR_CHECKSUM, 0, 1, 0]),            # a K byte
                      (128 + k_bytes + 3, [tk.TOPKV_ERR_CHECKSUM, 0, 0, 1]),  # a V byte
                      (24, [tk.TOPKV_ERR_CHECKSUM, 1 << 3, 0, 0])):           # seq_len field
        bad = blob.clone()
        bad[pos] ^= 0x40
        tk.topkv_kvcache1_verify(geo, n, 5, 6, bad, ws, res)
        torch.cuda.synchronize()
        assert res.cpu().tolist() == want, f"corruption at byte {pos}"
    tk.topkv_kvcache1_verify(geo, n, 5, 7, blob, ws, res)      # wrong model id expected
    torch.cuda.synchronize()
    assert res.cpu().tolist() == [tk.TOPKV_ERR_CHECKSUM, 1 << 2, 0, 0]
    roomy = torch.zeros(blob.numel() + 64, dtype=torch.uint8, device="cuda")   # misaligned blob
    with pytest.raises(tk.TopkvError) as e:
        tk.topkv_kvcache1_seal(geo, n, 5, 6, roomy.data_ptr() + 8, ws, blob_bytes=blob.numel())
    assert e.value.status == tk.TOPKV_ERR_UNSUPPORTED


def test_kvcache1_fullsize_70b(tk):
    """One 4096-token request of the 80-layer 70B pool: 1.34 GB blob (Eq. 1)."""
    wl = make_workload("llama3-70b-4k")
    say(f"[kvcache1] full size: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    n = int(wl.seq_lens[0])
    blob, ws = _blob_run(tk, wl, src, dst, 0, rid=42, mid=70, whole=True)   # all 80 layers in one call
    assert blob.numel() == 128 + 1_342_177_280
    hdr = okv.parse_header(blob[:128].cpu().numpy().tobytes())
    body = blob[128:].cpu().numpy()
    kb = hdr["k_bytes"]
    assert hdr["crc_k"] == crc64(body[:kb]) and hdr["crc_v"] == crc64(body[kb:])
    assert (hdr["seq_len"], hdr["layers"], hdr["kv_heads"], hdr["head_dim"]) == (4096, 80, 8, 128)
    row = 8 * 128 * 2
    for layer in (0, 41, 79):
        want = oracle.pack_request(to_host(src[layer])[None], 0, wl.block_tables[0], n)
        got_k = body[layer * n * row:(layer + 1) * n * row].view(np.uint16)
        got_v = body[kb + layer * n * row:kb + (layer + 1) * n * row].view(np.uint16)
        assert np.array_equal(got_k, want[0].reshape(-1)) and np.array_equal(got_v, want[1].reshape(-1))
        again = oracle.pack_request(to_host(dst[layer])[None], 0, wl.dst_block_tables[0], n)
        assert np.array_equal(again, want), f"layer {layer}: unpacked pool does not hold the request"
    del src, dst, blob
    torch.cuda.empty_cache()


@pytest.mark.parametrize("case", ["tiny", "mla", "reblock"])
def test_kvcache1_layer_ranges(tk, case):
    """Several layers per call (the whole request, or split ranges) give the
    same blob and the same destination pool as one call per layer."""
    if case == "tiny":
        wl = make_workload("tiny", dst_page_size=48)
    elif case == "mla":
        wl = make_workload("deepseek-v3-mla", num_layers=3, seq_lens=[700, 1, 64, 129])
    else:
        wl = make_workload("reblock-70b", num_layers=3, phys_layers=3, seq_lens=[300, 17, 4096])
    say(f"[kvcache1] layer ranges {case}")
    src = to_dev(host_src_pool(wl))
    dst0 = to_dev(host_dst_prefill(wl))
    geo = tk.pool_from_tensor(src)
    L = wl.num_layers
    for r in range(wl.num_reqs):
        n = int(wl.seq_lens[r])
        nbytes = tk.topkv_kvcache1_bytes(geo, n)
        bt, bt2 = to_dev(wl.block_tables[r]), to_dev(wl.dst_block_tables[r])
        ref = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
        for layer in range(L):
            tk.topkv_kvcache1_pack_layer(src, layer, bt, n, ref)
        ref_dst = dst0.clone()
        for layer in range(L):
            tk.topkv_kvcache1_unpack_layer(ref, ref_dst, layer, bt2, n)
        for ranges in ([(0, L)], [(0, 1), (1, L - 1)], [(L - 1, 1), (0, L - 1)], [(0, 0), (0, L)]):
            blob = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
            for first, count in ranges:
                tk.topkv_kvcache1_pack_layers(src, first, count, bt, n, blob)
            got_dst = dst0.clone()
            for first, count in ranges:
                tk.topkv_kvcache1_unpack_layers(ref, got_dst, first, count, bt2, n)
            torch.cuda.synchronize()
            assert torch.equal(blob, ref), f"{case} request {r} ranges {ranges}: blob differs"
            assert torch.equal(got_dst.view(torch.int16), ref_dst.view(torch.int16)), \
                f"{case} request {r} ranges {ranges}: pool differs"
    with pytest.raises(tk.TopkvError):
        tk.topkv_kvcache1_pack_layers(src, 1, L, to_dev(wl.block_tables[0]), int(wl.seq_lens[0]), blob)


# ---------------------------------------------------------------------------
# One-pass whole-request calls: topkv_kvcache1_pack_seal / verify_unpack
# ---------------------------------------------------------------------------

def _fused_case(case):
    if case == "tiny":
        return make_workload("tiny", dst_page_size=48)
    if case == "mla":
        return make_workload("deepseek-v3-mla", num_layers=3, seq_lens=[700, 1, 64, 129])
    if case == "reblock":
        return make_workload("reblock-70b", num_layers=2, phys_layers=2, seq_lens=[300, 17, 4096])
    # 16-byte rows and 7-token pages: many rows and page changes inside every 16-byte piece's sub-chunk
    return make_workload("tiny", num_heads=1, head_dim=8, page_size=7, dst_page_size=5, seq_lens=[333, 0, 2, 70])


@pytest.mark.parametrize("case", ["tiny", "mla", "reblock", "row16-p7"])
def test_kvcache1_pack_seal_verify_unpack(tk, case):
    """The one-pass sender writes the oracle's blob byte for byte (header and
    checksums included); the one-pass receiver reports no mismatch and leaves
    the pool the oracle's unpack gives."""
    wl = _fused_case(case)
    say(f"[kvcache1 one-pass] {case}: {wl.describe()}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    src, dst = to_dev(src_h), to_dev(dst_h)
    geo = tk.pool_from_tensor(src)
    want_dst = dst_h.copy()
    res = torch.full((4,), 99, dtype=torch.int32, device="cuda")
    for r in range(wl.num_reqs):
        n = int(wl.seq_lens[r])
        nbytes = tk.topkv_kvcache1_bytes(geo, n)
        blob = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
        ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
        tk.topkv_kvcache1_pack_seal(src, to_dev(wl.block_tables[r]), n, r + 1, 9, blob, ws)
        torch.cuda.synchronize()
        want = okv.serialize(src_h, wl.block_tables[r], n, r + 1, 9)
        assert blob.cpu().numpy().tobytes() == want, f"{case} request {r}: blob differs from the oracle"
        tk.topkv_kvcache1_verify_unpack(blob, dst, to_dev(wl.dst_block_tables[r]), n, r + 1, 9, ws, res)
        torch.cuda.synchronize()
        assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0], f"{case} request {r}"
        for layer in range(wl.num_layers):
            okv.unpack_layer(want, want_dst, layer, wl.dst_block_tables[r])
    assert np.array_equal(to_host(dst), want_dst), f"{case}: unpacked pool differs"


def test_kvcache1_one_pass_hostile_and_corrupt(tk):
    """Table entries outside the pool: the one-pass sender leaves those rows'
    blob bytes as they were and checksums them, exactly like the two calls it
    replaces; the receiver skips them like topkv_kvcache1_unpack_layers.
    Corrupted K or V bytes are reported (and the pool is still written)."""
    wl = make_workload("tiny", dst_page_size=16)
    say("[kvcache1 one-pass] hostile tables, corruption")
    src, dst0 = to_dev(host_src_pool(wl)), to_dev(host_dst_prefill(wl))
    geo = tk.pool_from_tensor(src)
    n = int(wl.seq_lens[0])                                  # 64 tokens, 4 pages
    bt = wl.block_tables[0].copy()
    bt[1], bt[3] = wl.num_pages, -2
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
    two = torch.full((nbytes,), 0x5C, dtype=torch.uint8, device="cuda")
    tk.topkv_kvcache1_pack_layers(src, 0, wl.num_layers, to_dev(bt), n, two)
    tk.topkv_kvcache1_seal(geo, n, 3, 4, two, ws)
    one = torch.full((nbytes,), 0x5C, dtype=torch.uint8, device="cuda")
    tk.topkv_kvcache1_pack_seal(src, to_dev(bt), n, 3, 4, one, ws)
    torch.cuda.synchronize()
    assert torch.equal(one, two), "one-pass blob differs from pack_layers + seal on a hostile table"
    bt2 = wl.dst_block_tables[0].copy()
    bt2[2] = 10 ** 6
    want_dst, got_dst = dst0.clone(), dst0.clone()
    tk.topkv_kvcache1_unpack_layers(two, want_dst, 0, wl.num_layers, to_dev(bt2), n)
    res = torch.zeros(4, dtype=torch.int32, device="cuda")
    tk.topkv_kvcache1_verify_unpack(two, got_dst, to_dev(bt2), n, 3, 4, ws, res)
    torch.cuda.synchronize()
    assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0]
    assert torch.equal(got_dst, want_dst), "one-pass receiver differs from unpack_layers on a hostile table"
    k_bytes = wl.num_layers * n * wl.num_heads * wl.head_dim * 2
    for pos, want in ((128 + 5, [tk.TOPKV_ERR_CHECKSUM, 0, 1, 0]), (128 + k_bytes + 11, [tk.TOPKV_ERR_CHECKSUM, 0, 0, 1])):
        bad = two.clone()
        bad[pos] ^= 0x01
        got = dst0.clone()
        tk.topkv_kvcache1_verify_unpack(bad, got, to_dev(bt2), n, 3, 4, ws, res)
        torch.cuda.synchronize()
        assert res.cpu().tolist() == want, f"corruption at byte {pos}"
        assert not torch.equal(got, dst0), "the receiver writes the pool whatever the verdict"


def test_kvcache1_one_pass_fullsize_70b(tk):
    """The 80-layer 70B request (1.34 GB blob): the one-pass sender's blob and
    the one-pass receiver's pool equal those of the two-step calls."""
    wl = make_workload("llama3-70b-4k")
    say(f"[kvcache1 one-pass] full size: {wl.describe()}")
    src, dst = device_src_pool(wl), device_dst_prefill(wl)
    geo = tk.pool_from_tensor(src)
    n = int(wl.seq_lens[0])
    bt, bt2 = to_dev(wl.block_tables[0]), to_dev(wl.dst_block_tables[0])
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
    one = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    tk.topkv_kvcache1_pack_seal(src, bt, n, 42, 70, one, ws)
    two = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    tk.topkv_kvcache1_pack_layers(src, 0, wl.num_layers, bt, n, two)
    tk.topkv_kvcache1_seal(geo, n, 42, 70, two, ws)
    torch.cuda.synchronize()
    assert torch.equal(one, two), "one-pass blob differs at full size"
    res = torch.zeros(4, dtype=torch.int32, device="cuda")
    tk.topkv_kvcache1_verify_unpack(one, dst, bt2, n, 42, 70, ws, res)
    torch.cuda.synchronize()
    assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0]
    for layer in (0, 37, 79):
        assert np.array_equal(oracle.pack_request(to_host(dst[layer])[None], 0, wl.dst_block_tables[0], n),
                              oracle.pack_request(to_host(src[layer])[None], 0, wl.block_tables[0], n)), layer
    del src, dst, one, two
    torch.cuda.empty_cache()

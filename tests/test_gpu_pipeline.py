"""Pipelined layer-by-layer transfer (Section 5.2) on one GPU: in every
placement (side stream, pack straight into mapped host memory, DMA shipper
with the pack on the prefill stream or on a second stream)
the layers shipped while the synthetic prefill runs arrive bit-exact in
pinned host memory; the staging and host buffers are poisoned before every
run, so a copy that read stale data would fail."""
import types

import numpy as np
import pytest

import oracle
from gpu_util import say, to_host
from paper_2607_28633_amd.workloads import device_src_pool, make_workload

pytestmark = pytest.mark.gpu


def test_pipelined_layers_arrive_intact():
    import bench
    wl = make_workload("llama3-8b")
    src = device_src_pool(wl)          # the same seeded pool the runner builds
    sample = (0, 15, 31)
    want = {l: oracle.pack_layer(to_host(src[l])[None], 0, wl.block_tables, wl.seq_lens) for l in sample}
    del src
    seen = []

    def check(variant, host):
        say(f"  checking {variant}")
        for l in sample:
            got = host[l].numpy().view(np.uint16)
            assert np.array_equal(got, want[l]), f"{variant}: layer {l} shipped over the pipeline differs"
        seen.append(variant)

    args = types.SimpleNamespace(workload="llama3-8b", steps=1, layer_ms=0.2)
    say("[pipeline] llama3-8b, 32 layers, 4 placements")
    out = bench.run_pipeline(args, check=check)
    say(f"  {out['ms']} {out['placements']}")
    assert seen == ["side", "fused", "dma", "dma_side_pack"]
    assert out["ms"]["serial"] >= out["ms"]["compute"]


def test_dma_shipper_copies_in_order():
    """The shipper moves device memory into pinned host memory after each
    producer event, completes tickets in order, and refuses memory it
    cannot address before touching the GPU."""
    import torch

    from paper_2607_28633_amd import topkv
    n = 3 << 20
    dev = torch.empty((6, n // 2), dtype=torch.int16, device="cuda")
    host = torch.zeros((6, n // 2), dtype=torch.int16, pin_memory=True)
    want = torch.randint(-32768, 32767, (6, n // 2), dtype=torch.int16)
    dma = topkv.topkv_dma_create()
    try:
        tickets, events = [], []                   # events stay alive until their copies finish
        for i in range(6):
            dev[i].fill_(-1)                       # poison, then the producer's real write
            dev[i].copy_(want[i].cuda(non_blocking=False))
            events.append(torch.cuda.Event())
            events[-1].record()
            tickets.append(topkv.topkv_dma_submit(dma, events[-1], host[i], dev[i], n))
        tickets.append(topkv.topkv_dma_submit(dma, None, host[0], dev[0], 0))      # ordering point
        assert tickets == list(range(1, 8))
        topkv.topkv_dma_wait(dma, tickets[-1])
        assert torch.equal(host, want)
        small = torch.zeros(2048, dtype=torch.int16, pin_memory=True)
        with pytest.raises(topkv.TopkvError) as e:
            topkv.topkv_dma_submit(dma, None, small, dev[0], n)                     # dst too small
        assert e.value.status == topkv.TOPKV_ERR_BOUNDS
        plain = torch.zeros(n // 2, dtype=torch.int16)                              # not pinned
        with pytest.raises(topkv.TopkvError) as e:
            topkv.topkv_dma_submit(dma, None, plain.data_ptr(), dev[0], n)
        assert e.value.status == topkv.TOPKV_ERR_BOUNDS
    finally:
        topkv.topkv_dma_destroy(dma)


def test_receive_side_ships_into_the_decode_pool():
    """The decode half of the pipeline (Section 5.2): each packed layer arrives
    in pinned host memory, the shipper copies it host -> device on a DMA
    engine, and the layer is unpacked into the decode pool (its own page
    order) as soon as its copy is done, while later layers' copies are still
    in flight.  The device staging buffer is poisoned first; every layer of
    the decode pool must match the oracle's unpack of the oracle's pack, and
    nothing outside the requests' slots may change."""
    import torch

    from paper_2607_28633_amd import topkv
    from paper_2607_28633_amd.workloads import host_dst_prefill, host_src_pool
    from gpu_util import to_dev

    wl = make_workload("llama3-8b", num_layers=4, num_pages=600, dst_num_pages=700, seq_lens=[4096, 1000, 17])
    say(f"[receive] llama3-8b shape, {wl.num_layers} layers, lengths {wl.seq_lens.tolist()}")
    src_h, dst_h = host_src_pool(wl), host_dst_prefill(wl)
    L = wl.num_layers
    wire = [oracle.pack_layer(src_h, l, wl.block_tables, wl.seq_lens) for l in range(L)]   # the sender's bytes
    nbytes = wire[0].size * 2
    host = torch.empty((L, nbytes // 2), dtype=torch.int16, pin_memory=True)
    for l in range(L):
        host[l].copy_(torch.from_numpy(wire[l].view(np.int16)))
    staging = torch.full((L, nbytes // 2), -1, dtype=torch.int16, device="cuda")
    dst = to_dev(dst_h)
    bt2, lens = to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    torch.cuda.synchronize()
    dma = topkv.topkv_dma_create()
    try:
        tickets = [topkv.topkv_dma_submit(dma, None, staging[l], host[l], nbytes) for l in range(L)]
        for l in range(L):
            topkv.topkv_dma_wait(dma, tickets[l])      # layer l is in HBM: unpack it, later copies continue
            topkv.topkv_unpack_layer_batched(staging[l], dst, l, wl.num_reqs, bt2, bt2.shape[1], lens,
                                             src_bytes=nbytes)
        torch.cuda.synchronize()
    finally:
        topkv.topkv_dma_destroy(dma)
    want = dst_h.copy()
    for l in range(L):
        oracle.unpack_layer(wire[l], want, l, wl.dst_block_tables, wl.seq_lens)
    got = to_host(dst)
    for l in range(L):
        assert np.array_equal(got[l], want[l]), \
            f"receive layer {l}: {int((got[l] != want[l]).sum())} elements differ"

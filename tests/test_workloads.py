"""Seeded input generator: determinism, table validity and the shapes each
workload promises.  CPU only."""
import numpy as np
import pytest

from paper_2607_28633_amd.workloads import (WORKLOADS, bf16_bits_from_f32, host_src_pool,
                                            make_workload)


def _pages(n, p):
    return -(-int(n) // int(p))


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_tables_valid_and_deterministic(name):
    a, b = make_workload(name), make_workload(name)
    assert np.array_equal(a.seq_lens, b.seq_lens)
    assert np.array_equal(a.block_tables, b.block_tables)
    assert np.array_equal(a.dst_block_tables, b.dst_block_tables)
    for bt, P, NP in ((a.block_tables, a.page_size, a.num_pages),
                      (a.dst_block_tables, a.dst_page_size, a.dst_num_pages)):
        used = []
        for r, n in enumerate(a.seq_lens):
            k = _pages(n, P)
            assert (bt[r, :k] >= 0).all() and (bt[r, :k] < NP).all()
            assert (bt[r, k:] == -1).all()
            used.extend(bt[r, :k].tolist())
        assert len(used) == len(set(used)), "a physical page is given to two token ranges"
        assert len(used) <= NP


def test_workload_shapes():
    t = make_workload("tiny")
    assert t.seq_lens.tolist() == [64, 48, 33, 17] and t.pool_shape() == (2, 64, 2, 16, 2, 64)
    b8 = make_workload("llama3-70b-batch8")
    assert b8.seq_lens[0] == 4096 and ((b8.seq_lens >= 1024) & (b8.seq_lens <= 8192)).all()
    need = sum(_pages(n, 16) for n in b8.seq_lens)
    assert b8.num_pages == int(np.ceil(1.25 * need))
    mla = make_workload("deepseek-v3-mla")
    assert mla.planes == 1 and mla.head_dim == 576 and mla.page_size == 64 and mla.num_reqs == 32
    assert ((mla.seq_lens >= 512) & (mla.seq_lens <= 16384)).all()
    rb = make_workload("reblock-70b")
    assert rb.page_size == 16 and rb.dst_page_size == 64 and rb.num_reqs == 100
    assert ((rb.seq_lens >= 256) & (rb.seq_lens <= 32768)).all()
    assert rb.phys_layers == 8 and rb.num_layers == 80
    # lognormal median 4096: the sample median sits near it
    assert 2500 < np.median(rb.seq_lens) < 6500
    h = make_workload("llama3-70b-4k")
    assert h.num_layers == 80 and h.seq_lens.tolist() == [4096] and h.num_pages == 4096
    tp8 = make_workload("llama3-70b-tp8")      # one GPU's eighth of the 70B heads
    assert tp8.num_heads * 8 == h.num_heads and tp8.pool_shape()[1:] == (4096, 2, 16, 1, 128)


def test_bf16_rounding_and_values():
    x = np.array([1.0, -2.5, 1.00390625, 1.01171875, 3.0e-39], dtype=np.float32)
    # 1.00390625 = 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 -> up to 1 + 2^-6
    assert bf16_bits_from_f32(x).tolist() == [0x3F80, 0xC020, 0x3F80, 0x3F82, 0x0021]
    pool = host_src_pool(make_workload("tiny"))
    f = (pool.astype(np.uint32) << 16).view(np.float32)
    assert abs(f.mean()) < 0.02 and 0.97 < f.std() < 1.03


def test_hybrid_layer_kinds_and_slots():
    """The hybrid workload: attention on every fourth layer, fixed-state layers
    elsewhere, each kind numbered among itself for its slabs, distinct slots on
    both sides, the state size of the stated shape, deterministic."""
    from paper_2607_28633_amd.workloads import HYBRID_STATE_BYTES, host_state_cache
    wl = make_workload("qwen3.5-397b-hybrid")
    assert wl.num_layers == 60 and sum(wl.layer_state) == 45
    assert [l for l in range(60) if not wl.is_state(l)] == list(range(3, 60, 4))
    assert (wl.planes, wl.num_heads, wl.head_dim) == (2, 2, 256)
    assert HYBRID_STATE_BYTES == 2 * (64 * 128 * 128 + 3 * (2 * 16 * 128 + 64 * 128)) == wl.state_bytes
    assert [wl.kv_slab(l) for l in range(3, 60, 4)] == list(range(15)) and wl.phys_layers == 15
    assert [wl.state_slab(l) for l in range(60) if wl.is_state(l)] == list(range(45))
    for slots, NS in ((wl.state_slots, wl.num_state_slots), (wl.dst_state_slots, wl.dst_num_state_slots)):
        assert slots.dtype == np.int32 and slots.size == wl.num_reqs == 32
        assert len(set(slots.tolist())) == slots.size and slots.min() >= 0 and slots.max() < NS == 40
    again = make_workload("qwen3.5-397b-hybrid")
    assert np.array_equal(again.state_slots, wl.state_slots) and np.array_equal(again.seq_lens, wl.seq_lens)
    small = make_workload("qwen3.5-397b-hybrid", num_layers=8, seq_lens=[5, 9], state_bytes=64)
    a, b = host_state_cache(small), host_state_cache(small)
    assert a.shape == (6, 3, 32) and np.array_equal(a, b)
    assert not np.array_equal(host_state_cache(small, dst=True), a)
    with pytest.raises(ValueError):
        make_workload("qwen3.5-397b-hybrid", state_bytes=7)

"""Fixed-state layers (Section 2.2) through the C ABI vs the CPU oracle, bit
for bit: state sizes from 1 byte to several tiles (16-, 8-, 2- and 1-byte
vector paths, ragged last tiles), slot permutations, hostile slots, more
requests than one grid dimension holds, a misaligned packed buffer, and a
reduced hybrid model (attention and state layers) swept layer by layer."""
import numpy as np
import pytest
import torch

import oracle
import oracle.state as so
from gpu_util import say, to_dev, to_host
from paper_2607_28633_amd.workloads import (host_dst_prefill, host_src_pool, host_state_cache, make_workload,
                                            random_words)

pytestmark = pytest.mark.gpu
SENTINEL = 0x3C


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _cache(seed, L, NS, nbytes):
    return random_words(np.random.default_rng(seed), (L, NS, nbytes), 1)


@pytest.mark.parametrize("state_bytes", [1, 2, 16, 1000, 4096, 32768, 40000, 100003, 2170880])
def test_state_pack_unpack(tk, state_bytes):
    """Pack R states from permuted slots, then unpack them into other slots."""
    L, NS, R = 3, 9, 6
    say(f"[state] bytes {state_bytes}")
    rng = np.random.default_rng(state_bytes)
    src_h, dst_h = _cache(1, L, NS, state_bytes), _cache(2, L, NS, state_bytes)
    s1 = rng.permutation(NS)[:R].astype(np.int32)
    s2 = rng.permutation(NS)[:R].astype(np.int32)
    src, dst = to_dev(src_h), to_dev(dst_h)
    n = R * state_bytes
    assert tk.topkv_packed_state_bytes(src, R) == n
    packed = torch.full((n + 64,), SENTINEL, dtype=torch.int8, device="cuda")
    for layer in (0, 2):
        tk.topkv_pack_state_layer(src, layer, R, to_dev(s1), packed, dst_bytes=n)
        tk.topkv_unpack_state_layer(packed, dst, layer, R, to_dev(s2), src_bytes=n)
        torch.cuda.synchronize()
        want = so.pack_state_layer(src_h, layer, s1)
        got = to_host(packed)
        assert np.array_equal(got[:n], want), f"layer {layer}: pack differs"
        assert (got[n:] == SENTINEL).all(), "write past the batch"
        so.unpack_state_layer(want, dst_h, layer, s2)
        assert np.array_equal(to_host(dst), dst_h), f"layer {layer}: unpack differs"


def test_state_words_and_bit_patterns(tk):
    """A bf16-shaped cache (2-byte words, every 16-bit pattern present) from the
    workload generator, all slots, request order reversed."""
    wl = make_workload("qwen3.5-397b-hybrid", num_layers=4, seq_lens=[30, 7, 64], state_bytes=65536 * 2)
    src_h = host_state_cache(wl)
    src_h.reshape(-1)[:65536] = np.arange(65536, dtype=np.uint16)
    slots = np.arange(wl.num_state_slots, dtype=np.int32)[::-1].copy()
    src = to_dev(src_h)
    n = slots.size * wl.state_bytes
    out = torch.empty(n // 2, dtype=torch.int16, device="cuda")
    say("[state] bit patterns")
    tk.topkv_pack_state_layer(src, 0, slots.size, to_dev(slots), out)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(out), so.pack_state_layer(src_h, 0, slots))


def test_state_hostile_slots(tk):
    """Slots outside [0, NS) are skipped: pack leaves that request's bytes
    alone, unpack writes nothing for it; the other requests still move."""
    L, NS, E = 2, 5, 3000
    src_h, dst_h = _cache(3, L, NS, E), _cache(4, L, NS, E)
    bad = np.array([2, -1, 4, NS, 0, 1 << 30, -7], dtype=np.int32)
    ok = (bad >= 0) & (bad < NS)
    src, dst = to_dev(src_h), to_dev(dst_h)
    R = bad.size
    say("[state] hostile slots")
    packed = torch.full((R * E,), SENTINEL, dtype=torch.int8, device="cuda")
    tk.topkv_pack_state_layer(src, 1, R, to_dev(bad), packed)
    torch.cuda.synchronize()
    want = np.full((R, E), SENTINEL, dtype=np.uint8)
    want[ok] = so.pack_state_layer(src_h, 1, bad[ok]).reshape(-1, E)
    assert np.array_equal(to_host(packed), want.reshape(-1))
    tk.topkv_unpack_state_layer(packed, dst, 0, R, to_dev(bad))
    torch.cuda.synchronize()
    so.unpack_state_layer(want[ok].reshape(-1), dst_h, 0, bad[ok])
    assert np.array_equal(to_host(dst), dst_h)


def test_state_many_requests(tk):
    """More requests (70,000) than the grid's second dimension holds: the
    workgroups stride over requests."""
    R, NS, E = 70_000, 70_003, 16
    rng = np.random.default_rng(9)
    src_h = _cache(5, 1, NS, E)
    s = rng.permutation(NS)[:R].astype(np.int32)
    say(f"[state] {R} requests")
    out = torch.zeros(R * E, dtype=torch.int8, device="cuda")
    tk.topkv_pack_state_layer(to_dev(src_h), 0, R, to_dev(s), out)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(out), so.pack_state_layer(src_h, 0, s))


def test_state_misaligned_packed(tk):
    """A packed buffer 2 bytes off 16-byte alignment takes the 2-byte path."""
    L, NS, E, R = 1, 4, 4096, 3
    src_h = _cache(6, L, NS, E)
    s = np.array([3, 1, 2], dtype=np.int32)
    raw = torch.zeros(R * E + 64, dtype=torch.uint8, device="cuda")
    say("[state] misaligned packed buffer")
    tk.topkv_pack_state_layer(to_dev(src_h), 0, R, to_dev(s), raw.data_ptr() + 2, dst_bytes=R * E)
    torch.cuda.synchronize()
    got = raw.cpu().numpy()
    assert np.array_equal(got[2:2 + R * E], so.pack_state_layer(src_h, 0, s))
    assert (got[:2] == 0).all() and (got[2 + R * E:] == 0).all()


def test_hybrid_model_sweep(tk):
    """A reduced hybrid model (8 layers: attention every fourth, state
    otherwise; 4 requests; 40 KiB states): pack every layer with the call its
    kind takes, unpack every layer, both against the oracle."""
    wl = make_workload("qwen3.5-397b-hybrid", num_layers=8, seq_lens=[100, 1, 37, 64], state_bytes=40960)
    say(f"[state] hybrid sweep {wl.describe()}")
    kv_src_h, kv_dst_h = host_src_pool(wl), host_dst_prefill(wl)
    st_src_h, st_dst_h = host_state_cache(wl), host_state_cache(wl, dst=True)
    kv_src, kv_dst = to_dev(kv_src_h), to_dev(kv_dst_h)
    st_src, st_dst = to_dev(st_src_h), to_dev(st_dst_h)
    bt, bt2, lens = to_dev(wl.block_tables), to_dev(wl.dst_block_tables), to_dev(wl.seq_lens)
    s1, s2 = to_dev(wl.state_slots), to_dev(wl.dst_state_slots)
    R = wl.num_reqs
    kv_bytes = tk.topkv_packed_layer_bytes(kv_src, wl.seq_lens)
    st_bytes = tk.topkv_packed_state_bytes(st_src, R)
    bufs = [torch.empty(max(kv_bytes, st_bytes) // 2, dtype=torch.int16, device="cuda") for _ in range(wl.num_layers)]
    for l in range(wl.num_layers):
        if wl.is_state(l):
            tk.topkv_pack_state_layer(st_src, wl.state_slab(l), R, s1, bufs[l], dst_bytes=st_bytes)
        else:
            tk.topkv_pack_layer_batched(kv_src, wl.kv_slab(l), R, bt, bt.shape[1], lens, bufs[l], dst_bytes=kv_bytes)
    for l in range(wl.num_layers):
        if wl.is_state(l):
            tk.topkv_unpack_state_layer(bufs[l], st_dst, wl.state_slab(l), R, s2, src_bytes=st_bytes)
        else:
            tk.topkv_unpack_layer_batched(bufs[l], kv_dst, wl.kv_slab(l), R, bt2, bt2.shape[1], lens,
                                          src_bytes=kv_bytes)
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        if wl.is_state(l):
            want = so.pack_state_layer(st_src_h, wl.state_slab(l), wl.state_slots)
            so.unpack_state_layer(want, st_dst_h, wl.state_slab(l), wl.dst_state_slots)
            n = st_bytes // 2
        else:
            want = oracle.pack_layer(kv_src_h, wl.kv_slab(l), wl.block_tables, wl.seq_lens)
            oracle.unpack_layer(want, kv_dst_h, wl.kv_slab(l), wl.dst_block_tables, wl.seq_lens)
            n = kv_bytes // 2
        assert np.array_equal(to_host(bufs[l])[:n], want), f"layer {l} pack differs"
    assert np.array_equal(to_host(kv_dst), kv_dst_h), "attention pools differ after the sweep"
    assert np.array_equal(to_host(st_dst), st_dst_h), "state caches differ after the sweep"


def test_check_state_slots(tk):
    """The checked path counts slots outside the cache and, when asked,
    slots named twice; a clean batch reports TOPKV_OK."""
    L, NS, E = 2, 40, 64
    cache = to_dev(_cache(7, L, NS, E))
    res = torch.full((4,), -9, dtype=torch.int32, device="cuda")
    ws = torch.empty(tk.topkv_check_state_workspace_bytes(cache) // 4, dtype=torch.int32, device="cuda")
    cases = [
        (np.arange(NS, dtype=np.int32)[::-1].copy(), True, [0, 0, 0]),
        (np.array([3, -1, 3, NS, 39, 3, 1 << 30, 0], dtype=np.int32), True, [3, 2, 0]),
        (np.array([3, -1, 3, NS, 39, 3, 1 << 30, 0], dtype=np.int32), False, [3, 0, 0]),
        (np.array([5, 5], dtype=np.int32), True, [0, 1, 0]),
        (np.zeros(0, dtype=np.int32), True, [0, 0, 0]),
    ]
    for slots, dup, want in cases:
        say(f"[state] check slots {slots.tolist()[:8]} duplicates={dup}")
        ws.fill_(-1)                      # the call must clear its own bitmap
        tk.topkv_check_state_slots(cache, slots.size, to_dev(slots) if slots.size else None, res,
                                   check_duplicates=dup, workspace=ws if dup else None)
        torch.cuda.synchronize()
        got = res.cpu().tolist()
        status = tk.TOPKV_OK if not any(want) else tk.TOPKV_ERR_BOUNDS
        assert got == [status] + want, f"{slots.tolist()} dup={dup}: {got}"

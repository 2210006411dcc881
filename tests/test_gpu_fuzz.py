"""Seeded random geometries through the C ABI vs the CPU oracle, bit for bit:
planes 1-2, 1-9 heads, head_dim 1-40, 1/2/4/8-byte words, page sizes 1-40 on
either side, up to 6 requests with empty and one-token ones, random windows
and head slices, tensor-parallel shards of a packed side, and every pair of
views (packed, slot-major, head-major).
Each case is small; together they cover piece widths 1-16 bytes, ragged
tiles and both grid modes.  A third set sends random KVCACHE1 geometries
through the one-pass sender and receiver."""
import random

import numpy as np
import pytest
import torch

import oracle
import oracle.reshard as rs
from gpu_util import say, to_dev, to_host

pytestmark = pytest.mark.gpu

WORDS = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}
N_CASES = 80


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _pages(n, p):
    return -(-int(n) // int(p))


def _case(seed):
    rng = random.Random(seed)
    c = dict(C=rng.choice([1, 2]), H=rng.randint(1, 9), D=rng.randint(1, 40), eb=rng.choice([1, 2, 4, 8]),
             P=rng.randint(1, 40), P2=rng.randint(1, 40), L=rng.randint(1, 3))
    R = rng.randint(1, 6)
    c["lens"] = np.array([rng.choice([0, 1, rng.randint(1, 90)]) for _ in range(R)], dtype=np.int32)
    for side, P in (("1", c["P"]), ("2", c["P2"])):
        need = [_pages(n, P) for n in c["lens"]]
        NP = sum(need) + rng.randint(1, 5)
        stride = max([1] + need) + rng.randint(0, 2)
        perm = list(range(NP))
        rng.shuffle(perm)
        bt = np.full((R, stride), -1, dtype=np.int32)
        cur = 0
        for r, k in enumerate(need):
            bt[r, :k] = perm[cur:cur + k]
            cur += k
        c["NP" + side], c["bt" + side] = NP, bt
    c["hc"] = rng.randint(1, c["H"])
    c["h0s"], c["h0d"] = rng.randint(0, c["H"] - c["hc"]), rng.randint(0, c["H"] - c["hc"])
    c["W"] = rng.choice([0, 0, rng.randint(1, 50)])
    c["kinds"] = rng.choice([("pool", "packed"), ("packed", "pool"), ("pool", "pool"), ("pool", "hm"),
                             ("hm", "packed"), ("packed", "hm"), ("hm", "hm"), ("hm", "pool")])
    c["layers"] = (rng.randint(0, c["L"] - 1), rng.randint(0, c["L"] - 1))
    c["S"] = rng.choice([d for d in range(1, c["hc"] + 1) if c["hc"] % d == 0]) if "packed" in c["kinds"] else 1
    c["slack"] = rng.choice([0, 0, 3])
    return c


def _pool(c, NP, P, head_major, npr):
    shape = (c["L"], NP, c["C"], c["H"], P, c["D"]) if head_major else (c["L"], NP, c["C"], P, c["H"], c["D"])
    return npr.integers(0, 1 << 63, size=shape, dtype=np.uint64).astype(WORDS[c["eb"]])


@pytest.mark.parametrize("seed", range(N_CASES))
def test_fuzz_pack_unpack(tk, seed):
    """The per-layer pack and unpack (windowed) on a random geometry."""
    c = _case(seed)
    say(f"[fuzz] pack/unpack seed {seed}: C{c['C']} H{c['H']} D{c['D']} u{8 * c['eb']} P{c['P']}->{c['P2']} "
        f"lens {c['lens'].tolist()} W{c['W']}")
    npr = np.random.default_rng(seed)
    src_h, dst_h = _pool(c, c["NP1"], c["P"], False, npr), _pool(c, c["NP2"], c["P2"], False, npr)
    src, dst = to_dev(src_h), to_dev(dst_h)
    bt, bt2, lens = to_dev(c["bt1"]), to_dev(c["bt2"]), to_dev(c["lens"])
    R, (ls, ld) = len(c["lens"]), c["layers"]
    n = oracle.packed_layer_elems(c["C"], c["H"], c["D"], c["lens"], c["W"])
    packed = torch.full((n + 16,), -3, dtype=src.dtype, device="cuda")
    tk.topkv_pack_layer_window(src, ls, R, bt, bt.shape[1], lens, c["W"], packed, dst_bytes=n * c["eb"])
    tk.topkv_unpack_layer_window(packed, dst, ld, R, bt2, bt2.shape[1], lens, c["W"], src_bytes=n * c["eb"])
    torch.cuda.synchronize()
    want = oracle.pack_layer(src_h, ls, c["bt1"], c["lens"], window=c["W"])
    got = to_host(packed)
    assert np.array_equal(got[:n], want), f"seed {seed}: pack differs"
    assert torch.equal(packed[n:], torch.full_like(packed[n:], -3)), f"seed {seed}: write past the batch"
    oracle.unpack_layer(want, dst_h, ld, c["bt2"], c["lens"], window=c["W"])
    assert np.array_equal(to_host(dst), dst_h), f"seed {seed}: unpack differs"


@pytest.mark.parametrize("seed", range(N_CASES))
def test_fuzz_layout_moves(tk, seed):
    """A random pair of views with a random head slice and window."""
    c = _case(1000 + seed)
    sk, dk = c["kinds"]
    say(f"[fuzz] move seed {seed}: {sk}->{dk} C{c['C']} H{c['H']} D{c['D']} u{8 * c['eb']} P{c['P']}->{c['P2']} "
        f"heads {c['h0s']}/{c['h0d']}+{c['hc']} shards {c['S']} lens {c['lens'].tolist()} W{c['W']}")
    npr = np.random.default_rng(1000 + seed)
    S = c["S"]
    cap = rs.packed_heads_elems(c["C"], c["hc"] // S, c["D"], c["lens"], c["W"]) + c["slack"]
    n = S * cap
    if sk == "packed":
        s_h = npr.integers(0, 1 << 63, size=n, dtype=np.uint64).astype(WORDS[c["eb"]])
    else:
        s_h = _pool(c, c["NP1"], c["P"], sk == "hm", npr)
    d_h = np.zeros(n, WORDS[c["eb"]]) if dk == "packed" else _pool(c, c["NP2"], c["P2"], dk == "hm", npr)
    lay = {"packed": rs.PACKED, "pool": rs.POOL, "hm": rs.POOL_HEAD_MAJOR}
    (ls, ld) = c["layers"]
    want = rs.move_layer(rs.View(lay[sk], s_h, ls, c["bt1"], c["h0s"] if sk != "packed" else 0, S, cap),
                         rs.View(lay[dk], d_h.copy(), ld, c["bt2"], c["h0d"] if dk != "packed" else 0, S, cap),
                         c["lens"], c["hc"], c["W"])
    s_d, d_d = to_dev(s_h), to_dev(d_h)
    bt, bt2, lens = to_dev(c["bt1"]), to_dev(c["bt2"]), to_dev(c["lens"])
    pk = dict(nbytes=cap * c["eb"], shards=S)
    sv = tk.packed_view(s_d, **pk) if sk == "packed" else tk.pool_view(s_d, ls, bt, bt.shape[1], c["h0s"], sk == "hm")
    dv = tk.packed_view(d_d, **pk) if dk == "packed" else tk.pool_view(d_d, ld, bt2, bt2.shape[1], c["h0d"], dk == "hm")
    tk.topkv_move_layer(sv, dv, len(c["lens"]), lens, c["hc"], c["W"])
    torch.cuda.synchronize()
    assert np.array_equal(to_host(d_d), want), f"seed {seed}: {sk} -> {dk} differs"


def _kv1_case(seed):
    rng = random.Random(seed)
    eb = rng.choice([1, 2, 4, 8])
    c = dict(C=rng.choice([1, 2]), H=rng.randint(1, 4), eb=eb, P=rng.randint(1, 40), P2=rng.randint(1, 40),
             L=rng.randint(1, 4))
    c["D"] = (16 // eb) * rng.randint(1, 6)                  # rows are whole 16-byte pieces (KVCACHE1 layout)
    c["n"] = rng.choice([0, 1, rng.randint(1, 700), rng.randint(1, 700)])
    for side, P in (("1", c["P"]), ("2", c["P2"])):
        k = _pages(c["n"], P)
        NP = k + rng.randint(1, 6)
        perm = list(range(NP))
        rng.shuffle(perm)
        c["NP" + side], c["bt" + side] = NP, np.array(perm[:max(k, 1)], dtype=np.int32)
    return c


@pytest.mark.parametrize("seed", range(40))
def test_fuzz_kvcache1_one_pass(tk, seed):
    """The one-pass KVCACHE1 sender and receiver on a random geometry: the blob
    is the oracle's serialization byte for byte and the receiver rebuilds the
    oracle's pool (every layer, the destination at another page size)."""
    import oracle.kvcache1 as okv
    c = _kv1_case(5000 + seed)
    say(f"[fuzz] kvcache1 seed {seed}: L{c['L']} C{c['C']} H{c['H']} D{c['D']} u{8 * c['eb']} "
        f"P{c['P']}->{c['P2']} n {c['n']}")
    npr = np.random.default_rng(5000 + seed)
    src_h, dst_h = _pool(c, c["NP1"], c["P"], False, npr), _pool(c, c["NP2"], c["P2"], False, npr)
    src, dst = to_dev(src_h), to_dev(dst_h)
    geo = tk.pool_from_tensor(src)
    n = c["n"]
    nbytes = tk.topkv_kvcache1_bytes(geo, n)
    blob = torch.full((nbytes,), 0x3B, dtype=torch.uint8, device="cuda")
    ws = torch.empty(tk.topkv_kvcache1_workspace_bytes(geo, n) // 8, dtype=torch.int64, device="cuda")
    res = torch.full((4,), 9, dtype=torch.int32, device="cuda")
    tk.topkv_kvcache1_pack_seal(src, to_dev(c["bt1"]), n, seed, 77, blob, ws)
    tk.topkv_kvcache1_verify_unpack(blob, dst, to_dev(c["bt2"]), n, seed, 77, ws, res)
    torch.cuda.synchronize()
    want = okv.serialize(src_h, c["bt1"], n, seed, 77)
    assert blob.cpu().numpy().tobytes() == want, f"seed {seed}: blob differs"
    assert res.cpu().tolist() == [tk.TOPKV_OK, 0, 0, 0], f"seed {seed}"
    for layer in range(c["L"]):
        okv.unpack_layer(want, dst_h, layer, c["bt2"])
    assert np.array_equal(to_host(dst), dst_h), f"seed {seed}: unpacked pool differs"

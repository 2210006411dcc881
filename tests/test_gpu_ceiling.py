"""The measurement kernels the bench reads the product against
(libtopkv_ceiling.so) do what they are reported as: the copies move exactly
the bytes named (ragged sizes too, nothing past them), the engine-schedule
copy moves every layer between its own strided blocks, the scattered-tile
copy moves each 32 KiB tile between the offsets it is given and skips tiles
whose offsets are misaligned or out of range, the read-only pass writes each
32 KiB tile's XOR, and the timeline's stamps are ordered."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

TILE = 32768


@pytest.fixture(scope="module")
def cl():
    from paper_2607_28633_amd import ceiling
    return ceiling


def _bytes(n, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randint(0, 256, (n,), dtype=torch.uint8, device="cuda", generator=g)


@pytest.mark.parametrize("n", [16, 4096, TILE, TILE + 16, 5 * TILE - 48, (16 << 20) + 272])
def test_copy_moves_exactly_n_bytes(cl, n):
    src = _bytes(n + 64, 1)
    dst = torch.full((n + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    cl.topkv_ceiling_copy(src, dst, n)
    torch.cuda.synchronize()
    assert torch.equal(dst[:n], src[:n])
    assert (dst[n:] == 0xA5).all()


def test_copy_layers_engine_schedule(cl):
    layers, lb, ss, ds = 7, 3 * TILE + 80, 4 * TILE, 5 * TILE
    src = _bytes(layers * ss, 2)
    dst = torch.full((layers * ds,), 0x3C, dtype=torch.uint8, device="cuda")
    for per_cu in (0, 1):
        dst.fill_(0x3C)
        cl.topkv_ceiling_copy_layers(src, ss, dst, ds, lb, layers, per_cu)
        torch.cuda.synchronize()
        for z in range(layers):
            assert torch.equal(dst[z * ds:z * ds + lb], src[z * ss:z * ss + lb]), (per_cu, z)
            assert (dst[z * ds + lb:(z + 1) * ds] == 0x3C).all(), (per_cu, z)


def test_copy_tiles_follows_the_offsets(cl):
    n_src, n_dst, tiles = 40 * TILE + 48, 30 * TILE + 16, 24
    src = _bytes(n_src, 4)
    dst = torch.full((n_dst,), 0x5A, dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(9)
    so = rng.integers(0, (n_src - TILE) // 16, size=tiles) * 16
    do = rng.permutation(np.arange(0, (n_dst - TILE) // TILE + 1) * TILE)[:tiles - 4]   # non-overlapping
    # misaligned, past the end (fits a 16-byte tile only, after every slot), negative, past
    do = np.concatenate([do, [8, n_dst - 16, -TILE, n_dst]])
    so[-1] = n_src - TILE + 32                                            # source past the end
    for lens in (None, rng.integers(1, TILE // 16 + 1, size=tiles) * 16):
        if lens is not None:
            lens[3], lens[5], lens[7] = 0, TILE + 16, 24                  # too short, too long, misaligned
        dst.fill_(0x5A)
        so_t, do_t = torch.tensor(so, device="cuda"), torch.tensor(do, device="cuda")
        ln_t = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
        cl.topkv_ceiling_copy_tiles(src, n_src, so_t, dst, n_dst, do_t, ln_t, tiles)
        torch.cuda.synchronize()
        want = np.full(n_dst, 0x5A, dtype=np.uint8)
        h = src.cpu().numpy()
        hit = np.zeros(n_dst, dtype=bool)
        for k in range(tiles):
            s0, d0, n = int(so[k]), int(do[k]), TILE if lens is None else int(lens[k])
            if (s0 | d0 | n) % 16 or n < 16 or n > TILE or s0 < 0 or d0 < 0 or s0 > n_src - n or d0 > n_dst - n:
                continue
            assert not hit[d0:d0 + n].any(), "copied tiles overlap: the result would depend on workgroup order"
            hit[d0:d0 + n] = True
            want[d0:d0 + n] = h[s0:s0 + n]
        assert np.array_equal(dst.cpu().numpy(), want), lens is None


@pytest.mark.parametrize("n", [16, TILE, 3 * TILE + 4096 + 16, (8 << 20) + 160])
def test_read_writes_each_tiles_xor(cl, n):
    src = _bytes(n, 3)
    tiles = -(-n // TILE)
    sink = torch.zeros(tiles + 1, dtype=torch.int32, device="cuda")
    cl.topkv_ceiling_read(src, n, sink)
    torch.cuda.synchronize()
    words = src.cpu().numpy().view(np.uint32)
    want = [int(np.bitwise_xor.reduce(words[b * TILE // 4:min(n, (b + 1) * TILE) // 4])) for b in range(tiles)]
    got = (sink[:tiles].cpu().numpy().view(np.uint32)).tolist()
    assert got == want
    assert int(sink[tiles]) == 0                    # nothing past the last tile's word


def test_timeline_copies_and_stamps_in_order(cl):
    n = 16 << 20
    src, dst = _bytes(n, 4), torch.zeros(n, dtype=torch.uint8, device="cuda")
    tiles = n // TILE
    stamps = torch.zeros(3 * tiles, dtype=torch.int64, device="cuda")
    cl.topkv_ceiling_copy_timeline(src, dst, n, stamps)
    cl.topkv_ceiling_empty()
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    t = stamps.view(tiles, 3).cpu().numpy()
    assert (t[:, 0] > 0).all() and (t[:, 0] <= t[:, 1]).all() and (t[:, 1] <= t[:, 2]).all()
    khz = cl.topkv_ceiling_wall_clock_khz()
    assert khz > 0 and (t[:, 2].max() - t[:, 0].min()) * 1e3 / khz < 1e6     # under a second, in us

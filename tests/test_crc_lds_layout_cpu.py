"""CPU model of the CRC-64 span kernel's LDS tables (csrc/kvcache1.hip): the
slicing-by-4 byte tables in 8 replicas and the sub-chunk advance's 8 byte
tables in 4 replicas, the fill that writes them, and every lane's lookups
(crc_word4's permute-built addresses, sub_advance's register rotation).
Checked: the fill writes every slot once with the right entry; each lane's
fold of a 64-byte piece equals the raw CRC register of those bytes (from the
oracle's CRC-64/XZ); each lane's advance equals the GF(2) product by
x^(8 * 64 Ki) mod P; and in every lookup instruction the 32 lanes an LDS
cycle serves sit in 32 different bank pairs (no bank conflict whatever the
data).  The model restates the kernel's layout constants and lane mapping,
so a change to them can be checked here before it reaches a GPU."""
import random
import struct

from oracle.crc64 import crc64

POLY = 0xC96C5795D7870F42          # ECMA-182, bit-reversed (bit 63 of a register is x^0)
M64 = (1 << 64) - 1
K_COPIES, K_SUB_COPIES = 8, 4
SUB = 1 << 16                      # bytes per sub-chunk


def mul_x(w):
    return (w >> 1) ^ (POLY if w & 1 else 0)


def mulmod(a, b):
    p = 0
    for _ in range(64):
        if a >> 63:
            p ^= b
        a = (a << 1) & M64
        b = mul_x(b)
    return p


def x8n(n):
    r, x = 1 << 63, 1 << 63
    for _ in range(8):
        x = mul_x(x)
    while n:
        if n & 1:
            r = mulmod(r, x)
        x = mulmod(x, x)
        n >>= 1
    return r


def raw_register(data):
    """The raw register (preset 0, no final complement) of `data`, from the
    oracle's CRC: crc = ~(~0 * x^(8N) + R)."""
    return (~crc64(bytes(data)) & M64) ^ mulmod(x8n(len(data)), M64)


def byte_set(m):
    t = [0] * (8 * 256)
    for k in range(8):
        for b in range(1, 256):
            low = (b & -b).bit_length() - 1
            t[k * 256 + b] = t[k * 256 + (b & (b - 1))] ^ m[8 * k + low]
    return t


def tables():
    p = [1 << 63]
    for _ in range(127):
        p.append(mul_x(p[-1]))
    slicing = byte_set([p[71 + 8 * (j // 8) - j % 8] for j in range(64)])
    m = [0] * 64
    m[63] = x8n(SUB)
    for j in range(63, 0, -1):
        m[j - 1] = mul_x(m[j])
    return slicing, byte_set(m)


def fill(slicing, advance):
    big, sub = bytearray(65536), bytearray(65536)
    for e in range(1024):
        t, b, u, c = e & 3, e >> 2, e & 7, e >> 3
        for i in range(K_COPIES):
            struct.pack_into("<Q", big, b * 256 + t * 64 + ((i + (e >> 2)) & 7) * 8, slicing[t * 256 + b])
        for i in range(K_SUB_COPIES):
            r = (i + (e >> 3)) & 3
            struct.pack_into("<Q", sub, c * 256 + u * 32 + r * 8, advance[u * 256 + c])
            struct.pack_into("<Q", sub, (c + 128) * 256 + u * 32 + r * 8, advance[u * 256 + c + 128])
    return big, sub


def perm(s0, s1, sel):
    out = 0
    for i in range(4):
        s = (sel >> (8 * i)) & 0xFF
        byte = (s1 >> (8 * s)) & 0xFF if s < 4 else (s0 >> (8 * (s - 4))) & 0xFF if s < 8 else 0
        assert s < 8 or s == 0x0C
        out |= byte << (8 * i)
    return out


def lane_constants(lane):
    rep8, grp4 = lane & 7, (lane >> 3) & 3
    L, sel = 0, []
    for k in range(4):
        t = (3 - k + grp4) & 3
        L |= (t * 64 + rep8 * 8) << (8 * k)
        sel.append(0x0C0C0000 | (3 - t) << 8 | (4 + k))
    rep4, grp8 = lane & 3, (lane >> 2) & 7
    la = lb = 0
    for k in range(4):
        la |= ((32 * k + 32 * grp8 + 8 * rep4) & 255) << (8 * k)
        lb |= ((32 * (k + 4) + 32 * grp8 + 8 * rep4) & 255) << (8 * k)
    return L, sel, la, lb, grp8 >= 4, 8 * (grp8 & 3)


def get(buf, off):
    return struct.unpack_from("<Q", buf, off)[0]


def crc_word4(big, lo, hi, w, L, sel, seen):
    x = lo ^ w
    e = []
    for k in range(4):
        a = perm(L, x, sel[k])
        seen[k].append(a)
        e.append(get(big, a))
    return (e[0] ^ e[1] ^ e[2] ^ e[3] ^ hi) & 0xFFFFFFFF, (e[0] ^ e[1] ^ e[2] ^ e[3]) >> 32


def sub_advance(sub, v, la, lb, swap, sh, seen):
    lo, hi = v & 0xFFFFFFFF, v >> 32
    a, b = (hi, lo) if swap else (lo, hi)
    w = [((b << 32 | a) >> sh) & 0xFFFFFFFF, ((a << 32 | b) >> sh) & 0xFFFFFFFF]
    r = 0
    for k in range(8):
        addr = perm(la if k < 4 else lb, w[k >> 2], 0x0C0C0000 | (k & 3) << 8 | (4 + (k & 3)))
        seen[k].append(addr)
        r ^= get(sub, addr)
    return r


def test_fill_writes_every_slot_once():
    slicing, advance = tables()
    big, sub = fill(slicing, advance)
    for b in range(256):
        for t in range(4):
            for r in range(K_COPIES):
                assert get(big, b * 256 + t * 64 + r * 8) == slicing[t * 256 + b]
        for t in range(8):
            for r in range(K_SUB_COPIES):
                assert get(sub, b * 256 + t * 32 + r * 8) == advance[t * 256 + b]


def test_lanes_fold_and_advance_without_bank_conflicts():
    slicing, advance = tables()
    big, sub = fill(slicing, advance)
    rng = random.Random(5)
    A = x8n(SUB)
    for half in (0, 32):                      # the two 32-lane groups of a wave
        fold_seen = [[] for _ in range(4)]
        adv_seen = [[] for _ in range(8)]
        for lane in range(half, half + 32):
            L, sel, la, lb, swap, sh = lane_constants(lane)
            piece = bytes(rng.getrandbits(8) for _ in range(64))
            lo = hi = 0
            for j in range(16):
                lo, hi = crc_word4(big, lo, hi, struct.unpack_from("<I", piece, 4 * j)[0], L, sel, fold_seen)
            assert (hi << 32 | lo) == raw_register(piece), lane
            v = rng.getrandbits(64)
            assert sub_advance(sub, v, la, lb, swap, sh, adv_seen) == mulmod(v, A), lane
        for k in range(4):                    # lookup k of word j, over the 32 lanes
            for j in range(16):
                pairs = {(fold_seen[k][lane * 16 + j] // 8) % 32 for lane in range(32)}
                assert len(pairs) == 32, (half, k, j)
        for k in range(8):
            assert len({(a // 8) % 32 for a in adv_seen[k]}) == 32, (half, k)

"""CPU model of the one-pass KVCACHE1 span kernels' addressing (the kGather /
kScatter source of crc64_span_kernel): every 16-byte piece of a tensor,
visited in the kernel's order (plane, span, sub-chunk, wave, lane, row j; the
planes' tensors share one launch, kMaxSpans / planes spans each), must land
on the pool byte the KVCACHE1 definition gives -- tensor byte o is layer
o // (s * row), token (o // row) % s, byte o % row of that token's row in its
page -- exactly once, inside the pool, with the front padding skipped.  The
model restates the kernel's integer steps (multiply-high division, the floor
quotient and remainder carried from sub-chunk to sub-chunk) so that a change
to them can be checked here before it reaches a GPU."""
import numpy as np

K_SUB_LOG2 = 16
K_SUB = 1 << K_SUB_LOG2
K_MAX_SPANS = 256
K_PIECE = 64
K_LOADS = 4
K_WAVES = 16


def make_div32(d):
    s = 0
    while (1 << s) < d:
        s += 1
    return d, ((((1 << 32) * ((1 << s) - d)) // d) + 1) & 0xFFFFFFFF, s


def div32(n, f):
    _, m, s = f
    assert 0 <= n < (1 << 31)
    return (((n * m) >> 32) + n) >> s


def span_geometry(n, inputs=1):
    max_spans = K_MAX_SPANS // inputs
    head = n - n % 16
    subs = (head + K_SUB - 1) // K_SUB
    span_subs = (subs + max_spans - 1) // max_spans if subs > 0 else 1
    span = span_subs * K_SUB
    return head, span_subs, span, (head + span - 1) // span


def test_div32_exact():
    rng = np.random.default_rng(0)
    divisors = list(range(1, 1100)) + [2048, 1152, 73728, 4095, 65537] + rng.integers(2, 1 << 30, 200).tolist()
    for d in divisors:
        f = make_div32(int(d))
        ns = {0, 1, d - 1, d, d + 1, 2 * d - 1, (1 << 31) - 1, (1 << 31) - 1 - ((1 << 31) - 1) % d}
        ns |= set(rng.integers(0, 1 << 31, 64).tolist())
        for n in ns:
            if 0 <= n < (1 << 31):
                assert div32(int(n), f) == n // d, (n, d)


def _check(L, NP, C, P, H, D, eb, s, seed=0):
    rng = np.random.default_rng(seed)
    row = H * D * eb
    page_bytes = C * P * row
    layer_bytes = NP * page_bytes
    table = rng.permutation(NP)[:-(-s // P)]
    tensor = L * s * row
    head, span_subs, span, spans = span_geometry(tensor, C)
    assert spans * C <= K_MAX_SPANS
    pad = spans * span - head
    d_row, d_seq, d_page = make_div32(row), make_div32(s), make_div32(P)
    step_q, step_r = K_SUB // row, K_SUB % row
    local = (np.arange(K_WAVES)[:, None] * 64 * K_PIECE + 16 * np.arange(64)[None, :]).reshape(-1)
    for c in range(C):
        seen = np.zeros(tensor // 16, np.int64)
        for blk in range(spans):
            span0 = blk * span_subs * K_SUB - pad
            q = span0 // row                                     # floor quotient (span0 < 0 in the padding)
            r0, in0 = q, span0 - q * row
            assert 0 <= in0 < row
            # every piece's table entry is loaded, a padding piece's as row 0's, and the receiver also
            # looks up the sub-chunk after a span's last one (past the tensor on the last span):
            # every such index lies within the request's table
            for sub in range(span_subs + 1):
                for j in range(K_LOADS):
                    for loc in local.tolist():
                        off = span0 + (sub << K_SUB_LOG2) + loc + 1024 * j
                        x = in0 + loc + 1024 * j
                        qq = div32(x, d_row)
                        r = r0 + qq
                        rr = max(r, 0)
                        i_any = div32(rr - div32(rr, d_seq) * s, d_page)
                        assert 0 <= i_any < len(table)
                        if sub == span_subs:
                            continue
                        if r < 0:
                            assert off < 0
                            continue
                        assert 0 <= off < head
                        inrow = x - qq * row
                        l = div32(r, d_seq)
                        t = r - l * s
                        i = div32(t, d_page)
                        assert (l, t, inrow) == (off // (s * row), (off // row) % s, off % row)
                        po = l * layer_bytes + int(table[i]) * page_bytes + c * P * row + (t - i * P) * row + inrow
                        assert 0 <= po and po + 16 <= L * layer_bytes
                        seen[off // 16] += 1
                in0 += step_r                                    # the next sub-chunk: + K_SUB bytes
                r0 += step_q
                if in0 >= row:
                    in0 -= row
                    r0 += 1
        assert (seen == 1).all()


def test_one_pass_addressing():
    _check(2, 20, 2, 16, 2, 64, 2, 100)          # 256-byte rows, ragged last page, front padding
    _check(3, 40, 2, 16, 1, 8, 2, 33)            # 16-byte rows: many rows per sub-chunk
    _check(8, 40, 1, 64, 1, 576, 2, 2000)        # MLA rows (1152 B, not dividing 64 KiB), 18 MB: carried remainder
    _check(4, 70, 2, 7, 3, 40, 2, 150)           # 240-byte rows, 7-token pages
    _check(2, 30, 2, 16, 8, 128, 2, 300)         # 2 KiB rows

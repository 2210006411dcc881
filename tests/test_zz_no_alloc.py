"""topkv_crc64_noalloc, the CRC-64 entry point that allocates nothing (its
workspace is the library's per-GPU file-scope array): called through the C
ABI twice in a row, the second time on a shorter input, each result equals
topkv_crc64's (caller-allocated workspace) on the same bytes, and the CRC of
the oracle's C byte loop.  A length the array could not hold does not exist
(the workspace does not grow with the length), so the refusal path is the
argument checks, tested on the CPU."""
import numpy as np
import pytest
import torch

from gpu_util import say
from oracle.crc64 import crc64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _with_workspace(tk, buf, n):
    ws = torch.empty(max(8, tk.topkv_crc64_workspace_bytes(n)) // 8, dtype=torch.int64, device="cuda")
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    tk.topkv_crc64(buf, n, ws, out)
    torch.cuda.synchronize()
    return int(out.item()) & 0xFFFFFFFFFFFFFFFF


def test_noalloc_matches_workspace_call(tk):
    g = torch.Generator(device="cuda")
    g.manual_seed(20261202)
    big = torch.randint(0, 256, ((64 << 20) + 4096,), dtype=torch.uint8, device="cuda", generator=g)
    host = big.cpu().numpy()
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    # the longer input first, then a shorter one: the second call must not see the first one's state
    for n in ((64 << 20) + 4093, (1 << 20) + 5, 100, 0):
        say(f"[noalloc] crc64 of {n} bytes")
        out.fill_(0x1234)
        tk.topkv_crc64_noalloc(big, n, out)
        torch.cuda.synchronize()
        got = int(out.item()) & 0xFFFFFFFFFFFFFFFF
        want = _with_workspace(tk, big, n)
        assert got == want, f"{n} bytes: {got:#x} != {want:#x} (workspace call)"
        assert got == crc64(host[:n]), f"{n} bytes: {got:#x} != oracle {crc64(host[:n]):#x}"


def test_noalloc_in_graph_replays(tk):
    """Captured into a HIP graph (the calls it is for): every replay, with
    eager work between replays, equals the workspace call."""
    buf = torch.arange(3 << 20, dtype=torch.int32, device="cuda").view(torch.uint8)
    n = buf.numel() - 7
    want = _with_workspace(tk, buf, n)
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    tk.topkv_crc64_noalloc(buf, 16, out)        # set-up call outside capture: looks the array's address up
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tk.topkv_crc64_noalloc(buf, n, out)
    for rep in range(3):
        out.fill_(0)
        _with_workspace(tk, buf, 12345)          # other work on the same GPU between replays
        g.replay()
        torch.cuda.synchronize()
        assert int(out.item()) & 0xFFFFFFFFFFFFFFFF == want, f"replay {rep}"

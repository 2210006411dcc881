"""topkv_check_tables on the device: valid tables pass; planted out-of-range
entries, repeated pages and bad lengths are counted exactly."""
import numpy as np
import pytest
import torch

from gpu_util import say
from paper_2607_28633_amd.workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tk():
    from paper_2607_28633_amd import topkv
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return topkv


def _run(tk, pool, bt, lens, dup):
    ws = torch.full((max(1, tk.topkv_check_workspace_bytes(pool) // 4),), -1, dtype=torch.int32, device="cuda")
    res = torch.full((4,), 77, dtype=torch.int32, device="cuda")
    tk.topkv_check_tables(pool, bt.shape[0], torch.from_numpy(bt).cuda(), bt.shape[1],
                          torch.from_numpy(lens).cuda(), dup, ws, res)
    torch.cuda.synchronize()
    return res.cpu().tolist()


@pytest.mark.parametrize("name", ["tiny", "reblock-70b"])
def test_valid_tables_pass(tk, name):
    wl = make_workload(name)
    say(f"[check] valid {name}")
    for bt, P, NP in ((wl.block_tables, wl.page_size, wl.num_pages),
                      (wl.dst_block_tables, wl.dst_page_size, wl.dst_num_pages)):
        pool = tk.make_pool(0x1000, num_pages=NP, num_layers=1, page_size=P, planes=wl.planes,
                            num_heads=wl.num_heads, head_dim=wl.head_dim)
        assert _run(tk, pool, bt, wl.seq_lens, 1) == [tk.TOPKV_OK, 0, 0, 0]
        assert _run(tk, pool, bt, wl.seq_lens, 0) == [tk.TOPKV_OK, 0, 0, 0]


def test_planted_errors_are_counted(tk):
    wl = make_workload("tiny")
    say("[check] planted errors")
    pool = tk.make_pool(0x1000, num_pages=wl.num_pages, num_layers=1, page_size=wl.page_size, planes=2,
                        num_heads=2, head_dim=64)
    bt = wl.block_tables.copy()
    lens = wl.seq_lens.copy()                  # 64/48/33/17 -> 4/3/3/2 pages, stride 4
    bt[0, 1] = wl.num_pages                    # out of range
    bt[1, 0] = -3                              # out of range
    bt[2, 2] = bt[3, 0]                        # a page named twice
    bt[3, 3] = 5000                            # past request 3's last page: never read, not counted
    assert _run(tk, pool, bt, lens, 1) == [tk.TOPKV_ERR_BOUNDS, 2, 1, 0]
    assert _run(tk, pool, bt, lens, 0) == [tk.TOPKV_ERR_BOUNDS, 2, 0, 0]   # pack sources may repeat pages
    lens2 = lens.copy()
    lens2[1] = -1
    lens2[2] = 4 * 16 + 1                      # beyond bt_stride * P
    bt2 = wl.block_tables.copy()
    bt2[2, 3] = sorted(set(range(wl.num_pages)) - set(bt2[bt2 >= 0].tolist()))[0]
    assert _run(tk, pool, bt2, lens2, 1) == [tk.TOPKV_ERR_BOUNDS, 0, 0, 2]

"""bench.py on the CPU: its byte accounting follows Eq. 1 (per launch: the
layer's bytes read and written, plus the table entries and lengths read), and it refuses more than one GPU before touching
one."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_headline_bytes_per_launch():
    import bench
    from paper_2607_28633_amd.workloads import make_workload
    wl = make_workload("llama3-70b-4k")
    # read + write of 2 planes x 4096 tokens x 2 KiB rows, 256 table entries, one length
    assert bench.layer_bytes(wl, 0) == (2 * 16_777_216 + 4 * 256 + 4,) * 2
    assert bench.step_bytes(wl) == (33_555_460, 33_555_460)


def test_windowed_bytes_count_kept_tokens_only():
    import bench
    from paper_2607_28633_amd.workloads import make_workload
    wl = make_workload("gpt-oss-120b")
    row = 8 * 64 * 2
    kept = int(np.minimum(wl.seq_lens, 128).sum())
    pack, _ = bench.layer_bytes(wl, 0)                   # layer 0 is windowed (W = 128)
    assert pack - 4 * wl.num_reqs - 2 * 2 * kept * row == 4 * sum(
        (int(n) - 1) // 16 - max(0, int(n) - 128) // 16 + 1 for n in wl.seq_lens)


def test_table_layouts_keep_the_pages_valid():
    """--tables sorted keeps every request's pages (sorted); consecutive gives
    each request its own run of the pool; runs8 gives each request runs of 8
    consecutive pages; all stay inside the pool, no page shared."""
    import bench
    from paper_2607_28633_amd.workloads import make_workload
    base = make_workload("llama3-70b-batch8")
    for layout in ("sorted", "consecutive", "runs8"):
        wl = make_workload("llama3-70b-batch8")
        bench.table_layout(wl, layout)
        for attr, P, NP in (("block_tables", wl.page_size, wl.num_pages),
                            ("dst_block_tables", wl.dst_page_size, wl.dst_num_pages)):
            tab, ref = getattr(wl, attr), getattr(base, attr)
            seen = []
            for r, n in enumerate(wl.seq_lens):
                k = -(-int(n) // P)
                row = tab[r, :k]
                assert row.min() >= 0 and row.max() < NP
                if layout == "sorted":
                    assert (np.diff(row) > 0).all() and sorted(ref[r, :k].tolist()) == row.tolist()
                elif layout == "runs8":
                    assert (row[::8] % 8 == 0).all()                      # runs start on 8-page slots
                    runs = [row[j:j + 8] for j in range(0, k, 8)]
                    assert all((np.diff(x) == 1).all() for x in runs)
                else:
                    assert (np.diff(row) == 1).all()
                seen += row.tolist()
            assert len(set(seen)) == len(seen)          # no page shared by two requests


def test_scattered_tiles_cover_every_page_run_once():
    """The ceiling's scattered-page copy (bench.scattered_tiles) moves exactly
    the workload's transfer: in each direction the tiles' packed intervals
    tile every layer's packed block once, and each tile's pool interval lies
    inside the page plane its table entry names, over the rows its request
    holds (five configurations; the re-blocking one unpacks into 64-token
    pages)."""
    import types

    import bench
    from paper_2607_28633_amd.workloads import make_workload
    for name in ("tiny", "llama3-70b-4k", "llama3-70b-batch8", "deepseek-v3-mla", "reblock-70b"):
        wl = make_workload(name)
        row = wl.num_heads * wl.head_dim * wl.elem_bytes
        layer_packed = int(wl.seq_lens.sum()) * wl.planes * row
        ring = bench.ring_slots(wl, layer_packed)
        st = types.SimpleNamespace(wl=wl, ring=ring, slice=layer_packed)
        for d, (tables, P, npages) in enumerate(((wl.block_tables, wl.page_size, wl.num_pages),
                                                 (wl.dst_block_tables, wl.dst_page_size, wl.dst_num_pages))):
            pool, packed, lens = bench.scattered_tiles(st, d)
            assert len(pool) == len(packed) == len(lens) and (lens >= 16).all() and (lens <= 32768).all()
            assert not ((pool | packed | lens.astype(np.int64)) % 16).any()
            per = len(pool) // wl.num_layers
            plane = P * row
            slab_bytes = npages * wl.planes * plane
            for l in sorted({0, wl.num_layers // 2, wl.num_layers - 1}):
                sl = slice(l * per, (l + 1) * per)
                o, n = packed[sl] - (l % ring) * layer_packed, lens[sl].astype(np.int64)
                k = np.argsort(o)
                assert o[k][0] == 0 and (o[k][1:] == (o[k] + n[k])[:-1]).all() and int((o + n).max()) == layer_packed
                # pool side: page plane of the tile, offset inside it, and the rows the request owns there
                q = pool[sl] - wl.kv_slab(l) * slab_bytes
                page, c, within = q // (wl.planes * plane), (q // plane) % wl.planes, q % plane
                tok = np.concatenate([[0], np.cumsum(wl.seq_lens.astype(np.int64))])
                r = np.searchsorted(tok, o // (wl.planes * row), side="right") - 1   # request of each tile
                first = (o - tok[r] * wl.planes * row - c * wl.seq_lens[r].astype(np.int64) * row) // row
                i = first // P                                                 # table entry of the tile
                assert (tables[r, i] == page).all() and (within == first % P * row + (o % row)).all()
                assert (within + n <= plane).all() and ((first * row + o % row + n) <= wl.seq_lens[r] * row).all()


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_kernel_code_digest():
    """The PMC summaries' staleness pin reads the built library's gfx950 code
    objects: every tagged translation unit is found, the digest is stable, and
    adding the state kernel changes it."""
    import bench
    from paper_2607_28633_amd.build import LIBRARY
    fat = bench._elf_sections(open(LIBRARY, "rb").read())[".hip_fatbin"]
    for tag in bench.KERNEL_TAGS + (bench.STATE_TAG,):
        assert tag in fat, tag
    a, b = bench.kernel_code_digest(), bench.kernel_code_digest()
    assert a == b and len(a) == 64
    assert bench.kernel_code_digest(True) != a


def _host_slabs(wl):
    from paper_2607_28633_amd.workloads import host_dst_prefill, host_src_pool, host_state_cache
    src, dst = host_src_pool(wl), host_dst_prefill(wl)
    slabs = list(range(min(wl.phys_layers, 2)))
    host = {s: (src[s][None].copy(), dst[s][None].copy()) for s in slabs}
    st = None
    if wl.layer_state:
        st = (host_state_cache(wl)[0][None].copy(), host_state_cache(wl, dst=True)[0][None].copy())
    return slabs, host, st


def test_threaded_host_baseline_matches_oracle():
    """The bench's threaded host pack/unpack equals the oracle (it checks each
    layer kind itself before timing) on full, re-blocked, windowed and
    fixed-state layers."""
    import bench
    from paper_2607_28633_amd.workloads import make_workload
    cases = [make_workload("tiny"),
             make_workload("tiny", dst_page_size=48, seq_lens=[100, 0, 37, 16]),
             make_workload("gpt-oss-120b", num_layers=2, seq_lens=[300, 17, 129, 128]),
             make_workload("qwen3.5-397b-hybrid", num_layers=4, seq_lens=[40, 3, 77], state_bytes=1000)]
    for wl in cases:
        hs, refs = _host_slabs(wl), {}
        bench.cpu_baseline(wl, hs, 0.05, refs)          # the oracle's results the threaded leg checks against
        res = bench.cpu_threaded(wl, hs, 0.05, refs, threads=3)
        assert res["value"] > 0 and res["threads"] == 3, wl.name


def test_kernel_launches_per_sweep():
    """The per-launch figures divide a sweep's time by its kernel launches:
    one per layer in the per-layer mode; in the engine mode, the grids the
    library issues for each engine call (topkv_engine_layers_per_grid over
    the call's layers and the packed slot size) and one launch for every
    layer that keeps its own call.  The ceiling copies run in the same layer
    groups."""
    import types

    import bench
    from paper_2607_28633_amd import topkv
    from paper_2607_28633_amd.workloads import make_workload

    def fake_setup(name):
        wl = make_workload(name)
        row = wl.num_heads * wl.head_dim * wl.elem_bytes
        nbytes = wl.planes * row * int(wl.seq_lens.astype(np.int64).sum())
        sl = max(nbytes, wl.num_reqs * wl.state_bytes if wl.layer_state else 0)
        ring = bench.ring_slots(wl, sl)
        return types.SimpleNamespace(wl=wl, tk=topkv, slice=sl, ring=ring, chunks=bench.engine_chunks(wl, ring))

    want = {"llama3-70b-4k": 3, "llama3-70b-batch8": 20, "deepseek-v3-mla": 21, "reblock-70b": 80,
            "llama3-8b": 1, "llama3-70b-tp8": 1}
    for name, grids in want.items():
        st = fake_setup(name)
        assert [bench.sweep_grids(st, "engine", d) for d in (0, 1)] == [grids, grids], name
        assert [bench.sweep_grids(st, "launches", d) for d in (0, 1)] == [st.wl.num_layers] * 2, name
    st = fake_setup("llama3-70b-4k")
    assert bench.layer_groups(st) == [(0, 27), (27, 27), (54, 26)]
    assert "27 layers per grid" in bench.engine_kernel(st.wl, st, "unpack")
    # windowed layers keep their own calls: gpt-oss alternates windowed and full-attention layers
    st = fake_setup("gpt-oss-120b")
    n_engine = sum(1 for kind, _, _ in st.chunks if kind == "engine")
    n_layer = sum(1 for kind, _, _ in st.chunks if kind == "layer")
    assert n_layer == 18 and bench.sweep_grids(st, "engine", 0) >= n_engine + n_layer

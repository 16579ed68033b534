"""The benchmark's split of selected blocks between the band and sparse kernels."""
import os
import sys

import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _sel(rows, ksel):
    out = torch.full((1, 1, len(rows), ksel), -1, dtype=torch.int32)
    for i, r in enumerate(rows):
        out[0, 0, i, :len(r)] = torch.tensor(sorted(r), dtype=torch.int32)
    return out


def test_band_blocks_whole_and_holed_windows():
    # m = 16, 2 init blocks, 64-token window (4 blocks); each row is the last
    # query of a sequence of pos + 1 keys.  The band takes a row's forced blocks
    # (init blocks 0 .. min(2, cur + 1) - 1 and local A .. cur) when it holds all.
    m, n_init, w = 16, 2, 64
    rows = [
        [0],                    # pos 0: cur 0, init {0}, A = 1 > cur: 1 band block
        [0, 1],                 # pos 16 (cur 1): init {0, 1}, A = 2 > cur: 2
        [0, 1, 2, 3, 4, 5, 6],  # pos 100 (cur 6): init {0, 1}, local 2..6: 7
        [0, 1, 2, 4, 5, 6],     # hole at 3: no band
        [0, 1, 2, 3, 4, 5, 6, 9],  # block 9 past cur is not valid: 7
        [1, 2, 3, 4, 5, 6],     # init block 0 missing: no band
    ]
    pos = [0, 16, 100, 100, 100, 100]
    want = [1, 2, 7, 0, 7, 0]
    want_init = [1, 2, 2, 0, 2, 0]
    for r, p, wv, wi in zip(rows, pos, want, want_init):
        nb, a, ni = bench.band_blocks(_sel([r], 8), p + 1, m, n_init, w)
        assert int(nb.item()) == wv, (r, p)
        assert int(ni.item()) == wi, (r, p)
        cur = p // m
        assert int(a.item()) == max(max(0, cur - w // m), min(n_init, cur + 1))


def test_band_blocks_without_window():
    # 64-token blocks, window 0, one init block: the forced blocks are block 0
    # and the row's own block
    m, n_init, w = 64, 1, 0
    rows = [[0], [0, 1], [0, 3, 5, 9], [3, 5, 9], [0, 3, 5]]
    pos = [10, 100, 600, 600, 600]          # cur 0, 1, 9, 9, 9
    want = [1, 2, 2, 0, 0]                  # row 3 lacks block 0, row 4 its own block
    for r, p, wv in zip(rows, pos, want):
        nb, a, ni = bench.band_blocks(_sel([r], 4), p + 1, m, n_init, w)
        assert int(nb.item()) == wv, (r, p)
    sel = _sel([[0, 3, 5, 9]], 4)
    nb, a, ni = bench.band_blocks(sel, 601, m, n_init, w)
    assert bench.sparse_part(sel, nb, a, ni).tolist() == [[[[-1, 3, 5, -1]]]]


def test_sparse_tiles_exclude_band_blocks():
    # m = 16: four blocks per 64-key tile
    m, n_init, w = 16, 1, 64
    row = [0, 5, 6, 7, 8, 9, 10]  # pos 170 (cur 10): A = 6, init 0 and local 6..10 whole
    sel = _sel([row], 8)
    Lk = 171
    nb, a, ni = bench.band_blocks(sel, Lk, m, n_init, w)
    assert int(nb.item()) == 6  # init block 0 and local 6..10
    sparse = bench.sparse_part(sel, nb, a, ni)
    # block 5 remains: tile 1
    assert bench.selected_tiles(sparse, Lk, m) == 1
    assert bench.selected_tiles(sel, Lk, m) == 3  # tiles 0, 1, 2 with the window


def test_cpu_baseline_times_one_slice_and_extrapolates():
    """The CPU baseline runs the oracle on one (batch, KV head) slice, all rows,
    reports the thread count the oracle ran on, and scales the slice's time to
    the whole workload by the selected-block ratio."""
    import oracle
    from paper_2601_02819_amd.inputs import Workload, make_inputs

    wl = Workload("tiny_train", 2, 512, 512, 4, 2, 64, 64, 3, 1, 0, "bf16", backward=True)
    host = make_inputs(wl, seed=0, with_grad_out=True)
    r = bench.cpu_baseline(host, wl, total_blocks=10_000)
    assert r["kind"] == "oracle" and r["unit"] == "TFLOP/s"
    assert r["cores"] == oracle.num_threads() >= 1
    assert r["value"] > 0 and r["seconds"] > 0
    assert "1 of its 4 independent (batch, KV head) slices" in r["sample"]
    # the slice holds 512 rows x 1 group x (1 init + 1 local + 3 picks, fewer early)
    nsel = r["extrapolated_full_seconds"] and 10_000 * r["seconds"] / r["extrapolated_full_seconds"]
    assert 512 * 2 < nsel <= 512 * 5
    assert bench.gpu_clocks().get("unavailable")        # no GPU here

"""The design premise of the simplex-sorted point order, reproduced from
tracked code (the oracle's lattice of the 128^3 d=5 benchmark volume): a tile
of 512 consecutive voxels touches about 290 distinct lattice vertices; after
grouping the points by their vertex 0 (buckets in a random order, as the
GPU's table-slot ids give them), a tile of 512 sorted points touches about 65,
and about one tile in nine has more rows than the forward slice stages in
LDS (112).  These are the figures the kernels are sized for; the test
recomputes them."""
import numpy as np

import synth

T = 512


def _rows_per_tile(vid: np.ndarray) -> np.ndarray:
    n = vid.shape[0] // T * T
    tiles = np.sort(vid[:n].reshape(-1, T * vid.shape[1]), axis=1)
    return 1 + np.count_nonzero(np.diff(tiles, axis=1), axis=1)


def test_sorted_tiles_touch_few_rows(O):
    f = synth.generate("C3")["f"]
    lat = O.lattice(f)
    vid = lat.vert.astype(np.int64)
    natural = _rows_per_tile(vid)
    order = np.random.default_rng(7).permutation(lat.M)  # a random bucket order
    perm = np.argsort(order[vid[:, 0]], kind="stable")
    sorted_rows = _rows_per_tile(vid[perm])
    assert 250 <= natural.mean() <= 330, natural.mean()
    assert 55 <= sorted_rows.mean() <= 80, sorted_rows.mean()
    assert natural.mean() / sorted_rows.mean() > 3.5
    assert 0.05 <= (sorted_rows > 112).mean() <= 0.2, (sorted_rows > 112).mean()

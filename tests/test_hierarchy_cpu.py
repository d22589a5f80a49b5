"""Host logic of the memory hierarchy (no GPU): frustum filtering of
camera-partition pairs against the oracle's linear program, on random boxes
and on the grid workloads' cameras and cells; the host cache's slot map."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_27735_amd import synthetic as S
from paper_2608_27735_amd.camera import look_at


def _hierarchy():
    pytest.importorskip("torch")
    from paper_2608_27735_amd import hierarchy
    return hierarchy


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_visible_boxes_matches_the_oracle(seed):
    H = _hierarchy()
    r = S.rng(300 + seed)
    cam = look_at(r.uniform(-8, 8, 3), r.uniform(-1, 1, 3), int(r.integers(32, 200)),
                  int(r.integers(32, 200)), fov_x_deg=float(r.uniform(30, 100)))
    n = 300
    c = r.uniform(-10, 10, (n, 3))
    ext = np.exp(r.uniform(np.log(0.02), np.log(3.0), (n, 3)))
    lo, hi = c - ext, c + ext
    got = H.visible_boxes(cam, lo, hi)
    n_vis = n_skip = 0
    for i in range(n):
        ok, s = O.box_meets_frustum(cam, lo[i], hi[i])
        if abs(s) < 1e-9:  # touching: either answer is right
            n_skip += 1
            continue
        assert got[i] == ok, (i, s)
        n_vis += ok
    assert 0 < n_vis < n - n_skip  # both outcomes occur


def test_visible_cells_of_the_workloads():
    H = _hierarchy()
    w = S.active_block_1m(n=16)
    for cam in w.cams[::25]:
        vis = H.visible_cells(cam, w.grid, margin=0.5)
        for c in range(w.grid.n_cells):
            lo, hi = w.grid.bounds(c)
            ok, s = O.box_meets_frustum(cam, lo - 0.5, hi + 0.5)
            if abs(s) > 1e-9:
                assert vis[c] == ok
        assert vis[w.active]

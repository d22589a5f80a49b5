"""GPU parity at the large workloads, through the launch path the bench times
(ActiveBlockStep: capacity mode, tile schedules, split backward, persistent
buffers):
  - the 1M-Gaussian active block (SH degree 3) at 1297x840 the bench measures,
    with uniform scales and with heavy-tailed scales;
  - the same block at 1920x1080, uniform and heavy-tailed (the large-block
    configuration);
  - the mid-scale scene's 300K-Gaussian active block at 1297x840 (ground plane
    and blobs);
  - the stress configuration's 4M-Gaussian active block of tiny Gaussians at
    2560x1440.

The oracle bins every workload whole; it cannot rasterise these frames in
seconds, so the images and gradients are checked on sampled outputs it can
compute on its own:
  - projection: the binning fields of all Gaussians, bit-exact;
  - binning: M, every tile range, the whole sorted value list and the whole
    sorted key list, bit-exact against the oracle's binning of all Gaussians;
  - forward: every pixel of the sampled tiles, max abs <= 1e-5 off the
    knife-edge pixels, `last` bit-exact there;
  - backward: with dL/dout zero outside the sampled tiles, every parameter
    gradient depends only on those tiles, so the oracle's gradients from the
    subset lists are the full answer: relative L2 <= 1e-4 per tensor.
The sampled tiles are the eight with the longest walks (where the schedules,
the split and long lists matter) and sixteen seeded random tiles.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_27735_amd import synthetic as S

pytestmark = pytest.mark.gpu

FWD_TOL = 1e-5
GRAD_TOL = 1e-4
# Knife-edge pixels: a threshold decision within the error the fp32 kernels
# can make on it. Alpha decisions take a relative 2e-6 (exp2 and opacity
# rounding) plus 8 x 2^-24 times the magnitude of the terms of the quadratic
# form in Cholesky form (the two products of its first square cancel for long
# thin splats far along their major axis; the oracle pin against an fp32
# emulation finds the actual error within 1/8 of that bound); the stop
# decision takes the accumulated bound of the transmittance. At most 2 % of
# the sampled pixels of any workload may be knife-edge.
KNIFE_REL = 2e-6
KNIFE_KAPPA = 8.0
KNIFE_FRAC = 0.02
WORKLOADS = {
    "1m-uniform-1297x840": lambda: S.active_block_1m(),
    "1m-heavy-tail-1297x840": lambda: S.active_block_1m(heavy_tail=True),
    "1m-uniform-1920x1080": lambda: S.active_block_1m(width=1920, height=1080),
    "1m-heavy-tail-1920x1080": lambda: S.active_block_1m(width=1920, height=1080, heavy_tail=True),
    "300k-midscale-1297x840": lambda: S.midscale_block(),
    "4m-stress-2560x1440": lambda: S.stress_block(),
}


def say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(scope="module", params=list(WORKLOADS), ids=list(WORKLOADS))
def full(request):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_27735_amd import api
    from paper_2608_27735_amd.step import ActiveBlockStep
    dev = torch.device("cuda:0")
    say("large workload", request.param)
    w = WORKLOADS[request.param]()
    cam, prm, scene = w.cam, w.params, w.scene
    r = S.rng(5)
    F, B = S.background_pair(r, cam.height, cam.width)
    params = {k: torch.from_numpy(v).to(dev) for k, v in scene.items()}
    st = ActiveBlockStep(cam, prm, params)
    st.project_and_bin(sync=True)
    Fd, Bd = torch.from_numpy(F).to(dev), torch.from_numpy(B).to(dev)
    st.forward(Fd, Bd)
    torch.cuda.synchronize()
    pb = O.project_bin(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                       scene["opacity_logits"])
    yield dict(api=api, st=st, cam=cam, prm=prm, scene=scene, F=F, B=B, Fd=Fd, Bd=Bd, r=r,
               pb=pb, name=request.param)
    del st, params
    torch.cuda.empty_cache()


def _tiles(cam):
    return (cam.width + 15) // 16, (cam.height + 15) // 16


def _sampled_tiles(full):
    cam, st = full["cam"], full["st"]
    ntx, nty = _tiles(cam)
    last = st.fwd["last"].cpu().numpy().astype(np.int64)
    H, W = cam.height, cam.width
    pad = np.zeros((nty * 16, ntx * 16), np.int64)
    pad[:H, :W] = last
    walk = pad.reshape(nty, 16, ntx, 16).max(axis=(1, 3)).reshape(-1)
    heavy = np.argsort(-walk, kind="stable")[:8]
    rnd = S.rng(77).choice(ntx * nty, 16, replace=False)
    return np.unique(np.concatenate([heavy, rnd]))


def _square_rect(pb, cam):
    """Tile rectangles and counts of the plain 3-sigma support squares (no cut
    to the alpha_min ellipse), in the fp32 steps of the binning chain."""
    f = np.float32
    u, v, r = pb["means2d"][:, 0], pb["means2d"][:, 1], pb["radius"]
    ntx, nty = _tiles(cam)
    x0 = np.maximum(np.floor((u - r) * f(0.0625)), f(0))
    x1 = np.minimum(np.floor((u + r) * f(0.0625)), f(ntx - 1))
    y0 = np.maximum(np.floor((v - r) * f(0.0625)), f(0))
    y1 = np.minimum(np.floor((v + r) * f(0.0625)), f(nty - 1))
    vis = (pb["tiles_touched"] > 0) & (x0 <= x1) & (y0 <= y1)
    rect = np.stack([x0, y0, x1, y1], 1).astype(np.int32)
    rect[~vis] = np.array([1, 0, 0, 0], np.int32)
    tiles = np.where(vis, (rect[:, 2] - rect[:, 0] + 1) * (rect[:, 3] - rect[:, 1] + 1), 0)
    return rect, tiles.astype(np.uint32)


def _oracle_subset(full, tiles, square=False):
    """Oracle projection of all Gaussians; oracle lists of the sampled tiles
    from the subset of Gaussians whose rectangle meets one of them (square:
    the uncut 3-sigma squares instead of the binning boxes)."""
    cam, pb = full["cam"], full["pb"]
    ntx, _ = _tiles(cam)
    if square:
        rect_sq, tiles_sq = _square_rect(pb, cam)
        pb = dict(pb, rect=rect_sq, tiles_touched=tiles_sq)
    rect = pb["rect"].astype(np.int64)  # tx0, ty0, tx1, ty1 (empty if tx1 < tx0)
    tx, ty = tiles % ntx, tiles // ntx
    meets = np.zeros(len(rect), bool)
    for a, b in zip(tx, ty):
        meets |= (rect[:, 0] <= a) & (a <= rect[:, 2]) & (rect[:, 1] <= b) & (b <= rect[:, 3])
    idx = np.nonzero(meets)[0]  # increasing: the subset keeps the index order
    _, vals, ranges = O.bin(cam.width, cam.height, pb["depth"][idx], pb["rect"][idx],
                            pb["tiles_touched"][idx])
    return pb, idx, vals, ranges


def test_fullsize_projection_and_binning(full):
    st, cam, pb = full["st"], full["cam"], full["pb"]
    say("projection + binning", full["name"])
    P = {k: v.cpu().numpy() for k, v in st.proj.items()}
    assert np.array_equal(P["means2d"].view(np.uint32), pb["means2d"].view(np.uint32))
    assert np.array_equal(P["depth"].view(np.uint32), pb["depth"].view(np.uint32))
    assert np.array_equal(P["extent"].view(np.uint32), pb["extent"].view(np.uint32))
    assert np.array_equal(P["tiles_touched"].view(np.uint32), pb["tiles_touched"])
    # M and every tile's list length from the oracle's rectangles
    ntx, nty = _tiles(cam)
    rect = pb["rect"].astype(np.int64)
    vis = rect[:, 2] >= rect[:, 0]
    diff = np.zeros((nty + 1, ntx + 1), np.int64)
    np.add.at(diff, (rect[vis, 1], rect[vis, 0]), 1)
    np.add.at(diff, (rect[vis, 1], rect[vis, 2] + 1), -1)
    np.add.at(diff, (rect[vis, 3] + 1, rect[vis, 0]), -1)
    np.add.at(diff, (rect[vis, 3] + 1, rect[vis, 2] + 1), 1)
    count = diff.cumsum(0).cumsum(1)[:nty, :ntx].reshape(-1)
    m = int(pb["tiles_touched"].astype(np.int64).sum())
    tr = st.tile_ranges.cpu().numpy().view(np.uint32).astype(np.int64)
    assert int(tr[-1, 1]) == m
    assert np.array_equal(tr[:, 1] - tr[:, 0], count)
    assert np.array_equal(tr[1:, 0], tr[:-1, 1]) and tr[0, 0] == 0
    # the whole sorted lists and keys against the oracle's binning of every
    # Gaussian
    say("whole lists and keys", full["name"], "M =", m)
    keys_o, vals_o, ranges_o = O.bin(cam.width, cam.height, pb["depth"], pb["rect"],
                                     pb["tiles_touched"])
    assert len(vals_o) == m
    assert np.array_equal(tr.astype(np.uint32), ranges_o)
    values = st.values[:m].cpu().numpy().view(np.uint32)
    assert np.array_equal(values, vals_o)
    del values
    api = full["api"]
    kb = api.bin_sort(cam.width, cam.height, st.proj, capacity=m, want_keys=True, sync=True)
    assert kb["n_isect"] == m
    keys = kb["keys"][:m].cpu().numpy().view(np.uint64)
    del kb
    torch.cuda.empty_cache()
    assert np.array_equal(keys, keys_o)
    print(f"  M = {m}: every tile range, value and key bit-exact")


def _subset_values(full, pb, idx):
    cam, prm, scene = full["cam"], full["prm"], full["scene"]
    sub = {k: v[idx] for k, v in scene.items()}
    pv = O.project_values(cam, prm, sub["means"], sub["log_scales"], sub["quats"],
                          sub["opacity_logits"], sub["sh"], pb["tiles_touched"][idx])
    return pb["means2d"][idx].astype(np.float64), pv


def _only(ranges, tiles):
    r = np.zeros_like(ranges)
    r[tiles] = ranges[tiles]
    return r


def test_fullsize_forward_on_sampled_tiles(full):
    st, cam, prm = full["st"], full["cam"], full["prm"]
    say("forward, sampled tiles", full["name"])
    tiles = _sampled_tiles(full)
    pb, idx, vals, ranges = _oracle_subset(full, tiles)
    m2d, pv = _subset_values(full, pb, idx)
    ref = O.render_fwd(cam, prm, _only(ranges, tiles), vals, m2d, pv["conic"], pv["opacity"],
                       pv["rgb"], full["F"], full["B"], rel_margin=KNIFE_REL, f32_kappa=KNIFE_KAPPA)
    out = st.fwd["out"].cpu().numpy()
    last = st.fwd["last"].cpu().numpy().view(np.uint32)
    ntx, _ = _tiles(cam)
    worst, knives, npx = 0.0, 0, 0
    for t in tiles:
        y0, x0 = (t // ntx) * 16, (t % ntx) * 16
        ys, xs = slice(y0, min(y0 + 16, cam.height)), slice(x0, min(x0 + 16, cam.width))
        kn = ref["knife"][ys, xs]
        err = np.abs(out[ys, xs] - ref["out"][ys, xs]).max(axis=-1)
        assert err[kn].max(initial=0.0) <= 0.02
        worst = max(worst, err[~kn].max(initial=0.0))
        assert np.array_equal(last[ys, xs][~kn], ref["last"][ys, xs][~kn]), t
        knives += int(kn.sum())
        npx += kn.size
    print(f"  {len(tiles)} tiles, max err {worst:.2e}, knife-edge pixels {knives} of {npx}")
    assert worst <= FWD_TOL
    assert knives <= max(8, KNIFE_FRAC * npx)


def test_fullsize_binning_box_changes_no_image(full):
    """The GPU's image on its cut lists against the oracle on the uncut 3-sigma
    squares, on the sampled tiles: the dropped pairs blend nothing."""
    st, cam, prm = full["st"], full["cam"], full["prm"]
    say("binning box vs squares, sampled tiles", full["name"])
    tiles = _sampled_tiles(full)
    pb, idx, vals, ranges = _oracle_subset(full, tiles, square=True)
    m2d, pv = _subset_values(full, pb, idx)
    ref = O.render_fwd(cam, prm, _only(ranges, tiles), vals, m2d, pv["conic"], pv["opacity"],
                       pv["rgb"], full["F"], full["B"], rel_margin=KNIFE_REL, f32_kappa=KNIFE_KAPPA)
    out = st.fwd["out"].cpu().numpy()
    ntx, _ = _tiles(cam)
    worst, knives, npx = 0.0, 0, 0
    for t in tiles:
        y0, x0 = (t // ntx) * 16, (t % ntx) * 16
        ys, xs = np.mgrid[y0:min(y0 + 16, cam.height), x0:min(x0 + 16, cam.width)]
        kn = ref["knife"][ys, xs]
        err = np.abs(out[ys, xs] - ref["out"][ys, xs]).max(axis=-1)
        worst = max(worst, err[~kn].max(initial=0.0))
        knives += int(kn.sum())
        npx += kn.size
    print(f"  {len(tiles)} tiles, max err {worst:.2e}, knife-edge pixels {knives} of {npx}")
    assert worst <= FWD_TOL
    assert knives <= max(8, KNIFE_FRAC * npx)


def test_fullsize_backward_from_sampled_tiles(full):
    api, st, cam, prm, scene = full["api"], full["st"], full["cam"], full["prm"], full["scene"]
    say("backward, upstream gradient on sampled tiles", full["name"])
    tiles = _sampled_tiles(full)
    pb, idx, vals, ranges = _oracle_subset(full, tiles)
    m2d, pv = _subset_values(full, pb, idx)
    rsub = _only(ranges, tiles)
    ref = O.render_fwd(cam, prm, rsub, vals, m2d, pv["conic"], pv["opacity"], pv["rgb"], full["F"],
                       full["B"], rel_margin=KNIFE_REL, f32_kappa=KNIFE_KAPPA)
    ntx, _ = _tiles(cam)
    mask = np.zeros((cam.height, cam.width), bool)
    for t in tiles:
        y0, x0 = (t // ntx) * 16, (t % ntx) * 16
        mask[y0:y0 + 16, x0:x0 + 16] = True
    G = S.upstream_grad(S.rng(78), cam.height, cam.width) * (mask & ~ref["knife"])[..., None]
    g2d_sub = O.render_bwd_2d(cam, prm, rsub, vals, m2d, pv["conic"], pv["opacity"], pv["rgb"],
                              full["F"], full["B"], G.astype(np.float64))
    g2d = np.zeros((len(scene["means"]), 9))
    g2d[idx] = g2d_sub
    refg = O.project_bwd(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                         scene["opacity_logits"], scene["sh"], pb["tiles_touched"], g2d)
    grads = st.backward(torch.from_numpy(G).to(st.dL_dout.device), full["Fd"], full["Bd"])
    torch.cuda.synchronize()
    for k in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        g = grads[k].cpu().numpy().astype(np.float64)
        gr = refg[k]
        rel = np.linalg.norm(g - gr) / max(np.linalg.norm(gr), 1e-30)
        print(f"  grad {k}: rel L2 {rel:.2e}")
        assert rel <= GRAD_TOL, (k, rel)

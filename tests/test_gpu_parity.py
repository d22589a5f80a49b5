"""GPU parity of every stage of the active-block step against the CPU oracle.

Bars (fp32 GPU path vs fp64 oracle on identical seeded inputs):
  - intersection count, sorted values, sorted keys, tile ranges, tiles_touched,
    pixel-space means, depths, radii: bit-exact;
  - composited RGBA and F/B: max abs <= 1e-5 per channel (pixels with a
    threshold decision within a relative 1e-4 of its threshold -- "knife-edge",
    where both precisions are legitimately different -- are reported and
    excluded; they must be few);
  - gradients: relative L2 <= 1e-4 per parameter tensor.
Every case prints its name and shape before touching the GPU.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_27735_amd import synthetic as S
from paper_2608_27735_amd.camera import RasterParams, look_at

pytestmark = pytest.mark.gpu

FWD_TOL = 1e-5
GRAD_TOL = 1e-4
KNIFE = 1e-4
# frames of at most this many tiles render, when not split, with four
# workgroups per tile (one pixel row per wave, four list entries per step)
ROWS_TILES = 256


@pytest.fixture(scope="module")
def api():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_27735_amd import api as A
    return A


def dev():
    return torch.device("cuda:0")


def to_dev(d):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev()) for k, v in d.items()}


def say(*a):
    print("[case]", *a, flush=True)


def cases():
    """(name, camera, params, scene) at sizes the oracle handles in seconds."""
    out = []
    w = S.tiny()
    out.append(("tiny-active", w.cams[0], w.params, S.subset(w.scene, w.cell_of == w.active)))
    out.append(("tiny-all", w.cams[0], w.params, w.scene))
    r = S.ring()
    sc = S.subset(r.scene, r.cell_of == r.active)
    out.append(("ring-active-cam0", r.cams[0], r.params, sc))
    out.append(("ring-active-cam3", r.cams[3], r.params, sc))
    # the whole 64K-Gaussian scene: several radix blocks and tile chunks
    out.append(("ring-all-cam5", r.cams[5], r.params, r.scene))
    # ragged image (not a multiple of 16), SH degree 2, bigger Gaussians
    rr = S.rng(21)
    cam = look_at((0.3, -3.0, 1.1), (0, 0, 0), 203, 117)
    prm = RasterParams(sh_degree=2)
    sc2 = S.gaussians(rr, rr.uniform(-1, 1, (3000, 3)), 2, math.log(0.05), 0.6)
    out.append(("ragged-203x117", cam, prm, sc2))
    # a deep tile: 24,000 faint sub-pixel Gaussians over a few tiles, so walks
    # run through lists of thousands of entries without saturating (more than
    # 64 chunks of 256: the split's open-ended last chunk)
    rd = S.rng(22)
    cam = look_at((0.0, -3.0, 0.0), (0, 0, 0), 48, 48)
    sc3 = S.gaussians(rd, rd.uniform((-0.5, -0.5, -0.5), (0.5, 0.5, 0.5), (24000, 3)), 0,
                      math.log(0.02), 0.2)
    sc3["opacity_logits"] = rd.normal(-4.0, 0.3, 24000).astype(np.float32)
    out.append(("deep-tile-48x48", cam, RasterParams(sh_degree=0), sc3))
    # small splats (1-3 pixels) in a ragged 100x75 image: most entries reach
    # only some of a tile's four-row strips, and the last tile row holds 11
    # rows (its third strip is clipped, its fourth empty)
    rs = S.rng(23)
    cam = look_at((0.0, -3.0, 0.4), (0, 0, 0), 100, 75)
    sc4 = S.gaussians(rs, rs.uniform((-0.8, -0.8, -0.6), (0.8, 0.8, 0.6), (6000, 3)), 1,
                      math.log(0.012), 0.4)
    out.append(("small-splats-100x75", cam, RasterParams(sh_degree=1), sc4))
    # small active blocks take the two-launch binning (at most 2,048 Gaussians,
    # 2,048 tiles): a ragged frame, and the largest block it takes next to one
    # Gaussian more (the general path)
    rk = S.rng(24)
    cam = look_at((0.2, -3.0, 0.9), (0, 0, 0), 203, 117)
    sc5 = S.gaussians(rk, rk.uniform(-1, 1, (1500, 3)), 2, math.log(0.05), 0.6)
    out.append(("small-path-ragged-203x117", cam, RasterParams(sh_degree=2), sc5))
    ring_n = {k: v[:2048] for k, v in r.scene.items()}
    out.append(("small-path-2048-cam1", r.cams[1], r.params, ring_n))
    # frames on both sides of the tile count up to which the blend kernels
    # give each tile four workgroups (256 = 16 x 16 tiles; 17 x 16 = 272)
    rb = S.rng(25)
    scb = S.gaussians(rb, rb.uniform(-1, 1, (2500, 3)), 1, math.log(0.04), 0.5)
    out.append(("rows-256-tiles-256x256", look_at((0.1, -3.0, 0.8), (0, 0, 0), 256, 256),
                RasterParams(sh_degree=1), scb))
    out.append(("general-272-tiles-272x256", look_at((0.1, -3.0, 0.8), (0, 0, 0), 272, 256),
                RasterParams(sh_degree=1), scb))
    out.append(("general-path-2049-cam1", r.cams[1], r.params,
                {k: v[:2049] for k, v in r.scene.items()}))
    return out


CASES = cases()


def gpu_project(api, cam, prm, scene):
    return api.project(cam, prm, **to_dev(scene))


def np32(t):
    return t.cpu().numpy()


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_project_bitexact_binning_fields_and_close_values(api, case):
    name, cam, prm, scene = case
    say("project", name, scene["means"].shape)
    p = gpu_project(api, cam, prm, scene)
    torch.cuda.synchronize()
    ob = O.project_bin(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                       scene["opacity_logits"])
    ov = O.project_values(cam, prm, **scene, tiles_touched=ob["tiles_touched"])
    assert np.array_equal(np32(p["tiles_touched"]).view(np.uint32), ob["tiles_touched"])
    assert np.array_equal(np32(p["means2d"]).view(np.uint32), ob["means2d"].view(np.uint32))
    assert np.array_equal(np32(p["depth"]).view(np.uint32), ob["depth"].view(np.uint32))
    assert np.array_equal(np32(p["extent"]).view(np.uint32), ob["extent"].view(np.uint32))
    vis = ob["tiles_touched"] > 0
    assert vis.sum() > 0
    co = np32(p["conic_opacity"])
    # the conic as its Cholesky factor (l11, l21, l22), relative to its scale
    ref = _factor_of(ov["conic"])
    scale = np.abs(ref).max(axis=1, keepdims=True) + 1e-30
    assert np.max(np.abs(co[vis, :3] - ref[vis]) / scale[vis]) < 1e-5
    assert np.max(np.abs(co[:, 3] - ov["opacity"])) < 1e-6
    assert np.max(np.abs(np32(p["rgb"]) - ov["rgb"])) < 1e-5


def _factor_of(conic):
    """Cholesky factor (l11, l21, l22) of conics (a, b, c): [[a, b], [b, c]] = L L^T
    with L = [[l11, 0], [l21, l22]] (zeros for a zero conic)."""
    a, b, c = conic[:, 0], conic[:, 1], conic[:, 2]
    l11 = np.sqrt(np.maximum(a, 0.0))
    safe = np.where(l11 > 0, l11, 1.0)
    l21 = np.where(l11 > 0, b / safe, 0.0)
    l22 = np.where(l11 > 0, np.sqrt(np.maximum(a * c - b * b, 0.0)) / safe, 0.0)
    return np.stack([l11, l21, l22], 1)


def _conic_of(co):
    """fp64 conic (a, b, c) = L L^T of fp32 factors stored as conic_opacity[:, :3]."""
    l = co[:, :3].astype(np.float64)
    return np.stack([l[:, 0] ** 2, l[:, 0] * l[:, 1], l[:, 1] ** 2 + l[:, 2] ** 2], 1)


def _oracle_inputs_f32(cam, prm, scene):
    """Oracle projection rounded to fp32 (the conic as its Cholesky factor, as
    the GPU stores it): the stage inputs both sides consume."""
    ob = O.project_bin(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                       scene["opacity_logits"])
    ov = O.project_values(cam, prm, **scene, tiles_touched=ob["tiles_touched"])
    co = np.concatenate([_factor_of(ov["conic"]), ov["opacity"][:, None]], 1).astype(np.float32)
    proj = dict(means2d=ob["means2d"], conic_opacity=co, depth=ob["depth"], extent=ob["extent"],
                tiles_touched=ob["tiles_touched"].view(np.int32), rgb=ov["rgb"].astype(np.float32))
    return ob, proj


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_bin_sort_bitexact(api, case):
    name, cam, prm, scene = case
    say("bin_sort", name, scene["means"].shape)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    keys, values, ranges = O.bin(cam.width, cam.height, ob["depth"], ob["rect"], ob["tiles_touched"])
    pd = to_dev(proj)
    b = api.bin_sort(cam.width, cam.height, pd, want_keys=True)
    torch.cuda.synchronize()
    m = b["n_isect"]
    assert m == len(values)
    assert np.array_equal(np32(b["values"][:m]).view(np.uint32), values)
    assert np.array_equal(np32(b["keys"][:m]).view(np.uint64), keys)
    assert np.array_equal(np32(b["tile_ranges"]).view(np.uint32), ranges)
    # the forward's schedule: tiles by decreasing quarter octave of list
    # length (the leading one and the two bits after it), stable
    length = (ranges[:, 1] - ranges[:, 0]).astype(np.int64)
    def quarter_octave(x):
        if x == 0:
            return 128
        nb = int(x).bit_length()
        sub = (int(x) >> (nb - 3)) & 3 if nb >= 3 else (int(x) << (3 - nb)) & 3
        return 4 * (32 - nb) + 3 - sub
    key = np.array([quarter_octave(x) for x in length])
    assert np.array_equal(np32(b["tile_order"]), np.argsort(key, kind="stable"))
    # determinism: a second call gives identical bytes
    b2 = api.bin_sort(cam.width, cam.height, pd, want_keys=True)
    torch.cuda.synchronize()
    assert torch.equal(b2["values"][:m], b["values"][:m])
    assert torch.equal(b2["keys"][:m], b["keys"][:m])



@pytest.mark.parametrize("width", [16400, 33000])
def test_bin_sort_wide_strip_frames(api, width):
    """Frames of many 8x8-tile blocks (129 and 258 in one block row; 2,050
    and 4,126 tiles): the level-2 sub-chunk lookup scans blocks in several
    64-lane rounds, and at 258 blocks each level-1 thread publishes and looks
    back for two blocks. 3,000 Gaussians along the horizon of a 32-pixel-high
    strip; lists, keys and ranges bit-exact against the oracle."""
    say("bin_sort wide strip", width)
    rr = S.rng(31)
    cam = look_at((0.0, -3.0, 0.0), (0, 0, 0), width, 32, fov_x_deg=120.0)
    prm = RasterParams(sh_degree=0)
    means = np.stack([rr.uniform(-4.5, 4.5, 3000), rr.uniform(-0.5, 0.5, 3000),
                      rr.uniform(-0.003, 0.003, 3000)], 1)
    scene = S.gaussians(rr, means, 0, math.log(0.003), 0.6)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    keys, values, ranges = O.bin(cam.width, cam.height, ob["depth"], ob["rect"], ob["tiles_touched"])
    assert len(values) > 3000
    pd = to_dev(proj)
    b = api.bin_sort(cam.width, cam.height, pd, want_keys=True)
    torch.cuda.synchronize()
    m = b["n_isect"]
    assert m == len(values)
    assert np.array_equal(np32(b["values"][:m]).view(np.uint32), values)
    assert np.array_equal(np32(b["keys"][:m]).view(np.uint64), keys)
    assert np.array_equal(np32(b["tile_ranges"]).view(np.uint32), ranges)

def _fwd_compare(got, ref, H, W):
    """Max error off the knife-edge pixels, and the number of knife-edge pixels.
    On a knife-edge pixel one threshold decision may legitimately differ
    between fp32 and fp64: a flipped skip changes the pixel by at most
    alpha_min, a flipped stop by at most t_min / (1 - alpha_max) = 0.01."""
    knife = ref["knife"]
    err = np.abs(got - ref["out"]).reshape(H, W, 4)
    off = err[~knife]
    on = err[knife]
    assert (on.max() if on.size else 0.0) <= 0.02
    assert knife.sum() <= max(8, 0.01 * H * W)
    return (off.max() if off.size else 0.0), int(knife.sum())


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("with_fb", [False, True])
def test_render_fwd_stage(api, case, with_fb):
    """Forward on identical fp32 screen-space inputs (oracle projection)."""
    name, cam, prm, scene = case
    say("render_fwd stage", name, with_fb)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    _, values, ranges = O.bin(cam.width, cam.height, ob["depth"], ob["rect"], ob["tiles_touched"])
    F = B = None
    if with_fb:
        F, B = S.background_pair(S.rng(31), cam.height, cam.width)
    ref = O.render_fwd(cam, prm, ranges, values, proj["means2d"].astype(np.float64),
                       _conic_of(proj["conic_opacity"]),
                       proj["conic_opacity"][:, 3].astype(np.float64),
                       proj["rgb"].astype(np.float64), F, B, rel_margin=KNIFE)
    pd = to_dev(proj)
    bins = api.bin_sort(cam.width, cam.height, pd)
    nb = torch.zeros(1, dtype=torch.int64, device=dev())
    fw = api.render_fwd(cam, prm, bins, pd, F=None if F is None else torch.from_numpy(F).to(dev()),
                        B=None if B is None else torch.from_numpy(B).to(dev()), n_blends=nb)
    torch.cuda.synchronize()
    err, nk = _fwd_compare(np32(fw["out"]), ref, cam.height, cam.width)
    print(f"  max err {err:.2e}, knife-edge pixels {nk} of {cam.width * cam.height}")
    assert err <= FWD_TOL
    ok = ~ref["knife"]
    assert np.array_equal(np32(fw["last"]).view(np.uint32)[ok], ref["last"][ok])
    assert np.max(np.abs(np32(fw["final_T"]) - ref["final_T"])[ok]) <= FWD_TOL
    assert abs(int(nb.item()) - ref["n_blends"]) <= nk * 4
    # the tile schedule changes no output: raster order gives identical bytes
    nb2 = torch.zeros(1, dtype=torch.int64, device=dev())
    fw2 = api.render_fwd(cam, prm, dict(bins, tile_order=None), pd,
                         F=None if F is None else torch.from_numpy(F).to(dev()),
                         B=None if B is None else torch.from_numpy(B).to(dev()), n_blends=nb2)
    torch.cuda.synchronize()
    for key in ("out", "final_T", "last"):
        assert torch.equal(fw2[key], fw[key])
    assert nb2.item() == nb.item()


def _square_rects(ob, cam):
    """Tile rectangles of the plain support squares [u +- r] x [v +- r] (no
    cut to the alpha_min ellipse), in the fp32 steps of the binning chain."""
    f = np.float32
    u, v = ob["means2d"][:, 0], ob["means2d"][:, 1]
    r = ob["radius"]
    ntx, nty = O.tile_grid(cam.width, cam.height)
    x0 = np.maximum(np.floor((u - r) * f(0.0625)), f(0))
    x1 = np.minimum(np.floor((u + r) * f(0.0625)), f(ntx - 1))
    y0 = np.maximum(np.floor((v - r) * f(0.0625)), f(0))
    y1 = np.minimum(np.floor((v + r) * f(0.0625)), f(nty - 1))
    vis = (ob["tiles_touched"] > 0) & (x0 <= x1) & (y0 <= y1)
    rect = np.stack([x0, y0, x1, y1], 1).astype(np.int32)
    rect[~vis] = 0
    tiles = np.where(vis, (rect[:, 2] - rect[:, 0] + 1) * (rect[:, 3] - rect[:, 1] + 1), 0)
    return rect, tiles.astype(np.uint32)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_binning_box_changes_no_image(api, case):
    """The GPU forward on its cut lists against the oracle on the uncut 3-sigma
    squares: the (tile, Gaussian) pairs the cut drops blend nothing, on the
    GPU's own fp32 alpha as well (the cut keeps the tile test's margin)."""
    name, cam, prm, scene = case
    say("binning box vs squares", name)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    rect, tiles = _square_rects(ob, cam)
    assert tiles.astype(np.int64).sum() >= ob["tiles_touched"].astype(np.int64).sum()
    _, values, ranges = O.bin(cam.width, cam.height, ob["depth"], rect, tiles)
    ref = O.render_fwd(cam, prm, ranges, values, proj["means2d"].astype(np.float64),
                       _conic_of(proj["conic_opacity"]),
                       proj["conic_opacity"][:, 3].astype(np.float64),
                       proj["rgb"].astype(np.float64), None, None, rel_margin=KNIFE)
    pd = to_dev(proj)
    bins = api.bin_sort(cam.width, cam.height, pd)
    nb = torch.zeros(1, dtype=torch.int64, device=dev())
    fw = api.render_fwd(cam, prm, bins, pd, n_blends=nb)
    torch.cuda.synchronize()
    err, nk = _fwd_compare(np32(fw["out"]), ref, cam.height, cam.width)
    print(f"  {int(tiles.astype(np.int64).sum())} square pairs, {bins['n_isect']} binned; "
          f"max err {err:.2e}, knife-edge pixels {nk}")
    assert err <= FWD_TOL
    assert abs(int(nb.item()) - ref["n_blends"]) <= nk * 4


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_render_cache_refresh(api, case):
    """The cached render of a partition: the forward with F = B = transparent
    as fp16 premultiplied RGBA. Against the fp64 oracle: off the knife-edge
    pixels within FWD_TOL plus half an fp16 ulp (the rounding of the store);
    against the fp32 forward of the same bins: bit-identical after numpy's
    round-to-nearest-even conversion."""
    name, cam, prm, scene = case
    say("render_cache", name)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    _, values, ranges = O.bin(cam.width, cam.height, ob["depth"], ob["rect"], ob["tiles_touched"])
    ref = O.render_fwd(cam, prm, ranges, values, proj["means2d"].astype(np.float64),
                       _conic_of(proj["conic_opacity"]),
                       proj["conic_opacity"][:, 3].astype(np.float64),
                       proj["rgb"].astype(np.float64), None, None, rel_margin=KNIFE)
    pd = to_dev(proj)
    bins = api.bin_sort(cam.width, cam.height, pd)
    img = torch.full((cam.height, cam.width, 4), float("nan"), dtype=torch.float16, device=dev())
    api.render_cache(cam, prm, bins, pd, image=img)
    fw = api.render_fwd(cam, prm, bins, pd)
    torch.cuda.synchronize()
    got = img.cpu().numpy()
    assert np.array_equal(got.view(np.uint16), np32(fw["out"]).astype(np.float16).view(np.uint16))
    g64 = got.astype(np.float64)
    half_ulp = np.spacing(np.abs(got)).astype(np.float64) / 2
    ok = ~ref["knife"]
    excess = (np.abs(g64 - ref["out"]) - half_ulp)[ok]
    print(f"  max error beyond the fp16 rounding {excess.max(initial=0.0):.2e}")
    assert excess.max(initial=0.0) <= FWD_TOL
    assert np.abs(g64 - ref["out"])[ref["knife"]].max(initial=0.0) <= 0.02


def test_render_cache_feeds_composite(api):
    """Cached renders of two partitions composited back over: equal to the
    forward of the middle partition between them (fp16 storage error only)."""
    r = S.ring()
    cam, prm = r.cams[2], r.params
    lab = S.rng(13).integers(0, 3, len(r.scene["means"]))
    say("render_cache -> composite", len(lab))

    def prep(sc):
        _, proj = _oracle_inputs_f32(cam, prm, sc)
        pd = to_dev(proj)
        return pd, api.bin_sort(cam.width, cam.height, pd)

    parts = [prep(S.subset(r.scene, lab == i)) for i in range(3)]
    imgs = torch.stack([api.render_cache(cam, prm, b, pd) for pd, b in (parts[0], parts[2])])
    F, B = api.composite_cache(imgs.view(torch.int16), [0, 1], 1)
    mid = api.render_fwd(cam, prm, parts[1][1], parts[1][0], F=F, B=B)
    ref = api.render_fwd(cam, prm, parts[1][1], parts[1][0],
                         F=api.render_fwd(cam, prm, parts[0][1], parts[0][0])["out"],
                         B=api.render_fwd(cam, prm, parts[2][1], parts[2][0])["out"])
    torch.cuda.synchronize()
    assert (mid["out"] - ref["out"]).abs().max().item() <= 2e-3


def test_cache_refresh_to_pinned_host(api):
    """Refresh of a partition's renders for several cameras (binning buffers
    grown on the way, double-buffered device staging, copies on a second
    stream): every host image equals that camera's own cached render."""
    from paper_2608_27735_amd.cache import CacheRefresher
    r = S.ring()
    prm = r.params
    sc = S.subset(r.scene, r.cell_of == r.active)
    cams = [r.cams[i] for i in (0, 3, 5, 1, 3)]
    say("cache refresh", len(cams), "cameras", sc["means"].shape)
    params = to_dev(sc)
    H, W = cams[0].height, cams[0].width
    hosts = [torch.full((H, W, 4), float("nan"), dtype=torch.float16).pin_memory()
             for _ in cams]
    ref = CacheRefresher(prm, params, W, H)
    rects = torch.zeros((len(cams), 4), dtype=torch.int32, device=dev())
    ref.refresh(cams, hosts, rects)
    for i, (cam, h) in enumerate(zip(cams, hosts)):
        pd = api.project(cam, prm, **params)
        bins = api.bin_sort(W, H, pd)
        rect = torch.zeros(4, dtype=torch.int32, device=dev())
        want = api.render_cache(cam, prm, bins, pd, rect=rect).cpu()
        assert torch.equal(h.view(torch.int16), want.view(torch.int16))
        assert torch.equal(rects[i], rect)
    assert any(h.float().abs().sum() > 0 for h in hosts)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_step_end_to_end(api, case):
    """Parameters -> composited image and parameter gradients, both sides from
    the same seeded parameters, F, B and upstream gradient."""
    name, cam, prm, scene = case
    say("end-to-end", name, scene["means"].shape)
    r = S.rng(41)
    F, B = S.background_pair(r, cam.height, cam.width)
    G = S.upstream_grad(r, cam.height, cam.width)
    ref0 = O.step(cam, prm, scene, F=F, B=B, rel_margin=KNIFE)
    # upstream gradient is zeroed on knife-edge pixels (the oracle decides which)
    G = G * (~ref0["fwd"]["knife"])[..., None]
    ref = O.step(cam, prm, scene, F=F, B=B, dL_dout=G.astype(np.float64))
    params = to_dev(scene)
    Fd, Bd = torch.from_numpy(F).to(dev()), torch.from_numpy(B).to(dev())
    p = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, p)
    fw = api.render_fwd(cam, prm, bins, p, F=Fd, B=Bd)
    grads = api.render_bwd(cam, prm, params, p, bins, fw, torch.from_numpy(G).to(dev()), F=Fd, B=Bd,
                           want_means2d=True)
    torch.cuda.synchronize()
    assert bins["n_isect"] == len(ref["sorted_values"])
    err, nk = _fwd_compare(np32(fw["out"]), ref0["fwd"], cam.height, cam.width)
    print(f"  fwd max err {err:.2e}, knife {nk}")
    assert err <= FWD_TOL
    for k in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        g = np32(grads[k]).astype(np.float64)
        gr = ref["grads"][k]
        rel = np.linalg.norm(g - gr) / max(np.linalg.norm(gr), 1e-30)
        print(f"  grad {k}: rel L2 {rel:.2e}")
        assert rel <= GRAD_TOL, (k, rel)
    g2 = np32(grads["means2d"]).astype(np.float64)
    rel = np.linalg.norm(g2 - ref["g2d"][:, :2]) / max(np.linalg.norm(ref["g2d"][:, :2]), 1e-30)
    assert rel <= GRAD_TOL


@pytest.mark.parametrize("hw", [(1, 1), (3, 5), (16, 16), (1, 17), (31, 2)])
def test_step_degenerate_frames(api, hw):
    """Frames of one pixel, one partial tile, one whole tile, a one-pixel
    column and a two-row strip: every tile's rows mostly clipped by the image
    (four workgroups per tile, most of their pixels outside)."""
    H, W = hw
    rr = S.rng(26)
    cam = look_at((0.0, -2.5, 0.3), (0, 0, 0), W, H, fov_x_deg=20.0)
    sc = S.gaussians(rr, rr.uniform(-0.3, 0.3, (300, 3)), 1, math.log(0.05), 0.6)
    test_step_end_to_end(api, (f"{W}x{H}", cam, RasterParams(sh_degree=1), sc))


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("chunk,n_slots", [(256, None), (512, None), (256, 3)])
def test_split_backward(api, case, chunk, n_slots):
    """Long tiles split into chunks for the backward: the forward's outputs are
    unchanged, the gradients match the oracle to the same bar and the unsplit
    backward up to rounding. n_slots = 3 leaves most tiles without slots
    (those run unsplit)."""
    name, cam, prm, scene = case
    say("split backward", name, chunk, n_slots)
    r = S.rng(43)
    F, B = S.background_pair(r, cam.height, cam.width)
    G = S.upstream_grad(r, cam.height, cam.width)
    ref0 = O.step(cam, prm, scene, F=F, B=B, rel_margin=KNIFE)
    G = G * (~ref0["fwd"]["knife"])[..., None]
    ref = O.step(cam, prm, scene, F=F, B=B, dL_dout=G.astype(np.float64))
    params = to_dev(scene)
    Fd, Bd = torch.from_numpy(F).to(dev()), torch.from_numpy(B).to(dev())
    Gd = torch.from_numpy(G).to(dev())
    p = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, p)
    if n_slots is None:
        n_slots = bins["n_isect"] // chunk + api.n_tiles(cam.width, cam.height) + 1
    split = api.make_split(n_slots, chunk)
    fw = api.render_fwd(cam, prm, bins, p, F=Fd, B=Bd, split=split)
    fw0 = api.render_fwd(cam, prm, bins, p, F=Fd, B=Bd)
    g0 = api.render_bwd(cam, prm, params, p, bins, fw0, Gd, F=Fd, B=Bd)
    gs = api.render_bwd(cam, prm, params, p, bins, fw, Gd, F=Fd, B=Bd, split=split)
    torch.cuda.synchronize()
    if api.n_tiles(cam.width, cam.height) > ROWS_TILES:
        for key in ("out", "final_T", "last"):
            assert torch.equal(fw[key], fw0[key])
    else:
        # the unsplit forward of a small frame takes the four-workgroups-per-
        # tile kernel: the same walk, rounded in another order
        ok = ~ref0["fwd"]["knife"]
        assert np.array_equal(np32(fw["last"])[ok], np32(fw0["last"])[ok])
        assert (fw["out"] - fw0["out"]).abs().max().item() <= FWD_TOL
        assert (fw["final_T"] - fw0["final_T"]).abs().max().item() <= FWD_TOL
    lens = np32(bins["tile_ranges"]).view(np.uint32).astype(np.int64)
    print(f"  tiles longer than a chunk: {int(((lens[:, 1] - lens[:, 0]) > chunk).sum())}")
    for k in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        a = np32(gs[k]).astype(np.float64)
        b = np32(g0[k]).astype(np.float64)
        gr = ref["grads"][k]
        rel = np.linalg.norm(a - gr) / max(np.linalg.norm(gr), 1e-30)
        rel0 = np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)
        print(f"  grad {k}: rel L2 {rel:.2e} vs oracle, {rel0:.2e} vs unsplit")
        assert rel <= GRAD_TOL, (k, rel)
        assert rel0 <= 2e-5, (k, rel0)


def test_render_bwd_stage_and_accumulate(api):
    """Backward on identical fp32 screen-space inputs; accumulate adds."""
    w = S.ring()
    cam, prm = w.cams[1], w.params
    scene = S.subset(w.scene, w.cell_of == w.active)
    say("render_bwd stage ring cam1", scene["means"].shape)
    r = S.rng(43)
    F, B = S.background_pair(r, cam.height, cam.width)
    G = S.upstream_grad(r, cam.height, cam.width)
    ob, proj = _oracle_inputs_f32(cam, prm, scene)
    _, values, ranges = O.bin(cam.width, cam.height, ob["depth"], ob["rect"], ob["tiles_touched"])
    args = (proj["means2d"].astype(np.float64), _conic_of(proj["conic_opacity"]),
            proj["conic_opacity"][:, 3].astype(np.float64), proj["rgb"].astype(np.float64))
    ref = O.render_fwd(cam, prm, ranges, values, *args, F, B, rel_margin=KNIFE)
    G = G * (~ref["knife"])[..., None]
    g2d = O.render_bwd_2d(cam, prm, ranges, values, *args, F, B, G.astype(np.float64))
    pd = to_dev(proj)
    params = to_dev(scene)
    bins = api.bin_sort(cam.width, cam.height, pd)
    Fd, Bd = torch.from_numpy(F).to(dev()), torch.from_numpy(B).to(dev())
    fw = api.render_fwd(cam, prm, bins, pd, F=Fd, B=Bd)
    Gd = torch.from_numpy(G).to(dev())
    grads = api.render_bwd(cam, prm, params, pd, bins, fw, Gd, F=Fd, B=Bd, want_means2d=True)
    torch.cuda.synchronize()
    rel = np.linalg.norm(np32(grads["means2d"]) - g2d[:, :2]) / np.linalg.norm(g2d[:, :2])
    assert rel <= GRAD_TOL
    before = {k: v.clone() for k, v in grads.items()}
    api.render_bwd(cam, prm, params, pd, bins, fw, Gd, F=Fd, B=Bd, grads=grads, accumulate=True)
    torch.cuda.synchronize()
    for k in before:
        assert torch.allclose(grads[k], 2 * before[k], rtol=1e-5, atol=1e-6 * before[k].abs().max().item())


def test_frozen_split_matches_joint_on_gpu(api):
    """The paper's equivalence (Method section) on the GPU path: the active slab
    rendered between F and B (rendered by the GPU from the front and back
    slabs) equals the joint render of all slabs, with t_min = 0."""
    rr = S.rng(50)
    cam = look_at((0.4, -3.2, 1.2), (0, 0, 0), 96, 80)
    prm = RasterParams(sh_degree=1, t_min=0.0)
    sc = S.gaussians(rr, rr.uniform(-1, 1, (2000, 3)), 1, math.log(0.08), 0.4)
    Rc = np.asarray(cam.R, np.float64)
    z = sc["means"].astype(np.float64) @ Rc[2] + cam.t[2]
    lab = np.searchsorted(np.quantile(z, [1 / 3, 2 / 3]), z)
    say("split vs joint", sc["means"].shape)

    def render(s, F=None, B=None):
        p = api.project(cam, prm, **to_dev(s))
        b = api.bin_sort(cam.width, cam.height, p)
        return api.render_fwd(cam, prm, b, p, F=F, B=B)["out"]

    joint = render(sc)
    F = render(S.subset(sc, lab == 0))
    B = render(S.subset(sc, lab == 2))
    split = render(S.subset(sc, lab == 1), F=F, B=B)
    torch.cuda.synchronize()
    assert (split - joint).abs().max().item() < 2e-5


@pytest.mark.parametrize("k,n_front,hw,acc", [(7, 3, (128, 128), False), (63, 20, (64, 96), False),
                                              (63, 63, (33, 17), False), (5, 0, (31, 31), True),
                                              (500, 211, (16, 24), False), (0, 0, (16, 16), False),
                                              (0, 0, (16, 16), True)])
def test_composite_cache(api, k, n_front, hw, acc):
    H, W = hw
    say("composite", k, n_front, hw, acc)
    r = S.rng(60 + k)
    imgs = S.half_bits(S.premultiplied_images(r, k, H, W, coverage=0.6)) if k else \
        np.zeros((0, H, W, 4), np.uint16)
    order = list(r.permutation(k))
    F0 = B0 = None
    if acc:
        F0, B0 = S.background_pair(r, H, W)
    Fo, Bo = O.composite(W, H, imgs, order, n_front, F=F0, B=B0)
    Fd = torch.from_numpy(F0).to(dev()) if acc else None
    Bd = torch.from_numpy(B0).to(dev()) if acc else None
    if k == 0 and not acc:  # k = 0 must overwrite with transparent
        Fd = torch.full((H, W, 4), 7.0, device=dev())
        Bd = torch.full((H, W, 4), 7.0, device=dev())
    img_d = torch.from_numpy(imgs.view(np.int16)).to(dev())
    Fg, Bg = api.composite_cache(img_d, order, n_front, F=Fd, B=Bd, accumulate=acc)
    torch.cuda.synchronize()
    assert np.abs(np32(Fg) - Fo).max() <= FWD_TOL
    assert np.abs(np32(Bg) - Bo).max() <= FWD_TOL


def test_composite_cache_worked_by_hand(api, over_by_hand):
    """The collapse kernel on the hand-worked cases (dyadic values, exact in
    fp32): every split into F and B gives F over B == the hand result."""
    for name, lay, res in over_by_hand:
        k = len(lay)
        say("composite by hand", name, k)
        imgs = S.half_bits(np.broadcast_to(lay.reshape(k, 1, 1, 4), (k, 3, 5, 4)).copy())
        img_d = torch.from_numpy(imgs.view(np.int16)).to(dev())
        for n in range(k + 1):
            Fg, Bg = api.composite_cache(img_d, list(range(k)), n)
            torch.cuda.synchronize()
            F, B = np32(Fg).astype(np.float64), np32(Bg).astype(np.float64)
            got = F + (1.0 - F[..., 3:4]) * B
            assert np.array_equal(got, np.broadcast_to(res, got.shape)), (name, n)


def test_edge_cases_empty_block_and_culled(api):
    w = S.tiny()
    cam, prm = w.cams[0], w.params
    r = S.rng(70)
    F, B = S.background_pair(r, cam.height, cam.width)
    Fd, Bd = torch.from_numpy(F).to(dev()), torch.from_numpy(B).to(dev())
    say("empty block")
    empty = S.subset(w.scene, np.zeros(len(w.scene["means"]), bool))
    params = to_dev(empty)
    p = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, p)
    fw = api.render_fwd(cam, prm, bins, p, F=Fd, B=Bd)
    torch.cuda.synchronize()
    assert bins["n_isect"] == 0
    assert np.array_equal(np32(bins["tile_order"]), np.arange(api.n_tiles(cam.width, cam.height)))
    exp = F.astype(np.float64) + (1 - F[..., 3:]) * B
    assert np.abs(np32(fw["out"]) - exp).max() <= FWD_TOL
    say("all culled (behind the camera)")
    behind = dict(w.scene)
    behind = {k: v[:100].copy() for k, v in behind.items()}
    behind["means"] = (np.asarray(cam.campos)[None] * 2.0 + 0.0 * behind["means"]).astype(np.float32)
    params = to_dev(behind)
    p = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, p)
    fw = api.render_fwd(cam, prm, bins, p, F=Fd, B=Bd)
    G = torch.from_numpy(S.upstream_grad(r, cam.height, cam.width)).to(dev())
    grads = api.render_bwd(cam, prm, params, p, bins, fw, G, F=Fd, B=Bd)
    torch.cuda.synchronize()
    assert bins["n_isect"] == 0 and int(p["tiles_touched"].sum()) == 0
    assert np.array_equal(np32(bins["tile_order"]), np.arange(api.n_tiles(cam.width, cam.height)))
    for v in grads.values():
        assert not torch.any(v != 0)
    say("all culled, general binning (more Gaussians than the one-workgroup sort takes)")
    many = {k: np.concatenate([v] * 30) for k, v in behind.items()}  # 3,000
    p = api.project(cam, prm, **to_dev(many))
    bins = api.bin_sort(cam.width, cam.height, p)
    torch.cuda.synchronize()
    assert bins["n_isect"] == 0
    assert torch.all(bins["tile_ranges"] == 0)
    assert np.array_equal(np32(bins["tile_order"]), np.arange(api.n_tiles(cam.width, cam.height)))


def test_capacity_overflow_writes_empty_ranges_only(api):
    """On overflow the lists are not written, every tile range is empty and
    the tile order is the identity, so the blend kernels read no entry."""
    from paper_2608_27735_amd._lib import AbcdError
    w = S.tiny()
    cam, prm = w.cams[0], w.params
    say("capacity overflow")
    p = api.project(cam, prm, **to_dev(w.scene))
    full = api.bin_sort(cam.width, cam.height, p)
    m = full["n_isect"]
    values = torch.full((m - 1,), -7, dtype=torch.int32, device=dev())
    ranges = torch.full_like(full["tile_ranges"], -7)
    order = torch.full_like(full["tile_order"], -7)
    with pytest.raises(AbcdError) as e:
        _raw_bin(api, cam, p, m - 1, values, ranges, order)
    assert e.value.status == 2
    torch.cuda.synchronize()
    assert torch.all(values == -7)
    assert torch.all(ranges == 0)
    assert np.array_equal(np32(order), np.arange(api.n_tiles(cam.width, cam.height)))


def test_step_overflow_is_flagged_and_renders_no_stale_list(api):
    """A step whose intersections outgrow the capacity it was sized for (no
    synchronisation inside the step) renders the active block as empty, not
    the previous call's lists, and overflowed() reports it."""
    from paper_2608_27735_amd.step import ActiveBlockStep
    w = S.tiny()
    cam, prm = w.cams[0], w.params
    act = S.subset(w.scene, w.cell_of == w.active)
    r = S.rng(71)
    F, B = S.background_pair(r, cam.height, cam.width)
    Fd, Bd = torch.from_numpy(F).to(dev()), torch.from_numpy(B).to(dev())
    params = to_dev(act)
    say("step overflow", len(act["means"]))
    st = ActiveBlockStep(cam, prm, params, headroom=1.0)  # capacity = M + 1024
    st.project_and_bin(sync=False)
    st.forward(Fd, Bd)
    torch.cuda.synchronize()
    assert not st.overflowed()
    assert int(st.n_blends.item()) > 0
    # grow every Gaussian 8x: many more intersections than the capacity
    params["log_scales"] += math.log(8.0)
    st.n_blends.zero_()
    target = torch.from_numpy(w.target).to(dev())
    grads = st.step(target, F=Fd, B=Bd)
    torch.cuda.synchronize()
    assert st.overflowed()
    assert int(st.n_blends.item()) == 0
    assert torch.all(st.tile_ranges == 0)
    exp = F.astype(np.float64) + (1 - F[..., 3:]) * B
    assert np.abs(np32(st.fwd["out"]) - exp).max() <= FWD_TOL
    for v in grads.values():
        assert not torch.any(v != 0)


def _raw_bin(api, cam, p, capacity, values, ranges, order):
    """bin_sort without the binding's automatic regrow."""
    import ctypes as C
    from paper_2608_27735_amd import _lib
    n = p["means2d"].shape[0]
    ws = torch.empty(api.bin_sort_workspace_size(n, cam.width, cam.height, capacity),
                     dtype=torch.uint8, device=dev())
    m = C.c_int64(0)
    st = _lib.load().abcd_bin_sort(cam.width, cam.height, n, p["means2d"].data_ptr(),
                                   p["extent"].data_ptr(), p["depth"].data_ptr(),
                                   p["tiles_touched"].data_ptr(), capacity, ws.data_ptr(),
                                   ws.numel(), None, values.data_ptr(), ranges.data_ptr(),
                                   order.data_ptr(), C.byref(m),
                                   torch.cuda.current_stream().cuda_stream)
    _lib.check(st)


@pytest.mark.parametrize("H,W", [(40, 56), (97, 131), (2100, 2048)])
def test_loss_l1_gradient(api, H, W):
    """Small, ragged, and past one launch's pass (4096 x 1024 pixels)."""
    r = S.rng(80)
    say("loss l1", H, W)
    out = np.concatenate([r.uniform(0, 1, (H, W, 3)), r.uniform(0, 1, (H, W, 1))], -1).astype(np.float32)
    tgt = r.uniform(0, 1, (H, W, 3)).astype(np.float32)
    bg = (0.2, 0.5, 0.9)
    loss = torch.zeros(1, device=dev())
    g = api.loss_l1_grad(torch.from_numpy(out).to(dev()), torch.from_numpy(tgt).to(dev()), bg=bg,
                         loss=loss)
    torch.cuda.synchronize()
    # the sign decision is taken on the fp32 image, as the kernel takes it
    img = out[..., :3] + (1 - out[..., 3:]) * np.array(bg, np.float32)
    ref_L, ref_g = O.loss_l1(out, tgt, bg=bg)
    s = np.sign(img - tgt) / (3 * H * W)
    exp = np.concatenate([s, -(s * np.array(bg)).sum(-1, keepdims=True)], -1)
    flip = np.sign(img - tgt) != np.sign(out[..., :3].astype(np.float64) + (1 - out[..., 3:].astype(np.float64)) * np.array(bg) - tgt)
    assert np.abs(np32(g) - exp).max() < 1e-9
    assert np.abs(np32(g)[~flip.any(-1)] - ref_g[~flip.any(-1)]).max() < 1e-9
    assert abs(loss.item() - ref_L) < 1e-5


def test_adam_step_matches_oracle(api):
    """Three Adam steps on the five parameter groups of 1003 Gaussians plus an
    unaligned group (scalar path), stage by stage against the fp64 oracle on the
    GPU's own fp32 state. Bar: fp32 evaluation of the formulas, with the
    rounding measured on the magnitudes of the terms (m = b1 m + (1 - b1) g can
    cancel): each moment within 3e-7 of the sum of its terms' magnitudes, theta
    within 4e-7 |theta| + 2e-6 (|update| + the same bound carried through the
    moment)."""
    r = S.rng(90)
    n = 1003
    shapes = dict(means=(n, 3), log_scales=(n, 3), quats=(n, 4), opacity_logits=(n,),
                  sh=(n, 16, 3), odd=(1001,))
    lr = dict(means=1.6e-4, log_scales=5e-3, quats=1e-3, opacity_logits=5e-2, sh=2.5e-3, odd=1e-2)
    say("adam", n)

    def mk(shape, scale=1.0):
        return torch.from_numpy((scale * r.normal(size=shape)).astype(np.float32)).to(dev())

    buf = {k: mk((int(np.prod(s)) + 1,)) for k, s in shapes.items()}
    # the odd group lives one float past a 16-byte boundary
    th = {k: (buf[k][1:] if k == "odd" else buf[k][:-1]).view(*shapes[k]) for k in shapes}
    m = {k: torch.zeros_like(th[k]) for k in shapes}
    v = {k: torch.zeros_like(th[k]) for k in shapes}
    for t in (1, 2, 3):
        g = {k: mk(shapes[k], 10.0 ** r.uniform(-4, 1)) for k in shapes}
        before = {k: (th[k].cpu().numpy().astype(np.float64), m[k].cpu().numpy().astype(np.float64),
                      v[k].cpu().numpy().astype(np.float64)) for k in shapes}
        api.adam_step(th, g, m, v, lr, t, beta1=0.9, beta2=0.999, eps=1e-15)
        torch.cuda.synchronize()
        for k in shapes:
            t0, m0, v0 = before[k]
            # the hyperparameters the kernel receives are fp32
            f32 = lambda x: float(np.float32(x))
            rt, rm, rv = O.adam(t0, g[k].cpu().numpy(), m0, v0, f32(lr[k]), f32(0.9), f32(0.999),
                                f32(1e-15), t)
            gk = g[k].cpu().numpy().astype(np.float64).ravel()
            mterm = f32(0.9) * np.abs(m0.ravel()) + (1 - f32(0.9)) * np.abs(gk)
            vterm = f32(0.999) * v0.ravel() + (1 - f32(0.999)) * gk * gk
            gm = m[k].cpu().numpy().astype(np.float64).ravel()
            gv = v[k].cpu().numpy().astype(np.float64).ravel()
            assert np.all(np.abs(gm - rm) <= 3e-7 * mterm), (k, t)
            assert np.all(np.abs(gv - rv) <= 3e-7 * vterm), (k, t)
            lr_t = f32(lr[k]) / (1 - f32(0.9) ** t)
            denom = np.sqrt(rv / (1 - f32(0.999) ** t)) + f32(1e-15)
            scale = np.abs(rt - t0.ravel()) + lr_t * mterm / denom
            gt = th[k].cpu().numpy().astype(np.float64).ravel()
            assert np.all(np.abs(gt - rt) <= 4e-7 * np.abs(rt) + 2e-6 * scale), (k, t)


def test_step_graph_replays_match_eager(api):
    """The step captured as a HIP graph: four replays, each after eager work
    that rewrites the parameters, F and B in place (and a synchronisation),
    each checked against an eager step on the same inputs."""
    from paper_2608_27735_amd.step import ActiveBlockStep
    r = S.ring()
    cam, prm = r.cams[2], r.params
    scene = S.subset(r.scene, r.cell_of == r.active)
    say("graph replay", scene["means"].shape)
    rr = S.rng(91)
    params = to_dev(scene)
    F0, B0 = S.background_pair(rr, cam.height, cam.width)
    F, B = torch.from_numpy(F0).to(dev()), torch.from_numpy(B0).to(dev())
    target = torch.from_numpy(rr.uniform(0, 1, (cam.height, cam.width, 3)).astype(np.float32)).to(dev())
    g_step = ActiveBlockStep(cam, prm, params)
    e_params = {k: v.clone() for k, v in params.items()}
    e_step = ActiveBlockStep(cam, prm, e_params, capacity=g_step.capacity)
    g_step.capture(target, F=F, B=B)
    torch.cuda.synchronize()
    for rep in range(4):
        # eager work between replays: new parameters and F/B, same for both steps
        with torch.no_grad():
            params["means"].add_(0.01 * torch.randn_like(params["means"]))
            params["opacity_logits"].mul_(0.9)
            F.mul_(0.95)
            B.mul_(0.97)
            for k in params:
                e_params[k].copy_(params[k])
        torch.cuda.synchronize()
        gg = g_step.replay()
        torch.cuda.synchronize()
        eg = e_step.step(target, F=F, B=B)
        torch.cuda.synchronize()
        assert torch.equal(g_step.fwd["out"], e_step.fwd["out"]), rep
        assert torch.equal(g_step.fwd["last"], e_step.fwd["last"]), rep
        assert torch.equal(g_step.values[:g_step.tile_ranges[-1, 1]],
                           e_step.values[:e_step.tile_ranges[-1, 1]]), rep
        for k in ("means", "log_scales", "quats", "opacity_logits", "sh"):
            rel = (torch.linalg.norm((gg[k] - eg[k]).double()) /
                   torch.linalg.norm(eg[k].double()).clamp_min(1e-30)).item()
            assert rel <= 1e-5, (rep, k, rel)  # same kernels; atomics order differs


def test_step_collapse_beside_binning(api):
    """The F/B collapse enqueued on a second stream beside projection and
    binning (step(collapse=...)) gives the step of the collapse run first,
    eagerly and as a replayed graph with the fork and join captured, across
    parameter and cache changes between steps."""
    from paper_2608_27735_amd.step import ActiveBlockStep
    r = S.ring()
    cam, prm = r.cams[2], r.params
    scene = S.subset(r.scene, r.cell_of == r.active)
    rr = S.rng(92)
    k, n_front = 9, 4
    imgs = torch.from_numpy(S.half_bits(S.premultiplied_images(rr, k, cam.height, cam.width,
                                                               coverage=0.6)).view(np.int16)).to(dev())
    order = list(rr.permutation(k))
    target = torch.from_numpy(rr.uniform(0, 1, (cam.height, cam.width, 3)).astype(np.float32)).to(dev())
    say("collapse beside binning", scene["means"].shape, k)
    params = to_dev(scene)
    probe = ActiveBlockStep(cam, prm, params)
    steps, FB = [], []
    for _ in range(3):  # sequential, overlapped eager, overlapped graph
        p = {kk: v.clone() for kk, v in params.items()}
        steps.append((ActiveBlockStep(cam, prm, p, capacity=2 * probe.capacity), p))
        FB.append((torch.empty((cam.height, cam.width, 4), device=dev()),
                   torch.empty((cam.height, cam.width, 4), device=dev())))

    def collapse(i):  # the overlapped ones on a bounded grid (same arithmetic per pixel)
        return lambda: api.composite_cache(imgs, order, n_front, F=FB[i][0], B=FB[i][1],
                                           beside=i > 0)

    steps[2][0].capture(target, F=FB[2][0], B=FB[2][1], before=collapse(2))
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.no_grad():
            for _, p in steps:
                p["means"].add_(0.003 * (rep + 1))
            if rep == 1:
                imgs.copy_(imgs.flip(0))
        torch.cuda.synchronize()
        collapse(0)()
        g0 = steps[0][0].step(target, F=FB[0][0], B=FB[0][1])
        g1 = steps[1][0].step(target, F=FB[1][0], B=FB[1][1], collapse=collapse(1))
        g2 = steps[2][0].replay()
        torch.cuda.synchronize()
        assert not any(s.overflowed() for s, _ in steps)
        for i in (1, 2):
            assert torch.equal(FB[i][0], FB[0][0]) and torch.equal(FB[i][1], FB[0][1]), (rep, i)
            assert torch.equal(steps[i][0].fwd["out"], steps[0][0].fwd["out"]), (rep, i)
            gi = (g1, g2)[i - 1]
            for kk in ("means", "log_scales", "quats", "opacity_logits", "sh"):
                rel = (torch.linalg.norm((gi[kk] - g0[kk]).double()) /
                       torch.linalg.norm(g0[kk].double()).clamp_min(1e-30)).item()
                assert rel <= 1e-5, (rep, i, kk, rel)  # same kernels; atomics order differs

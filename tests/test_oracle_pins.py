"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check uses an independent
route (closed forms, a library routine, quadrature, brute force, finite
differences, or the paper's own premise that "over" is associative so frozen
partitions collapse into F and B -- Abstract and Method section).
"""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

from oracle import oracle as O
from paper_2608_27735_amd import synthetic as S
from paper_2608_27735_amd.camera import Camera, RasterParams, look_at


def axis_camera(width=64, height=48, f=50.0):
    """Camera at the origin looking down +z (R = I, t = 0)."""
    return Camera(width=width, height=height, fx=f, fy=f, cx=width / 2, cy=height / 2,
                  R=np.eye(3, dtype=np.float32), t=np.zeros(3, np.float32),
                  campos=np.zeros(3, np.float32), near=0.2)


def scene_in_front(r, n, cam, sh_degree=0, depth=(2.0, 6.0), logscale=(math.log(0.15), 0.3),
                   spread=0.8):
    """n Gaussians in view of `cam` (means on rays through the image)."""
    z = r.uniform(*depth, n)
    px = r.uniform(0.1 * cam.width, 0.9 * cam.width, n)
    py = r.uniform(0.1 * cam.height, 0.9 * cam.height, n)
    xc = (px - cam.cx) / cam.fx * z
    yc = (py - cam.cy) / cam.fy * z
    pc = np.stack([xc, yc, z], 1)
    R = np.asarray(cam.R, np.float64)
    t = np.asarray(cam.t, np.float64)
    means = (pc - t) @ R  # world = R^T (cam - t)
    return S.gaussians(r, means, sh_degree, logscale[0], logscale[1])


# --------------------------------------------------------------- binary16

def test_half_decode_matches_numpy_all_patterns():
    bits = np.arange(65536, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([O.half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ------------------------------------------------------ spherical harmonics

def _sphere_quadrature(nz=24, nphi=48):
    z, wz = np.polynomial.legendre.leggauss(nz)
    phi = 2 * np.pi * np.arange(nphi) / nphi
    for zi, wi in zip(z, wz):
        s = math.sqrt(1 - zi * zi)
        for p in phi:
            yield np.array([s * math.cos(p), s * math.sin(p), zi]), wi * 2 * np.pi / nphi


def test_sh_basis_is_orthonormal_by_quadrature():
    G = np.zeros((16, 16))
    for d, w in _sphere_quadrature():
        y, _ = O.sh_basis(d)
        G += w * np.outer(y, y)
    assert np.allclose(G, np.eye(16), atol=1e-12)


def test_sh_degree_one_is_linear_in_y_z_x():
    r = S.rng(3)
    for _ in range(10):
        d = r.normal(size=3)
        d /= np.linalg.norm(d)
        y, _ = O.sh_basis(d)
        ratio = y[1:4] / d[[1, 2, 0]]
        assert np.allclose(ratio, ratio[0], rtol=1e-14)
        assert ratio[0] > 0


def test_sh_gradient_matches_finite_differences():
    r = S.rng(4)
    h = 1e-6
    for _ in range(8):
        d = r.normal(size=3)
        _, g = O.sh_basis(d)
        for k in range(3):
            e = np.zeros(3)
            e[k] = h
            fd = (O.sh_basis(d + e)[0] - O.sh_basis(d - e)[0]) / (2 * h)
            assert np.allclose(g[:, k], fd, atol=1e-8)


# ---------------------------------------------------------------- rotation

def test_quaternion_rotation_matches_scipy_and_is_proper():
    r = S.rng(5)
    for _ in range(20):
        q = r.normal(size=4)
        q /= np.linalg.norm(q)
        R = O.quat_to_rot(q)
        ref = Rotation.from_quat([q[1], q[2], q[3], q[0]]).as_matrix()  # scalar-last
        assert np.allclose(R, ref, atol=1e-14)
        assert np.allclose(R @ R.T, np.eye(3), atol=1e-14)
        assert abs(np.linalg.det(R) - 1) < 1e-13
        assert np.allclose(O.quat_to_rot(-q), R, atol=1e-15)


# -------------------------------------------------------------- projection

def _single(means, ls, q, op=0.0, sh=None, degree=0):
    means = np.asarray(means, np.float32).reshape(-1, 3)
    n = means.shape[0]
    nc = (degree + 1) ** 2
    return dict(means=means, log_scales=np.asarray(ls, np.float32).reshape(n, 3),
                quats=np.asarray(q, np.float32).reshape(n, 4),
                opacity_logits=np.full(n, op, np.float32),
                sh=np.zeros((n, nc, 3), np.float32) if sh is None else np.asarray(sh, np.float32))


def test_isotropic_gaussian_on_axis_closed_form():
    cam = axis_camera(64, 64, f=40.0)
    prm = RasterParams()
    for z, sig in [(2.0, 0.05), (3.5, 0.2), (5.0, 0.5)]:
        sc = _single([0, 0, z], [math.log(sig)] * 3, [1, 0, 0, 0])
        pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
        pv = O.project_values(cam, prm, **{k: sc[k] for k in ("means", "log_scales", "quats",
                                                                "opacity_logits", "sh")},
                              tiles_touched=pb["tiles_touched"])
        s32 = math.exp(float(np.float32(math.log(sig))))  # parameters are stored in fp32
        var = (cam.fx * s32 / z) ** 2 + float(np.float32(prm.eps2d))
        assert np.allclose(pv["conic"][0], [1 / var, 0, 1 / var], rtol=1e-12, atol=1e-15)
        assert np.allclose(pv["means2d"][0], [cam.cx, cam.cy], rtol=1e-14)
        assert abs(pb["radius"][0] - 3 * math.sqrt(var)) <= 2e-6 * 3 * math.sqrt(var)
        assert pb["depth"][0] == np.float32(z)
        assert abs(pv["opacity"][0] - 0.5) < 1e-15


def _perspective(cam, tcam):
    return np.array([cam.fx * tcam[0] / tcam[2] + cam.cx, cam.fy * tcam[1] / tcam[2] + cam.cy])


def _numeric_jacobian(cam, tcam, h=1e-6):
    J = np.zeros((2, 3))
    for k in range(3):
        e = np.zeros(3)
        e[k] = h * max(1.0, abs(tcam[k]))
        J[:, k] = (_perspective(cam, tcam + e) - _perspective(cam, tcam - e)) / (2 * e[k])
    return J


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ewa_covariance_matches_numeric_jacobian_and_scipy(seed):
    """Sigma' = J W Sigma W^T J^T + eps I with J the derivative of the pinhole
    map (evaluated at the guard-band-clamped point) and Sigma = R diag(s^2) R^T."""
    r = S.rng(100 + seed)
    cam = look_at((3.0, -2.0, 1.5), (0, 0, 0), 96, 64)
    prm = RasterParams(sh_degree=0)
    sc = S.gaussians(r, r.uniform(-1.5, 1.5, (40, 3)), 0, math.log(0.1), 0.5)
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
    pv = O.project_values(cam, prm, **sc, tiles_touched=pb["tiles_touched"])
    Rc = np.asarray(cam.R, np.float64)
    tc = np.asarray(cam.t, np.float64)
    g32 = float(np.float32(prm.guard))
    lim = np.array([g32 * 0.5 * cam.width / cam.fx, g32 * 0.5 * cam.height / cam.fy])
    checked = 0
    for i in range(40):
        if pb["tiles_touched"][i] == 0:
            continue
        t = Rc @ sc["means"][i].astype(np.float64) + tc
        ratio = t[:2] / t[2]
        tclamped = np.array([*(np.clip(ratio, -lim, lim) * t[2]), t[2]])
        J = _numeric_jacobian(cam, tclamped)
        q = sc["quats"][i].astype(np.float64)
        Rq = Rotation.from_quat([q[1], q[2], q[3], q[0]]).as_matrix()
        s = np.exp(sc["log_scales"][i].astype(np.float64))
        Sig = Rq @ np.diag(s * s) @ Rq.T
        Sp = J @ Rc @ Sig @ Rc.T @ J.T + float(np.float32(prm.eps2d)) * np.eye(2)
        a, b, c = pv["conic"][i]
        Q = np.array([[a, b], [b, c]])
        assert np.allclose(Q @ Sp, np.eye(2), atol=1e-6), i
        assert np.allclose(pv["means2d"][i], _perspective(cam, t), rtol=1e-12)
        # fp32 chain agrees with the fp64 values to fp32 accuracy
        assert np.allclose(pb["means2d"][i], pv["means2d"][i], rtol=2e-6, atol=1e-4)
        lmax = np.linalg.eigvalsh(Sp).max()
        assert abs(pb["radius"][i] - 3 * math.sqrt(lmax)) <= 1e-4 * 3 * math.sqrt(lmax)
        checked += 1
    assert checked >= 10


def test_guard_band_clamp_is_active_off_screen():
    """A Gaussian far right of the frame: its Jacobian uses the clamped ratio."""
    cam = axis_camera(64, 64, f=40.0)
    prm = RasterParams(guard=1.3)
    lim = float(np.float32(prm.guard)) * 0.5 * cam.width / cam.fx
    z = 4.0
    x = 1.8 * lim * z  # outside the guard band, but the huge footprint reaches the frame
    sig = 3.0
    sc = _single([x, 0.0, z], [math.log(sig)] * 3, [1, 0, 0, 0])
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
    assert pb["tiles_touched"][0] > 0
    pv = O.project_values(cam, prm, **sc, tiles_touched=pb["tiles_touched"])
    J = _numeric_jacobian(cam, np.array([lim * z, 0.0, z]))
    s32 = math.exp(float(np.float32(math.log(sig))))
    Sp = J @ (s32 * s32 * np.eye(3)) @ J.T + float(np.float32(prm.eps2d)) * np.eye(2)
    a, b, c = pv["conic"][0]
    assert np.allclose(np.array([[a, b], [b, c]]) @ Sp, np.eye(2), atol=1e-9)
    # the fp32 chain clamps the same way: its radius is 3 sqrt(lambda_max(Sigma'))
    lmax = np.linalg.eigvalsh(Sp).max()
    assert abs(pb["radius"][0] - 3 * math.sqrt(lmax)) <= 1e-5 * 3 * math.sqrt(lmax)


def test_culling_cases():
    cam = axis_camera()
    prm = RasterParams()
    sc = _single([[0, 0, 0.1],          # in front of the camera but before the near plane
                  [0, 0, -3.0],         # behind the camera
                  [0, 0, 3.0],          # zero quaternion
                  [np.nan, 0, 3.0],     # non-finite mean
                  [500.0, 0, 3.0],      # far outside the frame
                  [0, 0, 3.0]],         # visible
                 [[math.log(0.1)] * 3] * 6,
                 [[1, 0, 0, 0], [1, 0, 0, 0], [0, 0, 0, 0], [1, 0, 0, 0], [1, 0, 0, 0], [1, 0, 0, 0]])
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
    assert list(pb["tiles_touched"]) [:5] == [0, 0, 0, 0, 0]
    assert pb["tiles_touched"][5] > 0
    for k in ("means2d", "depth", "radius", "rect"):
        assert not np.any(pb[k][:5])


def test_tile_rectangle_is_the_overlap_of_the_binning_box():
    """tile (tx, ty) is in the rectangle iff [u-ex, u+ex] meets [16 tx, 16 tx + 16)
    and likewise in y with ey; the rectangle area is tiles_touched; the box
    lies inside the support square."""
    r = S.rng(7)
    cam = look_at((0.0, -4.0, 1.0), (0, 0, 0), 200, 120)
    prm = RasterParams()
    sc = S.gaussians(r, r.uniform(-1.5, 1.5, (400, 3)), 0, math.log(0.08), 0.6)
    sc["opacity_logits"][:100] = -4.0  # faint: alpha_min is reached well inside 3 sigma
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"], sc["opacity_logits"])
    ntx, nty = O.tile_grid(cam.width, cam.height)
    assert np.all(pb["extent"] <= pb["radius"][:, None])
    assert np.any(pb["extent"][:, 0] < pb["radius"])  # the cut does bind
    for i in np.nonzero(pb["tiles_touched"])[0]:
        u, v = pb["means2d"][i].astype(np.float64)
        ex, ey = (float(e) for e in pb["extent"][i])
        lo = np.float32(np.float32(u) - np.float32(ex)), np.float32(np.float32(v) - np.float32(ey))
        hi = np.float32(np.float32(u) + np.float32(ex)), np.float32(np.float32(v) + np.float32(ey))
        x0, y0, x1, y1 = pb["rect"][i]
        for tx in range(ntx):
            inx = float(lo[0]) < 16 * (tx + 1) and float(hi[0]) >= 16 * tx
            assert inx == (x0 <= tx <= x1), (i, tx)
        for ty in range(nty):
            iny = float(lo[1]) < 16 * (ty + 1) and float(hi[1]) >= 16 * ty
            assert iny == (y0 <= ty <= y1), (i, ty)
        assert pb["tiles_touched"][i] == (x1 - x0 + 1) * (y1 - y0 + 1)


def test_binning_box_drops_no_pixel_that_could_blend():
    """Every pixel centre of the support square outside the binning box gets
    alpha < alpha_min from the fp64 conic and opacity (so the cut changes no
    image), and for an isotropic opaque Gaussian the box is the square."""
    r = S.rng(17)
    cam = look_at((0.0, -4.0, 1.0), (0, 0, 0), 200, 120)
    prm = RasterParams()
    sc = S.gaussians(r, r.uniform(-1.0, 1.0, (300, 3)), 0, math.log(0.06), 0.8)
    sc["opacity_logits"] = r.normal(-1.0, 2.5, 300).astype(np.float32)
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"], sc["opacity_logits"])
    pv = O.project_values(cam, prm, sc["means"], sc["log_scales"], sc["quats"],
                          sc["opacity_logits"], sc["sh"], pb["tiles_touched"])
    checked = 0
    for i in np.nonzero(pb["tiles_touched"])[0]:
        u, v = pv["means2d"][i]
        a, b, c = pv["conic"][i]
        o = pv["opacity"][i]
        rad = float(pb["radius"][i])
        ex, ey = (float(e) for e in pb["extent"][i])
        xs = np.arange(math.floor(u - rad), math.ceil(u + rad) + 1) + 0.5
        ys = np.arange(math.floor(v - rad), math.ceil(v + rad) + 1) + 0.5
        X, Y = np.meshgrid(xs - u, ys - v)
        out = (np.abs(X) > ex + 1e-3) | (np.abs(Y) > ey + 1e-3)
        inside_sq = (np.abs(X) <= rad) & (np.abs(Y) <= rad)
        q = a * X * X + 2 * b * X * Y + c * Y * Y
        alpha = np.minimum(o * np.exp(-0.5 * q), prm.alpha_max)
        sel = out & inside_sq
        checked += int(sel.sum())
        assert np.all(alpha[sel] < prm.alpha_min), i
    assert checked > 1000
    # isotropic and opaque: the alpha_min ellipse reaches past 3 sigma, no cut
    iso = _single([[0, 0, 3.0]], [[math.log(0.1)] * 3], [[1, 0, 0, 0]])
    pb1 = O.project_bin(axis_camera(), prm, iso["means"], iso["log_scales"], iso["quats"],
                        np.array([4.0], np.float32))
    assert pb1["extent"][0, 0] == pb1["radius"][0] and pb1["extent"][0, 1] == pb1["radius"][0]


# ------------------------------------------------------------------ binning

def test_binning_equals_per_tile_brute_force():
    r = S.rng(8)
    cam = look_at((0.0, -4.0, 1.0), (0, 0, 0), 150, 100)
    prm = RasterParams()
    sc = S.gaussians(r, r.uniform(-1.5, 1.5, (600, 3)), 0, math.log(0.05), 0.6)
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
    keys, values, ranges = O.bin(cam.width, cam.height, pb["depth"], pb["rect"], pb["tiles_touched"])
    ntx, nty = O.tile_grid(cam.width, cam.height)
    assert len(values) == int(pb["tiles_touched"].astype(np.int64).sum())
    dbits = pb["depth"].view(np.uint32)
    pos = 0
    for t in range(ntx * nty):
        tx, ty = t % ntx, t // ntx
        rc = pb["rect"]
        inside = (pb["tiles_touched"] > 0) & (rc[:, 0] <= tx) & (tx <= rc[:, 2]) & \
                 (rc[:, 1] <= ty) & (ty <= rc[:, 3])
        idx = np.nonzero(inside)[0]
        idx = idx[np.lexsort((idx, dbits[idx]))]
        assert ranges[t, 0] == pos and ranges[t, 1] == pos + len(idx)
        assert np.array_equal(values[pos:pos + len(idx)], idx)
        assert np.all(keys[pos:pos + len(idx)] >> np.uint64(32) == t)
        assert np.array_equal((keys[pos:pos + len(idx)] & np.uint64(0xFFFFFFFF)).astype(np.uint32),
                              dbits[idx])
        pos += len(idx)


# --------------------------------------------------------------- "over"

def _imgs(r, k, h, w):
    return S.half_bits(S.premultiplied_images(r, k, h, w, coverage=0.7))


def test_over_two_layer_worked_example():
    """By hand: (0.25, 0, 0, 0.5) over (0, 0.5, 0, 0.5) = (0.25, 0.25, 0, 0.75) and
    (0, 0.5, 0, 0.5) over (0.25, 0, 0, 0.5) = (0.125, 0.5, 0, 0.75)."""
    a = np.array([0.25, 0, 0, 0.5])
    b = np.array([0, 0.5, 0, 0.5])
    imgs = S.half_bits(np.stack([a, b]).reshape(2, 1, 1, 4))
    F, B = O.composite(1, 1, imgs, [0, 1], 2)
    assert np.array_equal(F[0, 0], [0.25, 0.25, 0, 0.75])
    assert not np.any(B)
    F, B = O.composite(1, 1, imgs, [1, 0], 0)
    assert np.array_equal(B[0, 0], [0.125, 0.5, 0, 0.75])


def over_of(F, B):
    """F over B, premultiplied, per channel."""
    return F + (1.0 - F[..., 3:4]) * B


def test_over_cases_worked_by_hand(over_by_hand):
    """Every split of each hand-worked case (tests/golden/over_by_hand.txt) into
    F (the first n layers) and B (the rest) gives F over B == the hand result,
    and n = all layers leaves B transparent (Abstract; Method section)."""
    for name, lay, res in over_by_hand:
        k = len(lay)
        imgs = S.half_bits(lay.reshape(k, 1, 1, 4))
        assert np.array_equal(imgs.view(np.float16).astype(np.float64).reshape(k, 4), lay), name
        for n in range(k + 1):
            F, B = O.composite(1, 1, imgs, list(range(k)), n)
            assert np.array_equal(over_of(F, B)[0, 0], res), (name, n)
            if n == k:
                assert np.array_equal(F[0, 0], res) and not np.any(B), name
            if n == 0:
                assert np.array_equal(B[0, 0], res) and not np.any(F), name


def test_over_fold_equals_product_form():
    """alpha = 1 - prod(1 - a_k), rgb = sum_k c_k prod_{j<k}(1 - a_j)."""
    r = S.rng(9)
    imgs = _imgs(r, 6, 5, 7)
    order = [3, 0, 5, 1, 4, 2]
    F, _ = O.composite(7, 5, imgs, order, 6)
    x = imgs.view(np.float16).astype(np.float64)[order]
    trans = np.cumprod(np.concatenate([np.ones((1, 5, 7)), 1 - x[:-1, ..., 3]]), axis=0)
    rgb = (x[..., :3] * trans[..., None]).sum(0)
    alpha = 1 - np.prod(1 - x[..., 3], axis=0)
    assert np.allclose(F[..., :3], rgb, atol=1e-15)
    assert np.allclose(F[..., 3], alpha, atol=1e-15)


def test_over_associativity_chunks_identity_and_absorption():
    r = S.rng(10)
    k, h, w = 9, 6, 5
    imgs = _imgs(r, k, h, w)
    order = list(r.permutation(k))
    F_all, _ = O.composite(w, h, imgs, order, k)
    # chunked fold (a o b) o c == one-shot fold (associativity)
    for split in (1, 4, 8):
        F1, _ = O.composite(w, h, imgs, order[:split], split)
        F2, _ = O.composite(w, h, imgs, order[split:], k - split, F=F1, B=np.zeros_like(F1))
        assert np.allclose(F2, F_all, atol=1e-15)
    # F/B split: F over B equals the fold of everything
    F, B = O.composite(w, h, imgs, order, 4)
    FB, _ = O.composite(w, h, S.half_bits(B[None].astype(np.float32)), [0], 1, F=F, B=np.zeros_like(F))
    Bq = S.half_bits(B[None].astype(np.float32)).view(np.float16).astype(np.float64)[0]
    assert np.allclose(FB, F + (1 - F[..., 3:]) * Bq, atol=1e-15)
    # transparent layers are the identity
    z = np.zeros((1, h, w, 4), np.uint16)
    imgs_z = np.concatenate([imgs, z])
    F_z, _ = O.composite(w, h, imgs_z, order[:3] + [k] + order[3:], k + 1)
    assert np.array_equal(F_z, F_all)
    # an opaque front layer absorbs everything behind it
    opaque = S.half_bits(np.concatenate([r.uniform(0, 1, (1, h, w, 3)), np.ones((1, h, w, 1))], -1))
    imgs_o = np.concatenate([opaque, imgs])
    F_o, _ = O.composite(w, h, imgs_o, [0] + [i + 1 for i in order], k + 1)
    assert np.array_equal(F_o, opaque.view(np.float16).astype(np.float64)[0])
    # K = 0 gives transparent F and B
    F0, B0 = O.composite(w, h, np.zeros((0, h, w, 4), np.uint16), [], 0)
    assert not np.any(F0) and not np.any(B0)


# --------------------------------------------------------- forward render

def _splat_inputs(cam, means2d, conic, opacity, rgb, depth=None):
    """Hand-built screen-space Gaussians covering every tile."""
    n = len(opacity)
    ntx, nty = O.tile_grid(cam.width, cam.height)
    rect = np.tile(np.array([0, 0, ntx - 1, nty - 1], np.int32), (n, 1))
    depth = np.arange(1, n + 1, dtype=np.float32) if depth is None else np.asarray(depth, np.float32)
    tiles = np.full(n, ntx * nty, np.uint32)
    _, values, ranges = O.bin(cam.width, cam.height, depth, rect, tiles)
    return ranges, values, np.asarray(means2d, np.float64), np.asarray(conic, np.float64), \
        np.asarray(opacity, np.float64), np.asarray(rgb, np.float64)


def test_single_gaussian_pixels_closed_form():
    cam = axis_camera(40, 40)
    prm = RasterParams()
    var = 30.0
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [[17.3, 22.1]], [[1 / var, 0, 1 / var]],
                                                     [0.8], [[0.2, 0.5, 0.9]])
    fw = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb)
    for py in range(40):
        for px in range(40):
            d2 = (px + 0.5 - 17.3) ** 2 + (py + 0.5 - 22.1) ** 2
            a = min(0.99, 0.8 * math.exp(-0.5 * d2 / var))
            if a < 1 / 255:
                a = 0.0
            assert np.allclose(fw["out"][py, px], [0.2 * a, 0.5 * a, 0.9 * a, a], atol=1e-15)
            assert abs(fw["final_T"][py, px] - (1 - a)) < 1e-15
            assert fw["last"][py, px] == (1 if a > 0 else 0)


def test_two_nested_gaussians_closed_form_and_depth_order():
    cam = axis_camera(16, 16)
    prm = RasterParams()
    m2d = [[8.0, 8.0], [8.0, 8.0]]
    co = [[1 / 400, 0, 1 / 400], [1 / 900, 0, 1 / 900]]  # nearly flat over the tile
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, m2d, co, [0.6, 0.7],
                                                     [[1, 0, 0], [0, 1, 0]], depth=[5.0, 2.0])
    fw = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb)
    for py, px in [(0, 0), (8, 8), (15, 3)]:
        d2 = (px + 0.5 - 8) ** 2 + (py + 0.5 - 8) ** 2
        a_back = 0.6 * math.exp(-0.5 * d2 / 400)   # depth 5 -> behind
        a_front = 0.7 * math.exp(-0.5 * d2 / 900)  # depth 2 -> in front
        exp = [a_back * (1 - a_front), a_front, 0, 1 - (1 - a_front) * (1 - a_back)]
        assert np.allclose(fw["out"][py, px], exp, atol=1e-15)


def test_termination_before_transmittance_drops_below_t_min():
    """Flat layers of alpha 0.95: T = 0.05, 0.0025, 1.25e-4, then 6.25e-6 < 1e-4,
    so the fourth layer is not blended and last = 3."""
    cam = axis_camera(16, 16)
    prm = RasterParams()
    n = 6
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [[8, 8]] * n, [[0, 0, 0]] * n, [0.95] * n,
                                                     [[1, 1, 1]] * n)
    fw = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb)
    assert np.all(fw["last"] == 3)
    assert np.allclose(fw["final_T"], 0.05 ** 3, rtol=1e-14)
    assert np.allclose(fw["out"][..., 0], 1 - 0.05 ** 3, rtol=1e-14)
    assert np.allclose(fw["t_stop"], 0.05 ** 3, rtol=1e-14)
    assert fw["n_blends"] == 3 * 256


def test_alpha_clamp_and_skip_thresholds():
    cam = axis_camera(16, 16)
    prm = RasterParams()
    ranges, values, m2d, co, op, rgb = _splat_inputs(
        cam, [[8, 8], [8, 8]], [[0, 0, 0], [0, 0, 0]], [1.0, 0.003], [[1, 0, 0], [0, 1, 0]])
    fw = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb)
    # first clamps to 0.99, second (0.003 < 1/255) is skipped
    assert np.allclose(fw["out"][..., :], [0.99, 0, 0, 0.99], atol=1e-15)
    assert np.all(fw["last"] == 1)


def _fp32_alpha(px, py, mean32, conic, o):
    """Alpha at pixel (px, py) evaluated the way a fp32 rasteriser does: the
    conic's Cholesky factor rounded to fp32 and pre-scaled by sqrt(log2(e) / 2),
    offsets in fp32, q as a sum of two squares with fused multiply-adds, 2^(-q)
    rounded once, times the fp32 opacity. An emulation written here, not the
    oracle's arithmetic."""
    f = np.float32
    a, b, c = conic
    l11 = math.sqrt(a)
    l21 = b / l11
    l22 = math.sqrt(max(c - l21 * l21, 0.0))
    k = f(math.sqrt(math.log2(math.e) / 2))
    qa, qb, qc = k * f(l11), k * f(l21), k * f(l22)
    dx, dy = f(px + 0.5) - f(mean32[0]), f(py + 0.5) - f(mean32[1])

    def fma(x, y, z):
        return f(float(x) * float(y) + float(z))

    e1 = fma(qa, dx, f(qb * dy))
    e2 = f(qc * dy)
    p2 = -fma(e1, e1, f(e2 * e2))
    return f(f(o) * f(2.0 ** float(p2)))


def test_fp32_knife_margin_covers_every_fp32_alpha_decision():
    """With f32_kappa > 0 the oracle flags a pixel when an alpha decision lies
    within a bound of the fp32 evaluation's error. Splats placed so that one
    pixel sees alpha within +-1.5e-5 (relative) of alpha_min or alpha_max, with
    axis ratios up to 60:1 at every orientation and offsets of up to 200 px
    along the major axis (the cancellation the bound grows with): wherever the
    emulated fp32 decision differs from the fp64 one, the pixel is flagged,
    and the bound is not vacuous (pixels with alpha 1e-3 away from both
    thresholds are not flagged)."""
    r = S.rng(2024)
    cam = axis_camera(16, 16)
    prm = RasterParams()
    flips = flagged_flips = clear = clear_flagged = 0
    for case in range(2000):
        ang = r.uniform(0, math.pi)
        s_major = r.uniform(3.0, 120.0)
        s_minor = s_major / r.uniform(1.0, 60.0)
        cs, sn = math.cos(ang), math.sin(ang)
        Rm = np.array([[cs, -sn], [sn, cs]])
        cov = Rm @ np.diag([s_major ** 2, s_minor ** 2]) @ Rm.T
        conic = np.linalg.inv(cov)
        conic = (conic[0, 0], conic[0, 1], conic[1, 1])
        o = float(np.float32(r.uniform(0.05, 1.0)))
        near_max = case % 4 == 3
        far = case % 5 == 4
        rel = r.uniform(1e-3, 2e-3) * r.choice([-1, 1]) if far else r.uniform(-1.5e-5, 1.5e-5)
        target = (prm.alpha_max if near_max else prm.alpha_min) * (1 + rel)
        if target >= o:
            continue
        q = 2 * math.log(o / target)
        # direction: mostly along the major axis (long offsets), some at random
        th = ang + (r.normal(0, 0.02) if case % 2 else r.uniform(0, math.pi))
        u = np.array([math.cos(th), math.sin(th)])
        Q = np.array([[conic[0], conic[1]], [conic[1], conic[2]]])
        dist = math.sqrt(q / (u @ Q @ u))
        if dist > 200:
            continue
        px, py = 7, 9
        mean32 = np.array([px + 0.5, py + 0.5] - dist * u, np.float32)
        ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [mean32.astype(np.float64)], [conic],
                                                         [o], [[0.5, 0.5, 0.5]])
        fw = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb, rel_margin=2e-6,
                          f32_kappa=8.0)
        dx, dy = px + 0.5 - float(mean32[0]), py + 0.5 - float(mean32[1])
        power = -0.5 * (conic[0] * dx * dx + conic[2] * dy * dy) - conic[1] * dx * dy
        araw64 = o * math.exp(power)
        a32 = float(_fp32_alpha(px, py, mean32, conic, o))
        thr = prm.alpha_max if near_max else prm.alpha_min
        flip = (araw64 >= thr) != (a32 >= np.float32(thr))
        if flip:
            flips += 1
            flagged_flips += int(fw["knife"][py, px])
        if far:
            clear += 1
            clear_flagged += int(fw["knife"][py, px])
    assert flips >= 5, flips                       # the cases do reach the knife edge
    assert flagged_flips == flips, (flagged_flips, flips)
    assert clear >= 50 and clear_flagged == 0, (clear, clear_flagged)


def test_reductions_transparent_and_empty_and_opaque_front():
    r = S.rng(11)
    cam = look_at((0, -3.5, 1.0), (0, 0, 0), 48, 32)
    prm = RasterParams()
    sc = S.gaussians(r, r.uniform(-1, 1, (60, 3)), 0, math.log(0.1), 0.3)
    F, B = S.background_pair(r, 32, 48)
    base = O.step(cam, prm, sc)
    fb = O.step(cam, prm, sc, F=F, B=B)
    T = base["fwd"]["final_T"][..., None]
    # F = B = transparent: out = (C, 1 - T)
    assert np.allclose(base["fwd"]["out"][..., 3:], 1 - T, atol=1e-15)
    # generic: F over (C, 1-T) over B
    C = base["fwd"]["out"][..., :3]
    F64, B64 = F.astype(np.float64), B.astype(np.float64)
    exp_rgb = F64[..., :3] + (1 - F64[..., 3:]) * (C + T * B64[..., :3])
    exp_a = F64[..., 3:] + (1 - F64[..., 3:]) * (1 - T * (1 - B64[..., 3:]))
    assert np.allclose(fb["fwd"]["out"], np.concatenate([exp_rgb, exp_a], -1), atol=1e-14)
    # empty active block: out = F over B
    empty = S.subset(sc, np.zeros(60, bool))
    e = O.step(cam, prm, empty, F=F, B=B)
    assert np.allclose(e["fwd"]["out"], F64 + (1 - F64[..., 3:]) * B64, atol=1e-15)
    # opaque F hides the active block
    Fo = F.copy()
    Fo[..., 3] = 1.0
    o = O.step(cam, prm, sc, F=Fo, B=B)
    assert np.allclose(o["fwd"]["out"], Fo.astype(np.float64), atol=1e-15)


def _depth_slabs(cam, scene, n_slabs=3):
    Rc = np.asarray(cam.R, np.float64)
    z = scene["means"].astype(np.float64) @ Rc[2] + cam.t[2]
    qs = np.quantile(z, np.linspace(0, 1, n_slabs + 1)[1:-1])
    lab = np.searchsorted(qs, z)
    return lab


@pytest.mark.parametrize("t_min", [0.0, 1e-4])
def test_composited_split_equals_joint_render(t_min):
    """Paper premise (Method section): rendering the active partition between
    F and B equals rendering all partitions. Split by view depth so the
    partitions are depth-separated; with early termination the joint render
    may stop earlier, by at most its remaining transmittance."""
    r = S.rng(12)
    cam = look_at((0.4, -3.2, 1.2), (0, 0, 0), 64, 48)
    prm = RasterParams(t_min=t_min, sh_degree=1)
    sc = S.gaussians(r, r.uniform(-1, 1, (400, 3)), 1, math.log(0.12), 0.4)
    lab = _depth_slabs(cam, sc)
    joint = O.step(cam, prm, sc)
    parts = [O.step(cam, prm, S.subset(sc, lab == k)) for k in range(3)]
    F, A, B = (p["fwd"]["out"] for p in parts)
    split = O.step(cam, prm, S.subset(sc, lab == 1), F=F, B=B)["fwd"]["out"]
    diff = np.abs(split - joint["fwd"]["out"]).max(-1)
    if t_min == 0.0:
        assert diff.max() < 1e-12
    else:
        bound = joint["fwd"]["t_stop"] * 1.0 + 1e-12  # colours and alphas are <= 1 here
        assert np.all(diff <= bound)
        assert np.any(joint["fwd"]["t_stop"] > 0)


# ----------------------------------------------------------------- backward

def _loss(out, w):
    return float((out * w).sum())


def test_render_backward_2d_matches_finite_differences():
    r = S.rng(13)
    cam = axis_camera(48, 40)
    prm = RasterParams(t_min=0.0)
    sp = S.splats_2d(r, 24, 48, 40, sigma_px=(2.0, 9.0))
    sp["conic_opacity"][:, 3] = np.clip(sp["conic_opacity"][:, 3], 0.05, 0.95)
    m2d = sp["means2d"].astype(np.float64)
    co = sp["conic_opacity"][:, :3].astype(np.float64)
    op = sp["conic_opacity"][:, 3].astype(np.float64)
    rgb = sp["rgb"].astype(np.float64)
    ntx, nty = O.tile_grid(48, 40)
    rect = np.tile(np.array([0, 0, ntx - 1, nty - 1], np.int32), (24, 1))
    _, values, ranges = O.bin(48, 40, sp["depth"], rect, np.full(24, ntx * nty, np.uint32))
    F, B = S.background_pair(r, 40, 48)
    w = r.normal(size=(40, 48, 4))
    base = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb, F, B, rel_margin=1e-5)
    w[base["knife"]] = 0.0
    g2d = O.render_bwd_2d(cam, prm, ranges, values, m2d, co, op, rgb, F, B, w)

    def L(m2d_, co_, op_, rgb_):
        return _loss(O.render_fwd(cam, prm, ranges, values, m2d_, co_, op_, rgb_, F, B)["out"], w)

    h = 1e-6
    for i in range(24):
        for col, (arr, k) in enumerate([(m2d, 0), (m2d, 1), (co, 0), (co, 1), (co, 2), (op, None),
                                        (rgb, 0), (rgb, 1), (rgb, 2)]):
            hh = h * (1e-2 if arr is co else 1.0)
            ap, am = arr.copy(), arr.copy()
            if k is None:
                ap[i] += hh
                am[i] -= hh
            else:
                ap[i, k] += hh
                am[i, k] -= hh
            args_p = [m2d, co, op, rgb]
            args_m = [m2d, co, op, rgb]
            idx = {id(m2d): 0, id(co): 1, id(op): 2, id(rgb): 3}[id(arr)]
            args_p[idx], args_m[idx] = ap, am
            fd = (L(*args_p) - L(*args_m)) / (2 * hh)
            assert abs(fd - g2d[i, col]) <= 1e-6 * max(1.0, abs(fd)) + 1e-5 * abs(fd), (i, col, fd,
                                                                                          g2d[i, col])


def test_alpha_clamp_has_zero_gradient():
    """Where alpha is clamped to alpha_max, alpha does not depend on the opacity
    nor on the position; the finite difference agrees."""
    cam = axis_camera(16, 16)
    prm = RasterParams(t_min=0.0)
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [[8, 8]], [[1e-4, 0, 1e-4]], [1.0],
                                                     [[0.3, 0.6, 0.9]])
    w = np.ones((16, 16, 4))
    g2d = O.render_bwd_2d(cam, prm, ranges, values, m2d, co, op, rgb, None, None, w)
    assert g2d[0, 5] == 0.0 and g2d[0, 0] == 0.0 and g2d[0, 1] == 0.0
    opm = op - 1e-6
    Lp = _loss(O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb)["out"], w)
    Lm = _loss(O.render_fwd(cam, prm, ranges, values, m2d, co, opm, rgb)["out"], w)
    assert Lp == Lm


def _project_bwd_fd_case(seed, degree):
    r = S.rng(seed)
    cam = look_at((2.5, -2.0, 1.0), (0, 0, 0), 64, 48)
    prm = RasterParams(sh_degree=degree)
    sc = S.gaussians(r, r.uniform(-0.8, 0.8, (12, 3)), degree, math.log(0.1), 0.4, sh_hi_sd=0.3)
    # one Gaussian far to the side so the guard band clamps
    sc["means"][0] = np.array([0.2, -0.6, 3.4], np.float32)
    sc["log_scales"][0] = math.log(1.0)
    return r, cam, prm, sc


@pytest.mark.parametrize("degree", [0, 3])
def test_projection_backward_matches_finite_differences(degree):
    r, cam, prm, sc = _project_bwd_fd_case(200 + degree, degree)
    pb = O.project_bin(cam, prm, sc["means"], sc["log_scales"], sc["quats"])
    vis = pb["tiles_touched"]
    g2d = r.normal(size=(12, 9)) * (vis > 0)[:, None]
    g2d[:, 2:5] *= 100.0  # conic entries are small numbers

    def values_vec(s):
        pv = O.project_values(cam, prm, **s, tiles_touched=vis)
        return np.concatenate([pv["means2d"], pv["conic"], pv["opacity"][:, None], pv["rgb"]], 1)

    grads = O.project_bwd(cam, prm, **sc, tiles_touched=vis, g2d=g2d)
    h = 1e-5  # the step actually taken is the difference of the two fp32-rounded values
    for key in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        arr = sc[key]
        flat = arr.reshape(-1)
        for j in range(flat.size):
            sp, sm = dict(sc), dict(sc)
            xp = flat.astype(np.float64).copy()
            xm = xp.copy()
            step = h * max(1.0, abs(xp[j]))
            xp[j] += step
            xm[j] -= step
            # fp32 storage: use the exactly representable perturbed values
            vp = np.float32(xp[j])
            vm = np.float32(xm[j])
            ap = flat.copy()
            am = flat.copy()
            ap[j], am[j] = vp, vm
            sp[key], sm[key] = ap.reshape(arr.shape), am.reshape(arr.shape)
            Lp = float((values_vec(sp) * g2d).sum())
            Lm = float((values_vec(sm) * g2d).sum())
            fd = (Lp - Lm) / (float(vp) - float(vm))
            got = grads[key].reshape(-1)[j]
            assert abs(fd - got) <= 1e-5 * max(1.0, abs(fd)), (key, j, fd, got)


def _fd_scene(seed, n=16, degree=2):
    r = S.rng(seed)
    cam = look_at((0.3, -3.0, 1.0), (0, 0, 0), 40, 32)
    prm = RasterParams(sh_degree=degree, t_min=0.0)
    sc = S.gaussians(r, r.uniform(-0.7, 0.7, (n, 3)), degree, math.log(0.12), 0.3, sh_hi_sd=0.2)
    F, B = S.background_pair(r, 32, 40)
    w = r.normal(size=(32, 40, 4))
    return cam, prm, sc, F, B, w


def test_whole_step_backward_matches_finite_differences():
    """Smooth linear loss of the composited image; fp64 positions; perturbed
    entries whose binning or threshold decisions would change are skipped."""
    cam, prm, sc, F, B, w = _fd_scene(14)
    base = O.step(cam, prm, sc, F=F, B=B, dL_dout=w, pos32=False, rel_margin=1e-4)
    w = w * (~base["fwd"]["knife"])[..., None]
    base = O.step(cam, prm, sc, F=F, B=B, dL_dout=w, pos32=False)
    grads = base["grads"]
    checked = 0
    for key in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        flat = sc[key].reshape(-1)
        for j in range(0, flat.size, 3 if key == "sh" else 1):
            vals = []
            ok = True
            for sgn in (1, -1):
                a = flat.astype(np.float64).copy()
                a[j] += sgn * 1e-5 * max(1.0, abs(a[j]))
                s2 = dict(sc)
                s2[key] = a.astype(np.float32).reshape(sc[key].shape)
                res = O.step(cam, prm, s2, F=F, B=B, pos32=False, rel_margin=0)
                if not np.array_equal(res["sorted_values"], base["sorted_values"]) or \
                        not np.array_equal(res["tile_ranges"], base["tile_ranges"]):
                    ok = False
                vals.append((_loss(res["fwd"]["out"], w), float(s2[key].reshape(-1)[j])))
            if not ok:
                continue
            fd = (vals[0][0] - vals[1][0]) / (vals[0][1] - vals[1][1])
            got = grads[key].reshape(-1)[j]
            assert abs(fd - got) <= 1e-4 * max(1.0, abs(fd)), (key, j, fd, got)
            checked += 1
    assert checked > 100


def test_split_gradient_equals_joint_gradient_and_frozen_blocks_vanish():
    """Gradients of the active block through F o A o B equal those of the
    joint render restricted to the active Gaussians; the frozen Gaussians get
    no gradient from the split path by construction; opaque F zeroes them."""
    r = S.rng(15)
    cam = look_at((0.4, -3.2, 1.2), (0, 0, 0), 48, 40)
    prm = RasterParams(t_min=0.0, sh_degree=1)
    sc = S.gaussians(r, r.uniform(-1, 1, (240, 3)), 1, math.log(0.12), 0.4)
    lab = _depth_slabs(cam, sc)
    w = r.normal(size=(40, 48, 4))
    joint = O.step(cam, prm, sc, dL_dout=w)
    F = O.step(cam, prm, S.subset(sc, lab == 0))["fwd"]["out"]
    B = O.step(cam, prm, S.subset(sc, lab == 2))["fwd"]["out"]
    act = S.subset(sc, lab == 1)
    split = O.step(cam, prm, act, F=F, B=B, dL_dout=w)
    for key in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        gj = joint["grads"][key][lab == 1]
        gs = split["grads"][key]
        assert np.allclose(gs, gj, rtol=1e-9, atol=1e-12 * max(1.0, np.abs(gj).max())), key
    Fo = F.copy()
    Fo[..., 3] = 1.0
    hidden = O.step(cam, prm, act, F=Fo, B=B, dL_dout=w)
    for key in ("means", "log_scales", "quats", "opacity_logits", "sh"):
        assert not np.any(hidden["grads"][key]), key


# ------------------------------------------------------------------- Adam
# The optimizer is not named by the paper; the step follows Adam as published
# (Kingma and Ba 2015, Algorithm 1). Pins: closed forms of the bias-corrected
# moments, which a dropped bias correction, a swapped beta or a wrong sign
# would break.

def test_adam_first_step_is_normalised_gradient():
    r = np.random.default_rng(3)
    g = r.normal(size=50) * np.exp(r.uniform(-5, 5, 50))
    theta = r.normal(size=50)
    lr, eps = 0.01, 1e-8
    th, m, v = O.adam(theta, g, np.zeros(50), np.zeros(50), lr, 0.9, 0.999, eps, 1)
    # t = 1: m_hat = g and v_hat = g^2 exactly, so the step is lr g / (|g| + eps)
    assert np.allclose(th, theta - lr * g / (np.abs(g) + eps), rtol=0, atol=1e-15)
    assert np.allclose(m, 0.1 * g, rtol=1e-15) and np.allclose(v, 0.001 * g * g, rtol=1e-15)


def test_adam_constant_gradient_keeps_unit_step():
    # with a constant gradient the bias-corrected moments equal g and g^2 at
    # every step, so every step moves theta by lr g / (|g| + eps)
    g = np.array([2.0, -0.5, 1e-3, -7.0])
    theta = np.zeros(4)
    m, v = np.zeros(4), np.zeros(4)
    lr, eps = 0.1, 1e-12
    for t in range(1, 31):
        theta, m, v = O.adam(theta, g, m, v, lr, 0.9, 0.999, eps, t)
        assert np.allclose(theta, -t * lr * g / (np.abs(g) + eps), rtol=1e-12, atol=0)


def test_adam_zero_gradient_from_rest_stays():
    theta = np.array([1.0, -2.0, 3.0])
    th, m, v = O.adam(theta, np.zeros(3), np.zeros(3), np.zeros(3), 0.5, 0.9, 0.999, 1e-15, 1)
    assert np.array_equal(th, theta) and not m.any() and not v.any()


# ------------------------------------------- visibility-aware skipping (f2)

def test_fb_stop_worked_example():
    """Flat white layers of alpha 0.95 behind F with alpha 0.9 (weight 0.1 in the
    composite). T after each blend: 0.05, 0.0025, 1.25e-4. The plain rule
    blends three (1.25e-4 >= 1e-4); the compositing-aware rule weighs them by
    0.1 (5e-3, 2.5e-4, 1.25e-5) and stops before the third: last = 2,
    T = 0.0025, out = F + 0.1 (C + T B) with C = 1 - T per colour channel."""
    cam = axis_camera(16, 16)
    n = 6
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [[8, 8]] * n, [[0, 0, 0]] * n, [0.95] * n,
                                                     [[1, 1, 1]] * n)
    F = np.zeros((16, 16, 4))
    F[..., 0], F[..., 3] = 0.3, 0.9
    B = np.zeros((16, 16, 4))
    B[..., 1], B[..., 3] = 0.5, 0.5
    plain = O.render_fwd(cam, RasterParams(), ranges, values, m2d, co, op, rgb, F, B)
    assert np.all(plain["last"] == 3)
    fw = O.render_fwd(cam, RasterParams(fb_stop=True), ranges, values, m2d, co, op, rgb, F, B)
    assert np.all(fw["last"] == 2)
    T = 0.05 ** 2
    assert np.allclose(fw["final_T"], T, rtol=1e-14)
    C = 1 - T
    exp = [0.3 + 0.1 * C, 0.1 * (C + T * 0.5), 0.1 * C, 0.9 + 0.1 * (1 - T * 0.5)]
    assert np.allclose(fw["out"], exp, atol=1e-15)
    assert fw["n_blends"] == 2 * 256
    # transparent F: the weight is 1 and the rule is the plain one
    tr = O.render_fwd(cam, RasterParams(fb_stop=True), ranges, values, m2d, co, op, rgb, None, B)
    assert np.all(tr["last"] == 3)


def test_fb_stop_hidden_pixels_walk_nothing():
    """Behind an opaque F, or one that leaves less than t_min of weight, the
    compositing-aware rule blends nothing: last = 0, T = 1, out = F."""
    cam = axis_camera(16, 16)
    ranges, values, m2d, co, op, rgb = _splat_inputs(cam, [[8, 8]] * 3, [[0, 0, 0]] * 3, [0.5] * 3,
                                                     [[1, 0, 0]] * 3)
    for fa in (1.0, 1.0 - 5e-5):
        F = np.zeros((16, 16, 4))
        F[..., 2], F[..., 3] = 0.25, fa
        B = np.full((16, 16, 4), 0.5)
        fw = O.render_fwd(cam, RasterParams(fb_stop=True), ranges, values, m2d, co, op, rgb, F, B)
        assert np.all(fw["last"] == 0) and np.all(fw["final_T"] == 1.0)
        assert np.allclose(fw["out"], F + (1 - fa) * B, atol=1e-15)
        assert fw["n_blends"] == 0
    # just above the threshold the first blend still happens (0.5 * 2e-4 >= 1e-4)
    F[..., 3] = 1.0 - 2e-4
    fw = O.render_fwd(cam, RasterParams(fb_stop=True), ranges, values, m2d, co, op, rgb, F, B)
    assert np.all(fw["last"] == 1)


def test_fb_stop_backward_matches_finite_differences():
    """The backward replays the compositing-aware walk: gradients of the
    composited image agree with central differences of the forward, on a case
    where the rule ends many pixels early (F alpha 0.9 to 0.99)."""
    r = S.rng(17)
    cam = axis_camera(32, 32)
    prm = RasterParams(t_min=1e-2, fb_stop=True)
    n = 16
    sp = S.splats_2d(r, n, 32, 32, sigma_px=(3.0, 9.0))
    sp["conic_opacity"][:, 3] = np.clip(sp["conic_opacity"][:, 3], 0.3, 0.95)
    m2d = sp["means2d"].astype(np.float64)
    co = sp["conic_opacity"][:, :3].astype(np.float64)
    op = sp["conic_opacity"][:, 3].astype(np.float64)
    rgb = sp["rgb"].astype(np.float64)
    ntx, nty = O.tile_grid(32, 32)
    rect = np.tile(np.array([0, 0, ntx - 1, nty - 1], np.int32), (n, 1))
    _, values, ranges = O.bin(32, 32, sp["depth"], rect, np.full(n, ntx * nty, np.uint32))
    F = np.zeros((32, 32, 4))
    F[..., 3] = r.uniform(0.9, 0.99, (32, 32))
    F[..., :3] = F[..., 3:] * r.uniform(0, 1, (32, 32, 3))
    B = S.background_pair(r, 32, 32)[1].astype(np.float64)
    base = O.render_fwd(cam, prm, ranges, values, m2d, co, op, rgb, F, B, rel_margin=1e-3)
    plain = O.render_fwd(cam, RasterParams(t_min=1e-2), ranges, values, m2d, co, op, rgb, F, B)
    assert (base["last"] < plain["last"]).sum() > 50  # the rule bites
    w = r.normal(size=(32, 32, 4))
    w[base["knife"]] = 0.0
    g2d = O.render_bwd_2d(cam, prm, ranges, values, m2d, co, op, rgb, F, B, w)

    def L(arrs):
        return _loss(O.render_fwd(cam, prm, ranges, values, *arrs, F, B)["out"], w)

    h = 1e-7
    arrs = [m2d, co, op, rgb]
    for i in range(n):
        for col, (ai, k) in enumerate([(0, 0), (0, 1), (1, 0), (1, 1), (1, 2), (2, None),
                                       (3, 0), (3, 1), (3, 2)]):
            hh = h * (1e-2 if ai == 1 else 1.0)
            plus, minus = [a.copy() for a in arrs], [a.copy() for a in arrs]
            if k is None:
                plus[ai][i] += hh
                minus[ai][i] -= hh
            else:
                plus[ai][i, k] += hh
                minus[ai][i, k] -= hh
            fd = (L(plus) - L(minus)) / (2 * hh)
            assert abs(fd - g2d[i, col]) <= 1e-6 * max(1.0, abs(fd)) + 1e-4 * abs(fd), \
                (i, col, fd, g2d[i, col])


def test_collapse_stop_worked_example():
    """Three front layers of alpha 0.9 with stop_t = 0.05: the first two fold
    (weights 1 and 0.1), the third would get 0.01 < 0.05 and is dropped, and
    every back layer (weight 0.01 x 1) too."""
    lay = np.array([[0.9, 0, 0, 0.9], [0, 0.9, 0, 0.9], [0, 0, 0.9, 0.9], [0.2, 0.2, 0.2, 0.5]])
    imgs = S.half_bits(lay.reshape(4, 1, 1, 4))
    F, B = O.composite(1, 1, imgs, [0, 1, 2, 3], 3, stop_t=0.05)
    h = [float(np.float16(x)) for x in (0.9, 0.2, 0.5)]
    exp_F = [h[0], (1 - h[0]) * h[0], 0, h[0] + (1 - h[0]) * h[0]]
    assert np.allclose(F[0, 0], exp_F, atol=1e-15)
    assert not np.any(B)
    F0, B0 = O.composite(1, 1, imgs, [0, 1, 2, 3], 3)
    assert F0[0, 0, 2] > 0 and B0[0, 0, 3] == h[2]


def test_collapse_stop_is_chunk_invariant_and_bounded():
    """The rule looks only at what has been folded so far, so streaming the
    layers in chunks (accumulate) gives the one-pass result; and the dropped
    layers change F over B by at most 2 stop_t per channel."""
    r = S.rng(23)
    H, W, k, nf = 12, 10, 24, 14
    imgs = S.half_bits(S.premultiplied_images(r, k, H, W, alpha_max=0.9, coverage=0.8))
    order = list(r.permutation(k))
    st = 0.02
    F1, B1 = O.composite(W, H, imgs, order, nf, stop_t=st)
    Fc, Bc = O.composite(W, H, imgs, order[:9], 9, stop_t=st)
    Fc, Bc = O.composite(W, H, imgs, order[9:20], nf - 9, F=Fc, B=Bc, stop_t=st)
    Fc, Bc = O.composite(W, H, imgs, order[20:], 0, F=Fc, B=Bc, stop_t=st)
    assert np.allclose(Fc, F1, atol=1e-15) and np.allclose(Bc, B1, atol=1e-15)
    Fe, Be = O.composite(W, H, imgs, order, nf)
    over = lambda f, b: f + (1 - f[..., 3:]) * b
    d = np.abs(over(F1, B1) - over(Fe, Be))
    assert d.max() <= 2 * st
    assert d.max() > 0  # layers were dropped


# ------------------------------------------------- frustum visibility (f3)

def test_frustum_oracle_closed_cases():
    """A box around the viewed point is inside; one behind the camera, one past
    each image edge at a known depth are outside; their margins match the
    geometry."""
    cam = axis_camera(64, 48, f=50.0)  # camera at the origin looking down +z
    ok, s = O.box_meets_frustum(cam, [-0.1, -0.1, 4.9], [0.1, 0.1, 5.1])
    assert ok and s > 0
    ok, s = O.box_meets_frustum(cam, [-1, -1, -3], [1, 1, -1])
    assert not ok
    # at depth z the image spans x in [-cx z / fx, (W - cx) z / fx]
    z = 5.0
    xl = -cam.cx * z / cam.fx
    ok, _ = O.box_meets_frustum(cam, [xl - 0.5, -0.1, z], [xl - 0.05, 0.1, z])
    assert not ok
    ok, _ = O.box_meets_frustum(cam, [xl - 0.5, -0.1, z], [xl + 0.05, 0.1, z])
    assert ok
    yb = (cam.height - cam.cy) * z / cam.fy
    ok, _ = O.box_meets_frustum(cam, [-0.1, yb + 0.05, z], [0.1, yb + 0.5, z])
    assert not ok
    # between the camera and the near plane only
    ok, s = O.box_meets_frustum(cam, [-0.01, -0.01, 0.0], [0.01, 0.01, cam.near * 0.5])
    assert not ok and s < 0


def test_frustum_oracle_agrees_with_point_sampling():
    """Any sampled box point that projects into the image in front of the near
    plane proves visibility; boxes the oracle calls visible with a clear
    margin contain such points at a fine enough sampling."""
    r = S.rng(29)
    cam = look_at((3.0, -4.0, 2.0), (0.0, 0.0, 0.5), 80, 60)
    R = np.asarray(cam.R, np.float64)
    t = np.asarray(cam.t, np.float64)
    g = np.linspace(0, 1, 9)
    unit = np.stack(np.meshgrid(g, g, g, indexing="ij"), -1).reshape(-1, 3)
    for _ in range(60):
        c = r.uniform(-6, 6, 3)
        ext = r.uniform(0.05, 1.5, 3)
        lo, hi = c - ext, c + ext
        ok, s = O.box_meets_frustum(cam, lo, hi)
        p = (lo + unit * (hi - lo)) @ R.T + t
        z = p[:, 2]
        with np.errstate(divide="ignore", invalid="ignore"):
            u = cam.fx * p[:, 0] / z + cam.cx
            v = cam.fy * p[:, 1] / z + cam.cy
        hit = np.any((z >= cam.near) & (u >= 0) & (u <= cam.width) & (v >= 0) & (v <= cam.height))
        if hit:
            assert ok
        if ok and s > 0.2:
            assert hit


def test_loss_l1_worked_example_by_hand():
    """One pixel: rgb (0.5, 0.2, 0.1), a = 0.5 over bg (0, 0, 1) gives the
    image (0.5, 0.2, 0.6); against the target (0.4, 0.4, 0.5) the differences
    are (0.1, -0.2, 0.1), so L = 0.4 / 3, dL/drgb = (1, -1, 1) / 3 and
    dL/da = -(1 * 1) / 3 (only the blue background channel is non-zero)."""
    out = np.array([[[0.5, 0.2, 0.1, 0.5]]])
    tgt = np.array([[[0.4, 0.4, 0.5]]])
    L, g = O.loss_l1(out, tgt, bg=(0.0, 0.0, 1.0))
    assert abs(L - 0.4 / 3) < 1e-15
    assert np.allclose(g[0, 0], [1 / 3, -1 / 3, 1 / 3, -1 / 3], atol=1e-15)
    # a pixel that matches its target exactly has zero gradient (sign(0) = 0)
    L0, g0 = O.loss_l1(np.array([[[0.4, 0.4, 0.0, 0.5]]]), tgt, bg=(0.0, 0.0, 1.0))
    assert L0 == 0.0 and not g0.any()


def test_loss_l1_gradient_matches_finite_differences():
    """Away from the kinks (|img - target| > 1e-3 everywhere) the L1 loss is
    linear near the point, so central differences are exact up to rounding."""
    r = np.random.default_rng(12)
    h, w = 5, 7
    out = np.concatenate([r.uniform(0, 1, (h, w, 3)), r.uniform(0, 1, (h, w, 1))], -1)
    tgt = r.uniform(0, 1, (h, w, 3))
    bg = (0.3, 0.6, 0.1)
    img = out[..., :3] + (1 - out[..., 3:]) * np.array(bg)
    tgt = np.where(np.abs(img - tgt) < 1e-3, tgt + 0.01, tgt)
    _, g = O.loss_l1(out, tgt, bg=bg)
    eps = 1e-6
    for idx in [(0, 0, 0), (2, 3, 1), (4, 6, 2), (1, 5, 3), (3, 2, 3)]:
        op, om = out.copy(), out.copy()
        op[idx] += eps
        om[idx] -= eps
        fd = (O.loss_l1(op, tgt, bg)[0] - O.loss_l1(om, tgt, bg)[0]) / (2 * eps)
        assert abs(fd - g[idx]) < 1e-9, (idx, fd, g[idx])

"""numpy front end of the CPU oracle (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark use
this module. Every function forwards to the plain C oracle in abcd_oracle.c;
arrays are numpy, host memory, C-contiguous.

Camera and raster-parameter objects are duck-typed: any object with the
attributes width, height, fx, fy, cx, cy, R (3x3), t (3), campos (3), near and
alpha_min, alpha_max, t_min, eps2d, radius_sigmas, guard, sh_degree.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

TILE = 16

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_u64p = np.ctypeslib.ndpointer(np.uint64, flags="C_CONTIGUOUS")
_u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(np.uint8, flags="C_CONTIGUOUS")


class _Cam(C.Structure):
    _fields_ = [("width", C.c_int32), ("height", C.c_int32), ("fx", C.c_float),
                ("fy", C.c_float), ("cx", C.c_float), ("cy", C.c_float),
                ("R", C.c_float * 9), ("t", C.c_float * 3), ("campos", C.c_float * 3),
                ("near_plane", C.c_float)]


class _Prm(C.Structure):
    _fields_ = [("alpha_min", C.c_float), ("alpha_max", C.c_float), ("t_min", C.c_float),
                ("eps2d", C.c_float), ("radius_sigmas", C.c_float), ("guard", C.c_float),
                ("sh_degree", C.c_int32), ("fb_stop", C.c_int32)]


def _opt(ptr_type):
    """ndpointer that also accepts None (NULL)."""
    def from_param(cls, obj):
        if obj is None:
            return None
        return ptr_type.from_param(obj)
    return type("Opt" + ptr_type.__name__, (ptr_type,), {"from_param": classmethod(from_param)})


_lib = None


def lib():
    global _lib
    if _lib is not None:
        return _lib
    path = _build.LIB
    if not os.path.exists(path):
        _build.build()
    L = C.CDLL(path)
    cam_p, prm_p = C.POINTER(_Cam), C.POINTER(_Prm)
    L.orc_project_bin_f32.argtypes = [cam_p, prm_p, C.c_int64, _f32p, _f32p, _f32p, _f32p,
                                      _f32p, _f32p, _f32p, _f32p, _i32p, _u32p]
    L.orc_project_bin_f32.restype = None
    L.orc_project_values_f64.argtypes = [cam_p, prm_p, C.c_int64, _f32p, _f32p, _f32p, _f32p,
                                         _f32p, _u32p, _f64p, _f64p, _f64p, _f64p]
    L.orc_project_values_f64.restype = None
    L.orc_count_isect.argtypes = [C.c_int64, _u32p]
    L.orc_count_isect.restype = C.c_int64
    L.orc_bin.argtypes = [C.c_int32, C.c_int32, C.c_int64, _f32p, _i32p, _u32p, _u64p, _u32p,
                          _u32p]
    L.orc_bin.restype = None
    L.orc_render_fwd.argtypes = [cam_p, prm_p, _u32p, _u32p, _f64p, _f64p, _f64p, _f64p,
                                 _opt(_f64p), _opt(_f64p), _f64p, _f64p, _u32p,
                                 C.POINTER(C.c_uint64), C.c_double, C.c_double, _opt(_u8p),
                                 _opt(_f64p)]
    L.orc_render_fwd.restype = None
    L.orc_render_bwd_2d.argtypes = [cam_p, prm_p, C.c_int64, _u32p, _u32p, _f64p, _f64p, _f64p,
                                    _f64p, _opt(_f64p), _opt(_f64p), _f64p, _f64p]
    L.orc_render_bwd_2d.restype = None
    L.orc_project_bwd.argtypes = [cam_p, prm_p, C.c_int64, _f32p, _f32p, _f32p, _f32p, _f32p,
                                  _u32p, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p]
    L.orc_project_bwd.restype = None
    L.orc_composite.argtypes = [C.c_int32, C.c_int32, C.c_int32, _u16p, _i32p, C.c_int32,
                                _f64p, _f64p, C.c_int32, C.c_double, C.c_double, _u8p]
    L.orc_composite.restype = None
    L.orc_adam.argtypes = [C.c_int64, _f64p, _f64p, _f64p, _f64p, C.c_double, C.c_double,
                           C.c_double, C.c_double, C.c_int64]
    L.orc_adam.restype = None
    L.orc_half_to_double.argtypes = [C.c_uint16]
    L.orc_half_to_double.restype = C.c_double
    L.orc_sh_basis.argtypes = [_f64p, _f64p, _f64p]
    L.orc_sh_basis.restype = None
    L.orc_quat_to_rot.argtypes = [_f64p, _f64p]
    L.orc_quat_to_rot.restype = None
    _lib = L
    return L


def _cam(cam):
    c = _Cam()
    c.width, c.height = int(cam.width), int(cam.height)
    c.fx, c.fy, c.cx, c.cy = float(cam.fx), float(cam.fy), float(cam.cx), float(cam.cy)
    R = np.asarray(cam.R, dtype=np.float32).reshape(9)
    t = np.asarray(cam.t, dtype=np.float32).reshape(3)
    cp = np.asarray(cam.campos, dtype=np.float32).reshape(3)
    for i in range(9):
        c.R[i] = float(R[i])
    for i in range(3):
        c.t[i] = float(t[i])
        c.campos[i] = float(cp[i])
    c.near_plane = float(cam.near)
    return c


def _prm(p):
    q = _Prm()
    q.alpha_min, q.alpha_max, q.t_min = float(p.alpha_min), float(p.alpha_max), float(p.t_min)
    q.eps2d, q.radius_sigmas, q.guard = float(p.eps2d), float(p.radius_sigmas), float(p.guard)
    q.sh_degree = int(p.sh_degree)
    q.fb_stop = 1 if getattr(p, "fb_stop", False) else 0
    return q


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def tile_grid(width, height):
    return (width + TILE - 1) // TILE, (height + TILE - 1) // TILE


# ---------------------------------------------------------------- projection

def project_bin(cam, prm, means, log_scales, quats, opacity_logits=None):
    """fp32 chain: means2d, depth, radius (support), extent (half extents of the
    binning box), rect (tx0, ty0, tx1, ty1), tiles_touched. Without
    opacity_logits the opacity is bounded by 1 alone (logits of 0)."""
    means, log_scales, quats = _c(means, np.float32), _c(log_scales, np.float32), _c(quats, np.float32)
    n = means.shape[0]
    logits = np.zeros(n, np.float32) if opacity_logits is None else _c(opacity_logits, np.float32)
    out = dict(means2d=np.zeros((n, 2), np.float32), depth=np.zeros(n, np.float32),
               radius=np.zeros(n, np.float32), extent=np.zeros((n, 2), np.float32),
               rect=np.zeros((n, 4), np.int32), tiles_touched=np.zeros(n, np.uint32))
    lib().orc_project_bin_f32(C.byref(_cam(cam)), C.byref(_prm(prm)), n, means, log_scales, quats,
                              logits, out["means2d"], out["depth"], out["radius"], out["extent"],
                              out["rect"], out["tiles_touched"])
    return out


def project_values(cam, prm, means, log_scales, quats, opacity_logits, sh, tiles_touched):
    """fp64 means2d, conic (a, b, c), opacity and rgb of the visible Gaussians."""
    n = means.shape[0]
    out = dict(means2d=np.zeros((n, 2)), conic=np.zeros((n, 3)), opacity=np.zeros(n),
               rgb=np.zeros((n, 3)))
    lib().orc_project_values_f64(C.byref(_cam(cam)), C.byref(_prm(prm)), n, _c(means, np.float32),
                                 _c(log_scales, np.float32), _c(quats, np.float32),
                                 _c(opacity_logits, np.float32), _c(sh, np.float32),
                                 _c(tiles_touched, np.uint32), out["means2d"], out["conic"],
                                 out["opacity"], out["rgb"])
    return out


# ------------------------------------------------------------------- binning

def bin(width, height, depth, rect, tiles_touched):
    """Sorted (tile, depth, index) intersection list and per-tile [start, end)."""
    tiles_touched = _c(tiles_touched, np.uint32)
    n = tiles_touched.shape[0]
    m = int(lib().orc_count_isect(n, tiles_touched))
    ntx, nty = tile_grid(width, height)
    keys = np.zeros(max(m, 1), np.uint64)
    values = np.zeros(max(m, 1), np.uint32)
    ranges = np.zeros((ntx * nty, 2), np.uint32)
    lib().orc_bin(width, height, n, _c(depth, np.float32), _c(rect, np.int32), tiles_touched,
                  keys, values, ranges)
    return keys[:m], values[:m], ranges


# ------------------------------------------------------------- rasterisation

def _img(x, cam):
    if x is None:
        return None
    return _c(x, np.float64).reshape(cam.height * cam.width * 4)


def render_fwd(cam, prm, tile_ranges, values, means2d, conic, opacity, rgb, F=None, B=None,
               rel_margin=0.0, f32_kappa=0.0):
    """Forward blend and composite (fp64). knife marks pixels with a threshold
    decision within its margin (see orc_render_fwd): rel_margin for every
    decision, or, with f32_kappa > 0, per-decision margins from an error bound
    of the fp32 evaluation of alpha and of the transmittance."""
    H, W = cam.height, cam.width
    out = np.zeros((H, W, 4))
    final_T = np.zeros((H, W))
    last = np.zeros((H, W), np.uint32)
    knife = np.zeros((H, W), np.uint8)
    t_stop = np.zeros((H, W))
    nb = C.c_uint64(0)
    vals = _c(values, np.uint32) if len(values) else np.zeros(1, np.uint32)
    lib().orc_render_fwd(C.byref(_cam(cam)), C.byref(_prm(prm)), _c(tile_ranges, np.uint32), vals,
                         _c(means2d, np.float64), _c(conic, np.float64), _c(opacity, np.float64),
                         _c(rgb, np.float64), _img(F, cam), _img(B, cam), out, final_T, last,
                         C.byref(nb), float(rel_margin), float(f32_kappa), knife, t_stop)
    return dict(out=out, final_T=final_T, last=last, n_blends=int(nb.value), knife=knife.astype(bool),
                t_stop=t_stop)


def render_bwd_2d(cam, prm, tile_ranges, values, means2d, conic, opacity, rgb, F, B, dL_dout):
    n = means2d.shape[0]
    g2d = np.zeros((n, 9))
    vals = _c(values, np.uint32) if len(values) else np.zeros(1, np.uint32)
    lib().orc_render_bwd_2d(C.byref(_cam(cam)), C.byref(_prm(prm)), n, _c(tile_ranges, np.uint32),
                            vals, _c(means2d, np.float64), _c(conic, np.float64),
                            _c(opacity, np.float64), _c(rgb, np.float64), _img(F, cam), _img(B, cam),
                            _c(dL_dout, np.float64), g2d)
    return g2d


def project_bwd(cam, prm, means, log_scales, quats, opacity_logits, sh, tiles_touched, g2d):
    n = means.shape[0]
    nc = (prm.sh_degree + 1) ** 2
    out = dict(means=np.zeros((n, 3)), log_scales=np.zeros((n, 3)), quats=np.zeros((n, 4)),
               opacity_logits=np.zeros(n), sh=np.zeros((n, nc, 3)))
    lib().orc_project_bwd(C.byref(_cam(cam)), C.byref(_prm(prm)), n, _c(means, np.float32),
                          _c(log_scales, np.float32), _c(quats, np.float32),
                          _c(opacity_logits, np.float32), _c(sh, np.float32),
                          _c(tiles_touched, np.uint32), _c(g2d, np.float64), out["means"],
                          out["log_scales"], out["quats"], out["opacity_logits"], out["sh"])
    return out


# ------------------------------------------------------------------ collapse

def composite(width, height, images_f16, order, n_front, F=None, B=None, stop_t=0.0,
              rel_margin=0.0, with_knife=False):
    """Collapse K cached premultiplied fp16 RGBA renders into F and B (fp64).

    images_f16: uint16 view of binary16 data, shape [pool, H, W, 4]; the fold
    takes images[order[0]], images[order[1]], ... front to back, the first
    n_front into F and the rest into B. With F/B given, the fold continues
    behind them (accumulate mode). stop_t > 0 skips layers that can no longer
    be seen (see orc_composite); with_knife also returns the pixels whose skip
    decision lies within rel_margin of stop_t."""
    imgs = _c(images_f16, np.uint16)
    order = _c(order, np.int32).reshape(-1)
    k = int(order.shape[0])
    if k:
        pool = imgs.shape[0]
        assert imgs.shape[1:] == (height, width, 4) and order.min() >= 0 and order.max() < pool
    else:
        imgs = np.zeros(4, np.uint16)
        order = np.zeros(1, np.int32)
    acc = F is not None
    Fo = _c(F, np.float64).copy() if acc else np.zeros((height, width, 4))
    Bo = _c(B, np.float64).copy() if acc else np.zeros((height, width, 4))
    knife = np.zeros((height, width), np.uint8)
    lib().orc_composite(width, height, k, imgs, order, int(n_front), Fo, Bo, 1 if acc else 0,
                        float(stop_t), float(rel_margin), knife)
    if with_knife:
        return Fo, Bo, knife.astype(bool)
    return Fo, Bo


# ------------------------------------------------------------------- helpers

def loss_l1(out, target, bg=None):
    """L1 reconstruction loss of a step and its gradient (Method: the active
    block is optimised against a reconstruction loss of the composited image).

    out: H x W x 4 premultiplied RGBA render; target: H x W x 3; bg: background
    colour (black if None). The image is img = rgb + (1 - a) bg, the loss the
    mean over pixels and colour channels of |img - target|, and its gradient
    takes sign(0) = 0: dL/drgb = sign(img - target) / (3 H W), dL/da =
    -sum_c bg_c dL/drgb_c. fp64 throughout. Returns (loss, H x W x 4 gradient).
    """
    out = np.asarray(out, np.float64)
    target = np.asarray(target, np.float64)
    h, w = target.shape[:2]
    b = np.zeros(3) if bg is None else np.asarray(bg, np.float64)
    img = out[..., :3] + (1.0 - out[..., 3:4]) * b
    d = img - target
    n = 3.0 * h * w
    g_rgb = np.sign(d) / n
    g_a = -(g_rgb * b).sum(-1, keepdims=True)
    return float(np.abs(d).sum() / n), np.concatenate([g_rgb, g_a], -1)


def adam(theta, g, m, v, lr, b1=0.9, b2=0.999, eps=1e-15, t=1):
    """One Adam step in fp64; returns (theta, m, v) (new arrays)."""
    theta, m, v = (np.array(x, np.float64).ravel().copy() for x in (theta, m, v))
    g = _c(np.asarray(g, np.float64).ravel(), np.float64)
    lib().orc_adam(theta.size, theta, g, m, v, float(lr), float(b1), float(b2), float(eps), int(t))
    return theta, m, v


def sh_basis(direction):
    d = _c(direction, np.float64)
    y = np.zeros(16)
    g = np.zeros(48)
    lib().orc_sh_basis(d, y, g)
    return y, g.reshape(16, 3)


def quat_to_rot(q):
    r = np.zeros(9)
    lib().orc_quat_to_rot(_c(q, np.float64), r)
    return r.reshape(3, 3)


def half_to_double(h):
    return lib().orc_half_to_double(int(h))


# --------------------------------------------------------------- whole step

def step(cam, prm, scene, F=None, B=None, dL_dout=None, pos32=True, rel_margin=0.0):
    """Project -> bin -> forward (-> backward when dL_dout is given).

    pos32=True uses the fp32 pixel-space means of the binning chain for the
    blend (the GPU kernels' precision for positions); pos32=False keeps every
    value in fp64 (smooth in the parameters, for finite differences).
    """
    pb = project_bin(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                     scene["opacity_logits"])
    pv = project_values(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                        scene["opacity_logits"], scene["sh"], pb["tiles_touched"])
    m2d = pb["means2d"].astype(np.float64) if pos32 else pv["means2d"]
    keys, values, ranges = bin(cam.width, cam.height, pb["depth"], pb["rect"], pb["tiles_touched"])
    fw = render_fwd(cam, prm, ranges, values, m2d, pv["conic"], pv["opacity"], pv["rgb"], F, B,
                    rel_margin=rel_margin)
    res = dict(bin=pb, values=pv, keys=keys, sorted_values=values, tile_ranges=ranges, fwd=fw,
               means2d_used=m2d)
    if dL_dout is not None:
        g2d = render_bwd_2d(cam, prm, ranges, values, m2d, pv["conic"], pv["opacity"], pv["rgb"], F,
                            B, dL_dout)
        res["g2d"] = g2d
        res["grads"] = project_bwd(cam, prm, scene["means"], scene["log_scales"], scene["quats"],
                                   scene["opacity_logits"], scene["sh"], pb["tiles_touched"], g2d)
    return res


# ------------------------------------------------------ frustum visibility

def box_meets_frustum(cam, lo, hi):
    """Whether the world-space box [lo, hi] meets the camera's view frustum
    (points with view depth >= near whose projection lies in [0, W] x [0, H]),
    by its definition: the intersection is non-empty iff some box point
    satisfies every frustum half-space. Solved as a linear program that
    maximises the smallest signed distance s of a box point to the frustum's
    planes (unit normals); returns (s >= 0, s). |s| measures how far the case
    is from touching."""
    from scipy.optimize import linprog
    R = np.asarray(cam.R, np.float64).reshape(3, 3)
    t = np.asarray(cam.t, np.float64).reshape(3)
    fx, fy, cx, cy = (float(v) for v in (cam.fx, cam.fy, cam.cx, cam.cy))
    W, H = float(cam.width), float(cam.height)
    # half-spaces n . p_cam + d >= 0 in camera space
    planes = [((0.0, 0.0, 1.0), -float(cam.near)),      # in front of the near plane
              ((fx, 0.0, cx), 0.0),                       # u >= 0
              ((-fx, 0.0, W - cx), 0.0),                  # u <= W
              ((0.0, fy, cy), 0.0),                       # v >= 0
              ((0.0, -fy, H - cy), 0.0)]                  # v <= H
    A, b = [], []
    for n, d in planes:
        n = np.asarray(n) / np.linalg.norm(n)
        # n . (R x + t) + d >= s   <=>   -(n R) . x + s <= n . t + d
        A.append(np.concatenate([-(n @ R), [1.0]]))
        b.append(float(n @ t + d))
    lo = np.asarray(lo, np.float64)
    hi = np.asarray(hi, np.float64)
    bounds = [(lo[i], hi[i]) for i in range(3)] + [(None, 1e6)]
    res = linprog(np.array([0.0, 0.0, 0.0, -1.0]), A_ub=np.array(A), b_ub=np.array(b),
                  bounds=bounds, method="highs")
    assert res.status == 0, res.message
    s = -res.fun
    return s >= 0.0, s

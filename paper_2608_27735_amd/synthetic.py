"""Seeded synthetic inputs shaped like the paper's workloads.

The paper trains on two real scenes of about 200 cameras each, partitioned by a
regular grid of 5-unit cells (Results section); those datasets are not
available, so every input here is drawn from a numpy PCG64 generator with a
fixed seed, in the order means -> log-scales -> quaternions -> opacity logits
-> SH -> cameras -> targets. This module holds input recipes only: random
draws, grid bookkeeping and camera placement. It computes nothing the method
computes, and both the GPU library's tests and the oracle's consume it.
"""
import math

import numpy as np

from .camera import Camera, RasterParams, look_at


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ----------------------------------------------------------------- the grid

class Grid:
    """Regular 3D grid of convex cells (the paper's partition, Method section)."""

    def __init__(self, lo, hi, dims):
        self.lo = np.asarray(lo, np.float64)
        self.hi = np.asarray(hi, np.float64)
        self.dims = np.asarray(dims, np.int64)
        self.size = (self.hi - self.lo) / self.dims

    @property
    def n_cells(self):
        return int(np.prod(self.dims))

    def cell_index(self, lin):
        nx, ny, _ = self.dims
        return np.array([lin % nx, (lin // nx) % ny, lin // (nx * ny)])

    def linear(self, ijk):
        nx, ny, _ = self.dims
        return int(ijk[0] + nx * (ijk[1] + ny * ijk[2]))

    def bounds(self, lin):
        ijk = self.cell_index(lin)
        lo = self.lo + ijk * self.size
        return lo, lo + self.size

    def cell_of(self, points):
        """Cell of each point by its position (Gaussians are assigned by mean,
        Limitations section)."""
        ijk = np.floor((np.asarray(points, np.float64) - self.lo) / self.size).astype(np.int64)
        ijk = np.clip(ijk, 0, self.dims - 1)
        nx, ny, _ = self.dims
        return ijk[:, 0] + nx * (ijk[:, 1] + ny * ijk[:, 2])

    def order_from(self, campos):
        """Front-to-back order of all cells for a camera: sum over axes of the
        cell-index distance from the camera's (possibly virtual) cell, ties by
        linear id. Along any ray from the camera each per-axis distance is
        non-decreasing and every cell crossing raises the sum, so the order
        agrees with the traversal order of every ray."""
        cam = np.floor((np.asarray(campos, np.float64) - self.lo) / self.size).astype(np.int64)
        keys = []
        for lin in range(self.n_cells):
            ijk = self.cell_index(lin)
            keys.append((int(np.abs(ijk - cam).sum()), lin))
        return [lin for _, lin in sorted(keys)]

    def order_by_view_depth(self, cam: Camera):
        """Alternative order: view depth of the cell centres."""
        R = np.asarray(cam.R, np.float64)
        t = np.asarray(cam.t, np.float64)
        keys = []
        for lin in range(self.n_cells):
            lo, hi = self.bounds(lin)
            c = 0.5 * (lo + hi)
            keys.append(((R @ c + t)[2], lin))
        return [lin for _, lin in sorted(keys)]


# ------------------------------------------------------------ Gaussians

def gaussians(r, means, sh_degree, logscale_mean, logscale_sd, sh_hi_sd=0.1):
    """Parameter block for given means: log-scales N(mean, sd), unit quaternions
    from a normalised N(0, I), opacity logits N(0, 1), SH DC uniform on
    [-sqrt(pi), sqrt(pi)] (which the degree-0 band maps to a base colour
    uniform on [0, 1]) and higher bands N(0, sh_hi_sd)."""
    n = means.shape[0]
    ls = r.normal(logscale_mean, logscale_sd, (n, 3))
    q = r.normal(0.0, 1.0, (n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    op = r.normal(0.0, 1.0, n)
    nc = (sh_degree + 1) ** 2
    sh = np.zeros((n, nc, 3))
    sh[:, 0, :] = r.uniform(-math.sqrt(math.pi), math.sqrt(math.pi), (n, 3))
    if nc > 1:
        sh[:, 1:, :] = r.normal(0.0, sh_hi_sd, (n, nc - 1, 3))
    f = np.float32
    return dict(means=np.ascontiguousarray(means, f), log_scales=ls.astype(f), quats=q.astype(f),
                opacity_logits=op.astype(f), sh=sh.astype(f))


def subset(scene, mask):
    return {k: np.ascontiguousarray(v[mask]) for k, v in scene.items()}


def concat(scenes):
    return {k: np.ascontiguousarray(np.concatenate([s[k] for s in scenes])) for k in scenes[0]}


def uniform_in_cells(r, grid, per_cell):
    pts = []
    for lin in range(grid.n_cells):
        lo, hi = grid.bounds(lin)
        pts.append(r.uniform(lo, hi, (per_cell, 3)))
    return np.concatenate(pts)


# ------------------------------------------------------------- workloads

class Workload(dict):
    """dict with attribute access: scene, cams, grid, cell_of, active, ..."""
    __getattr__ = dict.__getitem__


def tiny(seed=1):
    """4,096 Gaussians, 2x2x2 grid over [-1, 1]^3 (512 uniform per cell), log-scales
    N(log 0.03, 0.3), SH degree 0; one 128x128 camera with a 60 degree field of
    view at distance 3 looking at the origin; the active cell is rank 3 of 8 in
    the camera's front-to-back order, so F and B both hold cells."""
    r = rng(seed)
    grid = Grid((-1, -1, -1), (1, 1, 1), (2, 2, 2))
    means = uniform_in_cells(r, grid, 512)
    scene = gaussians(r, means, 0, math.log(0.03), 0.3)
    d = np.array([0.3, -1.0, 0.4])
    cam = look_at(3.0 * d / np.linalg.norm(d), (0, 0, 0), 128, 128)
    order = grid.order_from(cam.campos)
    target = r.uniform(0.0, 1.0, (128, 128, 3)).astype(np.float32)
    return Workload(scene=scene, cams=[cam], grid=grid, cell_of=grid.cell_of(scene["means"]),
                    order=order, active=order[3], target=target,
                    params=RasterParams(sh_degree=0))


def ring(seed=2, n=65536, width=512, height=512, n_cams=8):
    """64K Gaussians, SH degree 3, 4x4x4 grid over [-1, 1]^3, means from a
    32-blob Gaussian mixture (centres uniform in the cube, sd 0.08, clipped to
    it), log-scales N(log 0.03, 0.3); 8 cameras at 512x512 on a ring of radius 3
    at 20 degrees elevation; the active cell is the one whose count is nearest
    1,024."""
    r = rng(seed)
    grid = Grid((-1, -1, -1), (1, 1, 1), (4, 4, 4))
    centres = r.uniform(-1.0, 1.0, (32, 3))
    comp = r.integers(0, 32, n)
    means = np.clip(centres[comp] + r.normal(0.0, 0.08, (n, 3)), -1.0, 1.0 - 1e-6)
    scene = gaussians(r, means, 3, math.log(0.03), 0.3)
    cams = []
    el = math.radians(20.0)
    for k in range(n_cams):
        az = math.radians(45.0 * k)
        pos = 3.0 * np.array([math.cos(el) * math.cos(az), math.cos(el) * math.sin(az), math.sin(el)])
        cams.append(look_at(pos, (0, 0, 0), width, height))
    cell = grid.cell_of(scene["means"])
    counts = np.bincount(cell, minlength=grid.n_cells)
    active = int(np.argmin(np.abs(counts - 1024)))
    target = r.uniform(0.0, 1.0, (n_cams, height, width, 3)).astype(np.float32)
    return Workload(scene=scene, cams=cams, grid=grid, cell_of=cell, active=active, target=target,
                    params=RasterParams(sh_degree=3))


def active_block_1m(seed=41, n=1_000_000, width=1297, height=840, heavy_tail=False, cam_index=0,
                    n_cams=200):
    """The large active block: a 5x5x4 grid of 5-unit cells (the paper's cell
    side) over [-12.5, 12.5]^2 x [0, 20]; the active cell (2, 2, 0) holds n
    Gaussians with means uniform in it, SH degree 3, log-scales N(log 0.25, 0.5)
    (sd 1.0 with heavy_tail); 200 cameras on the ellipse (20 cos p, 16 sin p, 8)
    looking at (0, 0, 2), rendered at width x height. Frozen cells are not drawn
    as Gaussians: their cached renders come from cached_cell_images()."""
    r = rng(seed)
    grid = Grid((-12.5, -12.5, 0.0), (12.5, 12.5, 20.0), (5, 5, 4))
    active = grid.linear((2, 2, 0))
    lo, hi = grid.bounds(active)
    means = r.uniform(lo, hi, (n, 3))
    scene = gaussians(r, means, 3, math.log(0.25), 1.0 if heavy_tail else 0.5)
    cams = []
    for k in range(n_cams):
        ph = 2.0 * math.pi * k / n_cams
        cams.append(look_at((20.0 * math.cos(ph), 16.0 * math.sin(ph), 8.0), (0, 0, 2), width, height))
    cam = cams[cam_index]
    order = grid.order_from(cam.campos)
    return Workload(scene=scene, cams=cams, cam=cam, grid=grid, active=active, order=order,
                    params=RasterParams(sh_degree=3))


def perturbed(r, scene, pos_sd=0.01, logit_shift=-1.0):
    """A starting point for training towards `scene`: means moved by N(0,
    pos_sd), opacity logits shifted by logit_shift, colours reset to the
    middle grey (SH DC 0, higher bands 0); scales and rotations kept."""
    out = {k: np.array(v, copy=True) for k, v in scene.items()}
    out["means"] = (out["means"] + r.normal(0.0, pos_sd, out["means"].shape)).astype(np.float32)
    out["opacity_logits"] = (out["opacity_logits"] + logit_shift).astype(np.float32)
    out["sh"] = np.zeros_like(out["sh"])
    return out


def midscale_block(seed=3, n=300_000, width=1297, height=840, n_cams=200, cam_index=0):
    """The mid-scale scene's active block: a 4x4x2 grid over [-10, 10]^2 x
    [0, 6]; the active cell (1, 1, 0) holds n Gaussians, 40% on a ground
    plane (z uniform on [0, 0.1]) and 60% in 8 Gaussian blobs (sd 0.5, centres
    uniform in the cell, clipped to it), log-scales N(log 0.2, 0.5), SH degree
    3; 200 cameras on the ellipse (16 cos p, 12 sin p, 5) looking at (0, 0, 1.5)."""
    r = rng(seed)
    grid = Grid((-10.0, -10.0, 0.0), (10.0, 10.0, 6.0), (4, 4, 2))
    active = grid.linear((1, 1, 0))
    lo, hi = grid.bounds(active)
    n_ground = int(0.4 * n)
    ground = np.stack([r.uniform(lo[0], hi[0], n_ground), r.uniform(lo[1], hi[1], n_ground),
                       r.uniform(0.0, 0.1, n_ground)], axis=1)
    centres = r.uniform(lo, hi, (8, 3))
    comp = r.integers(0, 8, n - n_ground)
    blobs = np.clip(centres[comp] + r.normal(0.0, 0.5, (n - n_ground, 3)), lo, hi - 1e-6)
    scene = gaussians(r, np.concatenate([ground, blobs]), 3, math.log(0.2), 0.5)
    cams = [look_at((16.0 * math.cos(2 * math.pi * k / n_cams), 12.0 * math.sin(2 * math.pi * k / n_cams),
                     5.0), (0, 0, 1.5), width, height) for k in range(n_cams)]
    cam = cams[cam_index]
    return Workload(scene=scene, cams=cams, cam=cam, grid=grid, active=active,
                    order=grid.order_from(cam.campos), params=RasterParams(sh_degree=3))


def midscale_scene(seed=31, n=5_000_000, width=1297, height=840, n_cams=200):
    """The whole mid-scale scene: n Gaussians over a 4x4x2 grid on
    [-10, 10]^2 x [0, 6], 40% on a ground plane (z uniform on [0, 0.1]) and 60%
    in 64 Gaussian blobs (sd 0.5, centres uniform in the box, clipped to it),
    log-scales N(log 0.2, 0.5) (0.01 of the 20-unit extent), SH degree 3;
    cameras on the ellipse (16 cos p, 12 sin p, 5) looking at (0, 0, 1.5)."""
    r = rng(seed)
    grid = Grid((-10.0, -10.0, 0.0), (10.0, 10.0, 6.0), (4, 4, 2))
    lo, hi = grid.lo, grid.hi
    n_ground = int(0.4 * n)
    ground = np.stack([r.uniform(lo[0], hi[0], n_ground), r.uniform(lo[1], hi[1], n_ground),
                       r.uniform(0.0, 0.1, n_ground)], axis=1)
    centres = r.uniform(lo, hi, (64, 3))
    comp = r.integers(0, 64, n - n_ground)
    blobs = np.clip(centres[comp] + r.normal(0.0, 0.5, (n - n_ground, 3)), lo, hi - 1e-6)
    scene = gaussians(r, np.concatenate([ground, blobs]), 3, math.log(0.2), 0.5)
    cams = [look_at((16.0 * math.cos(2 * math.pi * k / n_cams), 12.0 * math.sin(2 * math.pi * k / n_cams),
                     5.0), (0, 0, 1.5), width, height) for k in range(n_cams)]
    return Workload(scene=scene, cams=cams, grid=grid, cell_of=grid.cell_of(scene["means"]),
                    params=RasterParams(sh_degree=3))


def stress_block(seed=5, n=4_000_000, width=2560, height=1440, n_cams=200, cam_index=0):
    """The stress configuration's active block: an 8x8x2 grid over [-20, 20]^2 x
    [0, 10]; the active cell (3, 3, 0) holds n Gaussians with means uniform in
    it and tiny scales, log-scales N(log 0.08, 0.5) (0.002 of the 40-unit
    extent), SH degree 3; 200 cameras at 2560x1440 on the ellipse
    (30 cos p, 24 sin p, 12) looking at (0, 0, 2)."""
    r = rng(seed)
    grid = Grid((-20.0, -20.0, 0.0), (20.0, 20.0, 10.0), (8, 8, 2))
    active = grid.linear((3, 3, 0))
    lo, hi = grid.bounds(active)
    scene = gaussians(r, r.uniform(lo, hi, (n, 3)), 3, math.log(0.08), 0.5)
    cams = [look_at((30.0 * math.cos(2 * math.pi * k / n_cams), 24.0 * math.sin(2 * math.pi * k / n_cams),
                     12.0), (0, 0, 2.0), width, height) for k in range(n_cams)]
    cam = cams[cam_index]
    return Workload(scene=scene, cams=cams, cam=cam, grid=grid, active=active,
                    order=grid.order_from(cam.campos), params=RasterParams(sh_degree=3))


# ----------------------------------------------------------- image inputs

def premultiplied_images(r, k, height, width, alpha_max=0.95, coverage=0.5):
    """k premultiplied RGBA images (rgb <= alpha) as float32 [k, H, W, 4]: alpha
    uniform on [0, alpha_max] over a random axis-aligned rectangle covering
    about `coverage` of the frame (zero elsewhere), colour uniform on [0, 1]."""
    out = np.zeros((k, height, width, 4), np.float32)
    side = math.sqrt(coverage)
    for j in range(k):
        h0 = int(r.integers(0, max(1, int(height * (1 - side)) + 1)))
        w0 = int(r.integers(0, max(1, int(width * (1 - side)) + 1)))
        hh, ww = max(1, int(height * side)), max(1, int(width * side))
        a = r.uniform(0.0, alpha_max, (hh, ww, 1))
        c = r.uniform(0.0, 1.0, (hh, ww, 3))
        out[j, h0:h0 + hh, w0:w0 + ww, :3] = c * a
        out[j, h0:h0 + hh, w0:w0 + ww, 3:] = a
    return out


def half_bits(x):
    """binary16 bit patterns (uint16) of a float array, round-to-nearest-even."""
    return np.ascontiguousarray(np.asarray(x, np.float32).astype(np.float16)).view(np.uint16)


def background_pair(r, height, width):
    """A premultiplied F/B pair: F partly transparent, B denser."""
    f = premultiplied_images(r, 1, height, width, alpha_max=0.6, coverage=0.4)[0]
    b = premultiplied_images(r, 1, height, width, alpha_max=0.95, coverage=0.7)[0]
    return f, b


def dense_front(r, height, width, opaque_frac=0.2):
    """A premultiplied F that hides much of the frame: alpha uniform on
    [0.85, 1) over the left 70% of the columns, exactly 1 on a random
    `opaque_frac` of those pixels, 0.3 elsewhere; colour uniform on [0, 1]."""
    a = np.full((height, width, 1), 0.3, np.float32)
    cut = int(0.7 * width)
    a[:, :cut, 0] = r.uniform(0.85, 1.0, (height, cut))
    a[:, :cut, 0][r.uniform(0, 1, (height, cut)) < opaque_frac] = 1.0
    c = r.uniform(0.0, 1.0, (height, width, 3)).astype(np.float32)
    return np.concatenate([c * a, a], -1).astype(np.float32)


def upstream_grad(r, height, width, scale=1.0):
    """A smooth-free random dL/dout [H, W, 4]."""
    return (scale * r.normal(0.0, 1.0, (height, width, 4))).astype(np.float32)


def splats_2d(r, n, width, height, sigma_px=(1.0, 12.0), depth_range=(0.5, 20.0)):
    """Screen-space Gaussians for stage tests of binning and blending: centres
    uniform over a frame padded by 10%, depths uniform, covariance from two
    log-uniform sigmas and a uniform angle, conic = inverse covariance, radius
    between 2.5 and 3.5 sigmas of the major axis, opacity uniform on
    [0.05, 0.99], colour uniform on [0, 1]. Returns float32 arrays (means2d, conic_opacity [n, 4],
    depth, radius, rgb)."""
    pad = 0.1
    u = r.uniform(-pad * width, (1 + pad) * width, n)
    v = r.uniform(-pad * height, (1 + pad) * height, n)
    depth = r.uniform(*depth_range, n)
    s = np.exp(r.uniform(math.log(sigma_px[0]), math.log(sigma_px[1]), (n, 2)))
    th = r.uniform(0, math.pi, n)
    c, sn = np.cos(th), np.sin(th)
    cov_a = c * c * s[:, 0] ** 2 + sn * sn * s[:, 1] ** 2
    cov_b = c * sn * (s[:, 0] ** 2 - s[:, 1] ** 2)
    cov_c = sn * sn * s[:, 0] ** 2 + c * c * s[:, 1] ** 2
    det = cov_a * cov_c - cov_b ** 2
    op = r.uniform(0.05, 0.99, n)
    rgb = r.uniform(0.0, 1.0, (n, 3))
    rad = r.uniform(2.5, 3.5, n) * s.max(axis=1)
    f = np.float32
    co = np.stack([cov_c / det, -cov_b / det, cov_a / det, op], axis=1)
    return dict(means2d=np.stack([u, v], 1).astype(f), conic_opacity=co.astype(f),
                depth=depth.astype(f), radius=rad.astype(f), rgb=rgb.astype(f))


def cached_images_device(k, height, width, seed, device, coverage=0.35, alpha_max=0.9,
                         with_rects=False):
    """k premultiplied fp16 RGBA cached renders [k, H, W, 4] drawn on the GPU
    with a seeded torch generator (for workloads too large to draw on the
    host): per layer a random axis-aligned rectangle covering about
    `coverage` of the frame, alpha uniform on [0, alpha_max] inside, colour
    uniform on [0, 1], zero outside. with_rects also returns each layer's
    rectangle rounded out to 16-pixel tiles (int32 [k, 4] = x0, y0, x1, y1 on
    the device), the coverage box a cached render comes with."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = torch.zeros((k, height, width, 4), dtype=torch.float16, device=device)
    side = math.sqrt(coverage)
    hh, ww = max(1, int(height * side)), max(1, int(width * side))
    corners = torch.rand((k, 2), generator=g, device=device)
    boxes = []
    for j in range(k):
        h0 = int(corners[j, 0].item() * (height - hh + 1))
        w0 = int(corners[j, 1].item() * (width - ww + 1))
        a = torch.rand((hh, ww, 1), generator=g, device=device) * alpha_max
        c = torch.rand((hh, ww, 3), generator=g, device=device)
        out[j, h0:h0 + hh, w0:w0 + ww, :3] = (c * a).half()
        out[j, h0:h0 + hh, w0:w0 + ww, 3:] = a.half()
        boxes.append((w0 // 16 * 16, h0 // 16 * 16, min(width, -(-(w0 + ww) // 16) * 16),
                      min(height, -(-(h0 + hh) // 16) * 16)))
    if with_rects:
        return out, torch.tensor(boxes, dtype=torch.int32, device=device).reshape(k, 4)
    return out

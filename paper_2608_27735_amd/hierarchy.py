"""The memory hierarchy around the step (Method section: cached camera-partition
renders live on disk or in system memory, and only the active parameters and
the F/B pair a camera needs are on the GPU; Results section: the cache is read
when the active partition changes, so the transfer is amortised over many
steps).

  - visible_boxes: which partitions a camera can see (frustum filtering of the
    camera-partition pairs, so invisible pairs are never rendered or cached);
  - HostCache: the cached fp16 renders in pinned system memory, with their
    coverage boxes;
  - FBStreamer: F and B of one camera built from the host cache in chunks: two
    device staging chunks, uploads on a copy stream (only coverage boxes cross
    PCIe, abcd_stage_cached) overlapped with the collapse of the previous
    chunk (abcd_composite_cache, accumulating). Device memory is the two
    chunks plus F and B, whatever the number of partitions.
"""
import numpy as np
import torch

from . import api


# ------------------------------------------------------- frustum filtering

def _frustum(cam):
    """Near-plane corners (4, 3) and corner rays (4, 3) of the view frustum in
    camera space (z >= near, pixel coordinates within [0, W] x [0, H])."""
    fx, fy, cx, cy = (float(v) for v in (cam.fx, cam.fy, cam.cx, cam.cy))
    uv = np.array([[0.0, 0.0], [cam.width, 0.0], [cam.width, cam.height], [0.0, cam.height]])
    rays = np.stack([(uv[:, 0] - cx) / fx, (uv[:, 1] - cy) / fy, np.ones(4)], axis=1)
    return rays * float(cam.near), rays


def visible_boxes(cam, lo, hi):
    """Whether each world-space box [lo_i, hi_i] meets the camera's view
    frustum (unbounded far side). Exact separating-axis test between two
    convex polyhedra: the box is separated from the frustum iff their
    projections are disjoint on one of the box's face normals, the frustum's
    face normals, or a cross product of an edge direction of each (the
    frustum's edges are its four corner rays and the two near-rectangle
    directions). A projection of the frustum is unbounded where a corner ray
    points along the axis. Boxes that only touch the frustum count as
    visible."""
    lo = np.atleast_2d(np.asarray(lo, np.float64))
    hi = np.atleast_2d(np.asarray(hi, np.float64))
    R = np.asarray(cam.R, np.float64).reshape(3, 3)
    t = np.asarray(cam.t, np.float64).reshape(3)
    near_pts, rays = _frustum(cam)
    # box corners in camera space: (n, 8, 3)
    sel = np.array([[i & 1, (i >> 1) & 1, (i >> 2) & 1] for i in range(8)], bool)
    corners_w = np.where(sel[None], hi[:, None, :], lo[:, None, :])
    corners = corners_w @ R.T + t
    box_dirs = R.T  # rows: world axes in camera space
    fr_edges = np.concatenate([rays, np.eye(3)[:2]], axis=0)
    fr_normals = [np.array([0.0, 0.0, 1.0])] + [np.cross(rays[i], rays[(i + 1) % 4])
                                                 for i in range(4)]
    axes = list(box_dirs) + fr_normals + [np.cross(a, b) for a in box_dirs for b in fr_edges]
    axes = np.array([a / np.linalg.norm(a) for a in axes if np.linalg.norm(a) > 1e-12])
    # projections
    bp = corners @ axes.T                    # (n, 8, A)
    bmin, bmax = bp.min(axis=1), bp.max(axis=1)
    fp = near_pts @ axes.T                   # (4, A)
    rp = rays @ axes.T                       # (4, A)
    fmin = np.where((rp < 0).any(axis=0), -np.inf, fp.min(axis=0))
    fmax = np.where((rp > 0).any(axis=0), np.inf, fp.max(axis=0))
    separated = (bmax < fmin[None]) | (bmin > fmax[None])
    return ~separated.any(axis=1)


def visible_cells(cam, grid, margin=0.0):
    """Cells of a regular grid that the camera sees, each cell's box grown by
    `margin` (the reach of its Gaussians beyond the cell, e.g. three times
    their largest scale)."""
    los, his = zip(*(grid.bounds(c) for c in range(grid.n_cells)))
    return visible_boxes(cam, np.array(los) - margin, np.array(his) + margin)


# ------------------------------------------------------------ host cache

class HostCache:
    """Cached renders in pinned system memory: slot s holds one camera-partition
    image (fp16 [H, W, 4]) and its coverage box (x0, y0, x1, y1)."""

    def __init__(self, width, height, n_slots):
        self.W, self.H = width, height
        self.images = torch.zeros((n_slots, height, width, 4), dtype=torch.float16).pin_memory()
        self.rects = np.zeros((n_slots, 4), np.int32)
        self.rects[:, 0], self.rects[:, 1] = width, height  # empty until written
        self.index = {}

    def slot(self, key):
        """Slot of a (camera, partition) key, assigned on first use."""
        if key not in self.index:
            if len(self.index) == self.images.shape[0]:
                raise RuntimeError("host cache is full")
            self.index[key] = len(self.index)
        return self.index[key]

    def put(self, key, image, rect):
        """Store a device image and its coverage box (int32 [4], any device);
        synchronous."""
        s = self.slot(key)
        self.images[s].copy_(image)
        self.rects[s] = np.asarray(rect.cpu() if torch.is_tensor(rect) else rect, np.int32)
        return s


class FBStreamer:
    """Builds F and B for one camera from a HostCache, `chunk` images at a time."""

    def __init__(self, cache, chunk=16, device=None):
        self.cache = cache
        self.chunk = chunk
        dev = torch.device("cuda", torch.cuda.current_device()) if device is None else device
        H, W = cache.H, cache.W
        self.bufs = [torch.empty((chunk, H, W, 4), dtype=torch.float16, device=dev)
                     for _ in range(2)]
        self.copy_stream = torch.cuda.Stream(device=dev)
        self.consumed = [None, None]
        self.device = dev

    def build(self, slots, n_front, F, B, stop_t=0.0):
        """F = fold of slots[:n_front], B = fold of slots[n_front:] (front to
        back), written to the given fp32 [H, W, 4] tensors on the current
        stream. Returns once the work is queued; the host images must not change
        until the current stream reaches this point."""
        compute = torch.cuda.current_stream()
        slots = list(slots)
        if not slots:
            api.composite_cache(self.bufs[0][:0], [], 0, F=F, B=B)
            return F, B
        # coverage boxes of every layer, one small asynchronous upload
        rects = torch.from_numpy(np.ascontiguousarray(self.cache.rects[slots])).pin_memory()
        rects = rects.to(self.device, non_blocking=True)
        for c, a in enumerate(range(0, len(slots), self.chunk)):
            part = slots[a:a + self.chunk]
            buf = c & 1
            with torch.cuda.stream(self.copy_stream):
                # the chunk buffer is free once the collapse that read it is done
                if self.consumed[buf] is not None:
                    self.copy_stream.wait_event(self.consumed[buf])
                else:
                    self.copy_stream.wait_stream(compute)
                api.stage_cached([self.cache.images[s] for s in part], self.bufs[buf],
                                 rects=self.cache.rects[part])
                staged = torch.cuda.Event()
                staged.record(self.copy_stream)
            compute.wait_event(staged)
            nf = max(0, min(n_front, a + len(part)) - a)
            api.composite_cache(self.bufs[buf][:len(part)], list(range(len(part))), nf, F=F, B=B,
                                accumulate=c > 0, rects=rects[a:a + len(part)], stop_t=stop_t)
            ev = torch.cuda.Event()
            ev.record(compute)
            self.consumed[buf] = ev
        return F, B

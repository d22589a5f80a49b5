"""Block coordinate descent around the active-block step (Method section) and
the three training setups the paper compares (Results section), on synthetic
scenes whose ground truth is known.

BlockDescent keeps every partition's parameters and Adam moments in host
memory and puts one partition at a time on the GPU. Visiting partition b:
  1. the cameras that see b (frustum filtering) are gathered;
  2. for each, F and B are collapsed from the cached renders of the other
     partitions it sees, split at b in the camera's front-to-back order
     (streamed from the pinned host cache, FBStreamer);
  3. T steps: sample one of those cameras, project/bin/blend b alone between
     that camera's F and B, L1 loss against its image, backward into b only,
     Adam on b;
  4. b's parameters go back to host memory and its cached renders are
     redrawn for every camera that sees it.
Partitions are visited round robin (the paper leaves the schedule open).

Setups (mode): "abcd" (the method), "ablated" (F = B = transparent: each
partition is fitted to the whole image on its own) and "joint" (every
Gaussian in one partition: plain 3DGS training on the same renderer).
"""
import time

import numpy as np
import torch

from . import api
from .cache import CacheRefresher
from .hierarchy import FBStreamer, HostCache, visible_cells
from .step import ActiveBlockStep

NAMES = ("means", "log_scales", "quats", "opacity_logits", "sh")
DEFAULT_LR = dict(means=1.6e-4, log_scales=5e-3, quats=1e-3, opacity_logits=5e-2, sh=2.5e-3)


def render_joint(cam, prm, params):
    """The whole scene rendered at once (F = B = transparent): fp32 [H, W, 4]."""
    p = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, p)
    return api.render_fwd(cam, prm, bins, p)["out"]


def psnr(out, target):
    """PSNR of the composited colour over a black background against target."""
    mse = float(((out[..., :3] - target) ** 2).mean().item())
    return 10.0 * np.log10(1.0 / max(mse, 1e-20))


class BlockDescent:
    def __init__(self, grid, cell_of, scene, cams, targets, prm, mode="abcd", lr=None,
                 margin=None, seed=0, chunk=16, device=None):
        if mode not in ("abcd", "ablated", "joint"):
            raise ValueError(f"unknown mode {mode}")
        self.dev = device or torch.device("cuda", torch.cuda.current_device())
        self.grid, self.cams, self.prm, self.mode = grid, cams, prm, mode
        self.scene = {k: np.array(scene[k], np.float32, copy=True) for k in NAMES}
        self.m = {k: np.zeros_like(v) for k, v in self.scene.items()}
        self.v = {k: np.zeros_like(v) for k, v in self.scene.items()}
        self.lr = dict(DEFAULT_LR if lr is None else lr)
        self.rng = np.random.default_rng(seed)
        self.targets = torch.from_numpy(np.ascontiguousarray(targets, np.float32)).to(self.dev)
        cell_of = np.asarray(cell_of)
        if mode == "joint":
            cell_of = np.zeros_like(cell_of)
        self.blocks = [int(b) for b in np.unique(cell_of)]
        self.members = {b: np.nonzero(cell_of == b)[0] for b in self.blocks}
        self.t = {b: 0 for b in self.blocks}
        if margin is None:  # reach of a Gaussian beyond its cell: three sigmas of its largest axis
            margin = 3.0 * float(np.exp(self.scene["log_scales"].max()))
        if mode == "joint":
            self.sees = [set(self.blocks) for _ in cams]
        else:
            self.sees = [set(int(c) for c in np.nonzero(visible_cells(cam, grid, margin))[0])
                         & set(self.blocks) for cam in cams]
        W, H = cams[0].width, cams[0].height
        self.W, self.H = W, H
        self.cache = None
        if mode == "abcd":
            n_pairs = sum(len(s) for s in self.sees)
            self.cache = HostCache(W, H, max(n_pairs, 1))
            self.streamer = FBStreamer(self.cache, chunk=chunk, device=self.dev)
            for b in self.blocks:
                self._refresh(b, self._upload(b)[0])
        self.steps = 0

    # -------------------------------------------------------------- state

    def _upload(self, b):
        idx = self.members[b]
        up = lambda d: {k: torch.from_numpy(np.ascontiguousarray(d[k][idx])).to(self.dev)
                        for k in NAMES}
        return up(self.scene), up(self.m), up(self.v)

    def _download(self, b, params, m, v):
        idx = self.members[b]
        for k in NAMES:
            self.scene[k][idx] = params[k].cpu().numpy()
            self.m[k][idx] = m[k].cpu().numpy()
            self.v[k][idx] = v[k].cpu().numpy()

    def _cams_of(self, b):
        return [i for i, s in enumerate(self.sees) if b in s]

    def _refresh(self, b, params):
        """Redraw partition b's cached render for every camera that sees it."""
        cams = self._cams_of(b)
        if not cams:
            return
        ref = CacheRefresher(self.prm, params, self.W, self.H)
        slots = [self.cache.slot((i, b)) for i in cams]
        rects = torch.zeros((len(cams), 4), dtype=torch.int32, device=self.dev)
        ref.refresh([self.cams[i] for i in cams], [self.cache.images[s] for s in slots], rects)
        self.cache.rects[slots] = rects.cpu().numpy()

    def _fb(self, i, b):
        """F and B of camera i around partition b from the host cache."""
        order = [int(c) for c in self.grid.order_from(self.cams[i].campos)]
        seen = [c for c in order if c in self.sees[i]]
        pos = seen.index(b)
        front, back = seen[:pos], seen[pos + 1:]
        F = torch.empty((self.H, self.W, 4), dtype=torch.float32, device=self.dev)
        B = torch.empty_like(F)
        self.streamer.build([self.cache.slot((i, c)) for c in front + back], len(front), F, B)
        return F, B

    # ------------------------------------------------------------- training

    def visit(self, b, T):
        """T steps on partition b (see the module docstring)."""
        cams = self._cams_of(b)
        if not cams or len(self.members[b]) == 0:
            return
        params, m, v = self._upload(b)
        fb = {i: self._fb(i, b) for i in cams} if self.mode == "abcd" else {}
        st = ActiveBlockStep(self.cams[cams[0]], self.prm, params)
        for _ in range(T):
            i = int(self.rng.choice(cams))
            F, B = fb.get(i, (None, None))
            st.cam = self.cams[i]
            st.project_and_bin(sync=True)
            st.forward(F, B)
            st.loss_grad(self.targets[i])
            st.backward(st.dL_dout, F, B)
            self.t[b] += 1
            api.adam_step(params, st.grads, m, v, self.lr, self.t[b])
            self.steps += 1
        self._download(b, params, m, v)
        if self.mode == "abcd":
            self._refresh(b, params)

    def epoch(self, T):
        for b in self.blocks:
            self.visit(b, T)

    def evaluate(self):
        """Mean PSNR of the joint render of the current scene over all cameras."""
        params = {k: torch.from_numpy(self.scene[k]).to(self.dev) for k in NAMES}
        vals = [psnr(render_joint(cam, self.prm, params), self.targets[i])
                for i, cam in enumerate(self.cams)]
        return float(np.mean(vals))


def compare(gt_scene, init_scene, grid, cell_of, cams, prm, epochs=3, T=20, joint_T=None,
            seed=0, chunk=4, device=None):
    """The paper's three setups on a synthetic scene: targets are joint renders
    of gt_scene, training starts from init_scene. Returns per mode the PSNR
    before and after, steps, wall time and peak device memory."""
    dev = device or torch.device("cuda", torch.cuda.current_device())
    gt = {k: torch.from_numpy(np.ascontiguousarray(gt_scene[k], np.float32)).to(dev) for k in NAMES}
    targets = np.stack([render_joint(c, prm, gt)[..., :3].cpu().numpy() for c in cams])
    del gt
    out = {}
    for mode in ("joint", "ablated", "abcd"):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        bd = BlockDescent(grid, cell_of, init_scene, cams, targets, prm, mode=mode, seed=seed,
                          chunk=chunk, device=dev)
        before = bd.evaluate()
        t0 = time.perf_counter()
        steps_T = joint_T if (mode == "joint" and joint_T is not None) else T
        for _ in range(epochs):
            bd.epoch(steps_T)
        torch.cuda.synchronize()
        secs = time.perf_counter() - t0
        peak = torch.cuda.max_memory_allocated() - base
        out[mode] = dict(psnr_before=before, psnr_after=bd.evaluate(), steps=bd.steps,
                         seconds=secs, peak_device_bytes=int(peak), blocks=len(bd.blocks))
        del bd
    return out

"""Refresh of a partition's cached renders (Method section: after the T updates
of a block, the renders that the block contributes to every observing camera
are re-made; the cache holds them as compressed RGBA, here binary16).

For each camera: project -> bin -> cached render (abcd_render_cache) into one
of two device staging images, then an asynchronous copy of that image into the
caller's pinned host slot on a second stream, so that the copy of camera i
overlaps the rendering of camera i + 1. The intersection count is read back
per camera (binning grows its buffers when a camera needs more), the only
synchronisation on the compute stream.
"""
import torch

from . import api


class CacheRefresher:
    def __init__(self, prm, params, width, height):
        self.prm, self.params = prm, params
        n = params["means"].shape[0]
        dev = params["means"].device
        f32 = torch.float32
        self.W, self.H = width, height
        self.proj = dict(means2d=torch.empty((n, 2), dtype=f32, device=dev),
                         conic_opacity=torch.empty((n, 4), dtype=f32, device=dev),
                         depth=torch.empty((n,), dtype=f32, device=dev),
                         extent=torch.empty((n, 2), dtype=f32, device=dev),
                         tiles_touched=torch.empty((n,), dtype=torch.int32, device=dev),
                         rgb=torch.empty((n, 3), dtype=f32, device=dev))
        nt = api.n_tiles(width, height)
        self.tile_ranges = torch.empty((nt, 2), dtype=torch.int32, device=dev)
        self.tile_order = torch.empty((nt,), dtype=torch.int32, device=dev)
        self.values = None
        self.workspace = None
        self.capacity = 0
        self.staging = [torch.empty((height, width, 4), dtype=torch.float16, device=dev)
                        for _ in range(2)]
        self.copy_stream = torch.cuda.Stream(device=dev)
        self.copied = [None, None]  # event: staging slot free again

    def render(self, cam, image, rect=None):
        """Cached render of the partition on `cam` into `image` (fp16 [H, W, 4],
        on the GPU), and its coverage box into `rect` (int32 [4], optional), on
        the current stream. Returns the intersection count."""
        if (cam.width, cam.height) != (self.W, self.H):
            raise ValueError("camera size differs from the refresher's")
        api.project(cam, self.prm, **self.params, out=self.proj)
        b = api.bin_sort(self.W, self.H, self.proj, capacity=self.capacity,
                         workspace=self.workspace, values=self.values,
                         tile_ranges=self.tile_ranges, tile_order=self.tile_order, sync=True)
        self.values, self.workspace, self.capacity = b["values"], b["workspace"], b["capacity"]
        api.render_cache(cam, self.prm, b, self.proj, image=image, rect=rect)
        return b["n_isect"]

    def refresh(self, cams, host_images, rects=None):
        """Re-render the partition for every camera in `cams` into the pinned
        host fp16 images host_images[i] ([H, W, 4] each), and each image's
        coverage box into rects[i] (int32 [len(cams), 4] on the GPU, optional).
        Returns when every copy has landed."""
        if len(host_images) < len(cams):
            raise ValueError("one host image per camera is needed")
        for h in host_images[:len(cams)]:
            if h.is_cuda or not h.is_pinned() or h.dtype != torch.float16 or \
                    tuple(h.shape) != (self.H, self.W, 4):
                raise ValueError("host images must be pinned fp16 [H, W, 4] tensors")
        compute = torch.cuda.current_stream()
        for i, cam in enumerate(cams):
            slot = i & 1
            if self.copied[slot] is not None:
                compute.wait_event(self.copied[slot])
            img = self.staging[slot]
            self.render(cam, img, None if rects is None else rects[i])
            done = torch.cuda.Event()
            done.record(compute)
            with torch.cuda.stream(self.copy_stream):
                self.copy_stream.wait_event(done)
                host_images[i].copy_(img, non_blocking=True)
                ev = torch.cuda.Event()
                ev.record(self.copy_stream)
            self.copied[slot] = ev
        self.copy_stream.synchronize()

"""One ABCD active-block step on one camera, with every buffer allocated once.

The paper's inner loop (Method section): for a sampled camera observing the
active partition, render only the active partition, composite it with that
camera's F and B, evaluate the reconstruction loss and back-propagate into the
active parameters only. F and B come from collapsing the camera's cached
frozen-partition renders (composite_cache), done once per (block, camera).

This class only owns buffers and issues the C-ABI calls in order on the
current stream; it never synchronises unless asked for the intersection count.
"""
import torch

from . import api


class ActiveBlockStep:
    # below this many active Gaussians the backward's split does not pay for
    # its extra launches (the lists are short)
    SPLIT_MIN_GAUSSIANS = 16384

    def __init__(self, cam, prm, params, capacity=None, headroom=1.25, bg=None, chunk="auto"):
        self.cam, self.prm, self.params = cam, prm, params
        self.bg = bg
        n = params["means"].shape[0]
        dev = params["means"].device
        H, W = cam.height, cam.width
        f32 = torch.float32
        self.proj = dict(means2d=torch.empty((n, 2), dtype=f32, device=dev),
                         conic_opacity=torch.empty((n, 4), dtype=f32, device=dev),
                         depth=torch.empty((n,), dtype=f32, device=dev),
                         extent=torch.empty((n, 2), dtype=f32, device=dev),
                         tiles_touched=torch.empty((n,), dtype=torch.int32, device=dev),
                         rgb=torch.empty((n, 3), dtype=f32, device=dev))
        self.fwd = dict(out=torch.empty((H, W, 4), dtype=f32, device=dev),
                        final_T=torch.empty((H, W), dtype=f32, device=dev),
                        last=torch.empty((H, W), dtype=torch.int32, device=dev))
        self.dL_dout = torch.empty((H, W, 4), dtype=f32, device=dev)
        self.loss = torch.zeros((1,), dtype=f32, device=dev)
        self.n_blends = torch.zeros((1,), dtype=torch.int64, device=dev)
        self.bwd_ws = torch.empty(max(api.render_bwd_workspace_size(n), 256), dtype=torch.uint8,
                                  device=dev)
        self.tile_ranges = torch.zeros((api.n_tiles(W, H), 2), dtype=torch.int32, device=dev)
        self.tile_order = torch.empty((api.n_tiles(W, H),), dtype=torch.int32, device=dev)
        self.grads = {k: torch.zeros_like(params[k]) for k in
                      ("means", "log_scales", "quats", "opacity_logits", "sh")}
        if capacity is None:
            # size the intersection buffer from one synchronising pass
            api.project(cam, prm, **params, out=self.proj)
            b = api.bin_sort(W, H, self.proj, capacity=0, tile_ranges=self.tile_ranges,
                             tile_order=self.tile_order)
            capacity = int(b["n_isect"] * headroom) + 1024
        self.capacity = capacity
        self.bin_ws = torch.empty(max(api.bin_sort_workspace_size(n, W, H, capacity), 256),
                                  dtype=torch.uint8, device=dev)
        self.values = torch.empty((capacity,), dtype=torch.int32, device=dev)
        self.bins = dict(values=self.values, tile_ranges=self.tile_ranges,
                         tile_order=self.tile_order)
        # checkpoints for splitting long tiles in the backward (chunk=None: no
        # split); slots are taken as walks cross chunk boundaries, heaviest
        # tiles first, so a short pool only leaves light tiles whole
        self.split = None
        if chunk == "auto":
            chunk = 512 if n >= self.SPLIT_MIN_GAUSSIANS else None
        if chunk:
            self.split = api.make_split(self._split_slots(capacity, chunk), chunk, dev)

    def _split_slots(self, capacity, chunk):
        return capacity // (8 * chunk) + api.n_tiles(self.cam.width, self.cam.height) + 1

    def project_and_bin(self, sync=False):
        """With sync=True the intersection count is read back and the buffers
        grow when a camera needs more; without, the capacity must suffice."""
        api.project(self.cam, self.prm, **self.params, out=self.proj)
        b = api.bin_sort(self.cam.width, self.cam.height, self.proj, capacity=self.capacity,
                         workspace=self.bin_ws, values=self.values, tile_ranges=self.tile_ranges,
                         tile_order=self.tile_order,
                         sync=sync)
        if sync and b["values"] is not self.values:
            self.values, self.bin_ws, self.capacity = b["values"], b["workspace"], b["capacity"]
            self.bins["values"] = self.values
            if self.split is not None:
                chunk = self.split["chunk"]
                self.split = api.make_split(self._split_slots(self.capacity, chunk), chunk,
                                            self.values.device)
        return b["n_isect"]

    def overflowed(self):
        """Whether the last binning found more intersections than the capacity
        (reads the count back, so it synchronises). Such a step rendered the
        active block as empty (every tile range is empty) and its gradients
        are zero; call project_and_bin(sync=True) to grow the buffers."""
        return api.intersections(self.bin_ws) > self.capacity

    def forward(self, F=None, B=None):
        return api.render_fwd(self.cam, self.prm, self.bins, self.proj, F=F, B=B,
                              n_blends=self.n_blends, out=self.fwd, split=self.split)

    def loss_grad(self, target):
        return api.loss_l1_grad(self.fwd["out"], target, bg=self.bg, dL_dout=self.dL_dout,
                                loss=self.loss)

    def backward(self, dL_dout, F=None, B=None):
        return api.render_bwd(self.cam, self.prm, self.params, self.proj, self.bins, self.fwd,
                              dL_dout, F=F, B=B, workspace=self.bwd_ws, grads=self.grads,
                              split=self.split)

    def step(self, target, F=None, B=None):
        """project -> bin -> forward -> L1 gradient -> backward (no synchronisation)."""
        self.project_and_bin(sync=False)
        self.forward(F, B)
        self.loss_grad(target)
        return self.backward(self.dL_dout, F, B)

    def capture(self, target, F=None, B=None, before=None):
        """Record one step (and `before()`, e.g. the F/B collapse, ahead of it)
        as a HIP graph; replay() then launches the whole step at once. Every
        buffer the step touches is owned here or passed in, so a replay reads
        the current contents of params, target, F and B. The graph holds no
        memset nodes: the library clears with its own fill kernel."""
        def body():
            if before is not None:
                before()
            self.step(target, F, B)

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            body()  # one eager pass on the capture stream first
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            body()
        self.graph = graph
        return graph

    def replay(self):
        """Launch the captured step on the current stream (check overflowed()
        when the parameters or the camera may have grown the intersection
        count past the capacity)."""
        self.graph.replay()
        return self.grads

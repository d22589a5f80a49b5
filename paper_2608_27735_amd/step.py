"""One ABCD active-block step on one camera, with every buffer allocated once.

The paper's inner loop (Method section): for a sampled camera observing the
active partition, render only the active partition, composite it with that
camera's F and B, evaluate the reconstruction loss and back-propagate into the
active parameters only. F and B come from collapsing the camera's cached
frozen-partition renders (composite_cache), done once per (block, camera).

This class only owns buffers and issues the C-ABI calls in order on the
current stream; it never synchronises unless asked for the intersection count.
"""
import ctypes as C

import torch

from . import _lib, api


class ActiveBlockStep:
    # below this many active Gaussians the backward's split does not pay for
    # its extra launches (the lists are short)
    SPLIT_MIN_GAUSSIANS = 16384

    def __init__(self, cam, prm, params, capacity=None, headroom=1.25, bg=None, chunk="auto"):
        self._fast = None
        self._side = None  # second stream of step(collapse=...), made on first use
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

    @property
    def cam(self):
        return self._cam

    @cam.setter
    def cam(self, cam):
        self._cam = cam
        self._fast = None  # the prepared arguments hold the camera

    def _prepared(self):
        """ctypes arguments of the step's five calls, built once per camera and
        set of buffers: a step then passes only F, B, the target and the
        current stream (argument marshalling costs microseconds per call, which
        adds up for small active blocks whose kernels take a few)."""
        if self._fast is not None:
            return self._fast
        lib = _lib.load()
        cam_s, prm_s = _lib.camera_struct(self.cam), _lib.params_struct(self.prm)
        P, p, g = self.proj, self.params, self.grads
        n = p["means"].shape[0]
        W, H = self.cam.width, self.cam.height
        dev = p["means"].device
        nz = lambda t: api._ptr_nz(t, dev)
        split = None
        if self.split is not None:
            ws = self.split["workspace"]
            split = _lib.abcd_split(ws.data_ptr(), ws.numel(), int(self.split["chunk"]), 0)
        sp = C.byref(split) if split is not None else None
        bg = None if self.bg is None else (C.c_float * 3)(*[float(x) for x in self.bg])
        params = [p[k].data_ptr() for k in ("means", "log_scales", "quats", "opacity_logits", "sh")]
        self._fast = dict(
            keep=(cam_s, prm_s, split, bg), lib=lib, W=W, H=H, bg=bg,
            project=(C.byref(cam_s), C.byref(prm_s), n, *params, P["means2d"].data_ptr(),
                     P["conic_opacity"].data_ptr(), P["depth"].data_ptr(),
                     P["extent"].data_ptr(), P["tiles_touched"].data_ptr(), P["rgb"].data_ptr()),
            bin=(W, H, n, P["means2d"].data_ptr(), P["extent"].data_ptr(), P["depth"].data_ptr(),
                 P["tiles_touched"].data_ptr(), self.capacity, self.bin_ws.data_ptr(),
                 self.bin_ws.numel(), None, nz(self.values), self.tile_ranges.data_ptr(),
                 self.tile_order.data_ptr(), None),
            fwd_pre=(C.byref(cam_s), C.byref(prm_s), self.tile_ranges.data_ptr(),
                     self.tile_order.data_ptr(), nz(self.values), nz(P["means2d"]),
                     nz(P["conic_opacity"]), nz(P["rgb"])),
            fwd_post=(self.fwd["out"].data_ptr(), self.fwd["final_T"].data_ptr(),
                      self.fwd["last"].data_ptr(), self.n_blends.data_ptr(), sp),
            loss=(self.fwd["out"].data_ptr(),),
            loss_post=(bg, self.dL_dout.data_ptr(), self.loss.data_ptr()),
            bwd_pre=(C.byref(cam_s), C.byref(prm_s), n, *params, P["means2d"].data_ptr(),
                     P["conic_opacity"].data_ptr(), P["rgb"].data_ptr(), P["extent"].data_ptr(),
                     self.tile_ranges.data_ptr(), nz(self.values)),
            bwd_post=(self.fwd["final_T"].data_ptr(), self.fwd["last"].data_ptr()),
            bwd_tail=(self.bwd_ws.data_ptr(), self.bwd_ws.numel(),
                      *[g[k].data_ptr() for k in ("means", "log_scales", "quats",
                                                  "opacity_logits", "sh")],
                      None, 0, sp),
            checked=set())
        return self._fast

    def _image(self, t, name, channels, f):
        """Shape/dtype/device check of an image argument, once per tensor."""
        if t is None:
            return None
        if id(t) not in f["checked"]:
            api._need(t, name, torch.float32, (self.cam.height, self.cam.width, channels))
            f["checked"].add(id(t))
            f.setdefault("alive", []).append(t)  # keeps the id from being reused
        return t.data_ptr()

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
            self._fast = None
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

    def step(self, target, F=None, B=None, collapse=None):
        """project -> bin -> forward -> L1 gradient -> backward (no synchronisation),
        the same calls as project_and_bin(), forward(), loss_grad() and
        backward() with their arguments prepared once (see _prepared).

        collapse (optional callable): the work that writes F and B (the
        collapse of the frozen partitions' cached renders). It is enqueued on
        a second stream once the projection is done (so also the previous
        step's backward, which reads F and B), and runs beside the binning,
        which does not read F or B; the forward waits for it."""
        f = self._prepared()
        lib, st = f["lib"], api._stream()
        Fp, Bp = self._image(F, "F", 4, f), self._image(B, "B", 4, f)
        tp = self._image(target, "target", 3, f)
        main = torch.cuda.current_stream()
        _lib.check(lib.abcd_project(*f["project"], st))
        if collapse is not None:
            # after the projection (both are bound by memory bandwidth), beside
            # the binning (mostly bound by latency)
            if self._side is None:
                self._side = torch.cuda.Stream()  # default priority
                self._fork, self._join = torch.cuda.Event(), torch.cuda.Event()
            self._fork.record(main)
            self._side.wait_event(self._fork)
            with torch.cuda.stream(self._side):
                collapse()
            self._join.record(self._side)
        _lib.check(lib.abcd_bin_sort(*f["bin"], st))
        if collapse is not None:
            main.wait_event(self._join)
        _lib.check(lib.abcd_render_fwd(*f["fwd_pre"], Fp, Bp, *f["fwd_post"], st))
        _lib.check(lib.abcd_loss_l1_grad(f["W"], f["H"], *f["loss"], tp, *f["loss_post"], st))
        _lib.check(lib.abcd_render_bwd(*f["bwd_pre"], Fp, Bp, *f["bwd_post"], self.dL_dout.data_ptr(),
                                       *f["bwd_tail"], st))
        return self.grads

    def capture(self, target, F=None, B=None, before=None):
        """Record one step (and `before()`, e.g. the F/B collapse, beside its
        projection and binning as in step(collapse=...)) as a HIP graph;
        replay() then launches the whole step at once. Every buffer the step
        touches is owned here or passed in, so a replay reads the current
        contents of params, target, F and B. The graph holds no memset nodes:
        the library clears with its own fill kernel."""
        def body():
            self.step(target, F, B, collapse=before)

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

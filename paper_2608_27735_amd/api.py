"""Python binding of the ABCD C ABI (include/abcd.h) for torch tensors on the GPU.

Argument marshalling only: tensors are checked for device, dtype and layout,
their device pointers and the current HIP stream are passed to libabcd.so,
and every step runs in the library's kernels. There is no CPU fallback.
"""
import ctypes as C

import torch

from . import _lib
from ._lib import AbcdError, check

_lib.load()  # no fallback: the binding is unusable without the built library


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


_dummies = {}


def _ptr_nz(t, device):
    """Device pointer of t; for a missing or empty tensor (whose pointer may be
    NULL) a small placeholder buffer on the device that no kernel reads (the
    library requires these input pointers to be non-NULL)."""
    if t is not None and t.numel() > 0:
        return t.data_ptr()
    d = _dummies.get(device)
    if d is None:
        d = _dummies[device] = torch.zeros(64, dtype=torch.float32, device=device)
    return d.data_ptr()


def _need(t, name, dtype, shape=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _opt(t, name, dtype, shape=None):
    return None if t is None else _need(t, name, dtype, shape)


def n_tiles(width, height):
    return ((width + 15) // 16) * ((height + 15) // 16)


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def version():
    return _lib.load().abcd_version().decode()


# ------------------------------------------------------------------ project

def project(cam, prm, means, log_scales, quats, opacity_logits, sh, out=None):
    """EWA projection; returns dict(means2d, conic_opacity, depth, extent
    (n, 2: half extents of the binning box), tiles_touched (int32 view of
    uint32), rgb)."""
    n = means.shape[0]
    nc = (prm.sh_degree + 1) ** 2
    f32 = torch.float32
    _need(means, "means", f32, (n, 3))
    _need(log_scales, "log_scales", f32, (n, 3))
    _need(quats, "quats", f32, (n, 4))
    _need(opacity_logits, "opacity_logits", f32, (n,))
    _need(sh, "sh", f32, (n, nc, 3))
    dev = means.device
    if out is None:
        out = dict(means2d=_empty((n, 2), f32, dev), conic_opacity=_empty((n, 4), f32, dev),
                   depth=_empty((n,), f32, dev), extent=_empty((n, 2), f32, dev),
                   tiles_touched=_empty((n,), torch.int32, dev), rgb=_empty((n, 3), f32, dev))
    lib = _lib.load()
    check(lib.abcd_project(C.byref(_lib.camera_struct(cam)), C.byref(_lib.params_struct(prm)), n,
                           _ptr(means), _ptr(log_scales), _ptr(quats), _ptr(opacity_logits),
                           _ptr(sh), _ptr(out["means2d"]), _ptr(out["conic_opacity"]),
                           _ptr(out["depth"]), _ptr(out["extent"]), _ptr(out["tiles_touched"]),
                           _ptr(out["rgb"]), _stream()))
    return out


# ------------------------------------------------------------------ binning

def bin_sort_workspace_size(n, width, height, capacity=0):
    sz = C.c_size_t(0)
    check(_lib.load().abcd_bin_sort_workspace_size(n, capacity, width, height, C.byref(sz)))
    return sz.value


def bin_sort(width, height, proj, capacity=None, workspace=None, values=None, keys=None,
             tile_ranges=None, tile_order=None, want_keys=False, sync=True):
    """Per-tile depth-sorted lists. Returns dict(values, tile_ranges, tile_order,
    keys, n_isect); tile_order is the forward's schedule (heaviest lists first).

    With sync=True (default) M is read back (one stream synchronisation) and
    the buffers are grown to fit it; with sync=False the call never
    synchronises and `capacity`/`values` must already be large enough: an
    overflow leaves values unwritten and every tile range empty, and
    intersections(workspace) > capacity tells it afterwards."""
    means2d, extent = proj["means2d"], proj["extent"]
    depth, tiles = proj["depth"], proj["tiles_touched"]
    n = means2d.shape[0]
    dev = means2d.device
    _need(means2d, "means2d", torch.float32, (n, 2))
    _need(extent, "extent", torch.float32, (n, 2))
    _need(depth, "depth", torch.float32, (n,))
    _need(tiles, "tiles_touched", torch.int32, (n,))
    if tile_ranges is None:
        tile_ranges = _empty((n_tiles(width, height), 2), torch.int32, dev)
    if tile_order is None:
        tile_order = _empty((n_tiles(width, height),), torch.int32, dev)
    if capacity is None:
        capacity = 0 if values is None else values.numel()
    ws_bytes = bin_sort_workspace_size(n, width, height, capacity)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    if values is None and capacity > 0:
        values = _empty((capacity,), torch.int32, dev)
    if want_keys and (keys is None or keys.numel() < capacity):
        keys = _empty((max(capacity, 1),), torch.int64, dev)
    lib = _lib.load()
    m = C.c_int64(0)
    st = lib.abcd_bin_sort(width, height, n, _ptr(means2d), _ptr(extent), _ptr(depth), _ptr(tiles),
                           capacity, _ptr(workspace), workspace.numel(),
                           _ptr(keys) if want_keys else None, _ptr(values), _ptr(tile_ranges),
                           _ptr(tile_order), C.byref(m) if sync else None, _stream())
    if st == _lib.ABCD_E_CAPACITY and sync:
        capacity = int(m.value)
        values = _empty((max(capacity, 1),), torch.int32, dev)
        if want_keys:
            keys = _empty((max(capacity, 1),), torch.int64, dev)
        ws_bytes = bin_sort_workspace_size(n, width, height, capacity)
        if workspace.numel() < ws_bytes:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        st = lib.abcd_bin_sort(width, height, n, _ptr(means2d), _ptr(extent), _ptr(depth),
                               _ptr(tiles), capacity, _ptr(workspace), workspace.numel(),
                               _ptr(keys) if want_keys else None, _ptr(values), _ptr(tile_ranges),
                               _ptr(tile_order), C.byref(m), _stream())
    check(st)
    return dict(values=values, tile_ranges=tile_ranges, tile_order=tile_order,
                keys=keys if want_keys else None,
                n_isect=int(m.value) if sync else None, workspace=workspace, capacity=capacity)


def intersections(workspace):
    """The intersection count M the last abcd_bin_sort on this workspace found
    (the uint64 at the workspace's start; reading it synchronises with the
    stream). M > capacity means that call overflowed and rendered nothing."""
    return int(workspace[:8].cpu().view(torch.int64).item())


# -------------------------------------------------------------- rasterise

def split_workspace_size(n_slots):
    sz = C.c_size_t(0)
    check(_lib.load().abcd_split_workspace_size(int(n_slots), C.byref(sz)))
    return sz.value


def make_split(n_slots, chunk=2048, device=None):
    """A split workspace (see abcd_split) with n_slots checkpoint slots; give
    the same one to a forward and its backward."""
    dev = device or torch.device("cuda", torch.cuda.current_device())
    ws = torch.empty(split_workspace_size(n_slots), dtype=torch.uint8, device=dev)
    return dict(workspace=ws, chunk=int(chunk))


def _split_struct(split):
    if split is None:
        return None
    ws = split["workspace"]
    if not ws.is_cuda or ws.dtype != torch.uint8:
        raise ValueError("split workspace must be a uint8 GPU tensor")
    return C.byref(_lib.abcd_split(ws.data_ptr(), ws.numel(), int(split["chunk"]), 0))


def render_fwd(cam, prm, bins, proj, F=None, B=None, n_blends=None, out=None, split=None):
    """out = F over A over B; returns dict(out, final_T, last). split: see
    make_split (the backward must get the same one)."""
    H, W = cam.height, cam.width
    dev = proj["means2d"].device
    _opt(F, "F", torch.float32, (H, W, 4))
    _opt(B, "B", torch.float32, (H, W, 4))
    _opt(n_blends, "n_blends", torch.int64, (1,))
    if out is None:
        out = dict(out=_empty((H, W, 4), torch.float32, dev),
                   final_T=_empty((H, W), torch.float32, dev),
                   last=_empty((H, W), torch.int32, dev))
    lib = _lib.load()
    check(lib.abcd_render_fwd(C.byref(_lib.camera_struct(cam)), C.byref(_lib.params_struct(prm)),
                              _ptr(bins["tile_ranges"]), _ptr(bins.get("tile_order")),
                              _ptr_nz(bins["values"], dev), _ptr_nz(proj["means2d"], dev),
                              _ptr_nz(proj["conic_opacity"], dev), _ptr_nz(proj["rgb"], dev),
                              _ptr(F), _ptr(B), _ptr(out["out"]), _ptr(out["final_T"]),
                              _ptr(out["last"]), _ptr(n_blends), _split_struct(split), _stream()))
    return out


def render_cache(cam, prm, bins, proj, image=None, rect=None):
    """The partition rendered alone (F = B = transparent) as premultiplied fp16
    RGBA [H, W, 4] (torch.float16), the form abcd_composite_cache consumes.
    rect: optional int32 [4] GPU tensor that receives the coverage box."""
    H, W = cam.height, cam.width
    if image is None:
        image = _empty((H, W, 4), torch.float16, proj["means2d"].device)
    _need(image, "image", torch.float16, (H, W, 4))
    _opt(rect, "rect", torch.int32, (4,))
    dev = proj["means2d"].device
    check(_lib.load().abcd_render_cache(
        C.byref(_lib.camera_struct(cam)), C.byref(_lib.params_struct(prm)),
        _ptr(bins["tile_ranges"]), _ptr(bins.get("tile_order")), _ptr_nz(bins["values"], dev),
        _ptr_nz(proj["means2d"], dev), _ptr_nz(proj["conic_opacity"], dev),
        _ptr_nz(proj["rgb"], dev), _ptr(image),
        _ptr(rect), _stream()))
    return image


def render_bwd_workspace_size(n):
    sz = C.c_size_t(0)
    check(_lib.load().abcd_render_bwd_workspace_size(n, C.byref(sz)))
    return sz.value


def render_bwd(cam, prm, params, proj, bins, fwd, dL_dout, F=None, B=None, workspace=None,
               grads=None, accumulate=False, want_means2d=False, split=None):
    """Gradients of the active parameters; returns dict(means, log_scales, quats,
    opacity_logits, sh[, means2d])."""
    n = params["means"].shape[0]
    H, W = cam.height, cam.width
    dev = params["means"].device
    _need(dL_dout, "dL_dout", torch.float32, (H, W, 4))
    _opt(F, "F", torch.float32, (H, W, 4))
    _opt(B, "B", torch.float32, (H, W, 4))
    ws_bytes = render_bwd_workspace_size(n)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    if grads is None:
        grads = {k: torch.zeros_like(params[k]) for k in
                 ("means", "log_scales", "quats", "opacity_logits", "sh")}
        if want_means2d:
            grads["means2d"] = torch.zeros((n, 2), dtype=torch.float32, device=dev)
    lib = _lib.load()
    check(lib.abcd_render_bwd(
        C.byref(_lib.camera_struct(cam)), C.byref(_lib.params_struct(prm)), n,
        _ptr(params["means"]), _ptr(params["log_scales"]), _ptr(params["quats"]),
        _ptr(params["opacity_logits"]), _ptr(params["sh"]), _ptr(proj["means2d"]),
        _ptr(proj["conic_opacity"]), _ptr(proj["rgb"]), _ptr(proj["extent"]),
        _ptr(bins["tile_ranges"]), _ptr_nz(bins["values"], dev), _ptr(F), _ptr(B),
        _ptr(fwd["final_T"]),
        _ptr(fwd["last"]), _ptr(dL_dout), _ptr(workspace), workspace.numel(), _ptr(grads["means"]),
        _ptr(grads["log_scales"]), _ptr(grads["quats"]), _ptr(grads["opacity_logits"]),
        _ptr(grads["sh"]), _ptr(grads.get("means2d")), 1 if accumulate else 0,
        _split_struct(split), _stream()))
    return grads


def render_bwd_noalloc(cam, prm, params, proj, bins, fwd, dL_dout, F=None, B=None, grads=None,
                       accumulate=False, want_means2d=False, split=None):
    """render_bwd through abcd_render_bwd_noalloc: no workspace, the library's
    static per-GPU scratch instead (n <= NOALLOC_MAX_GAUSSIANS; calls that
    overlap on one GPU race). `grads` should be preallocated by callers that
    must not allocate."""
    n = params["means"].shape[0]
    H, W = cam.height, cam.width
    dev = params["means"].device
    _need(dL_dout, "dL_dout", torch.float32, (H, W, 4))
    _opt(F, "F", torch.float32, (H, W, 4))
    _opt(B, "B", torch.float32, (H, W, 4))
    if grads is None:
        grads = {k: torch.zeros_like(params[k]) for k in
                 ("means", "log_scales", "quats", "opacity_logits", "sh")}
        if want_means2d:
            grads["means2d"] = torch.zeros((n, 2), dtype=torch.float32, device=dev)
    check(_lib.load().abcd_render_bwd_noalloc(
        C.byref(_lib.camera_struct(cam)), C.byref(_lib.params_struct(prm)), n,
        _ptr(params["means"]), _ptr(params["log_scales"]), _ptr(params["quats"]),
        _ptr(params["opacity_logits"]), _ptr(params["sh"]), _ptr(proj["means2d"]),
        _ptr(proj["conic_opacity"]), _ptr(proj["rgb"]), _ptr(proj["extent"]),
        _ptr(bins["tile_ranges"]), _ptr_nz(bins["values"], dev), _ptr(F), _ptr(B),
        _ptr(fwd["final_T"]), _ptr(fwd["last"]), _ptr(dL_dout), _ptr(grads["means"]),
        _ptr(grads["log_scales"]), _ptr(grads["quats"]), _ptr(grads["opacity_logits"]),
        _ptr(grads["sh"]), _ptr(grads.get("means2d")), 1 if accumulate else 0,
        _split_struct(split), _stream()))
    return grads


# --------------------------------------------------------------- optimizer

PARAM_GROUPS = ("means", "log_scales", "quats", "opacity_logits", "sh")


def adam_step(params, grads, exp_avg, exp_avg_sq, lr, step, beta1=0.9, beta2=0.999, eps=1e-15):
    """One Adam update of the parameter groups (dicts of fp32 GPU tensors, in
    place); lr is a dict (one rate per group) or a float."""
    names = [k for k in params if params[k].numel() > 0]
    if len(names) > _lib.ADAM_MAX_GROUPS:
        raise ValueError("too many parameter groups")
    arr = (_lib.abcd_adam_group * max(len(names), 1))()
    for i, k in enumerate(names):
        for t, nm in ((params[k], "param"), (grads[k], "grad"), (exp_avg[k], "exp_avg"),
                      (exp_avg_sq[k], "exp_avg_sq")):
            _need(t, f"{nm}[{k}]", torch.float32, tuple(params[k].shape))
        arr[i].param, arr[i].grad = _ptr(params[k]), _ptr(grads[k])
        arr[i].exp_avg, arr[i].exp_avg_sq = _ptr(exp_avg[k]), _ptr(exp_avg_sq[k])
        arr[i].count = params[k].numel()
        arr[i].lr = float(lr[k] if isinstance(lr, dict) else lr)
    check(_lib.load().abcd_adam_step(arr, len(names), float(beta1), float(beta2), float(eps),
                                     int(step), _stream()))


# ---------------------------------------------------------------- collapse

def composite_cache(images, order, n_front, F=None, B=None, accumulate=False, rects=None,
                    stop_t=0.0, beside=False):
    """Collapse cached fp16 renders [K, H, W, 4] (torch.float16, or int16
    holding binary16 bits) into F and B (fp32 [H, W, 4]). rects: optional
    int32 [K, 4] GPU tensor of per-image coverage boxes (x0, y0, x1, y1);
    stop_t > 0 skips layers that can no longer be seen. beside: at most two
    workgroups per CU, for a collapse that runs beside other work on another
    stream (slower alone)."""
    if images.dtype not in (torch.float16, torch.int16):
        raise ValueError("images must be float16 (or int16 bit patterns)")
    if not images.is_cuda or not images.is_contiguous() or images.dim() != 4:
        raise ValueError("images must be a contiguous GPU tensor [K, H, W, 4]")
    k, H, W, c = images.shape
    if c != 4:
        raise ValueError("images must be RGBA")
    dev = images.device
    if F is None:
        F = _empty((H, W, 4), torch.float32, dev)
    if B is None:
        B = _empty((H, W, 4), torch.float32, dev)
    _need(F, "F", torch.float32, (H, W, 4))
    _need(B, "B", torch.float32, (H, W, 4))
    _opt(rects, "rects", torch.int32, (k, 4))
    order_arr = (C.c_int32 * max(k, 1))(*[int(x) for x in order])
    check(_lib.load().abcd_composite_cache(W, H, k, _ptr(images), order_arr, int(n_front),
                                           _ptr(rects), float(stop_t), _ptr(F), _ptr(B),
                                           (1 if accumulate else 0) | (2 if beside else 0),
                                           _stream()))
    return F, B


def stage_cached(host_images, dst, rects=None):
    """Copy pinned host fp16 images (a list of [H, W, 4] tensors) into the
    device chunk dst [>= k, H, W, 4], only inside each image's coverage box
    (rects: host int32 array [k, 4], or None for whole images), on the
    current stream."""
    k = len(host_images)
    if k == 0:
        return dst
    H, W = dst.shape[1], dst.shape[2]
    if dst.dtype not in (torch.float16, torch.int16) or not dst.is_cuda or \
            not dst.is_contiguous() or dst.shape[0] < k or dst.shape[3] != 4:
        raise ValueError("dst must be a contiguous fp16 GPU tensor [>= k, H, W, 4]")
    for h in host_images:
        if h.is_cuda or not h.is_pinned() or h.dtype not in (torch.float16, torch.int16) or \
                tuple(h.shape) != (H, W, 4) or not h.is_contiguous():
            raise ValueError("host images must be pinned contiguous fp16 [H, W, 4] tensors")
    ptrs = (C.c_void_p * k)(*[h.data_ptr() for h in host_images])
    r = None
    if rects is not None:
        import numpy as np
        ra = np.ascontiguousarray(np.asarray(rects, dtype=np.int32).reshape(-1, 4)[:k])
        r = ra.ctypes.data_as(C.POINTER(C.c_int32))
    check(_lib.load().abcd_stage_cached(W, H, k, ptrs, r, _ptr(dst), _stream()))
    return dst


def loss_l1_grad(out, target, bg=None, dL_dout=None, loss=None):
    H, W = out.shape[:2]
    _need(out, "out", torch.float32, (H, W, 4))
    _need(target, "target", torch.float32, (H, W, 3))
    _opt(loss, "loss", torch.float32, (1,))
    if dL_dout is None:
        dL_dout = torch.empty_like(out)
    bg_arr = None if bg is None else (C.c_float * 3)(*[float(x) for x in bg])
    check(_lib.load().abcd_loss_l1_grad(W, H, _ptr(out), _ptr(target), bg_arr, _ptr(dL_dout),
                                        _ptr(loss), _stream()))
    return dL_dout


# ------------------------------------------------------------------ timing

def timing_enable(flag=True):
    check(_lib.load().abcd_timing_enable(1 if flag else 0))


def timing_reset():
    check(_lib.load().abcd_timing_reset())


def timing_read(kernel):
    ms = C.c_double(0)
    cnt = C.c_int64(0)
    check(_lib.load().abcd_timing_read(kernel.encode(), C.byref(ms), C.byref(cnt)))
    return ms.value, cnt.value


__all__ = ["AbcdError", "project", "bin_sort", "bin_sort_workspace_size", "render_fwd",
           "render_bwd", "render_bwd_workspace_size", "composite_cache", "loss_l1_grad",
           "timing_enable", "timing_reset", "timing_read", "version", "n_tiles", "adam_step",
           "render_cache", "stage_cached", "make_split", "split_workspace_size", "intersections",
           "render_bwd_noalloc"]

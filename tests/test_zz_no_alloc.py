"""The allocation-free backward (abcd_render_bwd_noalloc) against the
workspace backward (abcd_render_bwd) through the C ABI: the same gradients
within the parity bar on two calls in a row, the second with a smaller input
(the static scratch keeps the first call's contents, which the second must
not see), and a size above the static scratch's limit rejected on the host."""
import math

import numpy as np
import pytest
import torch

from paper_2608_27735_amd import synthetic as S

pytestmark = pytest.mark.gpu

GRAD_TOL = 1e-4


def say(*a):
    print("[case]", *a, flush=True)


def _case(api, w, cam, mask, seed):
    dev = torch.device("cuda:0")
    sub = S.subset(w.scene, mask)
    params = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in sub.items()}
    r = S.rng(seed)
    F, B = S.background_pair(r, cam.height, cam.width)
    Fd, Bd = torch.from_numpy(F).to(dev), torch.from_numpy(B).to(dev)
    G = torch.from_numpy(S.upstream_grad(r, cam.height, cam.width)).to(dev)
    prm = w.params
    proj = api.project(cam, prm, **params)
    bins = api.bin_sort(cam.width, cam.height, proj)
    split = api.make_split(64, 256, dev)
    fwd = api.render_fwd(cam, prm, bins, proj, F=Fd, B=Bd, split=split)
    return params, proj, bins, fwd, Fd, Bd, G, split


def _rel(a, b):
    a, b = a.double().cpu().numpy(), b.double().cpu().numpy()
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)


def test_noalloc_backward_matches_workspace_backward_twice():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_27735_amd import api
    w = S.ring()
    cam = w.cams[2]
    # first call: the whole 64K scene; second: the active cell only (smaller)
    cases = []
    for name, mask, seed in (("ring-all-cam2", np.ones(len(w.scene["means"]), bool), 31),
                             ("ring-active-cam2", w.cell_of == w.active, 32)):
        say("workspace backward", name, int(mask.sum()))
        params, proj, bins, fwd, Fd, Bd, G, split = _case(api, w, cam, mask, seed)
        ref = api.render_bwd(cam, w.params, params, proj, bins, fwd, G, F=Fd, B=Bd,
                             want_means2d=True, split=split)
        cases.append((name, params, proj, bins, fwd, Fd, Bd, G, split, ref))
    torch.cuda.synchronize()
    got = []
    for name, params, proj, bins, fwd, Fd, Bd, G, split, ref in cases:  # two calls in a row
        say("noalloc backward", name)
        got.append(api.render_bwd_noalloc(cam, w.params, params, proj, bins, fwd, G, F=Fd, B=Bd,
                                          want_means2d=True, split=split))
    torch.cuda.synchronize()
    for (name, *_, ref), g in zip(cases, got):
        for k in ("means", "log_scales", "quats", "opacity_logits", "sh", "means2d"):
            rel = _rel(g[k], ref[k])
            print(f"  {name} {k}: rel L2 {rel:.2e}")
            assert torch.linalg.norm(ref[k].double()) > 0, k
            assert rel <= GRAD_TOL, (name, k, rel)


def test_noalloc_rejects_more_gaussians_than_its_scratch_holds():
    """Host-side rejection: nothing is enqueued (no GPU work happens)."""
    import ctypes as C
    from paper_2608_27735_amd import _lib
    lib = _lib.load()
    cam = S.ring().cams[0]
    c, p = _lib.camera_struct(cam), _lib.params_struct(S.ring().params)
    fake = 0x1000
    args = [fake] * 16 + [fake] * 6 + [0, None, None]
    st = lib.abcd_render_bwd_noalloc(C.byref(c), C.byref(p), _lib.NOALLOC_MAX_GAUSSIANS + 1,
                                     *args)
    assert st == _lib.ABCD_E_INVALID
    assert "static scratch" in lib.abcd_last_error().decode()

"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/abcd.h, and rejects invalid arguments on the host before
any HIP call (so these calls never launch a kernel)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2608_27735_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2608_27735_amd import build
        build.build()
    return _lib.load()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "abcd.h")).read()
    return sorted(set(re.findall(r"ABCD_API\s+[\w\s\*]*?\b(abcd_\w+)\s*\(", text)))


def test_header_declares_the_five_calls_and_helpers():
    names = declared_functions()
    for n in ("abcd_project", "abcd_bin_sort", "abcd_render_fwd", "abcd_render_bwd",
              "abcd_composite_cache", "abcd_bin_sort_workspace_size",
              "abcd_render_bwd_workspace_size", "abcd_last_error", "abcd_version"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    from paper_2608_27735_amd import _lib
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, n


def test_only_the_c_abi_is_exported():
    out = os.popen("nm -D --defined-only " + os.path.join(ROOT, "paper_2608_27735_amd",
                                                          "libabcd.so")).read()
    funcs = [l.split()[-1] for l in out.splitlines() if " T " in l]
    assert funcs and all(f.startswith("abcd_") for f in funcs), funcs


def test_version_and_status_strings(lib):
    assert lib.abcd_version().decode().startswith("abcd-gfx950")
    assert lib.abcd_status_string(2).decode() == "ABCD_E_CAPACITY"


def _cam(width=64, height=48):
    from paper_2608_27735_amd import _lib
    c = _lib.abcd_camera()
    c.width, c.height, c.fx, c.fy, c.cx, c.cy = width, height, 50.0, 50.0, 32.0, 24.0
    for i in range(9):
        c.R[i] = 1.0 if i in (0, 4, 8) else 0.0
    c.near_plane = 0.2
    return c


def _prm(**kw):
    from paper_2608_27735_amd import _lib
    p = _lib.abcd_raster_params()
    p.alpha_min, p.alpha_max, p.t_min, p.eps2d, p.radius_sigmas, p.guard = \
        1 / 255, 0.99, 1e-4, 0.3, 3.0, 1.3
    p.sh_degree, p.flags = 0, 0
    for k, v in kw.items():
        setattr(p, k, v)
    return p


FAKE = 0x1000  # never dereferenced: every call below fails validation first


@pytest.mark.parametrize("mutate", [
    lambda c, p: setattr(c, "width", 0),
    lambda c, p: setattr(c, "fx", -1.0),
    lambda c, p: setattr(c, "fx", float("nan")),
    lambda c, p: setattr(c, "near_plane", 0.0),   # depth keys need positive depths
    lambda c, p: setattr(c, "near_plane", -0.5),
    lambda c, p: setattr(p, "sh_degree", 4),
    lambda c, p: setattr(p, "alpha_max", 1.0),
    lambda c, p: setattr(p, "flags", 2),  # unknown flag bit
    lambda c, p: (setattr(c, "width", 16 * 400), setattr(c, "height", 16 * 100)),  # 40000 tiles
])
def test_project_rejects_bad_camera_or_params(lib, mutate):
    c, p = _cam(), _prm()
    mutate(c, p)
    st = lib.abcd_project(C.byref(c), C.byref(p), 10, *([FAKE] * 11), None)
    assert st == 1


def test_project_rejects_null_and_misaligned(lib):
    c, p = _cam(), _prm()
    assert lib.abcd_project(None, C.byref(p), 10, *([FAKE] * 11), None) == 1
    args = [FAKE] * 11
    args[3] = None  # opacity_logits
    assert lib.abcd_project(C.byref(c), C.byref(p), 10, *args, None) == 1
    args = [FAKE] * 11
    args[6] = FAKE + 4  # conic_opacity not 16-byte aligned
    assert lib.abcd_project(C.byref(c), C.byref(p), 10, *args, None) == 1
    assert lib.abcd_project(C.byref(c), C.byref(p), -1, *([FAKE] * 11), None) == 1
    assert "aligned" in lib.abcd_last_error().decode() or lib.abcd_last_error()


def test_workspace_size_helpers_are_host_only(lib):
    sz = C.c_size_t(0)
    assert lib.abcd_bin_sort_workspace_size(1_000_000, 0, 1297, 840, C.byref(sz)) == 0
    assert sz.value > 16 * 1_000_000
    big = C.c_size_t(0)
    assert lib.abcd_bin_sort_workspace_size(1_000_000, 10_000_000, 1297, 840, C.byref(big)) == 0
    assert big.value >= sz.value + 4 * 10_000_000
    small = C.c_size_t(0)
    assert lib.abcd_bin_sort_workspace_size(0, 0, 16, 16, C.byref(small)) == 0
    assert small.value >= 256
    assert lib.abcd_bin_sort_workspace_size(10, 0, 0, 16, C.byref(sz)) == 1
    assert lib.abcd_bin_sort_workspace_size(10, 1 << 33, 16, 16, C.byref(sz)) == 1
    assert lib.abcd_render_bwd_workspace_size(1000, C.byref(sz)) == 0
    assert sz.value >= 9 * 4 * 1000 + 16 * 32768 and sz.value % 256 == 0


def test_bin_sort_rejects_small_or_misaligned_workspace(lib):
    need = C.c_size_t(0)
    lib.abcd_bin_sort_workspace_size(100, 1000, 64, 48, C.byref(need))
    m = C.c_int64(0)
    base = [64, 48, 100, FAKE, FAKE, FAKE, FAKE, 1000]
    tail = [None, FAKE, FAKE, FAKE, C.byref(m), None]
    assert lib.abcd_bin_sort(*base, FAKE + 8, need.value, *tail) == 1
    assert lib.abcd_bin_sort(*base, FAKE, need.value - 1, *tail) == 1
    base[7] = -1  # negative capacity
    assert lib.abcd_bin_sort(*base, FAKE, need.value, *tail) == 1


def test_composite_rejects_bad_order(lib):
    def call(k, order, n_front, F=FAKE, rects=None, stop_t=0.0, flags=0):
        return lib.abcd_composite_cache(8, 8, k, FAKE, order, n_front, rects, stop_t, F, FAKE,
                                        flags, None)
    order = (C.c_int32 * 3)(0, 0, 2)
    assert call(3, order, 1) == 1
    order = (C.c_int32 * 3)(0, 1, 3)
    assert call(3, order, 1) == 1
    order = (C.c_int32 * 3)(2, 1, 0)
    assert call(3, order, 4) == 1
    assert call(-1, order, 0) == 1
    assert call(3, order, 1, F=None) == 1
    assert call(3, order, 1, rects=FAKE + 4) == 1   # rects misaligned
    assert call(3, order, 1, stop_t=-0.1) == 1
    assert call(3, order, 1, stop_t=1.0) == 1
    assert call(3, order, 1, stop_t=float("nan")) == 1
    assert call(3, order, 1, flags=4) == 1  # unknown flag bit
    assert call(3, order, 1, flags=-1) == 1


def test_render_calls_reject_bad_arguments(lib):
    c, p = _cam(), _prm()
    args = [FAKE] * 12
    args[0] = None  # tile_ranges
    assert lib.abcd_render_fwd(C.byref(c), C.byref(p), *args, None, None) == 1
    args = [FAKE] * 12
    args[6] = FAKE + 4  # F misaligned
    assert lib.abcd_render_fwd(C.byref(c), C.byref(p), *args, None, None) == 1
    cache = [FAKE] * 7 + [None]
    cache[6] = None  # image
    assert lib.abcd_render_cache(C.byref(c), C.byref(p), *cache, None) == 1
    cache = [FAKE] * 7 + [None]
    cache[6] = FAKE + 2  # image misaligned
    assert lib.abcd_render_cache(C.byref(c), C.byref(p), *cache, None) == 1
    cache = [FAKE] * 8
    cache[7] = FAKE + 2  # rect misaligned
    assert lib.abcd_render_cache(C.byref(c), C.byref(p), *cache, None) == 1
    bwd = [FAKE] * 16 + [FAKE, 1 << 20] + [FAKE] * 6 + [0, None, None]
    bwd[13] = None  # final_T
    assert lib.abcd_render_bwd(C.byref(c), C.byref(p), 10, *bwd) == 1
    bwd = [FAKE] * 16 + [FAKE, 8] + [FAKE] * 6 + [0, None, None]  # workspace too small
    assert lib.abcd_render_bwd(C.byref(c), C.byref(p), 10, *bwd) == 1
    assert lib.abcd_loss_l1_grad(0, 8, FAKE, FAKE, None, FAKE, None, None) == 1


@pytest.mark.parametrize("which", [2, 3, 4, 5])  # values_sorted, means2d, conic_opacity, rgb
def test_blend_inputs_may_not_be_null(lib, which):
    """A NULL list or splat array with non-empty tile ranges would fault the
    GPU; both blend entry points reject it on the host instead."""
    c, p = _cam(), _prm()
    args = [FAKE] * 12
    args[which] = None
    assert lib.abcd_render_fwd(C.byref(c), C.byref(p), *args, None, None) == 1
    cache = [FAKE] * 7 + [None]
    cache[which] = None
    assert lib.abcd_render_cache(C.byref(c), C.byref(p), *cache, None) == 1
    bwd = [FAKE] * 16 + [FAKE, 1 << 30] + [FAKE] * 6 + [0, None, None]
    bwd[10] = None  # values_sorted of the backward
    assert lib.abcd_render_bwd(C.byref(c), C.byref(p), 10, *bwd) == 1


def test_split_workspace_and_rejections(lib):
    from paper_2608_27735_amd import _lib
    sz = C.c_size_t(0)
    assert lib.abcd_split_workspace_size(1, C.byref(sz)) == 0
    one = sz.value
    assert lib.abcd_split_workspace_size(11, C.byref(sz)) == 0
    assert sz.value - one == 10 * (4096 + 8) or sz.value - one >= 10 * 4096
    assert lib.abcd_split_workspace_size(0, C.byref(sz)) == 1
    c, p = _cam(), _prm()
    args = [FAKE] * 12
    for ws, nbytes, chunk in ((FAKE + 8, 1 << 30, 256),   # misaligned
                              (FAKE, 1 << 30, 300),       # chunk not a multiple of 256
                              (FAKE, 1 << 30, 0),
                              (FAKE, 1 << 30, 1 << 25),   # chunk above 2^24
                              (FAKE, 64, 256)):           # no room for a slot
        sp = _lib.abcd_split(ws, nbytes, chunk, 0)
        assert lib.abcd_render_fwd(C.byref(c), C.byref(p), *args, C.byref(sp), None) == 1
    bwd = [FAKE] * 16 + [FAKE, 1 << 30] + [FAKE] * 6 + [0]
    sp = _lib.abcd_split(FAKE, 1 << 30, 100, 0)
    assert lib.abcd_render_bwd(C.byref(c), C.byref(p), 10, *bwd, C.byref(sp), None) == 1


def test_adam_rejects_bad_arguments(lib):
    from paper_2608_27735_amd import _lib
    g = (_lib.abcd_adam_group * 9)()
    for i in range(9):
        g[i].param = g[i].grad = g[i].exp_avg = g[i].exp_avg_sq = FAKE
        g[i].count, g[i].lr = 16, 1e-3
    assert lib.abcd_adam_step(g, 9, 0.9, 0.999, 1e-15, 1, None) == 1   # too many groups
    assert lib.abcd_adam_step(g, 1, 1.0, 0.999, 1e-15, 1, None) == 1   # beta1 = 1
    assert lib.abcd_adam_step(g, 1, 0.9, 0.999, -1.0, 1, None) == 1    # eps < 0
    assert lib.abcd_adam_step(g, 1, 0.9, 0.999, 1e-15, 0, None) == 1   # step 0
    g[0].grad = None
    assert lib.abcd_adam_step(g, 1, 0.9, 0.999, 1e-15, 1, None) == 1   # NULL array
    g[0].grad, g[0].count = FAKE, -1
    assert lib.abcd_adam_step(g, 1, 0.9, 0.999, 1e-15, 1, None) == 1   # count < 0
    assert lib.abcd_adam_step(None, 0, 0.9, 0.999, 1e-15, 1, None) == 0  # nothing to do


def test_noalloc_backward_rejects_n_beyond_its_static_scratch(lib):
    """abcd_render_bwd_noalloc holds at most ABCD_NOALLOC_MAX_GAUSSIANS in its
    static scratch; a larger n is rejected on the host before any HIP call."""
    from paper_2608_27735_amd import _lib
    c, p = _cam(), _prm()
    args = [FAKE] * 16 + [FAKE] * 6 + [0, None, None]
    assert lib.abcd_render_bwd_noalloc(C.byref(c), C.byref(p), _lib.NOALLOC_MAX_GAUSSIANS + 1,
                                       *args) == 1
    assert "static scratch" in lib.abcd_last_error().decode()
    args[9] = None  # tile_ranges
    assert lib.abcd_render_bwd_noalloc(C.byref(c), C.byref(p), 10, *args) == 1

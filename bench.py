"""Benchmark of one ABCD active-block step on one MI355X.

A step is one pass of the whole hot path on one camera:
  composite_cache (99 cached fp16 partition renders -> F, B)
  -> project -> bin_sort -> render_fwd (F over A over B) -> L1 gradient
  -> render_bwd (gradients of the active parameters).
Workload: the 1M-Gaussian active partition (SH degree 3, log-scales
N(log 0.25, 0.5), means uniform in one 5-unit cell of a 5x5x4 grid) seen by
camera 0 of a 200-camera elliptical orbit at 1297x840; F and B from the 99
frozen cells, ordered front to back for that camera; seeded synthetic data.

The metric is Gaussian-pixel blends per second: blended (pixel, Gaussian)
pairs of the step divided by the step time (all inputs resident in HBM).
Prints one JSON line.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Gaussian-pixel blends/sec (fwd+bwd) and ms per active-block step, 1 GPU"
HBM_PEAK_GBS = 8000.0
# MI355X vector issue: 256 CUs x 2.4 GHz x one wave64 VALU instruction per CU and clock (four
# 16-lane SIMDs, four clocks per wave64 instruction) = 39.3 T lane-operations/s; fp32 without
# packed instructions (which this build switches off) is 78.6 TFLOP/s counting an FMA as two
VALU_LANE_PEAK_T = 256 * 64 * 2.4e9 / 1e12
FP32_TFLOPS = 78.6
# algorithmic flops per evaluated (pixel, Gaussian) pair, an estimate kept as a cross-check:
# alpha of the pair (offset, quadratic form, exp, opacity, tests ~16) and, in the backward, its
# derivative terms and the sums over the tile's pixels (~45)
FLOPS_PER_PAIR = {"render_fwd": 16, "render_bwd": 45}
PROFILES = os.path.join(ROOT, "profiles")
HBM_PROFILE = "step_1m_1297x840_hbm_bytes.md"
SQ_PROFILE = "step_1m_1297x840_sq_counters.md"

KERNELS = ["composite", "project", "bin_zero", "depth_keys", "radix_pass", "l1_place", "l2_count",
           "l2_scatter", "bin_small_sort", "bin_small_collect", "render_fwd", "loss_l1",
           "zero_fill", "bwd_order", "render_bwd", "project_bwd", "adam"]
# the launches of abcd_bin_sort (general path, then the small-block path)
BIN_KERNELS = ["bin_zero", "depth_keys", "radix_pass", "l1_place", "l2_count", "l2_scatter",
               "bin_small_sort", "bin_small_collect"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--n", type=int, default=1_000_000)
    ap.add_argument("--width", type=int, default=1297)
    ap.add_argument("--height", type=int, default=840)
    ap.add_argument("--cpu-baseline", type=int, default=1, help="time the CPU oracle on a sample")
    ap.add_argument("--profile-kernels", type=int, default=1)
    ap.add_argument("--extras", type=int, default=1,
                    help="also time the graph replay, the 128x128 workload, Adam and the cache "
                         "refresh (0: only the step, e.g. under a profiler)")
    ap.add_argument("--configs", type=int, default=1,
                    help="also time the other workload configurations (ring scene, mid-scale "
                         "block over 100 sampled cameras, 1M block at 1920x1080, stress sweep "
                         "at 2560x1440); 0: skip them")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the steps, copy this many MiB device to device (a plain copy of "
                         "known size that scales the HBM byte counters)")
    return ap.parse_args()


def algorithmic_bytes(name, n, n_vis, m, npix, k, sh_coeffs, covered_px=None):
    """Bytes a kernel must move at minimum (inputs read once, outputs written once).
    covered_px: layer-pixels inside the cached images' coverage boxes (the
    collapse reads nothing outside them); None means every layer-pixel."""
    param = 4 * (3 + 3 + 4 + 1 + 3 * sh_coeffs)       # means, log-scales, quats, logit, SH
    proj = 4 * (2 + 4 + 1 + 2 + 1 + 3)                 # means2d, conic_opacity, depth, extent, tiles, rgb
    if name == "composite":
        return 8 * (npix * k if covered_px is None else covered_px) + 32 * npix
    if name == "project":
        return n * (param + proj)
    if name == "project_bwd":
        return n * (2 * param + 9 * 4 + 4)             # params in, grads out, g2d and extent.x in
    if name == "l2_scatter":
        return m * 4                                   # the sorted Gaussian indices
    return None


def library_digest():
    """Digest of the library's sources (kernels, shared headers, C ABI header):
    a counter summary taken on other sources no longer describes the kernels."""
    import glob
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2608_27735_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(ROOT, "paper_2608_27735_amd", "csrc", "*.h")) +
                   [os.path.join(ROOT, "include", "abcd.h")])
    for n in files:
        h.update(os.path.basename(n).encode())
        with open(n, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def profile_values(name):
    """The `- key = value` lines of a committed counter summary, if it was taken
    on the library sources built now; else {}."""
    path = os.path.join(PROFILES, name)
    if not os.path.exists(path):
        return {}
    vals = {}
    for line in open(path):
        if line.startswith("- ") and " = " in line:
            k, v = line[2:].strip().split(" = ", 1)
            vals[k.strip()] = v.strip().strip("`")
    return vals if vals.get("library_digest") == library_digest() else {}


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE runs, scaled by the plain-copy calibration), or
    None when it is missing or stale."""
    v = profile_values(HBM_PROFILE)
    try:
        return (float(v[f"{kernel}.fetch_kib"]) * float(v["fetch_factor"]) +
                float(v[f"{kernel}.write_kib"]) * float(v["write_factor"])) * 1024.0
    except (KeyError, ValueError):
        return None


def counted_valu(kernel):
    """Wave-level VALU instructions per launch of `kernel` (SQ_INSTS_VALU) from
    the committed counter summary, or None when it is missing or stale."""
    try:
        return float(profile_values(SQ_PROFILE)[f"{kernel}.sq_insts_valu"])
    except (KeyError, ValueError):
        return None


def roofline_of(name, d, pairs, bytes_):
    """Roofline of one kernel from its live-measured launch duration. HBM-bound
    kernels: algorithmic bytes per launch / duration against 8 TB/s. Blend
    kernels (bound by vector issue): counted VALU lane-operations per launch
    (SQ_INSTS_VALU x 64 lanes) / duration against the 39.3 T lane-op/s issue
    peak, with the HBM rate beside it; only without a current counter summary
    a flop estimate per list position walked (which counts entries the tile
    test drops before any arithmetic, so it is a rough upper figure)."""
    dur = d["ms_per_launch"] / 1e3
    traffic = measured_traffic(name)
    hbm = None if traffic is None else dict(achieved=traffic / dur / 1e9, peak=HBM_PEAK_GBS,
                                            unit="GB/s", frac=traffic / dur / 1e9 / HBM_PEAK_GBS)
    if bytes_ is not None:
        launch_bytes = bytes_ / d["launches_per_step"]
        achieved = launch_bytes / dur / 1e9
        return dict(bound="hbm", kernel=name, achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=achieved / HBM_PEAK_GBS, traffic=traffic,
                    algorithmic_bytes_per_launch=launch_bytes, basis="algorithmic bytes")
    if name not in FLOPS_PER_PAIR:
        return None
    est = pairs * FLOPS_PER_PAIR[name] / dur / 1e12
    insts = counted_valu(name)
    if insts is not None:
        achieved = insts * 64 / dur / 1e12
        return dict(bound="alu", kernel=name, achieved=achieved, peak=VALU_LANE_PEAK_T,
                    unit="Tlane-op/s", frac=achieved / VALU_LANE_PEAK_T, traffic=traffic,
                    basis="counted SQ_INSTS_VALU per launch x 64 lanes / live launch time",
                    valu_insts_per_launch=insts, hbm=hbm)
    return dict(bound="alu", kernel=name, achieved=est, peak=FP32_TFLOPS, unit="TFLOP/s",
                frac=est / FP32_TFLOPS, traffic=traffic,
                basis="estimated flops per evaluated pair (no current counter summary)",
                evaluated_pairs=pairs, flops_per_pair=FLOPS_PER_PAIR[name], hbm=hbm)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the path runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2608_27735_amd import api, synthetic as S
    from paper_2608_27735_amd.step import ActiveBlockStep

    dev = torch.device("cuda:0")
    t0 = time.time()
    w = S.active_block_1m(n=args.n, width=args.width, height=args.height)
    cam, prm = w.cam, w.params
    params = {k: torch.from_numpy(v).to(dev) for k, v in w.scene.items()}
    order = [c for c in w.order if c != w.active]          # 99 frozen cells, front to back
    n_front = w.order.index(w.active)
    k = len(order)
    images, rects = S.cached_images_device(k, cam.height, cam.width, seed=4101, device=dev,
                                           with_rects=True)
    order_idx = list(range(k))                              # images are stored in front-to-back order
    target = torch.from_numpy(S.rng(4102).uniform(0, 1, (cam.height, cam.width, 3))
                              .astype(np.float32)).to(dev)
    F = torch.empty((cam.height, cam.width, 4), dtype=torch.float32, device=dev)
    B = torch.empty_like(F)
    r4 = rects.cpu().to(torch.int64)
    covered = int(((r4[:, 2] - r4[:, 0]).clamp(min=0) * (r4[:, 3] - r4[:, 1]).clamp(min=0)).sum())
    st = ActiveBlockStep(cam, prm, params)
    m = st.project_and_bin(sync=True)
    n_vis = int((st.proj["tiles_touched"] > 0).sum().item())
    setup_s = time.time() - t0

    def one_step():
        # the collapse writes F and B on a second stream, beside projection
        # and binning (which do not read them); the forward waits for it
        st.step(target, F=F, B=B,
                collapse=lambda: api.composite_cache(images, order_idx, n_front, F=F, B=B,
                                                     rects=rects, beside=True))

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    st.n_blends.zero_()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        one_step()
    stop.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    blends_step = st.n_blends.item() / args.steps
    value = blends_step / (ms_step / 1e3)

    graph = small = optimizer = cache_refresh = visibility = hierarchy = comparison = None
    if args.extras:
        # the same step replayed as one HIP graph (collapse + step captured once)
        st.capture(target, F=F, B=B,
                   before=lambda: api.composite_cache(images, order_idx, n_front, F=F, B=B,
                                                      rects=rects, beside=True))
        for _ in range(args.warmup):
            st.replay()
        torch.cuda.synchronize()
        st.n_blends.zero_()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(args.steps):
            st.replay()
        g1.record()
        torch.cuda.synchronize()
        ms_graph = g0.elapsed_time(g1) / args.steps
        blends_graph = st.n_blends.item() / args.steps
        graph = dict(ms_per_step=ms_graph, value=blends_graph / (ms_graph / 1e3),
                     blends_per_step=blends_graph)

        # visibility-aware variant (reported beside the metric, not in it): the
        # collapse drops layers hidden below t_min and the forward stops a pixel
        # once (1 - F_alpha) T < t_min; the image differs from the exact step's
        # by at most t_min / (1 - alpha_max) (colour + 1) per channel
        import dataclasses
        prm_v = dataclasses.replace(prm, fb_stop=True)
        st_v = ActiveBlockStep(cam, prm_v, params, capacity=st.capacity)
        Fv, Bv = torch.empty_like(F), torch.empty_like(B)

        def vis_step():
            api.composite_cache(images, order_idx, n_front, F=Fv, B=Bv, rects=rects,
                                stop_t=prm.t_min)
            st_v.step(target, F=Fv, B=Bv)

        for _ in range(args.warmup):
            vis_step()
        torch.cuda.synchronize()
        st_v.n_blends.zero_()
        v0, v1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        v0.record()
        for _ in range(args.steps):
            vis_step()
        v1.record()
        torch.cuda.synchronize()
        ms_v = v0.elapsed_time(v1) / args.steps
        blends_v = st_v.n_blends.item() / args.steps
        hidden = float(((1.0 - Fv[..., 3]) < prm.t_min).float().mean().item())
        diff = float((st_v.fwd["out"] - st.fwd["out"]).abs().max().item())
        visibility = dict(ms_per_step=ms_v, blends_per_step=blends_v,
                          value=blends_v / (ms_v / 1e3), stop_t=prm.t_min,
                          hidden_pixel_fraction=hidden, max_abs_diff_vs_exact=diff,
                          note="compositing-aware stop (fb_stop) and thresholded collapse; "
                               "not the metric")
        del st_v, Fv, Bv

        # memory hierarchy (reported beside the metric): the cached renders held
        # in pinned host memory and streamed to the GPU by coverage box, 16 per
        # chunk, double-buffered against the collapse; device memory stays the
        # two chunks whatever the number of layers
        from paper_2608_27735_amd.hierarchy import FBStreamer, HostCache
        hcache = HostCache(cam.width, cam.height, k)
        hcache.images.copy_(images.cpu())
        hcache.rects[:] = rects.cpu().numpy()
        streamer = FBStreamer(hcache, chunk=16)
        Fh, Bh = torch.empty_like(F), torch.empty_like(B)
        hier = []
        for K in (25, 50, k):
            nf = min(n_front, K)
            slots = list(range(K))
            streamer.build(slots, nf, Fh, Bh)
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            reps = 5
            h0, h1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            h0.record()
            for _ in range(reps):
                streamer.build(slots, nf, Fh, Bh)
            h1.record()
            torch.cuda.synchronize()
            ms_h = h0.elapsed_time(h1) / reps
            rk = r4[:K]
            moved = int(8 * ((rk[:, 2] - rk[:, 0]).clamp(min=0) *
                             (rk[:, 3] - rk[:, 1]).clamp(min=0)).sum())
            hier.append(dict(layers=K, build_ms=ms_h, h2d_bytes=moved,
                             h2d_GBs=moved / (ms_h / 1e3) / 1e9,
                             resident_layers_bytes=K * cam.width * cam.height * 8,
                             device_peak_growth_bytes=torch.cuda.max_memory_allocated() - base))
        hierarchy = dict(per_layers=hier, chunk=16,
                         staging_bytes=2 * 16 * cam.width * cam.height * 8,
                         note="F/B built from pinned host memory; coverage boxes only cross "
                              "PCIe; device memory = two staging chunks + F/B")
        del hcache, streamer, Fh, Bh

        # the paper's three training setups on the 64K-Gaussian ring scene (4x4x4
        # grid, 8 cameras at 512x512) with a known ground truth: targets are
        # joint renders of the scene, training starts from a perturbed copy;
        # every setup gives each Gaussian the same number of Adam steps
        from paper_2608_27735_amd import train as TR
        rw = S.ring()
        comparison = TR.compare(rw.scene, S.perturbed(S.rng(5), rw.scene), rw.grid, rw.cell_of,
                                rw.cams, rw.params, epochs=2, T=20)
        comparison = dict(workload="64K Gaussians (SH 3), 4x4x4 grid, 8 cameras at 512x512; "
                                   "targets = joint renders of the ground truth; init = means "
                                   "jittered, opacity lowered, colours grey",
                          epochs=2, steps_per_gaussian=40, **comparison)

        # launch-bound regime (Results section: small active partitions leave the
        # rasterizer underused and launch costs dominate): the 512-Gaussian active
        # cell of the 4,096-Gaussian 128x128 workload, eager launches vs one graph
        # replay
        small = small_config(api, S, ActiveBlockStep, dev, args.steps, args.warmup)

    # per-kernel durations: HIP events around every launch, on the launch
    # stream, in steps that run the collapse first (not beside the binning),
    # so that each kernel's time is its own
    def one_step_alone():
        api.composite_cache(images, order_idx, n_front, F=F, B=B, rects=rects)
        st.step(target, F=F, B=B)

    kern = {}
    if args.profile_kernels:
        api.timing_reset()
        api.timing_enable(True)
        for _ in range(args.steps):
            one_step_alone()
        torch.cuda.synchronize()
        api.timing_enable(False)
        for name in KERNELS:
            ms, cnt = api.timing_read(name)
            if cnt:
                kern[name] = dict(ms_per_step=ms / args.steps, launches_per_step=cnt / args.steps,
                                  ms_per_launch=ms / cnt)
        api.timing_reset()
    sh_coeffs = (prm.sh_degree + 1) ** 2
    npix = cam.width * cam.height
    # evaluated pairs: every pixel walks its tile list up to its last blended entry
    pairs = int(st.fwd["last"].to(torch.int64).sum().item())
    dominant = max(kern, key=lambda x: kern[x]["ms_per_step"]) if kern else None
    roofline = None
    if dominant:
        roofline = roofline_of(dominant, kern[dominant], pairs,
                               algorithmic_bytes(dominant, args.n, n_vis, m, npix, k, sh_coeffs,
                                                 covered))
    for name in FLOPS_PER_PAIR:
        if name in kern:
            r = roofline_of(name, kern[name], pairs, None)
            kern[name]["roofline"] = {kk: r[kk] for kk in ("achieved", "peak", "unit", "frac",
                                                            "basis")}
    for name, d in kern.items():
        b = algorithmic_bytes(name, args.n, n_vis, m, npix, k, sh_coeffs, covered)
        if b is not None:
            d["algorithmic_GBs"] = b / d["launches_per_step"] / (d["ms_per_launch"] / 1e3) / 1e9
        t = measured_traffic(name)
        if t is not None:
            d["measured_GBs"] = t / (d["ms_per_launch"] / 1e3) / 1e9
            d["hbm_frac"] = d["measured_GBs"] / HBM_PEAK_GBS
        v = counted_valu(name)
        if v is not None:  # counted VALU lane-operations against the issue peak
            d["valu_issue_frac"] = v * 64 / (d["ms_per_launch"] / 1e3) / 1e12 / VALU_LANE_PEAK_T

    if args.extras:
        # the optimizer side of the step (reported beside the metric, not in it):
        # one Adam update of the five parameter groups
        exp_avg = {kk: torch.zeros_like(v) for kk, v in params.items()}
        exp_avg_sq = {kk: torch.zeros_like(v) for kk, v in params.items()}
        lrs = dict(means=1.6e-4, log_scales=5e-3, quats=1e-3, opacity_logits=5e-2, sh=2.5e-3)
        for t in range(1, 4):
            api.adam_step(params, st.grads, exp_avg, exp_avg_sq, lrs, t)
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record()
        for t in range(4, 4 + args.steps):
            api.adam_step(params, st.grads, exp_avg, exp_avg_sq, lrs, t)
        a1.record()
        torch.cuda.synchronize()
        adam_ms = a0.elapsed_time(a1) / args.steps
        n_el = sum(v.numel() for v in params.values())
        optimizer = dict(kernel="adam", ms_per_step=adam_ms, elements=n_el,
                         algorithmic_GBs=28.0 * n_el / (adam_ms / 1e3) / 1e9,
                         note="28 B per element (parameter, gradient, two moments read; "
                              "parameter and moments written); not part of ms_per_step")

        # the cache refresh after a block's T updates (reported beside the metric):
        # the block re-rendered for 8 cameras spread around the scene, fp16 images
        # copied into pinned host memory, copies overlapped with the next render
        from paper_2608_27735_amd.cache import CacheRefresher
        rcams = w.cams[::len(w.cams) // 8][:8]
        refresher = CacheRefresher(prm, params, cam.width, cam.height)
        hosts = [torch.empty((cam.height, cam.width, 4), dtype=torch.float16).pin_memory()
                 for _ in rcams]
        refresher.refresh(rcams, hosts)  # sizes the binning buffers
        torch.cuda.synchronize()
        r0 = time.perf_counter()
        refresher.refresh(rcams, hosts)
        refresh_ms = (time.perf_counter() - r0) * 1e3 / len(rcams)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for c in rcams:
            refresher.render(c, refresher.staging[0])
        c1.record()
        torch.cuda.synchronize()
        cache_refresh = dict(cameras=len(rcams), ms_per_camera=refresh_ms,
                             render_ms_per_camera=c0.elapsed_time(c1) / len(rcams),
                             image_bytes=cam.width * cam.height * 8,
                             note="project, bin (intersection count read back), fp16 cached "
                                  "render, async D2H into pinned memory; wall clock per camera")
        del hosts

    if args.copy_calibration_mb:
        nbytes = args.copy_calibration_mb << 20
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    configs = None
    if args.configs:
        del st, images, rects, F, B
        torch.cuda.empty_cache()
        configs = dict(
            tiny_512_128x128=small,
            ring_64k_8cams_512x512=config_ring(api, S, ActiveBlockStep, dev, args.steps,
                                               args.warmup),
            midscale_300k_100steps_1297x840=config_midscale(api, S, ActiveBlockStep, dev),
            block_1m_uniform_1920x1080=config_large(api, S, ActiveBlockStep, dev, False,
                                                    args.steps, args.warmup),
            block_1m_heavy_tail_1920x1080=config_large(api, S, ActiveBlockStep, dev, True,
                                                       args.steps, args.warmup),
            stress_2560x1440=config_stress(api, S, ActiveBlockStep, dev),
            comparison_midscale_5m_1297x840=comparison_midscale(S))

    cpu = None
    if args.cpu_baseline:
        cpu = cpu_baseline(w, cam, prm, k)

    out = {
        "metric": METRIC, "value": value, "unit": "blends/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"ABCD active-block step: {args.n} Gaussians (SH 3) at "
                               f"{cam.width}x{cam.height}, F/B collapsed from {k} cached fp16 "
                               "partition renders (with their coverage boxes)",
                   "n_gaussians": args.n, "width": cam.width, "height": cam.height,
                   "sh_degree": prm.sh_degree, "k_cached": k, "n_front": n_front,
                   "n_isect": m, "n_visible": n_vis, "blends_per_step": blends_step,
                   "cached_layer_pixels_covered": covered,
                   "evaluated_pairs_per_pass": pairs,
                   "sync_in_step": False},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "optimizer": optimizer,
        "graph": graph,
        "cache_refresh": cache_refresh,
        "visibility": visibility,
        "hierarchy": hierarchy,
        "comparison": comparison,
        "small_config": small,
        "configs": configs,
        "kernels": kern,
        "binning": ({"ms_per_step": sum(kern[x]["ms_per_step"] for x in BIN_KERNELS if x in kern),
                     "launches_per_step": sum(kern[x]["launches_per_step"] for x in BIN_KERNELS
                                              if x in kern)} if kern else None),
        "setup_s": setup_s,
    }
    print(json.dumps(out))


def small_config(api, S, ActiveBlockStep, dev, steps, warmup):
    import numpy as np
    import torch
    w = S.tiny()
    cam, prm = w.cams[0], w.params
    sub = S.subset(w.scene, w.cell_of == w.active)
    params = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in sub.items()}
    F0, B0 = S.background_pair(S.rng(4103), cam.height, cam.width)
    F, B = torch.from_numpy(F0).to(dev), torch.from_numpy(B0).to(dev)
    target = torch.from_numpy(w.target).to(dev)
    st = ActiveBlockStep(cam, prm, params)
    reps = max(steps, 50)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    eager = timed(lambda: st.step(target, F=F, B=B))
    st.capture(target, F=F, B=B)
    graph = timed(st.replay)
    return dict(workload=f"{len(sub['means'])} active Gaussians (SH 0) at {cam.width}x{cam.height}",
                eager_ms_per_step=eager, graph_ms_per_step=graph, steps=reps)


def _timed(fn, reps, warmup):
    """Mean milliseconds of fn() over reps calls after warm-up (HIP events on the
    current stream, synchronised on both sides)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def _blend_kernels(api, fn, reps, st):
    """Per-launch milliseconds of the two blend kernels (and the collapse) over
    reps calls of fn(), and the pairs blended per forward launch (st: the
    ActiveBlockStep fn runs)."""
    import torch
    st.n_blends.zero_()
    api.timing_reset()
    api.timing_enable(True)
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    api.timing_enable(False)
    out = {}
    fwd_calls = 0
    for name in ("render_fwd", "render_bwd", "composite"):
        ms, cnt = api.timing_read(name)
        if cnt:
            out[name] = ms / cnt
            if name == "render_fwd":
                fwd_calls = cnt
    api.timing_reset()
    return out, st.n_blends.item() / max(fwd_calls, 1)


def _blend_roofline(kern, blends_per_call):
    """Launch times of the blend kernels and their rate in blended pairs. Their
    VALU-issue roofline needs the counted instructions of the launch, which are
    taken on the headline workload only: a flop count per list position or per
    blend depends on the workload (how many list entries the tile test drops,
    how many lanes of a wave blend an entry) and does not transfer."""
    out = {}
    for name, ms in kern.items():
        row = dict(ms_per_launch=ms)
        if name in FLOPS_PER_PAIR:
            row.update(blends_per_launch=blends_per_call,
                       blends_per_s=blends_per_call / (ms / 1e3))
        out[name] = row
    return out


def _step_fields(st, ms, calls):
    import torch
    blends = st.n_blends.item() / calls
    pairs = int(st.fwd["last"].to(torch.int64).sum().item())
    return dict(ms_per_step=ms, value=blends / (ms / 1e3), unit="blends/s",
                blends_per_step=blends, evaluated_pairs_last_step=pairs,
                capacity=int(st.capacity))


def config_ring(api, S, ActiveBlockStep, dev, steps, warmup):
    """The 64K-Gaussian ring scene (SH 3, 4x4x4 grid over the unit cube's
    [-1, 1]^3, 32 blobs): its ~1K-Gaussian active cell, 8 cameras at 512x512.
    Every camera's F and B are collapsed from the 63 other cells' cached fp16
    renders (drawn by the cache-refresh path, with their coverage boxes), in
    the camera's front-to-back cell order; a step per camera."""
    import numpy as np
    import torch
    from paper_2608_27735_amd.cache import CacheRefresher
    w = S.ring()
    prm, cams = w.params, w.cams
    H, W = cams[0].height, cams[0].width
    cells = [c for c in range(w.grid.n_cells) if c != w.active]
    imgs = torch.zeros((len(cams), len(cells), H, W, 4), dtype=torch.float16, device=dev)
    rects = torch.zeros((len(cams), len(cells), 4), dtype=torch.int32, device=dev)
    for j, c in enumerate(cells):
        sub = S.subset(w.scene, w.cell_of == c)
        if len(sub["means"]) == 0:
            continue
        pc = {kk: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for kk, v in sub.items()}
        ref = CacheRefresher(prm, pc, W, H)
        for i, cam in enumerate(cams):
            ref.render(cam, imgs[i, j], rects[i, j])
    act = S.subset(w.scene, w.cell_of == w.active)
    params = {kk: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for kk, v in act.items()}
    st = ActiveBlockStep(cams[0], prm, params)
    for cam in cams[1:]:  # capacity for every camera
        st.cam = cam
        st.project_and_bin(sync=True)
    plan = []
    for cam in cams:
        order = [int(c) for c in w.grid.order_from(cam.campos)]
        nf = order.index(w.active)
        plan.append(([cells.index(c) for c in order if c != w.active], nf))
    targets = torch.from_numpy(w.target).to(dev)
    F = torch.empty((H, W, 4), dtype=torch.float32, device=dev)
    B = torch.empty_like(F)

    def cams_pass():
        for i, cam in enumerate(cams):
            st.cam = cam
            api.composite_cache(imgs[i], plan[i][0], plan[i][1], F=F, B=B, rects=rects[i])
            st.step(targets[i], F=F, B=B)

    reps = max(2, steps // 4)
    cams_pass()
    torch.cuda.synchronize()
    st.n_blends.zero_()
    ms = _timed(cams_pass, reps, 0) / len(cams)
    out = _step_fields(st, ms, reps * len(cams))
    kern, kb = _blend_kernels(api, cams_pass, 1, st)
    out.update(workload=f"{len(act['means'])} active Gaussians (SH 3) of the 64K ring scene, "
                        f"{len(cams)} cameras at {W}x{H}, F/B per camera from {len(cells)} "
                        "cached fp16 cell renders", cameras=len(cams), k_cached=len(cells),
               kernels_per_camera=_blend_roofline(kern, kb),
               note="ms_per_step = per camera: collapse of 63 layers + project, bin, forward, "
                    "L1 gradient, backward")
    return out


def config_midscale(api, S, ActiveBlockStep, dev, T=100):
    """The mid-scale scene's 300K-Gaussian active block (ground plane and
    blobs, SH 3) on 200 cameras at 1297x840: T = 100 steps, each on a camera
    drawn uniformly (seeded), with that camera's F and B collapsed from the 31
    other cells' cached renders (synthetic fp16 layers with coverage boxes,
    ordered by the camera's cell order)."""
    import numpy as np
    import torch
    w = S.midscale_block()
    prm, cams = w.params, w.cams
    H, W = cams[0].height, cams[0].width
    params = {kk: torch.from_numpy(v).to(dev) for kk, v in w.scene.items()}
    cells = [c for c in range(w.grid.n_cells) if c != w.active]
    images, rects = S.cached_images_device(len(cells), H, W, seed=3101, device=dev,
                                           with_rects=True)
    st = ActiveBlockStep(cams[0], prm, params)
    for cam in cams[1:]:
        st.cam = cam
        st.project_and_bin(sync=True)
    seq = S.rng(3102).integers(0, len(cams), T)
    plan = {}
    for i in set(int(x) for x in seq):
        order = [int(c) for c in w.grid.order_from(cams[i].campos)]
        plan[i] = ([cells.index(c) for c in order if c != w.active], order.index(w.active))
    target = torch.from_numpy(S.rng(3103).uniform(0, 1, (H, W, 3)).astype(np.float32)).to(dev)
    F = torch.empty((H, W, 4), dtype=torch.float32, device=dev)
    B = torch.empty_like(F)

    def run():
        for i in seq:
            i = int(i)
            st.cam = cams[i]
            api.composite_cache(images, plan[i][0], plan[i][1], F=F, B=B, rects=rects)
            st.step(target, F=F, B=B)

    run()
    torch.cuda.synchronize()
    st.n_blends.zero_()
    ms = _timed(run, 1, 0) / T
    out = _step_fields(st, ms, T)

    def last_cam():
        api.composite_cache(images, plan[int(seq[-1])][0], plan[int(seq[-1])][1], F=F, B=B,
                            rects=rects)
        st.step(target, F=F, B=B)

    kern, kb = _blend_kernels(api, last_cam, 3, st)
    out.update(kernels_last_camera=_blend_roofline(kern, kb))
    out.update(workload=f"{len(w.scene['means'])} active Gaussians (SH 3), mid-scale scene "
                        f"(4x4x2 grid), {T} steps over cameras drawn from {len(cams)} at {W}x{H}",
               steps=T, distinct_cameras=len(plan), k_cached=len(cells),
               note="ms_per_step = mean over the T steps, each: collapse of 31 layers + step")
    return out


def config_large(api, S, ActiveBlockStep, dev, heavy, steps, warmup):
    """The 1M-Gaussian active block (SH 3) at 1920x1080, uniform or heavy-tailed
    scales (log-normal sd 1.0), F and B from 99 cached layers."""
    import numpy as np
    import torch
    w = S.active_block_1m(width=1920, height=1080, heavy_tail=heavy)
    cam, prm = w.cam, w.params
    params = {kk: torch.from_numpy(v).to(dev) for kk, v in w.scene.items()}
    order = [c for c in w.order if c != w.active]
    n_front = w.order.index(w.active)
    k = len(order)
    images, rects = S.cached_images_device(k, cam.height, cam.width, seed=4101, device=dev,
                                           with_rects=True)
    target = torch.from_numpy(S.rng(4102).uniform(0, 1, (cam.height, cam.width, 3))
                              .astype(np.float32)).to(dev)
    F = torch.empty((cam.height, cam.width, 4), dtype=torch.float32, device=dev)
    B = torch.empty_like(F)
    st = ActiveBlockStep(cam, prm, params)
    m = st.project_and_bin(sync=True)

    def one():
        api.composite_cache(images, list(range(k)), n_front, F=F, B=B, rects=rects)
        st.step(target, F=F, B=B)

    one()
    torch.cuda.synchronize()
    st.n_blends.zero_()
    reps = max(5, steps // 2)
    ms = _timed(one, reps, warmup)
    out = _step_fields(st, ms, reps + warmup)
    kern, kb = _blend_kernels(api, one, 3, st)
    out.update(workload=f"1M active Gaussians (SH 3, {'heavy-tailed' if heavy else 'uniform'} "
                        f"scales) at {cam.width}x{cam.height}, F/B from {k} cached layers",
               n_isect=m, kernels=_blend_roofline(kern, kb))
    del st, images, rects
    torch.cuda.empty_cache()
    return out


def config_stress(api, S, ActiveBlockStep, dev, sizes=(262_144, 1_000_000, 4_000_000)):
    """The stress configuration at 2560x1440 (8x8x2 grid, tiny scales): steps of
    active blocks of 256K, 1M and 4M Gaussians, each with F and B collapsed
    from 127 cached layers (synthetic fp16 with coverage boxes), and the peak
    device memory of each point. Then, for the 1M block, F and B built from
    pinned host memory (coverage boxes streamed 16 layers at a time) for
    scenes of 10x, 50x, 100x and 128x the active block (9, 49, 99 and 127
    frozen cells of its size): the device peak should not grow with the scene."""
    import numpy as np
    import torch
    from paper_2608_27735_amd.hierarchy import FBStreamer, HostCache
    sweep = []
    k = 127
    for n in sizes:
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        w = S.stress_block(n=n)
        cam, prm = w.cam, w.params
        params = {kk: torch.from_numpy(v).to(dev) for kk, v in w.scene.items()}
        images, rects = S.cached_images_device(k, cam.height, cam.width, seed=5101, device=dev,
                                               with_rects=True)
        order = [c for c in w.order if c != w.active]
        n_front = w.order.index(w.active)
        target = torch.from_numpy(S.rng(5102).uniform(0, 1, (cam.height, cam.width, 3))
                                  .astype(np.float32)).to(dev)
        F = torch.empty((cam.height, cam.width, 4), dtype=torch.float32, device=dev)
        B = torch.empty_like(F)
        st = ActiveBlockStep(cam, prm, params)
        m = st.project_and_bin(sync=True)

        def one():
            api.composite_cache(images, list(range(len(order))), n_front, F=F, B=B, rects=rects)
            st.step(target, F=F, B=B)

        one()
        torch.cuda.synchronize()
        st.n_blends.zero_()
        reps = 5
        ms = _timed(one, reps, 1)
        row = _step_fields(st, ms, reps + 1)
        row["kernels"] = _blend_roofline(*_blend_kernels(api, one, 2, st))
        cm = _timed(lambda: api.composite_cache(images, list(range(len(order))), n_front, F=F,
                                                B=B, rects=rects), 5, 1)
        row.update(n_gaussians=n, n_isect=m, collapse_ms=cm,
                   device_peak_bytes=int(torch.cuda.max_memory_allocated() - base),
                   resident_layers_bytes=int(images.numel() * 2))
        sweep.append(row)
        del st, images, rects, params, F, B
    # device memory flat in the scene size: the cached layers live in pinned host memory
    w = S.stress_block(n=sizes[1])
    cam, prm = w.cam, w.params
    torch.cuda.empty_cache()
    hc = HostCache(cam.width, cam.height, k)
    dimgs, drects = S.cached_images_device(k, cam.height, cam.width, seed=5101, device=dev,
                                           with_rects=True)
    hc.images.copy_(dimgs.cpu())
    hc.rects[:] = drects.cpu().numpy()
    del dimgs, drects
    params = {kk: torch.from_numpy(v).to(dev) for kk, v in w.scene.items()}
    target = torch.from_numpy(S.rng(5102).uniform(0, 1, (cam.height, cam.width, 3))
                              .astype(np.float32)).to(dev)
    F = torch.empty((cam.height, cam.width, 4), dtype=torch.float32, device=dev)
    B = torch.empty_like(F)
    st = ActiveBlockStep(cam, prm, params)
    streamer = FBStreamer(hc, chunk=16)
    flat = []
    for K in (9, 49, 99, 127):
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        t0 = time.perf_counter()
        streamer.build(list(range(K)), K // 2, F, B)
        st.step(target, F=F, B=B)
        torch.cuda.synchronize()
        flat.append(dict(scene_over_active=K + 1, frozen_cells=K,
                         fb_build_and_step_ms=(time.perf_counter() - t0) * 1e3,
                         device_peak_growth_bytes=int(torch.cuda.max_memory_allocated() - base),
                         host_cache_bytes=int(K * cam.width * cam.height * 8)))
    resident = int(sum(v.numel() * v.element_size() for v in params.values()) +
                   2 * F.numel() * 4 + sum(b.numel() * b.element_size() for b in streamer.bufs))
    del st, streamer, hc, params, F, B
    torch.cuda.empty_cache()
    return dict(workload=f"stress block (tiny scales, SH 3) at {cam.width}x{cam.height}, "
                         f"{k} cached layers per camera", sweep=sweep, scene_growth=flat,
                resident_active_fb_staging_bytes=resident,
                note="scene_growth: the 1M block with F/B streamed from pinned host memory; "
                     "device_peak_growth_bytes is what building F/B and one step add on top of "
                     "the resident active set, F/B and staging chunks")


def comparison_midscale(S, n=5_000_000, n_cams=12, T=4):
    """The paper's three setups (Results section: 3DGS-style joint training,
    ABCD, ABCD without F/B) on the whole 5M-Gaussian mid-scale scene (32
    cells, 12 of its 200 cameras at 1297x840), targets = joint renders of the
    scene, training from a perturbed copy, T Adam steps per Gaussian (one
    epoch): PSNR, wall time and peak device memory of each. The ABCD setup
    keeps every camera's cached cell renders in pinned host memory and streams
    each camera's F/B to the GPU per visit."""
    from paper_2608_27735_amd import train as TR
    w = S.midscale_scene(n=n, n_cams=200)
    cams = w.cams[::200 // n_cams][:n_cams]
    t0 = time.perf_counter()
    res = TR.compare(w.scene, S.perturbed(S.rng(6), w.scene), w.grid, w.cell_of, cams, w.params,
                     epochs=1, T=T)
    return dict(workload=f"{n} Gaussians (SH 3), mid-scale scene (4x4x2 grid), {n_cams} cameras "
                         "at 1297x840; targets = joint renders of the ground truth; init = means "
                         "jittered, opacity lowered, colours grey", steps_per_gaussian=T,
                total_s=time.perf_counter() - t0, **res)


def cpu_baseline(w, cam, prm, k):
    """The oracle, as it stands, on a bounded sample of the same workload: the
    full step (projection of all Gaussians of a 1/4 random subset, binning,
    forward and backward over every pixel, and the F/B collapse of k cached
    renders over a 1/16 band of image rows), on this host's cores."""
    import numpy as np

    from oracle import oracle as O
    from paper_2608_27735_amd import synthetic as S

    cores = len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(cores))
    r = S.rng(4103)
    n = w.scene["means"].shape[0]
    sub = S.subset(w.scene, r.random(n) < 1.0 / 4)
    F, B = S.background_pair(r, cam.height, cam.width)
    G = S.upstream_grad(r, cam.height, cam.width)
    t0 = time.perf_counter()
    res = O.step(cam, prm, sub, F=F, B=B, dL_dout=G.astype(np.float64))
    t_step = time.perf_counter() - t0
    rows = max(1, cam.height // 16)
    imgs = S.half_bits(S.premultiplied_images(r, k, rows, cam.width, coverage=0.35))
    t1 = time.perf_counter()
    O.composite(cam.width, rows, imgs, list(range(k)), k // 2)
    t_comp = (time.perf_counter() - t1) * (cam.height / rows)  # scaled to the full frame
    blends = res["fwd"]["n_blends"]
    secs = t_step + t_comp
    return dict(value=blends / secs, unit="blends/s", cores=cores, kind="oracle",
                sample=f"1/4 random subset of the Gaussians ({len(sub['means'])}), full "
                       f"{cam.width}x{cam.height} frame: project+bin+fwd+bwd; F/B collapse of "
                       f"{k} layers timed on {rows} rows and scaled to the frame",
                step_s=t_step, composite_s_scaled=t_comp, blends=blends)


if __name__ == "__main__":
    main()

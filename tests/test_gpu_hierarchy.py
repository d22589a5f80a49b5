"""GPU tests of the memory hierarchy: cached renders kept in pinned host
memory, uploaded by coverage box (abcd_stage_cached) and collapsed in chunks
while the next chunk uploads. The collapse folds the same layers in the same
order as a one-pass collapse of device-resident images, so F and B must be
bit-identical to it; the one-pass collapse is held to the oracle by the
composite tests. Every case prints its name before touching the GPU."""
import numpy as np
import pytest
import torch

from paper_2608_27735_amd import synthetic as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mods():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_27735_amd import api, hierarchy
    return api, hierarchy


def dev():
    return torch.device("cuda:0")


def say(*a):
    print("[case]", *a, flush=True)


def _boxes(imgs, W, H, tile=16):
    k = imgs.shape[0]
    rects = np.zeros((k, 4), np.int32)
    for j in range(k):
        ys, xs = np.nonzero(np.any(imgs[j] != 0, axis=-1))
        if len(xs):
            rects[j] = (xs.min() // tile * tile, ys.min() // tile * tile,
                        min(W, (xs.max() // tile + 1) * tile), min(H, (ys.max() // tile + 1) * tile))
        else:
            rects[j] = (W, H, 0, 0)
    return rects


def test_host_cache_slots(mods):
    _, Hm = mods
    say("host cache slots")
    c = Hm.HostCache(8, 4, 2)
    assert c.slot(("cam0", 3)) == 0 and c.slot(("cam1", 3)) == 1 and c.slot(("cam0", 3)) == 0
    with pytest.raises(RuntimeError):
        c.slot(("cam2", 0))


def test_stage_cached_copies_only_the_boxes(mods):
    api, Hm = mods
    H, W, k = 37, 53, 5
    say("stage_cached boxes", k, H, W)
    r = S.rng(401)
    imgs = S.half_bits(S.premultiplied_images(r, k, H, W, coverage=0.3))
    rects = _boxes(imgs, W, H)
    rects[3] = (W, H, 0, 0)  # an empty box copies nothing
    host = [torch.from_numpy(imgs[j].view(np.float16)).pin_memory() for j in range(k)]
    dst = torch.full((k + 1, H, W, 4), -3.0, dtype=torch.float16, device=dev())
    api.stage_cached(host, dst, rects=rects)
    torch.cuda.synchronize()
    got = dst.cpu().numpy().view(np.uint16)
    sentinel = np.float16(-3.0).view(np.uint16)
    for j in range(k):
        x0, y0, x1, y1 = rects[j]
        inside = np.zeros((H, W), bool)
        inside[y0:y1, x0:x1] = x1 > x0
        assert np.array_equal(got[j][inside], imgs[j][inside])
        assert np.all(got[j][~inside] == sentinel)
    assert np.all(got[k] == sentinel)
    # whole images without boxes
    api.stage_cached(host, dst, rects=None)
    torch.cuda.synchronize()
    assert np.array_equal(dst[:k].cpu().numpy().view(np.uint16), imgs)


@pytest.mark.parametrize("k,n_front,hw,chunk,st", [(23, 9, (64, 96), 5, 0.0), (23, 9, (64, 96), 5, 0.01),
                                                   (40, 0, (33, 17), 16, 0.0), (7, 7, (128, 128), 3, 0.0),
                                                   (1, 1, (16, 24), 4, 0.0), (0, 0, (16, 24), 4, 0.0)])
def test_streamed_collapse_equals_resident_collapse(mods, k, n_front, hw, chunk, st):
    api, Hm = mods
    H, W = hw
    say("streamed collapse", k, n_front, hw, chunk, st)
    r = S.rng(410 + k)
    imgs = S.half_bits(S.premultiplied_images(r, k, H, W, alpha_max=0.9, coverage=0.4)) if k else \
        np.zeros((0, H, W, 4), np.uint16)
    rects = _boxes(imgs, W, H)
    cache = Hm.HostCache(W, H, max(k, 1) + 3)
    slots = []
    for j in range(k):  # stored out of order on purpose
        s = cache.put(("cam", (j * 7) % max(k, 1), j), torch.from_numpy(imgs[j].view(np.float16)),
                      rects[j])
        slots.append(s)
    order = list(r.permutation(k))
    streamer = Hm.FBStreamer(cache, chunk=chunk)
    F = torch.full((H, W, 4), 5.0, device=dev())
    B = torch.full((H, W, 4), 5.0, device=dev())
    streamer.build([slots[j] for j in order], n_front, F, B, stop_t=st)
    img_d = torch.from_numpy(imgs.view(np.int16)).to(dev())
    Fr, Br = api.composite_cache(img_d, order, n_front,
                                 rects=torch.from_numpy(rects).to(dev()) if k else None, stop_t=st)
    torch.cuda.synchronize()
    assert torch.equal(F, Fr) and torch.equal(B, Br)
    # a second build reuses the staging chunks
    streamer.build([slots[j] for j in order], n_front, F, B, stop_t=st)
    torch.cuda.synchronize()
    assert torch.equal(F, Fr) and torch.equal(B, Br)


def test_refresh_into_host_cache_then_stream(mods):
    """Partitions of the ring scene rendered per camera into the host cache
    (refresh), then F/B for the active cell streamed from it: equal to the
    collapse of the same renders kept on the device."""
    api, Hm = mods
    from paper_2608_27735_amd.cache import CacheRefresher
    w = S.ring()
    cam, prm = w.cams[1], w.params
    cells = [c for c in range(w.grid.n_cells) if (w.cell_of == c).sum() > 0]
    vis = Hm.visible_cells(cam, w.grid, margin=0.3)
    cells = [c for c in cells if vis[c] and c != w.active]
    order_all = [c for c in w.grid.order_from(cam.campos) if c in cells or c == w.active]
    front = [c for c in order_all[:order_all.index(w.active)] if c != w.active]
    back = [c for c in order_all[order_all.index(w.active) + 1:]]
    say("refresh -> host cache -> stream", len(front), len(back))
    H, W = cam.height, cam.width
    cache = Hm.HostCache(W, H, len(cells))
    dev_imgs, dev_rects = [], []
    for c in front + back:
        sc = {k: torch.from_numpy(np.ascontiguousarray(v[w.cell_of == c])).to(dev())
              for k, v in w.scene.items()}
        ref = CacheRefresher(prm, sc, W, H)
        host = [cache.images[cache.slot((1, c))]]
        rect = torch.zeros((1, 4), dtype=torch.int32, device=dev())
        ref.refresh([cam], host, rect)
        cache.rects[cache.slot((1, c))] = rect[0].cpu().numpy()
        img = torch.empty((H, W, 4), dtype=torch.float16, device=dev())
        ref.render(cam, img)
        dev_imgs.append(img)
        dev_rects.append(rect[0])
    torch.cuda.synchronize()
    streamer = Hm.FBStreamer(cache, chunk=4)
    F = torch.empty((H, W, 4), device=dev())
    B = torch.empty((H, W, 4), device=dev())
    streamer.build([cache.slot((1, c)) for c in front + back], len(front), F, B)
    Fr, Br = api.composite_cache(torch.stack(dev_imgs), list(range(len(dev_imgs))), len(front),
                                 rects=torch.stack(dev_rects).contiguous())
    torch.cuda.synchronize()
    assert torch.equal(F, Fr) and torch.equal(B, Br)
    assert F[..., 3].max().item() > 0 and B[..., 3].max().item() > 0

// abi.hip -- the extern "C" entry points declared in include/abcd.h: argument
// validation on the host (before any HIP call), dispatch to the kernels,
// error reporting and optional per-kernel event timing.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "abcd_internal.h"

#define ABCD_VERSION_STRING "abcd-gfx950 0.1.0"

namespace abcd {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

int32_t hip_fail(hipError_t e, const char* what) {
  set_error("%s failed: %s", what, hipGetErrorString(e));
  return ABCD_E_HIP;
}

// ------------------------------------------------------------ timing

namespace {
struct TimingRec {
  std::string name;
  hipEvent_t a, b;
};
thread_local bool g_timing = false;
thread_local std::vector<TimingRec> g_recs;
}  // namespace

TimedLaunch::TimedLaunch(const char* n, hipStream_t s) : name(n), stream(s), rec(nullptr) {
  if (!g_timing) return;
  TimingRec r{n, nullptr, nullptr};
  if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return;
  (void)hipEventRecord(r.a, s);
  g_recs.push_back(r);
  rec = &g_recs.back();
}

TimedLaunch::~TimedLaunch() {
  if (!rec) return;
  (void)hipEventRecord(g_recs.back().b, stream);
}

}  // namespace abcd

using namespace abcd;

namespace {

#define REQUIRE(cond, ...)            \
  do {                                \
    if (!(cond)) {                    \
      abcd::set_error(__VA_ARGS__);   \
      return ABCD_E_INVALID;          \
    }                                 \
  } while (0)

int32_t check_camera(const abcd_camera* c) {
  REQUIRE(c != nullptr, "camera is NULL");
  REQUIRE(c->width > 0 && c->height > 0, "image size %dx%d must be positive", c->width, c->height);
  const int64_t tiles = (int64_t)tiles_x(c->width) * tiles_y(c->height);
  REQUIRE(tiles <= ABCD_MAX_TILES, "%lld tiles exceed the limit %d", (long long)tiles,
          ABCD_MAX_TILES);
  REQUIRE(std::isfinite(c->fx) && std::isfinite(c->fy) && c->fx > 0 && c->fy > 0,
          "focal lengths must be positive and finite");
  REQUIRE(std::isfinite(c->cx) && std::isfinite(c->cy), "principal point must be finite");
  // depth keys are fp32 bit patterns, which order as unsigned integers only
  // for positive depths
  REQUIRE(std::isfinite(c->near_plane) && c->near_plane > 0.0f,
          "near_plane must be positive and finite");
  for (int i = 0; i < 9; ++i) REQUIRE(std::isfinite(c->R[i]), "R must be finite");
  for (int i = 0; i < 3; ++i)
    REQUIRE(std::isfinite(c->t[i]) && std::isfinite(c->campos[i]), "t and campos must be finite");
  return ABCD_OK;
}

int32_t check_params(const abcd_raster_params* p) {
  REQUIRE(p != nullptr, "raster params are NULL");
  REQUIRE(p->sh_degree >= 0 && p->sh_degree <= 3, "sh_degree %d not in [0, 3]", p->sh_degree);
  REQUIRE((p->flags & ~ABCD_FLAG_FB_STOP) == 0, "unknown flags 0x%x", p->flags);
  REQUIRE(p->alpha_min >= 0 && p->alpha_max > 0 && p->alpha_max < 1 && p->alpha_min <= p->alpha_max,
          "need 0 <= alpha_min <= alpha_max < 1");
  REQUIRE(p->t_min >= 0 && p->t_min < 1, "t_min must be in [0, 1)");
  REQUIRE(p->eps2d >= 0 && std::isfinite(p->eps2d), "eps2d must be finite and >= 0");
  REQUIRE(p->radius_sigmas > 0 && std::isfinite(p->radius_sigmas), "radius_sigmas must be > 0");
  REQUIRE(p->guard > 0 && std::isfinite(p->guard), "guard must be > 0");
  return ABCD_OK;
}

// The split workspace shared by a forward and its backward (NULL: no split).
int32_t check_split(const abcd_split* sp, SplitLayout* out) {
  *out = SplitLayout{};
  if (!sp) return ABCD_OK;
  REQUIRE(sp->workspace != nullptr && (reinterpret_cast<uintptr_t>(sp->workspace) & 255) == 0,
          "split workspace must be non-NULL and 256-byte aligned");
  REQUIRE(sp->chunk > 0 && sp->chunk % 256 == 0 && sp->chunk <= (1 << 24),
          "split chunk %d must be a positive multiple of 256, at most 2^24", sp->chunk);
  REQUIRE(split_slots(sp->bytes) > 0, "split workspace of %zu bytes holds no checkpoint slot",
          sp->bytes);
  *out = split_layout(sp->workspace, sp->bytes, sp->chunk);
  return ABCD_OK;
}

int32_t check_n(int64_t n) {
  REQUIRE(n >= 0 && n <= ABCD_MAX_GAUSSIANS, "n = %lld out of range", (long long)n);
  return ABCD_OK;
}

#define TRY(x)                    \
  do {                            \
    int32_t st_ = (x);            \
    if (st_ != ABCD_OK) return st_; \
  } while (0)

// Scratch of abcd_render_bwd_noalloc: the backward's workspace for up to
// ABCD_NOALLOC_MAX_GAUSSIANS Gaussians, as a static device array. Each GPU
// the library runs on holds its own copy at its own address until the process
// ends. In host code `scratch` names a host-side stand-in, not device memory:
// only the address hipGetSymbolAddress returns for the current device may be
// passed to kernels or copies.
constexpr size_t kNoAllocScratchBytes = bwd_workspace_bytes(ABCD_NOALLOC_MAX_GAUSSIANS);
static_assert(kNoAllocScratchBytes == ABCD_NOALLOC_SCRATCH_BYTES,
              "ABCD_NOALLOC_SCRATCH_BYTES states the static scratch size");
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch`, looked up once per device
// (with that device current) and kept.
int32_t noalloc_scratch(void** out) {
  int dev = -1;
  ABCD_HIP(hipGetDevice(&dev));
  REQUIRE(dev >= 0 && dev < kMaxDevices, "device %d beyond the %d the library tracks", dev,
          kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    ABCD_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    REQUIRE(p != nullptr, "no device address for the static scratch on device %d", dev);
    REQUIRE((reinterpret_cast<uintptr_t>(p) & 255) == 0, "static scratch is not 256-byte aligned");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ABCD_OK;
}

}  // namespace

extern "C" {

const char* abcd_last_error(void) { return g_err; }
const char* abcd_version(void) { return ABCD_VERSION_STRING; }

const char* abcd_status_string(int32_t s) {
  switch (s) {
    case ABCD_OK: return "ABCD_OK";
    case ABCD_E_INVALID: return "ABCD_E_INVALID";
    case ABCD_E_CAPACITY: return "ABCD_E_CAPACITY";
    case ABCD_E_OVERFLOW: return "ABCD_E_OVERFLOW";
    case ABCD_E_HIP: return "ABCD_E_HIP";
    default: return "unknown status";
  }
}

int32_t abcd_project(const abcd_camera* cam, const abcd_raster_params* prm, int64_t n,
                     const float* means, const float* log_scales, const float* quats,
                     const float* opacity_logits, const float* sh, float* means2d,
                     float* conic_opacity, float* depth, float* extent, uint32_t* tiles_touched,
                     float* rgb, hipStream_t stream) {
  TRY(check_camera(cam));
  TRY(check_params(prm));
  TRY(check_n(n));
  if (n > 0) {
    REQUIRE(means && log_scales && quats && opacity_logits && sh, "parameter array is NULL");
    REQUIRE(means2d && conic_opacity && depth && extent && tiles_touched && rgb,
            "output array is NULL");
    REQUIRE((reinterpret_cast<uintptr_t>(conic_opacity) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(quats) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(means2d) & 7) == 0 &&
                (reinterpret_cast<uintptr_t>(extent) & 7) == 0,
            "quats and conic_opacity must be 16-byte, means2d and extent 8-byte aligned");
  }
  return launch_project(*cam, *prm, n, means, log_scales, quats, opacity_logits, sh, means2d,
                        conic_opacity, depth, extent, tiles_touched, rgb, stream);
}

int32_t abcd_bin_sort_workspace_size(int64_t n, int64_t capacity, int32_t width, int32_t height,
                                     size_t* bytes) {
  TRY(check_n(n));
  REQUIRE(bytes != nullptr, "bytes is NULL");
  REQUIRE(capacity >= 0 && capacity < (1ll << 32), "capacity must be in [0, 2^32)");
  REQUIRE(width > 0 && height > 0, "image size must be positive");
  const int64_t tiles = (int64_t)tiles_x(width) * tiles_y(height);
  REQUIRE(tiles <= ABCD_MAX_TILES, "too many tiles");
  *bytes = bin_sort_workspace_bytes(n, capacity, width, height);
  return ABCD_OK;
}

int32_t abcd_bin_sort(int32_t width, int32_t height, int64_t n, const float* means2d,
                      const float* extent, const float* depth, const uint32_t* tiles_touched,
                      int64_t capacity, void* workspace, size_t ws_bytes, uint64_t* keys_sorted,
                      uint32_t* values_sorted, uint32_t* tile_ranges, uint32_t* tile_order,
                      int64_t* n_isect, hipStream_t stream) {
  TRY(check_n(n));
  REQUIRE(width > 0 && height > 0, "image size must be positive");
  const int64_t tiles = (int64_t)tiles_x(width) * tiles_y(height);
  REQUIRE(tiles <= ABCD_MAX_TILES, "too many tiles");
  REQUIRE(capacity >= 0 && capacity < (1ll << 32), "capacity must be in [0, 2^32)");
  REQUIRE(tile_ranges != nullptr, "tile_ranges is NULL");
  REQUIRE(workspace != nullptr, "workspace is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(workspace) & 255) == 0, "workspace must be 256-byte aligned");
  const size_t need = bin_sort_workspace_bytes(n, capacity, width, height);
  REQUIRE(ws_bytes >= need, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  if (n > 0) {
    REQUIRE(means2d && extent && depth && tiles_touched, "input array is NULL");
    REQUIRE((reinterpret_cast<uintptr_t>(means2d) & 7) == 0 &&
                (reinterpret_cast<uintptr_t>(extent) & 7) == 0,
            "means2d and extent must be 8-byte aligned");
  }
  REQUIRE(capacity == 0 || values_sorted != nullptr, "values_sorted is NULL with capacity > 0");
  TRY(launch_bin_sort(width, height, n, means2d, extent, depth, tiles_touched, capacity, workspace,
                      keys_sorted, values_sorted, tile_ranges, tile_order, stream));
  if (n_isect) {
    unsigned long long m = 0;
    ABCD_HIP(hipMemcpyAsync(&m, workspace, sizeof m, hipMemcpyDeviceToHost, stream));
    ABCD_HIP(hipStreamSynchronize(stream));
    *n_isect = (int64_t)m;
    if (m >= (1ull << 32)) {
      set_error("%llu intersections do not fit 32-bit indices", m);
      return ABCD_E_OVERFLOW;
    }
    if ((int64_t)m > capacity) {
      set_error("%llu intersections exceed the capacity %lld", m, (long long)capacity);
      return ABCD_E_CAPACITY;
    }
  }
  return ABCD_OK;
}

int32_t abcd_render_fwd(const abcd_camera* cam, const abcd_raster_params* prm,
                        const uint32_t* tile_ranges, const uint32_t* tile_order,
                        const uint32_t* values_sorted,
                        const float* means2d, const float* conic_opacity, const float* rgb,
                        const float* F, const float* B, float* out_rgba, float* final_T,
                        uint32_t* last, unsigned long long* n_blends, const abcd_split* split,
                        hipStream_t stream) {
  TRY(check_camera(cam));
  TRY(check_params(prm));
  SplitLayout sl;
  TRY(check_split(split, &sl));
  REQUIRE(tile_ranges && out_rgba && final_T && last, "tile_ranges or an output is NULL");
  REQUIRE(values_sorted && means2d && conic_opacity && rgb,
          "values_sorted, means2d, conic_opacity or rgb is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(out_rgba) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(F) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(B) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(conic_opacity) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(means2d) & 7) == 0,
          "RGBA images and conic_opacity must be 16-byte aligned, means2d 8-byte aligned");
  return launch_render_fwd(*cam, *prm, tile_ranges, values_sorted, means2d, conic_opacity, rgb, F,
                           B, out_rgba, final_T, last, n_blends, tile_order, sl, stream);
}

int32_t abcd_render_cache(const abcd_camera* cam, const abcd_raster_params* prm,
                          const uint32_t* tile_ranges, const uint32_t* tile_order,
                          const uint32_t* values_sorted, const float* means2d,
                          const float* conic_opacity, const float* rgb, uint16_t* image_f16,
                          int32_t* rect, hipStream_t stream) {
  TRY(check_camera(cam));
  TRY(check_params(prm));
  REQUIRE(tile_ranges && image_f16, "tile_ranges or image_f16 is NULL");
  REQUIRE(values_sorted && means2d && conic_opacity && rgb,
          "values_sorted, means2d, conic_opacity or rgb is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(image_f16) & 7) == 0 &&
              (reinterpret_cast<uintptr_t>(conic_opacity) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(means2d) & 7) == 0,
          "image_f16 and means2d must be 8-byte aligned, conic_opacity 16-byte aligned");
  REQUIRE((reinterpret_cast<uintptr_t>(rect) & 3) == 0, "rect must be 4-byte aligned");
  return launch_render_cache(*cam, *prm, tile_ranges, tile_order, values_sorted, means2d,
                             conic_opacity, rgb, image_f16, rect, stream);
}

int32_t abcd_split_workspace_size(int64_t n_slots, size_t* bytes) {
  REQUIRE(bytes != nullptr, "bytes is NULL");
  REQUIRE(n_slots >= 1 && n_slots <= 0x7FFF0000ll, "n_slots %lld not in [1, 2^31)",
          (long long)n_slots);
  *bytes = split_bytes((uint32_t)n_slots);
  return ABCD_OK;
}

int32_t abcd_render_bwd_workspace_size(int64_t n, size_t* bytes) {
  TRY(check_n(n));
  REQUIRE(bytes != nullptr, "bytes is NULL");
  *bytes = render_bwd_workspace_bytes(n);
  return ABCD_OK;
}

static int32_t render_bwd_impl(const abcd_camera* cam, const abcd_raster_params* prm, int64_t n,
                        const float* means, const float* log_scales, const float* quats,
                        const float* opacity_logits, const float* sh, const float* means2d,
                        const float* conic_opacity, const float* rgb, const float* extent,
                        const uint32_t* tile_ranges, const uint32_t* values_sorted,
                        const float* F, const float* B, const float* final_T, const uint32_t* last,
                        const float* dL_dout, void* workspace, size_t ws_bytes, float* d_means,
                        float* d_log_scales, float* d_quats, float* d_opacity_logits, float* d_sh,
                        float* d_means2d, int32_t accumulate, const abcd_split* split,
                        bool noalloc, hipStream_t stream) {
  TRY(check_camera(cam));
  TRY(check_params(prm));
  SplitLayout sl;
  TRY(check_split(split, &sl));
  TRY(check_n(n));
  REQUIRE(tile_ranges && final_T && last && dL_dout, "tile_ranges, final_T, last or dL_dout is NULL");
  REQUIRE(n == 0 || values_sorted, "values_sorted is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(dL_dout) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(F) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(B) & 15) == 0,
          "RGBA images must be 16-byte aligned");
  const size_t need = render_bwd_workspace_bytes(n);
  if (n > 0) {
    REQUIRE(means && log_scales && quats && opacity_logits && sh && means2d && conic_opacity &&
                rgb && extent,
            "input array is NULL");
    REQUIRE(d_means && d_log_scales && d_quats && d_opacity_logits && d_sh, "gradient array is NULL");
    if (noalloc) {
      REQUIRE(n <= ABCD_NOALLOC_MAX_GAUSSIANS,
              "n = %lld exceeds the %lld Gaussians the static scratch of "
              "abcd_render_bwd_noalloc holds; use abcd_render_bwd with a workspace",
              (long long)n, (long long)ABCD_NOALLOC_MAX_GAUSSIANS);
    } else {
      REQUIRE(workspace != nullptr && (reinterpret_cast<uintptr_t>(workspace) & 255) == 0,
              "workspace must be non-NULL and 256-byte aligned");
      REQUIRE(ws_bytes >= need, "workspace of %zu bytes, %zu needed", ws_bytes, need);
    }
    REQUIRE((reinterpret_cast<uintptr_t>(conic_opacity) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(quats) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(d_quats) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(means2d) & 7) == 0,
            "quats, d_quats and conic_opacity must be 16-byte and means2d 8-byte aligned");
  } else {
    return ABCD_OK;
  }
  // every argument is valid: only now the static scratch's address (a HIP call)
  if (noalloc) TRY(noalloc_scratch(&workspace));
  float* g2d = static_cast<float*>(workspace);
  TRY(launch_render_bwd_pixels(*cam, *prm, n, tile_ranges, values_sorted, means2d, conic_opacity,
                               rgb, F, B, final_T, last, dL_dout, g2d, sl, stream));
  return launch_project_bwd(*cam, *prm, n, means, log_scales, quats, opacity_logits, sh, extent,
                            g2d, d_means, d_log_scales, d_quats, d_opacity_logits, d_sh, d_means2d,
                            accumulate, stream);
}

int32_t abcd_render_bwd(const abcd_camera* cam, const abcd_raster_params* prm, int64_t n,
                        const float* means, const float* log_scales, const float* quats,
                        const float* opacity_logits, const float* sh, const float* means2d,
                        const float* conic_opacity, const float* rgb, const float* extent,
                        const uint32_t* tile_ranges, const uint32_t* values_sorted,
                        const float* F, const float* B, const float* final_T, const uint32_t* last,
                        const float* dL_dout, void* workspace, size_t ws_bytes, float* d_means,
                        float* d_log_scales, float* d_quats, float* d_opacity_logits, float* d_sh,
                        float* d_means2d, int32_t accumulate, const abcd_split* split,
                        hipStream_t stream) {
  return render_bwd_impl(cam, prm, n, means, log_scales, quats, opacity_logits, sh, means2d,
                         conic_opacity, rgb, extent, tile_ranges, values_sorted, F, B, final_T,
                         last, dL_dout, workspace, ws_bytes, d_means, d_log_scales, d_quats,
                         d_opacity_logits, d_sh, d_means2d, accumulate, split, false, stream);
}

int32_t abcd_render_bwd_noalloc(const abcd_camera* cam, const abcd_raster_params* prm, int64_t n,
                                const float* means, const float* log_scales, const float* quats,
                                const float* opacity_logits, const float* sh,
                                const float* means2d, const float* conic_opacity,
                                const float* rgb, const float* extent,
                                const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                const float* F, const float* B, const float* final_T,
                                const uint32_t* last, const float* dL_dout, float* d_means,
                                float* d_log_scales, float* d_quats, float* d_opacity_logits,
                                float* d_sh, float* d_means2d, int32_t accumulate,
                                const abcd_split* split, hipStream_t stream) {
  return render_bwd_impl(cam, prm, n, means, log_scales, quats, opacity_logits, sh, means2d,
                         conic_opacity, rgb, extent, tile_ranges, values_sorted, F, B, final_T,
                         last, dL_dout, nullptr, kNoAllocScratchBytes, d_means, d_log_scales,
                         d_quats, d_opacity_logits, d_sh, d_means2d, accumulate, split, true,
                         stream);
}

int32_t abcd_stage_cached(int32_t width, int32_t height, int32_t k,
                          const uint16_t* const* host_images, const int32_t* rects,
                          uint16_t* dst, hipStream_t stream) {
  REQUIRE(width > 0 && height > 0, "image size must be positive");
  REQUIRE(k >= 0, "k must be >= 0");
  if (k == 0) return ABCD_OK;
  REQUIRE(host_images && dst, "host_images or dst is NULL");
  for (int j = 0; j < k; ++j) {
    REQUIRE(host_images[j] != nullptr, "host_images[%d] is NULL", j);
    if (!rects) continue;
    const int32_t* r = rects + 4 * j;
    REQUIRE(r[0] >= 0 && r[1] >= 0 && r[2] <= width && r[3] <= height,
            "rect %d (%d, %d, %d, %d) leaves the %dx%d image", j, r[0], r[1], r[2], r[3], width,
            height);
  }
  return stage_cached(width, height, k, host_images, rects, dst, stream);
}

int32_t abcd_composite_cache(int32_t width, int32_t height, int32_t k, const uint16_t* images,
                             const int32_t* order, int32_t n_front, const int32_t* rects,
                             float stop_t, float* F, float* B, int32_t flags,
                             hipStream_t stream) {
  REQUIRE(width > 0 && height > 0, "image size must be positive");
  REQUIRE((flags & ~(ABCD_COMPOSITE_ACCUMULATE | ABCD_COMPOSITE_BESIDE)) == 0,
          "unknown composite flags 0x%x", (unsigned)flags);
  REQUIRE(stop_t >= 0.0f && stop_t < 1.0f, "stop_t must be in [0, 1)");
  REQUIRE((reinterpret_cast<uintptr_t>(rects) & 15) == 0, "rects must be 16-byte aligned");
  REQUIRE(k >= 0, "k must be >= 0");
  REQUIRE(n_front >= 0 && n_front <= k, "n_front %d not in [0, %d]", n_front, k);
  REQUIRE(F && B, "F or B is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(F) & 15) == 0 && (reinterpret_cast<uintptr_t>(B) & 15) == 0,
          "F and B must be 16-byte aligned");
  if (k > 0) {
    REQUIRE(images && order, "images or order is NULL");
    REQUIRE((reinterpret_cast<uintptr_t>(images) & 7) == 0, "images must be 8-byte aligned");
    std::vector<char> seen(k, 0);
    for (int j = 0; j < k; ++j) {
      REQUIRE(order[j] >= 0 && order[j] < k && !seen[order[j]], "order is not a permutation of 0..k-1");
      seen[order[j]] = 1;
    }
  }
  return launch_composite(width, height, k, images, order, n_front, rects, stop_t, F, B,
                          (flags & ABCD_COMPOSITE_ACCUMULATE) ? 1 : 0,
                          (flags & ABCD_COMPOSITE_BESIDE) != 0, stream);
}

int32_t abcd_loss_l1_grad(int32_t width, int32_t height, const float* out_rgba,
                          const float* target_rgb, const float* bg, float* dL_dout, float* loss,
                          hipStream_t stream) {
  REQUIRE(width > 0 && height > 0, "image size must be positive");
  REQUIRE(out_rgba && target_rgb && dL_dout, "image array is NULL");
  REQUIRE((reinterpret_cast<uintptr_t>(out_rgba) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(dL_dout) & 15) == 0,
          "RGBA images must be 16-byte aligned");
  const float b0 = bg ? bg[0] : 0.0f, b1 = bg ? bg[1] : 0.0f, b2 = bg ? bg[2] : 0.0f;
  return launch_loss_l1(width, height, out_rgba, target_rgb, b0, b1, b2, dL_dout, loss, stream);
}

int32_t abcd_adam_step(const abcd_adam_group* groups, int32_t n_groups, float beta1, float beta2,
                       float eps, int64_t step, hipStream_t stream) {
  REQUIRE(n_groups >= 0 && n_groups <= ABCD_ADAM_MAX_GROUPS, "n_groups must be in [0, %d]",
          ABCD_ADAM_MAX_GROUPS);
  REQUIRE(n_groups == 0 || groups != nullptr, "groups is NULL");
  REQUIRE(beta1 >= 0.0f && beta1 < 1.0f && beta2 >= 0.0f && beta2 < 1.0f,
          "beta1 and beta2 must be in [0, 1)");
  REQUIRE(eps >= 0.0f && std::isfinite(eps), "eps must be finite and >= 0");
  REQUIRE(step >= 1, "step must be >= 1");
  for (int32_t i = 0; i < n_groups; ++i) {
    const abcd_adam_group& g = groups[i];
    REQUIRE(g.count >= 0, "group %d: count < 0", i);
    REQUIRE(std::isfinite(g.lr), "group %d: lr is not finite", i);
    if (g.count > 0)
      REQUIRE(g.param && g.grad && g.exp_avg && g.exp_avg_sq, "group %d: array is NULL", i);
  }
  return launch_adam(groups, n_groups, beta1, beta2, eps, step, stream);
}

int32_t abcd_timing_enable(int32_t enable) {
  g_timing = enable != 0;
  return ABCD_OK;
}

int32_t abcd_timing_reset(void) {
  for (auto& r : g_recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_recs.clear();
  return ABCD_OK;
}

int32_t abcd_timing_read(const char* kernel, double* total_ms, int64_t* launches) {
  REQUIRE(kernel && total_ms && launches, "NULL argument");
  double tot = 0.0;
  int64_t cnt = 0;
  for (auto& r : g_recs) {
    if (r.name != kernel) continue;
    ABCD_HIP(hipEventSynchronize(r.b));
    float ms = 0.0f;
    ABCD_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    tot += ms;
    ++cnt;
  }
  *total_ms = tot;
  *launches = cnt;
  return ABCD_OK;
}

}  // extern "C"

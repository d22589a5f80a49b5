// composite.hip -- collapse of cached per-partition renders into F and B.
//
// The paper pre-renders every frozen partition per camera and, by the
// associativity of alpha compositing, collapses the renders in front of the
// active partition into F and those behind it into B (Abstract; Method
// section). Per pixel this is a left fold of premultiplied "over":
//   acc <- acc + (1 - acc_alpha) x,
// over the fp16 cached images in front-to-back order. The kernel is a pure
// HBM stream (8 bytes per layer-pixel read, 32 per pixel written): each thread
// owns two adjacent pixels, so every layer is one 16-byte load per thread;
// 16 loads are in flight per thread, marked non-temporal (each byte is read
// once), and the layer order travels in the kernel arguments. This runs at
// the rate of a device-to-device copy.
#include "abcd_internal.h"

namespace abcd {
namespace {

constexpr int kMaxLayers = 448;  // layers per launch (order table in kernel arguments)
constexpr int64_t kCompositeBesideGrid = 512;  // workgroups beside other work (two per CU)
constexpr int kBatch = 16;       // loads in flight per thread

struct LayerTable {
  int32_t idx[kMaxLayers];
};

// modes: 0 overwrite with the fold, 1 fold behind the incoming value, 2 leave untouched
struct FoldPlan {
  int nf, nb, mode_f, mode_b;
};

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 to_f4(uint2 bits) {
  const h4 h = __builtin_bit_cast(h4, bits);
  return make_float4((float)h[0], (float)h[1], (float)h[2], (float)h[3]);
}

__device__ __forceinline__ void over(float4& acc, const float4 x) {
  const float s = 1.0f - acc.w;
  acc.x += s * x.x;
  acc.y += s * x.y;
  acc.z += s * x.z;
  acc.w += s * x.w;
}

// Coordinates of the (one or two) pixels a thread folds.
struct PixPos {
  int x0, y0, x1, y1;
};

__device__ __forceinline__ bool in_rect(const int4 r, int x, int y) {
  return x >= r.x && x < r.z && y >= r.y && y < r.w;
}

// Fold layers tab[first .. first+count) at pixel pair `pp` (or single pixel).
// rects (may be NULL): per image, the pixel box outside which it is fully
// transparent; a layer is not read where it cannot contribute (folding a
// transparent layer leaves the accumulator bit-identical, so this changes no
// result). kStop: a pixel takes no further layer once the weight it could
// still give one, (1 - acc_alpha) vis, is below stop_t; a wave whose pixels
// have all stopped leaves the loop.
template <bool kPair, bool kStop>
__device__ __forceinline__ void fold(const uint2* __restrict__ img, int64_t npix, int64_t pp,
                                     const LayerTable& tab, int first, int count,
                                     const int4* __restrict__ rects, const PixPos& pos,
                                     float stop_t, float vis0, float vis1, float4& a0,
                                     float4& a1) {
  for (int j0 = 0; j0 < count; j0 += kBatch) {
    const int m = min(kBatch, count - j0);
    bool live = true;
    if (kStop) {
      live = (1.0f - a0.w) * vis0 >= stop_t || (kPair && (1.0f - a1.w) * vis1 >= stop_t);
      if (!__ballot(live)) break;  // wave-uniform
    }
    // which of the batch's layers any pixel of the wave needs (a wave-uniform
    // mask): layers whose box misses the whole wave cost no load and no fold
    bool need[kBatch];
    uint32_t wave_needs = 0;
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      need[b] = false;
      if (b < m) {
        need[b] = live;
        if (rects) {
          const int4 r = rects[tab.idx[first + j0 + b]];
          need[b] = need[b] && (in_rect(r, pos.x0, pos.y0) || (kPair && in_rect(r, pos.x1, pos.y1)));
        }
        if (__ballot(need[b])) wave_needs |= 1u << b;
      }
    }
    wave_needs = __builtin_amdgcn_readfirstlane(wave_needs);
    uint4 v[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      v[b] = make_uint4(0u, 0u, 0u, 0u);
      if ((wave_needs >> b) & 1u) {
        const int idx = tab.idx[first + j0 + b];
        if (need[b]) {
          const uint2* src = img + (int64_t)idx * npix + pp;
          if (kPair) {
            const u4v t = __builtin_nontemporal_load(reinterpret_cast<const u4v*>(src));
            v[b] = make_uint4(t[0], t[1], t[2], t[3]);
          } else {
            const uint2 s = *src;
            v[b] = make_uint4(s.x, s.y, 0u, 0u);
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      if ((wave_needs >> b) & 1u) {
        if (!kStop || (1.0f - a0.w) * vis0 >= stop_t) over(a0, to_f4(make_uint2(v[b].x, v[b].y)));
        if (kPair && (!kStop || (1.0f - a1.w) * vis1 >= stop_t))
          over(a1, to_f4(make_uint2(v[b].z, v[b].w)));
      }
    }
  }
}

template <bool kPair, bool kStop>
__global__ __launch_bounds__(256) void composite_kernel(int64_t npix, int width,
                                                        const uint2* __restrict__ img,
                                                        LayerTable tab, FoldPlan plan,
                                                        const int4* __restrict__ rects,
                                                        float stop_t, float4* __restrict__ F,
                                                        float4* __restrict__ B) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; (kPair ? 2 * t : t) < npix;
       t += stride) {
  const int64_t pp = kPair ? 2 * t : t;
  PixPos pos;
  pos.x0 = (int)((uint32_t)pp % (uint32_t)width);
  pos.y0 = (int)((uint32_t)pp / (uint32_t)width);
  pos.x1 = pos.x0 + 1;
  pos.y1 = pos.y0;
  if (pos.x1 == width) {
    pos.x1 = 0;
    pos.y1 += 1;
  }
  const float4 zero = make_float4(0, 0, 0, 0);
  // F
  float4 f0 = zero, f1 = zero;
  if (plan.mode_f != 2) {
    f0 = plan.mode_f == 1 ? F[pp] : zero;
    f1 = (kPair && plan.mode_f == 1) ? F[pp + 1] : zero;
    fold<kPair, kStop>(img, npix, pp, tab, 0, plan.nf, rects, pos, stop_t, 1.0f, 1.0f, f0, f1);
    F[pp] = f0;
    if (kPair) F[pp + 1] = f1;
  } else if (kStop && plan.mode_b != 2) {
    f0 = F[pp];
    if (kPair) f1 = F[pp + 1];
  }
  // B, weighted by what F leaves visible
  if (plan.mode_b != 2) {
    float4 a0 = plan.mode_b == 1 ? B[pp] : zero;
    float4 a1 = (kPair && plan.mode_b == 1) ? B[pp + 1] : zero;
    fold<kPair, kStop>(img, npix, pp, tab, plan.nf, plan.nb, rects, pos, stop_t, 1.0f - f0.w,
                       1.0f - f1.w, a0, a1);
    B[pp] = a0;
    if (kPair) B[pp + 1] = a1;
  }
  }
}

}  // namespace

int32_t launch_composite(int width, int height, int k, const uint16_t* images,
                         const int32_t* order, int n_front, const int32_t* rects, float stop_t,
                         float* F, float* B, int accumulate, bool beside, hipStream_t stream) {
  const int64_t npix = (int64_t)width * height;
  const uint2* img = reinterpret_cast<const uint2*>(images);
  // pairs need 16-byte alignment of every layer: even pixel count, aligned base
  const bool pair = (npix % 2 == 0) && ((reinterpret_cast<uintptr_t>(images) & 15) == 0) &&
                    ((reinterpret_cast<uintptr_t>(F) & 31) == 0) &&
                    ((reinterpret_cast<uintptr_t>(B) & 31) == 0);
  const int64_t threads = pair ? npix / 2 : npix;
  // beside: a bounded grid (each thread takes every grid-th pixel pair)
  // leaves room on the CUs for work on other streams (the binning of the step)
  int64_t blocks = (threads + kBlock - 1) / kBlock;
  if (beside) blocks = std::min<int64_t>(blocks, kCompositeBesideGrid);
  int fi = 0, bi = 0;
  const int nfront = n_front, nback = k - n_front;
  bool first = true;
  if (k == 0 && accumulate) return ABCD_OK;
  while (first || fi < nfront || bi < nback) {
    LayerTable tab;
    FoldPlan plan;
    plan.nf = std::min(nfront - fi, kMaxLayers);
    plan.nb = std::min(nback - bi, kMaxLayers - plan.nf);
    for (int j = 0; j < plan.nf; ++j) tab.idx[j] = order[fi + j];
    for (int j = 0; j < plan.nb; ++j) tab.idx[plan.nf + j] = order[n_front + bi + j];
    // a layer group that gets no layers in this launch is left alone, except
    // on the first launch without accumulation, which must write transparent
    plan.mode_f = (fi > 0 || accumulate) ? (plan.nf ? 1 : 2) : 0;
    plan.mode_b = (bi > 0 || accumulate) ? (plan.nb ? 1 : 2) : 0;
    if (!first && plan.nf == 0) plan.mode_f = 2;
    if (!first && plan.nb == 0) plan.mode_b = 2;
    const int4* r4 = reinterpret_cast<const int4*>(rects);
    float4* F4 = reinterpret_cast<float4*>(F);
    float4* B4 = reinterpret_cast<float4*>(B);
    if (pair && stop_t > 0.0f) {
      ABCD_LAUNCH("composite", (composite_kernel<true, true>), blocks, kBlock, 0, stream, npix,
                  width, img, tab, plan, r4, stop_t, F4, B4);
    } else if (pair) {
      ABCD_LAUNCH("composite", (composite_kernel<true, false>), blocks, kBlock, 0, stream, npix,
                  width, img, tab, plan, r4, stop_t, F4, B4);
    } else if (stop_t > 0.0f) {
      ABCD_LAUNCH("composite", (composite_kernel<false, true>), blocks, kBlock, 0, stream, npix,
                  width, img, tab, plan, r4, stop_t, F4, B4);
    } else {
      ABCD_LAUNCH("composite", (composite_kernel<false, false>), blocks, kBlock, 0, stream, npix,
                  width, img, tab, plan, r4, stop_t, F4, B4);
    }
    ABCD_HIP(hipGetLastError());
    fi += plan.nf;
    bi += plan.nb;
    first = false;
  }
  return ABCD_OK;
}

}  // namespace abcd

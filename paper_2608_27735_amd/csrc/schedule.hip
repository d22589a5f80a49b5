// schedule.hip -- the order in which the blend kernels take their tiles.
//
// Per-tile work in the blend kernels is very uneven (a tile's walk length
// ranges over two orders of magnitude), and a workgroup holds its CU slot
// until its slowest wave finishes. Launched in raster order, a few heavy tiles
// start late and run on an otherwise idle GPU. Taking tiles heaviest first
// (longest-processing-time order) lets the light tiles fill in around them.
//
// The work estimate is the tile's list length for the forward (known after
// binning) and, for the backward (known after the forward), the most entries
// the forward staged in one chunk of the tile's walk when the tile may be
// split, else the tile's largest per-pixel walk length; a tile's work items
// (its chunks) follow one another. The order is a stable bucket sort by the
// estimate's quarter octave (leading one and the two bits after it), so tiles
// of one bucket keep their raster order and neighbouring tiles stay close in
// launch order.
#include "schedule.h"

namespace abcd {
namespace {

// Largest per-pixel walk length (the forward's `last`) of each tile.
__global__ __launch_bounds__(kBlock) void tile_walk_kernel(int width, int height, int ntx,
                                                           const uint32_t* __restrict__ last,
                                                           uint32_t* __restrict__ work) {
  __shared__ uint32_t s_m;
  const int tile = blockIdx.x;
  const int px = (tile % ntx) * kTile + (threadIdx.x & 15);
  const int py = (tile / ntx) * kTile + (threadIdx.x >> 4);
  if (threadIdx.x == 0) s_m = 0;
  __syncthreads();
  uint32_t v = (px < width && py < height) ? last[(int64_t)py * width + px] : 0u;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
  if ((threadIdx.x & 63) == 0 && v) atomicMax(&s_m, v);
  __syncthreads();
  if (threadIdx.x == 0) work[tile] = s_m;
}

// Work items of the backward, in the order s_order (tiles by decreasing
// estimated work, workgroup memory): a tile with no walk has none, a tile
// the forward split (it has an end-of-walk slot) one per chunk its walk
// reaches, any other tile one (s_nt: items per tile, workgroup memory).
// Writes items (tile, chunk), queue[0] = their number and zeroes the
// counters of the kQueues queues (the heads the backward's workgroups
// advance). Wave w takes the positions of one contiguous range: their item
// count, then (once every wave's count is known) their items, 64 positions
// at a time with a running offset.
__device__ __forceinline__ void build_items(int ntiles, const uint16_t* s_order,
                                            const uint8_t* s_nt, uint2* __restrict__ items,
                                            uint32_t cap, uint32_t* __restrict__ queue) {
  __shared__ uint32_t s_wsum[kOrderWaves];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int per = (ntiles + kOrderWaves - 1) / kOrderWaves;
  const int i0 = min(ntiles, w * per), i1 = min(ntiles, i0 + per);
  uint32_t mine = 0;
  for (int i = i0 + l; i < i1; i += 64) mine += s_nt[s_order[i]];
  mine = wave_sum_u32(mine);
  if (l == 0) s_wsum[w] = mine;
  __syncthreads();
  uint32_t off = 0, total = 0;
#pragma unroll
  for (int v = 0; v < kOrderWaves; ++v) {
    const uint32_t c = s_wsum[v];
    off += v < w ? c : 0u;
    total += c;
  }
  for (int ib = i0; ib < i1; ib += 64) {
    const int i = ib + l;
    const uint32_t t = i < i1 ? s_order[i] : 0u;
    const uint32_t n = i < i1 ? s_nt[t] : 0u;
    uint32_t inc = n;  // inclusive prefix of n over the 64 positions
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)inc, d, 64);
      if (l >= d) inc += y;
    }
    const uint32_t at = off + inc - n;
    for (uint32_t jj = 0; jj < n && at + jj < cap; ++jj) items[at + jj] = make_uint2(t, jj);
    off += (uint32_t)__shfl((int)inc, 63, 64);
  }
  if (tid == 0) queue[0] = min(total, cap);
  if (tid < kQueues) queue[kQueueStride * tid + 1] = 0;
}

// The backward's schedule in one launch: workgroup 0 orders the tiles by
// `key` and writes the work items in that order (walk: each tile's largest
// per-pixel walk; every global load -- key, walk and the split slot of each
// tile -- is issued in its first loop, the rest works in workgroup memory);
// the other workgroups clear zero[0, zero_count) meanwhile (16-byte stores).
__global__ __launch_bounds__(kOrderThreads) void bwd_schedule_kernel(
    int ntiles, const uint32_t* __restrict__ key, const uint32_t* __restrict__ walk,
    uint32_t* __restrict__ order, SplitLayout sp, uint2* __restrict__ items, uint32_t cap,
    uint32_t* __restrict__ queue, float4* __restrict__ zero, int64_t zero4) {
  __shared__ uint8_t s_key[ABCD_MAX_TILES];      // bucket of each tile
  __shared__ uint8_t s_nt[ABCD_MAX_TILES];       // work items of each tile
  __shared__ uint16_t s_order[ABCD_MAX_TILES];   // the order
  static_assert(ABCD_MAX_TILES <= 65536, "tile indices are kept in 16 bits");
  if (blockIdx.x > 0) {
    const int64_t stride = (int64_t)(gridDim.x - 1) * kOrderThreads;
    for (int64_t j = (int64_t)(blockIdx.x - 1) * kOrderThreads + threadIdx.x; j < zero4; j += stride)
      zero[j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    return;
  }
  // eight tiles per thread at a time, their loads issued together (indices
  // clamped into the arrays, so that no load waits behind a branch). With a
  // split, key is the forward's per-tile work whose bit 31 marks a split tile
  // (reading slot_of instead, one 256-byte-strided word per tile, took 13 us).
  constexpr int kAt = 8;
  for (int tb = 0; tb < ntiles; tb += kAt * kOrderThreads) {
    uint32_t wk[kAt], kk[kAt];
#pragma unroll
    for (int u = 0; u < kAt; ++u) {
      const int tc = min(tb + u * kOrderThreads + (int)threadIdx.x, ntiles - 1);
      wk[u] = walk[tc];
      kk[u] = key[tc];
    }
#pragma unroll
    for (int u = 0; u < kAt; ++u) {
      const int t = tb + u * kOrderThreads + (int)threadIdx.x;
      uint32_t n = wk[u] > 0 ? 1u : 0u;
      const bool split = sp.ckpt && (kk[u] & kSplitTile);
      if (wk[u] > 0 && split) {
        const uint32_t ch = (uint32_t)sp.ch;
        n = min((wk[u] + ch - 1) / ch, kMaxChunks);
      }
      if (t < ntiles) {
        s_key[t] = (uint8_t)bucket_of(sp.ckpt ? kk[u] & ~kSplitTile : kk[u]);
        s_nt[t] = (uint8_t)n;
      }
    }
  }
  __syncthreads();
  order_keyed(ntiles, s_key, order, s_order);
  build_items(ntiles, s_order, s_nt, items, cap, queue);
}

}  // namespace

int32_t launch_bwd_schedule(int ntiles, const uint32_t* key, const uint32_t* walk,
                            uint32_t* order, const SplitLayout& split, void* items, uint32_t cap,
                            uint32_t* queue, float* zero, int64_t zero_count,
                            hipStream_t stream) {
  // workgroups hold ~137 KB of LDS each (one per CU): one schedules, up to
  // 255 clear
  const int64_t zero4 = zero_count / 4;
  const int grid = 1 + (int)std::min<int64_t>(255, (zero4 + kOrderThreads - 1) / kOrderThreads);
  ABCD_LAUNCH("bwd_order", bwd_schedule_kernel, grid, kOrderThreads, 0, stream, ntiles, key, walk,
              order, split, reinterpret_cast<uint2*>(items), cap, queue,
              reinterpret_cast<float4*>(zero), zero4);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_tile_walk(int width, int height, const uint32_t* last, uint32_t* work,
                         hipStream_t stream) {
  const int ntiles = tiles_x(width) * tiles_y(height);
  if (ntiles <= 0) return ABCD_OK;
  ABCD_LAUNCH("bwd_order", tile_walk_kernel, ntiles, kBlock, 0, stream, width, height,
              tiles_x(width), last, work);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd

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

__global__ __launch_bounds__(kOrderThreads) void tile_order_kernel(int ntiles,
                                                                   const uint32_t* __restrict__ work,
                                                                   uint32_t* __restrict__ order,
                                                                   const uint32_t* __restrict__ skip) {
  __shared__ uint8_t s_key[ABCD_MAX_TILES];
  if (skip && *skip) return;
  order_tiles(ntiles, work, order, s_key);
}

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

// Work items of the backward, in the order of `order` (tiles by decreasing
// estimated work): a tile with no walk has none, a tile the forward split (it
// has an end-of-walk slot) one per chunk its walk reaches, any other tile
// one. Writes items (tile, chunk), queue[0] = their number and zeroes the
// counters of the kQueues queues (the heads the backward's workgroups
// advance). s_n is workgroup memory of
// ABCD_MAX_TILES bytes.
__device__ __forceinline__ void build_items(int ntiles, const uint32_t* __restrict__ order,
                                            const uint32_t* __restrict__ walk,
                                            const SplitLayout& sp, uint2* __restrict__ items,
                                            uint32_t cap, uint32_t* __restrict__ queue,
                                            uint8_t* s_n) {
  __shared__ uint32_t s_wsum[kOrderWaves];
  __shared__ uint32_t s_off;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  if (tid == 0) s_off = 0;
  // items per position of the order, the dependent loads of eight positions
  // in flight at once
#pragma unroll 8
  for (int i = tid; i < ntiles; i += kOrderThreads) {
    const uint32_t t = order[i];
    const uint32_t wk = walk[t];
    uint32_t n = wk > 0 ? 1u : 0u;
    if (wk > 0 && sp.ckpt && sp.slot_of[(size_t)t * kMaxChunks] < sp.nslots) {
      const uint32_t ch = (uint32_t)sp.ch;
      n = min((wk + ch - 1) / ch, kMaxChunks);
    }
    s_n[i] = (uint8_t)n;
  }
  __syncthreads();
  for (int i0 = 0; i0 < ntiles; i0 += kOrderThreads) {
    const int i = i0 + tid;
    const uint32_t n = i < ntiles ? s_n[i] : 0u;
    const uint32_t t = n ? order[i] : 0u;
    // exclusive prefix of n over the workgroup
    uint32_t inc = n;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)inc, d, 64);
      if (l >= d) inc += y;
    }
    if (l == 63) s_wsum[w] = inc;
    __syncthreads();
    uint32_t before = 0, total = 0;
#pragma unroll
    for (int v = 0; v < kOrderWaves; ++v) {
      const uint32_t c = s_wsum[v];
      before += v < w ? c : 0u;
      total += c;
    }
    const uint32_t off = s_off + before + inc - n;
    for (uint32_t jj = 0; jj < n && off + jj < cap; ++jj) items[off + jj] = make_uint2(t, jj);
    __syncthreads();
    if (tid == 0) s_off += total;
    __syncthreads();
  }
  if (tid == 0) queue[0] = min(s_off, cap);
  if (tid < kQueues) queue[kQueueStride * tid + 1] = 0;
}

// The backward's schedule in one launch: tiles ordered by `key`, then the
// work items in that order (walk: each tile's largest per-pixel walk).
__global__ __launch_bounds__(kOrderThreads) void bwd_schedule_kernel(
    int ntiles, const uint32_t* __restrict__ key, const uint32_t* __restrict__ walk,
    uint32_t* __restrict__ order, SplitLayout sp, uint2* __restrict__ items, uint32_t cap,
    uint32_t* __restrict__ queue) {
  __shared__ uint8_t s_buf[ABCD_MAX_TILES];  // bucket keys, then items per position
  order_tiles(ntiles, key, order, s_buf);
  // the order is read back by other threads of this workgroup (the barrier
  // at the end of order_tiles also ends its use of s_buf)
  build_items(ntiles, order, walk, sp, items, cap, queue, s_buf);
}

}  // namespace

int32_t launch_bwd_schedule(int ntiles, const uint32_t* key, const uint32_t* walk,
                            uint32_t* order, const SplitLayout& split, void* items, uint32_t cap,
                            uint32_t* queue, hipStream_t stream) {
  ABCD_LAUNCH("bwd_order", bwd_schedule_kernel, 1, kOrderThreads, 0, stream, ntiles, key, walk,
              order, split, reinterpret_cast<uint2*>(items), cap, queue);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_tile_order(int ntiles, const uint32_t* work, uint32_t* order, const uint32_t* skip,
                          const char* name, hipStream_t stream) {
  if (ntiles <= 0) return ABCD_OK;
  ABCD_LAUNCH(name, tile_order_kernel, 1, kOrderThreads, 0, stream, ntiles, work, order, skip);
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

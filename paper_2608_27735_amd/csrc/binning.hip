// binning.hip -- per-tile, depth-ordered lists of the active Gaussians.
//
// The 3DGS renderer the paper builds on (Introduction) blends, per 16x16 tile,
// the Gaussians whose support rectangle covers the tile, front to back. The
// required order is key = tile << 32 | fp32 depth bits, ties by Gaussian
// index. Instead of sorting M (tile, depth) keys (M ~ 10^8 at the 1M-Gaussian
// block), this file sorts the n Gaussians once by depth (stable LSD radix
// sort, 8-bit digits) and then performs ONE stable counting sort by tile,
// generated directly from the support rectangles in depth order:
//
//   1. depth_keys       key = depth bits (culled -> 0xffffffff), value = index
//   2. radix passes     hist / scan / scatter, 4 x 8 bits, stable
//   3. bin_count        per chunk of consecutive depth ranks, per tile count
//                       (LDS histogram of every rectangle cell)
//   4. bin_scan_columns exclusive prefix of the chunk counts down each tile
//   5. bin_scan_tiles   exclusive prefix over tiles -> tile_ranges, M
//   6. bin_scatter      each wave walks its ranks IN ORDER, its lanes covering
//                       the cells of one rectangle (distinct tiles), so the
//                       position of every pair is its stable rank: the result
//                       is the unique sorted list, with no key array.
//
// HBM traffic is O(n) for the sort and ~4 bytes per intersection for the
// scatter (8 more if the keys are requested), against ~150 bytes per
// intersection for a six-pass LSD sort of 64-bit keys.
#include <algorithm>

#include "abcd_internal.h"

namespace abcd {
namespace {

constexpr int kRsItems = 16;
constexpr int kRsTile = kBlock * kRsItems;  // keys per radix block
constexpr int kScanThreads = 1024;
constexpr int kRanksPerWave = 256;

struct WsHeader {
  unsigned long long m;  // number of intersections
  uint32_t overflow;     // m exceeded the capacity
  uint32_t pad[61];
};
static_assert(sizeof(WsHeader) == 256, "header is one 256-byte slot");

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

inline int chunk_waves_for(int ntiles) {
  return std::min(4, std::max(1, 32768 / std::max(ntiles, 1)));
}

struct WsLayout {
  size_t hdr, keys_a, keys_b, vals_a, vals_b, hist, totals, counts, tile_total, tile_off, total;
  int64_t rs_blocks, chunks;
  int chunk_ranks, chunk_waves;
};

WsLayout ws_layout(int64_t n, int ntiles) {
  WsLayout L;
  L.rs_blocks = (n + kRsTile - 1) / kRsTile;
  L.chunk_waves = chunk_waves_for(ntiles);
  L.chunk_ranks = kRanksPerWave * L.chunk_waves;
  L.chunks = (n + L.chunk_ranks - 1) / L.chunk_ranks;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align256(bytes);
    return at;
  };
  L.hdr = take(sizeof(WsHeader));
  L.keys_a = take(sizeof(uint32_t) * n);
  L.keys_b = take(sizeof(uint32_t) * n);
  L.vals_a = take(sizeof(uint32_t) * n);
  L.vals_b = take(sizeof(uint32_t) * n);
  L.hist = take(sizeof(uint32_t) * 256 * L.rs_blocks);
  L.totals = take(sizeof(uint32_t) * 256);
  L.counts = take(sizeof(uint32_t) * (size_t)L.chunks * ntiles);
  L.tile_total = take(sizeof(uint32_t) * ntiles);
  L.tile_off = take(sizeof(uint32_t) * ntiles);
  L.total = off;
  return L;
}

// Lanes of the calling wave whose 8-bit digit equals this lane's (among the
// lanes in `active`).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, uint64_t active) {
  uint64_t peers = active;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return peers;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  return (1ull << __lane_id()) - 1ull;
}

// ---------------------------------------------------------- depth sort

__global__ __launch_bounds__(256) void depth_keys_kernel(int64_t n, const float* __restrict__ depth,
                                                         const uint32_t* __restrict__ tiles,
                                                         uint32_t* __restrict__ keys,
                                                         uint32_t* __restrict__ vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  keys[i] = tiles[i] ? __float_as_uint(depth[i]) : 0xffffffffu;
  vals[i] = (uint32_t)i;
}

__global__ __launch_bounds__(256) void radix_hist_kernel(const uint32_t* __restrict__ keys, int64_t n,
                                                         int shift, uint32_t* __restrict__ hist,
                                                         int64_t nblocks) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
#pragma unroll 4
  for (int it = 0; it < kRsItems; ++it) {
    const int64_t idx = base + it * kBlock + threadIdx.x;
    if (idx < n) {
      const uint32_t d = (keys[idx] >> shift) & 255u;
      const uint64_t peers = match_digit(d, __ballot(1));
      if (__lane_id() == __ffsll((unsigned long long)peers) - 1) atomicAdd(&h[d], (uint32_t)__popcll(peers));
    }
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblocks + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan of each digit's row of block counts in place (one
// workgroup per digit) and the digit totals.
__global__ __launch_bounds__(256) void radix_scan_rows_kernel(uint32_t* __restrict__ hist,
                                                              int64_t nblocks,
                                                              uint32_t* __restrict__ totals) {
  __shared__ uint32_t part[256];
  uint32_t* row = hist + (int64_t)blockIdx.x * nblocks;
  uint32_t carry = 0;
  for (int64_t b0 = 0; b0 < nblocks; b0 += 256) {
    const int64_t b = b0 + threadIdx.x;
    const uint32_t v = b < nblocks ? row[b] : 0u;
    part[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const uint32_t x = threadIdx.x >= off ? part[threadIdx.x - off] : 0u;
      __syncthreads();
      part[threadIdx.x] += x;
      __syncthreads();
    }
    if (b < nblocks) row[b] = carry + part[threadIdx.x] - v;
    carry += part[255];
    __syncthreads();
  }
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

__global__ __launch_bounds__(256) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in, int64_t n, int shift,
    const uint32_t* __restrict__ hist, int64_t nblocks, const uint32_t* __restrict__ totals,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out) {
  __shared__ uint32_t sbase[256];
  __shared__ uint32_t wcnt[4][256];
  const int tid = threadIdx.x, w = tid >> 6;
  // digit base = exclusive scan of the digit totals
  const uint32_t tot = totals[tid];
  sbase[tid] = tot;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const uint32_t x = tid >= off ? sbase[tid - off] : 0u;
    __syncthreads();
    sbase[tid] += x;
    __syncthreads();
  }
  sbase[tid] += hist[(int64_t)tid * nblocks + blockIdx.x] - tot;
#pragma unroll
  for (int k = 0; k < 4; ++k) wcnt[k][tid] = 0;
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
  uint32_t key[kRsItems], val[kRsItems];
#pragma unroll
  for (int it = 0; it < kRsItems; ++it) {
    const int64_t idx = base + it * kBlock + tid;
    key[it] = idx < n ? keys_in[idx] : 0u;
    val[it] = idx < n ? vals_in[idx] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kRsItems; ++it) {
    const int64_t idx = base + it * kBlock + tid;
    const bool valid = idx < n;
    const uint32_t d = (key[it] >> shift) & 255u;
    uint32_t rank = 0;
    if (valid) {
      const uint64_t peers = match_digit(d, __ballot(1));
      rank = __popcll(peers & lanemask_lt());
      if (__lane_id() == __ffsll((unsigned long long)peers) - 1) wcnt[w][d] = __popcll(peers);
    }
    __syncthreads();
    if (valid) {
      uint32_t pos = sbase[d] + rank;
      for (int k = 0; k < w; ++k) pos += wcnt[k][d];
      keys_out[pos] = key[it];
      vals_out[pos] = val[it];
    }
    __syncthreads();
    sbase[tid] += wcnt[0][tid] + wcnt[1][tid] + wcnt[2][tid] + wcnt[3][tid];
#pragma unroll
    for (int k = 0; k < 4; ++k) wcnt[k][tid] = 0;
    __syncthreads();
  }
}

// ------------------------------------------------- tile counting sort

struct Rect {
  int x0, y0, x1, y1;
  bool ok;
};

__device__ __forceinline__ Rect rect_of(uint32_t g, const float* __restrict__ means2d,
                                        const float* __restrict__ radius,
                                        const uint32_t* __restrict__ tiles, int ntx, int nty) {
  Rect r;
  r.ok = tiles[g] != 0;
  if (r.ok) {
    const float2 m = reinterpret_cast<const float2*>(means2d)[g];
    r.ok = tile_rect(m.x, m.y, radius[g], ntx, nty, r.x0, r.y0, r.x1, r.y1);
  }
  if (!r.ok) r.x0 = r.y0 = 0, r.x1 = r.y1 = -1;
  return r;
}

// cell -> (cx, cy) of a rectangle of width wr, row major; exact for cell < 2^22
__device__ __forceinline__ void cell_xy(int cell, int wr, float inv_wr, int& cx, int& cy) {
  int q = (int)((float)cell * inv_wr);
  if (q * wr > cell) --q;
  if ((q + 1) * wr <= cell) ++q;
  cy = q;
  cx = cell - q * wr;
}

__global__ __launch_bounds__(256) void bin_count_kernel(
    int64_t n, const uint32_t* __restrict__ order, const float* __restrict__ means2d,
    const float* __restrict__ radius, const uint32_t* __restrict__ tiles, int ntx, int nty,
    int chunk_ranks, uint32_t* __restrict__ counts) {
  extern __shared__ uint32_t cnt[];
  const int ntiles = ntx * nty;
  for (int t = threadIdx.x; t < ntiles; t += blockDim.x) cnt[t] = 0;
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * chunk_ranks;
  const int64_t r1 = std::min<int64_t>(n, r0 + chunk_ranks);
  for (int64_t r = r0 + threadIdx.x; r < r1; r += blockDim.x) {
    const Rect rc = rect_of(order[r], means2d, radius, tiles, ntx, nty);
    for (int y = rc.y0; y <= rc.y1; ++y)
      for (int x = rc.x0; x <= rc.x1; ++x) atomicAdd(&cnt[y * ntx + x], 1u);
  }
  __syncthreads();
  uint32_t* out = counts + (int64_t)blockIdx.x * ntiles;
  for (int t = threadIdx.x; t < ntiles; t += blockDim.x) out[t] = cnt[t];
}

// counts[chunk][tile] -> exclusive prefix down each tile column; column
// totals -> tile_total. Lane = tile, the 16 waves split the chunks.
__global__ __launch_bounds__(1024) void bin_scan_columns_kernel(uint32_t* __restrict__ counts,
                                                                int64_t chunks, int ntiles,
                                                                uint32_t* __restrict__ tile_total) {
  __shared__ uint32_t part[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int t = blockIdx.x * 64 + lane;
  const int64_t per = (chunks + 15) / 16;
  const int64_t c0 = std::min<int64_t>(chunks, per * w), c1 = std::min<int64_t>(chunks, c0 + per);
  uint32_t s = 0;
  if (t < ntiles)
    for (int64_t c = c0; c < c1; ++c) s += counts[c * ntiles + t];
  part[w][lane] = s;
  __syncthreads();
  uint32_t run = 0;
  for (int k = 0; k < w; ++k) run += part[k][lane];
  if (t < ntiles) {
    for (int64_t c = c0; c < c1; ++c) {
      const uint32_t v = counts[c * ntiles + t];
      counts[c * ntiles + t] = run;
      run += v;
    }
    if (w == 15) tile_total[t] = run;
  }
}

// Exclusive scan over tiles -> tile_off, tile_ranges, M; one workgroup.
__global__ __launch_bounds__(kScanThreads) void bin_scan_tiles_kernel(
    const uint32_t* __restrict__ tile_total, int ntiles, uint32_t* __restrict__ tile_off,
    uint32_t* __restrict__ tile_ranges, WsHeader* __restrict__ hdr, unsigned long long capacity) {
  __shared__ unsigned long long part[kScanThreads];
  const int per = (ntiles + kScanThreads - 1) / kScanThreads;
  const int lo = std::min(ntiles, per * (int)threadIdx.x), hi = std::min(ntiles, lo + per);
  unsigned long long s = 0;
  for (int i = lo; i < hi; ++i) s += tile_total[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = 1; off < kScanThreads; off <<= 1) {
    const unsigned long long v = threadIdx.x >= off ? part[threadIdx.x - off] : 0ull;
    __syncthreads();
    part[threadIdx.x] += v;
    __syncthreads();
  }
  const unsigned long long m = part[kScanThreads - 1];
  const bool fits = m <= capacity && m < (1ull << 32);
  unsigned long long run = part[threadIdx.x] - s;
  for (int i = lo; i < hi; ++i) {
    const uint32_t v = tile_total[i];
    tile_off[i] = (uint32_t)run;
    if (fits) {
      tile_ranges[2 * i] = (uint32_t)run;
      tile_ranges[2 * i + 1] = (uint32_t)(run + v);
    }
    run += v;
  }
  if (threadIdx.x == 0) {
    hdr->m = m;
    hdr->overflow = fits ? 0u : 1u;
  }
}

// Stable scatter of every (tile, Gaussian) pair of one chunk of depth ranks.
// Block = chunk_waves waves, wave w owns ranks [w * 256, w * 256 + 256) of the
// chunk. LDS holds, per wave and tile, the next free slot.
__global__ __launch_bounds__(256) void bin_scatter_kernel(
    int64_t n, const uint32_t* __restrict__ order, const float* __restrict__ means2d,
    const float* __restrict__ radius, const uint32_t* __restrict__ tiles,
    const float* __restrict__ depth, int ntx, int nty, int chunk_ranks,
    const uint32_t* __restrict__ counts, const uint32_t* __restrict__ tile_off,
    const WsHeader* __restrict__ hdr, uint32_t* __restrict__ values_sorted,
    unsigned long long* __restrict__ keys_sorted) {
  extern __shared__ uint32_t slot[];  // [waves][ntiles]
  if (hdr->overflow) return;
  const int ntiles = ntx * nty;
  const int nw = blockDim.x >> 6, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t rbase = (int64_t)blockIdx.x * chunk_ranks + (int64_t)w * kRanksPerWave;
  uint32_t* my = slot + (int64_t)w * ntiles;
  for (int t = threadIdx.x; t < nw * ntiles; t += blockDim.x) slot[t] = 0;
  __syncthreads();
  // this lane's 4 ranks: rbase + lane + 64 j
  uint32_t gj[4];
  Rect rj[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t r = rbase + lane + 64 * j;
    gj[j] = r < n ? order[r] : 0u;
    rj[j] = r < n ? rect_of(gj[j], means2d, radius, tiles, ntx, nty) : Rect{0, 0, -1, -1, false};
    for (int y = rj[j].y0; y <= rj[j].y1; ++y)
      for (int x = rj[j].x0; x <= rj[j].x1; ++x) atomicAdd(&my[y * ntx + x], 1u);
  }
  __syncthreads();
  // per-wave counts -> first free slot of each wave
  const uint32_t* crow = counts + (int64_t)blockIdx.x * ntiles;
  for (int t = threadIdx.x; t < ntiles; t += blockDim.x) {
    uint32_t run = tile_off[t] + crow[t];
    for (int k = 0; k < nw; ++k) {
      const uint32_t c = slot[k * ntiles + t];
      slot[k * ntiles + t] = run;
      run += c;
    }
  }
  __syncthreads();
  // in rank order: lanes spread over the cells of one rectangle (distinct tiles)
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll 1
    for (int l = 0; l < 64; ++l) {
      const int x0 = __builtin_amdgcn_readlane(rj[j].x0, l);
      const int y0 = __builtin_amdgcn_readlane(rj[j].y0, l);
      const int x1 = __builtin_amdgcn_readlane(rj[j].x1, l);
      const int y1 = __builtin_amdgcn_readlane(rj[j].y1, l);
      if (x1 < x0) continue;
      const uint32_t g = (uint32_t)__builtin_amdgcn_readlane((int)gj[j], l);
      const int wr = x1 - x0 + 1;
      const int area = wr * (y1 - y0 + 1);
      const float inv_wr = 1.0f / (float)wr;
      const unsigned long long dkey = keys_sorted ? (unsigned long long)__float_as_uint(depth[g]) : 0ull;
      for (int cell = lane; cell < area; cell += 64) {
        int cx, cy;
        cell_xy(cell, wr, inv_wr, cx, cy);
        const int t = (y0 + cy) * ntx + (x0 + cx);
        const uint32_t pos = my[t];
        my[t] = pos + 1;
        values_sorted[pos] = g;
        if (keys_sorted) keys_sorted[pos] = ((unsigned long long)t << 32) | dkey;
      }
    }
  }
}

__global__ void bin_empty_kernel(int ntiles, uint32_t* __restrict__ tile_ranges,
                                 WsHeader* __restrict__ hdr) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < 2 * ntiles; i += gridDim.x * blockDim.x)
    tile_ranges[i] = 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    hdr->m = 0;
    hdr->overflow = 0;
  }
}

int32_t set_max_lds(const void* fn, size_t bytes) {
  ABCD_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
  return ABCD_OK;
}

}  // namespace

size_t bin_sort_workspace_bytes(int64_t n, int ntiles) { return ws_layout(n, ntiles).total; }

int32_t launch_bin_sort(int width, int height, int64_t n, const float* means2d, const float* radius,
                        const float* depth, const uint32_t* tiles_touched, int64_t capacity,
                        void* workspace, uint64_t* keys_sorted, uint32_t* values_sorted,
                        uint32_t* tile_ranges, hipStream_t stream) {
  const int ntx = tiles_x(width), nty = tiles_y(height), ntiles = ntx * nty;
  const WsLayout L = ws_layout(n, ntiles);
  char* ws = static_cast<char*>(workspace);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  if (n == 0) {
    ABCD_LAUNCH("bin_scan_tiles", bin_empty_kernel, std::max(1, (2 * ntiles + 255) / 256), 256, 0,
                stream, ntiles, tile_ranges, hdr);
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  uint32_t* keys[2] = {reinterpret_cast<uint32_t*>(ws + L.keys_a), reinterpret_cast<uint32_t*>(ws + L.keys_b)};
  uint32_t* vals[2] = {reinterpret_cast<uint32_t*>(ws + L.vals_a), reinterpret_cast<uint32_t*>(ws + L.vals_b)};
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.hist);
  uint32_t* totals = reinterpret_cast<uint32_t*>(ws + L.totals);
  uint32_t* counts = reinterpret_cast<uint32_t*>(ws + L.counts);
  uint32_t* tile_total = reinterpret_cast<uint32_t*>(ws + L.tile_total);
  uint32_t* tile_off = reinterpret_cast<uint32_t*>(ws + L.tile_off);

  const int64_t gb = (n + kBlock - 1) / kBlock;
  ABCD_LAUNCH("depth_keys", depth_keys_kernel, gb, kBlock, 0, stream, n, depth, tiles_touched,
              keys[0], vals[0]);
  for (int pass = 0; pass < 4; ++pass) {
    const int src = pass & 1, dst = src ^ 1;
    ABCD_LAUNCH("radix_hist", radix_hist_kernel, L.rs_blocks, kBlock, 0, stream, keys[src], n,
                8 * pass, hist, L.rs_blocks);
    ABCD_LAUNCH("radix_scan", radix_scan_rows_kernel, 256, kBlock, 0, stream, hist, L.rs_blocks,
                totals);
    ABCD_LAUNCH("radix_scatter", radix_scatter_kernel, L.rs_blocks, kBlock, 0, stream, keys[src],
                vals[src], n, 8 * pass, hist, L.rs_blocks, totals, keys[dst], vals[dst]);
  }
  const uint32_t* order = vals[0];  // four passes: back in buffer 0

  const size_t count_lds = sizeof(uint32_t) * ntiles;
  const size_t scatter_lds = sizeof(uint32_t) * ntiles * L.chunk_waves;
  static bool attrs_set = false;
  if (!attrs_set) {
    int32_t st = set_max_lds((const void*)bin_count_kernel, sizeof(uint32_t) * 32768);
    if (st != ABCD_OK) return st;
    st = set_max_lds((const void*)bin_scatter_kernel, sizeof(uint32_t) * 32768);
    if (st != ABCD_OK) return st;
    attrs_set = true;
  }
  ABCD_LAUNCH("bin_count", bin_count_kernel, L.chunks, kBlock, count_lds, stream, n, order, means2d,
              radius, tiles_touched, ntx, nty, L.chunk_ranks, counts);
  ABCD_LAUNCH("bin_scan_columns", bin_scan_columns_kernel, (ntiles + 63) / 64, 1024, 0, stream,
              counts, L.chunks, ntiles, tile_total);
  ABCD_LAUNCH("bin_scan_tiles", bin_scan_tiles_kernel, 1, kScanThreads, 0, stream, tile_total,
              ntiles, tile_off, tile_ranges, hdr,
              (unsigned long long)std::max<int64_t>(capacity, 0));
  ABCD_LAUNCH("bin_scatter", bin_scatter_kernel, L.chunks, 64 * L.chunk_waves, scatter_lds, stream,
              n, order, means2d, radius, tiles_touched, depth, ntx, nty, L.chunk_ranks, counts,
              tile_off, hdr, values_sorted, reinterpret_cast<unsigned long long*>(keys_sorted));
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd

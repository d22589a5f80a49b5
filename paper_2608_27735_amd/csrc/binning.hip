// binning.hip -- per-tile, depth-ordered lists of the active Gaussians.
//
// The 3DGS renderer the paper builds on (Introduction) blends, per 16x16 tile,
// the Gaussians whose support rectangle covers the tile, front to back. The
// required order is key = tile << 32 | fp32 depth bits, ties by Gaussian
// index. Instead of sorting the M (tile, depth) keys (M ~ 10^8 at a 1M-Gaussian
// block), the n Gaussians are sorted once by depth (stable LSD radix sort,
// 8-bit digits) and the lists are then GENERATED in depth order by two stable
// counting sorts driven by the support rectangles:
//
//   level 1  Gaussians -> buckets of 8x8-tile blocks (a few per Gaussian)
//   level 2  each block's bucket -> its 64 tile lists
//
// Both levels place every pair at its stable rank. Level 1: a wave visits the
// distinct blocks its entries cover in increasing block order, and ballots
// rank the entries covering each block. Level 2: ballots give each of a
// block's 64 tiles the mask of a wave's entries covering it, and the entries
// of each mask store at their rank in it. Counts come from LDS atomics
// (level 1) and 2D difference arrays (level 2). Level 2 is
// split into sub-chunks of a bucket, each of which writes only 64 output
// streams, so consecutive writes of a stream meet in L2 and leave it as whole
// lines (a one-level scatter over all tiles of the frame writes every 4-byte
// entry into a different line and pays several times the payload in HBM
// writes).
//
//   bin_zero               header, counters and look-back states
//   depth_keys             keys, tile rectangles, digit counts, block totals,
//                          intersection count M
//   radix_pass x4          depth order of the n Gaussians
//   l1_place               (block, Gaussian) pairs, bucket-major, depth order;
//                          bucket offsets, sub-chunk and slice tables,
//                          overflow flag (on overflow nothing is placed: every
//                          tile range comes out empty)
//   l2_count               per slice of 16 sub-chunks: counts of its block's
//                          64 tiles per sub-chunk; per block (its last slice
//                          counted): the slices' prefix and the tile totals;
//                          last: tile_ranges
//   l2_scatter             values (and keys), tile-major, depth order; its
//                          first workgroup: the forward's tile order
#include <algorithm>

#include "schedule.h"

namespace abcd {
namespace {

constexpr int kDkItems = 4;                 // Gaussians per thread of depth_keys
constexpr int kDkTile = kBlock * kDkItems;
constexpr int kRsItems = 16;                // keys per thread of a radix pass
constexpr int kRsTile = kBlock * kRsItems;  // keys per radix partition
constexpr int kRsLook = 8;                  // partition states read at once looking back
// depth_keys adds the digit counts, block totals and intersection count of
// workgroup b into copy b mod kHistCopies, so that no counter takes more
// than a few dozen atomic adds; their readers sum the copies
constexpr int kHistCopies = 32;
constexpr int kScanThreads = 1024;
constexpr int kL1Items = 4;                 // level 1: depth ranks per lane
constexpr int kRanksPerWave = 64 * kL1Items;
constexpr int kChunk = 4 * kRanksPerWave;   // level 1: depth ranks per workgroup
constexpr int kSub = 256;                   // level 2: bucket entries per sub-chunk
constexpr int kSlice = 16;                  // level 2: sub-chunks per slice (a wave each)
constexpr int kBlk = 8;                     // block side in tiles
constexpr int kBlkTiles = kBlk * kBlk;
constexpr int kCountGrid = 512;             // workgroups of the grid-stride level-2 count
constexpr int kScatterGrid = 8192;          // workgroups of the grid-stride level-2 scatter

struct WsHeader {
  unsigned long long m;   // intersections (sum of tiles_touched)
  unsigned long long m1;  // (Gaussian, block) pairs
  uint32_t overflow;      // m > capacity or m >= 2^32: nothing is written
  uint32_t total_sub;     // level-2 sub-chunks
  uint32_t ticket[4];     // partitions taken by each radix pass
  uint32_t ticket_l1;     // chunks taken by l1_place
  uint32_t done_l2;       // blocks whose level-2 scan is done
  uint32_t nonempty;      // blocks holding at least one entry
  uint32_t pad[51];
};
static_assert(sizeof(WsHeader) == 256, "header is one 256-byte slot");

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Geo {
  int ntx, nty, nbx, nby, nblk;
};

inline Geo geo_of(int width, int height) {
  Geo g;
  g.ntx = tiles_x(width);
  g.nty = tiles_y(height);
  g.nbx = (g.ntx + kBlk - 1) / kBlk;
  g.nby = (g.nty + kBlk - 1) / kBlk;
  g.nblk = g.nbx * g.nby;
  return g;
}

struct WsLayout {
  size_t hdr, ghist, mcopy, bcopy, blk_done, lb1, st0, st1, keys_a, keys_b, vals_a, vals_b, rects, blk_off,
      sub_off, slice_off, pairs, c2, slice_tot, tile_total, tile_off, total;
  int64_t rs_parts, chunks, max_sub, max_slices;
};

WsLayout ws_layout(int64_t n, int64_t capacity, const Geo& g) {
  WsLayout L;
  const int64_t ntiles = (int64_t)g.ntx * g.nty;
  L.rs_parts = (n + kRsTile - 1) / kRsTile;
  L.chunks = (n + kChunk - 1) / kChunk;
  L.max_sub = (capacity + kSub - 1) / kSub + g.nblk;
  // (group of kSlice sub-chunks, block) pairs: each block start splits at
  // most one group
  L.max_slices = L.max_sub / kSlice + g.nblk + 2;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align256(bytes);
    return at;
  };
  // header, counters, level 1's and the first radix pass's look-back states
  // are one region, cleared by one launch
  L.hdr = take(sizeof(WsHeader));
  L.ghist = take(sizeof(uint32_t) * kHistCopies * 4 * 256);
  L.mcopy = take(sizeof(unsigned long long) * kHistCopies);
  L.bcopy = take(sizeof(uint32_t) * kHistCopies * g.nblk);
  L.blk_done = take(sizeof(uint32_t) * g.nblk);
  L.lb1 = take(sizeof(uint32_t) * (size_t)L.chunks * g.nblk);
  L.st0 = take(sizeof(unsigned long long) * 256 * L.rs_parts);
  L.st1 = take(sizeof(unsigned long long) * 256 * L.rs_parts);
  L.keys_a = take(sizeof(uint32_t) * n);
  L.keys_b = take(sizeof(uint32_t) * n);
  L.vals_a = take(sizeof(uint32_t) * n);
  L.vals_b = take(sizeof(uint32_t) * n);
  L.rects = take(sizeof(unsigned long long) * n);
  L.blk_off = take(sizeof(uint32_t) * (g.nblk + 1));
  L.sub_off = take(sizeof(uint32_t) * (g.nblk + 1));
  L.slice_off = take(sizeof(uint32_t) * (g.nblk + 1));
  L.pairs = take(sizeof(unsigned long long) * (size_t)capacity);  // m1 <= m <= capacity
  L.c2 = take(sizeof(uint32_t) * (size_t)L.max_sub * kBlkTiles);
  L.slice_tot = take(sizeof(uint32_t) * (size_t)L.max_slices * kBlkTiles);
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
//
// Stable LSD radix sort of the n depth keys, 8-bit digits, one launch per
// digit. The counts of every digit value over all keys do not depend on the
// order, so depth_keys takes them for all four digits at once; a pass then
// needs, per partition of kRsTile consecutive keys, the counts of each digit
// in the partitions before it. Each partition publishes its own counts as
// soon as it has them and reads its predecessors' (decoupled look-back):
// a state word per (partition, digit) holds a flag (aggregate: the
// partition's own count; inclusive: the count over it and every partition
// before it) and the count. Partitions take their index from a ticket
// counter in launch order, so every partition a workgroup waits for is
// already running and publishes without waiting itself: every wait ends.
// Keys are ranked and grouped by digit in LDS, then leave as runs of
// consecutive addresses.

constexpr unsigned long long kStAgg = 1ull << 62;   // the partition's own count
constexpr unsigned long long kStIncl = 2ull << 62;  // count over it and all before it

// Tile rectangle packed as x0 | x1 << 16 | y0 << 32 | y1 << 48 (empty: x0 = 1 > x1 = 0).
__device__ __forceinline__ unsigned long long pack_rect(int x0, int y0, int x1, int y1) {
  return (unsigned long long)x0 | ((unsigned long long)x1 << 16) | ((unsigned long long)y0 << 32) |
         ((unsigned long long)y1 << 48);
}

// Clears the header (with the radix passes' tickets), the digit counts and
// the first pass's partition states: one contiguous region of 16-byte words.
__global__ __launch_bounds__(256) void bin_zero_kernel(uint4* __restrict__ p, int64_t words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// Adds this wave's keys to the workgroup's counts h[4][256] of each digit
// value. A digit that every active lane shares (the high digits of nearby
// depths, the 0xff of off-screen Gaussians) is added once by the first lane.
__device__ __forceinline__ void count_digits(uint32_t (*h)[256], uint32_t key, bool valid) {
  const uint64_t act = __ballot(valid);
  if (!act) return;
  const int first = __ffsll((unsigned long long)act) - 1;
  const int lane = __lane_id();
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t d = (key >> (8 * b)) & 255u;
    const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)d, first);
    if (__ballot(valid && d == d0) == act) {
      if (lane == first) atomicAdd(&h[b][d0], (uint32_t)__popcll(act));
    } else if (valid) {
      atomicAdd(&h[b][d], 1u);
    }
  }
}

// Depth keys (fp32 bits; a Gaussian with no tile gets 0xffffffff and sorts
// last), packed tile rectangles, and, added into copy blockIdx mod
// kHistCopies (cleared before the launch): the counts of each value of each
// of the four key digits (ghist[copy][digit][value]), the Gaussians covering
// each 8x8-tile block (bcopy[copy][block]; s_blk: 4 x geo.nblk words of
// dynamic LDS, one row per wave so that waves do not contend) and the
// intersection count (mcopy[copy]).
__global__ __launch_bounds__(256) void depth_keys_kernel(
    int64_t n, const float* __restrict__ depth, const uint32_t* __restrict__ tiles,
    const float* __restrict__ means2d, const float* __restrict__ extent, Geo geo,
    uint32_t* __restrict__ keys, unsigned long long* __restrict__ rects,
    uint32_t* __restrict__ ghist, uint32_t* __restrict__ bcopy,
    unsigned long long* __restrict__ mcopy) {
  extern __shared__ uint32_t s_blk[];
  __shared__ uint32_t h[4][256];
  __shared__ unsigned long long s_m;
  const int tid = threadIdx.x;
#pragma unroll
  for (int b = 0; b < 4; ++b) h[b][tid] = 0;
  for (int b = tid; b < 4 * geo.nblk; b += kBlock) s_blk[b] = 0;
  if (tid == 0) s_m = 0;
  uint32_t* wblk = s_blk + (tid >> 6) * geo.nblk;
  const int64_t base = (int64_t)blockIdx.x * kDkTile;
  // every load of the thread's Gaussians in flight at once
  uint32_t tt[kDkItems];
  float dp[kDkItems];
  float2 mm[kDkItems], ee[kDkItems];
#pragma unroll
  for (int it = 0; it < kDkItems; ++it) {
    const int64_t i = base + it * kBlock + tid;
    const bool ok = i < n;
    tt[it] = ok ? tiles[i] : 0u;
    dp[it] = ok ? depth[i] : 0.0f;
    mm[it] = ok ? reinterpret_cast<const float2*>(means2d)[i] : make_float2(0.0f, 0.0f);
    ee[it] = ok ? reinterpret_cast<const float2*>(extent)[i] : make_float2(0.0f, 0.0f);
  }
  __syncthreads();
  uint32_t m = 0;  // at most kDkItems x 32768 tiles
#pragma unroll
  for (int it = 0; it < kDkItems; ++it) {
    const int64_t i = base + it * kBlock + tid;
    const bool ok = i < n;
    const bool vis = ok && tt[it] != 0;
    const uint32_t key = vis ? __float_as_uint(dp[it]) : 0xffffffffu;
    int x0 = 1, y0 = 0, x1 = 0, y1 = 0;
    const bool hit = vis && tile_rect(mm[it].x, mm[it].y, ee[it].x, ee[it].y, geo.ntx, geo.nty, x0,
                                      y0, x1, y1);
    if (!hit) x0 = 1, y0 = 0, x1 = 0, y1 = 0;
    if (ok) {
      keys[i] = key;
      rects[i] = pack_rect(x0, y0, x1, y1);
    }
    if (hit) {
      m += (uint32_t)((x1 - x0 + 1) * (y1 - y0 + 1));
      for (int by = y0 / kBlk; by <= y1 / kBlk; ++by)
        for (int bx = x0 / kBlk; bx <= x1 / kBlk; ++bx) atomicAdd(&wblk[by * geo.nbx + bx], 1u);
    }
    count_digits(h, key, ok);
  }
  const uint32_t wm = wave_sum_u32(m);
  if ((tid & 63) == 0 && wm) atomicAdd(&s_m, (unsigned long long)wm);
  __syncthreads();
  const int copy = (int)(blockIdx.x % kHistCopies);
  uint32_t* gh = ghist + copy * (4 * 256);
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t v = h[b][tid];
    if (v) atomicAdd(&gh[b * 256 + tid], v);
  }
  uint32_t* bc = bcopy + (size_t)copy * geo.nblk;
  for (int b = tid; b < geo.nblk; b += kBlock) {
    const uint32_t v = s_blk[b] + s_blk[geo.nblk + b] + s_blk[2 * geo.nblk + b] +
                       s_blk[3 * geo.nblk + b];
    if (v) atomicAdd(&bc[b], v);
  }
  if (tid == 0 && s_m) atomicAdd(&mcopy[copy], s_m);
}

// Exclusive prefix of one value per thread over the 256 threads; s4 is four
// words of LDS.
__device__ __forceinline__ uint32_t scan_256(uint32_t v, uint32_t* s4) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  uint32_t incl = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) s4[w] = incl;
  __syncthreads();
  uint32_t before = 0;
#pragma unroll
  for (int k = 0; k < 3; ++k) before += k < w ? s4[k] : 0u;
  __syncthreads();
  return before + incl - v;
}

// Look-back state words: the two top bits flag the count below them as the
// part's own (aggregate) or as the sum over it and every part before it
// (inclusive); 0 is not yet published.
template <typename W>
struct StateWord {
  static constexpr int kShift = 8 * (int)sizeof(W) - 2;
  static constexpr W kAgg = (W)1 << kShift;
  static constexpr W kIncl = (W)2 << kShift;
};

// Sum of the counts of item `idx` in the parts before `part` (part > 0; part
// q's word at st[q * stride + idx]), read back kRsLook parts at a time:
// aggregates are added until an inclusive count ends the walk; a word not yet
// published is read again (its part is running and publishes without
// waiting).
template <typename W>
__device__ __forceinline__ uint32_t look_back(const W* __restrict__ st, int64_t part,
                                              int64_t stride, int64_t idx) {
  using SW = StateWord<W>;
  uint32_t excl = 0;
  int64_t q = part - 1;
  while (true) {
    W s[kRsLook];
#pragma unroll
    for (int j = 0; j < kRsLook; ++j)
      s[j] = q - j >= 0 ? __hip_atomic_load(&st[(q - j) * stride + idx], __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT)
                        : SW::kIncl;
    int used = 0;
    bool open = true, found = false;
#pragma unroll
    for (int j = 0; j < kRsLook; ++j) {
      const W f = s[j] & ((W)3 << SW::kShift);
      if (open && f != 0) {
        excl += (uint32_t)(s[j] & (SW::kAgg - 1));
        ++used;
        if (f == SW::kIncl) found = true;
      }
      open = open && f == SW::kAgg;
    }
    if (found) return excl;
    if (used == 0) __builtin_amdgcn_s_sleep(1);
    q -= used;
  }
}

// One stable pass on digit `pass` (bits 8 pass .. 8 pass + 7) of partition
// `part` (from the ticket). Wave w ranks its consecutive quarter of the
// partition in order: the lanes holding one digit value find each other by
// ballots, and the first of them adds their number to the wave's running
// count of that value (an LDS atomic returning the count before it; a wave's
// atomics execute in program order, so the items are ranked in input order
// without waiting on each other). The partition's keys are then regrouped
// in LDS by digit (wave-major within a digit, which keeps the input order)
// and written out, each at the digit's global base + its place among the
// digit's keys of earlier partitions + its place in the partition. vals_in
// NULL: the values are the keys' input positions. st_next (NULL on the last
// pass): the next pass's states, whose row of this partition is cleared here.
__global__ __launch_bounds__(256) void radix_pass_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in, int64_t n, int pass,
    const uint32_t* __restrict__ ghist, unsigned long long* __restrict__ st,
    unsigned long long* __restrict__ st_next, uint32_t* __restrict__ ticket,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out) {
  constexpr int kPerWave = kRsTile / 4;
  constexpr int kWaveItems = kPerWave / 64;
  __shared__ uint32_t s_key[kRsTile];
  __shared__ uint32_t s_val[kRsTile];
  __shared__ uint32_t wcnt[4][256];  // per wave and digit: running counts, then first slots
  __shared__ uint32_t s_dst[256];    // per digit: global position of LDS slot 0
  __shared__ uint32_t s4[4];
  __shared__ uint32_t s_part;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int shift = 8 * pass;
  if (tid == 0) s_part = atomicAdd(ticket, 1u);
#pragma unroll
  for (int k = 0; k < 4; ++k) wcnt[k][tid] = 0;
  // global base of digit value tid: counts of the smaller values over all
  // keys (while the ticket is on its way)
  uint32_t total = 0;
  {
    uint32_t c[kHistCopies];
#pragma unroll
    for (int r = 0; r < kHistCopies; ++r) c[r] = ghist[(r * 4 + pass) * 256 + tid];
#pragma unroll
    for (int r = 0; r < kHistCopies; ++r) total += c[r];
  }
  const uint32_t gbase = scan_256(total, s4);  // its barriers publish s_part and the zeroed counts
  const int64_t part = s_part;
  const int64_t base = part * kRsTile;
  const int cnt = (int)min<int64_t>(kRsTile, n - base);
  uint32_t key[kWaveItems], val[kWaveItems], rank[kWaveItems];
#pragma unroll
  for (int it = 0; it < kWaveItems; ++it) {
    const int li = w * kPerWave + it * 64 + lane;
    const bool ok = li < cnt;
    key[it] = ok ? keys_in[base + li] : 0u;
    val[it] = ok ? (vals_in ? vals_in[base + li] : (uint32_t)(base + li)) : 0u;
  }
  if (st_next) st_next[part * 256 + tid] = 0ull;
  const uint64_t lt = lanemask_lt();
  // kRankGroup items at a time: their atomics are in flight together
  constexpr int kRankGroup = 4;
#pragma unroll
  for (int g = 0; g < kWaveItems; g += kRankGroup) {
    uint32_t before[kRankGroup];
    int first[kRankGroup];
#pragma unroll
    for (int u = 0; u < kRankGroup; ++u) {
      const int it = g + u;
      const bool ok = w * kPerWave + it * 64 + lane < cnt;
      const uint32_t d = (key[it] >> shift) & 255u;
      const uint64_t peers = match_digit(d, __ballot(ok));
      first[u] = __ffsll((unsigned long long)peers) - 1;
      rank[it] = __popcll(peers & lt);
      before[u] = 0;
      if (ok && lane == first[u]) before[u] = atomicAdd(&wcnt[w][d], (uint32_t)__popcll(peers));
    }
#pragma unroll
    for (int u = 0; u < kRankGroup; ++u)
      rank[g + u] += (uint32_t)__shfl((int)before[u], first[u] < 0 ? 0 : first[u], 64);
  }
  __syncthreads();
  // thread tid = digit value: publish the partition's count, then turn the
  // per-wave counts into LDS slots
  const uint32_t c0 = wcnt[0][tid], c1 = wcnt[1][tid], c2 = wcnt[2][tid], c3 = wcnt[3][tid];
  const uint32_t own = c0 + c1 + c2 + c3;
  __hip_atomic_store(&st[part * 256 + tid], (part == 0 ? kStIncl : kStAgg) | own, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t loc = scan_256(own, s4);
  wcnt[0][tid] = loc;
  wcnt[1][tid] = loc + c0;
  wcnt[2][tid] = loc + c0 + c1;
  wcnt[3][tid] = loc + c0 + c1 + c2;
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kWaveItems; ++it) {
    if (w * kPerWave + it * 64 + lane < cnt) {
      const uint32_t slot = wcnt[w][(key[it] >> shift) & 255u] + rank[it];
      s_key[slot] = key[it];
      s_val[slot] = val[it];
    }
  }
  uint32_t excl = 0;
  if (part > 0) {
    excl = look_back(st, part, 256, tid);
    __hip_atomic_store(&st[part * 256 + tid], kStIncl | (excl + own), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
  s_dst[tid] = gbase + excl - loc;
  __syncthreads();
  for (int i = tid; i < cnt; i += kBlock) {
    const uint32_t k = s_key[i];
    const uint32_t pos = s_dst[(k >> shift) & 255u] + (uint32_t)i;
    keys_out[pos] = k;
    vals_out[pos] = s_val[i];
  }
}

// ------------------------------------------------------------ rectangles

struct Rect {
  int x0, y0, x1, y1;  // inclusive tile rectangle; empty if x1 < x0
};

__device__ __forceinline__ Rect rect_of(uint32_t g, const unsigned long long* __restrict__ rects) {
  const unsigned long long p = rects[g];
  return Rect{(int)(p & 0xffff), (int)((p >> 32) & 0xffff), (int)((p >> 16) & 0xffff),
              (int)(p >> 48)};
}

__device__ __forceinline__ Rect block_rect(const Rect& t) {
  if (t.x1 < t.x0) return t;
  return Rect{t.x0 / kBlk, t.y0 / kBlk, t.x1 / kBlk, t.y1 / kBlk};
}

// the part of a tile rectangle inside block b, in local tile coordinates
__device__ __forceinline__ Rect clip_to_block(const Rect& t, int bx, int by) {
  Rect r;
  r.x0 = max(t.x0, bx * kBlk) - bx * kBlk;
  r.x1 = min(t.x1, bx * kBlk + kBlk - 1) - bx * kBlk;
  r.y0 = max(t.y0, by * kBlk) - by * kBlk;
  r.y1 = min(t.y1, by * kBlk + kBlk - 1) - by * kBlk;
  if (r.x0 > r.x1 || r.y0 > r.y1) r = Rect{0, 0, -1, -1};
  return r;
}

// local rectangle packed as x0 | y0 << 3 | x1 << 6 | y1 << 9 | 1 << 12 (0 = none)
__device__ __forceinline__ int pack_local(const Rect& r) {
  if (r.x1 < r.x0) return 0;
  return r.x0 | (r.y0 << 3) | (r.x1 << 6) | (r.y1 << 9) | (1 << 12);
}

// ------------------------------------------------------------- level 1

// Agent-scope relaxed atomic loads and stores of 32-bit words: they reach the
// memory side, past every XCD's L2, so words handed from one workgroup to
// another through them need no cache write-back or invalidation. The writer's
// waves wait for their stores to complete before a barrier, after which one
// thread counts the workgroup in with an agent-scope atomic; the workgroup
// whose count completes a total then reads the words.
__device__ __forceinline__ void store_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t load_agent(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr uint32_t kNoBlock = 0xffffffffu;

// Wave64 minimum with DPP row operations; the result is uniform.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  const int no = (int)kNoBlock;
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0xB1, 0xF, 0xF, false));
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0x4E, 0xF, 0xF, false));
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0x141, 0xF, 0xF, false));
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0x140, 0xF, 0xF, false));
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0x142, 0xA, 0xF, false));
  x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(no, (int)x, 0x143, 0xC, 0xF, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}


// Level 1, one workgroup per chunk of kChunk consecutive depth ranks (chunk
// index from a ticket, in launch order). Wave w owns ranks [w kRanksPerWave,
// (w + 1) kRanksPerWave) of the chunk and counts, per block, the pairs its Gaussians
// make (LDS atomics). The chunk publishes its count of each block and reads
// the earlier chunks' through one 32-bit state word per (chunk, block)
// (decoupled look-back, as in the radix passes), so that a pair's slot is
// the block's bucket offset + the block's pairs in earlier chunks + its
// place in the chunk. Bucket offsets, the sub-chunk table and the overflow
// decision come from the block totals and intersection count depth_keys
// added up; every workgroup derives them (chunk 0 also writes them out). On
// overflow nothing is placed. Dynamic LDS: 5 x geo.nblk words.
// Level-2 slices of a block whose sub-chunks are [s0, s1): its parts of the
// aligned groups of kSlice consecutive sub-chunks (one l2_count workgroup
// each).
__device__ __forceinline__ uint32_t slices_of(uint32_t s0, uint32_t s1) {
  return s1 > s0 ? (s1 - 1) / kSlice - s0 / kSlice + 1 : 0u;
}

__global__ __launch_bounds__(256) void l1_place_kernel(
    int64_t n, const uint32_t* __restrict__ order, const unsigned long long* __restrict__ rects,
    Geo geo, const uint32_t* __restrict__ bcopy, const unsigned long long* __restrict__ mcopy,
    unsigned long long capacity, int64_t chunks, uint32_t* __restrict__ lb,
    uint32_t* __restrict__ blk_off, uint32_t* __restrict__ sub_off, uint32_t* __restrict__ slice_off,
    WsHeader* __restrict__ hdr, unsigned long long* __restrict__ pairs,
    uint32_t* __restrict__ tile_total) {
  using SW = StateWord<uint32_t>;
  extern __shared__ uint32_t lds[];
  uint32_t* slot = lds;                    // [4][nblk]: per wave counts, then next free slots
  uint32_t* boff = lds + 4 * geo.nblk;     // [nblk]: block totals, then bucket offsets
  __shared__ uint32_t s4[4];
  __shared__ uint32_t s_chunk;
  __shared__ unsigned long long s_m;
  const int nblk = geo.nblk;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  if (tid == 0) s_chunk = atomicAdd(&hdr->ticket_l1, 1u);
  if (w == 0) {
    const unsigned long long v = wave_sum_u64(lane < kHistCopies ? mcopy[lane] : 0ull);
    if (lane == 0) s_m = v;
  }
  for (int t = tid; t < 4 * nblk; t += kBlock) slot[t] = 0;
  // block totals and their exclusive prefixes (buckets) in pairs and in
  // sub-chunks; thread tid takes the contiguous blocks [b0, b1)
  const int per = (nblk + kBlock - 1) / kBlock;
  const int b0 = min(nblk, per * tid), b1 = min(nblk, b0 + per);
  uint32_t tot = 0, stot = 0;
  for (int b = b0; b < b1; ++b) {
    uint32_t c[kHistCopies];
#pragma unroll
    for (int r = 0; r < kHistCopies; ++r) c[r] = bcopy[(size_t)r * nblk + b];
    uint32_t v = 0;
#pragma unroll
    for (int r = 0; r < kHistCopies; ++r) v += c[r];
    boff[b] = v;
    tot += v;
    stot += (v + kSub - 1) / kSub;
  }
  uint32_t run = scan_256(tot, s4);  // its barriers publish s_chunk, s_m and the cleared slots
  uint32_t srun = scan_256(stot, s4);
  const int64_t chunk = s_chunk;
  uint32_t lrun = 0;
  if (chunk == 0) {  // uniform: only chunk 0 writes the slice table
    uint32_t ltot = 0, sr = srun;
    for (int b = b0; b < b1; ++b) {
      const uint32_t ns = (boff[b] + kSub - 1) / kSub;
      ltot += slices_of(sr, sr + ns);
      sr += ns;
    }
    lrun = scan_256(ltot, s4);
  }
  const unsigned long long m = s_m;
  const bool over = m > capacity || m >= (1ull << 32);
  if (chunk == 0) {
    // blocks without entries (every block on overflow): their tiles' totals
    // are 0, and level 2 counts only the others
    uint32_t ne = 0;
    for (int b = b0; b < b1; ++b) {
      if (boff[b] != 0u && !over) {
        ++ne;
        continue;
      }
      const int bx = b % geo.nbx, by = b / geo.nbx;
      for (int t = 0; t < kBlkTiles; ++t) {
        const int tx = bx * kBlk + (t & 7), ty = by * kBlk + (t >> 3);
        if (tx < geo.ntx && ty < geo.nty) tile_total[ty * geo.ntx + tx] = 0u;
      }
    }
    ne = wave_sum_u32(ne);
    if (lane == 0 && ne) atomicAdd(&hdr->nonempty, ne);
  }
  for (int b = b0; b < b1; ++b) {
    const uint32_t v = boff[b];
    boff[b] = run;
    if (chunk == 0) {
      blk_off[b] = run;
      sub_off[b] = srun;
      slice_off[b] = lrun;
      lrun += slices_of(srun, srun + (v + kSub - 1) / kSub);
    }
    run += v;
    srun += (v + kSub - 1) / kSub;
  }
  if (chunk == 0 && tid == kBlock - 1) {  // the last range ends at the totals
    blk_off[nblk] = run;
    sub_off[nblk] = srun;
    slice_off[nblk] = lrun;
    hdr->m = m;
    hdr->m1 = run;
    hdr->overflow = over ? 1u : 0u;
    hdr->total_sub = over ? 0u : srun;
  }
  if (over) return;  // the same decision in every workgroup: nobody waits
  uint32_t* my = slot + w * nblk;
  const int64_t rbase = chunk * kChunk + (int64_t)w * kRanksPerWave;
  uint32_t gj[kL1Items];
  Rect bj[kL1Items], tj[kL1Items];
#pragma unroll
  for (int j = 0; j < kL1Items; ++j) {
    const int64_t r = rbase + lane + 64 * j;
    gj[j] = r < n ? order[r] : 0u;
    tj[j] = r < n ? rect_of(gj[j], rects) : Rect{0, 0, -1, -1};
    bj[j] = block_rect(tj[j]);
    for (int y = bj[j].y0; y <= bj[j].y1; ++y)
      for (int x = bj[j].x0; x <= bj[j].x1; ++x) atomicAdd(&my[y * geo.nbx + x], 1u);
  }
  __syncthreads();
  // publish this chunk's count of each of the thread's blocks, then read the
  // earlier chunks' and turn the per-wave counts into slots
  for (int b = b0; b < b1; ++b) {
    const uint32_t own = slot[b] + slot[nblk + b] + slot[2 * nblk + b] + slot[3 * nblk + b];
    __hip_atomic_store(&lb[chunk * nblk + b], (chunk == 0 ? SW::kIncl : SW::kAgg) | own,
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  for (int b = b0; b < b1; ++b) {
    uint32_t excl = 0;
    if (chunk > 0) {
      excl = look_back(lb, chunk, nblk, b);
      // the inclusive count of a chunk before the last stays below n <= 2^30
      if (chunk + 1 < chunks) {
        const uint32_t own = slot[b] + slot[nblk + b] + slot[2 * nblk + b] + slot[3 * nblk + b];
        __hip_atomic_store(&lb[chunk * nblk + b], SW::kIncl | (excl + own), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    uint32_t at = boff[b] + excl;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t c = slot[k * nblk + b];
      slot[k * nblk + b] = at;
      at += c;
    }
  }
  __syncthreads();
  // Placement, one distinct block at a time in increasing block order: each
  // entry walks its block rectangle row-major, so the smallest pending block
  // of the wave is the current cell of every entry that covers it; ballots
  // give each such entry its rank (entries in rank order: j, then lane).
  uint32_t nb[kL1Items];
  int cx[kL1Items], cy[kL1Items];
#pragma unroll
  for (int j = 0; j < kL1Items; ++j) {
    cx[j] = bj[j].x0;
    cy[j] = bj[j].y0;
    nb[j] = bj[j].x1 >= bj[j].x0 ? (uint32_t)(cy[j] * geo.nbx + cx[j]) : kNoBlock;
  }
  const uint64_t lt = lanemask_lt();
  while (true) {
    uint32_t lo = nb[0];
#pragma unroll
    for (int j = 1; j < kL1Items; ++j) lo = min(lo, nb[j]);
    const uint32_t B = wave_min_u32(lo);
    if (B == kNoBlock) break;
    uint32_t at = my[B];
#pragma unroll
    for (int j = 0; j < kL1Items; ++j) {
      const bool hit = nb[j] == B;
      const uint64_t bal = __ballot(hit);
      if (hit) {
        // the pair carries the rectangle clipped to its block, packed (the
        // slot is below m1 <= capacity; the test keeps any inconsistency in
        // the counts from writing past the array)
        const uint32_t pos = at + (uint32_t)__popcll(bal & lt);
        if (pos < capacity)
          pairs[pos] = (unsigned long long)gj[j] |
                       ((unsigned long long)pack_local(clip_to_block(tj[j], cx[j], cy[j])) << 32);
        if (cx[j] < bj[j].x1) {
          ++cx[j];
        } else {
          cx[j] = bj[j].x0;
          ++cy[j];
        }
        nb[j] = cy[j] <= bj[j].y1 ? (uint32_t)(cy[j] * geo.nbx + cx[j]) : kNoBlock;
      }
      at += (uint32_t)__popcll(bal);
    }
    if (lane == 0) my[B] = at;
  }
}

// ------------------------------------------------------------- level 2
//
// A block has 8 x 8 = 64 tiles (local tile l at x = l % 8, y = l / 8). Each
// bucket is cut into sub-chunks of kSub consecutive entries, and its
// sub-chunks into slices of kSlice. l2_count counts each tile's entries per
// sub-chunk and sums them over the slice: each sub-chunk's first slot in
// every tile list relative to its slice, and the slice's totals; a block's
// slice totals then become the slices' first slots (a block at the frame's
// centre can hold thousands of sub-chunks, and its scan runs on one
// workgroup: over slices it reads kSlice times fewer rows). l2_scatter writes
// the entries.

struct SubChunk {
  int bx, by, blk;   // block
  uint32_t e0, e1;   // entries [e0, e1) of the pair array
};

// The last b with off[b] <= x (off is nondecreasing over the blocks), with
// off[b] and other[b]. A wave finds it at once: lane b tests block b, 64
// blocks per round (coalesced loads instead of a binary search's chain of
// dependent ones), and the highest block that passes wins; its two values
// come from the same loads.
__device__ __forceinline__ int block_of_wave(uint32_t x, const uint32_t* __restrict__ off,
                                              const uint32_t* __restrict__ other, int nblk,
                                              uint32_t& off_b, uint32_t& other_b) {
  const int lane = threadIdx.x & 63;
  int lo = 0;
  off_b = other_b = 0;
  for (int b0 = 0; b0 < nblk; b0 += 64) {
    const int b = b0 + lane;
    const uint32_t o = b < nblk ? off[b] : 0u, t = b < nblk ? other[b] : 0u;
    const uint64_t ok = __ballot(b < nblk && o <= x);
    if (ok) {
      const int hi = 63 - __clzll(ok);
      lo = b0 + hi;
      off_b = (uint32_t)__builtin_amdgcn_readlane((int)o, hi);
      other_b = (uint32_t)__builtin_amdgcn_readlane((int)t, hi);
    }
  }
  return __builtin_amdgcn_readfirstlane(lo);
}

// Sub-chunk s of block b.
__device__ __forceinline__ SubChunk sub_chunk_of(uint32_t s, int b,
                                                 const uint32_t* __restrict__ sub_off,
                                                 const uint32_t* __restrict__ blk_off,
                                                 const Geo& geo) {
  SubChunk c;
  c.blk = b;
  c.bx = b % geo.nbx;
  c.by = b / geo.nbx;
  c.e0 = blk_off[b] + (s - sub_off[b]) * kSub;
  c.e1 = min(c.e0 + (uint32_t)kSub, blk_off[b + 1]);
  return c;
}

// Coverage counts of a wave's entries per local tile by a 2D difference
// array: an entry covering [x0, x1] x [y0, y1] adds +1 at (x0, y0), -1 at
// (x1 + 1, y0) and (x0, y1 + 1), +1 at (x1 + 1, y1 + 1) (corners outside the
// 8 x 8 block are dropped); the 2D inclusive prefix sum at tile (lx, ly) is
// the number of entries covering it. d is the wave's 64-word LDS array,
// zeroed by the caller; lane l returns the count of local tile l.
__device__ __forceinline__ void diff_add(uint32_t* d, int packed) {
  if (packed == 0) return;
  const int x0 = packed & 7, y0 = (packed >> 3) & 7, x1 = (packed >> 6) & 7, y1 = (packed >> 9) & 7;
  atomicAdd(&d[y0 * 8 + x0], 1u);
  if (x1 < 7) atomicAdd(&d[y0 * 8 + x1 + 1], 0xffffffffu);
  if (y1 < 7) atomicAdd(&d[(y1 + 1) * 8 + x0], 0xffffffffu);
  if (x1 < 7 && y1 < 7) atomicAdd(&d[(y1 + 1) * 8 + x1 + 1], 1u);
}

__device__ __forceinline__ uint32_t diff_prefix(uint32_t v, int lane) {
#pragma unroll
  for (int off = 1; off < 8; off <<= 1) {  // along the row (x)
    const uint32_t t = __shfl_up(v, off, 8);
    if ((lane & 7) >= off) v += t;
  }
#pragma unroll
  for (int off = 8; off < 64; off <<= 1) {  // down the columns (y)
    const uint32_t t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

__device__ __forceinline__ void load_entry(const unsigned long long* __restrict__ pairs,
                                           uint32_t e, uint32_t e1, uint32_t& g, int& packed) {
  g = 0;
  packed = 0;
  if (e < e1) {
    const unsigned long long p = pairs[e];
    g = (uint32_t)p;
    packed = (int)(p >> 32);
  }
}

// Exclusive scan over tiles -> tile_off and tile_ranges, by one workgroup of
// kScanThreads (on overflow every tile total is 0, so the ranges written
// are all empty and the blend kernels render nothing).
// s_key (workgroup memory, may be NULL): also each tile's schedule bucket,
// from the same loads.
__device__ __forceinline__ void scan_tiles(const uint32_t* __restrict__ tile_total, int ntiles,
                                           uint32_t* __restrict__ tile_off,
                                           uint32_t* __restrict__ tile_ranges, uint8_t* s_key) {
  // rounds of kScanThreads * kPer tiles, thread t taking kPer contiguous
  // tiles of each, all loads of a round in flight at once; the sums fit 32
  // bits (M < 2^32 unless overflowing, and then every total is 0)
  constexpr int kPer = 8;
  __shared__ uint32_t s_wave[kScanThreads / 64];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  uint32_t carry = 0;
  for (int r0 = 0; r0 < ntiles; r0 += kScanThreads * kPer) {
    const int lo = r0 + kPer * tid;
    uint32_t v[kPer];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      v[k] = lo + k < ntiles ? load_agent(&tile_total[lo + k]) : 0u;
      s += v[k];
    }
    if (s_key) {
#pragma unroll
      for (int k = 0; k < kPer; ++k)
        if (lo + k < ntiles) s_key[lo + k] = (uint8_t)bucket_of(v[k]);
    }
    uint32_t incl = s;  // inclusive prefix over the wave
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)incl, d, 64);
      if (lane >= d) incl += y;
    }
    if (lane == 63) s_wave[w] = incl;
    __syncthreads();
    uint32_t run = carry + incl - s, all = 0;
#pragma unroll
    for (int k = 0; k < kScanThreads / 64; ++k) {
      const uint32_t c = s_wave[k];
      run += k < w ? c : 0u;
      all += c;
    }
    __syncthreads();  // s_wave is rewritten by the next round
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (lo + k < ntiles) {
        tile_off[lo + k] = run;
        tile_ranges[2 * (lo + k)] = run;
        tile_ranges[2 * (lo + k) + 1] = run + v[k];
      }
      run += v[k];
    }
    carry += all;
  }
}

// Level 2's counts and scans in one launch. Workgroup k (grid stride) takes
// the sub-chunks [kSlice k, kSlice k + kSlice), wave w sub-chunk kSlice k + w,
// and counts its entries per tile; the group holds one slice of each block
// it meets. For each sub-chunk s, c2[s][tile] = entries of the earlier
// sub-chunks of its slice covering the tile, and slice_tot[slice][tile] =
// all of the slice's. The workgroup that completes a block's last slice turns
// the block's slice totals into each slice's first slot relative to the
// block (lane = local tile, the 16 waves split the slices, kScanRows rows in
// flight per wave) and writes the block's tile totals; the one that completes
// the last nonempty block scans the tile totals into tile_off and
// tile_ranges. With no sub-chunk at all (no entries, or overflow: every tile
// total is 0, which gives empty ranges) the first workgroup does that
// directly. Slice totals and tile totals pass between workgroups through
// store_agent and load_agent.
constexpr int kScanRows = 4;

__global__ __launch_bounds__(64 * kSlice) __attribute__((amdgpu_waves_per_eu(8))) void l2_count_kernel(
    const unsigned long long* __restrict__ pairs, Geo geo, const uint32_t* __restrict__ sub_off,
    const uint32_t* __restrict__ slice_off, const uint32_t* __restrict__ blk_off,
    WsHeader* __restrict__ hdr, uint32_t* __restrict__ c2, uint32_t* __restrict__ slice_tot,
    uint32_t* __restrict__ blk_done, uint32_t* __restrict__ tile_total,
    uint32_t* __restrict__ tile_off, uint32_t* __restrict__ tile_ranges) {
  static_assert(kSub == 4 * 64, "a sub-chunk is four entries per lane");
  static_assert(64 * kSlice == kScanThreads, "the tile scan takes the whole workgroup");
  __shared__ uint32_t d[kSlice][kBlkTiles];
  __shared__ int s_blk[kSlice];          // block of each wave's sub-chunk (-1: none)
  __shared__ uint32_t s_nsl[kSlice];     // slices of that block
  __shared__ uint32_t s_soff[kSlice];    // its first slice
  __shared__ int s_done[kSlice + 1];     // blocks completed here, then their count
  __shared__ uint32_t s_final;
  const uint32_t total = hdr->total_sub, nonempty = hdr->nonempty;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int ntiles = geo.ntx * geo.nty;
  bool final_step = total == 0u && blockIdx.x == 0;
  for (uint32_t g0 = blockIdx.x * (uint32_t)kSlice; g0 < total; g0 += gridDim.x * (uint32_t)kSlice) {
    const uint32_t s = g0 + (uint32_t)w;
    const bool live = s < total;  // uniform per wave
    int b = -1;
    uint32_t subb = 0, soff = 0, sub1 = 0, cnt = 0;
    int pk[4] = {0, 0, 0, 0};
    if (live) {
      b = block_of_wave(s, sub_off, slice_off, geo.nblk, subb, soff);
      sub1 = sub_off[b + 1];
      const uint32_t e0 = blk_off[b] + (s - subb) * kSub, e1 = blk_off[b + 1];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint32_t g;
        load_entry(pairs, e0 + lane + 64 * j, e1, g, pk[j]);
      }
    }
    d[w][lane] = 0;
    if (lane == 0) {
      s_blk[w] = b;
      s_nsl[w] = live ? slice_off[b + 1] - soff : 0u;
      s_soff[w] = soff;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) diff_add(d[w], pk[j]);  // 0 for no entry
    __syncthreads();
    cnt = diff_prefix(d[w][lane], lane);
    __syncthreads();
    d[w][lane] = cnt;
    __syncthreads();
    uint32_t before = 0;
    for (int v = 0; v < w; ++v) before += s_blk[v] == b ? d[v][lane] : 0u;
    if (live) {
      c2[(int64_t)s * kBlkTiles + lane] = before;
      // the slice's last sub-chunk here: the slice total
      if (w == kSlice - 1 || s + 1 == sub1)
        store_agent(&slice_tot[(int64_t)(soff + s / kSlice - subb / kSlice) * kBlkTiles + lane],
                    before + cnt);
    }
    // count this group's slices in, one per block met: lane v of the first
    // wave for the slice ending at sub-chunk v (all atomics in flight at once)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (w == 0) {
      bool done = false;
      if (lane < kSlice) {
        const int bv = s_blk[lane];
        if (bv >= 0 && (lane + 1 == kSlice || s_blk[lane + 1] != bv))
          done = __hip_atomic_fetch_add(&blk_done[bv], 1u, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT) + 1u == s_nsl[lane];
      }
      const uint64_t m = __ballot(done);
      if (done) s_done[__popcll(m & ((1ull << lane) - 1ull))] = lane;
      if (lane == 0) s_done[kSlice] = __popcll(m);
    }
    __syncthreads();
    const int nd = s_done[kSlice];
    for (int i = 0; i < nd; ++i) {
      // block bb's slices, all counted: prefix over them and the tile totals
      const int v = s_done[i], bb = s_blk[v];
      const uint32_t nsl = s_nsl[v], base = s_soff[v];
      const uint32_t per = (nsl + kSlice - 1) / kSlice;
      const uint32_t q0 = min(nsl, per * w) + base, q1 = min(nsl, per * w + per) + base;
      uint32_t sum = 0;
      for (uint32_t q = q0; q < q1; q += kScanRows) {
        uint32_t x[kScanRows];
#pragma unroll
        for (int u = 0; u < kScanRows; ++u)
          x[u] = q + u < q1 ? load_agent(&slice_tot[(int64_t)(q + u) * kBlkTiles + lane]) : 0u;
#pragma unroll
        for (int u = 0; u < kScanRows; ++u) sum += x[u];
      }
      __syncthreads();  // every wave is done reading d
      d[w][lane] = sum;
      __syncthreads();
      uint32_t run = 0;
      for (int k = 0; k < w; ++k) run += d[k][lane];
      for (uint32_t q = q0; q < q1; q += kScanRows) {
        uint32_t x[kScanRows];
#pragma unroll
        for (int u = 0; u < kScanRows; ++u)
          x[u] = q + u < q1 ? load_agent(&slice_tot[(int64_t)(q + u) * kBlkTiles + lane]) : 0u;
#pragma unroll
        for (int u = 0; u < kScanRows; ++u) {
          if (q + u < q1) slice_tot[(int64_t)(q + u) * kBlkTiles + lane] = run;
          run += x[u];
        }
      }
      if (w == kSlice - 1) {
        const int bx = bb % geo.nbx, by = bb / geo.nbx;
        const int tx = bx * kBlk + (lane & 7), ty = by * kBlk + (lane >> 3);
        if (tx < geo.ntx && ty < geo.nty) store_agent(&tile_total[ty * geo.ntx + tx], run);
      }
    }
    if (nd > 0) {  // uniform
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0)
        s_final = __hip_atomic_fetch_add(&hdr->done_l2, (uint32_t)nd, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT) + (uint32_t)nd == nonempty;
      __syncthreads();
      if (s_final) final_step = true;
    }
    __syncthreads();  // the shared arrays are rewritten by the next group
  }
  if (!final_step) return;
  scan_tiles(tile_total, ntiles, tile_off, tile_ranges, nullptr);
}

// Ordered scatter of one 256-entry sub-chunk into its block's 64 tile lists.
// Wave w owns entries [64 w, 64 w + 64) of the sub-chunk, lane l entry
// 64 w + l. Eight column and eight row ballots give, for every local tile t,
// the mask of the wave's entries whose rectangle holds it (column mask of
// t % 8 and row mask of t / 8, wave-uniform); the wave then walks the 64
// tiles and the entries of each tile's mask write their Gaussian at the
// wave's first slot in that tile's run plus their rank among the mask's
// lanes, one store of consecutive addresses per tile. A tile's run takes the
// waves' entries in wave order (per-wave counts by 2D difference arrays).
// Workgroup 0 first orders the tiles for the forward when tile_order is given
// (heaviest lists first; on overflow every total is 0, which gives the
// identity), beside the others' scatter; its buckets go to the dynamic
// workgroup memory (one byte per tile).
__global__ __launch_bounds__(kBlock) void l2_scatter_kernel(
    const unsigned long long* __restrict__ pairs, const float* __restrict__ depth, Geo geo,
    const uint32_t* __restrict__ sub_off, const uint32_t* __restrict__ slice_off,
    const uint32_t* __restrict__ blk_off, const uint32_t* __restrict__ c2,
    const uint32_t* __restrict__ slice_tot, const uint32_t* __restrict__ tile_off,
    const WsHeader* __restrict__ hdr, uint32_t* __restrict__ values_sorted,
    unsigned long long* __restrict__ keys_sorted, const uint32_t* __restrict__ tile_total,
    uint32_t* __restrict__ tile_order) {
  __shared__ uint32_t wcnt[4][kBlkTiles];   // per wave: entries covering each tile
  __shared__ uint32_t wdiff[4][kBlkTiles];  // per wave difference arrays
  extern __shared__ uint8_t s_key[];        // workgroup 0: bucket of each tile
  if (tile_order && blockIdx.x == 0) {  // uniform
    const int ntiles = geo.ntx * geo.nty;
    for (int t = threadIdx.x; t < ntiles; t += kBlock) s_key[t] = (uint8_t)bucket_of(tile_total[t]);
    __syncthreads();
    order_keyed<kBlock>(ntiles, s_key, tile_order, nullptr);
  }
  const uint32_t total = hdr->total_sub;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (uint32_t s = blockIdx.x; s < total; s += gridDim.x) {
    uint32_t subb, soff;
    const SubChunk sc =
        sub_chunk_of(s, block_of_wave(s, sub_off, slice_off, geo.nblk, subb, soff), sub_off, blk_off, geo);
    uint32_t g;
    int pk;
    load_entry(pairs, sc.e0 + threadIdx.x, sc.e1, g, pk);
    // global start of each tile's run in the sub-chunk (lane = local tile),
    // loaded now so that its latency overlaps the counting below
    uint32_t dst_l = 0u;
    {
      const int tx = sc.bx * kBlk + (lane & 7), ty = sc.by * kBlk + (lane >> 3);
      const uint32_t sl = soff + s / kSlice - subb / kSlice;
      if (tx < geo.ntx && ty < geo.nty)
        dst_l = tile_off[ty * geo.ntx + tx] + slice_tot[(int64_t)sl * kBlkTiles + lane] +
                c2[(int64_t)s * kBlkTiles + lane];
    }
    const uint32_t key_lo = keys_sorted && pk != 0 ? __float_as_uint(depth[g]) : 0u;
    wdiff[w][lane] = 0;
    __syncthreads();
    diff_add(wdiff[w], pk);
    __syncthreads();
    wcnt[w][lane] = diff_prefix(wdiff[w][lane], lane);
    __syncthreads();
    // this wave's first slot in the run of tile `lane`
    uint32_t base = dst_l;
#pragma unroll
    for (int k = 0; k < 3; ++k) base += k < w ? wcnt[k][lane] : 0u;
    uint64_t colm[kBlk], rowm[kBlk];
    {
      const int x0 = pk & 7, y0 = (pk >> 3) & 7, x1 = (pk >> 6) & 7, y1 = (pk >> 9) & 7;
      const bool v = pk != 0;
#pragma unroll
      for (int c = 0; c < kBlk; ++c) {
        colm[c] = __ballot(v && x0 <= c && c <= x1);
        rowm[c] = __ballot(v && y0 <= c && c <= y1);
      }
    }
#pragma unroll
    for (int t = 0; t < kBlkTiles; ++t) {
      const uint64_t m = colm[t & 7] & rowm[t >> 3];
      if (m == 0) continue;
      const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)base, t);
      if (__builtin_amdgcn_inverse_ballot_w64(m)) {  // this lane's bit of m
        const uint32_t pos =
            b + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        values_sorted[pos] = g;
        if (keys_sorted) {
          const uint32_t tile = (uint32_t)((sc.by * kBlk + (t >> 3)) * geo.ntx + sc.bx * kBlk + (t & 7));
          keys_sorted[pos] = ((unsigned long long)tile << 32) | key_lo;
        }
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------- small active blocks
//
// A small active block (the regime where ABCD's partitions hold few Gaussians
// and launch costs dominate) is binned in two launches instead of the general
// path's 22: one workgroup sorts the Gaussians by depth in LDS, counts each
// tile's list from the rectangles and scans the counts into the tile ranges;
// then one workgroup per tile collects, in depth order, the Gaussians whose
// rectangle covers it. The lists are the same as the general path's.

constexpr int kSmallN = 2048;        // Gaussians the one-workgroup sort holds
constexpr int kSmallTiles = 2048;    // tiles of the frame (each coordinate below 256)
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / 64;
constexpr int kSmallKeyBytes = kSmallN * 4;
static_assert(kSmallThreads == kOrderThreads, "the small path orders tiles with order_tiles");

bool small_path(int64_t n, const Geo& g) {
  return n <= kSmallN && (int64_t)g.ntx * g.nty <= kSmallTiles && g.ntx <= 256 && g.nty <= 256;
}

// tile rectangle in bytes: x0 | x1 << 8 | y0 << 16 | y1 << 24 (empty: x0 = 1 > x1 = 0)
__device__ __forceinline__ uint32_t pack_rect8(int x0, int y0, int x1, int y1) {
  return (uint32_t)x0 | ((uint32_t)x1 << 8) | ((uint32_t)y0 << 16) | ((uint32_t)y1 << 24);
}

// Exclusive scan over the threads of a workgroup of kSmallThreads: each wave
// scans its 64 values with shuffles, one barrier publishes the wave totals
// (s: kSmallWaves words of LDS), and each thread adds the totals of the waves
// before its own. Returns the exclusive prefix and the total in *tot.
__device__ __forceinline__ uint32_t scan_small(uint32_t v, uint32_t* s, uint32_t* tot) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  uint32_t incl = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) s[w] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < kSmallWaves; ++k) {
    const uint32_t c = s[k];
    before += k < w ? c : 0u;
    all += c;
  }
  *tot = all;
  __syncthreads();
  return before + incl - v;
}

// One workgroup: keys (fp32 depth bits; Gaussians with no tile last) and byte
// rectangles; a stable LSD radix sort by key in LDS (8-bit digits; wave w
// ranks its 128 consecutive entries with ballots, the waves' digit counts give
// the offsets), which keeps equal keys in index order; per-tile counts by LDS
// atomics over each rectangle; their exclusive scan (tile_off, tile_ranges);
// the sorted Gaussians and their rectangles for the per-tile collection; M
// and the overflow decision in the header (on overflow
// every range is empty), and the forward's tile order.
__global__ __launch_bounds__(kSmallThreads) void bin_small_sort_kernel(
    int n, const float* __restrict__ depth, const uint32_t* __restrict__ tiles,
    const float* __restrict__ means2d, const float* __restrict__ extent, Geo geo,
    unsigned long long capacity, uint32_t* __restrict__ sorted_g, uint32_t* __restrict__ sorted_rect,
    uint32_t* __restrict__ tile_off, uint32_t* __restrict__ tile_ranges,
    uint32_t* __restrict__ tile_order, WsHeader* __restrict__ hdr) {
  __shared__ uint32_t s_key[2][kSmallN];
  __shared__ uint16_t s_val[2][kSmallN];
  __shared__ uint32_t s_rect[kSmallN];
  __shared__ uint16_t s_cnt[kSmallWaves][256];
  __shared__ uint32_t s_tcount[kSmallTiles];
  __shared__ uint32_t s_scan[kSmallWaves];
  __shared__ unsigned long long s_m;
  __shared__ uint32_t s_kor, s_kand;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int ntiles = geo.ntx * geo.nty;
  for (int t = tid; t < ntiles; t += kSmallThreads) s_tcount[t] = 0;
  if (tid == 0) {
    s_m = 0;
    s_kor = 0u;
    s_kand = 0xffffffffu;
  }
  __syncthreads();
  unsigned long long m = 0;
  uint32_t kor = 0u, kand = 0xffffffffu;  // bits set in some key / in every key
  for (int i = tid; i < n; i += kSmallThreads) {
    const uint32_t tt = tiles[i];
    uint32_t key = 0xffffffffu;
    int x0 = 1, y0 = 0, x1 = 0, y1 = 0;
    if (tt != 0) {
      key = __float_as_uint(depth[i]);
      const float2 mm = reinterpret_cast<const float2*>(means2d)[i];
      const float2 ex = reinterpret_cast<const float2*>(extent)[i];
      if (!tile_rect(mm.x, mm.y, ex.x, ex.y, geo.ntx, geo.nty, x0, y0, x1, y1))
        x0 = 1, y0 = 0, x1 = 0, y1 = 0;
    }
    s_key[0][i] = key;
    s_val[0][i] = (uint16_t)i;
    s_rect[i] = pack_rect8(x0, y0, x1, y1);
    kor |= key;
    kand &= key;
    if (x1 >= x0) {
      m += tt;
      for (int y = y0; y <= y1; ++y)
        for (int x = x0; x <= x1; ++x) atomicAdd(&s_tcount[y * geo.ntx + x], 1u);
    }
  }
  const unsigned long long wm = wave_sum_u64(m);
  if (lane == 0 && wm) atomicAdd(&s_m, wm);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kor |= (uint32_t)__shfl_xor((int)kor, off, 64);
    kand &= (uint32_t)__shfl_xor((int)kand, off, 64);
  }
  if (lane == 0) {
    atomicOr(&s_kor, kor);
    atomicAnd(&s_kand, kand);
  }
  __syncthreads();
  const unsigned long long mt = s_m;
  const bool over = mt > capacity || mt >= (1ull << 32);
  // radix sort: wave w owns positions [128 w, 128 w + 128); the waves past
  // the last key (nw and on) hold nothing, and a digit that every key shares
  // would leave the order as it is, so its pass is skipped
  const uint64_t lt = lanemask_lt();
  const int nw = (n + 127) / 128;
  const uint32_t varying = s_kor ^ s_kand;
  int src = 0;  // buffer holding the order so far (uniform)
#pragma unroll 1
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 8 * pass;
    if (((varying >> shift) & 255u) == 0u) continue;  // uniform
    for (int i = tid; i < nw * 256; i += kSmallThreads) (&s_cnt[0][0])[i] = 0;
    __syncthreads();
    uint32_t key[2], rank[2];
    uint16_t val[2];
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int idx = 128 * w + 64 * it + lane;
      const bool valid = idx < n;
      key[it] = valid ? s_key[src][idx] : 0u;
      val[it] = valid ? s_val[src][idx] : (uint16_t)0;
      const uint32_t d = (key[it] >> shift) & 255u;
      const uint64_t peers = match_digit(d, __ballot(valid));
      rank[it] = 0;
      if (valid) {
        rank[it] = s_cnt[w][d] + (uint32_t)__popcll(peers & lt);
        if (lane == __ffsll((unsigned long long)peers) - 1)
          s_cnt[w][d] = (uint16_t)(s_cnt[w][d] + __popcll(peers));
      }
    }
    __syncthreads();
    // digit d: total over the waves, exclusive base over the digits, then the
    // waves' offsets in place
    uint32_t tot_d = 0;
    if (tid < 256)
      for (int v = 0; v < nw; ++v) tot_d += s_cnt[v][tid];
    uint32_t total;
    uint32_t base = scan_small(tid < 256 ? tot_d : 0u, s_scan, &total);
    if (tid < 256)
      for (int v = 0; v < nw; ++v) {
        const uint32_t c = s_cnt[v][tid];
        s_cnt[v][tid] = (uint16_t)base;
        base += c;
      }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int idx = 128 * w + 64 * it + lane;
      if (idx < n) {
        const uint32_t pos = s_cnt[w][(key[it] >> shift) & 255u] + rank[it];
        s_key[src ^ 1][pos] = key[it];
        s_val[src ^ 1][pos] = val[it];
      }
    }
    __syncthreads();
    src ^= 1;
  }
  for (int j = tid; j < n; j += kSmallThreads) {
    const uint32_t g = s_val[src][j];
    sorted_g[j] = g;
    sorted_rect[j] = s_rect[g];
  }
  // tile ranges: runs of `per` tiles per thread
  const int per = (ntiles + kSmallThreads - 1) / kSmallThreads;
  const int lo = min(ntiles, per * tid), hi = min(ntiles, lo + per);
  uint32_t sum = 0;
  for (int t = lo; t < hi; ++t) sum += over ? 0u : s_tcount[t];
  uint32_t total;
  uint32_t run = scan_small(sum, s_scan, &total);
  for (int t = lo; t < hi; ++t) {
    const uint32_t c = over ? 0u : s_tcount[t];
    tile_off[t] = run;
    tile_ranges[2 * t] = run;
    tile_ranges[2 * t + 1] = run + c;
    run += c;
    if (over) s_tcount[t] = 0u;
  }
  if (tile_order) {
    // the forward's schedule: heaviest lists first (identity on overflow); the
    // bucket keys go where the sort's second key buffer was
    static_assert(kSmallKeyBytes >= kSmallTiles, "bucket keys fit the spare key buffer");
    __syncthreads();
    order_tiles(ntiles, s_tcount, tile_order, reinterpret_cast<uint8_t*>(s_key[1]));
  }
  if (tid == 0) {
    hdr->m = mt;
    hdr->m1 = 0;
    hdr->overflow = over ? 1u : 0u;
    hdr->total_sub = 0;
  }
}

// One workgroup per tile: the sorted Gaussians whose rectangle covers the
// tile, in sorted order, 256 positions per round (ballots rank them).
__global__ __launch_bounds__(256) void bin_small_collect_kernel(
    int n, const float* __restrict__ depth, Geo geo, const uint32_t* __restrict__ sorted_g,
    const uint32_t* __restrict__ sorted_rect, const uint32_t* __restrict__ tile_off,
    const WsHeader* __restrict__ hdr, uint32_t* __restrict__ values_sorted,
    unsigned long long* __restrict__ keys_sorted) {
  __shared__ uint32_t s_w[4];
  if (hdr->overflow) return;
  const int t = blockIdx.x, tx = t % geo.ntx, ty = t / geo.ntx;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint64_t lt = lanemask_lt();
  uint32_t run = tile_off[t];
  for (int j0 = 0; j0 < n; j0 += 256) {
    const int j = j0 + threadIdx.x;
    bool hit = false;
    uint32_t g = 0;
    if (j < n) {
      const uint32_t r = sorted_rect[j];
      const int x0 = r & 255, x1 = (r >> 8) & 255, y0 = (r >> 16) & 255, y1 = r >> 24;
      hit = x0 <= tx && tx <= x1 && y0 <= ty && ty <= y1;
      g = sorted_g[j];
    }
    const uint64_t bal = __ballot(hit);
    if (lane == 0) s_w[w] = (uint32_t)__popcll(bal);
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const uint32_t c = s_w[v];
      before += v < w ? c : 0u;
      tot += c;
    }
    if (hit) {
      const uint32_t pos = run + before + (uint32_t)__popcll(bal & lt);
      values_sorted[pos] = g;
      if (keys_sorted) keys_sorted[pos] = ((unsigned long long)t << 32) | __float_as_uint(depth[g]);
    }
    run += tot;
    __syncthreads();
  }
}

__global__ void bin_empty_kernel(int ntiles, uint32_t* __restrict__ tile_ranges,
                                 uint32_t* __restrict__ tile_order, WsHeader* __restrict__ hdr) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < 2 * ntiles; i += gridDim.x * blockDim.x) {
    tile_ranges[i] = 0u;
    if (tile_order && i < ntiles) tile_order[i] = (uint32_t)i;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    hdr->m = 0;
    hdr->m1 = 0;
    hdr->overflow = 0;
    hdr->total_sub = 0;
  }
}

int32_t set_max_lds(const void* fn, size_t bytes) {
  ABCD_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
  return ABCD_OK;
}

}  // namespace

size_t bin_sort_workspace_bytes(int64_t n, int64_t capacity, int width, int height) {
  return ws_layout(n, capacity, geo_of(width, height)).total;
}

int32_t launch_bin_sort(int width, int height, int64_t n, const float* means2d, const float* extent,
                        const float* depth, const uint32_t* tiles_touched, int64_t capacity,
                        void* workspace, uint64_t* keys_sorted, uint32_t* values_sorted,
                        uint32_t* tile_ranges, uint32_t* tile_order, hipStream_t stream) {
  const Geo geo = geo_of(width, height);
  const int ntiles = geo.ntx * geo.nty;
  const WsLayout L = ws_layout(n, capacity, geo);
  char* ws = static_cast<char*>(workspace);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  if (n == 0) {
    ABCD_LAUNCH("bin_empty", bin_empty_kernel, std::max(1, (2 * ntiles + 255) / 256), 256, 0,
                stream, ntiles, tile_ranges, tile_order, hdr);
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  auto u32 = [&](size_t off) { return reinterpret_cast<uint32_t*>(ws + off); };
  if (small_path(n, geo)) {
    const unsigned long long cap_s = (unsigned long long)std::max<int64_t>(capacity, 0);
    ABCD_LAUNCH("bin_small_sort", bin_small_sort_kernel, 1, kSmallThreads, 0, stream, (int)n,
                depth, tiles_touched, means2d, extent, geo, cap_s, u32(L.keys_a), u32(L.keys_b),
                u32(L.tile_off), tile_ranges, tile_order, hdr);
    ABCD_LAUNCH("bin_small_collect", bin_small_collect_kernel, ntiles, kBlock, 0, stream, (int)n,
                depth, geo, u32(L.keys_a), u32(L.keys_b), u32(L.tile_off), hdr, values_sorted,
                reinterpret_cast<unsigned long long*>(keys_sorted));
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  uint32_t* keys[2] = {u32(L.keys_a), u32(L.keys_b)};
  uint32_t* vals[2] = {u32(L.vals_a), u32(L.vals_b)};
  unsigned long long* pstate[2] = {reinterpret_cast<unsigned long long*>(ws + L.st0),
                                   reinterpret_cast<unsigned long long*>(ws + L.st1)};
  uint32_t* ghist = u32(L.ghist);
  unsigned long long* rects = reinterpret_cast<unsigned long long*>(ws + L.rects);
  {
    const int64_t words = (int64_t)(L.st1 - L.hdr) / 16;
    ABCD_LAUNCH("bin_zero", bin_zero_kernel, std::min<int64_t>(1024, (words + kBlock - 1) / kBlock),
                kBlock, 0, stream, reinterpret_cast<uint4*>(ws + L.hdr), words);
  }
  static bool attrs_set = false;
  if (!attrs_set) {
    // depth_keys keeps 4 words and level 1 5 words per block of any frame of
    // at most ABCD_MAX_TILES tiles (at most ABCD_MAX_TILES / 8 blocks)
    int32_t st = set_max_lds((const void*)depth_keys_kernel,
                             4 * sizeof(uint32_t) * (ABCD_MAX_TILES / kBlk + 1));
    if (st != ABCD_OK) return st;
    st = set_max_lds((const void*)l1_place_kernel,
                     5 * sizeof(uint32_t) * (ABCD_MAX_TILES / kBlk + 1));
    if (st != ABCD_OK) return st;
    attrs_set = true;
  }
  uint32_t* bcopy = u32(L.bcopy);
  unsigned long long* mcopy = reinterpret_cast<unsigned long long*>(ws + L.mcopy);
  ABCD_LAUNCH("depth_keys", depth_keys_kernel, (n + kDkTile - 1) / kDkTile, kBlock,
              4 * sizeof(uint32_t) * geo.nblk, stream, n, depth, tiles_touched, means2d, extent, geo,
              keys[0], rects, ghist, bcopy, mcopy);
  for (int pass = 0; pass < 4; ++pass) {
    const int src = pass & 1, dst = src ^ 1;
    ABCD_LAUNCH("radix_pass", radix_pass_kernel, L.rs_parts, kBlock, 0, stream, keys[src],
                pass == 0 ? nullptr : vals[src], n, pass, ghist, pstate[pass & 1],
                pass < 3 ? pstate[(pass + 1) & 1] : nullptr, &hdr->ticket[pass], keys[dst],
                vals[dst]);
  }
  const uint32_t* order = vals[0];  // four passes: back in buffer 0

  const unsigned long long cap = (unsigned long long)std::max<int64_t>(capacity, 0);
  uint32_t* blk_off = u32(L.blk_off);
  uint32_t* sub_off = u32(L.sub_off);
  unsigned long long* pairs = reinterpret_cast<unsigned long long*>(ws + L.pairs);
  uint32_t* c2 = u32(L.c2);
  uint32_t* tile_total = u32(L.tile_total);
  uint32_t* tile_off = u32(L.tile_off);
  uint32_t* slice_off = u32(L.slice_off);
  uint32_t* slice_tot = u32(L.slice_tot);
  ABCD_LAUNCH("l1_place", l1_place_kernel, L.chunks, kBlock, 5 * sizeof(uint32_t) * geo.nblk,
              stream, n, order, rects, geo, bcopy, mcopy, cap, L.chunks, u32(L.lb1), blk_off,
              sub_off, slice_off, hdr, pairs, tile_total);
  ABCD_LAUNCH("l2_count", l2_count_kernel, kCountGrid, 64 * kSlice, 0, stream, pairs, geo, sub_off,
              slice_off, blk_off, hdr, c2, slice_tot, u32(L.blk_done), tile_total, tile_off,
              tile_ranges);
  ABCD_LAUNCH("l2_scatter", l2_scatter_kernel, kScatterGrid, kBlock,
              tile_order ? (size_t)((ntiles + 3) & ~3) : 0u, stream, pairs, depth, geo, sub_off,
              slice_off, blk_off, c2, slice_tot, tile_off, hdr, values_sorted,
              reinterpret_cast<unsigned long long*>(keys_sorted), tile_total, tile_order);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd

// schedule.h -- the stable bucket sort of tiles by decreasing quarter octave
// of a work estimate (heaviest first), shared by the backward's schedule
// (schedule.hip), the forward's tile order made at the end of binning, and
// the one-workgroup binning of small active blocks.
#pragma once

#include "abcd_internal.h"

namespace abcd {
namespace {

constexpr int kOrderThreads = 1024;
constexpr int kOrderWaves = kOrderThreads / 64;
constexpr int kBuckets = 129;  // 4 per leading-zero count of the work, 128 for no work
constexpr int kNone = 255;     // no tile (matches no bucket)

// Heavier work, smaller bucket: 4 lz + (3 - the two bits after the leading one).
__device__ __forceinline__ int bucket_of(uint32_t work) {
  if (!work) return 128;
  const int lz = __clz(work);
  const uint32_t sub = lz < 31 ? (work << (lz + 1)) >> 30 : 0u;
  return 4 * lz + 3 - (int)sub;
}

// Lanes of the calling wave holding the same bucket as this lane (buckets
// below 256; kNone never matches a real bucket).
__device__ __forceinline__ uint64_t match_bucket(int key) {
  uint64_t peers = __ballot(1);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return peers;
}

// Exclusive scan of s_base[0, kBuckets) in place by the first wave.
__device__ __forceinline__ void scan_buckets(uint32_t* s_base) {
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    uint32_t carry = 0;
    for (int b0 = 0; b0 < kBuckets; b0 += 64) {
      const uint32_t c = b0 + l < kBuckets ? s_base[b0 + l] : 0u;
      uint32_t inc = c;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = (uint32_t)__shfl_up((int)inc, d, 64);
        if (l >= d) inc += y;
      }
      if (b0 + l < kBuckets) s_base[b0 + l] = carry + inc - c;
      carry += (uint32_t)__shfl((int)inc, 63, 64);
    }
  }
}

// The ordering of tiles whose buckets are in s_key (workgroup memory, filled
// before the last barrier), by one workgroup of kThreads threads. Wave w
// takes the tiles of one contiguous range: it counts each bucket in the
// range (LDS atomics), the counts of all waves then give each wave its first
// slot in every bucket (buckets in order, waves in order within a bucket),
// and a second walk, 64 tiles at a time, places each tile at that slot plus
// its rank among the range's earlier tiles of its bucket (ballot match plus
// a running count). s_order (may be NULL): the order also into workgroup
// memory, as 16-bit tile indices.
template <int kThreads = kOrderThreads>
__device__ __forceinline__ void order_keyed(int ntiles, const uint8_t* s_key,
                                            uint32_t* __restrict__ order, uint16_t* s_order) {
  constexpr int kWaves = kThreads / 64;
  static_assert(kThreads >= kBuckets, "a thread per bucket");
  __shared__ uint32_t s_base[kBuckets];
  __shared__ uint32_t s_wc[kWaves][kBuckets];  // per wave counts, then first slots
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const uint64_t below = (1ull << l) - 1ull;
  for (int i = tid; i < kWaves * kBuckets; i += kThreads) (&s_wc[0][0])[i] = 0;
  __syncthreads();
  const int per = (ntiles + kWaves - 1) / kWaves;
  const int t0 = min(ntiles, w * per), t1 = min(ntiles, t0 + per);
  for (int t = t0 + l; t < t1; t += 64) atomicAdd(&s_wc[w][s_key[t]], 1u);
  __syncthreads();
  if (tid < kBuckets) {
    uint32_t tot = 0;
    for (int v = 0; v < kWaves; ++v) tot += s_wc[v][tid];
    s_base[tid] = tot;
  }
  __syncthreads();
  scan_buckets(s_base);
  __syncthreads();
  if (tid < kBuckets) {  // first slot of each wave in the bucket
    uint32_t run = s_base[tid];
    for (int v = 0; v < kWaves; ++v) {
      const uint32_t c = s_wc[v][tid];
      s_wc[v][tid] = run;
      run += c;
    }
  }
  __syncthreads();
  for (int tb = t0; tb < t1; tb += 64) {
    const int t = tb + l;
    const int key = t < t1 ? s_key[t] : kNone;
    const uint64_t peers = match_bucket(key);
    if (key != kNone) {
      const uint32_t pos = s_wc[w][key] + __popcll(peers & below);
      order[pos] = (uint32_t)t;
      if (s_order) s_order[pos] = (uint16_t)t;
      if ((peers & below) == 0) s_wc[w][key] += (uint32_t)__popcll(peers);
    }
  }
  __syncthreads();
}

// The ordering of tiles by the bucket of work[t]; s_key is workgroup memory
// of ABCD_MAX_TILES bytes.
__device__ __forceinline__ void order_tiles(int ntiles, const uint32_t* __restrict__ work,
                                            uint32_t* __restrict__ order, uint8_t* s_key) {
  // all loads in flight at once
#pragma unroll 8
  for (int t = threadIdx.x; t < ntiles; t += kOrderThreads) s_key[t] = (uint8_t)bucket_of(work[t]);
  __syncthreads();
  order_keyed(ntiles, s_key, order, nullptr);
}

}  // namespace
}  // namespace abcd

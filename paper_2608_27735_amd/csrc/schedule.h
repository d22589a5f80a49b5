// schedule.h -- the stable bucket sort of tiles by decreasing quarter octave
// of a work estimate (heaviest first), shared by the tile-order kernels of
// schedule.hip and the one-workgroup binning of small active blocks.
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

// The ordering itself, by one workgroup of kOrderThreads threads; s_key is
// workgroup memory of ABCD_MAX_TILES bytes.
__device__ __forceinline__ void order_tiles(int ntiles, const uint32_t* __restrict__ work,
                                            uint32_t* __restrict__ order, uint8_t* s_key) {
  __shared__ uint32_t s_base[kBuckets];
  __shared__ uint32_t s_wc[kOrderWaves][kBuckets];  // per wave counts, then exclusive offsets
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const uint64_t below = (1ull << l) - 1ull;
  if (tid < kBuckets) s_base[tid] = 0;
  // all loads in flight at once; buckets kept in LDS for both passes
#pragma unroll 8
  for (int t = tid; t < ntiles; t += kOrderThreads) s_key[t] = (uint8_t)bucket_of(work[t]);
  __syncthreads();
  // bucket totals: the first lane of each group of equal buckets adds the group
  for (int t0 = 0; t0 < ntiles; t0 += kOrderThreads) {
    const int t = t0 + tid;
    const int key = t < ntiles ? s_key[t] : kNone;
    const uint64_t peers = match_bucket(key);
    if (key != kNone && (peers & below) == 0) atomicAdd(&s_base[key], (uint32_t)__popcll(peers));
  }
  __syncthreads();
  scan_buckets(s_base);
  // stable placement, one chunk of tiles at a time
  for (int t0 = 0; t0 < ntiles; t0 += kOrderThreads) {
    for (int i = tid; i < kOrderWaves * kBuckets; i += kOrderThreads) (&s_wc[0][0])[i] = 0;
    __syncthreads();
    const int t = t0 + tid;
    const int key = t < ntiles ? s_key[t] : kNone;
    const uint64_t peers = match_bucket(key);
    if (key != kNone && (peers & below) == 0) s_wc[w][key] = (uint32_t)__popcll(peers);
    __syncthreads();
    if (tid < kBuckets) {  // exclusive offsets over the waves; advance the bucket base
      uint32_t run = s_base[tid];
      for (int v = 0; v < kOrderWaves; ++v) {
        const uint32_t c = s_wc[v][tid];
        s_wc[v][tid] = run;
        run += c;
      }
      s_base[tid] = run;
    }
    __syncthreads();
    if (key != kNone) order[s_wc[w][key] + __popcll(peers & below)] = (uint32_t)t;
    __syncthreads();
  }
}

}  // namespace
}  // namespace abcd

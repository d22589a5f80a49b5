// render_bwd.hip -- backward of the tile blend (paper, Method section:
// gradients reach the active parameters only).
//
// The backward walks each pixel's list back to front from its last blended
// entry, reduces each Gaussian's 9 screen-space gradients across the wave
// with cross-lane adds, combines the 4 waves in LDS and issues one global
// fp32 atomic per Gaussian and field per tile.
#include "blend.h"

namespace abcd {
namespace {

// DPP lane move inside the wave (all rows and banks enabled; every control
// used here reads a lane of the same row, so bound_ctrl never applies, and
// setting it lets the move fold into the add that consumes it).
template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xF, 0xF, true));
}

// Wave64 sum of nine values at once. Values 0-7 go through a butterfly that
// halves the set at each cross-row step without selects: v_permlane32_swap
// (v_permlane16_swap) of two registers leaves one value's upper-half (odd-row)
// partner in the other register, so the sum of the two results holds value
// 2q in the lower half (even rows) and 2q + 1 in the upper half (odd rows).
// Two such steps leave two registers, folded across lane bit 3 with one
// keep/send select pair, and the 8-lane groups finish with three DPP adds
// (quad xor 1, quad xor 2, row rotate 4). Value 8 is summed by DPP adds
// within rows and two row-broadcast adds. About 20 VALU instructions. On return each lane l with (l & 7) >= 4 holds the wave total
// of value sum9_slot(l) in `lo`, and lanes 48-63 the total of value 8 in `v8`.
struct Sum9 {
  float lo, v8;
};
__device__ __forceinline__ Sum9 wave_sum9(const float (&g)[9], int lane) {
  float a[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_int(g[2 * q]),
                                                    __float_as_int(g[2 * q + 1]), false, false);
    a[q] = __int_as_float(p[0]) + __int_as_float(p[1]);
  }
  float b[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_int(a[2 * q]),
                                                    __float_as_int(a[2 * q + 1]), false, false);
    b[q] = __int_as_float(p[0]) + __int_as_float(p[1]);
  }
  const bool b3 = lane & 8;
  float c = (b3 ? b[1] : b[0]) + dpp_mov<0x128>(b3 ? b[0] : b[1]);  // row rotate 8
  c += dpp_mov<0xB1>(c);   // quad [1,0,3,2]
  c += dpp_mov<0x4E>(c);   // quad [2,3,0,1]
  c += dpp_mov<0x124>(c);  // row rotate 4 (lane l reads l - 4): lanes with (l & 7) >= 4
                           // hold the 8-lane sum
  // value 8: row sums by DPP adds (every lane of a row ends with its row's
  // sum), then two row-broadcast adds over all rows: lane 15 of each row into
  // the next (row 3 now holds r2 + r3, row 1 r0 + r1), then lane 31 into rows
  // 2 and 3, so lanes 48-63 hold the wave total (the other rows hold partial
  // sums, which are not used)
  float v8 = g[8];
  v8 += dpp_mov<0xB1>(v8);   // quad [1,0,3,2]
  v8 += dpp_mov<0x4E>(v8);   // quad [2,3,0,1]
  v8 += dpp_mov<0x124>(v8);  // row rotate 4
  v8 += dpp_mov<0x128>(v8);  // row rotate 8
  v8 += dpp_mov<0x142>(v8);  // row broadcast 15
  v8 += dpp_mov<0x143>(v8);  // row broadcast 31
  return Sum9{c, v8};
}

// Which of the values 0-7 lane l holds in Sum9::lo: bit 3 of l picks the
// group of four, bit 4 the pair, bit 5 the member.
__device__ __forceinline__ int sum9_slot(int l) {
  return 4 * ((l >> 3) & 1) + 2 * ((l >> 4) & 1) + ((l >> 5) & 1);
}

// One work item of the backward: list positions [lo, hi) of `tile`, chunk j
// of a split tile (lo = j ch) or the whole walk (j = 0, hi = 2^32 - 1). Each
// pixel walks the positions below its walk length back to front, starting
// from its final state in its last chunk and from the forward's checkpoint at
// hi otherwise.
__device__ __forceinline__ void bwd_item(
    const BlendConsts& k, int tile, uint32_t j, const uint32_t* __restrict__ tile_ranges,
    const uint32_t* __restrict__ values, const float2* __restrict__ means2d,
    const float4* __restrict__ conic_opacity, const float* __restrict__ rgb,
    const float4* __restrict__ F, const float4* __restrict__ B, const float* __restrict__ final_T,
    const uint32_t* __restrict__ last, const float4* __restrict__ dL_dout, float* __restrict__ g2d,
    int64_t gs, const SplitLayout& sp) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float4 s_gc[256];  // a, b, c (conic), colour b
  __shared__ int s_pos[256];
  __shared__ uint32_t s_g[256];
  __shared__ float s_acc[9][256];  // field-major: [field][staged entry]
  __shared__ __align__(4) uint8_t s_idx[4][256];  // per wave: staged slots reaching its rows
  __shared__ int s_wcnt[5][4];
  __shared__ uint32_t s_max;
  const int tid = threadIdx.x;
  const int px = (tile % k.ntx) * kTile + (tid & 15);
  const int py = (tile / k.ntx) * kTile + (tid >> 4);
  const bool inside = px < k.width && py < k.height;
  const TileBox box = tile_box(k, tile);
  const uint32_t start = tile_ranges[2 * tile];
  // chunk bounds and checkpoint slots (a tile the forward did not split is
  // one item; all of this is uniform)
  uint32_t lo = 0, hi = 0xFFFFFFFFu, slot_hi = kNoSlot, slot_fin = kNoSlot;
  if (sp.ckpt) {
    const uint32_t* so = sp.slot_of + (size_t)tile * kMaxChunks;
    const uint32_t fin = so[0];
    if (fin < sp.nslots && j < kMaxChunks) {
      lo = j * (uint32_t)sp.ch;
      hi = chunk_hi(j, (uint32_t)sp.ch);
      slot_fin = fin;
      if (j + 1 < kMaxChunks && so[j + 1] < sp.nslots) slot_hi = so[j + 1];
    } else if (j != 0) {
      return;  // not an item of this split
    }
  }
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  float T = 1.0f, gcr = 0, gcg = 0, gcb = 0, gT = 0;
  uint32_t lastp = 0;
  float Tfin = 1.0f;
  // RG = sum over channels of gc_ch R_ch, where R is the colour accumulated
  // behind the current entry (normalised by its transmittance): the
  // alpha-derivative needs R only through this sum.
  float RG = 0.0f;
  __syncthreads();  // the previous item is done with the shared arrays
  if (tid == 0) s_max = 0;
  __syncthreads();
  if (inside) {
    const int64_t p = (int64_t)py * k.width + px;
    T = final_T[p];
    Tfin = T;
    lastp = last[p];
    const float4 G = dL_dout[p];
    const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
    const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
    const float s = 1.0f - f.w;
    gcr = s * G.x;
    gcg = s * G.y;
    gcb = s * G.z;
    gT = s * (G.x * bb.x + G.y * bb.y + G.z * bb.z - G.w * (1.0f - bb.w));
    if (lastp > hi && slot_hi != kNoSlot) {  // crossed hi: its slot was taken
      // the walk goes on past this chunk: start from the forward's state at
      // hi; the colour behind is what the rest of the walk added
      const float4 c = sp.ckpt[(size_t)slot_hi * 256 + tid];
      const float4 e = sp.ckpt[(size_t)slot_fin * 256 + tid];
      T = c.x;
      RG = (gcr * (e.y - c.y) + gcg * (e.z - c.z) + gcb * (e.w - c.w)) / c.x;
    }
    const uint32_t mine = min(lastp, hi);
    if (mine > lo) atomicMax(&s_max, mine);
  }
  __syncthreads();
  const uint32_t nent = __builtin_amdgcn_readfirstlane(s_max);  // end of this item's walk
  // d out / d T_final enters every entry's alpha-derivative as T_final g_T / (1 - alpha)
  const float TgT = Tfin * gT;
  // lanes 4, 12, ..., 60 add values 0-7 of an entry, lane 48 value 8
  const int lane = tid & 63;
  const bool adder = (lane & 7) == 4 || lane == 48;
  const int slot = lane == 48 ? 8 : sum9_slot(lane);
  float* const acc_lane = s_acc[slot];  // this lane's field, indexed by staged entry
  uint32_t wml = lastp;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) wml = max(wml, (uint32_t)__shfl_xor((int)wml, off, 64));
  wml = __builtin_amdgcn_readfirstlane(wml);  // uniform, so its tests compile to scalar branches
  // entry j of a batch is list position bend - 1 - j (back to front)
  const uint32_t bstop = start + lo;
  uint32_t bend = nent > lo ? start + nent : bstop;
  // Loads run two batches ahead of use, as in the forward: positions below
  // bstop read the entry at bstop (valid == false), so every load is
  // unconditional and in bounds.
  Rec rec{};
  uint32_t gid_next = 0;
  if (bend > bstop) {  // uniform
    const uint32_t b1 = bend - min(256u, bend - bstop);  // end of the next batch
    const uint32_t p0 = bend - 1 - tid, p1 = b1 - 1 - tid;
    const uint32_t gid0 = values[(uint32_t)tid < bend - bstop ? p0 : bstop];
    gid_next = values[(uint32_t)tid < b1 - bstop ? p1 : bstop];
    rec = gather_rec(gid0, (uint32_t)tid < bend - bstop, means2d, conic_opacity, rgb);
  }
  while (bend > bstop) {
    const uint32_t bbeg = bend - min(256u, bend - bstop);
    __syncthreads();
    const float3 cn = conic_of(rec.co);
    // each wave walks only the staged entries whose ellipse reaches its four
    // pixel rows: the others contribute nothing to any of its pixels
    const uint32_t rows =
        rec.valid ? splat_rows(rec.m.x, rec.m.y, cn.x, cn.y, cn.z, rec.co.w, k.alpha_min, box) : 0u;
    const bool keep = rows != 0u;
    int pos, wcnt;
    const int cnt = compact_rows(keep, rows, s_wcnt, s_idx, pos, wcnt);
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_gc[pos] = make_float4(cn.x, cn.y, cn.z, rec.b);
      s_pos[pos] = (int)(bend - 1 - tid - start);
      s_g[pos] = rec.gid;
#pragma unroll
      for (int q = 0; q < 9; ++q) s_acc[q][pos] = 0.0f;
    }
    __syncthreads();
    {
      // gathers of the next batch (ending at bbeg) and list values of the one
      // after (ending at b2) overlap the walk of this one
      const uint32_t b2 = bbeg - min(256u, bbeg - bstop);
      const uint32_t gid_after = values[(uint32_t)tid < b2 - bstop ? b2 - 1 - tid : bstop];
      rec = gather_rec(gid_next, (uint32_t)tid < bbeg - bstop, means2d, conic_opacity, rgb);
      gid_next = gid_after;
    }
    // Entries are read from LDS kGroup at a time, all reads issued before the
    // first is used, so the LDS latency is paid once per group.
    // The wave's list of staged slots, kBwdGroup at a time; slots past its end
    // hold stale bytes, which still index the staged arrays.
    static_assert(kBwdGroup == 4, "slot indices are read four at a time");
    const uint32_t* my_idx = reinterpret_cast<const uint32_t*>(s_idx[tid >> 6]);
    for (int j0 = 0; j0 < wcnt; j0 += kBwdGroup) {
    float4 gav[kBwdGroup], gbv[kBwdGroup];
    float cbv[kBwdGroup];  // colour b (the conic in s_gc is needed only at the flush)
    uint32_t kkv[kBwdGroup];
    const uint32_t iw = __builtin_amdgcn_readfirstlane(my_idx[j0 / 4]);  // four slots (uniform)
#pragma unroll
    for (int i = 0; i < kBwdGroup; ++i) {
      const int j = (int)((iw >> (8 * i)) & 255u);
      gav[i] = s_ga[j];
      gbv[i] = s_gb[j];
      cbv[i] = s_gc[j].w;
      kkv[i] = (uint32_t)s_pos[j];
    }
    // keep the group's reads ahead of the arithmetic (the compiler would
    // otherwise sink each read into the branch that uses it)
#pragma unroll
    for (int i = 0; i < kBwdGroup; ++i)
      asm volatile("" ::"v"(gav[i].x), "v"(gav[i].y), "v"(gav[i].z), "v"(gav[i].w), "v"(gbv[i].x),
                   "v"(gbv[i].y), "v"(gbv[i].z), "v"(gbv[i].w), "v"(cbv[i]));
#pragma unroll
    for (int i = 0; i < kBwdGroup; ++i) {
      if (j0 + i >= wcnt) break;  // wave-uniform
      const int j = (int)((iw >> (8 * i)) & 255u);  // staged slot (uniform)
      const uint32_t kk = __builtin_amdgcn_readfirstlane(kkv[i]);
      const float4 ga = gav[i], gb = gbv[i];
      if (kk >= wml) continue;  // wave-uniform: no pixel of this wave reaches entry kk
      const float dx = fx - ga.x, dy = fy - ga.y;
      const AlphaEval ae = eval_alpha(dx, dy, ga.z, ga.w, gb.x, gb.y, k.alpha_min, k.alpha_max);
      const bool contrib = kk < lastp && !ae.skip;
      if (!__ballot(contrib)) continue;  // wave-uniform
      // Branch-free per lane: a lane that does not blend this entry takes
      // alpha = 0, which leaves T and R unchanged, and a zero mask on the
      // alpha-derivative terms.
      const float a = contrib ? (ae.clamped ? k.alpha_max : ae.raw) : 0.0f;
      const float om = 1.0f - a;
      const float iom = __builtin_amdgcn_rcpf(om);  // om >= 1 - alpha_max > 0
      const float Tk = T * iom;
      const float wgt = a * Tk;
      float gr[9];
      gr[6] = wgt * gcr;
      gr[7] = wgt * gcg;
      gr[8] = wgt * gcb;
      const float CG = gb.z * gcr + gb.w * gcg + cbv[i] * gcb;
      const float dLda = Tk * (CG - RG) - iom * TgT;
      RG = a * CG + om * RG;
      T = Tk;
      const float dm = (contrib && !ae.clamped) ? dLda : 0.0f;
      const float gp = a * dm;
      // first and second moments of gp over the pixels; the conic and the
      // constant factors are applied once per entry at the flush
      const float q = gp * dx, r = gp * dy;
      gr[0] = q;
      gr[1] = r;
      gr[2] = q * dx;
      gr[3] = q * dy;
      gr[4] = r * dy;
      gr[5] = ae.e * dm;
      const Sum9 v = wave_sum9(gr, lane);
      float out = lane == 48 ? v.v8 : v.lo;
      asm volatile("" : "+v"(out));  // the last folds stay outside the branch (DPP add)
      if (adder) atomicAdd(acc_lane + j, out);
    }
    }
    __syncthreads();
    if (tid < cnt) {
      // moments -> dL/d(u, v, a, b, c): with q = dL/dpower * (dx, dy),
      // d power / d(u, v) = (a dx + b dy, b dx + c dy), d power / d(a, b, c)
      // = (-dx^2 / 2, -dx dy, -dy^2 / 2)
      const float4 co = s_gc[tid];
      float g[9];
#pragma unroll
      for (int q = 0; q < 9; ++q) g[q] = s_acc[q][tid];
      const float mx = g[0], my = g[1];
      g[0] = co.x * mx + co.y * my;
      g[1] = co.y * mx + co.z * my;
      g[2] = -0.5f * g[2];
      g[3] = -g[3];
      g[4] = -0.5f * g[4];
      float* dst = g2d + s_g[tid];
#pragma unroll
      for (int q = 0; q < 9; ++q)
        if (g[q] != 0.0f) atomicAdd(dst + q * gs, g[q]);
    }
    bend = bbeg;
  }
}

// Persistent workgroups take work items, heaviest first, from a queue until
// it is empty (every workgroup reaches the end of the queue and exits).
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void render_bwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    const float* __restrict__ final_T, const uint32_t* __restrict__ last,
    const float4* __restrict__ dL_dout, float* __restrict__ g2d, int64_t gs,
    const uint2* __restrict__ items,
    uint32_t* __restrict__ queue, uint32_t max_items, SplitLayout sp) {
  __shared__ uint2 s_item;
  const uint32_t n_items = min(queue[0], max_items);
  // Atomic adds to one address are serialised, and light items at the end
  // are taken faster than one counter can serve them. So item i belongs to
  // queue i mod nq (nq = kQueues, fewer for a smaller grid), each queue
  // heaviest first, and workgroup b takes from queue b mod nq (one per XCD,
  // which take workgroups round robin). The first item of workgroup b is item
  // b, taken without an atomic; later ones come from the queue's counter.
  const uint32_t nq = min(gridDim.x, (uint32_t)kQueues);
  const uint32_t q = blockIdx.x % nq;
  const uint32_t gq = (gridDim.x - q + nq - 1) / nq;  // workgroups of queue q
  bool first = true;
  for (;;) {
    if (threadIdx.x == 0) {
      const uint32_t r =
          first ? blockIdx.x / nq : gq + atomicAdd(&queue[kQueueStride * q + 1], 1u);
      const uint64_t i = (uint64_t)q + (uint64_t)nq * r;
      s_item = i < n_items ? items[i] : make_uint2(kNoSlot, 0u);
    }
    first = false;
    __syncthreads();
    const uint2 it = s_item;
    __syncthreads();
    if (it.x == kNoSlot) break;
    if (it.x < (uint32_t)k.ntiles)
      bwd_item(k, (int)it.x, it.y, tile_ranges, values, means2d, conic_opacity, rgb, F, B,
               final_T, last, dL_dout, g2d, gs, sp);
  }
}

// Small frames (few tiles, no split): one workgroup per tile in raster order,
// without the schedule's two launches (the launch-bound regime of small
// active partitions).
constexpr int kDirectTiles = 1024;

__global__ __launch_bounds__(256) void render_bwd_direct_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    const float* __restrict__ final_T, const uint32_t* __restrict__ last,
    const float4* __restrict__ dL_dout, float* __restrict__ g2d, int64_t gs) {
  bwd_item(k, (int)blockIdx.x, 0u, tile_ranges, values, means2d, conic_opacity, rgb, F, B, final_T,
           last, dL_dout, g2d, gs, SplitLayout{});
}

// Sums of nine values over each 16-lane row, by a butterfly over lane bits 3
// (row rotate 8), 2 (half-row mirror, which pairs lanes whose bit 2 differs),
// 1 and 0 (quad permutes): each step halves values 0-7 with one select pair
// and one DPP add. On return lane c of a row holds the row total of value
// rowsum9_slot(c), and every lane the total of value 8 in v8.
__device__ __forceinline__ float row_sum9(const float (&g)[9], int c, float& v8) {
  const bool b3 = c & 8, b2 = c & 4, b1 = c & 2;
  float h[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    h[i] = (b3 ? g[2 * i + 1] : g[2 * i]) + dpp_mov<0x128>(b3 ? g[2 * i] : g[2 * i + 1]);
  const float k0 = (b2 ? h[1] : h[0]) + dpp_mov<0x141>(b2 ? h[0] : h[1]);
  const float k1 = (b2 ? h[3] : h[2]) + dpp_mov<0x141>(b2 ? h[2] : h[3]);
  float m = (b1 ? k1 : k0) + dpp_mov<0x4E>(b1 ? k0 : k1);
  m += dpp_mov<0xB1>(m);
  v8 = g[8];
  v8 += dpp_mov<0x128>(v8);
  v8 += dpp_mov<0x141>(v8);
  v8 += dpp_mov<0x4E>(v8);
  v8 += dpp_mov<0xB1>(v8);
  return m;
}
__device__ __forceinline__ int rowsum9_slot(int c) {
  return 4 * ((c >> 1) & 1) + 2 * ((c >> 2) & 1) + ((c >> 3) & 1);
}

// Small frames, where one workgroup per tile leaves most of the chip idle and
// the longest list sets the launch's length: four workgroups per tile (rows
// 4q .. 4q + 3 for quarter q), one pixel row per wave, and four list entries
// per step of a wave. Lane l holds column l & 15 of the wave's row and entry
// l >> 4 of the step (entry 0 the backmost); the four copies of a pixel's
// state stay identical. Within a step the pixel's back-to-front recurrences
// over the four entries run as scans over lane bits 4 and 5: the
// transmittance before each entry is the running one times a prefix product
// of 1 / (1 - alpha), and the colour blended behind it a prefix sum S of
// alpha T (c . g), not normalised by the transmittance, so that the
// alpha-derivative is T (c . g) - (S + T_final g_T) / (1 - alpha).

__global__ __launch_bounds__(256) void render_bwd_rows_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    const float* __restrict__ final_T, const uint32_t* __restrict__ last,
    const float4* __restrict__ dL_dout, float* __restrict__ g2d, int64_t gs) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float4 s_gc[256];  // a, b, c (conic), colour b
  __shared__ int s_pos[256];
  __shared__ uint32_t s_g[256];
  __shared__ float s_acc[9][256];  // field-major: [field][staged entry]
  __shared__ __align__(4) uint8_t s_idx[4][256];  // per wave: staged slots reaching its row
  __shared__ int s_wcnt[5][4];
  __shared__ uint32_t s_max;
  const int tile = (int)(blockIdx.x >> 2), quarter = (int)(blockIdx.x & 3);
  const int tid = threadIdx.x, lane = tid & 63, col = lane & 15, e = lane >> 4;
  const int px = (tile % k.ntx) * kTile + col;
  const int py = (tile / k.ntx) * kTile + 4 * quarter + (tid >> 6);
  const bool inside = px < k.width && py < k.height;
  const TileBox box = tile_box(k, tile);
  const uint32_t start = tile_ranges[2 * tile];
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  float T = 1.0f, gcr = 0, gcg = 0, gcb = 0, gT = 0;
  uint32_t lastp = 0;
  if (tid == 0) s_max = 0;
  __syncthreads();
  if (inside) {
    const int64_t p = (int64_t)py * k.width + px;
    T = final_T[p];
    lastp = last[p];
    const float4 G = dL_dout[p];
    const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
    const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
    const float s = 1.0f - f.w;
    gcr = s * G.x;
    gcg = s * G.y;
    gcb = s * G.z;
    gT = s * (G.x * bb.x + G.y * bb.y + G.z * bb.z - G.w * (1.0f - bb.w));
    if (lastp > 0u) atomicMax(&s_max, lastp);
  }
  __syncthreads();
  const uint32_t nent = __builtin_amdgcn_readfirstlane(s_max);  // end of the quarter's walk
  const float TgT = T * gT;  // T is the final transmittance here
  float S = 0.0f;            // colour behind the step (sum of alpha T (c . g))
  uint32_t wml = lastp;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) wml = max(wml, (uint32_t)__shfl_xor((int)wml, off, 64));
  wml = __builtin_amdgcn_readfirstlane(wml);
  const bool odd = lane & 16, high = lane & 32;
  const bool adder = (col & 1) == 0 || col == 1;
  const int slot = col == 1 ? 8 : rowsum9_slot(col);
  const uint32_t bstop = start;
  uint32_t bend = start + nent;
  Rec rec{};
  uint32_t gid_next = 0;
  if (bend > bstop) {  // uniform
    const uint32_t b1 = bend - min(256u, bend - bstop);
    const uint32_t p0 = bend - 1 - tid, p1 = b1 - 1 - tid;
    const uint32_t gid0 = values[(uint32_t)tid < bend - bstop ? p0 : bstop];
    gid_next = values[(uint32_t)tid < b1 - bstop ? p1 : bstop];
    rec = gather_rec(gid0, (uint32_t)tid < bend - bstop, means2d, conic_opacity, rgb);
  }
  while (bend > bstop) {
    const uint32_t bbeg = bend - min(256u, bend - bstop);
    __syncthreads();
    const float3 cn = conic_of(rec.co);
    const uint32_t rows = rec.valid ? splat_rows_single(rec.m.x, rec.m.y, cn.x, cn.y, cn.z,
                                                        rec.co.w, k.alpha_min, box, 4 * quarter)
                                    : 0u;
    const bool keep = rows != 0u;
    int pos, wcnt;
    const int cnt = compact_rows(keep, rows, s_wcnt, s_idx, pos, wcnt);
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_gc[pos] = make_float4(cn.x, cn.y, cn.z, rec.b);
      s_pos[pos] = (int)(bend - 1 - tid - start);
      s_g[pos] = rec.gid;
#pragma unroll
      for (int q = 0; q < 9; ++q) s_acc[q][pos] = 0.0f;
    }
    __syncthreads();
    {
      const uint32_t b2 = bbeg - min(256u, bbeg - bstop);
      const uint32_t gid_after = values[(uint32_t)tid < b2 - bstop ? b2 - 1 - tid : bstop];
      rec = gather_rec(gid_next, (uint32_t)tid < bbeg - bstop, means2d, conic_opacity, rgb);
      gid_next = gid_after;
    }
    // slots past the end of the wave's list hold stale bytes: they still index
    // the staged arrays, and their lanes take part in nothing below
    const uint8_t* my_idx = s_idx[tid >> 6];
    for (int j0 = 0; j0 < wcnt; j0 += 4) {
      const bool valid = j0 + e < wcnt;
      const int j = my_idx[j0 + e];
      const float4 ga = s_ga[j], gb = s_gb[j];
      const float cb = s_gc[j].w;
      const uint32_t kk = (uint32_t)s_pos[j];
      if (!__ballot(valid && kk < wml)) continue;  // wave-uniform
      const float dx = fx - ga.x, dy = fy - ga.y;
      const AlphaEval ae = eval_alpha(dx, dy, ga.z, ga.w, gb.x, gb.y, k.alpha_min, k.alpha_max);
      const bool contrib = valid && kk < lastp && !ae.skip;
      if (!__ballot(contrib)) continue;  // wave-uniform
      const float a = contrib ? (ae.clamped ? k.alpha_max : ae.raw) : 0.0f;
      const float iom = __builtin_amdgcn_rcpf(1.0f - a);  // 1 - a >= 1 - alpha_max > 0
      // transmittance before each entry: T times the inclusive prefix product
      // of 1 / (1 - alpha) over the step's entries, back to front
      const Swapped p1 = swap_bit4(iom);
      const float t1 = p1.first * p1.second;
      const float in1 = odd ? t1 : iom;
      const Swapped p2 = swap_bit5(t1);
      const float Tk = T * (high ? in1 * p2.first : in1);
      const float ptot = p2.first * p2.second;
      const float CG = gb.z * gcr + gb.w * gcg + cb * gcb;
      const float wgt = a * Tk;
      // colour blended behind each entry within the step: exclusive prefix sum
      const float c0 = contrib ? wgt * CG : 0.0f;
      const Swapped s1 = swap_bit4(c0);
      const float u1 = s1.first + s1.second;
      const float ex1 = odd ? s1.first : 0.0f;
      const Swapped s2 = swap_bit5(u1);
      const float behind = S + (high ? ex1 + s2.first : ex1);
      const float stot = s2.first + s2.second;
      const float dLda = Tk * CG - iom * (behind + TgT);
      T *= ptot;
      S += stot;
      const float dm = (contrib && !ae.clamped) ? dLda : 0.0f;
      const float gp = a * dm;
      const float q = gp * dx, r = gp * dy;
      float gr[9];
      gr[0] = q;
      gr[1] = r;
      gr[2] = q * dx;
      gr[3] = q * dy;
      gr[4] = r * dy;
      gr[5] = ae.e * dm;
      gr[6] = wgt * gcr;
      gr[7] = wgt * gcg;
      gr[8] = wgt * gcb;
      float v8;
      const float m = row_sum9(gr, col, v8);
      float out = col == 1 ? v8 : m;
      asm volatile("" : "+v"(out));  // the last folds stay outside the branch (DPP add)
      if (adder && valid) atomicAdd(&s_acc[slot][j], out);
    }
    __syncthreads();
    if (tid < cnt) {
      const float4 co = s_gc[tid];
      float g[9];
#pragma unroll
      for (int q = 0; q < 9; ++q) g[q] = s_acc[q][tid];
      const float mx = g[0], my = g[1];
      g[0] = co.x * mx + co.y * my;
      g[1] = co.y * mx + co.z * my;
      g[2] = -0.5f * g[2];
      g[3] = -g[3];
      g[4] = -0.5f * g[4];
      float* dst = g2d + s_g[tid];
#pragma unroll
      for (int q = 0; q < 9; ++q)
        if (g[q] != 0.0f) atomicAdd(dst + q * gs, g[q]);
    }
    bend = bbeg;
  }
}

}  // namespace

static_assert(kQueueStride * kQueues == 64 * 8, "queue block of bwd_workspace_bytes");

// g2d (field-major), then the backward's tile work, tile order, work items (when
// not split) and queue.
size_t render_bwd_workspace_bytes(int64_t n) { return bwd_workspace_bytes(n); }

namespace {
// Workgroups of the persistent backward that fit the device at once.
int bwd_resident_blocks() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (cached[dev] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, render_bwd_kernel, kBlock, 0) !=
            hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        per_cu <= 0 || cus <= 0) {
      (void)hipGetLastError();
      return 1024;
    }
    cached[dev] = per_cu * cus;
  }
  return cached[dev];
}
}  // namespace

int32_t launch_render_bwd_pixels(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                                 const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                 const float* means2d, const float* conic_opacity,
                                 const float* rgb, const float* F, const float* B,
                                 const float* final_T, const uint32_t* last,
                                 const float* dL_dout, float* g2d, const SplitLayout& split,
                                 hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  const int64_t g2d_count = 9 * g2d_stride(n);
  if (!split.ckpt && k.ntiles <= kDirectTiles) {
    TRY_STATUS(launch_zero(g2d, g2d_count, stream));
    if (k.ntiles <= kRowsTiles)
      ABCD_LAUNCH("render_bwd", render_bwd_rows_kernel, 4 * k.ntiles, kBlock, 0, stream, k,
                  tile_ranges, values_sorted, reinterpret_cast<const float2*>(means2d),
                  reinterpret_cast<const float4*>(conic_opacity), rgb,
                  reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B), final_T,
                  last, reinterpret_cast<const float4*>(dL_dout), g2d, g2d_stride(n));
    else
      ABCD_LAUNCH("render_bwd", render_bwd_direct_kernel, k.ntiles, kBlock, 0, stream, k,
                  tile_ranges, values_sorted, reinterpret_cast<const float2*>(means2d),
                  reinterpret_cast<const float4*>(conic_opacity), rgb,
                  reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B), final_T,
                  last, reinterpret_cast<const float4*>(dL_dout), g2d, g2d_stride(n));
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  char* tail = reinterpret_cast<char*>(g2d) + bwd_g2d_bytes(n);
  uint32_t* work = reinterpret_cast<uint32_t*>(tail);
  uint32_t* order = work + ABCD_MAX_TILES;
  uint2* own_items = reinterpret_cast<uint2*>(order + ABCD_MAX_TILES);
  uint32_t* queue = reinterpret_cast<uint32_t*>(own_items + ABCD_MAX_TILES);
  uint2* items = split.ckpt ? split.items : own_items;
  const uint32_t max_items =
      (uint32_t)k.ntiles + (split.ckpt ? split.nslots : 0u);
  // each tile's largest walk: from the forward when split, else from `last`
  const uint32_t* walk = work;
  if (split.ckpt)
    walk = split.walk;
  else
    TRY_STATUS(launch_tile_walk(k.width, k.height, last, work, stream));
  // heaviest items first: by the forward's per-chunk estimate when split,
  // else by the walk
  TRY_STATUS(launch_bwd_schedule(k.ntiles, split.ckpt ? split.work : walk, walk, order, split,
                                 items, max_items, queue, g2d, g2d_count, stream));
  const int grid = (int)std::min<int64_t>(bwd_resident_blocks(), max_items);
  ABCD_LAUNCH("render_bwd", render_bwd_kernel, grid, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B), final_T,
              last, reinterpret_cast<const float4*>(dL_dout), g2d, g2d_stride(n), items, queue,
              max_items, split);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd

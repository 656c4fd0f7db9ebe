// Row-owned aggregation over a CSR matrix with a fixed work plan.
//
// Forward (Section 3.2's mean aggregator; Algorithm 1's P_i H):
//     A[v] = (1/d_v) * sum_{u in N(v) ∪ {v}} H_full[u]
// with fresh inner rows and stale boundary rows read from a second buffer.
// Backward (Algorithm 1's P_i^T (...)): the same kernel over the rows of
// P_i^T without a scale (the 1/d_v factor is applied to the GEMM output
// before this pass); output rows [0, n_inner) and [n_inner, n_inner+n_bd)
// go to two different buffers (inner feature gradient, outgoing boundary
// gradient).
//
// Mapping for CDNA4 (8 XCDs, 4 MB L2 each, wave64):
//  * A wave's vector load costs the per-CU texture data path the same time
//    whether or not all 64 lanes are active (measured: ~32 cycles per
//    64 x 16-byte load, about 20 TB/s for the chip on cache-resident rows),
//    so lanes are kept full: the float4 columns of a row are cut into full
//    slices of 64 float4 (S = 8, 4, 2 or 1 per launch) plus one remainder
//    launch of width SL < 64 in which G = 64 / SL lane groups share a wave.
//    Workgroup b works on slice b % S; the hardware deals workgroups to the
//    8 XCDs round robin, so an XCD only ever touches one slice of every row.
//  * The columns of the sparse matrix (the gathered rows) are cut into C
//    chunks of about 8,000 rows, one launch per chunk, so that the rows one
//    launch gathers from stay in the caches while they are reused (cache
//    blocking; C = 1 for short rows, where each gathered row is used only a
//    few times anyway).  Chunk c adds its partial sum to the output in chunk
//    order; the last chunk applies the row scale.
//  * Long runs: one wave owns one work item (a row's run of non-zeros inside
//    a chunk): G = 64 / SL lane groups take non-zeros k, k+1, ..., k+G-1, U
//    of them per group in flight (masked at the row's end), then the groups
//    are added in group order.  Short runs (fewer than G*U non-zeros): each
//    lane group owns its own item, U non-zeros in flight; items are sorted by
//    length, so the groups of a wave finish together.  Both kinds run in
//    one launch (long-run workgroups first).  Column indices are fetched by
//    one load of up to 64 per wave (one per lane) and handed out by
//    v_readlane or lane shuffles, which keeps index fetches off the texture
//    data path.
//  * A row with a run longer than a fixed segment is a split row: all its
//    runs are cut into segments that write partial sums, and one pass after
//    the last chunk adds them in (chunk, segment) order.  No floating-point
//    atomics: results are bitwise reproducible.
#include <cstdlib>

#include "internal.h"

namespace pgcn {

struct AggParams {
  const WorkItem *items;  // long-run items [0, n_long), then short-run items [n_long, n_items)
  int64_t n_items;
  int64_t n_long;
  int64_t long_blocks;    // workgroups of the long-run part (a multiple of slices)
  const int32_t *col;
  int64_t in_split;
  const float *in_lo;
  const float *in_hi;
  int64_t out_split;
  float *out_lo;          // fp32 rows [0, out_split) (final result or running sum)
  float *out_hi;          // fp32 rows [out_split, ...)
  uint16_t *out_bf16;     // bf16 copy of rows [0, out_split) (final chunk only)
  const float *scale;
  int32_t f;              // feature columns (total)
  int32_t c4_off;         // first float4 column of this launch
  int32_t c4_cnt;         // float4 columns of this launch
  int32_t slices;         // S
  int32_t mode;           // AGG_FIRST | AGG_LAST
  int32_t accum_lo;       // rows < out_split add to the output's previous content
  int32_t relu;           // final rows are max(x, 0)
  int64_t ld_in, ld_out, ld_bf16, ld_part;
  float *partials;
  float *send;            // or null: final rows [0, out_split) also to their send rows (stride ld_out)
  const int64_t *send_ptr;
  const int32_t *send_pos;
  const uint32_t *hub_init;  // or null: rows whose bit is set start from their dense-block sum
};

enum { AGG_FIRST = 1, AGG_LAST = 2 };

typedef float agg_f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);  // quiet NaN
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float *out_row(const AggParams &p, int64_t r) {
  if (r < p.out_split) return p.out_lo ? p.out_lo + r * p.ld_out : nullptr;
  return p.out_hi + (r - p.out_split) * p.ld_out;
}

// Combine this chunk's sum of float4 column c4 of row r with the running sum
// (or, with accum_lo, with what an inner row held before the first chunk)
// and store it (scaled, ReLU when asked, padding zeroed, bf16 copy) when this
// is the last chunk.
__device__ __forceinline__ void finish(const AggParams &p, int64_t r, int c4, float4 v) {
  const int c = 4 * c4;
  float *o = out_row(p, r);
  if (!(p.mode & AGG_FIRST) || (p.accum_lo && r < p.out_split) || (p.hub_init && ((p.hub_init[r >> 5] >> (r & 31)) & 1u)))
    v = add4(v, *reinterpret_cast<const float4 *>(o + c));
  if (!(p.mode & AGG_LAST)) {
    *reinterpret_cast<float4 *>(o + c) = v;
    return;
  }
  const float s = p.scale ? p.scale[r] : 1.0f;
  float4 q;
  q.x = (c + 0 < p.f) ? v.x * s : 0.0f;
  q.y = (c + 1 < p.f) ? v.y * s : 0.0f;
  q.z = (c + 2 < p.f) ? v.z * s : 0.0f;
  q.w = (c + 3 < p.f) ? v.w * s : 0.0f;
  if (p.relu) {
    q.x = q.x > 0.f ? q.x : 0.f;
    q.y = q.y > 0.f ? q.y : 0.f;
    q.z = q.z > 0.f ? q.z : 0.f;
    q.w = q.w > 0.f ? q.w : 0.f;
  }
  if (o) *reinterpret_cast<float4 *>(o + c) = q;
  if (p.send && r < p.out_split) {                     // four send slots per round, positions loaded together
    const agg_f32x4 qv = {q.x, q.y, q.z, q.w};
    const int64_t kb = p.send_ptr[r], ke = p.send_ptr[r + 1];
    for (int64_t k = kb; k < ke; k += 4) {
      int32_t pos[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) pos[e] = k + e < ke ? p.send_pos[k + e] : -1;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (pos[e] >= 0)   // read by no kernel of this step: kept out of the caches
          __builtin_nontemporal_store(qv, reinterpret_cast<agg_f32x4 *>(p.send + (int64_t)pos[e] * p.ld_out + c));
    }
  }
  if (p.out_bf16 && r < p.out_split) {
    uint2 w;
    w.x = (uint32_t)f32_to_bf16_rne(q.x) | ((uint32_t)f32_to_bf16_rne(q.y) << 16);
    w.y = (uint32_t)f32_to_bf16_rne(q.z) | ((uint32_t)f32_to_bf16_rne(q.w) << 16);
    *reinterpret_cast<uint2 *>(p.out_bf16 + r * p.ld_bf16 + c) = w;
  }
}

// Short runs: lane group g of a wave owns item n_long + (wave * G + g).
template <int SL, int U>
__device__ __forceinline__ void agg_short(const AggParams &p, int64_t blk) {
  constexpr int G = 64 / SL;
  constexpr int NL = (U + SL - 1) / SL;                 // index loads per step (G > 1)
  const int S = p.slices;
  const int slice = (int)(blk % S);
  const int lane = threadIdx.x % 64, g = lane / SL, j = lane % SL;
  const int64_t item = p.n_long + ((blk / S) * 4 + threadIdx.x / 64) * G + g;
  // a whole lane group leaves together (it is its own shuffle source)
  if (g >= G || item >= p.n_items) return;
  const int cs = slice * SL + j;
  const bool act = cs < p.c4_cnt;
  const int cbase = 4 * (p.c4_off + cs);
  const WorkItem it = p.items[item];
  const int32_t *cols = p.col + it.begin;
  const int len = it.len;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < len; k += U) {
    int32_t c[U];
    if (G == 1) {                                      // one item per wave: lane u loads index u
      const int32_t mine = (lane < U && k + lane < len) ? __builtin_nontemporal_load(cols + k + lane) : -1;
#pragma unroll
      for (int u = 0; u < U; ++u) c[u] = __builtin_amdgcn_readlane(mine, u);
    } else {
      int32_t mine[NL];
#pragma unroll
      for (int t = 0; t < NL; ++t) {
        const int q = k + t * SL + j;
        mine[t] = (t * SL + j < U && q < len) ? __builtin_nontemporal_load(cols + q) : -1;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) c[u] = __shfl(mine[u / SL], g * SL + u % SL);
    }
    float4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float *src = nullptr;
      if (c[u] >= 0) {
        if (c[u] < p.in_split) src = p.in_lo + (int64_t)c[u] * p.ld_in;
        else if (p.in_hi) src = p.in_hi + (int64_t)(c[u] - p.in_split) * p.ld_in;
      }
      x[u] = (act && src) ? *reinterpret_cast<const float4 *>(src + cbase) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc = add4(acc, x[u]);
  }
  if (!act) return;
  if (it.dst >= 0) finish(p, it.dst, p.c4_off + cs, acc);
  else *reinterpret_cast<float4 *>(p.partials + (int64_t)(-it.dst - 1) * p.ld_part + cbase) = acc;
}

// Long runs: one wave owns item (blk / S) * 4 + wave.
template <int SL, int U>
__device__ __forceinline__ void agg_long(const AggParams &p, int64_t blk) {
  constexpr int G = 64 / SL;
  const int S = p.slices;
  const int slice = (int)(blk % S);
  int64_t item = (blk / S) * 4 + threadIdx.x / 64;
  item = __builtin_amdgcn_readfirstlane((int)item);
  if (item >= p.n_long) return;
  const int lane = threadIdx.x % 64, g = lane / SL;
  const int cs = slice * SL + lane % SL;                // float4 column inside this launch
  const bool act = g < G && cs < p.c4_cnt;
  const int gg = g < G ? g : 0;
  const int cbase = 4 * (p.c4_off + cs);
  const WorkItem it = p.items[item];
  const int32_t *cols = p.col + it.begin;
  const int len = it.len;

  // column indices: one load of up to 64 per wave (one per lane), handed out
  // by v_readlane (one lane group) or lane shuffles (several groups)
  constexpr int GU = G * U;                            // non-zeros per step
  constexpr int KB = GU <= 64 ? (64 / GU) * GU : GU;   // non-zeros per index load (G divides 64 if GU > 64)
  constexpr int NB = (KB + 63) / 64;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < len; k0 += KB) {
    int32_t mine[NB];
#pragma unroll
    for (int t = 0; t < NB; ++t) {
      const int q = 64 * t + lane;
      mine[t] = (q < KB && k0 + q < len) ? __builtin_nontemporal_load(cols + k0 + q) : -1;
    }
    const int kn = len - k0 < KB ? len - k0 : KB;
    for (int j = 0; j < kn; j += GU) {
      int32_t c[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (G == 1) c[u] = __builtin_amdgcn_readlane(mine[0], j + u);
        else if (NB == 1) c[u] = __shfl(mine[0], j + u * G + gg);
        else c[u] = __shfl(mine[(u * G) / 64], (u * G) % 64 + gg);    // KB == GU: j == 0
      }
      float4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float *src = nullptr;
        if (c[u] >= 0) {
          if (c[u] < p.in_split) src = p.in_lo + (int64_t)c[u] * p.ld_in;
          else if (p.in_hi) src = p.in_hi + (int64_t)(c[u] - p.in_split) * p.ld_in;
        }
        x[u] = (act && src) ? *reinterpret_cast<const float4 *>(src + cbase) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) acc = add4(acc, x[u]);
    }
  }
  // groups are added in group order (fixed): ((g0 + g1) + g2) + ...
  float4 tot = acc;
#pragma unroll
  for (int q = 1; q < G; ++q) {
    const int from = lane % SL + q * SL;
    tot.x += __shfl(acc.x, from);
    tot.y += __shfl(acc.y, from);
    tot.z += __shfl(acc.z, from);
    tot.w += __shfl(acc.w, from);
  }
  if (g != 0 || cs >= p.c4_cnt) return;
  if (it.dst >= 0) {
    finish(p, it.dst, p.c4_off + cs, tot);
  } else {
    *reinterpret_cast<float4 *>(p.partials + (int64_t)(-it.dst - 1) * p.ld_part + cbase) = tot;
  }
}

// One launch per chunk and column range: the first long_blocks workgroups
// take the long runs, the rest the short runs.
template <int SL, int U>
__global__ __launch_bounds__(256) void agg_kernel(AggParams p) {
  if ((int64_t)blockIdx.x < p.long_blocks) agg_long<SL, U>(p, blockIdx.x);
  else agg_short<SL, U>(p, (int64_t)blockIdx.x - p.long_blocks);
}

// Sum the partial slots of each split row in slot order, then store.
__global__ __launch_bounds__(256) void agg_fixup_kernel(AggParams p, const SplitRow *splits) {
  const SplitRow s = splits[blockIdx.x];
  for (int c4 = p.c4_off + threadIdx.x; c4 < p.c4_off + p.c4_cnt; c4 += blockDim.x) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < s.nslots; ++j)
      acc = add4(acc, *reinterpret_cast<const float4 *>(p.partials + (int64_t)(s.first_slot + j) * p.ld_part + 4 * c4));
    finish(p, s.row, c4, acc);
  }
}

// ------------------------------------------------------------ dense block ---
//
// Block sums on the matrix cores: S[r] = sum over hub columns c of bit(r, c) H[c]
// for the hub rows r.  First hub_split_kernel (four workgroups per tile, two
// columns per thread) writes, per tile of kHubColTile =
// 32 hub columns and per block of 32 features of this launch's float4 slice,
// the tile's gathered rows as three bf16 parts (hi = bf16(x), mid = bf16(x -
// hi), lo = bf16(x - hi - mid): x = hi + mid + lo exactly for normal fp32 x),
// feature-major with the 32 columns contiguous, in exactly the layout the
// MFMA loop reads from LDS (an image of kHubImage bytes).  hub_kernel: a
// workgroup (8 waves) owns kHubRowTile = 512 hub rows (64 per wave), one
// feature block and a range of column tiles; it copies the next image into
// LDS while multiplying the current one (double buffered), several
// workgroups per CU.  v_mfma_f32_32x32x16_bf16 multiplies each part by the
// 0/1 bits (bf16 1.0 or 0, exact) with fp32 accumulation, so the products
// are exact and only the fp32 sums round, as in the gather.  Each fragment of
// a part read from LDS feeds the wave's four 32-row quarters.  The bits of a
// row for a tile are one 32-bit word, stored tile-major so that a wave's 32
// rows load as one contiguous 128-byte access.  Operand layout as in the update GEMMs:
// the feature side is the MFMA's first operand, so lane l holds hub row
// l % 32 (of its quarter) and registers 4q .. 4q+3 hold features
// 8q + 4(l / 32) .. +3 of the block; lane half h supplies columns
// 16 s + 8 h .. +7 of k-step s on both sides.  Column ranges ("groups") write
// partial sums that hub_combine_kernel adds in range order.

typedef float hub_f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 hub_bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int hub_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kHubLds = 40;                  // bf16 per feature row of an image: 32 columns + 8 pad
constexpr int kHubImage = 8192;              // bytes per (tile, feature block): 3 x 32 x 40 bf16 = 7,680, padded
constexpr int kHubFeatBlocks = 8;            // feature blocks of a 64-float4 slice
constexpr int kHubTargetWgs = 512;           // workgroups per launch the column ranges aim at

struct HubParams {
  const int32_t *row_ids;          // [rows]  output row of each hub row (-1: padding)
  const int32_t *col_ids;          // [cols]  gathered row of each hub column (-1: padding)
  const uint32_t *bits;            // [ntiles][rows]
  int32_t rows, ntiles, tiles_per_group, groups, nfb;
  int64_t in_split;
  const float *in_lo, *in_hi;
  int64_t ld_in;
  int32_t c4_off, c4_cnt;          // float4 columns of this pass (at most 64)
  uint16_t *img;                   // [kHubFeatBlocks][ntiles] images of this pass
  float *part;                     // [groups][rows][ld_part] block sums of each column range
  int64_t ld_part;
};

// Column ranges of a pass over nfb feature blocks: about kHubTargetWgs workgroups.
static int hub_groups(const Hub &h, int nfb) {
  const int64_t per = (int64_t)(h.rows / kHubRowTile) * nfb;
  const int64_t g = (kHubTargetWgs + per / 2) / per;
  return (int)std::max<int64_t>(1, std::min<int64_t>(g, h.cols / kHubColTile));
}

__device__ __forceinline__ uint16_t hub_bf16(float x) {
  uint32_t b = __float_as_uint(x);
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}
__device__ __forceinline__ float hub_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Four workgroups per tile (b = 4 tile + quarter): thread (w, l) splits columns
// 8 quarter + 2 w and + 1 of features 4 l .. 4 l + 3.
__global__ __launch_bounds__(256) void hub_split_kernel(HubParams p) {
  const int ct = blockIdx.x >> 2, t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int c0 = 8 * (blockIdx.x & 3) + 2 * wave;
  const bool f4_ok = lane < p.c4_cnt;
  const int cb = 4 * (p.c4_off + lane);
  float4 x2[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int c = p.col_ids[ct * kHubColTile + c0 + e];
    const float *src = nullptr;
    if (c >= 0) {
      if (c < p.in_split) src = p.in_lo + (int64_t)c * p.ld_in;
      else if (p.in_hi) src = p.in_hi + (int64_t)(c - p.in_split) * p.ld_in;
    }
    x2[e] = (f4_ok && src) ? *reinterpret_cast<const float4 *>(src + cb) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // features 4 lane .. 4 lane + 3 all sit in feature block lane / 8, rows 4 (lane % 8) .. +3
  uint16_t *img = p.img + ((int64_t)(lane >> 3) * p.ntiles + ct) * (kHubImage / 2);
#pragma unroll
  for (int fe = 0; fe < 4; ++fe) {
    uint32_t v[3] = {0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float x = fe == 0 ? x2[e].x : fe == 1 ? x2[e].y : fe == 2 ? x2[e].z : x2[e].w;
      const uint16_t hi = hub_bf16(x);
      const float r1 = x - hub_f32(hi);
      const uint16_t mi = hub_bf16(r1);
      const uint16_t lo = hub_bf16(r1 - hub_f32(mi));
      v[0] |= (uint32_t)hi << (16 * e);
      v[1] |= (uint32_t)mi << (16 * e);
      v[2] |= (uint32_t)lo << (16 * e);
    }
    const int fl = 4 * (lane & 7) + fe;
#pragma unroll
    for (int part = 0; part < 3; ++part)
      *reinterpret_cast<uint32_t *>(img + (part * 32 + fl) * kHubLds + c0) = v[part];
  }
}

// Workgroup b: row tile b / (groups nfb), column range (b / nfb) % groups, feature block b % nfb.
__global__ __launch_bounds__(512) void hub_kernel(HubParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t hs[2][kHubImage / 2];       // 16,384 bytes
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int fb = blockIdx.x % p.nfb, g = (blockIdx.x / p.nfb) % p.groups, rt = blockIdx.x / (p.nfb * p.groups);
  const int ct0 = g * p.tiles_per_group;
  const int ct1 = ct0 + p.tiles_per_group < p.ntiles ? ct0 + p.tiles_per_group : p.ntiles;
  const int h = lane >> 5, r32 = lane & 31;
  const int hrow0 = rt * kHubRowTile + wave * 64 + r32;          // this lane's rows: hrow0 + 32 i, i < 2
  const uint16_t *img = p.img + (int64_t)fb * p.ntiles * (kHubImage / 2);

  hub_u32x4 stg;
  uint32_t pat[2];
  auto load = [&](int ct) __attribute__((always_inline)) {
    const hub_u32x4 *src = reinterpret_cast<const hub_u32x4 *>(img + (int64_t)ct * (kHubImage / 2));
    stg = src[t];                                      // 512 threads x 16 bytes: the whole image
#pragma unroll
    for (int i = 0; i < 2; ++i) pat[i] = p.bits[(int64_t)ct * p.rows + hrow0 + 32 * i];
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
    reinterpret_cast<hub_u32x4 *>(hs[buf])[t] = stg;
  };
  auto expand = [](uint32_t byte) __attribute__((always_inline)) {
    hub_u32x4 aw;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      aw[w] = (((byte >> (2 * w)) & 1u) ? 0x3f80u : 0u) | (((byte >> (2 * w + 1)) & 1u) ? 0x3f800000u : 0u);
    return __builtin_bit_cast(hub_bf16x8, aw);
  };

  hub_f32x16 acc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) acc[i] = (hub_f32x16){};
  if (ct0 < ct1) {
    load(ct0);
    store(0);
  }
  __syncthreads();
  for (int ct = ct0; ct < ct1; ++ct) {
    const int cur = (ct - ct0) & 1;
    uint32_t pc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) pc[i] = pat[i];
    if (ct + 1 < ct1) load(ct + 1);
    const uint16_t *tile = hs[cur];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int sh = 16 * st + 8 * h;
      hub_bf16x8 a[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = expand((pc[i] >> sh) & 0xffu);
#pragma unroll
      for (int part = 0; part < 3; ++part) {
        const hub_bf16x8 b = __builtin_bit_cast(
            hub_bf16x8, *reinterpret_cast<const hub_u32x4 *>(tile + (part * 32 + r32) * kHubLds + 16 * st + 8 * h));
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a[i], acc[i], 0, 0, 0);
      }
    }
    if (ct + 1 < ct1) store(cur ^ 1);
    __syncthreads();
  }
  // partial sums of this column range: rows hrow0 + 32 i, features 32 fb + 8 q + 4 h .. +3
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float *dst = p.part + ((int64_t)g * p.rows + hrow0 + 32 * i) * p.ld_part + 4 * p.c4_off + 32 * fb;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = 32 * fb + 8 * q + 4 * h;
      if (f < 4 * p.c4_cnt)
        *reinterpret_cast<float4 *>(dst + 8 * q + 4 * h) =
            make_float4(acc[i][4 * q], acc[i][4 * q + 1], acc[i][4 * q + 2], acc[i][4 * q + 3]);
    }
  }
}

// Start value of every hub row: its block sum (groups added in group order),
// plus, with accum_lo, what an inner row held before.  One wave per hub row.
__global__ __launch_bounds__(256) void hub_combine_kernel(AggParams p, HubParams hp) {
  const int i = blockIdx.x * 4 + threadIdx.x / 64, lane = threadIdx.x % 64;
  if (i >= hp.rows || lane >= p.c4_cnt) return;
  const int r = hp.row_ids[i];
  if (r < 0) return;
  const int c = 4 * (p.c4_off + lane);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int g = 0; g < hp.groups; ++g)
    v = add4(v, *reinterpret_cast<const float4 *>(hp.part + ((int64_t)g * hp.rows + i) * hp.ld_part + c));
  float *o = out_row(p, r);
  if (p.accum_lo && r < p.out_split) v = add4(*reinterpret_cast<const float4 *>(o + c), v);
  *reinterpret_cast<float4 *>(o + c) = v;
}

template <int SL>
static void launch_sl(AggParams p, hipStream_t s) {
  constexpr int U = 8;
  constexpr int G = 64 / SL;
  p.long_blocks = (p.n_long + 3) / 4 * p.slices;
  const int64_t short_blocks = (p.n_items - p.n_long + 4 * G - 1) / (4 * G) * p.slices;
  hipLaunchKernelGGL((agg_kernel<SL, U>), dim3((unsigned)(p.long_blocks + short_blocks)), dim3(256), 0, s, p);
}

static void launch_dispatch(const AggParams &p, int sl, hipStream_t s) {
  switch (sl) {
    case 4: launch_sl<4>(p, s); break;
    case 8: launch_sl<8>(p, s); break;
    case 12: launch_sl<12>(p, s); break;
    case 16: launch_sl<16>(p, s); break;
    case 20: launch_sl<20>(p, s); break;
    case 24: launch_sl<24>(p, s); break;
    case 32: launch_sl<32>(p, s); break;
    case 40: launch_sl<40>(p, s); break;
    case 48: launch_sl<48>(p, s); break;
    default: launch_sl<64>(p, s); break;
  }
}

// First short run of chunk c: whole runs are sorted by decreasing length
// after the split segments (which always take the long-run path).
static int64_t first_short(const Plan &plan, int c, int threshold) {
  int64_t lo = plan.chunk_whole[c], hi = plan.chunk_items[c + 1];
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (plan.items[mid].len >= threshold) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Column launches of a row of f4 float4: full slices of W float4 (W = 64 by
// default; 8, 4, 2 or 1 slices per launch), then the remainder (if any) in one
// launch whose slice width is the smallest supported width that holds it.
struct ColLaunch {
  int off, cnt, S, SL;
};
constexpr int kMaxAggF4 = 31 * 512 + 63;                 // 32 launches at most
static_assert(4 * kMaxAggF4 == PGCN_MAX_WIDTH, "the entry points' width limit is the aggregation's");

static int slice_width() {
  const char *env = std::getenv("PGCN_AGG_SLICE_F4");    // tuning override: 16, 32 or 64
  const int v = env ? std::atoi(env) : 64;
  return (v == 16 || v == 32) ? v : 64;
}

static int col_launches(int f4, ColLaunch *out, int max_out) {
  const int W = slice_width();
  int n = 0;
  const int full = f4 / W * W;
  // full slices in launches of 8, 4, 2 or 1 slices: slice b % S of workgroup b
  // then matches its XCD b % 8
  for (int off = 0; off < full;) {
    int S = 8;
    while (S * W > full - off) S /= 2;
    if (n == max_out) return -1;
    out[n++] = ColLaunch{off, S * W, S, W};
    off += S * W;
  }
  if (f4 > full && n == max_out) return -1;
  const int rem = f4 - full;
  if (rem > 0) {
    static const int widths[] = {4, 8, 12, 16, 20, 24, 32, 40, 48, 64};
    int sl = 64;
    for (int w : widths)
      if (w >= rem) {
        sl = w;
        break;
      }
    out[n++] = ColLaunch{full, rem, 1, sl};
  }
  return n;
}

// Feature blocks of a dense-block pass over cnt float4 columns.
static int hub_nfb(int cnt) { return (4 * cnt + 31) / 32; }

// Rows of dense-block partial sums an aggregation over rows of f floats needs: the most
// that any of its passes uses.
static int64_t hub_sum_rows(const Plan &plan, int64_t f) {
  int64_t n = 0;
  if (plan.hub.rows == 0) return 0;
  ColLaunch cl[128];
  const int ncl = col_launches((int)((f + 3) / 4), cl, 128);
  for (int li = 0; li < ncl; ++li)
    for (int c0 = cl[li].off; c0 < cl[li].off + cl[li].cnt; c0 += 64) {
      const int cnt = std::min(64, cl[li].off + cl[li].cnt - c0);
      n = std::max<int64_t>(n, (int64_t)hub_groups(plan.hub, hub_nfb(cnt)) * plan.hub.rows);
    }
  return n;
}

// [split-row partial slots | dense-block sums of every column range | images of the block's columns]
size_t aggregate_workspace(const Plan &plan, int64_t f) {
  const int64_t ld_part = (f + 3) / 4 * 4;
  const size_t sums = ((size_t)plan.slots + (size_t)hub_sum_rows(plan, f)) * (size_t)ld_part * 4;
  return sums + (size_t)(plan.hub.cols / kHubColTile) * kHubFeatBlocks * (size_t)kHubImage;
}

int launch_aggregate(const AggArgs &a, hipStream_t s) {
  const Plan &plan = *a.plan;
  if (plan.items.empty()) return PGCN_OK;
  AggParams p{};
  const Hub &hub = plan.hub;
  p.col = hub.rows > 0 ? plan.d_col_rest : a.col;     // with a dense block the items index the rest
  p.hub_init = hub.rows > 0 ? hub.d_init : nullptr;
  p.in_split = a.in_split;
  p.in_lo = a.in_lo;
  p.in_hi = a.in_hi;
  p.out_split = a.out_split;
  p.out_lo = a.out_lo;
  p.out_hi = a.out_hi;
  p.out_bf16 = a.out_bf16;
  p.scale = a.scale;
  p.f = a.f;
  p.ld_in = a.ld_in;
  p.ld_out = a.ld_out;
  p.ld_bf16 = a.ld_bf16;
  p.ld_part = (a.f + 3) / 4 * 4;
  p.partials = a.partials;
  p.accum_lo = a.accum_lo;
  p.relu = a.relu;
  p.send = a.send;
  p.send_ptr = a.send_ptr;
  p.send_pos = a.send_pos;
  if (a.send && (!a.send_ptr || !a.send_pos || (reinterpret_cast<uintptr_t>(a.send) & 15) || a.ld_out % 4))
    return set_error(PGCN_EINVAL, "aggregation: send rows need the send map, 16-byte alignment and ld % 4 == 0");
  const int f4 = (a.f + 3) / 4;
  const int C = plan.chunks;
  if (f4 > kMaxAggF4) return set_error(PGCN_EINVAL, "aggregation: feature widths above 63,740 are not supported");
  ColLaunch cl[128];
  const int ncl = col_launches(f4, cl, 128);
  if (ncl < 0) return set_error(PGCN_EINVAL, "aggregation: too many column launches");
  for (int li = 0; li < ncl; ++li) {
    const int S = cl[li].S, SL = cl[li].SL;
    p.c4_off = cl[li].off;
    p.c4_cnt = cl[li].cnt;
    p.slices = S;
    const int U = 8;
    const int threshold = (64 / SL) * U;
    {
      TraceScope ts(a.trace_kind, s);      // one record for the chunk launches, which run back to back
      int32_t launched = 0;
      if (hub.rows > 0) {                  // block sums first: the rows' items add onto them
        HubParams hp{};
        hp.row_ids = hub.d_row_ids;
        hp.col_ids = hub.d_col_ids;
        hp.bits = hub.d_bits;
        hp.rows = hub.rows;
        hp.ntiles = hub.cols / kHubColTile;
        hp.in_split = a.in_split;
        hp.in_lo = a.in_lo;
        hp.in_hi = a.in_hi;
        hp.ld_in = a.ld_in;
        hp.c4_off = cl[li].off;
        hp.c4_cnt = cl[li].cnt < 64 ? cl[li].cnt : 64;
        hp.ld_part = p.ld_part;
        hp.part = a.partials + (size_t)plan.slots * (size_t)p.ld_part;
        hp.img = reinterpret_cast<uint16_t *>(hp.part + (size_t)hub_sum_rows(plan, a.f) * (size_t)p.ld_part);
        for (int c0 = cl[li].off; c0 < cl[li].off + cl[li].cnt; c0 += 64) {   // at most 64 float4 per pass
          hp.c4_off = c0;
          hp.c4_cnt = cl[li].off + cl[li].cnt - c0 < 64 ? cl[li].off + cl[li].cnt - c0 : 64;
          hp.nfb = hub_nfb(hp.c4_cnt);
          hp.groups = hub_groups(hub, hp.nfb);
          hp.tiles_per_group = (hp.ntiles + hp.groups - 1) / hp.groups;
          hipLaunchKernelGGL(hub_split_kernel, dim3((unsigned)(4 * hp.ntiles)), dim3(256), 0, s, hp);
          PGCN_HIP(hipGetLastError());
          hipLaunchKernelGGL(hub_kernel, dim3((unsigned)(hub.rows / kHubRowTile * hp.groups * hp.nfb)), dim3(512), 0,
                             s, hp);
          PGCN_HIP(hipGetLastError());
          AggParams pc = p;
          pc.c4_off = hp.c4_off;
          pc.c4_cnt = hp.c4_cnt;
          hipLaunchKernelGGL(hub_combine_kernel, dim3((unsigned)((hub.rows + 3) / 4)), dim3(256), 0, s, pc, hp);
          PGCN_HIP(hipGetLastError());
          launched += 3;
        }
      }
      for (int c = 0; c < C; ++c) {
        p.mode = (c == 0 ? AGG_FIRST : 0) | (c == C - 1 ? AGG_LAST : 0);
        const int64_t b = plan.chunk_items[c], e = plan.chunk_items[c + 1];
        if (e == b) continue;
        p.items = plan.d_items + b;
        p.n_items = e - b;
        p.n_long = first_short(plan, c, threshold) - b;
        launch_dispatch(p, SL, s);
        ++launched;
        PGCN_HIP(hipGetLastError());
      }
      ts.set_launches(launched);
    }
    if (!plan.splits.empty()) {       // split rows: all their slots, in (chunk, segment) order
      p.mode = AGG_FIRST | AGG_LAST;
      TraceScope ts(PGCN_TK_AGG_FIXUP, s);
      hipLaunchKernelGGL(agg_fixup_kernel, dim3((unsigned)plan.splits.size()), dim3(256), 0, s, p,
                         (const SplitRow *)plan.d_splits);
      PGCN_HIP(hipGetLastError());
    }
  }
  return PGCN_OK;
}

}  // namespace pgcn

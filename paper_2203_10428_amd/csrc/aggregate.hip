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
// Mapping for CDNA4 (wave64): a group of LPR lanes owns one work item (a
// whole row, or a fixed segment of a long row); each lane holds NV float4
// column vectors, so one nnz gathers one feature row with LPR*NV 16-byte
// loads.  Column indices are read once per nnz by every lane of the group
// (same address: one cache line per group).  No floating-point atomics: a
// long row's segments write partial sums that a second pass adds in segment
// order.
#include "internal.h"

namespace pgcn {

struct AggParams {
  const WorkItem *items;
  int64_t n_items;
  const int32_t *col;
  int64_t in_split;
  const float *in_lo;
  const float *in_hi;
  int64_t out_split;
  float *out_lo;
  float *out_hi;
  uint16_t *out_bf16;
  const float *scale;
  int32_t f;          // feature columns (total)
  int32_t c4_off;     // first float4 column of this launch
  int32_t c4_cnt;     // float4 columns of this launch
  int64_t ld_in, ld_out, ld_part;
  float *partials;
};

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);  // quiet NaN
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

__device__ __forceinline__ void store_row(const AggParams &p, int64_t r, int c4, float4 v) {
  const int c = 4 * c4;
  float s = p.scale ? p.scale[r] : 1.0f;
  float4 o;
  o.x = (c + 0 < p.f) ? v.x * s : 0.0f;
  o.y = (c + 1 < p.f) ? v.y * s : 0.0f;
  o.z = (c + 2 < p.f) ? v.z * s : 0.0f;
  o.w = (c + 3 < p.f) ? v.w * s : 0.0f;
  if (r < p.out_split) {
    if (p.out_lo) *reinterpret_cast<float4 *>(p.out_lo + r * p.ld_out + c) = o;
    if (p.out_bf16) {
      uint2 w;
      w.x = (uint32_t)f32_to_bf16_rne(o.x) | ((uint32_t)f32_to_bf16_rne(o.y) << 16);
      w.y = (uint32_t)f32_to_bf16_rne(o.z) | ((uint32_t)f32_to_bf16_rne(o.w) << 16);
      *reinterpret_cast<uint2 *>(p.out_bf16 + r * p.ld_out + c) = w;
    }
  } else {
    *reinterpret_cast<float4 *>(p.out_hi + (r - p.out_split) * p.ld_out + c) = o;
  }
}

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

template <int LPR, int NV, int U>
__global__ __launch_bounds__(256) void agg_kernel(AggParams p) {
  constexpr int GROUPS = 256 / LPR;
  const int lane = threadIdx.x % LPR;
  int64_t item = (int64_t)blockIdx.x * GROUPS + threadIdx.x / LPR;
  if (LPR == 64) item = __builtin_amdgcn_readfirstlane((int)item);
  if (item >= p.n_items) return;
  const WorkItem it = p.items[item];
  const int32_t *cols = p.col + it.begin;
  const int len = it.len;

  float4 acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = make_float4(0.f, 0.f, 0.f, 0.f);

  bool active[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) active[v] = (lane + v * LPR) < p.c4_cnt;
  const int cbase = 4 * (p.c4_off + lane);

  int k = 0;
  for (; k + U <= len; k += U) {
    int32_t c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) c[u] = cols[k + u];
    float4 x[U][NV];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float *src;
      if (c[u] < p.in_split) src = p.in_lo + (int64_t)c[u] * p.ld_in;
      else src = p.in_hi ? p.in_hi + (int64_t)(c[u] - p.in_split) * p.ld_in : nullptr;
#pragma unroll
      for (int v = 0; v < NV; ++v)
        x[u][v] = (src && active[v]) ? *reinterpret_cast<const float4 *>(src + cbase + 4 * v * LPR)
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int v = 0; v < NV; ++v) acc[v] = add4(acc[v], x[u][v]);
  }
  for (; k < len; ++k) {
    const int32_t c = cols[k];
    const float *src;
    if (c < p.in_split) src = p.in_lo + (int64_t)c * p.ld_in;
    else src = p.in_hi ? p.in_hi + (int64_t)(c - p.in_split) * p.ld_in : nullptr;
    if (src) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
        if (active[v]) acc[v] = add4(acc[v], *reinterpret_cast<const float4 *>(src + cbase + 4 * v * LPR));
    }
  }

  if (it.dst >= 0) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
      if (active[v]) store_row(p, it.dst, p.c4_off + lane + v * LPR, acc[v]);
  } else {
    float *dst = p.partials + (int64_t)(-it.dst - 1) * p.ld_part;
#pragma unroll
    for (int v = 0; v < NV; ++v)
      if (active[v]) *reinterpret_cast<float4 *>(dst + cbase + 4 * v * LPR) = acc[v];
  }
}

// Sum the partial slots of each split row in slot order, then scale and store.
__global__ __launch_bounds__(256) void agg_fixup_kernel(AggParams p, const SplitRow *splits) {
  const SplitRow s = splits[blockIdx.x];
  for (int c4 = p.c4_off + threadIdx.x; c4 < p.c4_off + p.c4_cnt; c4 += blockDim.x) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < s.nslots; ++j)
      acc = add4(acc, *reinterpret_cast<const float4 *>(p.partials + (int64_t)(s.first_slot + j) * p.ld_part + 4 * c4));
    store_row(p, s.row, c4, acc);
  }
}

template <int LPR, int NV>
static void launch_variant(const AggParams &p, hipStream_t s, int32_t trace_kind) {
  TraceScope ts(trace_kind, s);
  constexpr int U = NV >= 3 ? 2 : (NV == 2 ? 4 : 8);
  const int64_t groups = 256 / LPR;
  const int64_t blocks = (p.n_items + groups - 1) / groups;
  hipLaunchKernelGGL((agg_kernel<LPR, NV, U>), dim3((unsigned)blocks), dim3(256), 0, s, p);
}

size_t aggregate_workspace(const Plan &plan, int64_t f) {
  const int64_t ld_part = (f + 3) / 4 * 4;
  return (size_t)plan.slots * (size_t)ld_part * sizeof(float);
}

int launch_aggregate(const AggArgs &a, hipStream_t s) {
  const Plan &plan = *a.plan;
  AggParams p{};
  p.items = plan.d_items;
  p.n_items = (int64_t)plan.items.size();
  p.col = a.col;
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
  p.ld_part = (a.f + 3) / 4 * 4;
  p.partials = a.partials;
  if (p.n_items == 0) return PGCN_OK;
  const int f4 = (a.f + 3) / 4;
  // one launch per chunk of at most 256 float4 columns (1024 features)
  for (int off = 0; off < f4; off += 256) {
    const int cnt = f4 - off < 256 ? f4 - off : 256;
    p.c4_off = off;
    p.c4_cnt = cnt;
    if (cnt <= 4) launch_variant<4, 1>(p, s, a.trace_kind);
    else if (cnt <= 8) launch_variant<8, 1>(p, s, a.trace_kind);
    else if (cnt <= 16) launch_variant<16, 1>(p, s, a.trace_kind);
    else if (cnt <= 32) launch_variant<32, 1>(p, s, a.trace_kind);
    else if (cnt <= 64) launch_variant<64, 1>(p, s, a.trace_kind);
    else if (cnt <= 128) launch_variant<64, 2>(p, s, a.trace_kind);
    else if (cnt <= 192) launch_variant<64, 3>(p, s, a.trace_kind);
    else launch_variant<64, 4>(p, s, a.trace_kind);
    PGCN_HIP(hipGetLastError());
    if (!plan.splits.empty()) {
      TraceScope ts(PGCN_TK_AGG_FIXUP, s);
      hipLaunchKernelGGL(agg_fixup_kernel, dim3((unsigned)plan.splits.size()), dim3(256), 0, s, p,
                         plan.d_splits);
      PGCN_HIP(hipGetLastError());
    }
  }
  return PGCN_OK;
}

}  // namespace pgcn

// Bandwidth-bound kernels of the partition step:
//   - moving-average smoothing of stale features / gradients (Section 3.4);
//   - packing of the rows sent to peers (Algorithm 1's send of H_{S_{i,j}});
//   - accumulation of received stale gradients into their rows, in ascending
//     send-list order (Algorithm 1's loop over peers j);
//   - softmax cross-entropy / sigmoid BCE with their logit gradients
//     (Algorithm 1's J^(L)), with a fixed-order loss reduction;
//   - the SGD update (Algorithm 1's last line).
//   - dropout of a layer input with a Philox4x32-10 mask (after the boundary
//     receive, one mask for the forward and the backward: the paper's
//     implementation notes);
//   - the Adam update (the optimiser of the paper's experiments);
//   - the masked, row-scaled gradient diag(1/d) (J ∘ 1[H > 0]) that a
//     transform-first layer aggregates in its backward (Appendix A.1's
//     gradients in the other association).
// All are float4-vectorised over the feature dimension; no float atomics.
#include <algorithm>

#include "internal.h"

namespace pgcn {

// Row-block mapping shared by the streaming kernels: a 256-thread block covers
// 256 >> shift rows; the (1 << shift) lanes of a row stride over its float4
// columns.  shift is chosen so that 1 << shift is the smallest power of two
// >= the row's float4 count (at most 64 lanes).
static int lane_shift(int f4) {
  int sh = 0;
  while (sh < 6 && (1 << sh) < f4) ++sh;
  return sh;
}

static unsigned row_blocks(int64_t rows, int sh) {
  const int64_t rpb = 256 >> sh;
  return (unsigned)((rows + rpb - 1) / rpb);
}

typedef float ew_f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void ema_kernel(float *state, const float *in, int64_t rows, int f4, int64_t ld,
                                                  float gamma, int sh) {
  const int64_t r = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (r >= rows) return;
  const float g1 = 1.0f - gamma;
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    float4 *sp = reinterpret_cast<float4 *>(state + r * ld) + c4;
    // the incoming rows are read once (non-temporal); the state is read next by the aggregation
    const ew_f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const ew_f32x4 *>(in + r * ld) + c4);
    float4 v = *sp;
    v.x = gamma * v.x + g1 * x.x;
    v.y = gamma * v.y + g1 * x.y;
    v.z = gamma * v.z + g1 * x.z;
    v.w = gamma * v.w + g1 * x.w;
    *sp = v;
  }
}

// out[r, 4 c4 + e] = (H == null || H[r, .] > 0 ? J[r, .] : 0) * scale[r]; zero past cols
__global__ __launch_bounds__(256) void mask_scale_kernel(const float *J, int64_t ldj, const float *H, int64_t ldh,
                                                         const float *scale, int64_t rows, int cols, int f4,
                                                         float *out, int64_t ldo, int sh) {
  const int64_t r = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (r >= rows) return;
  const float sc = scale[r];
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    float4 j = reinterpret_cast<const float4 *>(J + r * ldj)[c4];
    if (H) {
      const float4 h = reinterpret_cast<const float4 *>(H + r * ldh)[c4];
      j.x = h.x > 0.f ? j.x : 0.f;
      j.y = h.y > 0.f ? j.y : 0.f;
      j.z = h.z > 0.f ? j.z : 0.f;
      j.w = h.w > 0.f ? j.w : 0.f;
    }
    const int c = 4 * c4;
    float4 o;
    o.x = c + 0 < cols ? j.x * sc : 0.f;
    o.y = c + 1 < cols ? j.y * sc : 0.f;
    o.z = c + 2 < cols ? j.z * sc : 0.f;
    o.w = c + 3 < cols ? j.w * sc : 0.f;
    reinterpret_cast<float4 *>(out + r * ldo)[c4] = o;
  }
}

int launch_mask_scale(const float *J, int64_t ldj, const float *H, int64_t ldh, const float *scale, int64_t rows,
                      int32_t cols, float *out, int64_t ldo, hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (rows == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_MASK_SCALE, s);
  hipLaunchKernelGGL(mask_scale_kernel, dim3(row_blocks(rows, sh)), dim3(256), 0, s, J, ldj, H, ldh, scale, rows,
                     cols, f4, out, ldo, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

int launch_ema(float *state, const float *in, int64_t rows, int32_t cols, int64_t ld, float gamma,
               hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (rows == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_EMA, s);
  hipLaunchKernelGGL(ema_kernel, dim3(row_blocks(rows, sh)), dim3(256), 0, s, state, in, rows, f4, ld, gamma, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}


__global__ __launch_bounds__(256) void pack_kernel(const int32_t *idx, int64_t count, const float *src,
                                                   float *dst, int f4, int64_t ld, int sh) {
  const int64_t k = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (k >= count) return;
  const float4 *from = reinterpret_cast<const float4 *>(src + (int64_t)idx[k] * ld);
  float4 *to = reinterpret_cast<float4 *>(dst + k * ld);
  // the sent rows are read by no kernel of this step: kept out of the caches
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    const float4 x = from[c4];
    __builtin_nontemporal_store((ew_f32x4){x.x, x.y, x.z, x.w}, reinterpret_cast<ew_f32x4 *>(to + c4));
  }
}

// Device-to-device refill: 16-byte vectors with non-temporal loads and stores
// (the copied rows are read in the next iteration, not in this one, so they
// stay out of the caches the gathers use).  One short-lived workgroup per
// 16 KB (four vectors per thread, loads issued together): the copy runs on a
// side stream beside the compute kernels, and workgroups that retire often
// let the dispatcher interleave theirs (a grid-stride copy that holds every
// wave slot until it ends starves a compute kernel launched meanwhile).
constexpr int kRefillVec = 4;
__global__ __launch_bounds__(256) void refill_copy_kernel(const ew_f32x4 *src, ew_f32x4 *dst, int64_t n16) {
  const int64_t base = (int64_t)blockIdx.x * (256 * kRefillVec) + threadIdx.x;
  ew_f32x4 v[kRefillVec];
#pragma unroll
  for (int j = 0; j < kRefillVec; ++j)
    if (base + 256 * j < n16) v[j] = __builtin_nontemporal_load(src + base + 256 * j);
#pragma unroll
  for (int j = 0; j < kRefillVec; ++j)
    if (base + 256 * j < n16) __builtin_nontemporal_store(v[j], dst + base + 256 * j);
}

int launch_refill_copy(void *dst, const void *src, size_t bytes, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  const int64_t blocks = (n16 + 256 * kRefillVec - 1) / (256 * kRefillVec);
  PGCN_REQUIRE(blocks <= 0x7fffffff, "pgcn_refill_async: copy too large for one launch");
  hipLaunchKernelGGL(refill_copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     reinterpret_cast<const ew_f32x4 *>(src), reinterpret_cast<ew_f32x4 *>(dst), n16);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

int launch_pack(const int32_t *idx, int64_t count, const float *src, float *dst, int32_t cols, int64_t ld,
                hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (count == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_PACK, s);
  hipLaunchKernelGGL(pack_kernel, dim3(row_blocks(count, sh)), dim3(256), 0, s, idx, count, src, dst, f4, ld, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

__global__ __launch_bounds__(256) void accum_kernel(const int64_t *__restrict__ inv_ptr,
                                                    const int32_t *__restrict__ inv_k, int64_t rows,
                                                    const float *__restrict__ src, float *__restrict__ dst, int f4,
                                                    int64_t ld, int sh) {
  const int64_t u = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (u >= rows) return;
  const int64_t b = inv_ptr[u], e = inv_ptr[u + 1];
  if (b == e) return;
  float4 *d = reinterpret_cast<float4 *>(dst + u * ld);
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    float4 v = d[c4];
#pragma unroll 4
    for (int64_t q = b; q < e; ++q) {   // ascending send-list position: ascending peer (loads are independent)
      const ew_f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const ew_f32x4 *>(src + (int64_t)inv_k[q] * ld) + c4);
      v.x += x.x;
      v.y += x.y;
      v.z += x.z;
      v.w += x.w;
    }
    d[c4] = v;
  }
}

// The gradient smoothing of Section 3.4 fused into the accumulation: every
// send row k belongs to exactly one inner row u (send_idx[k] == u), so the
// thread that adds row k into u also updates its moving average, once:
//     state[k] = gamma state[k] + (1 - gamma) src[k];  dst[u] += state[k]
// (the moving average is read once instead of twice).
// The three buffers are distinct allocations and the send rows k of one inner
// row are distinct, so the loads of later send rows may be issued ahead of the
// state stores of earlier ones (restrict); the sums keep ascending order.
__global__ __launch_bounds__(256) void accum_ema_kernel(const int64_t *__restrict__ inv_ptr,
                                                        const int32_t *__restrict__ inv_k, int64_t rows,
                                                        const float *__restrict__ src, float *__restrict__ state,
                                                        float gamma, float *__restrict__ dst, int f4, int64_t ld,
                                                        int sh) {
  const int64_t u = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (u >= rows) return;
  const int64_t b = inv_ptr[u], e = inv_ptr[u + 1];
  if (b == e) return;
  const float g1 = 1.0f - gamma;
  float4 *d = reinterpret_cast<float4 *>(dst + u * ld);
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    float4 v = d[c4];
    for (int64_t q0 = b; q0 < e; q0 += 4) {   // ascending send-list position: ascending peer
      // four send rows per round, their loads issued together; past the row's last slot the
      // round repeats that slot and neither stores nor adds it
      const int n = e - q0 < 4 ? (int)(e - q0) : 4;
      int64_t k[4];
      float4 x[4], m[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) k[j] = inv_k[q0 + (j < n ? j : n - 1)];
      // the received rows and the moving averages are next read in a later
      // iteration: non-temporal, so they leave the caches to the inner rows
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const ew_f32x4 xs = __builtin_nontemporal_load(reinterpret_cast<const ew_f32x4 *>(src + k[j] * ld) + c4);
        const ew_f32x4 ms = __builtin_nontemporal_load(reinterpret_cast<const ew_f32x4 *>(state + k[j] * ld) + c4);
        x[j] = make_float4(xs.x, xs.y, xs.z, xs.w);
        m[j] = make_float4(ms.x, ms.y, ms.z, ms.w);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        m[j].x = gamma * m[j].x + g1 * x[j].x;
        m[j].y = gamma * m[j].y + g1 * x[j].y;
        m[j].z = gamma * m[j].z + g1 * x[j].z;
        m[j].w = gamma * m[j].w + g1 * x[j].w;
        if (j < n)
          __builtin_nontemporal_store((ew_f32x4){m[j].x, m[j].y, m[j].z, m[j].w},
                                      reinterpret_cast<ew_f32x4 *>(state + k[j] * ld) + c4);
        const bool in = j < n;
        v.x = in ? v.x + m[j].x : v.x;
        v.y = in ? v.y + m[j].y : v.y;
        v.z = in ? v.z + m[j].z : v.z;
        v.w = in ? v.w + m[j].w : v.w;
      }
    }
    d[c4] = v;
  }
}

int launch_accum_ema(const int64_t *inv_ptr, const int32_t *inv_k, int64_t rows, const float *src, float *state,
                     float gamma, float *dst, int32_t cols, int64_t ld, hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (rows == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_ACCUM_EMA, s);
  hipLaunchKernelGGL(accum_ema_kernel, dim3(row_blocks(rows, sh)), dim3(256), 0, s, inv_ptr, inv_k, rows, src,
                     state, gamma, dst, f4, ld, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

int launch_accum(const int64_t *inv_ptr, const int32_t *inv_k, int64_t rows, const float *src, float *dst,
                 int32_t cols, int64_t ld, hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (rows == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_ACCUM, s);
  hipLaunchKernelGGL(accum_kernel, dim3(row_blocks(rows, sh)), dim3(256), 0, s, inv_ptr, inv_k, rows, src, dst, f4,
                     ld, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

// ---------------------------------------------------------------- losses ---

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Softmax cross-entropy, every row read once into registers where it fits:
// rows of at most 64 classes four to a wave (one class per lane, the four
// rows' loads in flight together), rows of at most 256 classes one to a wave
// (four classes per lane), wider rows one to a wave and read three times.
constexpr int kCeRegs = 4;

__device__ __forceinline__ float ce_row_loss(float m, float s, float zy, bool y_ok, float scale) {
  return y_ok ? scale * (m + __logf(s) - zy) : __builtin_nanf("");  // an out-of-range label poisons the loss
}

// Four rows per wave (C <= 64): slot i holds class `lane` of row r0 + i.
__global__ __launch_bounds__(256) void softmax_ce4_kernel(const float *Z, int64_t rows, int C, int64_t ld,
                                                          const int32_t *labels, float scale, float *J,
                                                          float *row_loss) {
  const int lane = threadIdx.x % 64;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + threadIdx.x / 64) * kCeRegs;
  if (r0 >= rows) return;
  float zr[kCeRegs], m[kCeRegs], s[kCeRegs];
#pragma unroll
  for (int i = 0; i < kCeRegs; ++i) zr[i] = (r0 + i < rows && lane < C) ? Z[(r0 + i) * ld + lane] : -INFINITY;
#pragma unroll
  for (int i = 0; i < kCeRegs; ++i) m[i] = wave_max(zr[i]);
#pragma unroll
  for (int i = 0; i < kCeRegs; ++i) s[i] = wave_sum(lane < C ? __expf(zr[i] - m[i]) : 0.f);
#pragma unroll
  for (int i = 0; i < kCeRegs; ++i) {
    const int64_t r = r0 + i;
    if (r >= rows) break;
    const int y = labels[r];
    const float inv_s = 1.0f / s[i];
    if (lane < C) J[r * ld + lane] = scale * (__expf(zr[i] - m[i]) * inv_s - (lane == y ? 1.0f : 0.0f));
    const bool y_ok = y >= 0 && y < C;
    const float zy = __shfl(zr[i], y_ok ? y : 0, 64);
    if (lane == 0) row_loss[r] = ce_row_loss(m[i], s[i], zy, y_ok, scale);
  }
}

// One row per wave.
__global__ __launch_bounds__(256) void softmax_ce_kernel(const float *Z, int64_t rows, int C, int64_t ld,
                                                         const int32_t *labels, float scale, float *J,
                                                         float *row_loss) {
  const int lane = threadIdx.x % 64;
  const int64_t r = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
  if (r >= rows) return;
  const float *z = Z + r * ld;
  const int y = labels[r];
  const bool y_ok = y >= 0 && y < C;
  float *j = J + r * ld;
  float m = -INFINITY, s = 0.f;
  if (C <= 64 * kCeRegs) {
    float zr[kCeRegs];
#pragma unroll
    for (int i = 0; i < kCeRegs; ++i) zr[i] = lane + 64 * i < C ? z[lane + 64 * i] : -INFINITY;
#pragma unroll
    for (int i = 0; i < kCeRegs; ++i) m = fmaxf(m, zr[i]);
    m = wave_max(m);
#pragma unroll
    for (int i = 0; i < kCeRegs; ++i)
      if (lane + 64 * i < C) s += __expf(zr[i] - m);
    s = wave_sum(s);
    const float inv_s = 1.0f / s;
#pragma unroll
    for (int i = 0; i < kCeRegs; ++i) {
      const int c = lane + 64 * i;
      if (c < C) j[c] = scale * (__expf(zr[i] - m) * inv_s - (c == y ? 1.0f : 0.0f));
    }
  } else {
    for (int c = lane; c < C; c += 64) m = fmaxf(m, z[c]);
    m = wave_max(m);
    for (int c = lane; c < C; c += 64) s += __expf(z[c] - m);
    s = wave_sum(s);
    const float inv_s = 1.0f / s;
    for (int c = lane; c < C; c += 64) {
      const float p = __expf(z[c] - m) * inv_s;
      j[c] = scale * (p - (c == y ? 1.0f : 0.0f));
    }
  }
  if (lane == 0) row_loss[r] = ce_row_loss(m, s, y_ok ? z[y] : 0.f, y_ok, scale);
}

__global__ __launch_bounds__(256) void sigmoid_bce_kernel(const float *Z, int64_t rows, int C, int64_t ld,
                                                          const float *T, int64_t ld_t, float scale, float *J,
                                                          float *row_loss) {
  const int lane = threadIdx.x % 64;
  const int64_t r = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
  if (r >= rows) return;
  const float *z = Z + r * ld;
  const float *y = T + r * ld_t;
  float *j = J + r * ld;
  float l = 0.f;
  for (int c = lane; c < C; c += 64) {
    const float x = z[c], t = y[c];
    l += fmaxf(x, 0.f) - x * t + log1pf(__expf(-fabsf(x)));
    const float sg = 1.0f / (1.0f + __expf(-x));
    j[c] = scale * (sg - t);
  }
  l = wave_sum(l);
  if (lane == 0) row_loss[r] = scale * l;
}

// Fixed-order reduction of the per-row losses in two passes, fp64 sums: block b
// of the first adds rows [b per, (b + 1) per) (a fixed tree over its threads'
// strided sums) and leaves the result, rounded to fp32, in the range's first
// element; one block then adds those kLossBlocks values the same way.
constexpr int kLossBlocks = 256;

__device__ __forceinline__ double block_sum_1024(double s, double *part) {
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  return part[0];
}

__global__ __launch_bounds__(1024) void loss_partial_kernel(float *row_loss, int64_t rows, int64_t per) {
  __shared__ double part[1024];
  const int64_t r0 = (int64_t)blockIdx.x * per, r1 = r0 + per < rows ? r0 + per : rows;
  double s = 0.0;
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 1024) s += (double)row_loss[r];
  s = block_sum_1024(s, part);             // every read of the range is done before this point
  if (threadIdx.x == 0 && r0 < r1) row_loss[r0] = (float)s;
}

__global__ __launch_bounds__(1024) void loss_reduce_kernel(const float *row_loss, int64_t rows, int64_t per,
                                                           float *out) {
  __shared__ double part[1024];
  double s = 0.0;
  for (int64_t r = (int64_t)threadIdx.x * per; r < rows; r += (int64_t)1024 * per) s += (double)row_loss[r];
  s = block_sum_1024(s, part);
  if (threadIdx.x == 0) *out = (float)s;
}

size_t loss_workspace(int64_t rows) { return (size_t)rows * sizeof(float); }

int launch_loss(int32_t kind, const float *Z, int64_t rows, int32_t C, int64_t ld, const int32_t *labels,
                const float *targets, int64_t ld_t, float scale, float *J, float *loss_out, float *ws,
                hipStream_t s) {
  TraceScope ts(PGCN_TK_LOSS, s);
  if (rows > 0) {
    const unsigned blocks = (unsigned)((rows + 3) / 4);
    if (kind == PGCN_SOFTMAX_CE && C <= 64)
      hipLaunchKernelGGL(softmax_ce4_kernel, dim3((unsigned)((rows + 4 * kCeRegs - 1) / (4 * kCeRegs))), dim3(256), 0,
                         s, Z, rows, C, ld, labels, scale, J, ws);
    else if (kind == PGCN_SOFTMAX_CE)
      hipLaunchKernelGGL(softmax_ce_kernel, dim3(blocks), dim3(256), 0, s, Z, rows, C, ld, labels, scale, J, ws);
    else
      hipLaunchKernelGGL(sigmoid_bce_kernel, dim3(blocks), dim3(256), 0, s, Z, rows, C, ld, targets, ld_t, scale,
                         J, ws);
    PGCN_HIP(hipGetLastError());
  }
  const int64_t per = rows > 0 ? (rows + kLossBlocks - 1) / kLossBlocks : 1;
  if (rows > 0) {
    hipLaunchKernelGGL(loss_partial_kernel, dim3((unsigned)((rows + per - 1) / per)), dim3(1024), 0, s, ws, rows, per);
    PGCN_HIP(hipGetLastError());
  }
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(1024), 0, s, (const float *)ws, rows, per, loss_out);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

__global__ __launch_bounds__(256) void sgd_kernel(float *W, const float *G, const float *G2, int64_t count,
                                                  float eta) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  const float g = G2 ? G[i] + G2[i] : G[i];
  W[i] = W[i] - eta * g;
}

int launch_sgd(float *W, const float *G, const float *G2, int64_t count, float eta, hipStream_t s) {
  if (count == 0) return PGCN_OK;
  TraceScope ts(PGCN_TK_SGD, s);
  hipLaunchKernelGGL(sgd_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, W, G, G2, count, eta);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

// float -> bf16 bits, round to nearest even (NaN stays a quiet NaN)
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): ten rounds of
// (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))
// with the key advanced by the Weyl constants after every round.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

__device__ __forceinline__ uint32_t word_of(const uint4 &a, int i) {
  return i == 0 ? a.x : i == 1 ? a.y : i == 2 ? a.z : a.w;
}

// Element q = (row0 + r) * cols + c is dropped when word q % 4 of
// Philox(counter = (q / 4 low, q / 4 high, layer, iteration), key = (seed, part))
// is below thr; kept elements are scaled.  Padding columns are written as 0.
__global__ __launch_bounds__(256) void dropout_kernel(float *out, const float *in, int64_t rows, int f4, int cols,
                                                      int64_t ld, int64_t row0, uint32_t thr, float scale,
                                                      uint32_t seed, uint32_t part, uint32_t layer, uint32_t iter,
                                                      uint16_t *out16, int64_t ld16, int sh) {
  const int64_t r = (int64_t)blockIdx.x * (256 >> sh) + (threadIdx.x >> sh);
  if (r >= rows) return;
  for (int c4 = threadIdx.x & ((1 << sh) - 1); c4 < f4; c4 += 1 << sh) {
    const int c = 4 * c4;
    const float4 x = *reinterpret_cast<const float4 *>(in + r * ld + c);
    float v[4] = {x.x, x.y, x.z, x.w};
    if (thr != 0u) {
      const uint64_t q0 = (uint64_t)(row0 + r) * (uint64_t)cols + (uint64_t)c;
      const uint64_t g = q0 >> 2;
      const int w0 = (int)(q0 & 3u);
      const uint4 a = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)(g >> 32), layer, iter), seed, part);
      uint4 b = a;
      if (w0 != 0)
        b = philox4x32_10(make_uint4((uint32_t)(g + 1), (uint32_t)((g + 1) >> 32), layer, iter), seed, part);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = w0 + e;
        const uint32_t u = i < 4 ? word_of(a, i) : word_of(b, i - 4);
        v[e] = u < thr ? 0.f : v[e] * scale;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (c + e >= cols) v[e] = 0.f;
    *reinterpret_cast<float4 *>(out + r * ld + c) = make_float4(v[0], v[1], v[2], v[3]);
    if (out16) {
      uint2 w;
      w.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
      w.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
      *reinterpret_cast<uint2 *>(out16 + r * ld16 + c) = w;
    }
  }
}

int launch_dropout(float *out, const float *in, int64_t rows, int32_t cols, int64_t ld, int64_t row0, uint32_t thr,
                   float scale, uint32_t seed, uint32_t part, uint32_t layer, uint32_t iteration, uint16_t *out16,
                   int64_t ld16, hipStream_t s) {
  const int f4 = (cols + 3) / 4;
  if (rows == 0 || f4 == 0) return PGCN_OK;
  const int sh = lane_shift(f4);
  TraceScope ts(PGCN_TK_DROPOUT, s);
  hipLaunchKernelGGL(dropout_kernel, dim3(row_blocks(rows, sh)), dim3(256), 0, s, out, in, rows, f4, cols, ld, row0,
                     thr, scale, seed, part, layer, iteration, out16, ld16, sh);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

// Adam (Kingma and Ba, Algorithm 1) with host-computed coefficients.
__global__ __launch_bounds__(256) void adam_kernel(float *W, const float *G, const float *Gp, float *m, float *v,
                                                   int64_t count, AdamCoef c) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= count) return;
  const float g = Gp ? G[i] + Gp[i] : G[i];
  const float mi = c.b1 * m[i] + c.omb1 * g;
  const float vi = c.b2 * v[i] + c.omb2 * (g * g);
  m[i] = mi;
  v[i] = vi;
  W[i] -= c.lr * (mi * c.c1) / (sqrtf(vi * c.c2) + c.eps);
}

int launch_adam(float *W, const float *G, const float *Gp, float *m, float *v, int64_t count, const AdamCoef &c,
                hipStream_t s) {
  if (count == 0) return PGCN_OK;
  TraceScope ts(PGCN_TK_ADAM, s);
  hipLaunchKernelGGL(adam_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, W, G, Gp, m, v, count, c);
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

}  // namespace pgcn

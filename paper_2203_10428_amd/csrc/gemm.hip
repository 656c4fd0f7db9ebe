// Dense update GEMMs of a GCN layer on CDNA4 matrix cores (Appendix A.1):
//   forward       Z = A W, H = relu(Z)                  (NN, ReLU epilogue)
//   feature grad  D = diag(1/d) ((J ∘ 1[H>0]) W^T)      (mask prologue, row-scale epilogue)
//   weight grad   G = A^T (J ∘ 1[H>0])                  (split over the node dimension,
//                                                         partials added in a fixed order)
// fp32 operands use v_mfma_f32_32x32x2f32; the bf16 path rounds operands to
// bf16 (round to nearest even) while staging them into LDS and uses
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//
// Tiling: 256 threads = 4 wave64s arranged 2x2 over a BM x BN tile; each wave
// owns (BM/2) x (BN/2) = several 32x32 MFMA tiles.  Tiles are staged through
// LDS with a register prefetch of the next K-slab while the current one is
// multiplied.  Block ids are remapped so that tiles sharing an A row-block run
// on the same XCD (same L2).
#include "internal.h"

namespace pgcn {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

enum AKind { A_MK_F32, A_MK_BF16, A_MK_MASK, A_KM_F32, A_KM_BF16 };
enum BKind { B_KN_W, B_NK_W, B_KN_MASK };
enum EKind { E_RELU, E_PLAIN, E_ROWSCALE, E_PARTIAL };

struct GP {
  int M, N, K;
  int kchunk;
  int tiles_n;
  const float *A;
  const uint16_t *A16;
  int64_t lda;
  const float *Am;       // mask source of A (A_MK_MASK), may be null
  int64_t ldam;
  const float *B;
  int64_t ldb;
  const float *Bm;       // mask source of B (B_KN_MASK), may be null
  int64_t ldbm;
  float *C;
  int64_t ldc;
  const float *rowscale;
};

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

__device__ __forceinline__ int xcd_remap(int b, int g) {
  if (g % 8 != 0) return b;
  return (b % 8) * (g / 8) + b / 8;
}

__device__ __forceinline__ float4 ld4_masked(const float *p, int valid) {
  float4 v = *reinterpret_cast<const float4 *>(p);
  if (valid < 4) {
    if (valid < 4) v.w = 0.f;
    if (valid < 3) v.z = 0.f;
    if (valid < 2) v.y = 0.f;
    if (valid < 1) v.x = 0.f;
  }
  return v;
}

__device__ __forceinline__ float4 apply_mask(float4 j, const float *h) {
  float4 m = *reinterpret_cast<const float4 *>(h);
  j.x = m.x > 0.f ? j.x : 0.f;
  j.y = m.y > 0.f ? j.y : 0.f;
  j.z = m.z > 0.f ? j.z : 0.f;
  j.w = m.w > 0.f ? j.w : 0.f;
  return j;
}

template <int EK>
__device__ __forceinline__ void epilogue_store(const GP &p, int row, int col, float v) {
  if (row >= p.M || col >= p.N) return;
  if (EK == E_RELU) {
    p.C[(int64_t)row * p.ldc + col] = v > 0.f ? v : 0.f;
  } else if (EK == E_PLAIN) {
    p.C[(int64_t)row * p.ldc + col] = v;
  } else if (EK == E_ROWSCALE) {
    p.C[(int64_t)row * p.ldc + col] = v * p.rowscale[row];
  } else {
    p.C[(int64_t)blockIdx.z * p.M * p.N + (int64_t)row * p.N + col] = v;
  }
}

// ------------------------------------------------------------------ fp32 ---

template <int BM, int BN, int AK, int BKd, int EK>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GP p) {
  constexpr int BK = 16, PAD = 4;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 4 / 256;       // float4 per thread for A
  constexpr int SB = BK * BN / 256;           // scalars per thread for W operands
  constexpr int VB = BK * BN / 4 / 256;       // float4 per thread for masked B
  static_assert(VA >= 1 && SB >= 1 && VB >= 1, "tile too small");
  __shared__ float As[BK][BM + PAD];
  __shared__ float Bs[BK][BN + PAD];

  const int t = threadIdx.x, lane = t % 64, wave = t / 64;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = blockIdx.z * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;

  float4 ra[VA];
  float rb[SB];
  float4 rbv[VB];

  auto load = [&](int kt) __attribute__((always_inline)) {
    if (AK == A_MK_F32 || AK == A_MK_MASK) {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, m = idx / (BK / 4), k4 = idx % (BK / 4);
        const int gm = m0 + m, gk = kt + 4 * k4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gm < p.M && gk < kend) {
          x = ld4_masked(p.A + (int64_t)gm * p.lda + gk, kend - gk);
          if (AK == A_MK_MASK && p.Am) x = apply_mask(x, p.Am + (int64_t)gm * p.ldam + gk);
        }
        ra[v] = x;
      }
    } else {  // A_KM_F32: element (m, k) at A[k * lda + m]
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, k = idx / (BM / 4), m4 = idx % (BM / 4);
        const int gk = kt + k, gm = m0 + 4 * m4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gk < kend && gm < p.M) x = ld4_masked(p.A + (int64_t)gk * p.lda + gm, p.M - gm);
        ra[v] = x;
      }
    }
    if (BKd == B_KN_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s, k = idx / BN, n = idx % BN;
        const int gk = kt + k, gn = n0 + n;
        rb[s] = (gk < kend && gn < p.N) ? p.B[(int64_t)gk * p.ldb + gn] : 0.f;
      }
    } else if (BKd == B_NK_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s, n = idx / BK, k = idx % BK;
        const int gk = kt + k, gn = n0 + n;
        rb[s] = (gk < kend && gn < p.N) ? p.B[(int64_t)gn * p.ldb + gk] : 0.f;
      }
    } else {  // B_KN_MASK
#pragma unroll
      for (int v = 0; v < VB; ++v) {
        const int idx = t + 256 * v, k = idx / (BN / 4), n4 = idx % (BN / 4);
        const int gk = kt + k, gn = n0 + 4 * n4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gk < kend && gn < p.N) {
          x = ld4_masked(p.B + (int64_t)gk * p.ldb + gn, p.N - gn);
          if (p.Bm) x = apply_mask(x, p.Bm + (int64_t)gk * p.ldbm + gn);
        }
        rbv[v] = x;
      }
    }
  };

  auto store = [&]() __attribute__((always_inline)) {
    if (AK == A_MK_F32 || AK == A_MK_MASK) {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, m = idx / (BK / 4), k4 = idx % (BK / 4);
        As[4 * k4 + 0][m] = ra[v].x;
        As[4 * k4 + 1][m] = ra[v].y;
        As[4 * k4 + 2][m] = ra[v].z;
        As[4 * k4 + 3][m] = ra[v].w;
      }
    } else {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, k = idx / (BM / 4), m4 = idx % (BM / 4);
        *reinterpret_cast<float4 *>(&As[k][4 * m4]) = ra[v];
      }
    }
    if (BKd == B_KN_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s;
        Bs[idx / BN][idx % BN] = rb[s];
      }
    } else if (BKd == B_NK_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s;
        Bs[idx % BK][idx / BK] = rb[s];
      }
    } else {
#pragma unroll
      for (int v = 0; v < VB; ++v) {
        const int idx = t + 256 * v, k = idx / (BN / 4), n4 = idx % (BN / 4);
        *reinterpret_cast<float4 *>(&Bs[k][4 * n4]) = rbv[v];
      }
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  if (kbeg < kend) {
    load(kbeg);
    store();
    __syncthreads();
    for (int kt = kbeg; kt < kend; kt += BK) {
      const bool more = kt + BK < kend;
      if (more) load(kt + BK);
#pragma unroll
      for (int kk = 0; kk < BK; kk += 2) {
        float a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[kk + lane / 32][wm0 + i * 32 + lane % 32];
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = Bs[kk + lane / 32][wn0 + j * 32 + lane % 32];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      __syncthreads();
      if (more) {
        store();
        __syncthreads();
      }
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + i * 32 + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
        const int col = n0 + wn0 + j * 32 + lane % 32;
        epilogue_store<EK>(p, row, col, acc[i][j][r]);
      }
}

// ------------------------------------------------------------------ bf16 ---

template <int BM, int BN, int AK, int BKd, int EK>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GP p) {
  constexpr int BK = 32, PAD = 8;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 8 / 256;       // 8-element vectors per thread for A
  constexpr int SB = BK * BN / 256;
  constexpr int VB = BK * BN / 4 / 256;
  static_assert(VA >= 1 && SB >= 1 && VB >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) uint16_t As[BM][BK + PAD];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN][BK + PAD];

  const int t = threadIdx.x, lane = t % 64, wave = t / 64;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = blockIdx.z * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;

  uint4 ra[VA];
  float rb[SB];
  float4 rbv[VB];

  auto pack8 = [](float4 a, float4 b) {
    uint4 r;
    r.x = (uint32_t)bf16_rne(a.x) | ((uint32_t)bf16_rne(a.y) << 16);
    r.y = (uint32_t)bf16_rne(a.z) | ((uint32_t)bf16_rne(a.w) << 16);
    r.z = (uint32_t)bf16_rne(b.x) | ((uint32_t)bf16_rne(b.y) << 16);
    r.w = (uint32_t)bf16_rne(b.z) | ((uint32_t)bf16_rne(b.w) << 16);
    return r;
  };
  auto mask16 = [](uint4 v, int valid) {   // zero bf16 elements >= valid
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (e >= valid) w[e / 2] &= (e % 2) ? 0x0000ffffu : 0xffff0000u;
    return make_uint4(w[0], w[1], w[2], w[3]);
  };

  auto load = [&](int kt) __attribute__((always_inline)) {
    if (AK == A_MK_BF16) {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, m = idx / (BK / 8), k8 = idx % (BK / 8);
        const int gm = m0 + m, gk = kt + 8 * k8;
        uint4 x = make_uint4(0, 0, 0, 0);
        if (gm < p.M && gk < kend) {
          x = *reinterpret_cast<const uint4 *>(p.A16 + (int64_t)gm * p.lda + gk);
          if (kend - gk < 8) x = mask16(x, kend - gk);
        }
        ra[v] = x;
      }
    } else if (AK == A_MK_MASK || AK == A_MK_F32) {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, m = idx / (BK / 8), k8 = idx % (BK / 8);
        const int gm = m0 + m, gk = kt + 8 * k8;
        float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
        if (gm < p.M && gk < kend) {
          const float *row = p.A + (int64_t)gm * p.lda + gk;
          x0 = ld4_masked(row, kend - gk);
          if (AK == A_MK_MASK && p.Am) x0 = apply_mask(x0, p.Am + (int64_t)gm * p.ldam + gk);
          if (gk + 4 < kend) {
            x1 = ld4_masked(row + 4, kend - gk - 4);
            if (AK == A_MK_MASK && p.Am) x1 = apply_mask(x1, p.Am + (int64_t)gm * p.ldam + gk + 4);
          }
        }
        ra[v] = pack8(x0, x1);
      }
    } else {  // A_KM_BF16: element (m, k) at A16[k * lda + m]
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, k = idx / (BM / 8), m8 = idx % (BM / 8);
        const int gk = kt + k, gm = m0 + 8 * m8;
        uint4 x = make_uint4(0, 0, 0, 0);
        if (gk < kend && gm < p.M) {
          x = *reinterpret_cast<const uint4 *>(p.A16 + (int64_t)gk * p.lda + gm);
          if (p.M - gm < 8) x = mask16(x, p.M - gm);
        }
        ra[v] = x;
      }
    }
    if (BKd == B_KN_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s, k = idx / BN, n = idx % BN;
        const int gk = kt + k, gn = n0 + n;
        rb[s] = (gk < kend && gn < p.N) ? p.B[(int64_t)gk * p.ldb + gn] : 0.f;
      }
    } else if (BKd == B_NK_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s, n = idx / BK, k = idx % BK;
        const int gk = kt + k, gn = n0 + n;
        rb[s] = (gk < kend && gn < p.N) ? p.B[(int64_t)gn * p.ldb + gk] : 0.f;
      }
    } else {
#pragma unroll
      for (int v = 0; v < VB; ++v) {
        const int idx = t + 256 * v, k = idx / (BN / 4), n4 = idx % (BN / 4);
        const int gk = kt + k, gn = n0 + 4 * n4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (gk < kend && gn < p.N) {
          x = ld4_masked(p.B + (int64_t)gk * p.ldb + gn, p.N - gn);
          if (p.Bm) x = apply_mask(x, p.Bm + (int64_t)gk * p.ldbm + gn);
        }
        rbv[v] = x;
      }
    }
  };

  auto store = [&]() __attribute__((always_inline)) {
    if (AK == A_KM_BF16) {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, k = idx / (BM / 8), m8 = idx % (BM / 8);
        const uint32_t w[4] = {ra[v].x, ra[v].y, ra[v].z, ra[v].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) As[8 * m8 + e][k] = (uint16_t)(w[e / 2] >> (16 * (e % 2)));
      }
    } else {
#pragma unroll
      for (int v = 0; v < VA; ++v) {
        const int idx = t + 256 * v, m = idx / (BK / 8), k8 = idx % (BK / 8);
        *reinterpret_cast<uint4 *>(&As[m][8 * k8]) = ra[v];
      }
    }
    if (BKd == B_KN_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s;
        Bs[idx % BN][idx / BN] = bf16_rne(rb[s]);
      }
    } else if (BKd == B_NK_W) {
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int idx = t + 256 * s;
        Bs[idx / BK][idx % BK] = bf16_rne(rb[s]);
      }
    } else {
#pragma unroll
      for (int v = 0; v < VB; ++v) {
        const int idx = t + 256 * v, k = idx / (BN / 4), n4 = idx % (BN / 4);
        Bs[4 * n4 + 0][k] = bf16_rne(rbv[v].x);
        Bs[4 * n4 + 1][k] = bf16_rne(rbv[v].y);
        Bs[4 * n4 + 2][k] = bf16_rne(rbv[v].z);
        Bs[4 * n4 + 3][k] = bf16_rne(rbv[v].w);
      }
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  if (kbeg < kend) {
    load(kbeg);
    store();
    __syncthreads();
    for (int kt = kbeg; kt < kend; kt += BK) {
      const bool more = kt + BK < kend;
      if (more) load(kt + BK);
#pragma unroll
      for (int ks = 0; ks < BK; ks += 16) {
        bf16x8 a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(&As[wm0 + i * 32 + lane % 32][ks + 8 * (lane / 32)]));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(&Bs[wn0 + j * 32 + lane % 32][ks + 8 * (lane / 32)]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      __syncthreads();
      if (more) {
        store();
        __syncthreads();
      }
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + i * 32 + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
        const int col = n0 + wn0 + j * 32 + lane % 32;
        epilogue_store<EK>(p, row, col, acc[i][j][r]);
      }
}

// Fixed-order sum of split partials.  A block owns 64 consecutive outputs and
// 4 quarters of the split range; quarter q adds its splits in ascending order,
// then the quarters are added in order q = 0, 1, 2, 3.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *ws, int splits, int64_t mn, float *out) {
  __shared__ float part[4][64];
  const int o = threadIdx.x % 64, q = threadIdx.x / 64;
  const int64_t i = (int64_t)blockIdx.x * 64 + o;
  const int per = (splits + 3) / 4;
  const int z0 = q * per, z1 = min(splits, z0 + per);
  float s = 0.f;
  if (i < mn)
    for (int z = z0; z < z1; ++z) s += ws[(int64_t)z * mn + i];
  part[q][o] = s;
  __syncthreads();
  if (q == 0 && i < mn) out[i] = ((part[0][o] + part[1][o]) + part[2][o]) + part[3][o];
}

// ---------------------------------------------------------------- launch ---

static int splitk_count(int M, int N, int K, int BM, int BN, int BK) {
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  int s = (1024 + tiles - 1) / tiles;
  const int max_s = (K + 255) / 256;
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  (void)BK;
  return s;
}

size_t gemm_workspace(Gemm kind, int32_t M, int32_t N, int32_t K) {
  if (kind != Gemm::TN_MASK_SPLITK) return 0;
  const int BN = N <= 64 ? 64 : 128;
  const int s = splitk_count(M, N, K, 128, BN, 16);
  return (size_t)s * (size_t)M * (size_t)N * sizeof(float);
}

template <int BN, int AK, int BKd, int EK>
static int run(const GP &p0, int bf16, int splits, hipStream_t s) {
  TraceScope ts(EK == E_PARTIAL ? PGCN_TK_GEMM_WGRAD : (EK == E_ROWSCALE ? PGCN_TK_GEMM_DGRAD : PGCN_TK_GEMM_FWD), s);
  constexpr int BM = 128;
  GP p = p0;
  const int tm = (p.M + BM - 1) / BM, tn = (p.N + BN - 1) / BN;
  p.tiles_n = tn;
  const int BK = bf16 ? 32 : 16;
  int kchunk = (p.K + splits - 1) / splits;
  kchunk = (kchunk + BK - 1) / BK * BK;
  if (kchunk == 0) kchunk = BK;
  p.kchunk = kchunk;
  dim3 grid((unsigned)(tm * tn), 1, (unsigned)splits);
  if (bf16) {
    constexpr int AKb = AK == A_MK_F32 ? A_MK_BF16 : (AK == A_KM_F32 ? A_KM_BF16 : AK);
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, AKb, BKd, EK>), grid, dim3(256), 0, s, p);
  } else {
    hipLaunchKernelGGL((gemm_f32_kernel<BM, BN, AK, BKd, EK>), grid, dim3(256), 0, s, p);
  }
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

template <int AK, int BKd, int EK>
static int run_bn(const GP &p, int bf16, int splits, hipStream_t s) {
  if (p.N <= 64) return run<64, AK, BKd, EK>(p, bf16, splits, s);
  return run<128, AK, BKd, EK>(p, bf16, splits, s);
}

int launch_gemm(Gemm kind, const GemmArgs &g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return PGCN_OK;
  GP p{};
  p.M = g.M;
  p.N = g.N;
  p.K = g.K;
  p.A = g.A;
  p.A16 = g.A16;
  p.lda = g.lda;
  p.B = g.B;
  p.ldb = g.ldb;
  p.C = g.C;
  p.ldc = g.ldc;
  p.rowscale = g.rowscale;
  const int bf16 = g.dtype == PGCN_BF16;
  switch (kind) {
    case Gemm::NN_RELU:
      return run_bn<A_MK_F32, B_KN_W, E_RELU>(p, bf16, 1, s);
    case Gemm::NN_PLAIN:
      return run_bn<A_MK_F32, B_KN_W, E_PLAIN>(p, bf16, 1, s);
    case Gemm::MASK_NT_ROWSCALE:
      p.Am = g.Hmask;
      p.ldam = g.ldm;
      return run_bn<A_MK_MASK, B_NK_W, E_ROWSCALE>(p, bf16, 1, s);
    case Gemm::TN_MASK_SPLITK: {
      p.Bm = g.Hmask;
      p.ldbm = g.ldm;
      const int BN = g.N <= 64 ? 64 : 128;
      const int splits = splitk_count(g.M, g.N, g.K, 128, BN, 16);
      const size_t need = (size_t)splits * (size_t)g.M * (size_t)g.N * sizeof(float);
      if (!g.workspace || g.workspace_bytes < need)
        return set_error(PGCN_EWORKSPACE, "weight-gradient GEMM: workspace too small");
      p.C = g.workspace;
      int rc = run_bn<A_KM_F32, B_KN_MASK, E_PARTIAL>(p, bf16, splits, s);
      if (rc) return rc;
      const int64_t mn = (int64_t)g.M * g.N;
      TraceScope ts(PGCN_TK_WGRAD_REDUCE, s);
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((mn + 63) / 64)), dim3(256), 0, s,
                         (const float *)g.workspace, splits, mn, g.C);
      PGCN_HIP(hipGetLastError());
      return PGCN_OK;
    }
  }
  return set_error(PGCN_EINVAL, "unknown GEMM kind");
}

}  // namespace pgcn

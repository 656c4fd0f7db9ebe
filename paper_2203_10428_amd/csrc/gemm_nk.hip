// Node-major update GEMMs of a GCN layer (Appendix A.1), C[M x N] = A[M x K] B^T
// with M = inner rows:
//   forward       Z = A W,                         A = aggregated features, B(n,k) = W[k][n]
//   feature grad  D = diag(1/d) ((J ∘ 1[H>0]) W^T), A = masked gradient,     B(n,k) = W[n][k]
// The GraphSAGE layer (Section 2's CONCAT update) uses the same kernels on
// the two halves of its weights: Z = z W_top, then Z = relu(Z + X W_bot)
// (accumulating epilogue), and the feature gradient without the row scale.
// On the bf16 path the feature gradient reads the masked operand as bf16,
// written once by the weight-gradient kernel (2 bytes per element instead of
// the 8 of fp32 J and H).
//
// The right operand (the layer's weights, at most a few MB) is first packed
// once per call into an n-major, k-contiguous matrix zero-padded to a 128-row
// and 64-column multiple (fp32, or bf16 rounded to nearest even for the bf16
// path), so the main loop loads both operands as 16-byte vectors with no
// bounds checks on the weights.
//
// Main loop for CDNA4: a 256-thread workgroup (4 wave64s, 2 x 2) computes a
// 128 x BN tile; both tiles sit in LDS with k contiguous and are double
// buffered, so one barrier per k-slab suffices while the next slab's global
// loads are in flight.  Slabs are short (16 fp32 / 32 bf16 values of k) so
// that three workgroups fit per CU: the staging of one workgroup's next slab
// (global load -> registers -> LDS) hides behind the others' MFMAs, which
// measured faster than longer slabs at two workgroups per CU.  The MFMA k
// order is permuted so that each lane's fragments over a slab are contiguous
// in LDS and load with 128-bit reads:
//   fp32, v_mfma_f32_32x32x2f32, slab of 16: step s uses k = 8*h + s for
//        lane half h (lanes 32h .. 32h+31);
//   bf16, v_mfma_f32_32x32x16_bf16, slab of 32: step j uses k = 16*h + 8*j
//        .. 16*h + 8*j + 7 for lane half h.
// Every k of the slab is used exactly once per output element.
#include "internal.h"

namespace pgcn {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct NKParams {
  int M, N, K;
  int tiles_n;
  const float *A;          // fp32 activations [M, lda] (k contiguous)
  const uint16_t *A16;     // bf16 activations [M, lda]
  int64_t lda;
  const float *Am;         // mask source of A (ReLU output), or null
  int64_t ldam;
  const void *B;           // packed weights [rows >= tiles_n * BN, ldb]
  int64_t ldb;
  float *C;
  int64_t ldc;
  const float *rowscale;
};

enum NKA { NK_A_F32, NK_A_BF16, NK_A_MASK };
enum NKE { NK_E_RELU, NK_E_PLAIN, NK_E_ROWSCALE, NK_E_ACC_RELU, NK_E_ACC_PLAIN };

__device__ __forceinline__ uint16_t nk_bf16(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7fffu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

__device__ __forceinline__ int nk_xcd_remap(int b, int g) {
  if (g % 8 != 0) return b;
  return (b % 8) * (g / 8) + b / 8;
}

// out[n][k] = (n < N && k < K) ? (trans ? W[k*ldw + n] : W[n*ldw + k]) : 0, for n < rows, k < ldk
template <bool BF16>
__global__ __launch_bounds__(256) void pack_b_kernel(const float *W, int ldw, int trans, int N, int K, int rows,
                                                     int ldk, void *out) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * ldk) return;
  const int n = i / ldk, k = i - n * ldk;
  const float v = (n < N && k < K) ? (trans ? W[(int64_t)k * ldw + n] : W[(int64_t)n * ldw + k]) : 0.f;
  if (BF16) reinterpret_cast<uint16_t *>(out)[i] = nk_bf16(v);
  else reinterpret_cast<float *>(out)[i] = v;
}

// Final value of one output element.
template <int EK>
__device__ __forceinline__ float nk_out(float v, float sc, float old) {
  if (EK == NK_E_RELU) return v > 0.f ? v : 0.f;
  if (EK == NK_E_PLAIN) return v;
  if (EK == NK_E_ROWSCALE) return v * sc;
  const float u = old + v;                             // accumulate onto C, then the activation
  return (EK == NK_E_ACC_RELU && u <= 0.f) ? 0.f : u;
}

// Stores the accumulators of one wave.  The values an epilogue reads (the row
// scales, or C for the accumulating forms) are loaded for a whole 32 x 32 tile
// before any of its stores, and tiles that lie inside C (all but the edge
// tiles; a wave-uniform test) store without per-element branches, so the
// loads are in flight together and the stores do not wait for one another.
template <int EK, int TM, int TN>
__device__ __forceinline__ void nk_epilogue(const NKParams &p, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                            int lane) {
  constexpr bool ACC = EK == NK_E_ACC_RELU || EK == NK_E_ACC_PLAIN;
  const int h = lane / 32, cl = lane % 32;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int rbase = m0 + i * 32 + 4 * h;
    const bool rows_in = m0 + i * 32 + 32 <= p.M;
    float sc[16];
    if (EK == NK_E_ROWSCALE) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = rbase + 8 * (r / 4) + (r % 4);
        sc[r] = (rows_in || row < p.M) ? p.rowscale[row] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + j * 32 + cl;
      float *c0 = p.C + (int64_t)rbase * p.ldc + col;
      float old[16];
      if (rows_in && n0 + j * 32 + 32 <= p.N) {
        if (ACC) {
#pragma unroll
          for (int r = 0; r < 16; ++r) old[r] = c0[(int64_t)(8 * (r / 4) + (r % 4)) * p.ldc];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r)
          c0[(int64_t)(8 * (r / 4) + (r % 4)) * p.ldc] = nk_out<EK>(acc[i][j][r], sc[r], old[r]);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = rbase + 8 * (r / 4) + (r % 4);
          if (row < p.M && col < p.N) {
            const float o = ACC ? c0[(int64_t)(8 * (r / 4) + (r % 4)) * p.ldc] : 0.f;
            c0[(int64_t)(8 * (r / 4) + (r % 4)) * p.ldc] = nk_out<EK>(acc[i][j][r], sc[r], o);
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ fp32 ---

template <int BM, int BN, int AK, int EK>
__global__ __launch_bounds__(256, 3) void gemm_nk_f32(NKParams p) {
  constexpr int BK = 16, LK = BK + 4, KV = BK / 4;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 4 / 256, VB = BN * BK / 4 / 256;
  __shared__ __attribute__((aligned(16))) float As[2][BM * LK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * LK];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  const int tile = nk_xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;
  const float *Bp = reinterpret_cast<const float *>(p.B);

  // raw loads only (whole vectors, predicated); the row-tail zeroing and the
  // ReLU mask are applied in store(), after the MFMAs that hide the loads
  f32x4 ra[VA], rh[VA], rb[VB];
  int kl = 0;                                          // k of the staged slab
  auto load = [&](int kt) __attribute__((always_inline)) {
    kl = kt;
#pragma unroll
    for (int v = 0; v < VA; ++v) {
      const int idx = t + 256 * v, m = idx / KV, k4 = idx % KV;
      const int gm = m0 + m, gk = kt + 4 * k4;
      const bool ok = gm < p.M && gk < p.K;
      ra[v] = ok ? *reinterpret_cast<const f32x4 *>(p.A + (int64_t)gm * p.lda + gk) : f32x4{0.f, 0.f, 0.f, 0.f};
      if (AK == NK_A_MASK)
        rh[v] = (ok && p.Am) ? *reinterpret_cast<const f32x4 *>(p.Am + (int64_t)gm * p.ldam + gk)
                             : f32x4{1.f, 1.f, 1.f, 1.f};
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v, n = idx / KV, k4 = idx % KV;
      rb[v] = *reinterpret_cast<const f32x4 *>(Bp + (int64_t)(n0 + n) * p.ldb + kt + 4 * k4);
    }
  };
  auto store = [&](int b) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < VA; ++v) {
      const int idx = t + 256 * v;
      f32x4 x = ra[v];
      const int valid = p.K - (kl + 4 * (idx % KV));   // zero the k >= K tail of the row
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e >= valid) x[e] = 0.f;
        if (AK == NK_A_MASK) x[e] = rh[v][e] > 0.f ? x[e] : 0.f;
      }
      *reinterpret_cast<f32x4 *>(&As[b][(idx / KV) * LK + 4 * (idx % KV)]) = x;
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      *reinterpret_cast<f32x4 *>(&Bs[b][(idx / KV) * LK + 4 * (idx % KV)]) = rb[v];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  load(0);
  store(0);
  __syncthreads();
  int it = 0;
  for (int kt = 0; kt < p.K; kt += BK, ++it) {
    const int cur = it & 1;
    // next slab's global loads in flight during this slab's MFMAs; the last
    // iteration reloads the current slab into the idle buffer (keeps the
    // staging registers free of control flow)
    load(kt + BK < p.K ? kt + BK : kt);
#pragma unroll
    for (int q = 0; q < BK / 8; ++q) {
      f32x4 a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        a[i] = *reinterpret_cast<const f32x4 *>(&As[cur][(wm0 + i * 32 + r) * LK + (BK / 2) * h + 4 * q]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = *reinterpret_cast<const f32x4 *>(&Bs[cur][(wn0 + j * 32 + r) * LK + (BK / 2) * h + 4 * q]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
    store(cur ^ 1);
    __syncthreads();
  }
  nk_epilogue<EK, TM, TN>(p, acc, m0 + wm0, n0 + wn0, lane);
}

// ------------------------------------------------------------------ bf16 ---

template <int BM, int BN, int AK, int EK>
__global__ __launch_bounds__(256, 3) void gemm_nk_bf16(NKParams p) {
  constexpr int BK = 32, LK = BK + 8, KV = BK / 8;     // bf16 elements; 80-byte rows
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 8 / 256, VB = BN * BK / 8 / 256;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LK];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  const int tile = nk_xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;
  const uint16_t *Bp = reinterpret_cast<const uint16_t *>(p.B);

  // raw loads only (whole vectors, predicated); the row-tail zeroing, the ReLU
  // mask and the bf16 rounding are applied in store(), after the MFMAs
  constexpr bool SRC32 = AK != NK_A_BF16;              // fp32 source rounded to bf16 in store()
  u32x4 ra[VA], rb[VB];
  f32x4 rx[SRC32 ? 2 * VA : 1], rh[AK == NK_A_MASK ? 2 * VA : 1];
  int kl = 0;                                          // k of the staged slab
  auto load = [&](int kt) __attribute__((always_inline)) {
    kl = kt;
#pragma unroll
    for (int v = 0; v < VA; ++v) {
      const int idx = t + 256 * v, m = idx / KV, k8 = idx % KV;
      const int gm = m0 + m, gk = kt + 8 * k8;
      const bool ok = gm < p.M && gk < p.K;
      if (!SRC32) {
        ra[v] = ok ? *reinterpret_cast<const u32x4 *>(p.A16 + (int64_t)gm * p.lda + gk) : u32x4{0u, 0u, 0u, 0u};
      } else {
        // the second half-vector exists when gk + 4 < K (ld is a multiple of 4)
        const float *row = p.A + (int64_t)gm * p.lda + gk;
        const bool ok1 = ok && gk + 4 < p.K;
        rx[2 * v] = ok ? *reinterpret_cast<const f32x4 *>(row) : f32x4{0.f, 0.f, 0.f, 0.f};
        rx[2 * v + 1] = ok1 ? *reinterpret_cast<const f32x4 *>(row + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        if (AK == NK_A_MASK) {
          const float *hrow = p.Am + (int64_t)gm * p.ldam + gk;
          rh[2 * v] = (ok && p.Am) ? *reinterpret_cast<const f32x4 *>(hrow) : f32x4{1.f, 1.f, 1.f, 1.f};
          rh[2 * v + 1] = (ok1 && p.Am) ? *reinterpret_cast<const f32x4 *>(hrow + 4) : f32x4{1.f, 1.f, 1.f, 1.f};
        }
      }
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v, n = idx / KV, k8 = idx % KV;
      rb[v] = *reinterpret_cast<const u32x4 *>(Bp + (int64_t)(n0 + n) * p.ldb + kt + 8 * k8);
    }
  };
  auto store = [&](int b) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < VA; ++v) {
      const int idx = t + 256 * v;
      const int valid = p.K - (kl + 8 * (idx % KV));   // zero the k >= K tail of the row
      u32x4 o;
      if (!SRC32) {
        o = ra[v];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e >= valid) o[e / 2] &= (e % 2) ? 0x0000ffffu : 0xffff0000u;
      } else {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          x[e] = rx[2 * v + e / 4][e % 4];
          if (AK == NK_A_MASK) x[e] = rh[2 * v + e / 4][e % 4] > 0.f ? x[e] : 0.f;
          if (e >= valid) x[e] = 0.f;
        }
#pragma unroll
        for (int w = 0; w < 4; ++w)
          o[w] = (uint32_t)nk_bf16(x[2 * w]) | ((uint32_t)nk_bf16(x[2 * w + 1]) << 16);
      }
      *reinterpret_cast<u32x4 *>(&As[b][(idx / KV) * LK + 8 * (idx % KV)]) = o;
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      *reinterpret_cast<u32x4 *>(&Bs[b][(idx / KV) * LK + 8 * (idx % KV)]) = rb[v];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  load(0);
  store(0);
  __syncthreads();
  int it = 0;
  for (int kt = 0; kt < p.K; kt += BK, ++it) {
    const int cur = it & 1;
    // next slab's global loads in flight during this slab's MFMAs; the last
    // iteration reloads the current slab into the idle buffer (keeps the
    // staging registers free of control flow)
    load(kt + BK < p.K ? kt + BK : kt);
#pragma unroll
    for (int q = 0; q < BK / 16; ++q) {
      bf16x8 a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(&As[cur][(wm0 + i * 32 + r) * LK + (BK / 2) * h + 8 * q]));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(&Bs[cur][(wn0 + j * 32 + r) * LK + (BK / 2) * h + 8 * q]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    store(cur ^ 1);
    __syncthreads();
  }
  nk_epilogue<EK, TM, TN>(p, acc, m0 + wm0, n0 + wn0, lane);
}

// ---------------------------------------------------------------- launch ---

static int64_t nk_ldk(int K) { return ((int64_t)K + 63) / 64 * 64; }
static int64_t nk_rows(int N) { return ((int64_t)N + 127) / 128 * 128; }

size_t gemm_nk_workspace(int32_t N, int32_t K, int32_t dtype) {
  const size_t el = dtype == PGCN_BF16 ? 2 : 4;
  return align_up((size_t)nk_rows(N) * (size_t)nk_ldk(K) * el, 256);
}

template <int BN, int AK, int EK>
static void nk_launch(const NKParams &p0, bool bf16, hipStream_t s) {
  constexpr int BM = 128;
  NKParams p = p0;
  const int tm = (p.M + BM - 1) / BM, tn = (p.N + BN - 1) / BN;
  p.tiles_n = tn;
  if (bf16) {
    constexpr int AKb = AK == NK_A_F32 ? NK_A_BF16 : AK;
    hipLaunchKernelGGL((gemm_nk_bf16<BM, BN, AKb, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  } else {
    hipLaunchKernelGGL((gemm_nk_f32<BM, BN, AK, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  }
}

template <int AK, int EK>
static void nk_launch_bn(const NKParams &p, bool bf16, hipStream_t s) {
  if (p.N <= 64) nk_launch<64, AK, EK>(p, bf16, s);
  else nk_launch<128, AK, EK>(p, bf16, s);
}

// kind: NN_* (forward: B(n,k) = W[k][n]) or MASK_NT_* (feature gradient:
// B(n,k) = W[n][k]); g.workspace holds the packed weights.
int launch_gemm_nk(Gemm kind, const GemmArgs &g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return PGCN_OK;
  const bool bf16 = g.dtype == PGCN_BF16;
  const size_t need = gemm_nk_workspace(g.N, g.K, g.dtype);
  if (!g.workspace || g.workspace_bytes < need)
    return set_error(PGCN_EWORKSPACE, "update GEMM: workspace too small for the packed weights");
  const int rows = (int)nk_rows(g.N), ldk = (int)nk_ldk(g.K);
  const bool fwd = kind == Gemm::NN_RELU || kind == Gemm::NN_PLAIN || kind == Gemm::NN_ACC_RELU ||
                   kind == Gemm::NN_ACC_PLAIN;
  {
    TraceScope ts(PGCN_TK_GEMM_PACK, s);
    const unsigned blocks = (unsigned)(((int64_t)rows * ldk + 255) / 256);
    if (bf16)
      hipLaunchKernelGGL(pack_b_kernel<true>, dim3(blocks), dim3(256), 0, s, g.B, (int)g.ldb, fwd ? 1 : 0, g.N, g.K,
                         rows, ldk, (void *)g.workspace);
    else
      hipLaunchKernelGGL(pack_b_kernel<false>, dim3(blocks), dim3(256), 0, s, g.B, (int)g.ldb, fwd ? 1 : 0, g.N,
                         g.K, rows, ldk, (void *)g.workspace);
    PGCN_HIP(hipGetLastError());
  }
  NKParams p{};
  p.M = g.M;
  p.N = g.N;
  p.K = g.K;
  p.A = g.A;
  p.A16 = g.A16;
  p.lda = g.lda;
  p.Am = g.Hmask;
  p.ldam = g.ldm;
  p.B = g.workspace;
  p.ldb = ldk;
  p.C = g.C;
  p.ldc = g.ldc;
  p.rowscale = g.rowscale;
  TraceScope ts(fwd ? PGCN_TK_GEMM_FWD : PGCN_TK_GEMM_DGRAD, s);
  switch (kind) {
    case Gemm::NN_RELU: nk_launch_bn<NK_A_F32, NK_E_RELU>(p, bf16, s); break;
    case Gemm::NN_PLAIN: nk_launch_bn<NK_A_F32, NK_E_PLAIN>(p, bf16, s); break;
    case Gemm::NN_ACC_RELU: nk_launch_bn<NK_A_F32, NK_E_ACC_RELU>(p, bf16, s); break;
    case Gemm::NN_ACC_PLAIN: nk_launch_bn<NK_A_F32, NK_E_ACC_PLAIN>(p, bf16, s); break;
    case Gemm::MASK_NT_ROWSCALE: nk_launch_bn<NK_A_MASK, NK_E_ROWSCALE>(p, bf16, s); break;
    case Gemm::MASK_NT_PLAIN: nk_launch_bn<NK_A_MASK, NK_E_PLAIN>(p, bf16, s); break;
    case Gemm::NT16_ROWSCALE:
    case Gemm::NT16_PLAIN:
      if (!bf16 || !p.A16) return set_error(PGCN_EINVAL, "launch_gemm_nk: NT16 needs the bf16 path and A16");
      if (kind == Gemm::NT16_ROWSCALE) nk_launch_bn<NK_A_F32, NK_E_ROWSCALE>(p, true, s);
      else nk_launch_bn<NK_A_F32, NK_E_PLAIN>(p, true, s);
      break;
    default: return set_error(PGCN_EINVAL, "launch_gemm_nk: not a node-major GEMM");
  }
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

}  // namespace pgcn

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
// (bf16) or 256-row (fp32) and 64-column multiple (bf16 rounded to nearest
// even for the bf16 path; three exact bf16 parts for fp32 by parts, below;
// fp32 for the plain fp32 kernel), so the main loop loads both operands as
// 16-byte vectors with no bounds checks on the weights.
//
// fp32 GEMMs run by parts on the bf16 matrix cores (gemm_nk_f32s) unless
// PGCN_GEMM_F32=native selects the fp32 matrix-core kernel (gemm_nk_f32).
//
// Main loop for CDNA4: a 256-thread workgroup (4 wave64s, 2 x 2) computes a
// 128 x BN tile; both tiles sit in LDS with k contiguous (rows of four
// 16-byte groups, XOR-swizzled by row so that staging writes and fragment
// reads are free of bank conflicts) and are double buffered, so one barrier
// per k-slab suffices while the next slab's global loads are in flight.
// Slabs are short (16 fp32 / 32 bf16 values of k) so that four workgroups fit
// per CU (32 KB of LDS, at most 128 VGPRs; three for the bf16 kernel with an
// fp32 masked operand): the staging of one workgroup's next slab (global load
// -> registers -> LDS) hides behind the others' MFMAs, which measured faster
// than longer slabs or deeper prefetch at two workgroups per CU.  The MFMA k
// order is permuted so that each lane's fragments over a slab are contiguous
// in LDS and load with 128-bit reads:
//   fp32, v_mfma_f32_32x32x2f32, slab of 16: step s uses k = 8*h + s for
//        lane half h (lanes 32h .. 32h+31);
//   fp32 by parts, v_mfma_f32_32x32x16_bf16, slab of 16: k = 8*h .. 8*h + 7;
//   bf16, v_mfma_f32_32x32x16_bf16, slab of 32: step j uses k = 16*h + 8*j
//        .. 16*h + 8*j + 7 for lane half h.
// Every k of the slab is used exactly once per output element.
#include <cstdlib>
#include <cstring>

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
  int64_t bplane;          // fp32 by parts: elements from one bf16 part of the packed weights to the next
  float *C;
  int64_t ldc;
  const float *rowscale;
  int vec;                 // C rows 16-byte aligned: ldc % 4 == 0 and C 16-byte aligned
  float *send;             // or null: final rows of C also written to send rows (stride ldc)
  const int64_t *send_ptr; // send rows of output row r: send_pos[send_ptr[r] .. send_ptr[r + 1])
  const int32_t *send_pos;
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
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;   // rows x ldk may pass 2^31 at the widest layers
  if (i >= (int64_t)rows * ldk) return;
  const int n = (int)(i / ldk), k = (int)(i - (int64_t)n * ldk);
  const float v = (n < N && k < K) ? (trans ? W[(int64_t)k * ldw + n] : W[(int64_t)n * ldw + k]) : 0.f;
  if (BF16) reinterpret_cast<uint16_t *>(out)[i] = nk_bf16(v);
  else reinterpret_cast<float *>(out)[i] = v;
}

// fp32 by parts: x = hi + mid + lo exactly, each part a bf16 (8 significant
// bits): hi is x with its low 16 bits cleared (never overflows), mid is
// x - hi rounded to nearest, and lo is what remains (at most 8 significant
// bits, so exact while |x| >= 2^-111; below, lo is a bf16 subnormal rounded
// to nearest).  Both differences are exact.  |mid| < 2^-7 |x| and
// |lo| <= 2^-15 |x|.  A non-finite x makes mid and lo NaN (Inf - Inf), so
// its products are NaN.  Two values at a time: returns the bf16 pairs
// (element 0 in the low half).
typedef __bf16 nk_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void nk_split3x2(float x0, float x1, uint32_t &hi, uint32_t &mid, uint32_t &lo) {
  const uint32_t b0 = __float_as_uint(x0), b1 = __float_as_uint(x1);
  const float r0 = x0 - __uint_as_float(b0 & 0xffff0000u), r1 = x1 - __uint_as_float(b1 & 0xffff0000u);
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);    // the high halves of b0 (low) and b1 (high)
  mid = __builtin_bit_cast(uint32_t, (nk_bf16x2){(__bf16)r0, (__bf16)r1});
  const float l0 = r0 - __uint_as_float(mid << 16), l1 = r1 - __uint_as_float(mid & 0xffff0000u);
  lo = __builtin_bit_cast(uint32_t, (nk_bf16x2){(__bf16)l0, (__bf16)l1});
}

// The packed weights as three bf16 planes (hi, mid, lo), `plane` elements apart;
// same indexing as pack_b_kernel.
__global__ __launch_bounds__(256) void pack_b_split_kernel(const float *W, int ldw, int trans, int N, int K, int rows,
                                                           int ldk, uint16_t *out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t plane = (int64_t)rows * ldk;
  if (i >= plane) return;
  const int n = (int)(i / ldk), k = (int)(i - (int64_t)n * ldk);
  const float v = (n < N && k < K) ? (trans ? W[(int64_t)k * ldw + n] : W[(int64_t)n * ldw + k]) : 0.f;
  uint32_t hi, mid, lo;
  nk_split3x2(v, 0.f, hi, mid, lo);
  out[i] = (uint16_t)hi;
  out[plane + i] = (uint16_t)mid;
  out[2 * plane + i] = (uint16_t)lo;
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

// Orders a wave's LDS accesses before and after this point (LDS operations of
// one wave complete in order; this keeps the compiler from moving them).
__device__ __forceinline__ void nk_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

constexpr int kNkStageLd = 36;                         // floats per staged row (32 + 4)
constexpr int kNkStageFloats = 4 * 32 * kNkStageLd;    // one 32 x 32 block per wave

// Stores the accumulators of one wave.  The MFMAs compute every 32 x 32 block
// transposed (the packed weights are the matrix core's left operand), so lane
// l holds output row l % 32 and, in registers 4q .. 4q+3, the columns
// 8q + 4(l / 32) .. +3 of the block; one row scale per lane suffices.  Each
// block passes through the wave's own LDS region and leaves as 16-byte
// vectors, eight lanes per row: every store instruction writes 8 whole rows of
// the block (128 contiguous bytes each).  Blocks inside C (all but the edge
// blocks; a wave-uniform test) load the old C of the accumulating forms before
// any store and store without per-element branches.
template <int EK, int TM, int TN>
__device__ __forceinline__ void nk_epilogue(const NKParams &p, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                            int lane, float *stage) {
  constexpr bool ACC = EK == NK_E_ACC_RELU || EK == NK_E_ACC_PLAIN;
  const int h = lane / 32, cl = lane % 32;
  const int rr = lane / 8, g = lane % 8;               // read layout: rows rr + 8s, columns 4g .. 4g+3
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = m0 + i * 32;
    const bool rows_in = mb + 32 <= p.M;
    const float sc = (EK == NK_E_ROWSCALE && mb + cl < p.M) ? p.rowscale[mb + cl] : 0.f;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = ACC ? acc[i][j][4 * q + e] : nk_out<EK>(acc[i][j][4 * q + e], sc, 0.f);
        *reinterpret_cast<f32x4 *>(stage + cl * kNkStageLd + 8 * q + 4 * h) = v;
      }
      nk_wave_sync();
      f32x4 v[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) v[s] = *reinterpret_cast<const f32x4 *>(stage + (rr + 8 * s) * kNkStageLd + 4 * g);
      nk_wave_sync();                                  // the next block's staging comes after these reads
      const int cb = n0 + j * 32 + 4 * g;
      float *c0 = p.C + (int64_t)(mb + rr) * p.ldc + cb;
      if (p.vec && rows_in && n0 + j * 32 + 32 <= p.N) {
        if (ACC) {
          f32x4 old[4];
#pragma unroll
          for (int s = 0; s < 4; ++s) old[s] = *reinterpret_cast<const f32x4 *>(c0 + (int64_t)(8 * s) * p.ldc);
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[s][e] = nk_out<EK>(v[s][e], 0.f, old[s][e]);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) *reinterpret_cast<f32x4 *>(c0 + (int64_t)(8 * s) * p.ldc) = v[s];
        if (p.send) {                                  // the same rows to their send slots
          int64_t kb[4], ke[4];
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            kb[s] = p.send_ptr[mb + rr + 8 * s];
            ke[s] = p.send_ptr[mb + rr + 8 * s + 1];
          }
          // one slot of each of the four rows per round: their position loads are issued together
          for (int i = 0;; ++i) {
            int32_t pos[4];
            bool any = false;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
              pos[s] = kb[s] + i < ke[s] ? p.send_pos[kb[s] + i] : -1;
              any |= pos[s] >= 0;
            }
            if (!any) break;
#pragma unroll
            for (int s = 0; s < 4; ++s)
              if (pos[s] >= 0)   // read by no kernel of this step: kept out of the caches
                __builtin_nontemporal_store(v[s], reinterpret_cast<f32x4 *>(p.send + (int64_t)pos[s] * p.ldc + cb));
          }
        }
      } else {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int row = mb + rr + 8 * s;
          if (row >= p.M) continue;
          float *c = c0 + (int64_t)(8 * s) * p.ldc;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (cb + e < p.N) {
              v[s][e] = ACC ? nk_out<EK>(v[s][e], 0.f, c[e]) : v[s][e];
              c[e] = v[s][e];
            }
          if (p.send)
            for (int64_t k = p.send_ptr[row]; k < p.send_ptr[row + 1]; ++k) {
              float *d = p.send + (int64_t)p.send_pos[k] * p.ldc + cb;
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (cb + e < p.N) d[e] = v[s][e];
            }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ fp32 ---

// 16-byte group g of LDS row `row` (4 groups per row) is stored at group
// g ^ ((row >> 2) & 3): the 16 lanes of one 16-byte access pass, whether 4
// rows x 4 groups (staging writes) or 16 rows x 1 group (fragment reads), then
// fall on 16 distinct 16-byte bank groups.
__device__ __forceinline__ int nk_sw(int row, int g) { return g ^ ((row >> 2) & 3); }

template <int BM, int BN, int AK, int EK>
__global__ __launch_bounds__(256, 4) void gemm_nk_f32(NKParams p) {
  constexpr int BK = 16, LK = BK, KV = BK / 4;        // rows of 4 16-byte groups, XOR-swizzled (nk_sw)
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 4 / 256, VB = BN * BK / 4 / 256;
  constexpr int SM = 2 * (BM + BN) * LK > kNkStageFloats ? 2 * (BM + BN) * LK : kNkStageFloats;
  __shared__ __attribute__((aligned(16))) float smem[SM];
  float(*As)[BM * LK] = reinterpret_cast<float(*)[BM * LK]>(smem);
  float(*Bs)[BN * LK] = reinterpret_cast<float(*)[BN * LK]>(smem + 2 * BM * LK);

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
      *reinterpret_cast<f32x4 *>(&As[b][(idx / KV) * LK + 4 * nk_sw(idx / KV, idx % KV)]) = x;
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      *reinterpret_cast<f32x4 *>(&Bs[b][(idx / KV) * LK + 4 * nk_sw(idx / KV, idx % KV)]) = rb[v];
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
        a[i] = *reinterpret_cast<const f32x4 *>(&As[cur][(wm0 + i * 32 + r) * LK + 4 * nk_sw(wm0 + i * 32 + r, 2 * h + q)]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = *reinterpret_cast<const f32x4 *>(&Bs[cur][(wn0 + j * 32 + r) * LK + 4 * nk_sw(wn0 + j * 32 + r, 2 * h + q)]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(b[j][e], a[i][e], acc[i][j], 0, 0, 0);
    }
    store(cur ^ 1);
    __syncthreads();
  }
  // the last barrier of the loop ends every LDS read of the main loop
  nk_epilogue<EK, TM, TN>(p, acc, m0 + wm0, n0 + wn0, lane, smem + wave * 32 * kNkStageLd);
}

// ------------------------------------------------------- fp32 by parts ---
//
// The fp32 GEMM on the bf16 matrix cores: both operands enter as three exact
// bf16 parts (nk_split3), and each 32 x 32 block accumulates, in fp32, the six
// part products whose order is at most 2^-16 of the full product:
//   hi.hi + hi.mid + mid.hi + hi.lo + mid.mid + lo.hi.
// The three dropped ones (mid.lo, lo.mid, lo.lo) are below 2^-21 (1 + 2^-7)
// |a b| together, and every part product is exact in fp32 (8 x 8 significant
// bits), so the result carries fp32 accuracy.  Six v_mfma_f32_32x32x16_bf16 per 16
// values of k take 192 matrix-core cycles, against 512 for the eight
// v_mfma_f32_32x32x2f32 of the plain fp32 kernel.  The weights arrive already
// split (pack_b_split_kernel); the activations are split once per workgroup
// while staged.  Slabs of 16 values of k: per operand three bf16 planes of
// 32-byte rows (two 16-byte groups, the second group first in rows 8 .. 15 of
// every 16 so that the 16 lanes of one 16-byte access pass fall on distinct
// banks), double buffered: 48 KB and three workgroups per CU for 128 x 128
// tiles, 72 KB and two for 128 x 256 (64 x 128 per wave: 48 matrix-core
// instructions per slab and wave, half the split work per instruction).  Lane
// half h takes k = 8h .. 8h + 7 of the slab on both operands.

__device__ __forceinline__ int nk_sw2(int row, int g) { return g ^ ((row >> 3) & 1); }

template <int BM, int BN, int AK, int EK>
__global__ __launch_bounds__(256, BN == 256 ? 2 : 3) void gemm_nk_f32s(NKParams p) {
  constexpr int BK = 16;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int PA = BM * BK, PB = BN * BK;             // bf16 elements of one plane
  constexpr int NB = 3 * BN * 2;                       // 16-byte vectors of the three weight planes
  constexpr int VB = (NB + 255) / 256;
  static_assert(BM == 128, "one 8-value vector of A per thread");
  constexpr int SMB = 2 * 3 * (PA + PB) * 2;
  constexpr int SM = SMB > kNkStageFloats * 4 ? SMB : kNkStageFloats * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SM];
  uint16_t *As = reinterpret_cast<uint16_t *>(smem);   // [2][3][PA]
  uint16_t *Bs = As + 2 * 3 * PA;                      // [2][3][PB]

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  const int tile = nk_xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;
  const uint16_t *Bp = reinterpret_cast<const uint16_t *>(p.B);

  // raw loads only; the row tail, the ReLU mask and the split are applied in
  // store(), after the MFMAs that hide the loads
  const int am = t / 2, ag = t % 2;                    // A: row am, values 8 ag .. 8 ag + 7 of the slab
  f32x4 rx[2], rh[AK == NK_A_MASK ? 2 : 1];
  u32x4 rb[VB];
  int kl = 0;
  auto load = [&](int kt) __attribute__((always_inline)) {
    kl = kt;
    const int gm = m0 + am, gk = kt + 8 * ag;
    const bool ok = gm < p.M && gk < p.K, ok1 = ok && gk + 4 < p.K;   // ld is a multiple of 4
    const float *row = p.A + (int64_t)gm * p.lda + gk;
    rx[0] = ok ? *reinterpret_cast<const f32x4 *>(row) : f32x4{0.f, 0.f, 0.f, 0.f};
    rx[1] = ok1 ? *reinterpret_cast<const f32x4 *>(row + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (AK == NK_A_MASK) {
      const float *hrow = p.Am + (int64_t)gm * p.ldam + gk;
      rh[0] = (ok && p.Am) ? *reinterpret_cast<const f32x4 *>(hrow) : f32x4{1.f, 1.f, 1.f, 1.f};
      rh[1] = (ok1 && p.Am) ? *reinterpret_cast<const f32x4 *>(hrow + 4) : f32x4{1.f, 1.f, 1.f, 1.f};
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      if (NB % 256 == 0 || idx < NB) {
        const int pl = idx / (2 * BN), n = (idx % (2 * BN)) / 2, g = idx % 2;
        rb[v] = *reinterpret_cast<const u32x4 *>(Bp + pl * p.bplane + (int64_t)(n0 + n) * p.ldb + kt + 8 * g);
      }
    }
  };
  auto store = [&](int b) __attribute__((always_inline)) {
    float x[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      x[q] = rx[q / 4][q % 4];
      if constexpr (AK == NK_A_MASK) x[q] = rh[q / 4][q % 4] > 0.f ? x[q] : 0.f;
    }
    if (kl + BK > p.K) {                               // the last slab (uniform): zero the k >= K tail
      const int valid = p.K - (kl + 8 * ag);
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q >= valid) x[q] = 0.f;
    }
    u32x4 oh, om, ol;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t hi, mid, lo;
      nk_split3x2(x[2 * w], x[2 * w + 1], hi, mid, lo);
      oh[w] = hi;
      om[w] = mid;
      ol[w] = lo;
    }
    const int off = am * BK + 8 * nk_sw2(am, ag);
    *reinterpret_cast<u32x4 *>(As + (b * 3 + 0) * PA + off) = oh;
    *reinterpret_cast<u32x4 *>(As + (b * 3 + 1) * PA + off) = om;
    *reinterpret_cast<u32x4 *>(As + (b * 3 + 2) * PA + off) = ol;
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      if (NB % 256 == 0 || idx < NB) {
        const int pl = idx / (2 * BN), n = (idx % (2 * BN)) / 2, g = idx % 2;
        *reinterpret_cast<u32x4 *>(Bs + (b * 3 + pl) * PB + n * BK + 8 * nk_sw2(n, g)) = rb[v];
      }
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
    load(kt + BK < p.K ? kt + BK : kt);                // as in gemm_nk_f32
    bf16x8 a[3][TM], b[3][TN];
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm0 + i * 32 + r;
        a[pl][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(
                                                  As + (cur * 3 + pl) * PA + row * BK + 8 * nk_sw2(row, h)));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = wn0 + j * 32 + r;
        b[pl][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(
                                                  Bs + (cur * 3 + pl) * PB + row * BK + 8 * nk_sw2(row, h)));
      }
    }
    // smallest products first; the TM x TN independent blocks between dependent steps
    constexpr int PW[6] = {2, 1, 0, 1, 0, 0}, PX[6] = {0, 1, 2, 0, 1, 0};   // parts of weights / activations
#pragma unroll
    for (int u = 0; u < 6; ++u)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[PW[u]][j], a[PX[u]][i], acc[i][j], 0, 0, 0);
    store(cur ^ 1);
    __syncthreads();
  }
  nk_epilogue<EK, TM, TN>(p, acc, m0 + wm0, n0 + wn0, lane, reinterpret_cast<float *>(smem) + wave * 32 * kNkStageLd);
}

// ------------------------------------------------------------------ bf16 ---

template <int BM, int BN, int AK, int EK>
__global__ __launch_bounds__(256, AK == NK_A_MASK ? 3 : 4) void gemm_nk_bf16(NKParams p) {
  constexpr int BK = 32, LK = BK, KV = BK / 8;         // bf16 elements; 64-byte rows, XOR-swizzled (nk_sw)
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  constexpr int VA = BM * BK / 8 / 256, VB = BN * BK / 8 / 256;
  constexpr int SM = 2 * (BM + BN) * LK * 2 > kNkStageFloats * 4 ? 2 * (BM + BN) * LK * 2 : kNkStageFloats * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SM];
  uint16_t(*As)[BM * LK] = reinterpret_cast<uint16_t(*)[BM * LK]>(smem);
  uint16_t(*Bs)[BN * LK] = reinterpret_cast<uint16_t(*)[BN * LK]>(smem + 2 * BM * LK * 2);

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
      *reinterpret_cast<u32x4 *>(&As[b][(idx / KV) * LK + 8 * nk_sw(idx / KV, idx % KV)]) = o;
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int idx = t + 256 * v;
      *reinterpret_cast<u32x4 *>(&Bs[b][(idx / KV) * LK + 8 * nk_sw(idx / KV, idx % KV)]) = rb[v];
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
        a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(
                                              &As[cur][(wm0 + i * 32 + r) * LK + 8 * nk_sw(wm0 + i * 32 + r, 2 * h + q)]));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(
                                              &Bs[cur][(wn0 + j * 32 + r) * LK + 8 * nk_sw(wn0 + j * 32 + r, 2 * h + q)]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
    }
    store(cur ^ 1);
    __syncthreads();
  }
  nk_epilogue<EK, TM, TN>(p, acc, m0 + wm0, n0 + wn0, lane, reinterpret_cast<float *>(smem) + wave * 32 * kNkStageLd);
}

// ---------------------------------------------------------------- launch ---

static int64_t nk_ldk(int K) { return ((int64_t)K + 63) / 64 * 64; }
static int64_t nk_rows(int N, bool bf16) { return bf16 ? ((int64_t)N + 127) / 128 * 128 : ((int64_t)N + 255) / 256 * 256; }

// fp32 GEMMs by parts (the default) or on the fp32 matrix cores
// (PGCN_GEMM_F32=native, a tuning override read per call)
static bool nk_f32_by_parts() {
  const char *e = std::getenv("PGCN_GEMM_F32");
  return !(e && std::strcmp(e, "native") == 0);
}

// fp32: room for the three bf16 planes of the split weights (6 bytes per element) in either mode
size_t gemm_nk_workspace(int32_t N, int32_t K, int32_t dtype) {
  const size_t el = dtype == PGCN_BF16 ? 2 : 6;
  return align_up((size_t)nk_rows(N, dtype == PGCN_BF16) * (size_t)nk_ldk(K) * el, 256);
}

template <int BN, int AK, int EK>
static void nk_launch(const NKParams &p0, bool bf16, hipStream_t s) {
  constexpr int BM = 128;
  NKParams p = p0;
  const int tm = (p.M + BM - 1) / BM, tn = (p.N + BN - 1) / BN;
  p.tiles_n = tn;
  if constexpr (BN == 256) {                           // fp32 by parts only
    hipLaunchKernelGGL((gemm_nk_f32s<BM, BN, AK, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  } else if (bf16) {
    constexpr int AKb = AK == NK_A_F32 ? NK_A_BF16 : AK;
    hipLaunchKernelGGL((gemm_nk_bf16<BM, BN, AKb, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  } else if (p.bplane > 0) {
    hipLaunchKernelGGL((gemm_nk_f32s<BM, BN, AK, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  } else {
    hipLaunchKernelGGL((gemm_nk_f32<BM, BN, AK, EK>), dim3((unsigned)(tm * tn)), dim3(256), 0, s, p);
  }
}

// Tile width: 64 for narrow outputs; by parts, 256 (twice the matrix-core work
// per staged A value and per slab) where that pads no more columns than 128.
template <int AK, int EK>
static void nk_launch_bn(const NKParams &p, bool bf16, hipStream_t s) {
  if (p.N <= 64) nk_launch<64, AK, EK>(p, bf16, s);
  else if (p.bplane > 0 && (p.N + 255) / 256 * 2 == (p.N + 127) / 128) nk_launch<256, AK, EK>(p, bf16, s);
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
  const int rows = (int)nk_rows(g.N, bf16), ldk = (int)nk_ldk(g.K);
  const bool fwd = kind == Gemm::NN_RELU || kind == Gemm::NN_PLAIN || kind == Gemm::NN_ACC_RELU ||
                   kind == Gemm::NN_ACC_PLAIN || kind == Gemm::NN_SRC32_PLAIN || kind == Gemm::NN_SRC32_ROWSCALE ||
                   kind == Gemm::NN_SRC32_RELU;
  const bool parts = !bf16 && nk_f32_by_parts();
  {
    TraceScope ts(PGCN_TK_GEMM_PACK, s);
    const unsigned blocks = (unsigned)(((int64_t)rows * ldk + 255) / 256);
    if (parts)
      hipLaunchKernelGGL(pack_b_split_kernel, dim3(blocks), dim3(256), 0, s, g.B, (int)g.ldb, fwd ? 1 : 0, g.N, g.K,
                         rows, ldk, reinterpret_cast<uint16_t *>(g.workspace));
    else if (bf16)
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
  p.bplane = parts ? (int64_t)rows * ldk : 0;
  p.C = g.C;
  p.ldc = g.ldc;
  p.rowscale = g.rowscale;
  p.vec = (g.ldc % 4 == 0 && (reinterpret_cast<uintptr_t>(g.C) & 15) == 0) ? 1 : 0;
  if (g.send) {
    if (!fwd || !g.send_ptr || !g.send_pos || ((reinterpret_cast<uintptr_t>(g.send) & 15) && p.vec))
      return set_error(PGCN_EINVAL, "update GEMM: send rows need a forward kind, the send map and 16-byte alignment");
    p.send = g.send;
    p.send_ptr = g.send_ptr;
    p.send_pos = g.send_pos;
  }
  TraceScope ts(fwd ? PGCN_TK_GEMM_FWD : PGCN_TK_GEMM_DGRAD, s);
  switch (kind) {
    case Gemm::NN_RELU: nk_launch_bn<NK_A_F32, NK_E_RELU>(p, bf16, s); break;
    case Gemm::NN_PLAIN: nk_launch_bn<NK_A_F32, NK_E_PLAIN>(p, bf16, s); break;
    case Gemm::NN_ACC_RELU: nk_launch_bn<NK_A_F32, NK_E_ACC_RELU>(p, bf16, s); break;
    case Gemm::NN_ACC_PLAIN: nk_launch_bn<NK_A_F32, NK_E_ACC_PLAIN>(p, bf16, s); break;
    case Gemm::NN_SRC32_PLAIN:                         // fp32 operand; on the bf16 path rounded while staged
    case Gemm::NN_SRC32_ROWSCALE:
    case Gemm::NN_SRC32_RELU:
      if (!p.A) return set_error(PGCN_EINVAL, "launch_gemm_nk: NN_SRC32 needs the fp32 operand");
      if (kind == Gemm::NN_SRC32_ROWSCALE && !p.rowscale)
        return set_error(PGCN_EINVAL, "launch_gemm_nk: NN_SRC32_ROWSCALE needs the row scales");
      p.Am = nullptr;
      if (kind == Gemm::NN_SRC32_PLAIN) {
        if (bf16) nk_launch_bn<NK_A_MASK, NK_E_PLAIN>(p, true, s);
        else nk_launch_bn<NK_A_F32, NK_E_PLAIN>(p, false, s);
      } else if (kind == Gemm::NN_SRC32_RELU) {
        if (bf16) nk_launch_bn<NK_A_MASK, NK_E_RELU>(p, true, s);
        else nk_launch_bn<NK_A_F32, NK_E_RELU>(p, false, s);
      } else {
        if (bf16) nk_launch_bn<NK_A_MASK, NK_E_ROWSCALE>(p, true, s);
        else nk_launch_bn<NK_A_F32, NK_E_ROWSCALE>(p, false, s);
      }
      break;
    case Gemm::MASK_NT_ROWSCALE: nk_launch_bn<NK_A_MASK, NK_E_ROWSCALE>(p, bf16, s); break;
    case Gemm::MASK_NT_PLAIN: nk_launch_bn<NK_A_MASK, NK_E_PLAIN>(p, bf16, s); break;
    case Gemm::NT_SRC32_ACC_PLAIN:                     // C += A W^T, fp32 A rounded while staged on bf16
      if (!p.A) return set_error(PGCN_EINVAL, "launch_gemm_nk: NT_SRC32 needs the fp32 operand");
      p.Am = nullptr;
      if (bf16) nk_launch_bn<NK_A_MASK, NK_E_ACC_PLAIN>(p, true, s);
      else nk_launch_bn<NK_A_F32, NK_E_ACC_PLAIN>(p, false, s);
      break;
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

// Weight-gradient GEMM of a GCN layer (Appendix A.1; the G of Algorithm 1):
//     G = A^T (J ∘ 1[H > 0])        [f_in x f_out], a sum over the inner rows
// A [n, f_in], J and H [n, f_out] are node-major, so the reduction index k is
// the node.  The node range is cut into fixed splits; each workgroup computes
// one output tile over one split into a partial tile, and a second kernel adds
// the partials in split order (deterministic, no atomics).
//
// Main loop for CDNA4: 256 threads (4 wave64s, 2 x 2) per 128 x BN tile; slabs
// of nodes are staged through double-buffered LDS, one barrier per slab, with
// the next slab's global loads in flight during the MFMAs.  Both operands are
// transposed on the way into LDS (one row per feature, nodes contiguous) so a
// lane's MFMA fragments over a slab are contiguous and load with 128-bit
// reads: a thread loads a block of 4 nodes x 4 features (fp32; 8 features for
// bf16 A) as 16-byte vectors and writes one node-contiguous vector per
// feature.  Feature 4u + e (8u + e for bf16 A) is kept in LDS row e * U + u
// (U = tile width / 4 or / 8), which puts the lanes of one LDS write on
// distinct banks; the epilogue maps rows back to features.  The ReLU mask and
// the bf16 rounding are applied after the MFMAs, just before the LDS write, so
// the global loads stay in flight under the MFMAs.
//   fp32: slabs of 16 nodes, v_mfma_f32_32x32x2f32; step e of group q uses
//         node 8h + 4q + e for lane half h;
//   bf16: slabs of 32 nodes, A already bf16 in memory, J ∘ mask rounded to
//         bf16 (nearest even); v_mfma_f32_32x32x16_bf16, step q uses nodes
//         16q + 8h .. 16q + 8h + 7 for lane half h.  The first row of tiles
//         can also write the rounded J ∘ mask node-major for the feature
//         gradient.
// The grid is one-dimensional over (split, tile) with the tiles of a split
// adjacent and on the same XCD, so each split's rows of A, J and H come from
// HBM about once and are re-read from that XCD's L2.
// A transform-first layer sums over inner and boundary rows: rows k >= ksplit
// of the left operand come from a second matrix (A_hi), and on the bf16 path
// that operand is fp32 in memory and rounded while staged (template A32).
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "internal.h"

namespace pgcn {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct TNParams {
  int M, N, K;            // M = f_in, N = f_out, K = node count
  int kchunk;             // nodes per split (a multiple of the slab)
  int tiles, tiles_n;
  const float *A;         // fp32 [min(K, ksplit), lda]
  const uint16_t *A16;    // bf16 [K, lda]
  int64_t lda;
  const float *A_hi;      // fp32 rows k >= ksplit (row k - ksplit, stride lda), or null: zero rows
  int ksplit;             // K when there is no second matrix
  const float *J;         // [K, ldb]
  int64_t ldb;
  const float *H;         // mask source [K, ldh], or null (no ReLU)
  int64_t ldh;
  float *partials;        // [splits, M, N]
  uint16_t *M16;          // bf16 path: bf16(J ∘ mask) [K, ldm16] written by the first row of tiles, or null
  int64_t ldm16;
};

__device__ __forceinline__ uint32_t tn_bf16(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (b >> 16) | 0x40u;
  b += 0x7fffu + ((b >> 16) & 1u);
  return b >> 16;
}

// (split, tile) of this workgroup: logical index l = split * tiles + tile, with
// workgroup b (dispatched to XCD b % 8) taking l = (b % 8) * (G / 8) + b / 8
__device__ __forceinline__ void tn_coords(int tiles, int &split, int &tile) {
  const int g = gridDim.x, b = blockIdx.x;
  const int l = (g % 8 == 0) ? (b % 8) * (g / 8) + b / 8 : b;
  split = l / tiles;
  tile = l - split * tiles;
}

// partial[split][fm][fn] for the accumulators of one wave; LDS row c holds
// feature 4 * (c % UA) + c / UA of the A tile (VA features per vector)
template <int TM, int TN, int UA, int VA, int UB>
__device__ __forceinline__ void tn_store_partial(const TNParams &p, const f32x16 (&acc)[TM][TN], int split, int m0,
                                                 int n0, int wm0, int wn0, int lane) {
  float *out = p.partials + (int64_t)split * p.M * p.N;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int cn = wn0 + j * 32 + lane % 32;
    const int fn = n0 + 4 * (cn % UB) + cn / UB;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int cm = wm0 + i * 32 + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
        const int fm = m0 + VA * (cm % UA) + cm / UA;
        if (fm < p.M && fn < p.N) out[(int64_t)fm * p.N + fn] = acc[i][j][r];
      }
  }
}

// ------------------------------------------------------------------ fp32 ---
//
// v_mfma_f32_32x32x2f32 takes one node per lane half (k = lane / 32), so the
// fp32 kernel keeps both tiles node-major in LDS (rows of 128 + 32 floats: the
// two lane halves read rows k and k + 1 on disjoint banks) and needs no
// transpose: every thread stages 16-byte vectors of whole node rows (A, J and
// H alike, coalesced over the row), and the next-but-one slab is loaded into a
// second register set, so each load has two slabs of MFMAs to arrive.

template <int BM, int BN>
__global__ __launch_bounds__(256, BN == 128 ? 2 : 3) void gemm_tn_f32(TNParams p) {
  constexpr int BK = 16;                               // BK nodes per slab
  constexpr int LDA = BM + 32, LDB = BN + 32;
  constexpr int VA = BK * BM / 4 / 256, VB = BK * BN / 4 / 256;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  static_assert(VA >= 1 && VB >= 1, "slab smaller than the workgroup");
  __shared__ __attribute__((aligned(16))) float As[2][BK * LDA];
  __shared__ __attribute__((aligned(16))) float Bs[2][BK * LDB];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  int split, tile;
  tn_coords(p.tiles, split, tile);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = split * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;
  const bool masked = p.H != nullptr;
  // vector v of this thread: node (t + 256 v) / (B/4) of the slab, features 4 ((t + 256 v) % (B/4)) ..
  const int ca = 4 * (t % (BM / 4)), na = t / (BM / 4);
  const int cb = 4 * (t % (BN / 4)), nb = t / (BN / 4);
  constexpr int SA = 256 / (BM / 4), SB = 256 / (BN / 4);   // node step between a thread's vectors
  const bool fa = m0 + ca < p.M, fb = n0 + cb < p.N;

  struct Regs {
    f32x4 a[VA], b[VB], h[VB];
  };
  auto load = [&](Regs &R, int kt) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < VA; ++v) {
      const int node = kt + na + SA * v;
      const bool hi = node >= p.ksplit;                 // boundary rows of a transform-first layer
      const float *src = hi ? p.A_hi : p.A;
      const bool ok = fa && node < kend && src != nullptr;
      const int64_t row = hi ? node - p.ksplit : node;
      R.a[v] = ok ? *reinterpret_cast<const f32x4 *>(src + row * p.lda + m0 + ca) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      const int node = kt + nb + SB * v;
      const bool ok = fb && node < kend;
      R.b[v] = ok ? *reinterpret_cast<const f32x4 *>(p.J + (int64_t)node * p.ldb + n0 + cb)
                  : f32x4{0.f, 0.f, 0.f, 0.f};
      if (masked)
        R.h[v] = ok ? *reinterpret_cast<const f32x4 *>(p.H + (int64_t)node * p.ldh + n0 + cb)
                    : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto store = [&](Regs &R, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < VA; ++v) *reinterpret_cast<f32x4 *>(&As[buf][(na + SA * v) * LDA + ca]) = R.a[v];
#pragma unroll
    for (int v = 0; v < VB; ++v) {
      f32x4 x = R.b[v];
      if (masked) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = R.h[v][e] > 0.f ? x[e] : 0.f;
      }
      *reinterpret_cast<f32x4 *>(&Bs[buf][(nb + SB * v) * LDB + cb]) = x;
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < BK / 2; ++s) {                 // nodes 2s (lanes 0-31) and 2s + 1 (lanes 32-63)
      const float *ar = &As[buf][(2 * s + h) * LDA + wm0 + r];
      const float *br = &Bs[buf][(2 * s + h) * LDB + wn0 + r];
      float a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = ar[i * 32];
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = br[j * 32];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  const int ns = (kend - kbeg + BK - 1) / BK;          // slabs of this split (<= 0: none)
  if (ns > 0 && BM == 128) {
    Regs R0, R1;
    load(R0, kbeg);
    load(R1, kbeg + BK);                               // past kend: zero vectors, no loads
    store(R0, 0);
    __syncthreads();
    for (int sl = 0; sl < ns; sl += 2) {
      load(R0, kbeg + (sl + 2) * BK);
      compute(0);
      store(R1, 1);
      __syncthreads();
      if (sl + 1 >= ns) break;
      load(R1, kbeg + (sl + 3) * BK);
      compute(1);
      store(R0, 0);
      __syncthreads();
    }
  } else if (ns > 0) {
    // 256-row tiles: a slab's MFMAs take twice as long, so loads one slab
    // ahead have time to arrive, and one register set leaves room for the
    // 128 accumulators
    Regs R0;
    load(R0, kbeg);
    store(R0, 0);
    __syncthreads();
    for (int sl = 0; sl < ns; ++sl) {
      load(R0, kbeg + (sl + 1) * BK);
      compute(sl & 1);
      store(R0, (sl + 1) & 1);
      __syncthreads();
    }
  }

  // output: row = A feature m0 + wm0 + 32 i + 8 (reg / 4) + 4 h + reg % 4, column = J feature n0 + wn0 + 32 j + r
  float *out = p.partials + (int64_t)split * p.M * p.N;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int fn = n0 + wn0 + j * 32 + r;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int fm = m0 + wm0 + i * 32 + 8 * (q / 4) + 4 * h + (q % 4);
        if (fm < p.M && fn < p.N) out[(int64_t)fm * p.N + fn] = acc[i][j][q];
      }
  }
}

// -------------------------------------------------------- fp32 by parts ---
//
// The fp32 weight gradient on the bf16 matrix cores, as the node-major fp32
// GEMMs do it: A and J ∘ mask enter as three exact bf16 parts each (hi = x
// with its low 16 bits cleared, mid = x - hi rounded to nearest, lo = the
// rest), and each block accumulates in fp32 the six part products hi.hi,
// hi.mid, mid.hi, hi.lo, mid.mid, lo.hi (the three dropped ones are below
// 2^-21 (1 + 2^-7) |a b| together).  Slabs of 16 nodes, one
// v_mfma_f32_32x32x16_bf16 step per part product; both operands transposed
// into LDS (one row per feature, 16 nodes = two 16-byte groups, the groups
// swapped in rows 8 .. 15 of every 16), three planes each, double buffered
// (48 KB, three workgroups per CU).  Thread item: 4 nodes x 4 features of A
// (threads 0 .. 127) or of J (threads 128 ..), node quad fastest, so the 32
// lanes of one 8-byte LDS write pass cover 8 whole rows; feature 4u + e sits
// in LDS row e U + u.  Lane half h takes nodes 8h .. 8h + 7 of the slab.

__device__ __forceinline__ void tn_split3x2(float x0, float x1, uint32_t &hi, uint32_t &mid, uint32_t &lo) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const uint32_t b0 = __float_as_uint(x0), b1 = __float_as_uint(x1);
  const float r0 = x0 - __uint_as_float(b0 & 0xffff0000u), r1 = x1 - __uint_as_float(b1 & 0xffff0000u);
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);    // the high halves of b0 (low) and b1 (high)
  mid = __builtin_bit_cast(uint32_t, (bf16x2){(__bf16)r0, (__bf16)r1});
  const float l0 = r0 - __uint_as_float(mid << 16), l1 = r1 - __uint_as_float(mid & 0xffff0000u);
  lo = __builtin_bit_cast(uint32_t, (bf16x2){(__bf16)l0, (__bf16)l1});
}

__device__ __forceinline__ int tn_sw2(int row, int g) { return g ^ ((row >> 3) & 1); }

// Raw loads of one thread item: nodes nq .. nq + 3 (zero past kend or for an
// absent operand), features col .. col + 3; rows >= ksplit come from src_hi
// (row - ksplit).  hsrc: the mask source (left at 1 when null).
__device__ __forceinline__ void tn_parts_load(f32x4 (&x)[4], f32x4 (&hm)[4], const float *src_lo, const float *src_hi,
                                              const float *hsrc, int64_t ld_src, int64_t ld_h, int ksplit, int nq,
                                              int kend, int col, bool fok) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int node = nq + s;
    const bool hi = node >= ksplit;
    const float *src = hi ? src_hi : src_lo;
    const bool ok = fok && node < kend && src != nullptr;
    const int64_t row = hi ? node - ksplit : node;
    x[s] = ok ? *reinterpret_cast<const f32x4 *>(src + row * ld_src + col) : f32x4{0.f, 0.f, 0.f, 0.f};
    if (hsrc) hm[s] = (fok && node < kend) ? *reinterpret_cast<const f32x4 *>(hsrc + (int64_t)node * ld_h + col)
                                           : f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// Masks, splits and writes one thread item into the three planes at base
// (plane elements apart): feature e of quad uq in row e U + uq, node quad kq.
__device__ __forceinline__ void tn_parts_store(const f32x4 (&x)[4], const f32x4 (&hm)[4], uint16_t *base, int plane,
                                               int U, int uq, int kq) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float v0 = hm[0][e] > 0.f ? x[0][e] : 0.f, v1 = hm[1][e] > 0.f ? x[1][e] : 0.f;
    const float v2 = hm[2][e] > 0.f ? x[2][e] : 0.f, v3 = hm[3][e] > 0.f ? x[3][e] : 0.f;
    uint32_t hi01, mi01, lo01, hi23, mi23, lo23;
    tn_split3x2(v0, v1, hi01, mi01, lo01);
    tn_split3x2(v2, v3, hi23, mi23, lo23);
    const int row = e * U + uq;
    const int off = row * 16 + 8 * tn_sw2(row, kq / 2) + 4 * (kq % 2);
    *reinterpret_cast<u32x2 *>(base + off) = u32x2{hi01, hi23};
    *reinterpret_cast<u32x2 *>(base + plane + off) = u32x2{mi01, mi23};
    *reinterpret_cast<u32x2 *>(base + 2 * plane + off) = u32x2{lo01, lo23};
  }
}

template <int BN>
__global__ __launch_bounds__(256, 3) void gemm_tn_f32s(TNParams p) {
  constexpr int BM = 128, BK = 16;
  constexpr int UA = BM / 4, UB = BN / 4;              // feature quads of the tiles
  constexpr int PA = BM * BK, PB = BN * BK;            // bf16 elements of one plane
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  static_assert(UA * 4 == 128 && UB * 4 <= 128, "one item per thread");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][3][PA];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][3][PB];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  int split, tile;
  tn_coords(p.tiles, split, tile);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = split * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;

  const bool isA = t < 128;                            // wave-uniform
  const int it = isA ? t : t - 128;
  const int kq = it % 4, uq = it / 4;                  // node quad, feature quad
  const bool hasB = !isA && uq < UB;
  const bool fok = isA ? m0 + 4 * uq < p.M : (hasB && n0 + 4 * uq < p.N);

  // this thread's operand rows: A (rows >= ksplit from A_hi) or J and its mask source H
  const float *src_lo = isA ? p.A : p.J, *src_hi = isA ? p.A_hi : nullptr, *hsrc = isA ? nullptr : p.H;
  const int64_t ld_src = isA ? p.lda : p.ldb, ld_h = p.ldh;
  const int ksplit = isA ? p.ksplit : p.K, col = (isA ? m0 : n0) + 4 * uq;
  f32x4 x[4], hm[4];                                   // node s of the quad: features col .. col + 3
#pragma unroll
  for (int s = 0; s < 4; ++s) hm[s] = f32x4{1.f, 1.f, 1.f, 1.f};
  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  if (kbeg < kend) {
    tn_parts_load(x, hm, src_lo, src_hi, hsrc, ld_src, ld_h, ksplit, kbeg + 4 * kq, kend, col, fok);
    if (isA || hasB)
      tn_parts_store(x, hm, isA ? &As[0][0][0] : &Bs[0][0][0], isA ? PA : PB, isA ? UA : UB, uq, kq);
    __syncthreads();
    int itn = 0;
    for (int kt = kbeg; kt < kend; kt += BK, ++itn) {
      const int cur = itn & 1;
      tn_parts_load(x, hm, src_lo, src_hi, hsrc, ld_src, ld_h, ksplit, (kt + BK < kend ? kt + BK : kt) + 4 * kq,
                    kend, col, fok);
      bf16x8 a[3][TM], b[3][TN];
#pragma unroll
      for (int pl = 0; pl < 3; ++pl) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int row = wm0 + i * 32 + r;
          a[pl][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(&As[cur][pl][row * BK + 8 * tn_sw2(row, h)]));
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int row = wn0 + j * 32 + r;
          b[pl][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(&Bs[cur][pl][row * BK + 8 * tn_sw2(row, h)]));
        }
      }
      constexpr int PX[6] = {2, 1, 0, 1, 0, 0}, PY[6] = {0, 1, 2, 0, 1, 0};   // parts of A / of J, smallest first
#pragma unroll
      for (int u = 0; u < 6; ++u)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[PX[u]][i], b[PY[u]][j], acc[i][j], 0, 0, 0);
      if (isA || hasB)
        tn_parts_store(x, hm, isA ? &As[cur ^ 1][0][0] : &Bs[cur ^ 1][0][0], isA ? PA : PB, isA ? UA : UB, uq, kq);
      __syncthreads();
    }
  }
  tn_store_partial<TM, TN, UA, 4, UB>(p, acc, split, m0, n0, wm0, wn0, lane);
}

// 256 x 128 tiles by parts (each wave 128 x 64): twice the matrix-core work
// of a 128 x 128 tile for 4/3 of its staged bytes, since the staging (the
// vector-memory path), not the matrix cores, bounds the narrower tile.  Every
// thread stages an A item (4 nodes x 4 of the 256 features); threads 0 .. 127
// also stage a J item.  72 KB of LDS, two workgroups per CU; the A parts are
// read from LDS one plane at a time to leave room for the 128 accumulators.
__global__ __launch_bounds__(256, 2) void gemm_tn_f32s_wide(TNParams p) {
  constexpr int BM = 256, BN = 128, BK = 16;
  constexpr int UA = BM / 4, UB = BN / 4;
  constexpr int PA = BM * BK, PB = BN * BK;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][3][PA];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][3][PB];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  int split, tile;
  tn_coords(p.tiles, split, tile);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = split * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;

  const int kq = t % 4, uq = t / 4;                    // node quad; feature quad (A: all, J: t < 128)
  const bool hasB = t < 128;                           // waves 0 and 1
  const bool fa = m0 + 4 * uq < p.M, fb = hasB && n0 + 4 * uq < p.N;
  f32x4 xa[4], ha[4], xb[4], hb[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    ha[s] = f32x4{1.f, 1.f, 1.f, 1.f};
    hb[s] = f32x4{1.f, 1.f, 1.f, 1.f};
  }
  auto load = [&](int kt) __attribute__((always_inline)) {
    const int nq = kt + 4 * kq;
    tn_parts_load(xa, ha, p.A, p.A_hi, nullptr, p.lda, 0, p.ksplit, nq, kend, m0 + 4 * uq, fa);
    if (hasB) tn_parts_load(xb, hb, p.J, nullptr, p.H, p.ldb, p.ldh, p.K, nq, kend, n0 + 4 * uq, fb);
  };
  auto store = [&](int b) __attribute__((always_inline)) {
    tn_parts_store(xa, ha, &As[b][0][0], PA, UA, uq, kq);
    if (hasB) tn_parts_store(xb, hb, &Bs[b][0][0], PB, UB, uq, kq);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  if (kbeg < kend) {
    load(kbeg);
    store(0);
    __syncthreads();
    int itn = 0;
    for (int kt = kbeg; kt < kend; kt += BK, ++itn) {
      const int cur = itn & 1;
      load(kt + BK < kend ? kt + BK : kt);
      bf16x8 b[3][TN];
#pragma unroll
      for (int pl = 0; pl < 3; ++pl)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int row = wn0 + j * 32 + r;
          b[pl][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(&Bs[cur][pl][row * BK + 8 * tn_sw2(row, h)]));
        }
      // A parts lo, mid, hi in turn, each with the J parts that keep its products (smallest first)
#pragma unroll
      for (int pa = 2; pa >= 0; --pa) {
        bf16x8 a[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int row = wm0 + i * 32 + r;
          a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(&As[cur][pa][row * BK + 8 * tn_sw2(row, h)]));
        }
#pragma unroll
        for (int pb = 2 - pa; pb >= 0; --pb)
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[pb][j], acc[i][j], 0, 0, 0);
      }
      store(cur ^ 1);
      __syncthreads();
    }
  }
  tn_store_partial<TM, TN, UA, 4, UB>(p, acc, split, m0, n0, wm0, wn0, lane);
}

// ------------------------------------------------------------------ bf16 ---

template <int BN, bool A32>
__global__ __launch_bounds__(256, (BN == 128 && A32) ? 2 : 3) void gemm_tn_bf16(TNParams p) {
  constexpr int BM = 128, BK = 32, LK = BK + 8;       // bf16 elements; 80-byte rows
  constexpr int UA = BM / 8, UB = BN / 4;
  constexpr int NA = UA * (BK / 4), NB = UB * (BK / 4);
  static_assert(NA <= 256 && NB <= 256 && (NB == 256 || NA + NB <= 256), "staging items exceed the workgroup");
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LK];

  const int t = threadIdx.x, lane = t % 64, wave = __builtin_amdgcn_readfirstlane(t / 64);
  int split, tile;
  tn_coords(p.tiles, split, tile);
  const int m0 = (tile / p.tiles_n) * BM, n0 = (tile % p.tiles_n) * BN;
  const int kbeg = split * p.kchunk;
  const int kend = min(p.K, kbeg + p.kchunk);
  const int wm0 = (wave / 2) * WM, wn0 = (wave % 2) * WN;

  // A blocks (4 nodes x 8 features) on threads [0, NA); J/H blocks (4 nodes x
  // 4 features) on every thread when there are 256 of them, else after the A threads
  const bool hasA = t < NA;
  const int ua = t % UA, ka = t / UA;
  const bool aok = hasA && m0 + 8 * ua < p.M;
  const int ib = NB == 256 ? t : t - NA;
  const bool hasB = ib >= 0 && ib < NB;
  const int ub = ib % UB, kb = ib / UB;
  const bool bok = hasB && n0 + 4 * ub < p.N;
  const bool masked = p.H != nullptr;

  const bool write_m16 = p.M16 != nullptr && m0 == 0 && bok;
  const bool aok1 = aok && m0 + 8 * ua + 4 < p.M;     // A32: the second half-vector lies inside the row
  u32x4 xa[4];
  f32x4 xf[A32 ? 8 : 1];                               // A32: fp32 rows, rounded in store()
  f32x4 xb[4], hm[4];
  int kl = 0;                                          // node of the staged slab
  auto load = [&](int kt) __attribute__((always_inline)) {
    kl = kt;
    if (hasA) {
      const int gk = kt + 4 * ka;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (A32) {
          const int node = gk + s;
          const bool hi = node >= p.ksplit;
          const float *src = hi ? p.A_hi : p.A;
          const bool ok = aok && node < kend && src != nullptr;
          const float *row = src + (int64_t)(hi ? node - p.ksplit : node) * p.lda + m0 + 8 * ua;
          xf[2 * s] = ok ? *reinterpret_cast<const f32x4 *>(row) : f32x4{0.f, 0.f, 0.f, 0.f};
          xf[2 * s + 1] = (ok && aok1) ? *reinterpret_cast<const f32x4 *>(row + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        } else {
          xa[s] = (aok && gk + s < kend)
                      ? *reinterpret_cast<const u32x4 *>(p.A16 + (int64_t)(gk + s) * p.lda + m0 + 8 * ua)
                      : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
    if (hasB) {
      const int gk = kt + 4 * kb;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bool ok = bok && gk + s < kend;
        xb[s] = ok ? *reinterpret_cast<const f32x4 *>(p.J + (int64_t)(gk + s) * p.ldb + n0 + 4 * ub)
                   : f32x4{0.f, 0.f, 0.f, 0.f};
        if (masked)
          hm[s] = ok ? *reinterpret_cast<const f32x4 *>(p.H + (int64_t)(gk + s) * p.ldh + n0 + 4 * ub)
                     : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  auto store = [&](int b) __attribute__((always_inline)) {
    if (hasA) {
      if (A32) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int w = 0; w < 4; ++w)
            xa[s][w] = tn_bf16(xf[2 * s + w / 2][2 * (w % 2)]) | (tn_bf16(xf[2 * s + w / 2][2 * (w % 2) + 1]) << 16);
      }
#pragma unroll
      for (int w = 0; w < 4; ++w) {            // features 2w (low halves) and 2w + 1 (high halves)
        const u32x2 lo{(xa[0][w] & 0xffffu) | (xa[1][w] << 16), (xa[2][w] & 0xffffu) | (xa[3][w] << 16)};
        const u32x2 hi{(xa[0][w] >> 16) | (xa[1][w] & 0xffff0000u), (xa[2][w] >> 16) | (xa[3][w] & 0xffff0000u)};
        *reinterpret_cast<u32x2 *>(&As[b][((2 * w) * UA + ua) * LK + 4 * ka]) = lo;
        *reinterpret_cast<u32x2 *>(&As[b][((2 * w + 1) * UA + ua) * LK + 4 * ka]) = hi;
      }
    }
    if (hasB) {
      if (masked) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int e = 0; e < 4; ++e) xb[s][e] = hm[s][e] > 0.f ? xb[s][e] : 0.f;
      }
      uint32_t q[4][4];                                // bf16 bits of node s, feature e
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e) q[s][e] = tn_bf16(xb[s][e]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const u32x2 v{q[0][e] | (q[1][e] << 16), q[2][e] | (q[3][e] << 16)};
        *reinterpret_cast<u32x2 *>(&Bs[b][(e * UB + ub) * LK + 4 * kb]) = v;
      }
      if (write_m16) {                                 // the masked operand, node-major, for the feature gradient
        const int gk = kl + 4 * kb;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (gk + s < kend)
            *reinterpret_cast<u32x2 *>(p.M16 + (int64_t)(gk + s) * p.ldm16 + n0 + 4 * ub) =
                u32x2{q[s][0] | (q[s][1] << 16), q[s][2] | (q[s][3] << 16)};
      }
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  const int h = lane >> 5, r = lane & 31;
  if (kbeg < kend) {
    load(kbeg);
    store(0);
    __syncthreads();
    int it = 0;
    for (int kt = kbeg; kt < kend; kt += BK, ++it) {
      const int cur = it & 1;
      load(kt + BK < kend ? kt + BK : kt);
#pragma unroll
      for (int q = 0; q < BK / 16; ++q) {
        bf16x8 a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          a[i] = __builtin_bit_cast(bf16x8,
                                    *reinterpret_cast<const u32x4 *>(&As[cur][(wm0 + i * 32 + r) * LK + 16 * q + 8 * h]));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          b[j] = __builtin_bit_cast(bf16x8,
                                    *reinterpret_cast<const u32x4 *>(&Bs[cur][(wn0 + j * 32 + r) * LK + 16 * q + 8 * h]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      store(cur ^ 1);
      __syncthreads();
    }
  }
  tn_store_partial<TM, TN, UA, 8, UB>(p, acc, split, m0, n0, wm0, wn0, lane);
}

// Fixed-order sum of split partials.  A block owns OUT consecutive outputs
// (64, or 16 for small outputs) and G = 256 V / OUT ranges of the split
// index: thread (g, c) adds the splits of range g in ascending order for
// outputs V c .. V c + V - 1 (16-byte loads when mn % 4 == 0, V = 4), then
// the G range sums of each output are added in order g = 0 .. G - 1.  Many
// short independent sums keep enough loads in flight for partials that
// number in the hundreds per output.
template <int V, int OUT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *ws, int splits, int64_t mn, float *out) {
  constexpr int C = OUT / V, G = 256 / C;
  __shared__ float part[G][OUT];
  const int c = threadIdx.x % C, g = threadIdx.x / C;
  const int64_t i0 = (int64_t)blockIdx.x * OUT + V * c;
  const int per = (splits + G - 1) / G;
  const int z0 = g * per, z1 = min(splits, z0 + per);
  float s[V];
#pragma unroll
  for (int e = 0; e < V; ++e) s[e] = 0.f;
  if (i0 < mn) {                                       // V = 4: mn % 4 == 0, so i0 + 3 < mn
#pragma unroll 4
    for (int z = z0; z < z1; ++z) {
      if constexpr (V == 4) {
        const float4 x = *reinterpret_cast<const float4 *>(ws + (int64_t)z * mn + i0);
        s[0] += x.x;
        s[1] += x.y;
        s[2] += x.z;
        s[3] += x.w;
      } else {
        s[0] += ws[(int64_t)z * mn + i0];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < V; ++e) part[g][V * c + e] = s[e];
  __syncthreads();
  const int o = threadIdx.x;
  const int64_t i = (int64_t)blockIdx.x * OUT + o;
  if (o < OUT && i < mn) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < G; ++k) t += part[k][o];
    out[i] = t;
  }
}

// ---------------------------------------------------------------- launch ---

// Tile height of the fp32 kernels (plain and by parts): 256 (each wave
// 128 x 64: the same staged bytes feed twice the MFMAs, and staging, not the
// matrix cores, bounds the 128-row tile) for 128-wide tiles when f_in >= 384
// and 256-row tiles pad it no further than 128-row tiles would; 128
// otherwise and on bf16 (at f_in = 256 the two tiles leave the grid short of
// one round of resident workgroups: measured slower).  PGCN_TN_BM=128
// (environment) keeps 128.
static int tn_bm(int M, int N, bool bf16) {
  static const bool only128 = [] {
    const char *e = std::getenv("PGCN_TN_BM");
    return e && std::atoi(e) == 128;
  }();
  if (bf16 || N <= 64 || only128 || M < 384) return 128;
  return (M + 255) / 256 * 256 <= (M + 127) / 128 * 128 ? 256 : 128;
}

// fp32 weight gradients by parts (the default) or on the fp32 matrix cores
// (PGCN_GEMM_F32=native, read per call)
static bool tn_f32_by_parts() {
  const char *e = std::getenv("PGCN_GEMM_F32");
  return !(e && std::strcmp(e, "native") == 0);
}

static int tn_tiles(int M, int N, int bm) {
  const int BN = N <= 64 ? 64 : 128;
  return ((M + bm - 1) / bm) * ((N + BN - 1) / BN);
}

// Resident workgroups of a variant on 256 CUs: three per CU, two for the
// 128-wide tiles whose staging holds two slabs (fp32) or fp32 rows (bf16 with
// an fp32 left operand).
static int tn_slots(int N, bool bf16, bool a32) {
  return (N > 64 && (!bf16 || a32)) ? 512 : 768;
}

// Splits over the nodes: tiles x splits about one round of resident
// workgroups, at least 256 nodes per split, and tiles x splits a multiple of 8
// when possible (XCD mapping).
static int splitk_count(int M, int N, int K, int slots, int bm) {
  const int tiles = tn_tiles(M, N, bm);
  int s = slots / tiles;
  const int max_s = (K + 255) / 256;
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  int r = s;
  while (r > 1 && (tiles * r) % 8 != 0) --r;
  if ((tiles * r) % 8 == 0 && 2 * r >= s) s = r;
  return s;
}

size_t gemm_workspace(Gemm kind, int32_t M, int32_t N, int32_t K) {
  if (kind != Gemm::TN_MASK_SPLITK) return 0;
  const int s = std::max({splitk_count(M, N, K, 512, 128), splitk_count(M, N, K, 768, 128),
                           splitk_count(M, N, K, 512, 256)});                     // any variant
  return (size_t)s * (size_t)M * (size_t)N * sizeof(float);
}

template <int BM, int BN>
static void tn_launch(TNParams p, bool bf16, bool a32, bool parts, int splits, hipStream_t s) {
  p.tiles_n = (p.N + BN - 1) / BN;
  p.tiles = ((p.M + BM - 1) / BM) * p.tiles_n;
  const int slab = bf16 ? 32 : 16;
  int kchunk = (p.K + splits - 1) / splits;
  kchunk = (kchunk + slab - 1) / slab * slab;
  if (kchunk == 0) kchunk = slab;
  p.kchunk = kchunk;
  const dim3 grid((unsigned)(p.tiles * splits));
  if (bf16 && a32) hipLaunchKernelGGL((gemm_tn_bf16<BN, true>), grid, dim3(256), 0, s, p);
  else if (bf16) hipLaunchKernelGGL((gemm_tn_bf16<BN, false>), grid, dim3(256), 0, s, p);
  else if (parts && BM == 128) hipLaunchKernelGGL((gemm_tn_f32s<BN>), grid, dim3(256), 0, s, p);
  else if (parts && BN == 128) hipLaunchKernelGGL(gemm_tn_f32s_wide, grid, dim3(256), 0, s, p);
  else hipLaunchKernelGGL((gemm_tn_f32<BM, BN>), grid, dim3(256), 0, s, p);
}

int launch_gemm(Gemm kind, const GemmArgs &g, hipStream_t s) {
  if (kind != Gemm::TN_MASK_SPLITK) return set_error(PGCN_EINVAL, "launch_gemm: only the weight-gradient GEMM");
  if (g.M <= 0 || g.N <= 0) return PGCN_OK;
  const bool bf16 = g.dtype == PGCN_BF16;
  const bool a32 = g.k_split > 0;                      // second left matrix; fp32 left operand on both paths
  const bool parts = !bf16 && tn_f32_by_parts();
  const int bm = tn_bm(g.M, g.N, bf16);
  const int splits = splitk_count(g.M, g.N, g.K, parts ? (bm == 256 ? 512 : 768) : tn_slots(g.N, bf16, a32), bm);
  const size_t need = (size_t)splits * (size_t)g.M * (size_t)g.N * sizeof(float);
  if (!g.workspace || g.workspace_bytes < need)
    return set_error(PGCN_EWORKSPACE, "weight-gradient GEMM: workspace too small");
  TNParams p{};
  p.M = g.M;
  p.N = g.N;
  p.K = g.K;
  p.A = g.A;
  p.A16 = g.A16;
  p.lda = g.lda;
  p.J = g.B;
  p.ldb = g.ldb;
  p.H = g.Hmask;
  p.ldh = g.ldm;
  p.partials = g.workspace;
  p.A_hi = a32 ? g.A_hi : nullptr;
  p.ksplit = a32 ? (int)g.k_split : g.K;
  if (a32 && (!g.A || g.k_split > g.K || (g.lda % 4) != 0))
    return set_error(PGCN_EINVAL, "weight-gradient GEMM: bad split left operand");
  if (g.M16) {
    if (!bf16 || g.ldm16 < g.N || g.ldm16 % 4 != 0 || ((uintptr_t)g.M16 & 7u))
      return set_error(PGCN_EINVAL, "weight-gradient GEMM: bad bf16 operand output");
    p.M16 = g.M16;
    p.ldm16 = g.ldm16;
  }
  {
    TraceScope ts(PGCN_TK_GEMM_WGRAD, s);
    if (g.N <= 64) tn_launch<128, 64>(p, bf16, a32, parts, splits, s);
    else if (bm == 256) tn_launch<256, 128>(p, bf16, a32, parts, splits, s);
    else tn_launch<128, 128>(p, bf16, a32, parts, splits, s);
    PGCN_HIP(hipGetLastError());
  }
  const int64_t mn = (int64_t)g.M * g.N;
  TraceScope ts(PGCN_TK_WGRAD_REDUCE, s);
  // 64 outputs per workgroup, or 16 (64 split ranges each) when that would
  // leave fewer than four workgroups per CU: the sums stay short and many
  const bool narrow = (mn + 63) / 64 < 1024;
  const dim3 rgrid((unsigned)(narrow ? (mn + 15) / 16 : (mn + 63) / 64));
  const float *ws = (const float *)g.workspace;
  if (mn % 4 == 0 && ((uintptr_t)g.workspace & 15u) == 0) {   // every partial [M x N] starts 16-byte aligned
    if (narrow) hipLaunchKernelGGL((splitk_reduce_kernel<4, 16>), rgrid, dim3(256), 0, s, ws, splits, mn, g.C);
    else hipLaunchKernelGGL((splitk_reduce_kernel<4, 64>), rgrid, dim3(256), 0, s, ws, splits, mn, g.C);
  } else {
    if (narrow) hipLaunchKernelGGL((splitk_reduce_kernel<1, 16>), rgrid, dim3(256), 0, s, ws, splits, mn, g.C);
    else hipLaunchKernelGGL((splitk_reduce_kernel<1, 64>), rgrid, dim3(256), 0, s, ws, splits, mn, g.C);
  }
  PGCN_HIP(hipGetLastError());
  return PGCN_OK;
}

}  // namespace pgcn

// Internal declarations shared by the libpgcn translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "pgcn.h"

namespace pgcn {

// Aggregation work item: a contiguous run of one CSR row.  `dst >= 0` is the
// output row (the item covers the whole row); `dst < 0` means partial-sum
// slot (-dst - 1) of a row that was split into fixed segments.
struct WorkItem {
  int64_t begin;
  int32_t len;
  int32_t dst;
};

// A split row: partial slots [first_slot, first_slot + nslots) are summed in
// slot order into output row `row`.
struct SplitRow {
  int32_t row;
  int32_t first_slot;
  int32_t nslots;
  int32_t pad;
};

// Fixed work plan over one CSR matrix (rows of P_i or of P_i^T).  The
// matrix columns are cut into `chunks` equal ranges; chunk c's items are
// items[chunk_items[c] .. chunk_items[c+1]): first the segments of split rows
// (items[.. chunk_whole[c])), then one item per other row's run, longest
// first.  Split rows own `slots` partial slots in total, contiguous per row in
// (chunk, segment) order; `splits` lists them for the fix-up pass.
// Dense block of the matrix taken by the matrix cores instead of the gather:
// the hub rows (most non-zeros) x the hub columns (most referenced), as one
// bit per (row, column).  The block's sum of each hub row is formed first
// (workgroups of kHubRowTile rows, column tiles of kHubColTile staged in LDS,
// the gathered rows split exactly into three bf16 parts, fp32 accumulation;
// several workgroups share a row tile, each over its own range of column
// tiles, and their partial sums are added in range order), and the plan's
// items then add the rest of the row onto it.
constexpr int kHubRowTile = 512;
constexpr int kHubColTile = 32;
struct Hub {
  int32_t rows = 0, rows_real = 0;      // hub rows, padded to kHubRowTile (padding: row id -1)
  int32_t cols = 0, cols_real = 0;      // hub columns, padded to kHubColTile (padding: column id -1)
  int64_t nnz = 0;                      // non-zeros inside the block
  std::vector<int32_t> row_ids, col_ids;
  std::vector<uint32_t> bits;           // [cols / kHubColTile][rows]: bit k = column tile*32 + k
  std::vector<uint32_t> init;           // over all output rows: the row starts from its block sum
  int32_t *d_row_ids = nullptr, *d_col_ids = nullptr;
  uint32_t *d_bits = nullptr, *d_init = nullptr;
};

struct Plan {
  int32_t chunks = 1;
  std::vector<WorkItem> items;
  std::vector<SplitRow> splits;
  std::vector<int64_t> chunk_items, chunk_whole;
  int64_t slots = 0;            // partial slots of all split rows
  WorkItem *d_items = nullptr;
  SplitRow *d_splits = nullptr;
  Hub hub;                      // hub.rows == 0: no dense block
  // with a dense block the items index the matrix without it (col_rest); otherwise the
  // partition's column array
  std::vector<int32_t> col_rest;
  int32_t *d_col_rest = nullptr;
};

}  // namespace pgcn

struct pgcn_partition {
  int32_t nparts = 0, self = 0, host_only = 0, segment = 0, self_loop = 1, symmetric = 0;
  int64_t n_inner = 0, n_bd = 0, nnz = 0, n_send = 0;
  int64_t max_row = 0, max_row_t = 0;
  int device = -1;
  // host copies (canonical numbering)
  std::vector<int64_t> inner_gid, bd_gid, recv_ptr, rowptr, rowptr_t, send_ptr, inv_ptr;
  std::vector<int32_t> col, col_t, send_idx, inv_k;
  std::vector<float> inv_deg;
  std::vector<int64_t> deg;        // whole-graph degree + 1 of the n_inner + n_bd local nodes
  std::vector<float> sym_scale;    // d̃^{-1/2} of the local nodes (symmetric partitions)
  pgcn::Plan plan, plan_t;
  // plans for gathered rows of at most kNarrowRow floats, whose chunks hold
  // more rows for the same bytes; chunks == 0: not built (same as plan, plan_t)
  pgcn::Plan plan_n, plan_tn;
  // device copies
  int32_t *d_col = nullptr, *d_col_t = nullptr, *d_send_idx = nullptr, *d_inv_k = nullptr;
  int64_t *d_inv_ptr = nullptr;
  float *d_inv_deg = nullptr;
  float *d_sym_scale = nullptr;
  // P_i = diag(row_scale) pattern diag(col_scale): the mean (1/d, no column scale) or the
  // symmetric normalisation (d̃^{-1/2} on both sides)
  const float *d_row_scale = nullptr;   // [n_inner]
  const float *d_col_scale = nullptr;   // [n_inner + n_bd] or null
};

namespace pgcn {

// Aggregations of rows of at most this many floats use the narrow plans.
constexpr int64_t kNarrowRow = 64;

// The work plan for an aggregation of P_i (transposed: P_i^T) over rows of f floats.
inline const Plan &agg_plan(const pgcn_partition *p, bool transposed, int64_t f) {
  const Plan &narrow = transposed ? p->plan_tn : p->plan_n;
  if (f <= kNarrowRow && narrow.chunks > 0) return narrow;
  return transposed ? p->plan_t : p->plan;
}

int set_error(int code, const std::string &msg) noexcept;
// The status of an exception caught at an entry point (call from a catch handler): no C++
// exception crosses the C interface; std::bad_alloc is PGCN_ENOMEM, anything else PGCN_EINVAL.
int exception_status(const char *fn) noexcept;

// Workspace bytes one pgcn_layer_fwd call needs (0 for arguments it rejects).
size_t layer_fwd_workspace(const pgcn_partition *p, const pgcn_fwd_args *a);
// Resolves this library's fixed scratch array on device `dev` (which must be
// current) once; pgcn_partition_setup calls it for the device it builds on.
int noalloc_scratch_init(int dev);

// Records a HIP event pair around a kernel launch on stream `s` while tracing
// is enabled (pgcn_trace_enable); does nothing otherwise.  A scope around
// several back-to-back launches says how many with set_launches.
class TraceScope {
 public:
  TraceScope(int32_t kind, hipStream_t s);
  ~TraceScope();
  void set_launches(int32_t n);
  TraceScope(const TraceScope &) = delete;
  TraceScope &operator=(const TraceScope &) = delete;

 private:
  hipStream_t s_;
  int64_t slot_ = -1;
};
int check_hip(hipError_t e, const char *what);

#define PGCN_HIP(call)                                   \
  do {                                                   \
    hipError_t _e = (call);                              \
    if (_e != hipSuccess) return ::pgcn::check_hip(_e, #call); \
  } while (0)

#define PGCN_REQUIRE(cond, msg)                                  \
  do {                                                           \
    if (!(cond)) return ::pgcn::set_error(PGCN_EINVAL, (msg));   \
  } while (0)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---- kernel launchers (defined in the .hip files) -------------------------

// Aggregation over a fixed plan.  Column c < in_split reads in_lo[c], else
// in_hi[c - in_split] (in_hi == nullptr: zero rows).  Output row r < out_split
// goes to out_lo[r], else out_hi[r - out_split].  When `scale` is non-null
// each output row is multiplied by scale[r].  Partial slots go to `partials`.
struct AggArgs {
  const Plan *plan;
  const int32_t *col;
  int64_t in_split;
  const float *in_lo, *in_hi;
  int64_t out_split;
  float *out_lo, *out_hi;
  uint16_t *out_bf16;      // optional bf16 copy of out_lo rows (forward, bf16 GEMM path)
  const float *scale;
  int32_t f;
  int64_t ld_in, ld_out, ld_bf16;
  float *partials;
  int32_t trace_kind;      // PGCN_TK_AGG_FWD or PGCN_TK_AGG_BWD
  int32_t accum_lo;        // 1: rows [0, out_split) add to what out_lo holds (GraphSAGE self term)
  int32_t relu;            // 1: the final rows are max(x, 0) (transform-first forward)
  // optional: the final rows [0, out_split) also go to the send rows that carry them:
  // send[k] for k in send_pos[send_ptr[r] .. send_ptr[r + 1]) (stride ld_out)
  float *send;
  const int64_t *send_ptr;
  const int32_t *send_pos;
};
int launch_aggregate(const AggArgs &a, hipStream_t s);
size_t aggregate_workspace(const Plan &plan, int64_t f);

// NN_*: C (=|+=) A W, with ReLU for *_RELU (ACC: C = act(C + A W));
// MASK_NT_*: C = (J ∘ mask) W^T, row-scaled or plain (fp32 J and mask; rounded to bf16 on the
// bf16 path); NT16_*: the same with the masked operand already bf16 in A16;
// NT_SRC32_ACC_PLAIN: C += A W^T from the fp32 operand on both paths;
// NN_SRC32_PLAIN / _ROWSCALE / _RELU: C = act((diag(rowscale)) A W) from the fp32 operand on both paths
// (rounded to bf16 while staged on the bf16 path); TN_MASK_SPLITK: C = A^T (J ∘ mask)
enum class Gemm {
  NN_RELU, NN_PLAIN, NN_ACC_RELU, NN_ACC_PLAIN, MASK_NT_ROWSCALE, MASK_NT_PLAIN, NT16_ROWSCALE, NT16_PLAIN,
  NN_SRC32_PLAIN, NN_SRC32_ROWSCALE, NN_SRC32_RELU, NT_SRC32_ACC_PLAIN, TN_MASK_SPLITK
};
struct GemmArgs {
  int32_t M, N, K;
  int32_t dtype;            // PGCN_F32 / PGCN_BF16
  const float *A;           // fp32 operand
  const uint16_t *A16;      // bf16 operand (activations)
  int64_t lda;
  const float *B;           // weights or masked operand source
  int64_t ldb;
  const float *Hmask;       // mask source for the masked operand (may be null: no mask)
  int64_t ldm;
  float *C;
  int64_t ldc;
  const float *rowscale;    // per output row scale (MASK_NT_ROWSCALE)
  float *workspace;
  size_t workspace_bytes;
  uint16_t *M16;            // TN_MASK_SPLITK, bf16 path: also write bf16(B ∘ mask) [K, ldm16] (or null)
  int64_t ldm16;
  // TN_MASK_SPLITK with k_split > 0: rows k >= k_split of the left operand come from
  // A_hi[k - k_split] (null: zero rows), and on the bf16 path A (fp32) is rounded
  // while staged instead of reading A16
  const float *A_hi;
  int64_t k_split;
  // NN_* (launch_gemm_nk): the final rows of C also go to the send rows that carry them,
  // send[k] for k in send_pos[send_ptr[r] .. send_ptr[r + 1]) (stride ldc); null: not written
  float *send;
  const int64_t *send_ptr;
  const int32_t *send_pos;
};
int launch_gemm(Gemm kind, const GemmArgs &g, hipStream_t s);
size_t gemm_workspace(Gemm kind, int32_t M, int32_t N, int32_t K);
// forward and feature-gradient GEMMs: weights packed into g.workspace first
int launch_gemm_nk(Gemm kind, const GemmArgs &g, hipStream_t s);
size_t gemm_nk_workspace(int32_t N, int32_t K, int32_t dtype);

// out[r, c] = (H == null || H[r, c] > 0 ? J[r, c] : 0) * scale[r] for c < cols, 0 for c in [cols, ld4(cols))
int launch_mask_scale(const float *J, int64_t ldj, const float *H, int64_t ldh, const float *scale, int64_t rows,
                      int32_t cols, float *out, int64_t ldo, hipStream_t s);
int launch_ema(float *state, const float *in, int64_t rows, int32_t cols, int64_t ld, float gamma,
               hipStream_t s);
int launch_dropout(float *out, const float *in, int64_t rows, int32_t cols, int64_t ld, int64_t row0, uint32_t thr,
                   float scale, uint32_t seed, uint32_t part, uint32_t layer, uint32_t iteration, uint16_t *out16,
                   int64_t ld16, hipStream_t s);
// Adam coefficients, each computed in double on the host and rounded once
struct AdamCoef {
  float lr, eps, b1, b2, omb1, omb2, c1, c2;   // omb = 1 - beta; c = 1 / (1 - beta^t)
};
int launch_adam(float *W, const float *G, const float *Gp, float *m, float *v, int64_t count, const AdamCoef &c,
                hipStream_t s);
// Device-to-device copy of `bytes` (a multiple of 16, both pointers 16-byte aligned) with
// non-temporal loads and stores.
int launch_refill_copy(void *dst, const void *src, size_t bytes, hipStream_t s);
int launch_pack(const int32_t *idx, int64_t count, const float *src, float *dst, int32_t cols,
                int64_t ld, hipStream_t s);
int launch_accum(const int64_t *inv_ptr, const int32_t *inv_k, int64_t rows, const float *src,
                 float *dst, int32_t cols, int64_t ld, hipStream_t s);
int launch_accum_ema(const int64_t *inv_ptr, const int32_t *inv_k, int64_t rows, const float *src, float *state,
                     float gamma, float *dst, int32_t cols, int64_t ld, hipStream_t s);
int launch_loss(int32_t kind, const float *Z, int64_t rows, int32_t classes, int64_t ld,
                const int32_t *labels, const float *targets, int64_t ld_t, float scale, float *J,
                float *loss_out, float *ws, hipStream_t s);
size_t loss_workspace(int64_t rows);
int launch_sgd(float *W, const float *G, const float *G2, int64_t count, float eta, hipStream_t s);

}  // namespace pgcn

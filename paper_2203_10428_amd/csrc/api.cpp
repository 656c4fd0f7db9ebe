// C ABI entry points of libpgcn: argument checking and kernel composition.
#include <cmath>
#include <cstring>

#include "internal.h"

using namespace pgcn;

namespace {

int check_part(const pgcn_partition *p, const char *fn) {
  if (!p) return set_error(PGCN_EINVAL, std::string(fn) + ": null partition");
  if (p->host_only) return set_error(PGCN_EINVAL, std::string(fn) + ": partition was built host-only");
  int dev = -1;
  PGCN_HIP(hipGetDevice(&dev));
  if (dev != p->device) return set_error(PGCN_EINVAL, std::string(fn) + ": current device differs from set-up device");
  return PGCN_OK;
}

bool aligned16(const void *q) { return ((uintptr_t)q & 15u) == 0; }

int64_t ld4(int64_t f) { return (f + 3) / 4 * 4; }
// Row stride of a workspace matrix that an aggregation gathers from: a
// multiple of 8 floats.  A 41-float row then spans 192 bytes, three whole
// 64-byte lines, where a 44-float stride spreads rows over 3.5 lines on
// average (measured: the Reddit-like 41-wide aggregation 7% faster).
int64_t ldw(int64_t f) { return (f + 7) / 8 * 8; }

// forward: split-row partials, plus an fp32 running sum over the column chunks
// when the caller keeps no fp32 A (bf16 path)
size_t fwd_acc_bytes(const pgcn_partition *p, int32_t f_in, int32_t gemm_dtype) {
  const Plan &pl = agg_plan(p, false, f_in);
  if ((pl.chunks <= 1 && pl.hub.rows == 0) || gemm_dtype != PGCN_BF16) return 0;
  return align_up((size_t)p->n_inner * (size_t)ld4(f_in) * sizeof(float), 256);
}
// forward workspace: [aggregation partials | running sum | packed weights]
size_t fwd_agg_bytes(const pgcn_partition *p, int32_t f_in, int32_t gemm_dtype) {
  return align_up(aggregate_workspace(agg_plan(p, false, f_in), f_in), 256) + fwd_acc_bytes(p, f_in, gemm_dtype);
}
// symmetric normalisation, aggregate-first: the gathered rows scaled by d̃_u^{-1/2}
size_t fwd_sym_off(const pgcn_partition *p, int32_t f_in, int32_t f_out, int32_t gemm_dtype) {
  return fwd_agg_bytes(p, f_in, gemm_dtype) + gemm_nk_workspace(f_out, f_in, gemm_dtype);
}
size_t fwd_ws(const pgcn_partition *p, int32_t f_in, int32_t f_out, int32_t gemm_dtype) {
  const size_t sym = p->symmetric ? align_up((size_t)(p->n_inner + p->n_bd) * (size_t)ldw(f_in) * sizeof(float), 256)
                                  : 0;
  return fwd_sym_off(p, f_in, f_out, gemm_dtype) + sym;
}

// Region 0 of the backward workspace first holds the split-K partials of the
// weight gradient, which are consumed before it is reused for D and the
// transposed aggregation's partials.
size_t bwd_region0(const pgcn_partition *p, int32_t f_in, int32_t f_out, bool input_grad) {
  size_t g = gemm_workspace(Gemm::TN_MASK_SPLITK, f_in, f_out, (int32_t)p->n_inner);
  size_t d = 0;
  if (input_grad)
    d = align_up((size_t)p->n_inner * (size_t)ldw(f_in) * sizeof(float), 256) +
        align_up(aggregate_workspace(agg_plan(p, true, f_in), f_in), 256);
  return align_up(g > d ? g : d, 256);
}
// bf16 path with a feature gradient: the masked operand in bf16, written by the
// weight-gradient kernel and read by the feature-gradient GEMM
int64_t ld_m16(int32_t f_out) { return ((int64_t)f_out + 7) / 8 * 8; }
size_t m16_bytes(const pgcn_partition *p, int32_t f_out, bool input_grad, int32_t gemm_dtype) {
  if (!input_grad || gemm_dtype != PGCN_BF16) return 0;
  return align_up((size_t)p->n_inner * (size_t)ld_m16(f_out) * sizeof(uint16_t), 256);
}
// backward workspace: [region 0 | packed weights | bf16 masked operand]
size_t bwd_ws(const pgcn_partition *p, int32_t f_in, int32_t f_out, bool input_grad, int32_t gemm_dtype) {
  return bwd_region0(p, f_in, f_out, input_grad) + (input_grad ? gemm_nk_workspace(f_in, f_out, gemm_dtype) : 0) +
         m16_bytes(p, f_out, input_grad, gemm_dtype);
}
uint16_t *m16_ptr(const pgcn_partition *p, void *ws, int32_t f_in, int32_t f_out, bool input_grad, int32_t dt) {
  if (!m16_bytes(p, f_out, input_grad, dt)) return nullptr;
  return (uint16_t *)((char *)ws + bwd_region0(p, f_in, f_out, input_grad) + gemm_nk_workspace(f_in, f_out, dt));
}

// Transform-first layers.  Forward workspace: [Y (n+b rows, f_out wide) |
// aggregation partials | packed weights].  Backward workspace: [T (n+b rows,
// f_out wide) | region R | packed weights]; region R first holds D = diag(1/d)
// M and the transposed aggregation's partials, then (both consumed) the
// split-K partials of the weight gradient.
int64_t ld_y(int32_t f_out) { return ldw(f_out); }
size_t y_bytes(const pgcn_partition *p, int32_t f_out) {
  return align_up((size_t)(p->n_inner + p->n_bd) * (size_t)ld_y(f_out) * sizeof(float), 256);
}
size_t fwd_tf_agg_off(const pgcn_partition *p, int32_t f_out) { return y_bytes(p, f_out); }
size_t fwd_tf_gemm_off(const pgcn_partition *p, int32_t f_out) {
  return y_bytes(p, f_out) + align_up(aggregate_workspace(agg_plan(p, false, f_out), f_out), 256);
}
size_t fwd_ws_tf(const pgcn_partition *p, int32_t f_in, int32_t f_out, int32_t dt) {
  return fwd_tf_gemm_off(p, f_out) + gemm_nk_workspace(f_out, f_in, dt);
}
size_t bwd_tf_region(const pgcn_partition *p, int32_t f_in, int32_t f_out) {
  const size_t g = gemm_workspace(Gemm::TN_MASK_SPLITK, f_in, f_out, (int32_t)(p->n_inner + p->n_bd));
  const size_t d = align_up((size_t)p->n_inner * (size_t)ld_y(f_out) * sizeof(float), 256) +
                   align_up(aggregate_workspace(agg_plan(p, true, f_out), f_out), 256);
  return align_up(g > d ? g : d, 256);
}
size_t bwd_ws_tf(const pgcn_partition *p, int32_t f_in, int32_t f_out, bool input_grad, int32_t dt) {
  return y_bytes(p, f_out) + bwd_tf_region(p, f_in, f_out) + (input_grad ? gemm_nk_workspace(f_in, f_out, dt) : 0);
}

}  // namespace

// Workspace bytes one pgcn_layer_fwd call needs (0 for arguments it rejects).
size_t pgcn::layer_fwd_workspace(const pgcn_partition *p, const pgcn_fwd_args *a) {
  if (!p || !a || a->f_in < 1 || a->f_out < 1 || a->f_in > PGCN_MAX_WIDTH || a->f_out > PGCN_MAX_WIDTH) return 0;
  if (a->gemm_dtype != PGCN_F32 && a->gemm_dtype != PGCN_BF16) return 0;
  if (a->order == PGCN_ORDER_TRANSFORM) return fwd_ws_tf(p, a->f_in, a->f_out, a->gemm_dtype);
  if (a->order != PGCN_ORDER_AGG) return 0;
  if (a->a_given) return gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
  return fwd_ws(p, a->f_in, a->f_out, a->gemm_dtype);
}

extern "C" size_t pgcn_layer_workspace_size(const pgcn_partition *p, int32_t f_in, int32_t f_out, int32_t gemm_dtype,
                                            int32_t order) try {
  if (order == PGCN_ORDER_AGG) return pgcn_workspace_size(p, f_in, f_out, gemm_dtype);
  if (order != PGCN_ORDER_TRANSFORM || !p || f_in <= 0 || f_out <= 0) return 0;
  const size_t w = fwd_ws_tf(p, f_in, f_out, gemm_dtype);
  const size_t b = bwd_ws_tf(p, f_in, f_out, true, gemm_dtype) + m16_bytes(p, f_out, true, gemm_dtype);
  const size_t l = align_up(loss_workspace(p->n_inner), 256);
  const size_t m = w > b ? w : b;
  return m > l ? m : l;
} catch (...) {
  (void)exception_status("pgcn_layer_workspace_size");
  return 0;
}

extern "C" size_t pgcn_workspace_size(const pgcn_partition *p, int32_t f_in, int32_t f_out, int32_t gemm_dtype) try {
  if (!p || f_in <= 0 || f_out <= 0) return 0;
  size_t w = fwd_ws(p, f_in, f_out, gemm_dtype);
  size_t b = bwd_ws(p, f_in, f_out, true, gemm_dtype);
  size_t l = align_up(loss_workspace(p->n_inner), 256);
  size_t m = w > b ? w : b;
  return m > l ? m : l;
} catch (...) {
  (void)exception_status("pgcn_workspace_size");
  return 0;
}

namespace {

// Y = [H_in ; H_bd] W, then H_out = act(P_i Y): the layer function of
// Appendix A.1 in the association P (H W).
// Rows of the layer output that this partition sends, written by the kernel
// that produces them (send_idx order, via the inverse send map).
template <class Args>
void set_send(Args &x, const pgcn_partition *p, float *send_out) {
  if (!send_out || p->n_send == 0) return;
  x.send = send_out;
  x.send_ptr = p->d_inv_ptr;
  x.send_pos = p->d_inv_k;
}

int layer_fwd_transform(const pgcn_partition *p, const pgcn_fwd_args *a, hipStream_t s) {
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->H_in && a->W && a->H_out, "pgcn_layer_fwd: null H_in, W or H_out");
    PGCN_REQUIRE(aligned16(a->H_in) && aligned16(a->H_bd) && aligned16(a->H_out),
                 "pgcn_layer_fwd: H_in/H_bd/H_out must be 16-byte aligned");
  }
  const size_t need = fwd_ws_tf(p, a->f_in, a->f_out, a->gemm_dtype);
  if (!a->workspace || a->workspace_bytes < need) return set_error(PGCN_EWORKSPACE, "pgcn_layer_fwd: workspace too small");
  if (p->n_inner == 0) return PGCN_OK;
  const int64_t ldy = ld_y(a->f_out);
  float *Y = (float *)a->workspace;
  const bool bd = p->n_bd > 0 && a->H_bd != nullptr;
  GemmArgs m{};
  m.N = a->f_out;
  m.K = a->f_in;
  m.dtype = a->gemm_dtype;
  m.lda = a->ld_in;
  m.B = a->W;
  m.ldb = a->f_out;
  m.ldc = ldy;
  m.workspace = (float *)((char *)a->workspace + fwd_tf_gemm_off(p, a->f_out));
  m.workspace_bytes = gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
  for (int part = 0; part < (bd ? 2 : 1); ++part) {    // symmetric: rows of Y scaled by d̃_u^{-1/2}
    m.M = (int32_t)(part ? p->n_bd : p->n_inner);
    m.A = part ? a->H_bd : a->H_in;
    m.C = part ? Y + p->n_inner * ldy : Y;
    m.rowscale = p->d_col_scale ? p->d_col_scale + (part ? p->n_inner : 0) : nullptr;
    int rc = launch_gemm_nk(p->d_col_scale ? Gemm::NN_SRC32_ROWSCALE : Gemm::NN_SRC32_PLAIN, m, s);
    if (rc) return rc;
  }
  AggArgs g{};
  g.plan = &agg_plan(p, false, a->f_out);
  g.col = p->d_col;
  g.in_split = p->n_inner;
  g.in_lo = Y;
  g.in_hi = bd ? Y + p->n_inner * ldy : nullptr;
  g.out_split = p->n_inner;
  g.out_lo = a->H_out;
  g.scale = p->d_row_scale;
  g.f = a->f_out;
  g.ld_in = ldy;
  g.ld_out = a->ld_out;
  g.partials = (float *)((char *)a->workspace + fwd_tf_agg_off(p, a->f_out));
  g.relu = a->relu ? 1 : 0;
  g.trace_kind = PGCN_TK_AGG_FWD;
  set_send(g, p, a->send_out);
  return launch_aggregate(g, s);
}

// T = P_i^T M, dW = [H_in ; H_bd]^T T, J_full = T W^T.
int layer_bwd_transform(const pgcn_partition *p, const pgcn_bwd_args *a, hipStream_t s) {
  const bool input_grad = a->J_in != nullptr || a->J_bd_out != nullptr;
  PGCN_REQUIRE(a->dW, "pgcn_layer_bwd: null dW");
  if (input_grad) {
    PGCN_REQUIRE(a->J_in && (a->J_bd_out || p->n_bd == 0),
                 "pgcn_layer_bwd: J_in and J_bd_out must both be given (or both NULL)");
    PGCN_REQUIRE(aligned16(a->J_in) && aligned16(a->J_bd_out), "pgcn_layer_bwd: J_in/J_bd_out must be 16-byte aligned");
  }
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->J_out && a->W && a->H_in, "pgcn_layer_bwd: null J_out, W or H_in");
    PGCN_REQUIRE(!a->relu || a->H_out, "pgcn_layer_bwd: relu needs H_out as mask source");
    PGCN_REQUIRE(aligned16(a->J_out) && aligned16(a->H_out) && aligned16(a->H_in) && aligned16(a->H_bd),
                 "pgcn_layer_bwd: J_out/H_out/H_in/H_bd must be 16-byte aligned");
  }
  const size_t need = bwd_ws_tf(p, a->f_in, a->f_out, input_grad, a->gemm_dtype);
  if (!a->workspace || a->workspace_bytes < need) return set_error(PGCN_EWORKSPACE, "pgcn_layer_bwd: workspace too small");
  if (p->n_inner == 0) {             // no rows (so no boundary rows): dW = 0, a split-K GEMM over no nodes
    GemmArgs z{};
    z.M = a->f_in;
    z.N = a->f_out;
    z.dtype = a->gemm_dtype;
    z.C = a->dW;
    z.workspace = (float *)a->workspace;
    z.workspace_bytes = a->workspace_bytes;
    return launch_gemm(Gemm::TN_MASK_SPLITK, z, s);
  }
  const int64_t ldt = ld_y(a->f_out);
  float *T = (float *)a->workspace;
  char *R = (char *)a->workspace + y_bytes(p, a->f_out);
  float *D = (float *)R;
  float *partials = (float *)(R + align_up((size_t)p->n_inner * ldt * sizeof(float), 256));
  int rc = launch_mask_scale(a->J_out, a->ld_out, a->relu ? a->H_out : nullptr, a->ld_out, p->d_row_scale, p->n_inner,
                             a->f_out, D, ldt, s);
  if (rc) return rc;
  AggArgs t{};
  t.plan = &agg_plan(p, true, a->f_out);
  t.col = p->d_col_t;
  t.in_split = p->n_inner;
  t.in_lo = D;
  t.out_split = p->n_inner;
  t.out_lo = T;
  t.out_hi = T + p->n_inner * ldt;
  t.scale = p->d_col_scale;
  t.f = a->f_out;
  t.ld_in = ldt;
  t.ld_out = ldt;
  t.partials = partials;
  t.trace_kind = PGCN_TK_AGG_BWD;
  rc = launch_aggregate(t, s);
  if (rc) return rc;

  GemmArgs g{};
  g.M = a->f_in;
  g.N = a->f_out;
  g.K = (int32_t)(p->n_inner + p->n_bd);
  g.dtype = a->gemm_dtype;
  g.A = a->H_in;
  g.A_hi = p->n_bd > 0 ? a->H_bd : nullptr;
  g.k_split = p->n_inner;
  g.lda = a->ld_in;
  g.B = T;
  g.ldb = ldt;
  g.C = a->dW;
  g.ldc = a->f_out;
  g.workspace = (float *)R;
  g.workspace_bytes = bwd_tf_region(p, a->f_in, a->f_out);
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, g, s);
  if (rc || !input_grad) return rc;

  GemmArgs d{};
  d.N = a->f_in;
  d.K = a->f_out;
  d.dtype = a->gemm_dtype;
  d.lda = ldt;
  d.B = a->W;
  d.ldb = a->f_out;
  d.ldc = a->ld_in;
  d.workspace = (float *)(R + bwd_tf_region(p, a->f_in, a->f_out));
  d.workspace_bytes = gemm_nk_workspace(a->f_in, a->f_out, a->gemm_dtype);
  for (int part = 0; part < (p->n_bd > 0 ? 2 : 1); ++part) {
    d.M = (int32_t)(part ? p->n_bd : p->n_inner);
    d.A = part ? T + p->n_inner * ldt : T;
    d.C = part ? a->J_bd_out : a->J_in;
    rc = launch_gemm_nk(Gemm::MASK_NT_PLAIN, d, s);
    if (rc) return rc;
  }
  return PGCN_OK;
}

}  // namespace

extern "C" int pgcn_layer_fwd(const pgcn_partition *p, const pgcn_fwd_args *a, hipStream_t s) try {
  int rc = check_part(p, "pgcn_layer_fwd");
  if (rc) return rc;
  PGCN_REQUIRE(p->self_loop, "pgcn_layer_fwd: the GCN layer needs a partition built with self loops");
  PGCN_REQUIRE(a, "pgcn_layer_fwd: null args");
  PGCN_REQUIRE(a->f_in >= 1 && a->f_out >= 1, "pgcn_layer_fwd: widths must be >= 1");
  PGCN_REQUIRE(a->f_in <= PGCN_MAX_WIDTH && a->f_out <= PGCN_MAX_WIDTH, "pgcn_layer_fwd: widths above PGCN_MAX_WIDTH");
  PGCN_REQUIRE(aligned16(a->send_out), "pgcn_layer_fwd: send_out must be 16-byte aligned");
  PGCN_REQUIRE(a->gemm_dtype == PGCN_F32 || a->gemm_dtype == PGCN_BF16, "pgcn_layer_fwd: bad gemm_dtype");
  PGCN_REQUIRE(a->ld_in >= a->f_in && a->ld_in % 4 == 0, "pgcn_layer_fwd: ld_in must be >= f_in and a multiple of 4");
  PGCN_REQUIRE(a->ld_out >= a->f_out && a->ld_out % 4 == 0, "pgcn_layer_fwd: ld_out must be >= f_out and a multiple of 4");
  PGCN_REQUIRE(a->order == PGCN_ORDER_AGG || a->order == PGCN_ORDER_TRANSFORM, "pgcn_layer_fwd: bad order");
  PGCN_REQUIRE(a->a_given == 0 || a->a_given == 1, "pgcn_layer_fwd: a_given must be 0 or 1");
  PGCN_REQUIRE(!(a->a_given && a->order == PGCN_ORDER_TRANSFORM),
               "pgcn_layer_fwd: a given aggregate needs the aggregate-first order");
  if (a->order == PGCN_ORDER_TRANSFORM) return layer_fwd_transform(p, a, s);
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  if (a->a_given) {                  // only the update: Z = A W from the given fp32 aggregate
    if (p->n_inner > 0) {
      PGCN_REQUIRE(a->A && a->W && a->H_out, "pgcn_layer_fwd: a_given needs A, W and H_out");
      PGCN_REQUIRE(aligned16(a->A), "pgcn_layer_fwd: A must be 16-byte aligned");
    }
    const size_t gneed = gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
    if (!a->workspace || a->workspace_bytes < gneed) return set_error(PGCN_EWORKSPACE, "pgcn_layer_fwd: workspace too small");
    if (p->n_inner == 0) return PGCN_OK;
    GemmArgs m{};
    m.M = (int32_t)p->n_inner;
    m.N = a->f_out;
    m.K = a->f_in;
    m.dtype = a->gemm_dtype;
    m.A = a->A;
    m.lda = a->ld_in;
    m.B = a->W;
    m.ldb = a->f_out;
    m.C = a->H_out;
    m.ldc = a->ld_out;
    m.workspace = (float *)a->workspace;
    m.workspace_bytes = gneed;
    set_send(m, p, a->send_out);
    return launch_gemm_nk(a->relu ? Gemm::NN_SRC32_RELU : Gemm::NN_SRC32_PLAIN, m, s);
  }
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->H_in && a->W && a->H_out, "pgcn_layer_fwd: null H_in, W or H_out");
    PGCN_REQUIRE(aligned16(a->H_in) && aligned16(a->H_bd), "pgcn_layer_fwd: H_in/H_bd must be 16-byte aligned");
    if (bf16 && !a->A) {
      PGCN_REQUIRE(a->A_bf16 && aligned16(a->A_bf16) && a->ld_in % 8 == 0,
                   "pgcn_layer_fwd: bf16 path needs A_bf16 (16-byte aligned, ld_in % 8 == 0) or A");
    } else {
      PGCN_REQUIRE(a->A, "pgcn_layer_fwd: fp32 path needs A");
    }
    PGCN_REQUIRE(!a->A || aligned16(a->A), "pgcn_layer_fwd: A must be 16-byte aligned");
    PGCN_REQUIRE(!a->A_bf16 || (aligned16(a->A_bf16) && a->ld_in % 8 == 0),
                 "pgcn_layer_fwd: A_bf16 must be 16-byte aligned with ld_in % 8 == 0");
  }
  const size_t need = fwd_ws(p, a->f_in, a->f_out, a->gemm_dtype);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need))
    return set_error(PGCN_EWORKSPACE, "pgcn_layer_fwd: workspace too small");
  if (p->n_inner == 0) return PGCN_OK;

  const float *in_lo = a->H_in, *in_hi = p->n_bd > 0 ? a->H_bd : nullptr;
  int64_t ld_agg = a->ld_in;
  if (p->d_col_scale) {              // symmetric: the gathered rows scaled by d̃_u^{-1/2} first
    const int64_t lds = ldw(a->f_in);
    float *Hs = (float *)((char *)a->workspace + fwd_sym_off(p, a->f_in, a->f_out, a->gemm_dtype));
    rc = launch_mask_scale(a->H_in, a->ld_in, nullptr, 0, p->d_col_scale, p->n_inner, a->f_in, Hs, lds, s);
    if (!rc && in_hi)
      rc = launch_mask_scale(in_hi, a->ld_in, nullptr, 0, p->d_col_scale + p->n_inner, p->n_bd, a->f_in,
                             Hs + p->n_inner * lds, lds, s);
    if (rc) return rc;
    in_lo = Hs;
    in_hi = in_hi ? Hs + p->n_inner * lds : nullptr;
    ld_agg = lds;
  }
  AggArgs g{};
  g.plan = &agg_plan(p, false, a->f_in);
  g.col = p->d_col;
  g.in_split = p->n_inner;
  g.in_lo = in_lo;
  g.in_hi = in_hi;
  g.out_split = p->n_inner;
  g.out_lo = a->A;
  g.out_hi = nullptr;
  g.out_bf16 = bf16 ? a->A_bf16 : nullptr;
  g.scale = p->d_row_scale;
  g.f = a->f_in;
  g.ld_in = ld_agg;
  g.ld_out = a->ld_in;
  g.ld_bf16 = a->ld_in;
  g.partials = (float *)a->workspace;
  if (!a->A && (g.plan->chunks > 1 || g.plan->hub.rows > 0)) {   // running sum over chunks (and the block sum)
    g.out_lo = (float *)((char *)a->workspace + align_up(aggregate_workspace(*g.plan, a->f_in), 256));
    g.ld_out = ld4(a->f_in);
  }
  g.trace_kind = PGCN_TK_AGG_FWD;
  rc = launch_aggregate(g, s);
  if (rc) return rc;

  GemmArgs m{};
  m.M = (int32_t)p->n_inner;
  m.N = a->f_out;
  m.K = a->f_in;
  m.dtype = a->gemm_dtype;
  m.A = a->A;
  m.A16 = a->A_bf16;
  m.lda = a->ld_in;
  m.B = a->W;
  m.ldb = a->f_out;
  m.C = a->H_out;
  m.ldc = a->ld_out;
  m.workspace = (float *)((char *)a->workspace + fwd_agg_bytes(p, a->f_in, a->gemm_dtype));
  m.workspace_bytes = gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
  set_send(m, p, a->send_out);
  if (bf16 && !a->A_bf16)           // bf16 path without the bf16 copy: A rounded while staged (same values)
    return launch_gemm_nk(a->relu ? Gemm::NN_SRC32_RELU : Gemm::NN_SRC32_PLAIN, m, s);
  return launch_gemm_nk(a->relu ? Gemm::NN_RELU : Gemm::NN_PLAIN, m, s);
} catch (...) {
  return exception_status("pgcn_layer_fwd");
}

extern "C" int pgcn_layer_bwd(const pgcn_partition *p, const pgcn_bwd_args *a, hipStream_t s) try {
  int rc = check_part(p, "pgcn_layer_bwd");
  if (rc) return rc;
  PGCN_REQUIRE(p->self_loop, "pgcn_layer_bwd: the GCN layer needs a partition built with self loops");
  PGCN_REQUIRE(a, "pgcn_layer_bwd: null args");
  PGCN_REQUIRE(a->f_in >= 1 && a->f_out >= 1, "pgcn_layer_bwd: widths must be >= 1");
  PGCN_REQUIRE(a->f_in <= PGCN_MAX_WIDTH && a->f_out <= PGCN_MAX_WIDTH, "pgcn_layer_bwd: widths above PGCN_MAX_WIDTH");
  PGCN_REQUIRE(a->gemm_dtype == PGCN_F32 || a->gemm_dtype == PGCN_BF16, "pgcn_layer_bwd: bad gemm_dtype");
  PGCN_REQUIRE(a->ld_in >= a->f_in && a->ld_in % 4 == 0, "pgcn_layer_bwd: ld_in must be >= f_in and a multiple of 4");
  PGCN_REQUIRE(a->ld_out >= a->f_out && a->ld_out % 4 == 0, "pgcn_layer_bwd: ld_out must be >= f_out and a multiple of 4");
  PGCN_REQUIRE(a->order == PGCN_ORDER_AGG || a->order == PGCN_ORDER_TRANSFORM, "pgcn_layer_bwd: bad order");
  if (a->order == PGCN_ORDER_TRANSFORM) return layer_bwd_transform(p, a, s);
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  const bool input_grad = a->J_in != nullptr || a->J_bd_out != nullptr;
  PGCN_REQUIRE(a->dW, "pgcn_layer_bwd: null dW");
  if (input_grad) {
    PGCN_REQUIRE(a->J_in && (a->J_bd_out || p->n_bd == 0),
                 "pgcn_layer_bwd: J_in and J_bd_out must both be given (or both NULL)");
    PGCN_REQUIRE(aligned16(a->J_in) && aligned16(a->J_bd_out), "pgcn_layer_bwd: J_in/J_bd_out must be 16-byte aligned");
  }
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->J_out && a->W, "pgcn_layer_bwd: null J_out or W");
    PGCN_REQUIRE(!a->relu || a->H_out, "pgcn_layer_bwd: relu needs H_out as mask source");
    PGCN_REQUIRE(aligned16(a->J_out) && aligned16(a->H_out), "pgcn_layer_bwd: J_out/H_out must be 16-byte aligned");
    if (bf16 && !a->A)
      PGCN_REQUIRE(a->A_bf16 && aligned16(a->A_bf16) && a->ld_in % 8 == 0,
                   "pgcn_layer_bwd: bf16 path needs A_bf16 (16-byte aligned, ld_in % 8 == 0) or A");
    else
      PGCN_REQUIRE(a->A && aligned16(a->A), "pgcn_layer_bwd: fp32 path needs A (16-byte aligned)");
  }
  const size_t need = bwd_ws(p, a->f_in, a->f_out, input_grad, a->gemm_dtype);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need))
    return set_error(PGCN_EWORKSPACE, "pgcn_layer_bwd: workspace too small");

  // dW = A^T (J ∘ 1[H > 0]); with no inner rows it is zero
  GemmArgs g{};
  g.M = a->f_in;
  g.N = a->f_out;
  g.K = (int32_t)p->n_inner;
  g.dtype = a->gemm_dtype;
  g.A = a->A;
  g.A16 = a->A_bf16;
  g.lda = a->ld_in;
  g.B = a->J_out;
  g.ldb = a->ld_out;
  g.Hmask = a->relu ? a->H_out : nullptr;
  g.ldm = a->ld_out;
  g.C = a->dW;
  g.ldc = a->f_out;
  g.workspace = (float *)a->workspace;
  g.workspace_bytes = a->workspace_bytes;
  uint16_t *M16 = p->n_inner > 0 ? m16_ptr(p, a->workspace, a->f_in, a->f_out, input_grad, a->gemm_dtype) : nullptr;
  g.M16 = M16;
  g.ldm16 = ld_m16(a->f_out);
  if (bf16 && !a->A_bf16) g.k_split = p->n_inner;    // fp32 A rounded while staged (every row from A)
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, g, s);
  if (rc) return rc;
  if (!input_grad || p->n_inner == 0) return PGCN_OK;

  // D = diag(1/d) ((J ∘ 1[H > 0]) W^T), then J_full = (P_i^T without the scale) D
  const int64_t ld_d = ldw(a->f_in);
  float *D = (float *)a->workspace;
  float *partials = (float *)((char *)a->workspace + align_up((size_t)p->n_inner * ld_d * sizeof(float), 256));
  GemmArgs d{};
  d.M = (int32_t)p->n_inner;
  d.N = a->f_in;
  d.K = a->f_out;
  d.dtype = a->gemm_dtype;
  d.A = a->J_out;
  d.lda = a->ld_out;
  d.Hmask = a->relu ? a->H_out : nullptr;
  d.ldm = a->ld_out;
  d.B = a->W;
  d.ldb = a->f_out;
  d.C = D;
  d.ldc = ld_d;
  d.rowscale = p->d_row_scale;
  d.workspace = (float *)((char *)a->workspace + bwd_region0(p, a->f_in, a->f_out, input_grad));
  d.workspace_bytes = gemm_nk_workspace(a->f_in, a->f_out, a->gemm_dtype);
  if (M16) {                       // bf16 path: the masked operand as the weight-gradient kernel rounded it
    d.A = nullptr;
    d.A16 = M16;
    d.lda = ld_m16(a->f_out);
    d.Hmask = nullptr;
  }
  rc = launch_gemm_nk(M16 ? Gemm::NT16_ROWSCALE : Gemm::MASK_NT_ROWSCALE, d, s);
  if (rc) return rc;

  AggArgs t{};
  t.plan = &agg_plan(p, true, a->f_in);
  t.col = p->d_col_t;
  t.in_split = p->n_inner;
  t.in_lo = D;
  t.in_hi = nullptr;
  t.out_split = p->n_inner;
  t.out_lo = a->J_in;
  t.out_hi = a->J_bd_out;
  t.out_bf16 = nullptr;
  t.scale = p->d_col_scale;           // symmetric: d̃_u^{-1/2} of the gradient's rows
  t.f = a->f_in;
  t.ld_in = ld_d;
  t.ld_out = a->ld_in;
  t.ld_bf16 = 0;
  t.partials = partials;
  t.trace_kind = PGCN_TK_AGG_BWD;
  return launch_aggregate(t, s);
} catch (...) {
  return exception_status("pgcn_layer_bwd");
}

// ---------------------------------------------------------------- GraphSAGE ---

namespace {

// GraphSAGE forward with z W_top evaluated as P_i (X W_top): Y = [X_in ; X_bd]
// W_top, H_out = P_i Y, then H_out = act(H_out + X_in W_bot).
int sage_fwd_transform(const pgcn_partition *p, const pgcn_sage_fwd_args *a, hipStream_t s) {
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->X_in && a->W && a->H_out, "pgcn_sage_layer_fwd: null X_in, W or H_out");
    PGCN_REQUIRE(aligned16(a->X_in) && aligned16(a->X_bd) && aligned16(a->H_out),
                 "pgcn_sage_layer_fwd: X_in/X_bd/H_out must be 16-byte aligned");
    if (bf16)
      PGCN_REQUIRE(a->X_in_bf16 && aligned16(a->X_in_bf16) && a->ld_in % 8 == 0,
                   "pgcn_sage_layer_fwd: bf16 path needs X_in_bf16 (16-byte aligned) and ld_in % 8 == 0");
  }
  const size_t need = fwd_ws_tf(p, a->f_in, a->f_out, a->gemm_dtype);
  if (!a->workspace || a->workspace_bytes < need)
    return set_error(PGCN_EWORKSPACE, "pgcn_sage_layer_fwd: workspace too small");
  if (p->n_inner == 0) return PGCN_OK;
  const int64_t ldy = ld_y(a->f_out);
  float *Y = (float *)a->workspace;
  const bool bd = p->n_bd > 0 && a->X_bd != nullptr;
  GemmArgs m{};
  m.N = a->f_out;
  m.K = a->f_in;
  m.dtype = a->gemm_dtype;
  m.lda = a->ld_in;
  m.B = a->W;
  m.ldb = a->f_out;
  m.ldc = ldy;
  m.workspace = (float *)((char *)a->workspace + fwd_tf_gemm_off(p, a->f_out));
  m.workspace_bytes = gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
  for (int part = 0; part < (bd ? 2 : 1); ++part) {
    m.M = (int32_t)(part ? p->n_bd : p->n_inner);
    m.A = part ? a->X_bd : a->X_in;
    m.C = part ? Y + p->n_inner * ldy : Y;
    int rc = launch_gemm_nk(Gemm::NN_SRC32_PLAIN, m, s);
    if (rc) return rc;
  }
  AggArgs g{};
  g.plan = &agg_plan(p, false, a->f_out);
  g.col = p->d_col;
  g.in_split = p->n_inner;
  g.in_lo = Y;
  g.in_hi = bd ? Y + p->n_inner * ldy : nullptr;
  g.out_split = p->n_inner;
  g.out_lo = a->H_out;
  g.scale = p->d_inv_deg;
  g.f = a->f_out;
  g.ld_in = ldy;
  g.ld_out = a->ld_out;
  g.partials = (float *)((char *)a->workspace + fwd_tf_agg_off(p, a->f_out));
  g.trace_kind = PGCN_TK_AGG_FWD;
  int rc = launch_aggregate(g, s);
  if (rc) return rc;
  GemmArgs b{};                      // the self term, accumulated onto P_i Y, then the activation
  b.M = (int32_t)p->n_inner;
  b.N = a->f_out;
  b.K = a->f_in;
  b.dtype = a->gemm_dtype;
  b.A = a->X_in;
  b.A16 = a->X_in_bf16;
  b.lda = a->ld_in;
  b.B = a->W + (size_t)a->f_in * a->f_out;
  b.ldb = a->f_out;
  b.C = a->H_out;
  b.ldc = a->ld_out;
  b.workspace = m.workspace;
  b.workspace_bytes = m.workspace_bytes;
  set_send(b, p, a->send_out);
  return launch_gemm_nk(a->relu ? Gemm::NN_ACC_RELU : Gemm::NN_ACC_PLAIN, b, s);
}

// T = P_i^T M; dW = [[X_in ; X_bd]^T T ; X_in^T M]; J_full = T W_top^T (+ M W_bot^T on inner rows).
int sage_bwd_transform(const pgcn_partition *p, const pgcn_sage_bwd_args *a, hipStream_t s) {
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  const bool input_grad = a->J_in != nullptr || a->J_bd_out != nullptr;
  PGCN_REQUIRE(a->dW, "pgcn_sage_layer_bwd: null dW");
  if (input_grad) {
    PGCN_REQUIRE(a->J_in && (a->J_bd_out || p->n_bd == 0),
                 "pgcn_sage_layer_bwd: J_in and J_bd_out must both be given (or both NULL)");
    PGCN_REQUIRE(aligned16(a->J_in) && aligned16(a->J_bd_out),
                 "pgcn_sage_layer_bwd: J_in/J_bd_out must be 16-byte aligned");
  }
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->J_out && a->W && a->X_in, "pgcn_sage_layer_bwd: null J_out, W or X_in");
    PGCN_REQUIRE(!a->relu || a->H_out, "pgcn_sage_layer_bwd: relu needs H_out as mask source");
    PGCN_REQUIRE(aligned16(a->J_out) && aligned16(a->H_out) && aligned16(a->X_in) && aligned16(a->X_bd),
                 "pgcn_sage_layer_bwd: J_out/H_out/X_in/X_bd must be 16-byte aligned");
    if (bf16)
      PGCN_REQUIRE(a->X_in_bf16 && aligned16(a->X_in_bf16) && a->ld_in % 8 == 0,
                   "pgcn_sage_layer_bwd: bf16 path needs X_in_bf16 (16-byte aligned) and ld_in % 8 == 0");
  }
  const size_t need = bwd_ws_tf(p, a->f_in, a->f_out, input_grad, a->gemm_dtype) +
                      m16_bytes(p, a->f_out, input_grad, a->gemm_dtype);
  if (!a->workspace || a->workspace_bytes < need)
    return set_error(PGCN_EWORKSPACE, "pgcn_sage_layer_bwd: workspace too small");
  const size_t half = (size_t)a->f_in * a->f_out;
  if (p->n_inner == 0) {             // no rows (so no boundary rows): both halves of dW are zero
    GemmArgs z{};
    z.M = a->f_in;
    z.N = a->f_out;
    z.dtype = a->gemm_dtype;
    z.workspace = (float *)a->workspace;
    z.workspace_bytes = a->workspace_bytes;
    for (int hlf = 0; hlf < 2; ++hlf) {
      z.C = a->dW + hlf * half;
      int rc = launch_gemm(Gemm::TN_MASK_SPLITK, z, s);
      if (rc) return rc;
    }
    return PGCN_OK;
  }
  const int64_t ldt = ld_y(a->f_out);
  float *T = (float *)a->workspace;
  char *R = (char *)a->workspace + y_bytes(p, a->f_out);
  const size_t region = bwd_tf_region(p, a->f_in, a->f_out);
  float *D = (float *)R;
  float *partials = (float *)(R + align_up((size_t)p->n_inner * ldt * sizeof(float), 256));
  int rc = launch_mask_scale(a->J_out, a->ld_out, a->relu ? a->H_out : nullptr, a->ld_out, p->d_inv_deg, p->n_inner,
                             a->f_out, D, ldt, s);
  if (rc) return rc;
  AggArgs t{};
  t.plan = &agg_plan(p, true, a->f_out);
  t.col = p->d_col_t;
  t.in_split = p->n_inner;
  t.in_lo = D;
  t.out_split = p->n_inner;
  t.out_lo = T;
  t.out_hi = T + p->n_inner * ldt;
  t.f = a->f_out;
  t.ld_in = ldt;
  t.ld_out = ldt;
  t.partials = partials;
  t.trace_kind = PGCN_TK_AGG_BWD;
  rc = launch_aggregate(t, s);
  if (rc) return rc;

  GemmArgs g{};                      // top half: [X_in ; X_bd]^T T over n + b nodes
  g.M = a->f_in;
  g.N = a->f_out;
  g.K = (int32_t)(p->n_inner + p->n_bd);
  g.dtype = a->gemm_dtype;
  g.A = a->X_in;
  g.A_hi = p->n_bd > 0 ? a->X_bd : nullptr;
  g.k_split = p->n_inner;
  g.lda = a->ld_in;
  g.B = T;
  g.ldb = ldt;
  g.C = a->dW;
  g.ldc = a->f_out;
  g.workspace = (float *)R;
  g.workspace_bytes = region;
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, g, s);
  if (rc) return rc;
  uint16_t *M16 = (bf16 && input_grad)
                      ? (uint16_t *)(R + region + gemm_nk_workspace(a->f_in, a->f_out, a->gemm_dtype)) : nullptr;
  GemmArgs h{};                      // bottom half: X_in^T (J ∘ 1[H > 0]); bf16: also writes the rounded M
  h.M = a->f_in;
  h.N = a->f_out;
  h.K = (int32_t)p->n_inner;
  h.dtype = a->gemm_dtype;
  h.A = a->X_in;
  h.A16 = a->X_in_bf16;
  h.lda = a->ld_in;
  h.B = a->J_out;
  h.ldb = a->ld_out;
  h.Hmask = a->relu ? a->H_out : nullptr;
  h.ldm = a->ld_out;
  h.C = a->dW + half;
  h.ldc = a->f_out;
  h.workspace = (float *)R;
  h.workspace_bytes = region;
  h.M16 = M16;
  h.ldm16 = ld_m16(a->f_out);
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, h, s);
  if (rc || !input_grad) return rc;

  GemmArgs d{};                      // J_in = M W_bot^T, then J_in += T_in W_top^T; J_bd_out = T_bd W_top^T
  d.M = (int32_t)p->n_inner;
  d.N = a->f_in;
  d.K = a->f_out;
  d.dtype = a->gemm_dtype;
  d.A = a->J_out;
  d.lda = a->ld_out;
  d.Hmask = a->relu ? a->H_out : nullptr;
  d.ldm = a->ld_out;
  d.B = a->W + half;
  d.ldb = a->f_out;
  d.C = a->J_in;
  d.ldc = a->ld_in;
  d.workspace = (float *)(R + region);
  d.workspace_bytes = gemm_nk_workspace(a->f_in, a->f_out, a->gemm_dtype);
  if (M16) {
    d.A = nullptr;
    d.A16 = M16;
    d.lda = ld_m16(a->f_out);
    d.Hmask = nullptr;
  }
  rc = launch_gemm_nk(M16 ? Gemm::NT16_PLAIN : Gemm::MASK_NT_PLAIN, d, s);
  if (rc) return rc;
  GemmArgs e{};
  e.N = a->f_in;
  e.K = a->f_out;
  e.dtype = a->gemm_dtype;
  e.lda = ldt;
  e.B = a->W;
  e.ldb = a->f_out;
  e.ldc = a->ld_in;
  e.workspace = d.workspace;
  e.workspace_bytes = d.workspace_bytes;
  e.M = (int32_t)p->n_inner;
  e.A = T;
  e.C = a->J_in;
  rc = launch_gemm_nk(Gemm::NT_SRC32_ACC_PLAIN, e, s);
  if (rc || p->n_bd == 0) return rc;
  e.M = (int32_t)p->n_bd;
  e.A = T + p->n_inner * ldt;
  e.C = a->J_bd_out;
  return launch_gemm_nk(Gemm::MASK_NT_PLAIN, e, s);
}

}  // namespace

extern "C" int pgcn_sage_layer_fwd(const pgcn_partition *p, const pgcn_sage_fwd_args *a, hipStream_t s) try {
  int rc = check_part(p, "pgcn_sage_layer_fwd");
  if (rc) return rc;
  PGCN_REQUIRE(!p->self_loop, "pgcn_sage_layer_fwd: the partition must be built with PGCN_SETUP_NO_SELF_LOOP");
  PGCN_REQUIRE(a, "pgcn_sage_layer_fwd: null args");
  PGCN_REQUIRE(a->f_in >= 1 && a->f_out >= 1, "pgcn_sage_layer_fwd: widths must be >= 1");
  PGCN_REQUIRE(a->f_in <= PGCN_MAX_WIDTH && a->f_out <= PGCN_MAX_WIDTH, "pgcn_sage_layer_fwd: widths above PGCN_MAX_WIDTH");
  PGCN_REQUIRE(aligned16(a->send_out), "pgcn_sage_layer_fwd: send_out must be 16-byte aligned");
  PGCN_REQUIRE(a->gemm_dtype == PGCN_F32 || a->gemm_dtype == PGCN_BF16, "pgcn_sage_layer_fwd: bad gemm_dtype");
  PGCN_REQUIRE(a->ld_in >= a->f_in && a->ld_in % 4 == 0, "pgcn_sage_layer_fwd: ld_in must be >= f_in and a multiple of 4");
  PGCN_REQUIRE(a->ld_out >= a->f_out && a->ld_out % 4 == 0,
               "pgcn_sage_layer_fwd: ld_out must be >= f_out and a multiple of 4");
  PGCN_REQUIRE(a->order == PGCN_ORDER_AGG || a->order == PGCN_ORDER_TRANSFORM, "pgcn_sage_layer_fwd: bad order");
  if (a->order == PGCN_ORDER_TRANSFORM) return sage_fwd_transform(p, a, s);
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->X_in && a->W && a->H_out, "pgcn_sage_layer_fwd: null X_in, W or H_out");
    PGCN_REQUIRE(aligned16(a->X_in) && aligned16(a->X_bd), "pgcn_sage_layer_fwd: X_in/X_bd must be 16-byte aligned");
    if (bf16) {
      PGCN_REQUIRE(a->A_bf16 && a->X_in_bf16 && aligned16(a->A_bf16) && aligned16(a->X_in_bf16) && a->ld_in % 8 == 0,
                   "pgcn_sage_layer_fwd: bf16 path needs A_bf16 and X_in_bf16 (16-byte aligned) and ld_in % 8 == 0");
    } else {
      PGCN_REQUIRE(a->A, "pgcn_sage_layer_fwd: fp32 path needs A");
    }
    PGCN_REQUIRE(!a->A || aligned16(a->A), "pgcn_sage_layer_fwd: A must be 16-byte aligned");
  }
  const size_t need = fwd_ws(p, a->f_in, a->f_out, a->gemm_dtype);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need))
    return set_error(PGCN_EWORKSPACE, "pgcn_sage_layer_fwd: workspace too small");
  if (p->n_inner == 0) return PGCN_OK;

  // z = P_i [X_in ; X_bd] (mean over N(v))
  AggArgs g{};
  g.plan = &agg_plan(p, false, a->f_in);
  g.col = p->d_col;
  g.in_split = p->n_inner;
  g.in_lo = a->X_in;
  g.in_hi = p->n_bd > 0 ? a->X_bd : nullptr;
  g.out_split = p->n_inner;
  g.out_lo = a->A;
  g.out_bf16 = bf16 ? a->A_bf16 : nullptr;
  g.scale = p->d_inv_deg;
  g.f = a->f_in;
  g.ld_in = a->ld_in;
  g.ld_out = a->ld_in;
  g.ld_bf16 = a->ld_in;
  g.partials = (float *)a->workspace;
  if (!a->A && (g.plan->chunks > 1 || g.plan->hub.rows > 0)) {
    g.out_lo = (float *)((char *)a->workspace + align_up(aggregate_workspace(*g.plan, a->f_in), 256));
    g.ld_out = ld4(a->f_in);
  }
  g.trace_kind = PGCN_TK_AGG_FWD;
  rc = launch_aggregate(g, s);
  if (rc) return rc;

  // H_out = z W_top, then H_out = act(H_out + X_in W_bot)
  GemmArgs m{};
  m.M = (int32_t)p->n_inner;
  m.N = a->f_out;
  m.K = a->f_in;
  m.dtype = a->gemm_dtype;
  m.A = a->A;
  m.A16 = a->A_bf16;
  m.lda = a->ld_in;
  m.B = a->W;
  m.ldb = a->f_out;
  m.C = a->H_out;
  m.ldc = a->ld_out;
  m.workspace = (float *)((char *)a->workspace + fwd_agg_bytes(p, a->f_in, a->gemm_dtype));
  m.workspace_bytes = gemm_nk_workspace(a->f_out, a->f_in, a->gemm_dtype);
  rc = launch_gemm_nk(Gemm::NN_PLAIN, m, s);
  if (rc) return rc;
  m.A = a->X_in;
  m.A16 = a->X_in_bf16;
  m.B = a->W + (size_t)a->f_in * a->f_out;
  set_send(m, p, a->send_out);
  return launch_gemm_nk(a->relu ? Gemm::NN_ACC_RELU : Gemm::NN_ACC_PLAIN, m, s);
} catch (...) {
  return exception_status("pgcn_sage_layer_fwd");
}

extern "C" int pgcn_sage_layer_bwd(const pgcn_partition *p, const pgcn_sage_bwd_args *a, hipStream_t s) try {
  int rc = check_part(p, "pgcn_sage_layer_bwd");
  if (rc) return rc;
  PGCN_REQUIRE(!p->self_loop, "pgcn_sage_layer_bwd: the partition must be built with PGCN_SETUP_NO_SELF_LOOP");
  PGCN_REQUIRE(a, "pgcn_sage_layer_bwd: null args");
  PGCN_REQUIRE(a->f_in >= 1 && a->f_out >= 1, "pgcn_sage_layer_bwd: widths must be >= 1");
  PGCN_REQUIRE(a->f_in <= PGCN_MAX_WIDTH && a->f_out <= PGCN_MAX_WIDTH, "pgcn_sage_layer_bwd: widths above PGCN_MAX_WIDTH");
  PGCN_REQUIRE(a->gemm_dtype == PGCN_F32 || a->gemm_dtype == PGCN_BF16, "pgcn_sage_layer_bwd: bad gemm_dtype");
  PGCN_REQUIRE(a->ld_in >= a->f_in && a->ld_in % 4 == 0, "pgcn_sage_layer_bwd: ld_in must be >= f_in and a multiple of 4");
  PGCN_REQUIRE(a->ld_out >= a->f_out && a->ld_out % 4 == 0,
               "pgcn_sage_layer_bwd: ld_out must be >= f_out and a multiple of 4");
  PGCN_REQUIRE(a->order == PGCN_ORDER_AGG || a->order == PGCN_ORDER_TRANSFORM, "pgcn_sage_layer_bwd: bad order");
  if (a->order == PGCN_ORDER_TRANSFORM) return sage_bwd_transform(p, a, s);
  const bool bf16 = a->gemm_dtype == PGCN_BF16;
  const bool input_grad = a->J_in != nullptr || a->J_bd_out != nullptr;
  PGCN_REQUIRE(a->dW, "pgcn_sage_layer_bwd: null dW");
  if (input_grad) {
    PGCN_REQUIRE(a->J_in && (a->J_bd_out || p->n_bd == 0),
                 "pgcn_sage_layer_bwd: J_in and J_bd_out must both be given (or both NULL)");
    PGCN_REQUIRE(aligned16(a->J_in) && aligned16(a->J_bd_out),
                 "pgcn_sage_layer_bwd: J_in/J_bd_out must be 16-byte aligned");
  }
  if (p->n_inner > 0) {
    PGCN_REQUIRE(a->J_out && a->W, "pgcn_sage_layer_bwd: null J_out or W");
    PGCN_REQUIRE(!a->relu || a->H_out, "pgcn_sage_layer_bwd: relu needs H_out as mask source");
    PGCN_REQUIRE(aligned16(a->J_out) && aligned16(a->H_out), "pgcn_sage_layer_bwd: J_out/H_out must be 16-byte aligned");
    if (bf16)
      PGCN_REQUIRE(a->A_bf16 && a->X_in_bf16 && aligned16(a->A_bf16) && aligned16(a->X_in_bf16) && a->ld_in % 8 == 0,
                   "pgcn_sage_layer_bwd: bf16 path needs A_bf16 and X_in_bf16 (16-byte aligned) and ld_in % 8 == 0");
    else
      PGCN_REQUIRE(a->A && a->X_in && aligned16(a->A) && aligned16(a->X_in),
                   "pgcn_sage_layer_bwd: fp32 path needs A and X_in (16-byte aligned)");
  }
  const size_t need = bwd_ws(p, a->f_in, a->f_out, input_grad, a->gemm_dtype);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need))
    return set_error(PGCN_EWORKSPACE, "pgcn_sage_layer_bwd: workspace too small");

  // dW = [z, X_in]^T (J ∘ 1[H > 0]): the two row blocks of dW; zero without inner rows
  const size_t half = (size_t)a->f_in * a->f_out;
  GemmArgs g{};
  g.M = a->f_in;
  g.N = a->f_out;
  g.K = (int32_t)p->n_inner;
  g.dtype = a->gemm_dtype;
  g.A = a->A;
  g.A16 = a->A_bf16;
  g.lda = a->ld_in;
  g.B = a->J_out;
  g.ldb = a->ld_out;
  g.Hmask = a->relu ? a->H_out : nullptr;
  g.ldm = a->ld_out;
  g.C = a->dW;
  g.ldc = a->f_out;
  g.workspace = (float *)a->workspace;
  g.workspace_bytes = a->workspace_bytes;
  uint16_t *M16 = p->n_inner > 0 ? m16_ptr(p, a->workspace, a->f_in, a->f_out, input_grad, a->gemm_dtype) : nullptr;
  g.M16 = M16;
  g.ldm16 = ld_m16(a->f_out);
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, g, s);
  if (rc) return rc;
  g.A = a->X_in;
  g.A16 = a->X_in_bf16;
  g.C = a->dW + half;
  g.M16 = nullptr;
  rc = launch_gemm(Gemm::TN_MASK_SPLITK, g, s);
  if (rc) return rc;
  if (!input_grad || p->n_inner == 0) return PGCN_OK;

  // J_in = (J ∘ 1[H > 0]) W_bot^T (the self term), D = diag(1/d) ((J ∘ 1[H > 0]) W_top^T),
  // then J_full = (P_i^T without the scale) D, added to the inner rows
  const int64_t ld_d = ldw(a->f_in);
  float *D = (float *)a->workspace;
  float *partials = (float *)((char *)a->workspace + align_up((size_t)p->n_inner * ld_d * sizeof(float), 256));
  GemmArgs d{};
  d.M = (int32_t)p->n_inner;
  d.N = a->f_in;
  d.K = a->f_out;
  d.dtype = a->gemm_dtype;
  d.A = a->J_out;
  d.lda = a->ld_out;
  d.Hmask = a->relu ? a->H_out : nullptr;
  d.ldm = a->ld_out;
  d.B = a->W + half;
  d.ldb = a->f_out;
  d.C = a->J_in;
  d.ldc = a->ld_in;
  d.workspace = (float *)((char *)a->workspace + bwd_region0(p, a->f_in, a->f_out, input_grad));
  d.workspace_bytes = gemm_nk_workspace(a->f_in, a->f_out, a->gemm_dtype);
  if (M16) {                       // bf16 path: the masked operand as the weight-gradient kernel rounded it
    d.A = nullptr;
    d.A16 = M16;
    d.lda = ld_m16(a->f_out);
    d.Hmask = nullptr;
  }
  rc = launch_gemm_nk(M16 ? Gemm::NT16_PLAIN : Gemm::MASK_NT_PLAIN, d, s);
  if (rc) return rc;
  d.B = a->W;
  d.C = D;
  d.ldc = ld_d;
  d.rowscale = p->d_inv_deg;
  rc = launch_gemm_nk(M16 ? Gemm::NT16_ROWSCALE : Gemm::MASK_NT_ROWSCALE, d, s);
  if (rc) return rc;

  AggArgs t{};
  t.plan = &agg_plan(p, true, a->f_in);
  t.col = p->d_col_t;
  t.in_split = p->n_inner;
  t.in_lo = D;
  t.out_split = p->n_inner;
  t.out_lo = a->J_in;
  t.out_hi = a->J_bd_out;
  t.f = a->f_in;
  t.ld_in = ld_d;
  t.ld_out = a->ld_in;
  t.partials = partials;
  t.trace_kind = PGCN_TK_AGG_BWD;
  t.accum_lo = 1;
  return launch_aggregate(t, s);
} catch (...) {
  return exception_status("pgcn_sage_layer_bwd");
}

extern "C" int pgcn_dropout(float *out, const float *in, int64_t rows, int32_t cols, int64_t ld, int64_t row0,
                            double p, uint32_t seed, uint32_t part, uint32_t layer, uint32_t iteration,
                            uint16_t *out_bf16, int64_t ld_bf16, hipStream_t s) try {
  PGCN_REQUIRE(rows >= 0 && cols >= 0 && ld >= cols && ld % 4 == 0 && row0 >= 0, "pgcn_dropout: bad shape or stride");
  PGCN_REQUIRE(p >= 0.0 && p < 1.0, "pgcn_dropout: p must be in [0, 1)");
  if (rows == 0 || cols == 0) return PGCN_OK;
  PGCN_REQUIRE(out && in && aligned16(out) && aligned16(in), "pgcn_dropout: null or unaligned buffer");
  PGCN_REQUIRE(!out_bf16 || (aligned16(out_bf16) && ld_bf16 >= ld4(cols) && ld_bf16 % 8 == 0),
               "pgcn_dropout: out_bf16 needs 16-byte alignment and ld_bf16 % 8 == 0, >= cols");
  const double t = std::floor(p * 4294967296.0);
  const uint32_t thr = t >= 4294967295.0 ? 0xffffffffu : (uint32_t)t;
  const float scale = (float)(1.0 / (1.0 - p));
  return launch_dropout(out, in, rows, cols, ld, row0, thr, scale, seed, part, layer, iteration, out_bf16, ld_bf16, s);
} catch (...) {
  return exception_status("pgcn_dropout");
}

extern "C" int pgcn_adam_update(float *W, const float *G, const float *G_peer, float *m, float *v, int64_t count,
                                double lr, double beta1, double beta2, double eps, int32_t t, hipStream_t s) try {
  PGCN_REQUIRE(count >= 0 && t >= 1, "pgcn_adam_update: count must be >= 0 and t >= 1");
  PGCN_REQUIRE(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0, "pgcn_adam_update: betas must be in [0, 1)");
  if (count == 0) return PGCN_OK;
  PGCN_REQUIRE(W && G && m && v, "pgcn_adam_update: null buffer");
  AdamCoef c;
  c.lr = (float)lr;
  c.eps = (float)eps;
  c.b1 = (float)beta1;
  c.b2 = (float)beta2;
  c.omb1 = (float)(1.0 - beta1);
  c.omb2 = (float)(1.0 - beta2);
  c.c1 = (float)(1.0 / (1.0 - std::pow(beta1, (double)t)));
  c.c2 = (float)(1.0 / (1.0 - std::pow(beta2, (double)t)));
  return launch_adam(W, G, G_peer, m, v, count, c, s);
} catch (...) {
  return exception_status("pgcn_adam_update");
}

extern "C" int pgcn_smooth_ema(float *state, const float *incoming, int64_t rows, int32_t cols, int64_t ld,
                               float gamma, hipStream_t s) try {
  PGCN_REQUIRE(rows >= 0 && cols >= 0 && ld >= cols && ld % 4 == 0, "pgcn_smooth_ema: bad shape or stride");
  if (rows == 0 || cols == 0) return PGCN_OK;
  PGCN_REQUIRE(state && incoming && aligned16(state) && aligned16(incoming),
               "pgcn_smooth_ema: null or unaligned buffer");
  return launch_ema(state, incoming, rows, cols, ld, gamma, s);
} catch (...) {
  return exception_status("pgcn_smooth_ema");
}

extern "C" int pgcn_pack_boundary(const pgcn_partition *p, int32_t kind, const float *src, float *dst, int32_t cols,
                                  int64_t ld, hipStream_t s) try {
  int rc = check_part(p, "pgcn_pack_boundary");
  if (rc) return rc;
  PGCN_REQUIRE(kind == PGCN_PACK_FEAT || kind == PGCN_ACCUM_GRAD, "pgcn_pack_boundary: bad kind");
  PGCN_REQUIRE(cols >= 0 && ld >= cols && ld % 4 == 0, "pgcn_pack_boundary: bad shape or stride");
  if (p->n_send == 0 || cols == 0) return PGCN_OK;
  PGCN_REQUIRE(src && dst && aligned16(src) && aligned16(dst), "pgcn_pack_boundary: null or unaligned buffer");
  if (kind == PGCN_PACK_FEAT) return launch_pack(p->d_send_idx, p->n_send, src, dst, cols, ld, s);
  return launch_accum(p->d_inv_ptr, p->d_inv_k, p->n_inner, src, dst, cols, ld, s);
} catch (...) {
  return exception_status("pgcn_pack_boundary");
}

extern "C" int pgcn_accum_smoothed(const pgcn_partition *p, const float *incoming, float *state, float gamma,
                                   float *dst, int32_t cols, int64_t ld, hipStream_t s) try {
  int rc = check_part(p, "pgcn_accum_smoothed");
  if (rc) return rc;
  PGCN_REQUIRE(cols >= 0 && ld >= cols && ld % 4 == 0, "pgcn_accum_smoothed: bad shape or stride");
  PGCN_REQUIRE(std::isfinite(gamma), "pgcn_accum_smoothed: gamma must be finite");
  if (p->n_send == 0 || cols == 0) return PGCN_OK;
  PGCN_REQUIRE(incoming && state && dst && aligned16(incoming) && aligned16(state) && aligned16(dst),
               "pgcn_accum_smoothed: null or unaligned buffer");
  PGCN_REQUIRE(state != incoming && state != dst, "pgcn_accum_smoothed: state aliases another buffer");
  return launch_accum_ema(p->d_inv_ptr, p->d_inv_k, p->n_inner, incoming, state, gamma, dst, cols, ld, s);
} catch (...) {
  return exception_status("pgcn_accum_smoothed");
}

extern "C" int pgcn_loss_fwd_bwd(int32_t kind, const float *Z, int64_t rows, int32_t classes, int64_t ld,
                                 const int32_t *labels, const float *targets, int64_t ld_t, float scale, float *J,
                                 float *loss_out, void *workspace, size_t workspace_bytes, hipStream_t s) try {
  PGCN_REQUIRE(kind == PGCN_SOFTMAX_CE || kind == PGCN_SIGMOID_BCE, "pgcn_loss_fwd_bwd: bad kind");
  PGCN_REQUIRE(rows >= 0 && classes >= 1 && ld >= classes, "pgcn_loss_fwd_bwd: bad shape or stride");
  PGCN_REQUIRE(loss_out, "pgcn_loss_fwd_bwd: null loss_out");
  if (rows > 0) {
    PGCN_REQUIRE(Z && J, "pgcn_loss_fwd_bwd: null Z or J");
    if (kind == PGCN_SOFTMAX_CE) PGCN_REQUIRE(labels, "pgcn_loss_fwd_bwd: softmax-CE needs labels");
    else PGCN_REQUIRE(targets && ld_t >= classes, "pgcn_loss_fwd_bwd: BCE needs targets with ld_t >= classes");
  }
  if (!workspace || workspace_bytes < loss_workspace(rows))
    return set_error(PGCN_EWORKSPACE, "pgcn_loss_fwd_bwd: workspace too small");
  return launch_loss(kind, Z, rows, classes, ld, labels, targets, ld_t, scale, J, loss_out, (float *)workspace, s);
} catch (...) {
  return exception_status("pgcn_loss_fwd_bwd");
}

extern "C" int pgcn_sgd_update(float *W, const float *G, const float *G_peer, int64_t count, float eta,
                               hipStream_t s) try {
  PGCN_REQUIRE(count >= 0, "pgcn_sgd_update: negative count");
  if (count == 0) return PGCN_OK;
  PGCN_REQUIRE(W && G, "pgcn_sgd_update: null W or G");
  return launch_sgd(W, G, G_peer, count, eta, s);
} catch (...) {
  return exception_status("pgcn_sgd_update");
}

namespace {
// True when `p` is device memory of this process (not host memory, pinned or not).
bool is_device_memory(const void *p) {
  hipPointerAttribute_t attr{};
  const hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();        // unregistered host memory: clear the sticky error
    return false;
  }
  return attr.type == hipMemoryTypeDevice;
}
}  // namespace

extern "C" int pgcn_refill_async(void *dst, const void *src, size_t bytes, uint32_t flags, hipStream_t s) try {
  if (bytes == 0) return PGCN_OK;
  PGCN_REQUIRE(dst && src, "pgcn_refill_async: null buffer");
  PGCN_REQUIRE((flags & ~(uint32_t)(PGCN_REFILL_DMA | PGCN_REFILL_FROM_HOST)) == 0, "pgcn_refill_async: unknown flags");
  if (flags & PGCN_REFILL_FROM_HOST) {
    hipPointerAttribute_t attr{};
    const hipError_t e = hipPointerGetAttributes(&attr, src);
    if (e != hipSuccess) (void)hipGetLastError();        // unregistered host memory: clear the sticky error
    PGCN_REQUIRE(e == hipSuccess && attr.type == hipMemoryTypeHost,
                 "pgcn_refill_async: PGCN_REFILL_FROM_HOST needs a pinned host source");
    TraceScope ts(PGCN_TK_REFILL, s);
    PGCN_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s));
    return PGCN_OK;
  }
  TraceScope ts(PGCN_TK_REFILL, s);
  // flags = 0, at least kRefillKernelMin bytes, 16-byte-aligned device buffers: the library's
  // non-temporal copy kernel.  Anything else goes to the runtime's copy, which validates host
  // pointers itself; small copies skip the pointer lookups (microseconds each) that the
  // kernel path needs.
  constexpr size_t kRefillKernelMin = size_t(4) << 20;
  const bool vec = (bytes % 16) == 0 && ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 15) == 0;
  if (!(flags & PGCN_REFILL_DMA) && vec && bytes >= kRefillKernelMin && is_device_memory(dst) && is_device_memory(src))
    return launch_refill_copy(dst, src, bytes, s);
  PGCN_HIP(hipMemcpyAsync(dst, src, bytes, (flags & PGCN_REFILL_DMA) ? hipMemcpyDeviceToDeviceNoCU : hipMemcpyDeviceToDevice, s));
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_refill_async");
}

/*
 * pgcn.h — C ABI of libpgcn: one partition's PipeGCN training step on
 * AMD Instinct MI355X (gfx950).
 *
 * The operations follow the paper "PipeGCN: Efficient Full-Graph Training of
 * Graph Convolutional Networks with Pipelined Feature Communication"
 * (ICLR 2022):
 *   - Algorithm 1 (per-partition view): set-up of the inner, boundary and
 *     send sets; forward, loss, backward, AllReduce and SGD per iteration;
 *   - Section 3.2: the mean aggregator with one-iteration-stale boundary
 *     features and boundary feature gradients;
 *   - Section 3.4: moving-average smoothing of stale features and gradients;
 *   - Appendix A.1: the layer function Z = P H W, H' = σ(Z) and its two
 *     gradients, with P split into intra- and inter-partition parts.
 *
 * Conventions shared by every call
 * --------------------------------
 * Status:    every int-returning call returns PGCN_OK (0) or a PGCN_E* code;
 *            pgcn_last_error() gives a thread-local message for the last
 *            failure.  No C++ exception crosses this interface.
 * Memory:    the caller owns every activation, weight, gradient and buffer
 *            (device memory, fp32 unless stated).  The library owns only the
 *            partition handle's index arrays.  Scratch memory is passed in as
 *            `workspace` (size from pgcn_workspace_size()).
 * Layout:    dense matrices are row-major with an explicit row stride `ld`
 *            (in elements).  fp32 matrices read by the aggregation kernels
 *            need ld % 4 == 0 and 16-byte aligned bases; bf16 matrices need
 *            ld % 8 == 0.  Columns [f, ld) are padding: never read as data;
 *            the aggregation kernels write zeros there.  Weight matrices W
 *            and weight gradients dW are compact [f_in x f_out].
 * Streams:   compute calls only enqueue work on the given stream; nothing
 *            synchronises the host except pgcn_partition_setup/destroy.
 * Threads:   a partition handle is immutable after set-up; concurrent calls
 *            on different streams with disjoint outputs and workspaces are
 *            safe.
 * Determinism: no floating-point atomics are used; results are bitwise
 *            reproducible for identical inputs and launch configuration.
 */
#ifndef PGCN_H
#define PGCN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PGCN_VERSION 165

enum pgcn_status {
  PGCN_OK = 0,
  PGCN_EINVAL = 1,        /* null pointer, bad size, bad stride, bad enum       */
  PGCN_ENOMEM = 2,        /* device or host allocation failed during set-up     */
  PGCN_EHIP = 3,          /* a HIP runtime call failed (message has its text)   */
  PGCN_EUNSUPPORTED = 4,  /* device is not gfx950, or an unsupported combination */
  PGCN_EWORKSPACE = 5     /* workspace missing or smaller than required          */
};

/* Arithmetic of the update GEMMs.  PGCN_F32: fp32 operands, fp32 results
 * and fp32 accumulation.  Each product is formed from an exact split of
 * both fp32 operands into three bf16 parts (x = hi + mid + lo), six part
 * products each, on the bf16 matrix cores.  Each part product is exact in
 * fp32, and the three dropped ones are together below 2^-21 (1 + 2^-7) of
 * the product, so results carry fp32 accuracy.  The environment variable
 * PGCN_GEMM_F32=native (read per call) selects the fp32 matrix cores
 * instead.  A non-finite operand gives a non-finite (NaN) result.
 * PGCN_BF16: operands rounded once to bf16 (nearest even), products
 * accumulated in fp32. */
enum pgcn_dtype { PGCN_F32 = 0, PGCN_BF16 = 1 };

enum pgcn_setup_flags {
  PGCN_SETUP_HOST_ONLY = 1,     /* build the index structures on the host only: no
                                   device upload; compute calls on such a handle
                                   return PGCN_EINVAL (used to test the builder
                                   without a GPU) */
  PGCN_SETUP_NO_SELF_LOOP = 2,  /* P_i is the mean over N(v) without the self loop
                                   (the GraphSAGE layer's aggregation, Section 2):
                                   entries 1/d_v with d_v = degree; a row without
                                   neighbours is zero.  The sets V_i, B_i, S_{i,j}
                                   are unchanged. */
  PGCN_SETUP_SYMMETRIC = 4      /* P_i is the symmetric normalisation of Appendix
                                   A.1, rows of D̃^{-1/2} (A + I) D̃^{-1/2}: entries
                                   1 / sqrt(d̃_v d̃_u) with d̃ the whole-graph degree + 1
                                   of every inner and boundary node (the boundary
                                   nodes' degrees come from their full rows of the
                                   global CSR).  GCN layers only; not with
                                   PGCN_SETUP_NO_SELF_LOOP. */
};

enum pgcn_pack_kind {
  PGCN_PACK_FEAT = 0,     /* dst[k, :] = src[send_idx[k], :] for k in [0, n_send)       */
  PGCN_ACCUM_GRAD = 1     /* dst[u, :] += sum_{k : send_idx[k] == u} src[k, :], ascending k */
};

enum pgcn_loss_kind { PGCN_SOFTMAX_CE = 0, PGCN_SIGMOID_BCE = 1 };

/* Association in which a GCN layer evaluates its product P H W (Appendix
 * A.1's layer function; the paper fixes none): aggregate first, (P H) W, or
 * transform first, P (H W), which aggregates f_out instead of f_in columns
 * and pays when the layer narrows (f_out < f_in). */
enum pgcn_layer_order { PGCN_ORDER_AGG = 0, PGCN_ORDER_TRANSFORM = 1 };

/* Global graph on the host.  Must be symmetric (u in N(v) <=> v in N(u)).
 * Duplicate entries and self loops are allowed and removed; exactly one
 * self loop per inner row is added (Ã = A + I, Appendix A.1) unless the
 * partition is built with PGCN_SETUP_NO_SELF_LOOP. */
typedef struct {
  int64_t n;               /* global node count                     */
  const int64_t *rowptr;   /* [n+1], rowptr[0] == 0, non-decreasing */
  const int32_t *col;      /* [rowptr[n]], values in [0, n)         */
} pgcn_csr;

/* Which partition owns each node (Algorithm 1's input: partition id i, count n). */
typedef struct {
  int32_t nparts;          /* partition count, >= 1                 */
  int32_t self;            /* the partition to build, in [0, nparts) */
  const int32_t *owner;    /* [n] host, values in [0, nparts)        */
} pgcn_boundary_map;

typedef struct pgcn_partition pgcn_partition;

/* Tuning overrides (environment variables; none is needed for correct use):
 *   PGCN_AGG_CHUNKS    column chunks of the aggregation plans, 1..64 (read by
 *                      pgcn_partition_setup; default: about 8,000 gathered rows
 *                      per chunk, 32,000 for rows of at most 64 floats, while
 *                      rows keep >= 32 non-zeros per chunk);
 *   PGCN_AGG_CHUNKS_T  the same for the plans of P_i^T alone (takes precedence);
 *   PGCN_AGG_CHUNKS_NARROW  the same for the plans of rows of at most 64 floats
 *                      (takes precedence over both);
 *   PGCN_SEGMENT       length at which long rows are split into segments,
 *                      16..1048576 (read by pgcn_partition_setup; default 512);
 *   PGCN_AGG_SLICE_F4  float4 columns per aggregation lane slice: 16, 32 or 64
 *                      (read per call; default 64);
 *   PGCN_TN_BM=128     keeps the fp32 weight-gradient GEMM in 128-row tiles
 *                      (read once; default: 256-row tiles for f_in >= 384);
 *   PGCN_GEMM_F32=native  fp32 update GEMMs on the fp32 matrix cores instead of
 *                      by bf16 parts (read per call; see pgcn_dtype);
 *   PGCN_HUB=0         no dense block on the matrix cores (read by
 *                      pgcn_partition_setup; default: a block of the rows with
 *                      the most non-zeros x the most referenced columns where it
 *                      saves >= 5% of the gathers, reported by pgcn_info);
 *   PGCN_HUB_ROWS, PGCN_HUB_COLS  both > 0: force the block to that many rows
 *                      and columns (clamped to the matrix).
 * Chunks, segments and the dense block set the order in which a row's terms are
 * added (results stay deterministic for a given setting and row width); the
 * slice width and PGCN_TN_BM change only speed; PGCN_GEMM_F32 changes the
 * order of the GEMMs' fp32 sums within the same rounding bound. */

/* Largest layer width (f_in, f_out) the layer entry points accept: the
 * aggregation covers a row in at most 32 launches of up to 512 float4
 * columns.  Wider layers are rejected with PGCN_EINVAL before any launch. */
#define PGCN_MAX_WIDTH 63740

/* Sizes of a built partition. */
typedef struct {
  int64_t n_inner;         /* |V_i|                                           */
  int64_t n_bd;            /* |B_i|                                           */
  int64_t nnz;             /* non-zeros of P_i (with one self loop per inner row
                              unless built with PGCN_SETUP_NO_SELF_LOOP)      */
  int64_t n_send;          /* sum_j |S_{i,j}|                                 */
  int64_t max_row_len;     /* longest row of P_i                              */
  int64_t max_row_len_t;   /* longest row of P_i^T                            */
  int32_t nparts;
  int32_t self;
  int32_t host_only;       /* 1 if built with PGCN_SETUP_HOST_ONLY            */
  int32_t spmm_segment;    /* rows longer than this are split (fixed order)   */
  int64_t spmm_items;      /* work items of the forward aggregation           */
  int64_t spmm_split_slots;/* partial-sum slots of split rows (forward)       */
  int64_t spmmt_items;     /* work items of the transposed aggregation        */
  int64_t spmmt_split_slots;
  int32_t spmm_chunks;     /* column chunks (cache blocking) of P_i           */
  int32_t spmmt_chunks;    /* column chunks of P_i^T                          */
  int32_t symmetric;       /* 1 if built with PGCN_SETUP_SYMMETRIC            */
  int32_t self_loop;       /* 0 if built with PGCN_SETUP_NO_SELF_LOOP         */
  int32_t spmm_chunks_narrow;  /* column chunks of P_i when the aggregated rows
                                  have at most 64 floats                      */
  int32_t spmmt_chunks_narrow; /* the same for P_i^T                          */
  int32_t spmm_hub_rows;   /* rows x columns of the dense block of P_i taken  */
  int32_t spmm_hub_cols;   /* by the matrix cores (0: none)                   */
  int64_t spmm_hub_nnz;    /* its non-zeros                                   */
  int32_t spmmt_hub_rows;  /* the same for P_i^T                              */
  int32_t spmmt_hub_cols;
  int64_t spmmt_hub_nnz;
} pgcn_info;

/* Caller-allocated host buffers for pgcn_partition_export, sized from pgcn_info.
 * Local numbering: inner local id = rank of the global id among owner == self;
 * boundary local id = n_inner + rank by (owner, global id).  Rows of P_i and
 * P_i^T list columns in ascending local id.  The send list holds S_{i,j} for
 * ascending j, each in ascending global id. */
typedef struct {
  int64_t *inner_gid;      /* [n_inner]                       */
  int64_t *bd_gid;         /* [n_bd]                          */
  int64_t *recv_ptr;       /* [nparts+1] boundary rows of owner j: [recv_ptr[j], recv_ptr[j+1]) */
  int64_t *rowptr;         /* [n_inner+1]                     */
  int32_t *col;            /* [nnz]                           */
  int64_t *rowptr_t;       /* [n_inner+n_bd+1]                */
  int32_t *col_t;          /* [nnz]                           */
  int64_t *send_ptr;       /* [nparts+1]                      */
  int32_t *send_idx;       /* [n_send] inner local ids        */
  int64_t *inv_ptr;        /* [n_inner+1]                     */
  int32_t *inv_k;          /* [n_send] positions into send_idx, ascending per row */
  int64_t *deg;            /* [n_inner+n_bd] whole-graph degree + 1 (distinct
                              neighbours, no self loop, plus one) */
} pgcn_arrays;

/*
 * Partition set-up (Algorithm 1, set-up block; Section 3.1).
 * Builds V_i, B_i, the CSR of P_i (entries 1/d_v, d_v = row length = degree
 * + 1), its transpose, the send sets S_{i,j} = B_j ∩ V_i, the inverse send
 * map and the fixed-order work plan of the aggregation kernels; uploads them
 * to the current device.  Host-synchronous.  `flags` is a mask of
 * pgcn_setup_flags.  On success *out receives a handle freed by
 * pgcn_partition_destroy.  Errors: PGCN_EINVAL (bad graph or map),
 * PGCN_ENOMEM, PGCN_EHIP, PGCN_EUNSUPPORTED (current device not gfx950).
 */
int pgcn_partition_setup(const pgcn_csr *csr, const pgcn_boundary_map *bmap, uint32_t flags,
                         pgcn_partition **out);
int pgcn_partition_info(const pgcn_partition *part, pgcn_info *out);
/* Copies every index array into caller buffers (host).  Any member may be NULL to skip it. */
int pgcn_partition_export(const pgcn_partition *part, const pgcn_arrays *host_out);
void pgcn_partition_destroy(pgcn_partition *part);

/* Bytes of workspace that pgcn_layer_fwd / pgcn_layer_bwd / pgcn_loss_fwd_bwd need
 * for these widths (the maximum over the three), aggregate-first layers. */
size_t pgcn_workspace_size(const pgcn_partition *part, int32_t f_in, int32_t f_out, int32_t gemm_dtype);
/* The same for a GCN or GraphSAGE layer evaluated in `order`
 * (pgcn_layer_order); returns 0 for a bad order.  PGCN_ORDER_AGG gives
 * pgcn_workspace_size. */
size_t pgcn_layer_workspace_size(const pgcn_partition *part, int32_t f_in, int32_t f_out, int32_t gemm_dtype,
                                 int32_t order);

/*
 * One layer forward (Algorithm 1's forward update; Section 3.2 forward
 * equation; Appendix A.1 layer function):
 *     A = P_i [H_in ; H_bd]        fresh inner rows, stale boundary rows
 *     Z = A W ;  H_out = relu(Z) if relu else Z
 * H_bd holds the boundary rows to use (the received stale buffer, or its
 * smoothing state); NULL means all-zero boundary rows (iteration 1).
 * With gemm_dtype == PGCN_BF16, A is rounded once to bf16 (round to nearest
 * even) into A_bf16, W is rounded to bf16 and the product accumulates in
 * fp32; A (fp32) may then be NULL, or A_bf16 may be NULL when A is given
 * (A is then rounded while staged: the same values).  With PGCN_F32, A is
 * required and A_bf16 ignored.
 * order == PGCN_ORDER_TRANSFORM evaluates the same layer as
 *     Y = [H_in ; H_bd] W            (n_inner + n_bd rows, in the workspace)
 *     H_out = relu(P_i Y) if relu else P_i Y
 * (bf16 path: H and W rounded to bf16, fp32 accumulation; the aggregation
 * stays fp32).  A and A_bf16 are then unused and may be NULL; the backward
 * takes the layer input instead.  Workspace: pgcn_layer_workspace_size with
 * the same order.
 * a_given == 1 (aggregate first only) skips the aggregation: A is an input
 * holding P_i [H_in ; H_bd], e.g. a layer-1 aggregate kept across iterations
 * (the input features are constant); H_in / H_bd are then not read.
 */
typedef struct {
  int32_t f_in, f_out;         /* 1 .. PGCN_MAX_WIDTH                            */
  int32_t gemm_dtype;          /* pgcn_dtype                                    */
  int32_t relu;                /* 1: H_out = relu(Z); 0: H_out = Z (last layer)  */
  int64_t ld_in;               /* stride of H_in, H_bd, A, A_bf16 (elements)     */
  int64_t ld_out;              /* stride of H_out                                */
  const float *H_in;           /* [n_inner, ld_in]                               */
  const float *H_bd;           /* [n_bd, ld_in] or NULL                          */
  const float *W;              /* [f_in, f_out]                                  */
  float *A;                    /* [n_inner, ld_in] out                           */
  uint16_t *A_bf16;            /* [n_inner, ld_in] out (bf16 bits)               */
  float *H_out;                /* [n_inner, ld_out] out                          */
  void *workspace;
  size_t workspace_bytes;
  int32_t order;               /* pgcn_layer_order (0: aggregate first)           */
  int32_t a_given;             /* 1: A (fp32) already holds P_i [H_in ; H_bd]; only
                                  the update runs (aggregate first; on the bf16
                                  path A is rounded while staged, A_bf16 unused) */
  float *send_out;             /* [n_send, ld_out] or NULL: also writes the rows of
                                  H_out that this partition sends (Algorithm 1's
                                  forward send of the next layer's input), row k =
                                  H_out[send_idx[k]], columns [0, f_out); the kernel
                                  that writes H_out writes them (no second pass over
                                  H_out). 16-byte aligned. */
} pgcn_fwd_args;
int pgcn_layer_fwd(const pgcn_partition *part, const pgcn_fwd_args *args, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * layer forward as pgcn_layer_fwd (same kernels, same results bit for bit),
 * with its workspace taken from a fixed array inside this library instead of
 * args->workspace.  Nothing is allocated by the call.
 *
 * args->workspace must be NULL and args->workspace_bytes 0 (else
 * PGCN_EINVAL); every other argument is as for pgcn_layer_fwd, and the
 * caller still owns and passes every input and output.  A layer whose
 * workspace (pgcn_layer_workspace_size's forward share) exceeds
 * PGCN_NOALLOC_SCRATCH_BYTES is rejected with PGCN_EWORKSPACE before any
 * launch.  The array holds PGCN_NOALLOC_SCRATCH_BYTES on every GPU the
 * library runs on, until the process ends; its address on a device is
 * resolved when a partition is set up there.
 *
 * All calls on one GPU share that GPU's array and it keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on one
 * GPU (two streams, two threads, two graphs replayed concurrently) race and
 * must be serialised by the caller.
 */
#define PGCN_NOALLOC_SCRATCH_BYTES (32u << 20)
int pgcn_layer_fwd_noalloc(const pgcn_partition *part, const pgcn_fwd_args *args, hipStream_t stream);

/*
 * One layer backward (Algorithm 1's weight- and feature-gradient lines;
 * Appendix A.1 gradients):
 *     M      = J_out ∘ 1[H_out > 0] if relu else J_out
 *     dW     = A^T M
 *     J_full = P_i^T (M W^T)      rows [0, n_inner) -> J_in,
 *                                 rows [n_inner, n_inner+n_bd) -> J_bd_out
 * J_in and J_bd_out are both NULL for the first layer (no feature gradient).
 * Stale gradients from peers are added afterwards with pgcn_pack_boundary
 * (PGCN_ACCUM_GRAD), as Algorithm 1 does after waiting for them.
 * dW accumulates split-K partials in a fixed order (deterministic).
 * order == PGCN_ORDER_TRANSFORM (the layer's forward used that order):
 *     T      = P_i^T M               [n_inner + n_bd, f_out], in the workspace
 *     dW     = [H_in ; H_bd]^T T
 *     J_full = T W^T                 rows split into J_in / J_bd_out as above
 * H_in / H_bd are the input rows the forward used (stride ld_in; H_bd NULL
 * means zero boundary rows); A and A_bf16 are unused.  bf16 path: H, T and W
 * rounded to bf16 (nearest even) for the products, fp32 accumulation.
 * Aggregate first on the bf16 path, A_bf16 may be NULL when A (fp32) is
 * given: A is then rounded to bf16 while staged (the same values).
 */
typedef struct {
  int32_t f_in, f_out;
  int32_t gemm_dtype;
  int32_t relu;
  int64_t ld_in, ld_out;
  const float *J_out;          /* [n_inner, ld_out]                              */
  const float *H_out;          /* [n_inner, ld_out] mask source (when relu)      */
  const float *A;              /* [n_inner, ld_in] (PGCN_F32)                    */
  const uint16_t *A_bf16;      /* [n_inner, ld_in] (PGCN_BF16)                   */
  const float *W;              /* [f_in, f_out]                                  */
  float *dW;                   /* [f_in, f_out] out                              */
  float *J_in;                 /* [n_inner, ld_in] out or NULL                   */
  float *J_bd_out;             /* [n_bd, ld_in] out or NULL                      */
  void *workspace;
  size_t workspace_bytes;
  int32_t order;               /* pgcn_layer_order (0: aggregate first)           */
  const float *H_in;           /* [n_inner, ld_in] layer input (PGCN_ORDER_TRANSFORM) */
  const float *H_bd;           /* [n_bd, ld_in] or NULL       (PGCN_ORDER_TRANSFORM) */
} pgcn_bwd_args;
int pgcn_layer_bwd(const pgcn_partition *part, const pgcn_bwd_args *args, hipStream_t stream);

/*
 * Moving-average smoothing of stale features or gradients (Section 3.4):
 *     state[r, c] = gamma * state[r, c] + (1 - gamma) * incoming[r, c]
 * for r < rows, c < cols; both matrices share stride ld (ld % 4 == 0).
 */
int pgcn_smooth_ema(float *state, const float *incoming, int64_t rows, int32_t cols, int64_t ld,
                     float gamma, hipStream_t stream);

/*
 * Boundary packing (Algorithm 1's send of H_{S_{i,j}} and the accumulation of
 * received gradients C_j into rows S_{i,j}, ascending j):
 *   PGCN_PACK_FEAT : dst[k, :] = src[send_idx[k], :],   src [n_inner, ld], dst [n_send, ld]
 *   PGCN_ACCUM_GRAD: dst[u, :] += src[k, :] for each k with send_idx[k] == u, in
 *                    ascending k;                      src [n_send, ld], dst [n_inner, ld]
 */
int pgcn_pack_boundary(const pgcn_partition *part, int32_t kind, const float *src, float *dst,
                       int32_t cols, int64_t ld, hipStream_t stream);

/*
 * Smoothing of the received gradients (Section 3.4) fused with their
 * accumulation (Algorithm 1's loop over peers j): for every send row k,
 *     state[k, :] = gamma * state[k, :] + (1 - gamma) * incoming[k, :]
 * and dst[u, :] += state[k, :] for each k with send_idx[k] == u, in ascending
 * k.  The same values as pgcn_smooth_ema(state, incoming, n_send, ...)
 * followed by pgcn_pack_boundary(PGCN_ACCUM_GRAD, state, dst, ...), in one
 * pass.  incoming and state: [n_send, ld]; dst: [n_inner, ld]; ld % 4 == 0,
 * 16-byte aligned; state must not alias incoming or dst.
 */
int pgcn_accum_smoothed(const pgcn_partition *part, const float *incoming, float *state, float gamma, float *dst,
                        int32_t cols, int64_t ld, hipStream_t stream);

/*
 * Loss and its gradient w.r.t. the logits (Algorithm 1's J^(L)):
 *   PGCN_SOFTMAX_CE : loss = scale * sum_r -log softmax(Z_r)[labels[r]]
 *                     J_r  = scale * (softmax(Z_r) - onehot(labels[r]))
 *   PGCN_SIGMOID_BCE: loss = scale * sum_{r,c} BCE(sigmoid(Z_rc), targets_rc)
 *                     J_rc = scale * (sigmoid(Z_rc) - targets_rc)
 * Z and J: [rows, ld]; labels: [rows] int32 in [0, classes); targets: [rows, ld_t].
 * loss_out: one device float, written (not accumulated), reduced in a fixed order.
 */
int pgcn_loss_fwd_bwd(int32_t kind, const float *Z, int64_t rows, int32_t classes, int64_t ld,
                      const int32_t *labels, const float *targets, int64_t ld_t, float scale,
                      float *J, float *loss_out, void *workspace, size_t workspace_bytes,
                      hipStream_t stream);

/* Algorithm 1's update after the AllReduce (a sum): W -= eta * (G + G_peer).
 * G_peer may be NULL (one partition: the AllReduce is the identity). */
int pgcn_sgd_update(float *W, const float *G, const float *G_peer, int64_t count, float eta,
                    hipStream_t stream);

/*
 * Adam update after the AllReduce (the optimiser of the paper's experiments,
 * its setup table; Kingma and Ba, ICLR 2015, Algorithm 1), element-wise for
 * i < count, with g = G + G_peer (G_peer may be NULL):
 *     m = beta1 m + (1 - beta1) g ;  v = beta2 v + (1 - beta2) g^2
 *     W -= lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * t >= 1 is the step count; m and v (caller-owned, zero before the first
 * step) are updated in place.  The coefficients (beta, 1 - beta, the bias
 * corrections) are computed on the host in double precision and rounded
 * once to fp32; the element-wise update runs in fp32.
 */
int pgcn_adam_update(float *W, const float *G, const float *G_peer, float *m, float *v, int64_t count, double lr,
                     double beta1, double beta2, double eps, int32_t t, hipStream_t stream);

/*
 * Dropout of a layer input, applied after the boundary receive with one mask
 * for the forward and the backward (the paper's implementation notes; rates
 * in its setup table).  For r < rows, c < cols, with global row R = row0 + r
 * (the partition's local numbering: inner rows, then boundary rows at
 * row0 = n_inner) and element index q = R * cols + c:
 *     u = word (q mod 4) of Philox4x32-10(counter = (lo32(q / 4), hi32(q / 4),
 *         layer, iteration), key = (seed, part))
 *     out[r, c] = u < floor(p * 2^32) ? 0 : in[r, c] * (1 / (1 - p))
 * Philox4x32-10 is the counter-based generator of Salmon, Moraes, Dror and
 * Shaw (SC 2011).  The same call on a gradient (same arguments) applies the
 * forward's mask in the backward.  in and out share stride ld (ld % 4 == 0,
 * 16-byte aligned) and may alias.  out_bf16 (optional, stride ld_bf16,
 * ld_bf16 % 8 == 0) receives out rounded to bf16 (nearest even).  0 <= p < 1.
 */
int pgcn_dropout(float *out, const float *in, int64_t rows, int32_t cols, int64_t ld, int64_t row0, double p,
                 uint32_t seed, uint32_t part, uint32_t layer, uint32_t iteration, uint16_t *out_bf16,
                 int64_t ld_bf16, hipStream_t stream);

/*
 * GraphSAGE layer forward (Section 2: the update function takes
 * CONCAT(z_v, h_v); the model of the paper's experiments), on a partition
 * built with PGCN_SETUP_NO_SELF_LOOP:
 *     z = P_i [X_in ; X_bd]          (mean over N(v); stale boundary rows)
 *     Z = [z, X_in] W ;  H_out = relu(Z) if relu else Z
 * X_in / X_bd are the layer input after dropout (pgcn_dropout); X_bd NULL
 * means all-zero boundary rows.  W is [2 f_in, f_out]: rows [0, f_in) act
 * on z, rows [f_in, 2 f_in) on X_in.  The product is evaluated as z W_top
 * followed by an accumulation of X_in W_bot (two passes over H_out).
 * PGCN_F32: z -> A (required).  PGCN_BF16: z rounded once to bf16 -> A_bf16,
 * and X_in_bf16 (the bf16 copy of X_in, e.g. from pgcn_dropout) is the
 * self operand; W is rounded to bf16; fp32 accumulation.
 * Workspace: pgcn_workspace_size(part, f_in, f_out, gemm_dtype).
 * order == PGCN_ORDER_TRANSFORM evaluates z W_top as P_i (X W_top):
 *     Y = [X_in ; X_bd] W_top        (n_inner + n_bd rows, in the workspace)
 *     H_out = act(P_i Y + X_in W_bot)
 * (bf16 path: X and W rounded to bf16 for the products); A and A_bf16 are
 * unused.  Workspace: pgcn_layer_workspace_size with that order.
 */
typedef struct {
  int32_t f_in, f_out;
  int32_t gemm_dtype;
  int32_t relu;
  int64_t ld_in, ld_out;       /* strides of X_in, X_bd, A, A_bf16, X_in_bf16 / of H_out */
  const float *X_in;           /* [n_inner, ld_in]                               */
  const uint16_t *X_in_bf16;   /* [n_inner, ld_in] (PGCN_BF16)                   */
  const float *X_bd;           /* [n_bd, ld_in] or NULL                          */
  const float *W;              /* [2 f_in, f_out]                                */
  float *A;                    /* [n_inner, ld_in] out: z (PGCN_F32)             */
  uint16_t *A_bf16;            /* [n_inner, ld_in] out: z in bf16 (PGCN_BF16)    */
  float *H_out;                /* [n_inner, ld_out] out                          */
  void *workspace;
  size_t workspace_bytes;
  int32_t order;               /* pgcn_layer_order (0: aggregate first)           */
  float *send_out;             /* [n_send, ld_out] or NULL: the sent rows of H_out,
                                  as in pgcn_fwd_args                            */
} pgcn_sage_fwd_args;
int pgcn_sage_layer_fwd(const pgcn_partition *part, const pgcn_sage_fwd_args *args, hipStream_t stream);

/*
 * GraphSAGE layer backward (gradients of the forward above):
 *     M        = J_out ∘ 1[H_out > 0] if relu else J_out
 *     dW       = [z, X_in]^T M          (rows [0, f_in): z^T M; rows [f_in, 2 f_in): X_in^T M)
 *     [dz, ds] = M W^T
 *     J_full   = P_i^T dz, plus ds on the inner rows:
 *                rows [0, n_inner) -> J_in, rows [n_inner, n_inner + n_bd) -> J_bd_out
 * J_full is the gradient of the dropped input; apply the dropout mask to it
 * with pgcn_dropout (same arguments as in the forward) before it is sent or
 * accumulated.  J_in and J_bd_out are both NULL for the first layer.
 * order == PGCN_ORDER_TRANSFORM (the forward used that order):
 *     T = P_i^T M                    [n_inner + n_bd, f_out], in the workspace
 *     dW rows [0, f_in) = [X_in ; X_bd]^T T,  rows [f_in, 2 f_in) = X_in^T M
 *     J_full = T W_top^T, plus M W_bot^T on the inner rows
 * X_bd is the (dropped) boundary input the forward used (NULL: zero rows); A
 * and A_bf16 are unused.  bf16 path: X, T, M and W rounded to bf16 for the
 * products.
 */
typedef struct {
  int32_t f_in, f_out;
  int32_t gemm_dtype;
  int32_t relu;
  int64_t ld_in, ld_out;
  const float *J_out;          /* [n_inner, ld_out]                              */
  const float *H_out;          /* [n_inner, ld_out] mask source (when relu)      */
  const float *A;              /* [n_inner, ld_in] z (PGCN_F32)                  */
  const uint16_t *A_bf16;      /* [n_inner, ld_in] z (PGCN_BF16)                 */
  const float *X_in;           /* [n_inner, ld_in] (PGCN_F32)                    */
  const uint16_t *X_in_bf16;   /* [n_inner, ld_in] (PGCN_BF16)                   */
  const float *W;              /* [2 f_in, f_out]                                */
  float *dW;                   /* [2 f_in, f_out] out                            */
  float *J_in;                 /* [n_inner, ld_in] out or NULL                   */
  float *J_bd_out;             /* [n_bd, ld_in] out or NULL                      */
  void *workspace;
  size_t workspace_bytes;
  int32_t order;               /* pgcn_layer_order (0: aggregate first)           */
  const float *X_bd;           /* [n_bd, ld_in] or NULL        (PGCN_ORDER_TRANSFORM) */
} pgcn_sage_bwd_args;
int pgcn_sage_layer_bwd(const pgcn_partition *part, const pgcn_sage_bwd_args *args, hipStream_t stream);

/* Refill of a stale buffer (Algorithm 1's send/receive threads; the paper runs
 * them on a second stream): an asynchronous copy of `bytes` bytes into device
 * memory `dst`, enqueued on `stream`.  flags = 0: device-to-device on the
 * compute units; copies of at least 4 MiB between 16-byte-aligned device
 * buffers (`bytes` a multiple of 16) by the library's copy kernel with
 * non-temporal loads and stores (the copied rows are read in the next
 * iteration, so they bypass the caches the current one uses), others by
 * the runtime's copy; PGCN_REFILL_DMA:
 * device-to-device by the DMA engines, using no compute units (as a transfer
 * arriving from a peer GPU would); PGCN_REFILL_FROM_HOST: `src` is pinned
 * (page-locked) host memory, copied by DMA over the host link (the paper's
 * CPU-staged exchange); other host memory is rejected with PGCN_EINVAL. */
enum pgcn_refill_flags { PGCN_REFILL_DMA = 1, PGCN_REFILL_FROM_HOST = 2 };
int pgcn_refill_async(void *dst, const void *src, size_t bytes, uint32_t flags, hipStream_t stream);

/*
 * Kernel tracing (measurement support).  While enabled, every kernel launch
 * (and every refill copy) of the library is bracketed by a HIP event pair
 * recorded on the launch stream, except that the chunk launches of one
 * aggregation column range (PGCN_TK_AGG_FWD / _BWD), which run back to back,
 * share one pair: each event record costs the stream several microseconds.
 * pgcn_trace_collect waits for the recorded pairs and returns each record's
 * kind (pgcn_trace_kind), duration in ms and the number of launches it spans
 * (`launches`, may be NULL; 1 except for the shared aggregation records,
 * which may span 0 launches when every chunk is empty), then clears the
 * record.  pgcn_trace_enable creates `capacity` event pairs
 * up front (timing-only events without the system-scope cache flush a
 * default event record performs, so tracing does not disturb the caches of
 * the kernels it brackets) and resets the kind filter to "all kinds";
 * launches beyond the capacity are not recorded.  pgcn_trace_filter limits
 * recording to the kinds whose bit (1u << kind) is set in `kind_mask`.  Not
 * for use under graph capture.
 */
enum pgcn_trace_kind {
  PGCN_TK_AGG_FWD = 0, PGCN_TK_AGG_BWD = 1, PGCN_TK_AGG_FIXUP = 2, PGCN_TK_GEMM_FWD = 3,
  PGCN_TK_GEMM_DGRAD = 4, PGCN_TK_GEMM_WGRAD = 5, PGCN_TK_WGRAD_REDUCE = 6, PGCN_TK_EMA = 7,
  PGCN_TK_PACK = 8, PGCN_TK_ACCUM = 9, PGCN_TK_LOSS = 10, PGCN_TK_SGD = 11, PGCN_TK_REFILL = 12,
  PGCN_TK_GEMM_PACK = 13, PGCN_TK_DROPOUT = 14, PGCN_TK_ADAM = 15, PGCN_TK_MASK_SCALE = 16,
  PGCN_TK_ACCUM_EMA = 17
};
int pgcn_trace_enable(int32_t capacity);
int pgcn_trace_filter(uint32_t kind_mask);
int pgcn_trace_collect(int32_t *kinds, float *ms, int32_t *launches, int32_t max_records, int32_t *count);
int pgcn_trace_disable(void);

const char *pgcn_last_error(void);
int pgcn_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PGCN_H */

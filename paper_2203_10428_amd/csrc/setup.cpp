// Partition set-up (Algorithm 1's set-up block; Section 3.1): inner set V_i,
// boundary set B_i, local propagation matrix P_i and its transpose, send sets
// S_{i,j} = B_j ∩ V_i, the inverse send map and the fixed work plans of the
// aggregation kernels.  Host code; the result is uploaded once.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <new>
#include <numeric>
#include <utility>

#include "internal.h"

namespace pgcn {

static thread_local std::string g_error;
// Set when the message itself could not be stored (out of host memory).
static thread_local const char *g_error_static = nullptr;

int set_error(int code, const std::string &msg) noexcept {
  try {
    g_error = msg;
    g_error_static = nullptr;
  } catch (...) {
    g_error_static = "libpgcn: out of host memory while reporting an error";
  }
  return code;
}

static void set_message(const char *fn, const char *what) noexcept {
  try {
    g_error = std::string(fn) + ": " + what;
    g_error_static = nullptr;
  } catch (...) {
    g_error_static = "libpgcn: out of host memory while reporting an error";
  }
}

int exception_status(const char *fn) noexcept {
  int code = PGCN_EINVAL;
  try {
    throw;
  } catch (const std::bad_alloc &) {
    code = PGCN_ENOMEM;
    set_message(fn, "out of host memory");
  } catch (const std::exception &e) {
    set_message(fn, e.what());
  } catch (...) {
    set_message(fn, "unexpected C++ exception");
  }
  return code;
}

int check_hip(hipError_t e, const char *what) {
  return set_error(PGCN_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Number of column chunks of a CSR matrix for cache blocking: chunks of about
// 8,000 gathered rows of 1 KB (measured on MI355X: the Reddit-like forward is
// fastest at 10-11 chunks of its 88,000 columns, the transposed aggregation at
// 7-8 of its 58,000), or 32,000 rows for the narrow plans (rows of at most 256
// bytes: the Reddit-like 41-wide output layer is fastest at 2-4 chunks), but
// only while a row keeps >= 32 non-zeros per chunk on average.
// PGCN_AGG_CHUNKS overrides every plan, PGCN_AGG_CHUNKS_T the transposed ones,
// PGCN_AGG_CHUNKS_NARROW the narrow ones (before the other two).
static int32_t choose_chunks(int64_t nrows, int64_t ncols, int64_t nnz, bool transposed, int64_t rows_per_chunk,
                             bool narrow = false) {
  for (const char *name : {narrow ? "PGCN_AGG_CHUNKS_NARROW" : "", transposed ? "PGCN_AGG_CHUNKS_T" : "",
                           "PGCN_AGG_CHUNKS"}) {
    const char *env = *name ? std::getenv(name) : nullptr;
    if (!env) continue;
    int v = std::atoi(env);
    if (v >= 1 && v <= 64) return v;
  }
  if (nrows == 0 || ncols == 0) return 1;
  const int64_t by_cache = (ncols + rows_per_chunk - 1) / rows_per_chunk;
  const int64_t by_len = (nnz / nrows) / 32;
  int64_t c = std::min(by_cache, by_len);
  return (int32_t)std::max<int64_t>(1, std::min<int64_t>(c, 16));
}

// Cost of one (row, column) pair of a dense block on the matrix cores, in
// units of one gathered non-zero of the same width, measured on MI355X for
// 1 KB rows: each non-zero the block takes off the gather saves about 28.5 ps
// there (the block's columns are the most referenced rows, mostly served by
// the L2, so they cost the gather less than its average non-zero), and the
// block costs 1.6-2.4 ps per pair.  A sweep of this constant on the
// Reddit-like partition (0.02 to 0.08) put the best step at 0.057.
constexpr double kHubPairCost = 0.057;

static int64_t env_int(const char *name, int64_t dflt) {
  const char *v = std::getenv(name);
  return v ? std::atoll(v) : dflt;
}

// The dense block of a CSR matrix for the matrix cores: the rows with the
// most non-zeros x the most referenced columns, sizes on a grid of
// 512 x 2^i (and the full extent), chosen to maximise the non-zeros moved off
// the gather minus kHubPairCost x the block's area; no block when that saving
// is under 5% of the non-zeros or the matrix is small.  PGCN_HUB=0 disables
// it; PGCN_HUB_ROWS / PGCN_HUB_COLS force its size (tests).  Fills the block's
// rows, columns and bits, and the matrix without the block (rowptr_rest,
// col_rest; columns stay ascending).
static void choose_hub(const std::vector<int64_t> &rowptr, const std::vector<int32_t> &col, int64_t nrows,
                       int64_t ncols, Hub &h, std::vector<int64_t> &rowptr_rest, std::vector<int32_t> &col_rest) {
  h = Hub();
  rowptr_rest.clear();
  col_rest.clear();
  const int64_t nnz = (int64_t)col.size();
  if (env_int("PGCN_HUB", 1) == 0 || nrows == 0 || ncols == 0 || nnz == 0) return;
  const int64_t force_r = env_int("PGCN_HUB_ROWS", 0), force_c = env_int("PGCN_HUB_COLS", 0);
  // ranks: rows by decreasing length, columns by decreasing reference count (ties by id)
  std::vector<int64_t> ccount(ncols, 0);
  for (int32_t c : col) ccount[c]++;
  std::vector<int64_t> rord(nrows), cord(ncols);
  std::iota(rord.begin(), rord.end(), 0);
  std::iota(cord.begin(), cord.end(), 0);
  std::stable_sort(rord.begin(), rord.end(),
                   [&](int64_t a, int64_t b) { return rowptr[a + 1] - rowptr[a] > rowptr[b + 1] - rowptr[b]; });
  std::stable_sort(cord.begin(), cord.end(), [&](int64_t a, int64_t b) { return ccount[a] > ccount[b]; });
  std::vector<int64_t> rrank(nrows), crank(ncols);
  for (int64_t i = 0; i < nrows; ++i) rrank[rord[i]] = i;
  for (int64_t i = 0; i < ncols; ++i) crank[cord[i]] = i;
  int64_t R = 0, C = 0;
  if (force_r > 0 && force_c > 0) {
    R = std::min(force_r, nrows);
    C = std::min(force_c, ncols);
  } else {
    if (force_r < 0 || force_c < 0 || nnz < (int64_t)1 << 20) return;
    // grid sizes and a 2D histogram of the non-zeros by (row size class, column size class)
    std::vector<int64_t> gr, gc;
    for (int64_t v = 512; v < nrows; v *= 2) gr.push_back(v);
    gr.push_back(nrows);
    for (int64_t v = 512; v < ncols; v *= 2) gc.push_back(v);
    gc.push_back(ncols);
    auto cls = [](const std::vector<int64_t> &g, int64_t rank) {
      return (int64_t)(std::upper_bound(g.begin(), g.end(), rank) - g.begin());
    };
    const int64_t nr = (int64_t)gr.size(), nc = (int64_t)gc.size();
    std::vector<int64_t> hist((size_t)nr * nc, 0);
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t a = cls(gr, rrank[r]);
      for (int64_t k = rowptr[r]; k < rowptr[r + 1]; ++k) hist[(size_t)a * nc + cls(gc, crank[col[k]])]++;
    }
    double best = 0.05 * (double)nnz;
    for (int64_t i = 0; i < nr; ++i)
      for (int64_t j = 0; j < nc; ++j) {
        int64_t in = 0;
        for (int64_t a = 0; a <= i; ++a)
          for (int64_t b = 0; b <= j; ++b) in += hist[(size_t)a * nc + b];
        const double net = (double)in - kHubPairCost * (double)gr[i] * (double)gc[j];
        if (net > best) {
          best = net;
          R = gr[i];
          C = gc[j];
        }
      }
    if (R == 0) return;
  }
  // hub rows and columns in ascending id; positions of the columns
  std::vector<int32_t> rows, cols;
  for (int64_t r = 0; r < nrows; ++r)
    if (rrank[r] < R) rows.push_back((int32_t)r);
  for (int64_t c = 0; c < ncols; ++c)
    if (crank[c] < C) cols.push_back((int32_t)c);
  std::vector<int32_t> cpos(ncols, -1);
  for (size_t i = 0; i < cols.size(); ++i) cpos[cols[i]] = (int32_t)i;
  h.rows_real = (int32_t)rows.size();
  h.cols_real = (int32_t)cols.size();
  h.rows = (h.rows_real + kHubRowTile - 1) / kHubRowTile * kHubRowTile;
  h.cols = (h.cols_real + kHubColTile - 1) / kHubColTile * kHubColTile;
  h.row_ids.assign(h.rows, -1);
  std::copy(rows.begin(), rows.end(), h.row_ids.begin());
  h.col_ids.assign(h.cols, -1);
  std::copy(cols.begin(), cols.end(), h.col_ids.begin());
  const int64_t ntiles = h.cols / kHubColTile;
  h.bits.assign((size_t)h.rows * ntiles, 0u);
  h.init.assign((size_t)(nrows + 31) / 32, 0u);
  std::vector<int32_t> rpos(nrows, -1);
  for (size_t i = 0; i < rows.size(); ++i) {
    rpos[rows[i]] = (int32_t)i;
    h.init[rows[i] >> 5] |= 1u << (rows[i] & 31);
  }
  rowptr_rest.assign(nrows + 1, 0);
  col_rest.reserve(nnz);
  for (int64_t r = 0; r < nrows; ++r) {
    for (int64_t k = rowptr[r]; k < rowptr[r + 1]; ++k) {
      const int32_t c = col[k];
      if (rpos[r] >= 0 && cpos[c] >= 0) {
        h.bits[(size_t)(cpos[c] / kHubColTile) * h.rows + rpos[r]] |= 1u << (cpos[c] % kHubColTile);
        h.nnz++;
      } else {
        col_rest.push_back(c);
      }
    }
    rowptr_rest[r + 1] = (int64_t)col_rest.size();
  }
}

// Work plan of one aggregation.  A row whose run inside some chunk is longer
// than `segment` is a split row: every run of it, in every chunk, is cut into
// segments of at most `segment` non-zeros that write partial slots; the row's
// slots are contiguous in (chunk, segment) order, and one fix-up pass after
// the last chunk adds them in that order, so results never depend on timing.
// Every other row adds its run of each chunk to the output in chunk order
// (empty runs are skipped except in the first and last chunk, which write
// and finish the row).  Whole runs are scheduled longest first.
static void build_plan(const std::vector<int64_t> &rowptr, const std::vector<int32_t> &col, int64_t nrows,
                       int64_t ncols, int32_t segment, int32_t chunks, Plan &p) {
  p.items.clear();
  p.splits.clear();
  p.slots = 0;
  p.chunks = chunks;
  const int32_t C = p.chunks;
  p.chunk_items.assign(C + 1, 0);
  p.chunk_whole.assign(C, 0);
  // run bounds: row r's run in chunk c is [bnd[r*(C+1)+c], bnd[r*(C+1)+c+1])
  std::vector<int64_t> bnd((size_t)nrows * (C + 1));
  for (int64_t r = 0; r < nrows; ++r) {
    const int32_t *rb = col.data() + rowptr[r], *re = col.data() + rowptr[r + 1];
    int64_t *q = bnd.data() + (size_t)r * (C + 1);
    q[0] = rowptr[r];
    for (int32_t c = 1; c < C; ++c) q[c] = rowptr[r] + (std::lower_bound(rb, re, (int32_t)(ncols * c / C)) - rb);
    q[C] = rowptr[r + 1];
  }
  // split rows and their slot ranges
  std::vector<int64_t> cursor(nrows, -1);
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t *q = bnd.data() + (size_t)r * (C + 1);
    bool split = false;
    int64_t nseg = 0;
    for (int32_t c = 0; c < C; ++c) {
      const int64_t len = q[c + 1] - q[c];
      split |= len > segment;
      nseg += (len + segment - 1) / segment;
    }
    if (!split) continue;
    p.splits.push_back(SplitRow{(int32_t)r, (int32_t)p.slots, (int32_t)nseg, 0});
    cursor[r] = p.slots;
    p.slots += nseg;
  }
  std::vector<int64_t> order;
  order.reserve(nrows);
  for (int32_t c = 0; c < C; ++c) {
    order.clear();
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t b = bnd[(size_t)r * (C + 1) + c], e = bnd[(size_t)r * (C + 1) + c + 1];
      if (cursor[r] >= 0) {
        for (int64_t sb = b; sb < e; sb += segment) {
          const int64_t se = std::min<int64_t>(sb + segment, e);
          p.items.push_back(WorkItem{sb, (int32_t)(se - sb), (int32_t)(-cursor[r]++ - 1)});
        }
      } else if (e > b || c == 0 || c == C - 1) {
        order.push_back(r);
      }
    }
    p.chunk_whole[c] = (int64_t)p.items.size();
    std::stable_sort(order.begin(), order.end(), [&](int64_t x, int64_t y) {
      const int64_t *qx = bnd.data() + (size_t)x * (C + 1) + c, *qy = bnd.data() + (size_t)y * (C + 1) + c;
      return qx[1] - qx[0] > qy[1] - qy[0];
    });
    for (int64_t r : order) {
      const int64_t b = bnd[(size_t)r * (C + 1) + c], e = bnd[(size_t)r * (C + 1) + c + 1];
      p.items.push_back(WorkItem{b, (int32_t)(e - b), (int32_t)r});
    }
    p.chunk_items[c + 1] = (int64_t)p.items.size();
  }
}

template <class T>
static int upload(T **dptr, const std::vector<T> &h) {
  *dptr = nullptr;
  if (h.empty()) return PGCN_OK;
  hipError_t e = hipMalloc((void **)dptr, h.size() * sizeof(T));
  if (e != hipSuccess) {
    *dptr = nullptr;
    return set_error(PGCN_ENOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
  }
  PGCN_HIP(hipMemcpy(*dptr, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
  return PGCN_OK;
}

// A narrow plan of a matrix takes its wide plan's dense block: the block's sizes, and its
// device arrays once uploaded (borrowed: free_device frees them through the wide plan).
static void share_hub(const Plan &wide, Plan &narrow) {
  narrow.hub.rows = wide.hub.rows;
  narrow.hub.rows_real = wide.hub.rows_real;
  narrow.hub.cols = wide.hub.cols;
  narrow.hub.cols_real = wide.hub.cols_real;
  narrow.hub.nnz = wide.hub.nnz;
  narrow.hub.d_row_ids = wide.hub.d_row_ids;
  narrow.hub.d_col_ids = wide.hub.d_col_ids;
  narrow.hub.d_bits = wide.hub.d_bits;
  narrow.hub.d_init = wide.hub.d_init;
  narrow.d_col_rest = wide.d_col_rest;
}

static void free_device(pgcn_partition *p) {
  void *ptrs[] = {p->d_col, p->d_col_t, p->d_send_idx, p->d_inv_k, p->d_inv_ptr, p->d_inv_deg, p->d_sym_scale,
                  p->plan.d_items, p->plan.d_splits, p->plan_t.d_items, p->plan_t.d_splits,
                  p->plan_n.d_items, p->plan_n.d_splits, p->plan_tn.d_items, p->plan_tn.d_splits};
  for (void *q : ptrs)
    if (q) (void)hipFree(q);
  for (Plan *q : {&p->plan, &p->plan_t}) {
    void *hp[] = {q->d_col_rest, q->hub.d_row_ids, q->hub.d_col_ids, q->hub.d_bits, q->hub.d_init};
    for (void *x : hp)
      if (x) (void)hipFree(x);
  }
  for (Plan *q : {&p->plan, &p->plan_t, &p->plan_n, &p->plan_tn}) {   // the narrow plans' are borrowed
    q->d_col_rest = nullptr;
    q->hub.d_row_ids = q->hub.d_col_ids = nullptr;
    q->hub.d_bits = q->hub.d_init = nullptr;
  }
  p->d_col = p->d_col_t = p->d_send_idx = p->d_inv_k = nullptr;
  p->d_inv_ptr = nullptr;
  p->d_inv_deg = p->d_sym_scale = nullptr;
  p->d_row_scale = p->d_col_scale = nullptr;
  p->plan.d_items = p->plan_t.d_items = p->plan_n.d_items = p->plan_tn.d_items = nullptr;
  p->plan.d_splits = p->plan_t.d_splits = p->plan_n.d_splits = p->plan_tn.d_splits = nullptr;
}

// The graph must be undirected: v lists u exactly when u lists v (self loops
// and repeated entries ignored).  Compares every row with the same row of the
// transpose, both sorted and deduplicated.
static bool graph_is_symmetric(int64_t n, const int64_t *rp, const int32_t *cl) {
  std::vector<int64_t> tp(n + 1, 0);
  for (int64_t v = 0; v < n; ++v)
    for (int64_t k = rp[v]; k < rp[v + 1]; ++k)
      if (cl[k] != v) tp[cl[k] + 1]++;
  for (int64_t v = 0; v < n; ++v) tp[v + 1] += tp[v];
  std::vector<int32_t> tc(tp[n]);
  {
    std::vector<int64_t> fill(tp.begin(), tp.end() - 1);
    for (int64_t v = 0; v < n; ++v)           // rows visited in ascending v: transposed rows come out sorted
      for (int64_t k = rp[v]; k < rp[v + 1]; ++k)
        if (cl[k] != v) tc[fill[cl[k]]++] = (int32_t)v;
  }
  std::vector<int32_t> row;
  for (int64_t v = 0; v < n; ++v) {
    row.clear();
    for (int64_t k = rp[v]; k < rp[v + 1]; ++k)
      if (cl[k] != v) row.push_back(cl[k]);
    std::sort(row.begin(), row.end());
    row.erase(std::unique(row.begin(), row.end()), row.end());
    auto tb = tc.begin() + tp[v], te = tc.begin() + tp[v + 1];
    te = std::unique(tb, te);
    if ((int64_t)row.size() != (int64_t)(te - tb) || !std::equal(row.begin(), row.end(), tb)) return false;
  }
  return true;
}

static int check_device() {
  int dev = 0;
  PGCN_HIP(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  PGCN_HIP(hipGetDeviceProperties(&prop, dev));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return set_error(PGCN_EUNSUPPORTED, std::string("libpgcn is built for gfx950, device is ") + prop.gcnArchName);
  return PGCN_OK;
}

static int default_segment() {
  const char *s = std::getenv("PGCN_SEGMENT");
  if (s) {
    int v = std::atoi(s);
    if (v >= 16 && v <= (1 << 20)) return v;
  }
  return 512;
}

}  // namespace pgcn

using namespace pgcn;

extern "C" int pgcn_partition_setup(const pgcn_csr *csr, const pgcn_boundary_map *bmap, uint32_t flags,
                                    pgcn_partition **out) try {
  PGCN_REQUIRE(csr && bmap && out, "pgcn_partition_setup: null argument");
  *out = nullptr;
  const int64_t n = csr->n;
  PGCN_REQUIRE(n >= 0 && n <= INT32_MAX, "pgcn_partition_setup: n out of range");
  PGCN_REQUIRE(csr->rowptr && bmap->owner, "pgcn_partition_setup: null rowptr or owner");
  PGCN_REQUIRE(bmap->nparts >= 1 && bmap->self >= 0 && bmap->self < bmap->nparts,
               "pgcn_partition_setup: bad partition count or self");
  PGCN_REQUIRE((flags & ~(uint32_t)(PGCN_SETUP_HOST_ONLY | PGCN_SETUP_NO_SELF_LOOP | PGCN_SETUP_SYMMETRIC)) == 0,
               "pgcn_partition_setup: unknown flags");
  PGCN_REQUIRE(!((flags & PGCN_SETUP_SYMMETRIC) && (flags & PGCN_SETUP_NO_SELF_LOOP)),
               "pgcn_partition_setup: the symmetric normalisation needs the self loops");
  const int64_t *rp = csr->rowptr;
  const int32_t *cl = csr->col;
  const int32_t *owner = bmap->owner;
  const int32_t self = bmap->self, nparts = bmap->nparts;
  PGCN_REQUIRE(rp[0] == 0, "pgcn_partition_setup: rowptr[0] != 0");
  for (int64_t v = 0; v < n; ++v)
    PGCN_REQUIRE(rp[v + 1] >= rp[v], "pgcn_partition_setup: rowptr decreases");
  PGCN_REQUIRE(rp[n] == 0 || cl, "pgcn_partition_setup: null col");
  for (int64_t k = 0; k < rp[n]; ++k)
    PGCN_REQUIRE(cl[k] >= 0 && cl[k] < n, "pgcn_partition_setup: column out of range");
  for (int64_t v = 0; v < n; ++v)
    PGCN_REQUIRE(owner[v] >= 0 && owner[v] < nparts, "pgcn_partition_setup: owner out of range");
  PGCN_REQUIRE(graph_is_symmetric(n, rp, cl),
               "pgcn_partition_setup: the graph is not symmetric (some v lists u but u does not list v)");
  if (!(flags & PGCN_SETUP_HOST_ONLY)) {
    int rc = check_device();
    if (rc) return rc;
  }

  // owned here until it is handed out: every early return frees it (device arrays included)
  struct Release {
    void operator()(pgcn_partition *q) const noexcept {
      if (!q->host_only) free_device(q);
      delete q;
    }
  };
  std::unique_ptr<pgcn_partition, Release> holder(new (std::nothrow) pgcn_partition());
  pgcn_partition *p = holder.get();
  if (!p) return set_error(PGCN_ENOMEM, "pgcn_partition_setup: out of host memory");
  p->nparts = nparts;
  p->self = self;
  p->host_only = (flags & PGCN_SETUP_HOST_ONLY) ? 1 : 0;
  p->segment = default_segment();

  // V_i in ascending global id; local id = rank
  std::vector<int64_t> local_of(n, -1);
  for (int64_t v = 0; v < n; ++v)
    if (owner[v] == self) {
      local_of[v] = (int64_t)p->inner_gid.size();
      p->inner_gid.push_back(v);
    }
  const int64_t n_in = (int64_t)p->inner_gid.size();
  p->n_inner = n_in;

  // N(v) of inner rows: self loops and duplicates removed
  std::vector<int64_t> nb_ptr(n_in + 1, 0);
  std::vector<int32_t> nb;
  {
    size_t total = 0;
    for (int64_t i = 0; i < n_in; ++i) total += rp[p->inner_gid[i] + 1] - rp[p->inner_gid[i]];
    nb.reserve(total);
  }
  for (int64_t i = 0; i < n_in; ++i) {
    int64_t v = p->inner_gid[i];
    size_t start = nb.size();
    for (int64_t k = rp[v]; k < rp[v + 1]; ++k)
      if (cl[k] != v) nb.push_back(cl[k]);
    std::sort(nb.begin() + start, nb.end());
    nb.erase(std::unique(nb.begin() + start, nb.end()), nb.end());
    nb_ptr[i + 1] = (int64_t)nb.size();
  }

  // B_i ordered by (owner, global id)
  {
    std::vector<int32_t> bd;
    for (int32_t u : nb)
      if (owner[u] != self) bd.push_back(u);
    std::sort(bd.begin(), bd.end(), [&](int32_t a, int32_t b) {
      return owner[a] != owner[b] ? owner[a] < owner[b] : a < b;
    });
    bd.erase(std::unique(bd.begin(), bd.end()), bd.end());
    p->bd_gid.assign(bd.begin(), bd.end());
  }
  const int64_t n_bd = (int64_t)p->bd_gid.size();
  p->n_bd = n_bd;
  for (int64_t k = 0; k < n_bd; ++k) local_of[p->bd_gid[k]] = n_in + k;
  p->recv_ptr.assign(nparts + 1, 0);
  for (int64_t g : p->bd_gid) p->recv_ptr[owner[g] + 1]++;
  for (int32_t j = 0; j < nparts; ++j) p->recv_ptr[j + 1] += p->recv_ptr[j];

  // whole-graph degree + 1 of every local node: inner rows from N(v), boundary
  // nodes from their own rows of the global CSR (distinct neighbours, no self loop)
  p->deg.resize(n_in + n_bd);
  for (int64_t i = 0; i < n_in; ++i) p->deg[i] = nb_ptr[i + 1] - nb_ptr[i] + 1;
  {
    std::vector<int32_t> row;
    for (int64_t k = 0; k < n_bd; ++k) {
      const int64_t u = p->bd_gid[k];
      row.clear();
      for (int64_t q = rp[u]; q < rp[u + 1]; ++q)
        if (cl[q] != u) row.push_back(cl[q]);
      std::sort(row.begin(), row.end());
      p->deg[n_in + k] = (int64_t)(std::unique(row.begin(), row.end()) - row.begin()) + 1;
    }
  }

  // P_i: N(v) ∪ {v} (N(v) alone for the GraphSAGE aggregation), ascending local id
  const bool self_loop = !(flags & PGCN_SETUP_NO_SELF_LOOP);
  p->self_loop = self_loop ? 1 : 0;
  p->symmetric = (flags & PGCN_SETUP_SYMMETRIC) ? 1 : 0;
  if (p->symmetric) {                // d̃^{-1/2}, computed in double and rounded once
    p->sym_scale.resize(n_in + n_bd);
    for (int64_t k = 0; k < n_in + n_bd; ++k) p->sym_scale[k] = (float)(1.0 / std::sqrt((double)p->deg[k]));
  }
  p->rowptr.assign(n_in + 1, 0);
  p->col.reserve(nb.size() + n_in);
  for (int64_t i = 0; i < n_in; ++i) {
    size_t start = p->col.size();
    if (self_loop) p->col.push_back((int32_t)i);
    for (int64_t k = nb_ptr[i]; k < nb_ptr[i + 1]; ++k) p->col.push_back((int32_t)local_of[nb[k]]);
    std::sort(p->col.begin() + start, p->col.end());
    p->rowptr[i + 1] = (int64_t)p->col.size();
  }
  std::vector<int32_t>().swap(nb);
  p->nnz = (int64_t)p->col.size();
  p->inv_deg.resize(n_in);
  for (int64_t i = 0; i < n_in; ++i) {
    int64_t len = p->rowptr[i + 1] - p->rowptr[i];
    p->inv_deg[i] = len > 0 ? 1.0f / (float)len : 0.0f;     // a row without neighbours is zero
    p->max_row = std::max(p->max_row, len);
  }

  // P_i^T by counting sort; rows visited in ascending order keep columns ascending
  const int64_t n_all = n_in + n_bd;
  p->rowptr_t.assign(n_all + 1, 0);
  for (int32_t c : p->col) p->rowptr_t[c + 1]++;
  for (int64_t r = 0; r < n_all; ++r) p->rowptr_t[r + 1] += p->rowptr_t[r];
  p->col_t.resize(p->nnz);
  {
    std::vector<int64_t> fill(p->rowptr_t.begin(), p->rowptr_t.end() - 1);
    for (int64_t i = 0; i < n_in; ++i)
      for (int64_t k = p->rowptr[i]; k < p->rowptr[i + 1]; ++k) p->col_t[fill[p->col[k]]++] = (int32_t)i;
  }
  for (int64_t r = 0; r < n_all; ++r) p->max_row_t = std::max(p->max_row_t, p->rowptr_t[r + 1] - p->rowptr_t[r]);

  // S_{i,j} = B_j ∩ V_i: inner u adjacent to some w owned by j (w's row lists u)
  p->send_ptr.assign(nparts + 1, 0);
  {
    // (j, local u) for every edge from a node w owned by j != self to an inner u; sorted and
    // deduplicated, this is S_{i,j} for ascending j, each by ascending local (= global) id
    std::vector<std::pair<int32_t, int32_t>> su;
    for (int64_t w = 0; w < n; ++w) {
      int32_t j = owner[w];
      if (j == self) continue;
      for (int64_t k = rp[w]; k < rp[w + 1]; ++k) {
        int32_t u = cl[k];
        if (u != w && owner[u] == self) su.emplace_back(j, (int32_t)local_of[u]);
      }
    }
    std::sort(su.begin(), su.end());
    su.erase(std::unique(su.begin(), su.end()), su.end());
    p->send_idx.reserve(su.size());
    for (const auto &e : su) {
      p->send_idx.push_back(e.second);
      p->send_ptr[e.first + 1]++;
    }
    for (int32_t j = 0; j < nparts; ++j) p->send_ptr[j + 1] += p->send_ptr[j];
  }
  p->n_send = (int64_t)p->send_idx.size();

  // inverse send map: positions k per inner row, ascending k
  p->inv_ptr.assign(n_in + 1, 0);
  for (int32_t u : p->send_idx) p->inv_ptr[u + 1]++;
  for (int64_t u = 0; u < n_in; ++u) p->inv_ptr[u + 1] += p->inv_ptr[u];
  p->inv_k.resize(p->n_send);
  {
    std::vector<int64_t> fill(p->inv_ptr.begin(), p->inv_ptr.end() - 1);
    for (int64_t k = 0; k < p->n_send; ++k) p->inv_k[fill[p->send_idx[k]]++] = (int32_t)k;
  }

  {
    const int64_t nnz = p->nnz, wide = 8000, narrow = 32000;
    const int32_t c = choose_chunks(n_in, n_all, nnz, false, wide), ct = choose_chunks(n_all, n_in, nnz, true, wide);
    const int32_t cn = choose_chunks(n_in, n_all, nnz, false, narrow, true);
    const int32_t ctn = choose_chunks(n_all, n_in, nnz, true, narrow, true);
    // a matrix may have a dense block on the matrix cores; every plan of it then indexes the
    // rest, and the narrow plans use the wide plan's block (the same matrix, the same block)
    std::vector<int64_t> rp_rest, rpt_rest;
    choose_hub(p->rowptr, p->col, n_in, n_all, p->plan.hub, rp_rest, p->plan.col_rest);
    choose_hub(p->rowptr_t, p->col_t, n_all, n_in, p->plan_t.hub, rpt_rest, p->plan_t.col_rest);
    const bool hub = p->plan.hub.rows > 0, hub_t = p->plan_t.hub.rows > 0;
    build_plan(hub ? rp_rest : p->rowptr, hub ? p->plan.col_rest : p->col, n_in, n_all, p->segment, c, p->plan);
    build_plan(hub_t ? rpt_rest : p->rowptr_t, hub_t ? p->plan_t.col_rest : p->col_t, n_all, n_in, p->segment, ct,
               p->plan_t);
    p->plan_n.chunks = p->plan_tn.chunks = 0;
    if (cn != c) {
      build_plan(hub ? rp_rest : p->rowptr, hub ? p->plan.col_rest : p->col, n_in, n_all, p->segment, cn, p->plan_n);
      share_hub(p->plan, p->plan_n);
    }
    if (ctn != ct) {
      build_plan(hub_t ? rpt_rest : p->rowptr_t, hub_t ? p->plan_t.col_rest : p->col_t, n_all, n_in, p->segment, ctn,
                 p->plan_tn);
      share_hub(p->plan_t, p->plan_tn);
    }
  }

  if (!p->host_only) {
    PGCN_HIP(hipGetDevice(&p->device));
    int rc = noalloc_scratch_init(p->device);
    if (!rc) rc = upload(&p->d_col, p->col);
    if (!rc) rc = upload(&p->d_col_t, p->col_t);
    if (!rc) rc = upload(&p->d_send_idx, p->send_idx);
    if (!rc) rc = upload(&p->d_inv_k, p->inv_k);
    if (!rc) rc = upload(&p->d_inv_ptr, p->inv_ptr);
    if (!rc) rc = upload(&p->d_inv_deg, p->inv_deg);
    if (!rc && p->symmetric) rc = upload(&p->d_sym_scale, p->sym_scale);
    if (!rc) rc = upload(&p->plan.d_items, p->plan.items);
    if (!rc) rc = upload(&p->plan.d_splits, p->plan.splits);
    if (!rc) rc = upload(&p->plan_t.d_items, p->plan_t.items);
    if (!rc) rc = upload(&p->plan_t.d_splits, p->plan_t.splits);
    if (!rc) rc = upload(&p->plan_n.d_items, p->plan_n.items);
    if (!rc) rc = upload(&p->plan_n.d_splits, p->plan_n.splits);
    if (!rc) rc = upload(&p->plan_tn.d_items, p->plan_tn.items);
    if (!rc) rc = upload(&p->plan_tn.d_splits, p->plan_tn.splits);
    for (Plan *q : {&p->plan, &p->plan_t}) {
      if (!rc) rc = upload(&q->d_col_rest, q->col_rest);
      if (!rc) rc = upload(&q->hub.d_row_ids, q->hub.row_ids);
      if (!rc) rc = upload(&q->hub.d_col_ids, q->hub.col_ids);
      if (!rc) rc = upload(&q->hub.d_bits, q->hub.bits);
      if (!rc) rc = upload(&q->hub.d_init, q->hub.init);
    }
    if (rc) return rc;
    if (p->plan_n.chunks > 0) share_hub(p->plan, p->plan_n);
    if (p->plan_tn.chunks > 0) share_hub(p->plan_t, p->plan_tn);
    p->d_row_scale = p->symmetric ? p->d_sym_scale : p->d_inv_deg;
    p->d_col_scale = p->symmetric ? p->d_sym_scale : nullptr;
  }
  *out = holder.release();
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_partition_setup");
}

extern "C" int pgcn_partition_info(const pgcn_partition *p, pgcn_info *o) try {
  PGCN_REQUIRE(p && o, "pgcn_partition_info: null argument");
  o->n_inner = p->n_inner;
  o->n_bd = p->n_bd;
  o->nnz = p->nnz;
  o->n_send = p->n_send;
  o->max_row_len = p->max_row;
  o->max_row_len_t = p->max_row_t;
  o->nparts = p->nparts;
  o->self = p->self;
  o->host_only = p->host_only;
  o->spmm_segment = p->segment;
  o->spmm_items = (int64_t)p->plan.items.size();
  o->spmm_split_slots = p->plan.slots;
  o->spmmt_items = (int64_t)p->plan_t.items.size();
  o->spmmt_split_slots = p->plan_t.slots;
  o->spmm_chunks = p->plan.chunks;
  o->spmmt_chunks = p->plan_t.chunks;
  o->spmm_chunks_narrow = p->plan_n.chunks ? p->plan_n.chunks : p->plan.chunks;
  o->spmmt_chunks_narrow = p->plan_tn.chunks ? p->plan_tn.chunks : p->plan_t.chunks;
  o->spmm_hub_rows = p->plan.hub.rows_real;
  o->spmm_hub_cols = p->plan.hub.cols_real;
  o->spmm_hub_nnz = p->plan.hub.nnz;
  o->spmmt_hub_rows = p->plan_t.hub.rows_real;
  o->spmmt_hub_cols = p->plan_t.hub.cols_real;
  o->spmmt_hub_nnz = p->plan_t.hub.nnz;
  o->symmetric = p->symmetric;
  o->self_loop = p->self_loop;
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_partition_info");
}

template <class T>
static void copy_out(T *dst, const std::vector<T> &src) {
  if (dst && !src.empty()) std::memcpy(dst, src.data(), src.size() * sizeof(T));
}

extern "C" int pgcn_partition_export(const pgcn_partition *p, const pgcn_arrays *h) try {
  PGCN_REQUIRE(p && h, "pgcn_partition_export: null argument");
  copy_out(h->inner_gid, p->inner_gid);
  copy_out(h->bd_gid, p->bd_gid);
  copy_out(h->recv_ptr, p->recv_ptr);
  copy_out(h->rowptr, p->rowptr);
  copy_out(h->col, p->col);
  copy_out(h->rowptr_t, p->rowptr_t);
  copy_out(h->col_t, p->col_t);
  copy_out(h->send_ptr, p->send_ptr);
  copy_out(h->send_idx, p->send_idx);
  copy_out(h->inv_ptr, p->inv_ptr);
  copy_out(h->inv_k, p->inv_k);
  copy_out(h->deg, p->deg);
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_partition_export");
}

extern "C" void pgcn_partition_destroy(pgcn_partition *p) try {
  if (!p) return;
  if (!p->host_only) free_device(p);
  delete p;
} catch (...) {
  (void)exception_status("pgcn_partition_destroy");
}

extern "C" const char *pgcn_last_error(void) { return g_error_static ? g_error_static : g_error.c_str(); }

extern "C" int pgcn_version(void) { return PGCN_VERSION; }

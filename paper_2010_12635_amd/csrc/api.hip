// C ABI of libgcn: argument validation on the host, then the kernel
// sequence of each call on the caller's stream.  Nothing here allocates
// device memory; scratch comes from the caller's workspace.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <mutex>

#include "gcn.h"
#include "internal.h"

using namespace gcn;

namespace {

constexpr int64_t DEFAULT_HEAVY = 128;
constexpr int64_t DEFAULT_CHUNK = 256;
// One column range by default: on R-MAT scale 21, 16 ranges cut the L2-miss
// traffic of the aggregation by 28 % but made it slower (more, shorter
// pieces and their partial rows), so the die-mapped launch is opt-in.
constexpr int64_t DEFAULT_PARTS = 1;

int64_t parts_or_default(int64_t, int64_t parts) { return parts > 0 ? parts : DEFAULT_PARTS; }
bool valid_parts(int64_t parts) { return parts == 1 || parts == 8 || parts == 16 || parts == 32 || parts == 64; }

bool valid_prec(int32_t p) { return p == GCN_F32 || p == GCN_F16 || p == GCN_BF16; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t elem_bytes(int32_t prec) { return prec == GCN_F32 ? 4 : 2; }
bool debug_sync() {
  const char* e = std::getenv("GCN_DEBUG_SYNC");
  return e && e[0] && e[0] != '0';
}

gcn_status finish(hipError_t e, hipStream_t s) {
  if (e != hipSuccess) return GCN_ERR_DEVICE;
  if (debug_sync()) {
    if (hipStreamSynchronize(s) != hipSuccess) return GCN_ERR_DEVICE;
    if (hipGetLastError() != hipSuccess) return GCN_ERR_DEVICE;
  }
  return GCN_OK;
}

#define GCN_HIP(x) do { hipError_t _e = (x); if (_e != hipSuccess) return finish(_e, s); } while (0)

gcn_status check_layer(const gcn_layer* L) {
  if (!L) return GCN_ERR_INVALID_ARG;
  if (L->f_in <= 0 || L->f_out <= 0) return GCN_ERR_SHAPE;
  if (L->ld_in < L->f_in || L->ld_out < L->f_out) return GCN_ERR_SHAPE;
  if (L->ld_in % 8 || L->ld_out % 8) return GCN_ERR_ALIGNMENT;
  if (L->act != GCN_ACT_NONE && L->act != GCN_ACT_RELU) return GCN_ERR_INVALID_ARG;
  if (!(L->dropout_p >= 0.f && L->dropout_p < 1.f)) return GCN_ERR_INVALID_ARG;
  return GCN_OK;
}

gcn_status check_adj(const gcn_adj* A, int32_t prec) {
  if (!A) return GCN_ERR_INVALID_ARG;
  if (A->n <= 0) return GCN_ERR_SHAPE;
  if (A->format == GCN_DENSE || A->format == GCN_DENSE_TILED) {
    if (!A->dense) return GCN_ERR_INVALID_ARG;
    if (A->value_prec != prec) return GCN_ERR_UNSUPPORTED;
    if (!aligned16(A->dense)) return GCN_ERR_ALIGNMENT;
    if (A->format == GCN_DENSE_TILED) return GCN_OK;
    if (A->ld_dense < A->n) return GCN_ERR_SHAPE;
    if (A->ld_dense % 8) return GCN_ERR_ALIGNMENT;
    return GCN_OK;
  }
  if (A->format != GCN_CSR) return GCN_ERR_INVALID_ARG;
  if (A->index != GCN_I32 && A->index != GCN_I64) return GCN_ERR_INVALID_ARG;
  if (A->nnz < 0) return GCN_ERR_SHAPE;
  if (!A->rowptr || (A->nnz > 0 && !A->colidx)) return GCN_ERR_INVALID_ARG;
  if (A->values) {
    if (A->value_prec != prec) return GCN_ERR_UNSUPPORTED;
  } else if (!A->dinv) {
    return GCN_ERR_INVALID_ARG;
  }
  if (A->n_heavy > 0) {
    if (!A->heavy_rows || !A->heavy_chunk_off || !A->chunk_heavy || !A->chunk_beg) return GCN_ERR_INVALID_ARG;
    if (A->chunk_nnz <= 0 || A->heavy_threshold <= 0 || A->n_chunks <= 0) return GCN_ERR_INVALID_ARG;
    if (!valid_parts(A->col_parts)) return GCN_ERR_INVALID_ARG;
    if (A->col_parts > 1 && (!A->part_off || A->part_slots <= 0)) return GCN_ERR_INVALID_ARG;
    if (!A->chunk_order || !A->piece_desc || !A->piece_pos) return GCN_ERR_INVALID_ARG;
    if (A->n_fix < 0 || A->n_fix > A->n_heavy || A->n_fix_big < 0 || A->n_fix_big > A->n_fix) return GCN_ERR_SHAPE;
    if (A->n_chunks > A->n_heavy && A->n_fix == 0) return GCN_ERR_INVALID_ARG;  // rows of several pieces unlisted
    if (A->n_fix > 0 && !A->fix_rows) return GCN_ERR_INVALID_ARG;
  }
  if (A->row_perm && !A->row_desc) return GCN_ERR_INVALID_ARG;
  if (A->n_heavy > 0 && !A->row_perm) return GCN_ERR_INVALID_ARG;   // the light rows must be listed
  if (A->row_perm && (A->n_light < 0 || A->n_light > A->n)) return GCN_ERR_SHAPE;
  if (A->row_perm && (A->n_light_single < 0 || A->n_light_single > A->n_light)) return GCN_ERR_SHAPE;
  return GCN_OK;
}

CsrView view_of(const gcn_adj* A) {
  CsrView v;
  v.n = A->n; v.nnz = A->nnz; v.idx64 = A->index == GCN_I64;
  v.rowptr = A->rowptr; v.colidx = A->colidx; v.values = A->values; v.dinv = A->dinv;
  v.heavy_threshold = A->heavy_threshold; v.chunk_nnz = A->chunk_nnz;
  v.n_heavy = A->n_heavy > 0 ? A->n_heavy : 0; v.n_chunks = A->n_chunks;
  v.heavy_rows = A->heavy_rows; v.heavy_chunk_off = A->heavy_chunk_off; v.chunk_heavy = A->chunk_heavy;
  v.n_light = A->row_perm ? A->n_light : 0;
  v.row_perm = A->row_perm;
  v.chunk_order = A->n_heavy > 0 ? A->chunk_order : nullptr;
  v.chunk_beg = A->n_heavy > 0 ? A->chunk_beg : nullptr;
  v.part_off = A->n_heavy > 0 ? A->part_off : nullptr;
  v.parts = A->n_heavy > 0 ? A->col_parts : 1;
  v.part_slots = A->n_heavy > 0 ? A->part_slots : 0;
  v.piece_desc = A->n_heavy > 0 ? static_cast<const RowDesc*>(A->piece_desc) : nullptr;
  v.piece_pos = A->n_heavy > 0 ? A->piece_pos : nullptr;
  v.row_desc = A->row_perm ? static_cast<const RowDesc*>(A->row_desc) : nullptr;
  v.n_light_single = A->row_perm ? A->n_light_single : 0;
  v.n_fix = A->n_heavy > 0 ? A->n_fix : 0;
  v.n_fix_big = A->n_heavy > 0 ? A->n_fix_big : 0;
  v.fix_rows = A->n_heavy > 0 ? A->fix_rows : nullptr;
  return v;
}

// Workspace of a layer call: the column-sum partials of dZ (kept from the
// aggregation step to the final reduction) at the front, then the scratch
// of one step at a time.
struct LayerPlan {
  int s_split;       // S = H W
  int agg_split;     // dense aggregation
  int dw_split;      // dW = H^T G_S
  int dh_split;      // dZ_below = G_S W^T
  int64_t cs_floats; // column-sum partial region (multiple of 64 floats)
  int64_t cb_floats; // column-sum partials of dZ_below (multiple of 64 floats)
  int64_t floats;    // total
};

LayerPlan plan_layer(const gcn_adj* A, const gcn_layer* L, int32_t prec) {
  LayerPlan p;
  const int64_t n = A->n;
  const bool ident = L->identity_input != 0;    // no product with H = I
  p.s_split = ident ? 1 : gemm_choose_splits(prec, n, L->f_out, L->f_in);
  p.dh_split = ident ? 1 : gemm_choose_splits(prec, n, L->f_in, L->f_out);
  p.dw_split = ident ? 0 : wgrad_splits(prec, n, L->f_in, L->f_out);
  p.agg_split = 1;
  int64_t f = 0;
  auto upd = [&](int64_t x) { if (x > f) f = x; };
  if (p.s_split > 1) upd(p.s_split * n * L->f_out);
  if (p.dh_split > 1) upd(p.dh_split * n * L->f_in);
  upd((int64_t)p.dw_split * L->f_in * L->f_out);
  int64_t cs = 0;
  if (A->format != GCN_CSR) {
    upd((int64_t)(dense_agg_workspace_bytes(prec, n, L->f_out, A->format == GCN_DENSE_TILED) / sizeof(float)) + 1);
    cs = dense_agg_colsum_rows(prec, n) * L->f_out;
  } else {
    upd(spmm_partials_floats(view_of(A), prec, L->f_out));
    cs = colsum_partials_floats(n, L->ld_out);
  }
  p.cs_floats = (cs + 63) / 64 * 64;
  // column sums of dZ_below: one row per product workgroup, or the
  // column-sum pass over dZ_below where the generic GEMM computes it
  const int64_t cb = std::max<int64_t>((int64_t)tsgemm_colsum_rows_max() * L->f_in, colsum_partials_floats(n, L->ld_in));
  p.cb_floats = ident ? 0 : (cb + 63) / 64 * 64;
  p.floats = p.cs_floats + p.cb_floats + f;
  return p;
}

size_t plan_bytes(const LayerPlan& p) { return (size_t)p.floats * sizeof(float) + 256; }

Epilogue base_epi(void* out, int64_t ldo, int64_t rows, int64_t cols, int mode, int32_t* flag) {
  Epilogue e{};
  e.out = out; e.ldo = ldo; e.rows = rows; e.cols = cols; e.mode = mode; e.flag = flag;
  e.keep_scale = 1.f;
  return e;
}

hipError_t run_gemm(int32_t prec, bool akc, bool bkc, const void* A, int64_t lda, const void* B, int64_t ldb,
                    int64_t M, int64_t N, int64_t K, int splits, bool force_partials, float* ws,
                    const Epilogue& epi, hipStream_t s) {
  GemmCall c;
  c.prec = prec; c.a_kc = akc; c.b_kc = bkc; c.A = A; c.lda = lda; c.B = B; c.ldb = ldb;
  c.M = M; c.N = N; c.K = K; c.splits = splits;
  const bool use_partials = splits > 1 || force_partials;
  c.partials = use_partials ? ws : nullptr;
  c.epi = epi;
  hipError_t e = gemm_launch(c, s);
  if (e != hipSuccess || !use_partials) return e;
  return reduce_partials(prec, ws, splits, M, N, epi, s);
}

// Row-streaming product C = A B for the n-row operands of the layer
// (S = H W, dZ_below = G_S W^T); the generic tiled GEMM covers the rest.
bool use_tsgemm(int32_t prec, int64_t M, int64_t K) { return M >= 1024 && tsgemm_supported(prec, K); }

hipError_t row_product(int32_t prec, const void* A, int64_t lda, const void* B, int64_t ldb, bool b_kc, int64_t M,
                       int64_t N, int64_t K, int splits, float* ws, const Epilogue& epi, hipStream_t s) {
  if (use_tsgemm(prec, M, K)) return tsgemm_launch(prec, A, lda, B, ldb, b_kc, M, N, K, epi, s);
  return run_gemm(prec, true, b_kc, A, lda, B, ldb, M, N, K, splits, false, ws, epi, s);
}

// Y = epilogue(A_hat X).  For dense A_hat, colsum (may be NULL) receives the
// column-sum partials of X computed during its transposition.
hipError_t aggregate(const gcn_adj* A, int32_t prec, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                     float* ws, float* colsum, hipStream_t s) {
  if (A->format != GCN_CSR)
    return dense_agg_launch(prec, A->dense, A->ld_dense, A->format == GCN_DENSE_TILED, A->n, X, ldx, F, epi, ws,
                            colsum, s);
  return spmm_launch(view_of(A), prec, X, ldx, F, epi, ws, s);
}

size_t aggregate_bytes(const gcn_adj* A, int32_t prec, int64_t F) {
  int64_t f = 0;
  if (A->format != GCN_CSR) {
    f = (int64_t)(dense_agg_workspace_bytes(prec, A->n, F, A->format == GCN_DENSE_TILED) / sizeof(float)) + 1;
  } else {
    f = spmm_partials_floats(view_of(A), prec, F);
  }
  return (size_t)f * sizeof(float) + 256;
}

Epilogue agg_epi(void* Y, int64_t ldy, int64_t n, int64_t F, const float* bias, int32_t act, float p,
                 int32_t training, uint64_t seed, int32_t layer_id, uint64_t epoch, int32_t* overflow,
                 const gcn_scaler* epoch_from = nullptr) {
  Epilogue ea = base_epi(Y, ldy, n, F, EPI_AGG, overflow);
  ea.bias = bias;
  ea.relu = act == GCN_ACT_RELU;
  ea.dropout = ea.relu && training && p > 0.f;
  if (ea.dropout) {
    const double t = std::floor((double)p * 4294967296.0);
    ea.thr = (uint32_t)(t > 4294967295.0 ? 4294967295.0 : t);
    ea.keep_scale = 1.f / (1.f - p);
  }
  ea.seed = seed;
  ea.layer = (uint64_t)(uint32_t)layer_id;
  ea.epoch = epoch;
  ea.epoch_ctr = epoch_from ? &epoch_from->step : nullptr;   // step and skipped are adjacent int32
  return ea;
}

}  // namespace

extern "C" {

const char* gcn_status_string(int32_t status) {
  switch (status) {
    case GCN_OK: return "GCN_OK";
    case GCN_ERR_INVALID_ARG: return "GCN_ERR_INVALID_ARG: missing pointer or invalid enum/scalar argument";
    case GCN_ERR_SHAPE: return "GCN_ERR_SHAPE: non-positive or inconsistent sizes";
    case GCN_ERR_ALIGNMENT: return "GCN_ERR_ALIGNMENT: leading dimension not a multiple of 8 or pointer not 16-byte aligned";
    case GCN_ERR_UNSUPPORTED: return "GCN_ERR_UNSUPPORTED: combination not implemented";
    case GCN_ERR_CAPACITY: return "GCN_ERR_CAPACITY: output buffer too small";
    case GCN_ERR_WORKSPACE: return "GCN_ERR_WORKSPACE: workspace missing or too small";
    case GCN_ERR_DEVICE: return "GCN_ERR_DEVICE: HIP runtime or kernel launch failure";
    case GCN_ERR_GRAPH: return "GCN_ERR_GRAPH: vertex id outside [0, n)";
  }
  return "unknown gcn_status";
}

int32_t gcn_abi_version(void) { return GCN_ABI_VERSION; }

gcn_status gcn_normalize_workspace_size(int64_t n, int64_t num_edges, size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || num_edges < 0) return GCN_ERR_SHAPE;
  *bytes = normalize_workspace_bytes(n, num_edges);
  return GCN_OK;
}

gcn_status gcn_normalize(int64_t n, int64_t num_edges, const int32_t* src, const int32_t* dst, int32_t index,
                         void* rowptr, int32_t* colidx, int64_t nnz_capacity, int32_t* deg, float* dinv,
                         int32_t value_prec, void* values, void* dense, int64_t ld_dense, int64_t* nnz_out,
                         void* workspace, size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n <= 0 || num_edges < 0) return GCN_ERR_SHAPE;
  if (n > INT32_MAX) return GCN_ERR_UNSUPPORTED;
  if (num_edges > 0 && (!src || !dst)) return GCN_ERR_INVALID_ARG;
  if (!rowptr || !colidx || !dinv || !nnz_out) return GCN_ERR_INVALID_ARG;
  if (index != GCN_I32 && index != GCN_I64) return GCN_ERR_INVALID_ARG;
  if ((values || dense) && !valid_prec(value_prec)) return GCN_ERR_INVALID_ARG;
  const int64_t max_nnz = 2 * num_edges + n;
  if (nnz_capacity < max_nnz) return GCN_ERR_CAPACITY;
  if (index == GCN_I32 && max_nnz >= INT32_MAX) return GCN_ERR_UNSUPPORTED;
  if (dense) {
    if (ld_dense < n) return GCN_ERR_SHAPE;
    if (ld_dense % 8 || !aligned16(dense)) return GCN_ERR_ALIGNMENT;
  }
  if (!workspace || workspace_bytes < normalize_workspace_bytes(n, num_edges)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  int64_t nnz = 0;
  int32_t bad = 0;
  hipError_t e = normalize_run(n, num_edges, src, dst, index == GCN_I64, rowptr, colidx, deg, dinv, value_prec,
                               values, dense, ld_dense, &nnz, &bad, workspace, workspace_bytes, s);
  if (e != hipSuccess) return GCN_ERR_DEVICE;
  if (bad) return GCN_ERR_GRAPH;
  *nnz_out = nnz;
  return finish(hipSuccess, s);
}

gcn_status gcn_dense_tiled_elems(int64_t n, int32_t prec, int64_t* elems) {
  if (!elems || !valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0) return GCN_ERR_SHAPE;
  *elems = dense_tiled_elems(prec, n);
  return GCN_OK;
}

gcn_status gcn_densify(const gcn_adj* A, int32_t format, int32_t value_prec, void* dense, int64_t ld_dense,
                       void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!A || !dense || !valid_prec(value_prec)) return GCN_ERR_INVALID_ARG;
  if (A->format != GCN_CSR || (format != GCN_DENSE && format != GCN_DENSE_TILED)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, value_prec);
  if (st != GCN_OK) return st;
  if (!aligned16(dense)) return GCN_ERR_ALIGNMENT;
  if (format == GCN_DENSE) {
    if (ld_dense < A->n) return GCN_ERR_SHAPE;
    if (ld_dense % 8) return GCN_ERR_ALIGNMENT;
  }
  GCN_HIP(densify_launch(view_of(A), value_prec, format == GCN_DENSE_TILED, dense, ld_dense, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_schedule_size(int64_t n, int64_t nnz, int64_t heavy_threshold, int64_t chunk_nnz, int64_t col_parts,
                             size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || nnz < 0) return GCN_ERR_SHAPE;
  if (heavy_threshold <= 0) heavy_threshold = DEFAULT_HEAVY;
  if (chunk_nnz <= 0) chunk_nnz = DEFAULT_CHUNK;
  col_parts = parts_or_default(n, col_parts);
  if (!valid_parts(col_parts)) return GCN_ERR_INVALID_ARG;
  *bytes = schedule_bytes(n, nnz, heavy_threshold, chunk_nnz, col_parts);
  return GCN_OK;
}

gcn_status gcn_schedule(gcn_adj* A, int64_t heavy_threshold, int64_t chunk_nnz, int64_t col_parts, void* sched,
                        size_t sched_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!A || !sched) return GCN_ERR_INVALID_ARG;
  if (A->format != GCN_CSR || !A->rowptr || (A->nnz > 0 && !A->colidx)) return GCN_ERR_INVALID_ARG;
  if (A->index != GCN_I32 && A->index != GCN_I64) return GCN_ERR_INVALID_ARG;
  if (A->n <= 0 || A->nnz < 0) return GCN_ERR_SHAPE;
  if (heavy_threshold <= 0) heavy_threshold = DEFAULT_HEAVY;
  if (chunk_nnz <= 0) chunk_nnz = DEFAULT_CHUNK;
  col_parts = parts_or_default(A->n, col_parts);
  if (!valid_parts(col_parts)) return GCN_ERR_INVALID_ARG;
  if (sched_bytes < schedule_bytes(A->n, A->nnz, heavy_threshold, chunk_nnz, col_parts)) return GCN_ERR_WORKSPACE;
  if (!aligned16(sched)) return GCN_ERR_ALIGNMENT;
  SchedOut o{};
  hipError_t e = schedule_run(A->n, A->nnz, A->index == GCN_I64, A->rowptr, A->colidx, heavy_threshold, chunk_nnz,
                              col_parts, sched, sched_bytes, &o, s);
  if (e != hipSuccess) return GCN_ERR_DEVICE;
  A->heavy_threshold = heavy_threshold;
  A->chunk_nnz = chunk_nnz;
  A->n_heavy = o.n_heavy;
  A->n_chunks = o.n_chunks;
  A->heavy_rows = o.heavy_rows;
  A->heavy_chunk_off = o.heavy_chunk_off;
  A->chunk_heavy = o.chunk_heavy;
  A->row_perm = o.row_perm;
  A->n_light = o.n_light;
  A->chunk_order = o.chunk_order;
  A->chunk_beg = o.chunk_beg;
  A->part_off = o.part_off;
  A->col_parts = col_parts;
  A->part_slots = o.part_slots;
  A->piece_desc = o.piece_desc;
  A->piece_pos = o.piece_pos;
  A->row_desc = o.row_desc;
  A->n_light_single = o.n_light_single;
  A->n_fix = o.n_fix;
  A->n_fix_big = o.n_fix_big;
  A->fix_rows = o.fix_rows;
  return finish(hipSuccess, s);
}

gcn_status gcn_layer_workspace_size(const gcn_adj* A, const gcn_layer* L, int32_t prec, size_t* bytes) {
  if (!bytes || !valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, prec);
  if (st != GCN_OK) return st;
  st = check_layer(L);
  if (st != GCN_OK) return st;
  *bytes = plan_bytes(plan_layer(A, L, prec));
  return GCN_OK;
}

gcn_status gcn_layer_fwd(const gcn_adj* A, const gcn_layer* L, int32_t prec, int32_t training, const void* H,
                         const void* W, const float* bias, uint64_t seed, uint64_t epoch, void* S, void* H_out,
                         int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, prec);
  if (st != GCN_OK) return st;
  st = check_layer(L);
  if (st != GCN_OK) return st;
  const bool ident = L->identity_input != 0;
  if (ident && L->f_in != A->n) return GCN_ERR_SHAPE;
  if ((!ident && (!H || !S)) || !W || !H_out) return GCN_ERR_INVALID_ARG;
  if ((H && !aligned16(H)) || !aligned16(W) || (S && !aligned16(S)) || !aligned16(H_out)) return GCN_ERR_ALIGNMENT;
  const LayerPlan plan = plan_layer(A, L, prec);
  if (!workspace || workspace_bytes < plan_bytes(plan)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  float* ws = static_cast<float*>(workspace);
  const int64_t n = A->n;

  // S = H W; with H = I, S is W itself (n x f_out, ld_out)
  const void* Sx = W;
  if (!ident) {
    Epilogue es = base_epi(S, L->ld_out, n, L->f_out, EPI_STORE, overflow);
    GCN_HIP(row_product(prec, H, L->ld_in, W, L->ld_out, false, n, L->f_out, L->f_in, plan.s_split, ws, es, s));
    Sx = S;
  }

  Epilogue ea = agg_epi(H_out, L->ld_out, n, L->f_out, bias, L->act, L->dropout_p, training, seed, L->layer_id,
                        epoch, overflow, L->epoch_from);
  GCN_HIP(aggregate(A, prec, Sx, L->ld_out, L->f_out, ea, ws, nullptr, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_transform_workspace_size(int64_t n, int64_t f_in, int64_t f_out, int32_t prec, size_t* bytes) {
  if (!bytes || !valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || f_in <= 0 || f_out <= 0) return GCN_ERR_SHAPE;
  const int sp = gemm_choose_splits(prec, n, f_out, f_in);
  *bytes = (size_t)(sp > 1 ? sp * n * f_out : 0) * sizeof(float) + 256;
  return GCN_OK;
}

gcn_status gcn_transform(int64_t n, int64_t f_in, int64_t f_out, int32_t prec, const void* H, int64_t ld_in,
                         const void* W, int64_t ld_w, void* S, int64_t ld_s, int32_t* overflow, void* workspace,
                         size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || f_in <= 0 || f_out <= 0 || ld_in < f_in || ld_w < f_out || ld_s < f_out) return GCN_ERR_SHAPE;
  if (ld_in % 8 || ld_w % 8 || ld_s % 8) return GCN_ERR_ALIGNMENT;
  if (!H || !W || !S) return GCN_ERR_INVALID_ARG;
  if (!aligned16(H) || !aligned16(W) || !aligned16(S)) return GCN_ERR_ALIGNMENT;
  const int sp = gemm_choose_splits(prec, n, f_out, f_in);
  const size_t need = (size_t)(sp > 1 ? sp * n * f_out : 0) * sizeof(float) + 256;
  if (sp > 1 && (!workspace || workspace_bytes < need)) return GCN_ERR_WORKSPACE;
  if (workspace && !aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  Epilogue es = base_epi(S, ld_s, n, f_out, EPI_STORE, overflow);
  GCN_HIP(row_product(prec, H, ld_in, W, ld_w, false, n, f_out, f_in, sp, static_cast<float*>(workspace), es, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_aggregate_workspace_size(const gcn_adj* A, int64_t F, int32_t prec, size_t* bytes) {
  if (!bytes || !valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, prec);
  if (st != GCN_OK) return st;
  if (F <= 0) return GCN_ERR_SHAPE;
  *bytes = aggregate_bytes(A, prec, F);
  return GCN_OK;
}

gcn_status gcn_aggregate(const gcn_adj* A, int64_t F, int32_t prec, const void* X, int64_t ldx, const float* bias,
                         int32_t act, float dropout_p, int32_t training, uint64_t seed, int32_t layer_id,
                         uint64_t epoch, void* Y, int64_t ldy, int32_t* overflow, void* workspace,
                         size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, prec);
  if (st != GCN_OK) return st;
  if (F <= 0 || ldx < F || ldy < F) return GCN_ERR_SHAPE;
  if (ldx % 8 || ldy % 8) return GCN_ERR_ALIGNMENT;
  if (act != GCN_ACT_NONE && act != GCN_ACT_RELU) return GCN_ERR_INVALID_ARG;
  if (!(dropout_p >= 0.f && dropout_p < 1.f)) return GCN_ERR_INVALID_ARG;
  if (!X || !Y) return GCN_ERR_INVALID_ARG;
  if (!aligned16(X) || !aligned16(Y)) return GCN_ERR_ALIGNMENT;
  if (workspace_bytes < aggregate_bytes(A, prec, F) || (!workspace && aggregate_bytes(A, prec, F) > 256))
    return GCN_ERR_WORKSPACE;
  if (workspace && !aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  Epilogue ea = agg_epi(Y, ldy, A->n, F, bias, act, dropout_p, training, seed, layer_id, epoch, overflow);
  GCN_HIP(aggregate(A, prec, X, ldx, F, ea, static_cast<float*>(workspace), nullptr, s));
  return finish(hipSuccess, s);
}

namespace {

// Argument checks of gcn_layer_bwd that do not concern the workspace.
gcn_status layer_bwd_check(const gcn_adj* A, const gcn_layer* L, int32_t prec, const void* H, const void* W,
                           const void* dZ, int32_t act_below, float p_below, const float* dW, const float* dbias,
                           const void* dZ_below, const float* dbias_below, const void* GS) {
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  gcn_status st = check_adj(A, prec);
  if (st != GCN_OK) return st;
  st = check_layer(L);
  if (st != GCN_OK) return st;
  const bool ident = L->identity_input != 0;
  if (ident && L->f_in != A->n) return GCN_ERR_SHAPE;
  if (ident && dZ_below) return GCN_ERR_INVALID_ARG;
  if (dbias_below && !dZ_below) return GCN_ERR_INVALID_ARG;
  if ((!ident && !H) || !W || !dZ || !dW || !GS) return GCN_ERR_INVALID_ARG;
  if (act_below != GCN_ACT_NONE && act_below != GCN_ACT_RELU) return GCN_ERR_INVALID_ARG;
  if (!(p_below >= 0.f && p_below < 1.f)) return GCN_ERR_INVALID_ARG;
  if ((H && !aligned16(H)) || !aligned16(W) || !aligned16(dZ) || !aligned16(dW) || !aligned16(GS) ||
      (dZ_below && !aligned16(dZ_below)) || (dbias && !aligned16(dbias)) || (dbias_below && !aligned16(dbias_below)))
    return GCN_ERR_ALIGNMENT;
  return GCN_OK;
}

// The kernel sequence of gcn_layer_bwd on checked arguments; `workspace`
// holds at least plan_bytes(plan) bytes, 16-byte aligned.  Every scratch
// word is written before it is read (column-sum, wgrad and chunk partials
// are stored whole by their producers), so the workspace need not be
// cleared between calls.
gcn_status layer_bwd_run(const gcn_adj* A, const gcn_layer* L, int32_t prec, const LayerPlan& plan,
                         const void* H, const void* W, const void* dZ, int32_t act_below, float p_below, float* dW,
                         float* dbias, void* dZ_below, float* dbias_below, void* GS, int32_t* overflow,
                         float* workspace, hipStream_t s) {
  const bool ident = L->identity_input != 0;
  float* cs = workspace;                           // column-sum partials of dZ
  float* cb = cs + plan.cs_floats;                 // column-sum partials of dZ_below
  float* ws = cb + plan.cb_floats;                 // per-step scratch
  const int64_t n = A->n;
  const bool dense = A->format != GCN_CSR;

  // G_S = A_hat^T dZ = A_hat dZ (A_hat symmetric); for dense A_hat the
  // transposition of dZ also yields the column-sum partials for dbias
  Epilogue eg = base_epi(GS, L->ld_out, n, L->f_out, EPI_STORE, overflow);
  GCN_HIP(aggregate(A, prec, dZ, L->ld_out, L->f_out, eg, ws, dbias && dense ? cs : nullptr, s));
  RedJob jb{};
  if (dbias) {
    Epilogue eb = base_epi(dbias, L->ld_out, 1, L->f_out, EPI_F32, overflow);
    if (dense) {
      jb = make_job(cs, (int)dense_agg_colsum_rows(prec, n), 1, L->f_out, eb);
    } else {
      int nb = 0;
      GCN_HIP(colsum_partial_launch(prec, dZ, n, L->f_out, L->ld_out, cs, L->ld_out, &nb, s));
      eb.cols = L->ld_out;
      jb = make_job(cs, nb, 1, L->ld_out, eb);
    }
  }
  if (ident) {
    // dW = I^T G_S = G_S: widened to fp32, padding columns zeroed
    GCN_HIP(cast_launch(prec, 0, n, L->f_out, GS, L->ld_out, dW, L->ld_out, overflow, s, L->ld_out));
    if (dbias) GCN_HIP(reduce_partials2(prec, jb, nullptr, s));
    return finish(hipSuccess, s);
  }
  // dW = H^T G_S (fp32, split over vertices), then one launch reduces the dW
  // spans and the dbias partials, each in a fixed order
  Epilogue ew = base_epi(dW, L->ld_out, L->f_in, L->f_out, EPI_F32, overflow);
  GCN_HIP(wgrad_launch(prec, H, L->ld_in, GS, L->ld_out, n, L->f_in, L->f_out, plan.dw_split, ws, s));
  const RedJob jw = make_job(ws, plan.dw_split, L->f_in, L->f_out, ew);
  GCN_HIP(reduce_partials2(prec, jw, dbias ? &jb : nullptr, s));
  // dZ_below = (G_S W^T) * [H > 0] / (1 - p_below)
  if (dZ_below) {
    Epilogue ed = base_epi(dZ_below, L->ld_in, n, L->f_in, EPI_DMASK, overflow);
    ed.relu = act_below == GCN_ACT_RELU;
    ed.keep_scale = 1.f / (1.f - p_below);
    ed.hmask = H;
    ed.ldh = L->ld_in;
    if (!dbias_below) {
      GCN_HIP(row_product(prec, GS, L->ld_out, W, L->ld_out, true, n, L->f_in, L->f_out, plan.dh_split, ws, ed, s));
    } else {
      // the bias gradient of the layer below, the column sums of dZ_below:
      // from the product's own workgroups where the row-streaming kernel
      // runs, else from a column-sum pass over the stored dZ_below
      Epilogue eb = base_epi(dbias_below, L->ld_in, 1, L->f_in, EPI_F32, overflow);
      RedJob jc{};
      if (use_tsgemm(prec, n, L->f_out)) {
        int rows = 0;
        GCN_HIP(tsgemm_launch(prec, GS, L->ld_out, W, L->ld_out, true, n, L->f_in, L->f_out, ed, s, cb, &rows));
        jc = make_job(cb, rows, 1, L->f_in, eb);
      } else {
        GCN_HIP(run_gemm(prec, true, true, GS, L->ld_out, W, L->ld_out, n, L->f_in, L->f_out, plan.dh_split, false,
                         ws, ed, s));
        int nb = 0;
        GCN_HIP(colsum_partial_launch(prec, dZ_below, n, L->f_in, L->ld_in, cb, L->ld_in, &nb, s));
        eb.cols = L->ld_in;
        jc = make_job(cb, nb, 1, L->ld_in, eb);
      }
      GCN_HIP(reduce_partials2(prec, jc, nullptr, s));
    }
  }
  return finish(hipSuccess, s);
}


}  // namespace

gcn_status gcn_layer_bwd(const gcn_adj* A, const gcn_layer* L, int32_t prec, const void* H, const void* W,
                         const void* dZ, int32_t act_below, float p_below, float* dW, float* dbias, void* dZ_below,
                         float* dbias_below, void* GS, int32_t* overflow, void* workspace, size_t workspace_bytes,
                         void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  gcn_status st = layer_bwd_check(A, L, prec, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, dbias_below, GS);
  if (st != GCN_OK) return st;
  const LayerPlan plan = plan_layer(A, L, prec);
  if (!workspace || workspace_bytes < plan_bytes(plan)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  return layer_bwd_run(A, L, prec, plan, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, dbias_below, GS, overflow,
                       static_cast<float*>(workspace), s);
}

// ---------------------------------------------------------------------------
// gcn_layer_bwd_noalloc: gcn_layer_bwd with its scratch in a fixed device
// array of this library instead of a caller workspace.  In host code the
// array's name is only a stand-in: the kernels get the device address that
// hipGetSymbolAddress returns for the current device, fetched once per
// device and kept.

__device__ __align__(256) unsigned char scratch[GCN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_addr[MAX_DEVICES];

gcn_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return GCN_ERR_DEVICE;
  if (dev < 0 || dev >= MAX_DEVICES) return GCN_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_addr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return GCN_ERR_DEVICE;
    scratch_addr[dev] = ptr;
  }
  *out = scratch_addr[dev];
  return GCN_OK;
}

}  // namespace

gcn_status gcn_layer_bwd_noalloc(const gcn_adj* A, const gcn_layer* L, int32_t prec, const void* H, const void* W,
                                 const void* dZ, int32_t act_below, float p_below, float* dW, float* dbias,
                                 void* dZ_below, float* dbias_below, void* GS, int32_t* overflow, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  gcn_status st = layer_bwd_check(A, L, prec, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, dbias_below, GS);
  if (st != GCN_OK) return st;
  const LayerPlan plan = plan_layer(A, L, prec);
  if (plan_bytes(plan) > (size_t)GCN_NOALLOC_SCRATCH_BYTES) return GCN_ERR_CAPACITY;
  void* scr = nullptr;
  st = scratch_of_current_device(&scr);
  if (st != GCN_OK) return st;
  return layer_bwd_run(A, L, prec, plan, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, dbias_below, GS, overflow,
                       static_cast<float*>(scr), s);
}

gcn_status gcn_loss_workspace_size(int64_t n, int64_t C, size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || C <= 0) return GCN_ERR_SHAPE;
  *bytes = loss_workspace_bytes(n, C);
  return GCN_OK;
}

gcn_status gcn_loss(int64_t n, int64_t C, int64_t ld, int32_t prec, const void* logits, const int32_t* labels,
                    const uint8_t* mask, int64_t n_mask, const float* loss_scale, float* loss, void* dlogits,
                    float* dlogits_colsum, int32_t* n_correct, int32_t* overflow, void* workspace,
                    size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || C <= 0 || ld < C || n_mask <= 0 || n_mask > n) return GCN_ERR_SHAPE;
  if (ld % 8) return GCN_ERR_ALIGNMENT;
  if (C > 64 * (prec == GCN_F32 ? 4 : 8)) return GCN_ERR_UNSUPPORTED;
  if (!logits || !labels || !loss || !dlogits) return GCN_ERR_INVALID_ARG;
  if (!aligned16(logits) || !aligned16(dlogits) || (dlogits_colsum && !aligned16(dlogits_colsum)))
    return GCN_ERR_ALIGNMENT;
  if (!workspace || workspace_bytes < loss_workspace_bytes(n, C)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  GCN_HIP(loss_launch(prec, n, C, ld, logits, labels, mask, n_mask, loss_scale, loss, dlogits, dlogits_colsum,
                      n_correct, overflow, workspace, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_optimizer_step(int64_t count, float* master, const float* grad, float* m, float* v, void* working,
                              int32_t prec, const gcn_adam_config* cfg, gcn_scaler* state, int32_t* overflow_flag,
                              void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (count <= 0) return GCN_ERR_SHAPE;
  if (!master || !grad || !m || !v || !cfg || !state || !overflow_flag) return GCN_ERR_INVALID_ARG;
  if (working && !valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (!(cfg->lr > 0.f) || !(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) || !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f) ||
      !(cfg->eps >= 0.f) || !(cfg->backoff > 0.f && cfg->backoff <= 1.f) || !(cfg->growth >= 1.f) ||
      cfg->interval <= 0 || !(cfg->min_scale > 0.f) || !(cfg->max_scale >= cfg->min_scale))
    return GCN_ERR_INVALID_ARG;
  AdamHyper hp;
  hp.lr = cfg->lr; hp.beta1 = cfg->beta1; hp.beta2 = cfg->beta2; hp.eps = cfg->eps;
  hp.backoff = cfg->backoff; hp.growth = cfg->growth; hp.interval = cfg->interval;
  hp.min_scale = cfg->min_scale; hp.max_scale = cfg->max_scale;
  static_assert(sizeof(gcn_scaler) == sizeof(ScalerState), "scaler layout");
  GCN_HIP(optimizer_launch(count, master, grad, m, v, working, prec, hp, reinterpret_cast<ScalerState*>(state),
                           overflow_flag, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_cast(int64_t rows, int64_t cols, int32_t src_prec, const void* src, int64_t ld_src, int32_t dst_prec,
                    void* dst, int64_t ld_dst, int32_t* overflow, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(src_prec) || !valid_prec(dst_prec) || !src || !dst) return GCN_ERR_INVALID_ARG;
  if (rows <= 0 || cols <= 0) return GCN_ERR_SHAPE;
  if (rows > 1 && (ld_src < cols || ld_dst < cols)) return GCN_ERR_SHAPE;
  if (!aligned16(src) || !aligned16(dst)) return GCN_ERR_ALIGNMENT;
  if (rows > 1 && (ld_src % 8 || ld_dst % 8)) return GCN_ERR_ALIGNMENT;
  GCN_HIP(cast_launch(src_prec, dst_prec, rows, cols, src, rows > 1 ? ld_src : 0, dst, rows > 1 ? ld_dst : 0,
                      overflow, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_optimizer_step_half(int64_t count, void* w, const float* grad, void* m, void* v, float* widened,
                                   int32_t prec, const gcn_adam_config* cfg, gcn_scaler* state,
                                   int32_t* overflow_flag, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (count <= 0) return GCN_ERR_SHAPE;
  if (!w || !grad || !m || !v || !cfg || !state || !overflow_flag) return GCN_ERR_INVALID_ARG;
  if (prec != GCN_F16 && prec != GCN_BF16) return GCN_ERR_INVALID_ARG;
  if (!(cfg->lr > 0.f) || !(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) || !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f) ||
      !(cfg->eps >= 0.f))
    return GCN_ERR_INVALID_ARG;
  AdamHyper hp{};
  hp.lr = cfg->lr; hp.beta1 = cfg->beta1; hp.beta2 = cfg->beta2; hp.eps = cfg->eps;
  GCN_HIP(adam_half_launch(count, w, grad, m, v, widened, prec, hp, reinterpret_cast<ScalerState*>(state),
                           overflow_flag, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_sample_pairs(int64_t n, const int32_t* edge_u, const int32_t* edge_v, int64_t n_edges, int64_t n_pos,
                            int64_t n_neg, uint64_t seed, uint64_t epoch, int32_t* pair_u, int32_t* pair_v,
                            void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n < 2 || n > INT32_MAX || n_pos < 0 || n_neg < 0 || n_pos + n_neg <= 0) return GCN_ERR_SHAPE;
  if (n_pos + n_neg > INT32_MAX) return GCN_ERR_UNSUPPORTED;
  if (n_pos > 0 && (n_edges < 1 || !edge_u || !edge_v)) return GCN_ERR_INVALID_ARG;
  if (!pair_u || !pair_v) return GCN_ERR_INVALID_ARG;
  GCN_HIP(sample_pairs_launch(n, edge_u, edge_v, n_edges, n_pos, n_neg, seed, epoch, pair_u, pair_v, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_pair_loss_workspace_size(int64_t n_pairs, size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n_pairs <= 0) return GCN_ERR_SHAPE;
  *bytes = pair_loss_workspace_bytes(n_pairs);
  return GCN_OK;
}

gcn_status gcn_pair_loss(int64_t n, int64_t F, int64_t ld, int32_t prec, const void* Z, const int32_t* pair_u,
                         const int32_t* pair_v, int64_t n_pos, int64_t n_neg, const float* loss_scale, float* loss,
                         float* scores, float* g, int32_t* overflow, void* workspace, size_t workspace_bytes,
                         void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || F <= 0 || ld < F || n_pos < 0 || n_neg < 0 || n_pos + n_neg <= 0) return GCN_ERR_SHAPE;
  if (n_pos + n_neg > INT32_MAX) return GCN_ERR_UNSUPPORTED;
  if (ld % 8) return GCN_ERR_ALIGNMENT;
  if (F > 64 * (prec == GCN_F32 ? 4 : 8)) return GCN_ERR_UNSUPPORTED;
  if (!Z || !pair_u || !pair_v || !loss || !g) return GCN_ERR_INVALID_ARG;
  if (!aligned16(Z)) return GCN_ERR_ALIGNMENT;
  if (!workspace || workspace_bytes < pair_loss_workspace_bytes(n_pos + n_neg)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  GCN_HIP(pair_loss_launch(prec, n, F, ld, Z, pair_u, pair_v, n_pos, n_neg, loss_scale, loss, scores, g, overflow,
                           workspace, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_pair_backward_workspace_size(int64_t n, int64_t n_pairs, int64_t F, size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || n_pairs < 0 || F <= 0) return GCN_ERR_SHAPE;
  *bytes = pair_backward_workspace_bytes(n, n_pairs, F);
  return GCN_OK;
}

gcn_status gcn_pair_backward(int64_t n, int64_t F, int64_t ld, int32_t prec, const void* Z, const int32_t* pair_u,
                             const int32_t* pair_v, int64_t n_pairs, const float* g, void* dZ, int64_t ldz,
                             int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!valid_prec(prec)) return GCN_ERR_INVALID_ARG;
  if (n <= 0 || n > INT32_MAX || F <= 0 || ld < F || ldz < F || n_pairs < 0) return GCN_ERR_SHAPE;
  if (n_pairs > INT32_MAX / 2) return GCN_ERR_UNSUPPORTED;
  if (ld % 8 || ldz % 8) return GCN_ERR_ALIGNMENT;
  if (F > 64 * (prec == GCN_F32 ? 4 : 8)) return GCN_ERR_UNSUPPORTED;
  if (!Z || !dZ || (n_pairs > 0 && (!pair_u || !pair_v || !g))) return GCN_ERR_INVALID_ARG;
  if (!aligned16(Z) || !aligned16(dZ)) return GCN_ERR_ALIGNMENT;
  if (!workspace || workspace_bytes < pair_backward_workspace_bytes(n, n_pairs, F)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  GCN_HIP(pair_backward_launch(prec, n, F, ld, Z, pair_u, pair_v, n_pairs, g, dZ, ldz, overflow, workspace, s));
  return finish(hipSuccess, s);
}

gcn_status gcn_pair_metrics_workspace_size(int64_t n_pos, int64_t n_neg, size_t* bytes) {
  if (!bytes) return GCN_ERR_INVALID_ARG;
  if (n_pos <= 0 || n_neg <= 0 || n_pos + n_neg > INT32_MAX) return GCN_ERR_SHAPE;
  *bytes = pair_metrics_workspace_bytes(n_pos, n_neg);
  return GCN_OK;
}

gcn_status gcn_pair_metrics(const float* scores, int64_t n_pos, int64_t n_neg, double* auc_ap, void* workspace,
                            size_t workspace_bytes, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n_pos <= 0 || n_neg <= 0 || n_pos + n_neg > INT32_MAX) return GCN_ERR_SHAPE;
  if (!scores || !auc_ap) return GCN_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < pair_metrics_workspace_bytes(n_pos, n_neg)) return GCN_ERR_WORKSPACE;
  if (!aligned16(workspace)) return GCN_ERR_ALIGNMENT;
  GCN_HIP(pair_metrics_launch(scores, n_pos, n_neg, auc_ap, workspace, s));
  return finish(hipSuccess, s);
}

}  // extern "C"

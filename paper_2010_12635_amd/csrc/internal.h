// Host-side launch functions of the libgcn kernels (internal; not exported).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"
#include "gcn.h"

namespace gcn {

// Accelerator complex dies of gfx950 (MI355X): consecutive workgroups of a
// launch are dealt to them in turn, workgroup w to die w % XCDS, each die
// with its own L2.
constexpr int64_t XCDS = 8;

// ----------------------------------------------------------------- GEMM ----
// C[M x N] = sum_k A(m, k) * B(k, n) with fp32 accumulation on MFMA.
// A(m, k) = a_kc ? A[m * lda + k] : A[k * lda + m]
// B(k, n) = b_kc ? B[n * ldb + k] : B[k * ldb + n]
// With splits > 1 the K range is cut into `splits` pieces (multiples of the
// K tile) whose fp32 partial sums go to `partials` [splits][M][N]; the
// caller then runs reduce_partials.  With splits == 1 the epilogue is
// applied directly.
struct GemmCall {
  int prec;              // gcn_precision
  bool a_kc, b_kc;
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  int64_t M, N, K;
  int splits;
  float* partials;
  Epilogue epi;
};
// Number of K splits the GEMM would use for these sizes (1 = none).
int gemm_choose_splits(int prec, int64_t M, int64_t N, int64_t K);
hipError_t gemm_launch(const GemmCall& c, hipStream_t s);

// out = epilogue(sum over s < splits of partials[s][r][c]) for r < M, c < N,
// splits added in order; for EPI_F32 columns [N, ldo) are written 0.
struct RedJob {
  const float* part;
  int splits;
  int64_t M, N, width, blocks;
  int64_t ld;                   // floats between partial rows of one split (N unless given)
  int opw;                      // outputs per workgroup: 64, 16, 4 or 1 (256 / opw groups of splits)
  Epilogue ep;
};
RedJob make_job(const float* partials, int splits, int64_t M, int64_t N, const Epilogue& epi);
// The same for partial rows ld >= N floats apart (split stride M * ld).
RedJob make_job_ld(const float* partials, int splits, int64_t M, int64_t N, int64_t ld, const Epilogue& epi);
// One launch for job a and, if b != NULL, job b.
hipError_t reduce_partials2(int prec, const RedJob& a, const RedJob* b, hipStream_t s);
hipError_t reduce_partials(int prec, const float* partials, int splits, int64_t M, int64_t N,
                           const Epilogue& epi, hipStream_t s);

// Column-sum partials of X (rows x cols, ld): partials[b][c] for c < ldp
// (zero for c >= cols), *splits = number of row blocks b; reduce with
// make_job(partials, *splits, 1, ldp, epi).  partials needs
// colsum_partials_floats() floats.
int64_t colsum_partials_floats(int64_t rows, int64_t ld);
hipError_t colsum_partial_launch(int prec, const void* X, int64_t rows, int64_t cols, int64_t ld, float* partials,
                                 int64_t ldp, int* splits, hipStream_t s);

// ----------------------------------------------------------------- SpMM ----
// Where a light row or a heavy-row piece lies: first entry, row, number of
// entries (pieces: bit 31 set when the piece is its row's only one).
struct RowDesc {
  int64_t beg;
  int32_t row;
  int32_t len;
};
static_assert(sizeof(RowDesc) == 16, "one 16-byte load per descriptor");

struct CsrView {
  int64_t n, nnz;
  bool idx64;
  const void* rowptr;
  const int32_t* colidx;
  const void* values;    // storage type == prec, or NULL (dinv product)
  const float* dinv;
  int64_t heavy_threshold, chunk_nnz, n_heavy, n_chunks;
  const int32_t* heavy_rows;
  const int32_t* heavy_chunk_off;
  const int32_t* chunk_heavy;
  int64_t n_light;
  const int32_t* row_perm;   // light rows, degree descending (NULL: index order)
  const int32_t* chunk_order;  // pieces by first column, grouped by column range
  const int64_t* chunk_beg;    // [n_chunks + 1] first entry of each piece
  const int64_t* part_off;     // [parts + 1] ranges of chunk_order per column range
  int64_t parts, part_slots;   // column ranges (1 or a multiple of XCDS); most pieces per XCD
  const RowDesc* piece_desc;   // [n_chunks] in chunk_order positions
  const int32_t* piece_pos;    // [n_chunks] chunk_order position of each piece
  const RowDesc* row_desc;     // [n_light] in row_perm order
  int64_t n_light_single;      // the last rows of row_perm / row_desc with exactly one entry
  int64_t n_fix, n_fix_big;    // heavy rows of > 1 piece; of them, rows of > GCN_FIX_BIG_PIECES
  const int32_t* fix_rows;     // [n_fix] their heavy-row slots, the big ones first
};
// Y = A_hat X (+ epilogue) for X: n x F (ld), Y described by epi.
int64_t spmm_partials_floats(const CsrView& A, int prec, int64_t F);
hipError_t spmm_launch(const CsrView& A, int prec, const void* X, int64_t ldx, int64_t F,
                       const Epilogue& epi, float* partials, hipStream_t s);

// ------------------------------------------------- tall-skinny products ----
// C (M x N) = A (M x K, row-major, lda) . B, B(k, n) = b_kc ? B[n * ldb + k]
// : B[k * ldb + n]; epilogue EPI_STORE or EPI_DMASK (16-byte row stores).
// With colsum (B k-contiguous only), each workgroup also writes the column
// sums of what it stored, as stored, to row w of colsum ([rows][N] floats,
// *colsum_rows = the workgroups per column block, at most
// tsgemm_colsum_rows_max()).
bool tsgemm_supported(int prec, int64_t K);
int tsgemm_colsum_rows_max();
hipError_t tsgemm_launch(int prec, const void* A, int64_t lda, const void* B, int64_t ldb, bool b_kc, int64_t M,
                         int64_t N, int64_t K, const Epilogue& epi, hipStream_t s, float* colsum = nullptr,
                         int* colsum_rows = nullptr);

// ----------------------------------------------------- weight gradient ----
// partials[s][m][n] = sum over the s-th vertex span of H[k][m] * G[k][n];
// reduce_partials then adds the spans in order.
int wgrad_splits(int prec, int64_t n, int64_t M, int64_t N);
hipError_t wgrad_launch(int prec, const void* H, int64_t ldh, const void* G, int64_t ldg, int64_t n, int64_t M,
                        int64_t N, int splits, float* partials, hipStream_t s);

// ------------------------------------------------ dense-A_hat aggregation ----
// Y = epilogue(A_hat X) for dense A_hat (n x lda); ws holds the padded
// transpose of X and, for the wide kernel with k ranges, their fp32
// partials (dense_agg_workspace_bytes).  With colsum != NULL the
// transposition also writes column-sum partials of X, [rows][F] floats with
// rows = dense_agg_colsum_rows(); reduce with make_job(colsum, rows, 1, F, ..).
size_t dense_agg_workspace_bytes(int prec, int64_t n, int64_t F, bool tiled);
int64_t dense_agg_colsum_rows(int prec, int64_t n);
hipError_t dense_agg_launch(int prec, const void* A, int64_t lda, bool tiled, int64_t n, const void* X, int64_t ldx,
                            int64_t F, const Epilogue& epi, void* ws, float* colsum, hipStream_t s);
// Elements of the tiled dense A_hat (rows padded to 64, columns to the chunk).
int64_t dense_tiled_elems(int prec, int64_t n);
// Dense A_hat from CSR: row-major (ld) or tiled operand order.
hipError_t densify_launch(const CsrView& A, int prec, bool tiled, void* dense, int64_t ld, hipStream_t s);

// ------------------------------------------------------------ normalize ----
size_t normalize_workspace_bytes(int64_t n, int64_t num_edges);
hipError_t normalize_run(int64_t n, int64_t num_edges, const int32_t* src, const int32_t* dst,
                         bool idx64, void* rowptr, int32_t* colidx, int32_t* deg, float* dinv,
                         int value_prec, void* values, void* dense, int64_t ld_dense,
                         int64_t* nnz_out, int32_t* bad_ids, void* ws, size_t ws_bytes,
                         hipStream_t s);
// Heavy-row pieces and light-row order (see gcn_schedule in gcn.h); the
// pointers returned point into `sched`.
struct SchedOut {
  int32_t *heavy_rows, *heavy_chunk_off, *chunk_heavy, *row_perm, *chunk_order, *piece_pos, *fix_rows;
  int64_t *chunk_beg, *part_off;
  RowDesc *piece_desc, *row_desc;
  int64_t n_heavy, n_chunks, n_light, part_slots, n_fix, n_fix_big, n_light_single;
};
size_t schedule_bytes(int64_t n, int64_t nnz, int64_t threshold, int64_t chunk_nnz, int64_t parts);
hipError_t schedule_run(int64_t n, int64_t nnz, bool idx64, const void* rowptr, const int32_t* colidx,
                        int64_t threshold, int64_t chunk_nnz, int64_t parts, void* sched, size_t sched_bytes,
                        SchedOut* out, hipStream_t s);

// ----------------------------------------------------------------- loss ----
size_t loss_workspace_bytes(int64_t n, int64_t C);
hipError_t loss_launch(int prec, int64_t n, int64_t C, int64_t ld, const void* logits,
                       const int32_t* labels, const uint8_t* mask, int64_t n_mask,
                       const float* loss_scale, float* loss, void* dlogits, float* dlogits_colsum,
                       int32_t* n_correct, int32_t* flag, void* ws, hipStream_t s);

// ------------------------------------------------------------ optimiser ----
struct AdamHyper {
  float lr, beta1, beta2, eps, backoff, growth, min_scale, max_scale;
  int32_t interval;
};
struct ScalerState { float scale; int32_t good_steps; int32_t step; int32_t skipped; };
hipError_t optimizer_launch(int64_t count, float* master, const float* grad, float* m, float* v,
                            void* working, int prec, const AdamHyper& hp, ScalerState* state,
                            int32_t* flag, hipStream_t s);
hipError_t adam_half_launch(int64_t count, void* w, const float* grad, void* m, void* v, float* widened, int prec,
                            const AdamHyper& hp, ScalerState* state, int32_t* flag, hipStream_t s);
// dst[:, :cols] = src converted; with zcols > cols, dst[:, cols:zcols] = 0.
hipError_t cast_launch(int src_prec, int dst_prec, int64_t rows, int64_t cols, const void* src, int64_t lds,
                       void* dst, int64_t ldd, int32_t* flag, hipStream_t s, int64_t zcols = 0);

// --------------------------------------------------------------- helpers ----
hipError_t fill_zero(void* p, size_t bytes, hipStream_t s);
// In-place exclusive scan of int64 data[0..count); scratch holds
// segment_scan_scratch_elems(count) int64.
int64_t segment_scan_scratch_elems(int64_t count);
hipError_t segment_scan_exclusive(int64_t* data, int64_t count, int64_t* scratch, hipStream_t s);

// ------------------------------------------------------ link prediction ----
// Pair decoder of Eq. (2) on sampled pairs (see gcn.h for the definitions).
hipError_t sample_pairs_launch(int64_t n, const int32_t* edge_u, const int32_t* edge_v, int64_t n_edges, int64_t n_pos,
                               int64_t n_neg, uint64_t seed, uint64_t epoch, int32_t* pair_u, int32_t* pair_v,
                               hipStream_t s);
size_t pair_loss_workspace_bytes(int64_t n_pairs);
hipError_t pair_loss_launch(int prec, int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pair_u,
                            const int32_t* pair_v, int64_t n_pos, int64_t n_neg, const float* loss_scale, float* loss,
                            float* scores, float* g, int32_t* flag, void* ws, hipStream_t s);
size_t pair_backward_workspace_bytes(int64_t n, int64_t n_pairs, int64_t F);
hipError_t pair_backward_launch(int prec, int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pair_u,
                                const int32_t* pair_v, int64_t n_pairs, const float* g, void* dZ, int64_t ldz,
                                int32_t* flag, void* ws, hipStream_t s);
size_t pair_metrics_workspace_bytes(int64_t n_pos, int64_t n_neg);
hipError_t pair_metrics_launch(const float* scores, int64_t n_pos, int64_t n_neg, double* auc_ap, void* ws,
                               hipStream_t s);

}  // namespace gcn

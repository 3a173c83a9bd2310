/*
 * gcn.h -- C ABI of libgcn: forward and backward of the graph convolutional
 * layer on AMD Instinct MI355X (gfx950).
 *
 * The operation is the layer of Kipf & Welling that the paper studies
 * (Section "Graph Convolutions", Eq. (1)):
 *
 *     H' = sigma(A_hat (H W) + b),   A_hat = D^-1/2 (A + I) D^-1/2,
 *
 * for an undirected graph G = (V, E) whose edges are unordered vertex pairs
 * (Section "Introduction", definition of A), with A: n x n, H: n x f_in,
 * W: f_in x f_out (the shape list of Section "Graph Convolutions").  sigma is
 * ReLU followed by inverted dropout on hidden layers and the identity on the
 * output layer.  Storage precision follows the optimisation levels of Section
 * "Background and Motivation": GCN_F32 is the all-fp32 level O0; GCN_F16 and
 * GCN_BF16 are the O2 "almost fp16" level (16-bit weights and activations,
 * fp32 master weights, fp32 optimiser, dynamic loss scaling).  Every product
 * accumulates in fp32 in every mode.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.    Every array argument is device memory allocated and owned by the
 *            caller (this library allocates nothing and keeps no global
 *            state), except the documented host outputs (nnz_out, sizes).
 *            Base pointers must be 16-byte aligned.
 * Layout.    Row-major.  A matrix with logical width f has a leading
 *            dimension ld >= f with ld % 8 == 0: the paper pads matrices to
 *            multiples of 8 for 16-bit matrix units (Section "Reduced
 *            Precision Changes"); here that rule is a layout rule and the
 *            logical widths stay arbitrary.  Columns [f, ld) of an input are
 *            ignored; columns [f, ld) of an output may be overwritten with 0.
 * Streams.   `stream` is a hipStream_t (NULL = default stream).  All calls are
 *            asynchronous on it, except gcn_normalize and gcn_schedule, which
 *            synchronise it (once and twice) to return sizes to the host.
 * Errors.    Every call validates its arguments on the host before it
 *            launches anything and returns a gcn_status; a call that returns
 *            an argument error has had no effect.  GCN_ERR_DEVICE reports a
 *            failed launch or runtime call.  Numeric overflow is not an
 *            error: it sets *overflow (a device int32) to 1.
 * Precision. `prec` (gcn_precision) is the storage type of H, W, S, H_out,
 *            dZ, G_S and dZ_below.  Biases, gradients of W and b, dinv,
 *            losses and optimiser state are fp32.
 */
#ifndef GCN_H
#define GCN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GCN_ABI_VERSION 11

typedef enum gcn_status {
  GCN_OK = 0,
  GCN_ERR_INVALID_ARG = 1,  /* NULL required pointer, bad enum, bad scalar   */
  GCN_ERR_SHAPE = 2,        /* non-positive or inconsistent sizes            */
  GCN_ERR_ALIGNMENT = 3,    /* ld % 8 != 0 or pointer not 16-byte aligned   */
  GCN_ERR_UNSUPPORTED = 4,  /* valid but not implemented combination        */
  GCN_ERR_CAPACITY = 5,     /* an output buffer is too small                 */
  GCN_ERR_WORKSPACE = 6,    /* workspace missing or smaller than required   */
  GCN_ERR_DEVICE = 7,       /* HIP runtime or launch failure                */
  GCN_ERR_GRAPH = 8         /* edge list holds a vertex id outside [0, n)    */
} gcn_status;

typedef enum gcn_precision { GCN_F32 = 0, GCN_F16 = 1, GCN_BF16 = 2 } gcn_precision;
typedef enum gcn_index { GCN_I32 = 0, GCN_I64 = 1 } gcn_index;       /* rowptr width */
typedef enum gcn_adj_format { GCN_CSR = 0, GCN_DENSE = 1, GCN_DENSE_TILED = 2 } gcn_adj_format;
typedef enum gcn_act { GCN_ACT_NONE = 0, GCN_ACT_RELU = 1 } gcn_act;

/* Normalised adjacency A_hat (device arrays, caller-owned).
 * CSR: rows sorted, columns sorted and unique within a row, A_hat symmetric
 * (gcn_layer_bwd uses A_hat^T = A_hat).  values == NULL means
 * A_hat_ij = dinv[i] * dinv[j] computed on the fly.
 * DENSE: dense[i * ld_dense + j] = A_hat_ij in value_prec.
 * DENSE_TILED: the dense matrix stored in matrix-core operand order (see
 * gcn_densify); ld_dense is ignored.
 * The heavy-row schedule (filled by gcn_schedule) lets the CSR product split
 * rows with more than heavy_threshold entries into pieces that separate lane
 * groups sum, each into an fp32 partial row, the partials of a row then
 * added in a fixed order (run-to-run deterministic); with n_heavy == 0 every
 * row is processed whole.  With col_parts = P > 1 the columns are cut into
 * P ranges [p n / P, (p + 1) n / P) and a heavy row's pieces never cross a
 * range boundary; the pieces of range p run on the chip's XCD p mod 8, so
 * each XCD's L2 caches the rows of X of its own column ranges only.
 * gcn_schedule also lists the other ("light") rows in order of decreasing
 * degree (row_perm), so that the rows a wavefront processes together have
 * similar lengths, the rows of a single entry last (n_light_single of them,
 * which a lane group takes four at a time); with row_perm == NULL rows
 * are processed in index order. */
typedef struct gcn_adj {
  int64_t n;
  int64_t nnz;
  int32_t format;        /* gcn_adj_format */
  int32_t index;         /* gcn_index of rowptr; colidx is always int32 */
  int32_t value_prec;    /* gcn_precision of values / dense (== layer prec) */
  int32_t reserved0;
  const void* rowptr;    /* [n + 1] */
  const int32_t* colidx; /* [nnz]   */
  const void* values;    /* [nnz] or NULL */
  const float* dinv;     /* [n]: deg^-1/2, deg counting the self-loop */
  const void* dense;     /* [n x ld_dense] (GCN_DENSE) */
  int64_t ld_dense;
  int64_t heavy_threshold;        /* rows with more entries are "heavy"      */
  int64_t chunk_nnz;              /* most entries in one piece of a heavy row */
  int64_t n_heavy;                /* number of heavy rows                    */
  int64_t n_chunks;               /* total pieces over all heavy rows        */
  const int32_t* heavy_rows;      /* [n_heavy] ascending row ids             */
  const int32_t* heavy_chunk_off; /* [n_heavy + 1] first piece of each row   */
  const int32_t* chunk_heavy;     /* [n_chunks] heavy-row slot of a piece    */
  int64_t n_light;                /* rows listed in row_perm                 */
  const int32_t* row_perm;        /* [n_light] light rows, degree descending */
  const int32_t* chunk_order;     /* [n_chunks] pieces by the column of their
                                     first entry (grouped by column range)  */
  const int64_t* chunk_beg;       /* [n_chunks + 1] first entry of each piece
                                     (pieces of a row are consecutive)      */
  const int64_t* part_off;        /* [col_parts + 1] pieces of column range p
                                     are chunk_order[part_off[p] ..
                                     part_off[p + 1])                       */
  int64_t col_parts;              /* column ranges P: 1 or a multiple of 8   */
  int64_t part_slots;             /* most pieces on one XCD (P > 1)          */
  const void* piece_desc;         /* [n_chunks] 16-byte piece descriptors in
                                     chunk_order positions                  */
  const int32_t* piece_pos;       /* [n_chunks] chunk_order position of each
                                     piece                                  */
  const void* row_desc;           /* [n_light] 16-byte light-row descriptors
                                     in row_perm order (required with
                                     row_perm)                              */
  int64_t n_light_single;         /* the last n_light_single rows of row_perm
                                     (and row_desc) have exactly one entry  */
  int64_t n_fix;                  /* heavy rows of more than one piece       */
  int64_t n_fix_big;              /* how many of them have more than
                                     GCN_FIX_BIG_PIECES pieces              */
  const int32_t* fix_rows;        /* [n_fix] heavy-row slots (indices into
                                     heavy_rows) of the rows of more than one
                                     piece: the n_fix_big rows of more than
                                     GCN_FIX_BIG_PIECES pieces first, each
                                     group in ascending order               */
} gcn_adj;

/* A heavy row of more than this many pieces has its partials added by a
 * whole workgroup (contiguous runs of pieces per lane group, then the runs
 * in order); fewer, by one lane group in piece order. */
#define GCN_FIX_BIG_PIECES 32

/* One layer: H (n x f_in, ld_in) -> H_out (n x f_out, ld_out); W is
 * f_in x f_out with leading dimension ld_out; bias has f_out entries.
 * identity_input != 0 declares H = I (the featureless input of the paper's
 * run-time experiments, Section "Run-Time and Memory Usage Analysis"):
 * f_in must equal n, H is not read (may be NULL), H W = W exactly, and the
 * calls below skip the products with I. */
typedef struct gcn_layer {
  int64_t f_in;
  int64_t f_out;
  int64_t ld_in;
  int64_t ld_out;
  int32_t act;           /* gcn_act applied after aggregation              */
  float dropout_p;       /* in [0, 1); only with GCN_ACT_RELU and training  */
  int32_t layer_id;      /* dropout stream id                               */
  int32_t identity_input;/* 1: H is the n x n identity (f_in == n)         */
  const struct gcn_scaler* epoch_from;
                         /* NULL, or the device loss-scale state whose
                            step + skipped (optimiser calls so far) is added
                            to the epoch argument of gcn_layer_fwd when its
                            kernels run: a training epoch captured into a
                            HIP graph then draws a new dropout mask at every
                            replay                                          */
} gcn_layer;

/* Dynamic loss-scale state, device-resident (16 bytes). */
typedef struct gcn_scaler {
  float scale;           /* current loss scale S                            */
  int32_t good_steps;    /* consecutive steps without overflow              */
  int32_t step;          /* Adam step count t (applied steps only)          */
  int32_t skipped;       /* total skipped steps                             */
} gcn_scaler;

typedef struct gcn_adam_config {
  float lr, beta1, beta2, eps;
  float backoff;         /* scale multiplier on overflow (0.5)              */
  float growth;          /* scale multiplier after `interval` good steps (2)*/
  int32_t interval;      /* good steps before growth (2000)                 */
  float min_scale;       /* lower clamp of S (1)                            */
  float max_scale;       /* upper clamp of S (2^24)                         */
} gcn_adam_config;

/* Human-readable name of a status code (static string). */
const char* gcn_status_string(int32_t status);
/* GCN_ABI_VERSION of the built library. */
int32_t gcn_abi_version(void);

/* ---------------------------------------------------------------------------
 * gcn_normalize: build A_hat from an undirected edge list.
 *
 * Input: num_edges pairs (src[k], dst[k]) of vertex ids in [0, n).  A pair is
 * an unordered edge {u, v} (Section "Introduction", definition of A):
 * (u, v) and (v, u) are the same edge, repeats collapse, u == v pairs are
 * dropped, and one self-loop per vertex is added (A + I).  Output is the
 * canonical CSR (rows ascending, columns ascending and unique) with
 * deg[i] = |N(i)| + 1, dinv[i] = float(1 / sqrt(double(deg[i]))),
 * values[k] = dinv[row] * dinv[col] rounded to value_prec, and optionally
 * the dense n x ld_dense matrix (all other entries zero).
 *
 * rowptr: [n + 1] of `index` width; colidx: [nnz_capacity] with
 * nnz_capacity >= 2 * num_edges + n (always sufficient); deg (int32, may be
 * NULL), dinv (required), values (may be NULL), dense (may be NULL).
 * GCN_I32 requires 2 * num_edges + n < 2^31.  workspace: at least
 * gcn_normalize_workspace_size() bytes.  *nnz_out (host) receives nnz.
 * Synchronises `stream` once.  Returns GCN_ERR_GRAPH if a vertex id lies
 * outside [0, n) (outputs are then undefined).  The result is bit-identical
 * from run to run.
 * ------------------------------------------------------------------------- */
gcn_status gcn_normalize_workspace_size(int64_t n, int64_t num_edges, size_t* bytes);
gcn_status gcn_normalize(int64_t n, int64_t num_edges, const int32_t* src, const int32_t* dst,
                         int32_t index, void* rowptr, int32_t* colidx, int64_t nnz_capacity,
                         int32_t* deg, float* dinv, int32_t value_prec, void* values,
                         void* dense, int64_t ld_dense, int64_t* nnz_out,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_densify: write the dense form of a CSR A_hat (values, or dinv[i] *
 * dinv[j] when values is NULL, rounded to value_prec) into `dense`, every
 * other entry zero.
 *   format GCN_DENSE:       dense[i * ld_dense + j], ld_dense >= n, % 8 == 0.
 *   format GCN_DENSE_TILED: rows are grouped in blocks of 64, columns in
 *     chunks of KC = 32 (16-bit) or 16 (fp32) elements; with VE = KC / 4,
 *     element (i, j) lives at
 *       (((i / 64) * NC + j / KC) * 4 + (i % 64) / 16) * 16 * KC
 *       + ((j % KC) / VE * 16 + i % 16) * VE + j % VE,
 *     NC = ceil(n / KC): each 16-row x KC-column piece is one contiguous
 *     1 KiB block in the lane order of a 16x16 MFMA operand, and the 64 rows
 *     of a block are contiguous along k.  Size: gcn_dense_tiled_elems().
 *     This is the layout the dense aggregation streams at full bandwidth.
 * Asynchronous on `stream`.
 * ------------------------------------------------------------------------- */
gcn_status gcn_dense_tiled_elems(int64_t n, int32_t prec, int64_t* elems);
gcn_status gcn_densify(const gcn_adj* A, int32_t format, int32_t value_prec, void* dense, int64_t ld_dense,
                       void* stream);

/* ---------------------------------------------------------------------------
 * gcn_schedule: fill the heavy-row fields of a CSR gcn_adj (n, nnz, index,
 * rowptr, colidx must be set).  Rows with more than heavy_threshold entries
 * are cut into pieces: first at the boundaries of the col_parts column
 * ranges, then every chunk_nnz entries; a lane group sums each piece into
 * an fp32 partial row and a fix-up adds a row's partials in a fixed order
 * (run-to-run deterministic; fix_rows lists the rows it visits).  The
 * pieces are launched grouped by column
 * range (range p on XCD p mod 8) and, inside a range, in order of the
 * column of their first entry (chunk_order; pieces of different hubs that
 * cover the same columns then run together and share the cached rows of
 * X).  The remaining rows are listed by decreasing length (row_perm).  The
 * launch orders are permutations whose ties may come out in any order;
 * results do not depend on them.  heavy_threshold <= 0, chunk_nnz <= 0 and
 * col_parts <= 0 select the defaults (heavy_threshold 128, chunk_nnz 256,
 * col_parts 1); col_parts must
 * otherwise be 1, 8, 16, 32 or 64 (GCN_ERR_INVALID_ARG).  sched: device
 * buffer of at least gcn_schedule_size() bytes (same arguments) that must
 * outlive every use of *A.  Synchronises `stream` twice.
 * ------------------------------------------------------------------------- */
gcn_status gcn_schedule_size(int64_t n, int64_t nnz, int64_t heavy_threshold, int64_t chunk_nnz,
                             int64_t col_parts, size_t* bytes);
gcn_status gcn_schedule(gcn_adj* A, int64_t heavy_threshold, int64_t chunk_nnz, int64_t col_parts,
                        void* sched, size_t sched_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_layer_fwd: one layer of Eq. (1), computed as A_hat (H W) + b.
 *   S     = H W                               (n x f_out, ld_out, prec)
 *   Z     = A_hat S + bias                    (bias fp32 [f_out], may be NULL)
 *   H_out = dropout(ReLU(Z)) if act == RELU, else Z     (n x f_out, ld_out)
 * Inverted dropout (training != 0, dropout_p > 0): element (i, j) with
 * e = i * f_out + j is kept iff output word (e % 4) of Philox-4x32-10 with
 * counter (b mod 2^32, b / 2^32, epoch mod 2^32, layer_id), b = e / 4, and
 * key (seed mod 2^32, seed / 2^32) is >= floor(p * 2^32); kept values are
 * multiplied by 1 / (1 - p) in fp32.
 * S is caller scratch that the backward pass does not need.  workspace: at
 * least gcn_layer_workspace_size() bytes.  *overflow is set to 1 if any
 * stored element of H_out is not finite.
 * With L->identity_input, S = W and the aggregation reads W in place (S is
 * not written and may be NULL); GCN_ERR_SHAPE unless f_in == n.
 * ------------------------------------------------------------------------- */
gcn_status gcn_layer_workspace_size(const gcn_adj* A, const gcn_layer* L, int32_t prec, size_t* bytes);
gcn_status gcn_layer_fwd(const gcn_adj* A, const gcn_layer* L, int32_t prec, int32_t training,
                         const void* H, const void* W, const float* bias,
                         uint64_t seed, uint64_t epoch, void* S, void* H_out,
                         int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_transform and gcn_aggregate: the two halves of gcn_layer_fwd, for
 * callers that schedule or time them separately (Eq. (1) read as
 * A_hat (H W); the product is never re-associated).
 *   gcn_transform:  S = H W     H: n x f_in (ld_in), W: f_in x f_out (ld_w),
 *                               S: n x f_out (ld_s), all prec, fp32 accumulation.
 *   gcn_aggregate:  Y = sigma(A_hat X + bias) with the epilogue of
 *                   gcn_layer_fwd (act, dropout with key (seed, layer_id),
 *                   counter (e / 8, epoch, 0, 0), e = i * F + j).
 *                   X, Y: n x F (ldx, ldy), prec.
 * Workspace sizes come from the matching *_workspace_size call.
 * ------------------------------------------------------------------------- */
gcn_status gcn_transform_workspace_size(int64_t n, int64_t f_in, int64_t f_out, int32_t prec, size_t* bytes);
gcn_status gcn_transform(int64_t n, int64_t f_in, int64_t f_out, int32_t prec, const void* H, int64_t ld_in,
                         const void* W, int64_t ld_w, void* S, int64_t ld_s, int32_t* overflow,
                         void* workspace, size_t workspace_bytes, void* stream);
gcn_status gcn_aggregate_workspace_size(const gcn_adj* A, int64_t F, int32_t prec, size_t* bytes);
gcn_status gcn_aggregate(const gcn_adj* A, int64_t F, int32_t prec, const void* X, int64_t ldx,
                         const float* bias, int32_t act, float dropout_p, int32_t training,
                         uint64_t seed, int32_t layer_id, uint64_t epoch, void* Y, int64_t ldy,
                         int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_layer_bwd: gradients of gcn_layer_fwd given dZ = dLoss/dZ (n x f_out,
 * ld_out, prec, already multiplied by the loss scale).  The chain rule through
 * one layer of Eq. (1) (Section "Graph Convolutions"), Z = A_hat (H W) + b,
 * with A_hat symmetric because G is undirected (Section "Introduction");
 * gradients stay multiplied by the dynamic loss scale of the O1/O2 levels
 * (Section "Background and Motivation") until the optimiser step:
 *   G_S      = A_hat^T dZ = A_hat dZ           (GS: n x f_out, ld_out, prec)
 *   dW       = H^T G_S                          (f_in x ld_out fp32; cols >= f_out set to 0)
 *   dbias    = column sums of dZ                (ld_out fp32, may be NULL)
 *   dZ_below = (G_S W^T) * [H > 0] / (1 - p_below)   if act_below == RELU
 *            =  G_S W^T                               if act_below == NONE
 *              (n x f_in, ld_in, prec; NULL skips it, e.g. for the first layer)
 *   dbias_below = column sums of dZ_below as stored (ld_in fp32, cols >=
 *              f_in set to 0; may be NULL, needs dZ_below): the bias
 *              gradient of the layer below, which its own gcn_layer_bwd call
 *              then need not compute (pass dbias = NULL there); summed by
 *              the workgroups that write dZ_below, without a pass of its own
 * The ReLU derivative at 0 is 0.  *overflow is set to 1 if any stored
 * element of GS, dW, dbias, dZ_below or dbias_below is not finite.  dW,
 * dbias and dbias_below are summed in a fixed order (run-to-run
 * deterministic).
 * With L->identity_input, dW = I^T G_S = G_S widened to fp32 (exactly what
 * the product with I gives); dZ_below must be NULL (GCN_ERR_INVALID_ARG
 * otherwise: there is nothing below an input layer).
 * ------------------------------------------------------------------------- */
gcn_status gcn_layer_bwd(const gcn_adj* A, const gcn_layer* L, int32_t prec,
                         const void* H, const void* W, const void* dZ,
                         int32_t act_below, float p_below,
                         float* dW, float* dbias, void* dZ_below, float* dbias_below, void* GS,
                         int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_layer_bwd_noalloc: gcn_layer_bwd without a workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid hipMalloc).  The call's scratch lives in a fixed
 * device array of GCN_NOALLOC_SCRATCH_BYTES bytes inside this library, one
 * per GPU, held until the process ends; the call itself allocates nothing.
 * Arguments, results and errors are those of gcn_layer_bwd (same kernels,
 * bit-identical outputs), plus GCN_ERR_CAPACITY when the call would need
 * more scratch than the array holds (gcn_layer_workspace_size() tells how
 * much it needs).  Every call on one GPU shares that GPU's array and leaves
 * its contents behind: calls that overlap on one GPU (several streams or
 * host threads) race, and the caller must serialise them.  The current HIP
 * device must be the device of `stream`.
 * ------------------------------------------------------------------------- */
#define GCN_NOALLOC_SCRATCH_BYTES (64u << 20)
gcn_status gcn_layer_bwd_noalloc(const gcn_adj* A, const gcn_layer* L, int32_t prec,
                                 const void* H, const void* W, const void* dZ,
                                 int32_t act_below, float p_below,
                                 float* dW, float* dbias, void* dZ_below, float* dbias_below, void* GS,
                                 int32_t* overflow, void* stream);

/* ---------------------------------------------------------------------------
 * gcn_loss: masked mean softmax cross-entropy over logits (n x C, ld, prec)
 * and labels (int32 in [0, C)); mask (uint8, NULL = every row) selects the
 * n_mask training rows (n_mask = number of nonzero mask entries, > 0).
 * This is the training loss of the semi-supervised vertex classification
 * that the paper scores by accuracy (Section "Experimental Setup", its
 * experiments subsection; the GCN of Section "Graph Convolutions" with the
 * original model's architecture), and the seed of
 * the backward pass: dlogits carries the loss scale S of the O1/O2 levels
 * (Section "Background and Motivation").
 *   *loss        = mean over masked rows of logsumexp(z_i) - z_i[y_i]   (fp32, unscaled)
 *   dlogits      = S * (softmax(z_i) - onehot(y_i)) / n_mask on masked rows, 0 elsewhere
 *   *n_correct   = masked rows whose arg-max (lowest index on ties) is y_i (may be NULL)
 *   dlogits_colsum = column sums of dlogits as stored (fp32 [ld], entries
 *                  [C, ld) set to 0; may be NULL): the output layer's bias
 *                  gradient, which its gcn_layer_bwd call then need not
 *                  compute (dbias = NULL there); summed by the loss kernel's
 *                  own workgroups, without a pass of its own over dlogits
 * S is *loss_scale (device float; NULL means 1).  Class padding [C, ld) is
 * excluded from the softmax.  The loss and the column sums are reduced in a
 * fixed order.
 * ------------------------------------------------------------------------- */
gcn_status gcn_loss_workspace_size(int64_t n, int64_t C, size_t* bytes);
gcn_status gcn_loss(int64_t n, int64_t C, int64_t ld, int32_t prec, const void* logits,
                    const int32_t* labels, const uint8_t* mask, int64_t n_mask,
                    const float* loss_scale, float* loss, void* dlogits, float* dlogits_colsum,
                    int32_t* n_correct, int32_t* overflow, void* workspace, size_t workspace_bytes,
                    void* stream);

/* ---------------------------------------------------------------------------
 * gcn_optimizer_step: one step of Adam on fp32 master weights with dynamic
 * loss scaling (Section "Background and Motivation", levels O1/O2), on
 * `count` flat parameters.  grad holds loss-scaled gradients.
 *   overflow = *overflow_flag != 0 or any grad element is not finite.
 *   overflow: no parameter changes; S = max(S * backoff, min_scale);
 *             good_steps = 0; skipped += 1.
 *   else:     g = grad / S; step += 1; m = b1 m + (1 - b1) g;
 *             v = b2 v + (1 - b2) g^2;
 *             master -= lr * (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps);
 *             working = master rounded to prec (may be NULL);
 *             good_steps += 1; if good_steps == interval:
 *             S = min(S * growth, max_scale), good_steps = 0.
 * *overflow_flag is cleared to 0 for the next step.  state and
 * overflow_flag are device memory; no host synchronisation happens.
 * ------------------------------------------------------------------------- */
gcn_status gcn_optimizer_step(int64_t count, float* master, const float* grad, float* m, float* v,
                              void* working, int32_t prec, const gcn_adam_config* cfg,
                              gcn_scaler* state, int32_t* overflow_flag, void* stream);

/* ===========================================================================
 * Other optimisation levels (Section "Background and Motivation"): O0 is the
 * fp32 path (prec = GCN_F32 everywhere), O2 the path above.  The two calls
 * below supply what O1 and O3 need beyond it.
 * ======================================================================== */

/* gcn_cast: dst = src converted to dst_prec, for a rows x cols block
 * (row-major, leading dimensions ld_src / ld_dst in elements; with rows == 1
 * the leading dimensions are ignored and cols may be any length, e.g. a
 * whole flat buffer).  16-bit results are rounded to nearest, ties to even;
 * widening is exact; src_prec == dst_prec copies.  This is the cast of the
 * O1 cast lists: GEMM-class operations run on 16-bit copies of fp32
 * operands, the loss on an fp32 copy of 16-bit logits.
 * *overflow is set to 1 when an output element is not finite (NULL ok).
 * Columns [cols, ld_dst) of dst are not written.
 * Errors: GCN_ERR_SHAPE (rows, cols <= 0, or rows > 1 with ld < cols),
 * GCN_ERR_ALIGNMENT (src/dst not 16-byte aligned, or rows > 1 with
 * ld_src or ld_dst not a multiple of 8), GCN_ERR_INVALID_ARG (NULL, or a
 * bad precision).  Asynchronous on `stream`. */
gcn_status gcn_cast(int64_t rows, int64_t cols, int32_t src_prec, const void* src, int64_t ld_src,
                    int32_t dst_prec, void* dst, int64_t ld_dst, int32_t* overflow, void* stream);

/* gcn_optimizer_step_half: one Adam step of level O3 ("full 16-bit"):
 * parameters w and moments m, v are `count` elements of prec (GCN_F16 or
 * GCN_BF16), with no fp32 master copy and no loss scale.  Each line is one
 * elementwise operation, evaluated in fp32 (one rounding per arithmetic
 * operation, no fused multiply-add) and rounded to prec by r(), with
 * t = state->step + 1 and c1 = 1 - b1^t, c2 = 1 - b2^t computed in double
 * and rounded to fp32:
 *   g = r(grad);  m = r(b1 * m + (1 - b1) * g);  v = r(b2 * v + ((1 - b2) * g) * g);
 *   mh = r(m / c1);  vh = r(v / c2);
 *   d = r(r(sqrt(vh)) + eps);  w = r(w - r((lr * mh) / d)).
 * Non-finite values are applied like any other (in binary16, eps = 1e-8
 * and small second moments round to 0, and the update becomes infinite:
 * the instability of level O3).  widened (NULL ok) receives w as fp32
 * (e.g. the bias operand of the layer epilogue).  state->step += 1 always;
 * state->skipped counts steps whose grad or *overflow_flag was non-finite;
 * state->scale is left as it is (the loss kernel should read 1).  Only
 * cfg's lr, beta1, beta2 and eps are used.  *overflow_flag is cleared.
 * Errors: GCN_ERR_SHAPE (count <= 0), GCN_ERR_INVALID_ARG (NULL required
 * pointer, prec not 16-bit, bad hyper-parameters).  Asynchronous. */
gcn_status gcn_optimizer_step_half(int64_t count, void* w, const float* grad, void* m, void* v,
                                   float* widened, int32_t prec, const gcn_adam_config* cfg,
                                   gcn_scaler* state, int32_t* overflow_flag, void* stream);

/* ===========================================================================
 * Link prediction: the graph auto-encoder of Section "Graph Auto-Encoders",
 * Eq. (2), A' = sigmoid(Z Z^T) with Z = GCN(A_hat, X), evaluated on sampled
 * vertex pairs (k = 0 .. K-1, K = n_pos + n_neg; pairs k < n_pos are
 * positives with label 1, the others negatives with label 0).  Vertex ids
 * are int32 in [0, n); Z is n x F (ld, prec).
 * ======================================================================== */

/* gcn_sample_pairs: the pairs of one training epoch.  Pair k takes the
 * Philox-4x64-10 block with key (seed, 0x50414952) and counter
 * (k, epoch, 0, 0), outputs w0, w1:
 *   k <  n_pos: e = w0 mod n_edges, pair = (edge_u[e], edge_v[e]);
 *   k >= n_pos: u = w0 mod n, v = (u + 1 + (w1 mod (n - 1))) mod n (v != u).
 * pair_u, pair_v: [n_pos + n_neg] int32 device outputs.  Requires n >= 2 and,
 * with n_pos > 0, n_edges >= 1.  Asynchronous. */
gcn_status gcn_sample_pairs(int64_t n, const int32_t* edge_u, const int32_t* edge_v, int64_t n_edges,
                            int64_t n_pos, int64_t n_neg, uint64_t seed, uint64_t epoch,
                            int32_t* pair_u, int32_t* pair_v, void* stream);

/* gcn_pair_loss: decoder scores and the logistic loss on pairs.
 *   s_k    = <Z[u_k], Z[v_k]>                       (fp32 accumulation)
 *   *loss  = mean_k softplus(s_k) - y_k s_k          (binary cross-entropy of sigmoid(s_k))
 *   g[k]   = S (sigmoid(s_k) - y_k) / K              (fp32; S = *loss_scale, NULL means 1)
 *   scores[k] = s_k (fp32, may be NULL)
 * The loss is summed in a fixed order.  A pair with an id outside [0, n) is
 * skipped (g = 0, score NaN) and sets *overflow, as does a non-finite score,
 * g or loss.  F <= 64 * (16 / element size).  workspace: at least
 * gcn_pair_loss_workspace_size() bytes. */
gcn_status gcn_pair_loss_workspace_size(int64_t n_pairs, size_t* bytes);
gcn_status gcn_pair_loss(int64_t n, int64_t F, int64_t ld, int32_t prec, const void* Z,
                         const int32_t* pair_u, const int32_t* pair_v, int64_t n_pos, int64_t n_neg,
                         const float* loss_scale, float* loss, float* scores, float* g,
                         int32_t* overflow, void* workspace, size_t workspace_bytes, void* stream);

/* gcn_pair_backward: dZ = d(sum_k g_k s_k)/dZ: row r sums g_k Z[v_k] over
 * the pairs with u_k = r and g_k Z[u_k] over the pairs with v_k = r, in
 * increasing k, rows that span several blocks of 64 pair endpoints being
 * summed block by block in order (run-to-run deterministic); rows in no
 * pair are 0.  dZ: n x F (ldz, prec; padding columns may be overwritten
 * with 0).  Pairs with an id outside [0, n) are skipped.  n_pairs <= 2^30.
 * *overflow is set if a stored element is not finite.  workspace:
 * gcn_pair_backward_workspace_size(n, n_pairs, F) bytes. */
gcn_status gcn_pair_backward_workspace_size(int64_t n, int64_t n_pairs, int64_t F, size_t* bytes);
gcn_status gcn_pair_backward(int64_t n, int64_t F, int64_t ld, int32_t prec, const void* Z,
                             const int32_t* pair_u, const int32_t* pair_v, int64_t n_pairs,
                             const float* g, void* dZ, int64_t ldz, int32_t* overflow,
                             void* workspace, size_t workspace_bytes, void* stream);

/* gcn_pair_metrics: the paper's link-prediction metrics (Section
 * "Experimental Setup": AUC and AP) of held-out pairs from their fp32
 * scores (scores[0 .. n_pos) positives, then n_neg negatives; all finite):
 *   auc_ap[0] = AUC = #{(i, j): s_i > s_j} + #{s_i == s_j} / 2, over P x N, divided by P N;
 *   auc_ap[1] = AP  = mean over positives i of #{pos with s >= s_i} / #{all with s >= s_i}.
 * Exact counts from one sort of the P + N scores (-0 and +0 are equal), a
 * count of the negatives before every sorted position and two binary
 * searches per positive: O((P + N) log(P + N)); fixed-order sums.  auc_ap is
 * a device array of 2 doubles.  n_pos + n_neg <= 2^31 - 1, else
 * GCN_ERR_SHAPE.  workspace: gcn_pair_metrics_workspace_size(), about
 * 32 (P + N) bytes. */
gcn_status gcn_pair_metrics_workspace_size(int64_t n_pos, int64_t n_neg, size_t* bytes);
gcn_status gcn_pair_metrics(const float* scores, int64_t n_pos, int64_t n_neg, double* auc_ap,
                            void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GCN_H */

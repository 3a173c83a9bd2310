// Neighbourhood aggregation Y = A_hat X for A_hat in CSR (the sparse
// product the paper could not run in half precision, Section "Reduced
// Precision Changes"), with the layer epilogue fused into the store.
//
// Work mapping (wave64):
//  * Light rows (<= heavy_threshold entries): a group of LPR lanes owns one
//    row; lane li of the group owns the 16-byte column slice li of the
//    feature row (8 x 16-bit or 4 x fp32), so one neighbour row of X is a
//    single coalesced LPR * 16-byte read.  Neighbours are walked 8 at a
//    time to keep several gathers in flight.  Rows are taken in the order of
//    the schedule's permutation (decreasing degree), so the groups of a
//    wave walk rows of similar length; rows of a single entry (isolated
//    vertices: the self-loop only) come last and go four per lane group
//    and round.  fp32 accumulation.
//  * Heavy rows (power-law hubs): cut by the schedule into pieces that never
//    cross a column range [q n / P, (q + 1) n / P) and hold at most
//    chunk_nnz entries; a lane group sums one piece, like a light row, into
//    an fp32 partial row.  The pieces of range q run on XCD q mod 8 (the
//    launch deals workgroup w to XCD w mod 8), so the L2 of each die only
//    caches rows of X from its own 1/P-th of the columns: on R-MAT graphs,
//    whose hubs' neighbours are spread over every column, this is what
//    makes the gathered rows of the hubs hit in L2.  Inside a range the
//    pieces run in order of their first column.  A fix-up adds the
//    partials of each row of several pieces in a fixed order (a lane group
//    per row in piece order; a workgroup per row of more than
//    GCN_FIX_BIG_PIECES pieces, contiguous runs per lane group, then the
//    runs in order) and applies the epilogue; a row of one piece is stored
//    by its piece.  No atomics: results are run-to-run identical.
#pragma once
#include "internal.h"

namespace gcn {

namespace {

template <typename IdxT>
struct SpmmParams {
  int64_t n;
  int64_t n_rows;               // rows to process: n_light with descriptors, else n
  int64_t n_single;             // the last n_single descriptors are rows of one entry
  const RowDesc* row_desc;      // light rows in schedule order (NULL: every row, index order)
  const IdxT* rowptr;
  const int32_t* colidx;
  const void* values;
  const float* dinv;
  const void* X;
  int64_t ldx;
  int64_t F;
  Epilogue epi;
};

template <typename T, bool HAS_VAL>
__device__ __forceinline__ float edge_value(const void* values, const float* dinv, float drow, int64_t e, int32_t c) {
  if (HAS_VAL) return to_f32<T>(reinterpret_cast<const T*>(values)[e]);
  return drow * dinv[c];
}

template <typename T>
__device__ __forceinline__ void fma_vec(float* acc, float v, uint4 raw) {
  float x[Vec<T>::N];
  unpack<T>(raw, x);
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) acc[i] = fmaf(v, x[i], acc[i]);
}

template <typename T, bool HAS_VAL, int U>
__device__ __forceinline__ void gather_block(float* acc, const T* __restrict__ X, int64_t ldx, const int32_t* __restrict__ colidx,
                                             const void* values, const float* dinv, float drow, int64_t e, int64_t stride) {
  int32_t c[U];
  uint4 x[U];
  float v[U];
#pragma unroll
  for (int u = 0; u < U; ++u) c[u] = colidx[e + u * stride];
#pragma unroll
  for (int u = 0; u < U; ++u) x[u] = ldg16(X + (int64_t)c[u] * ldx);
#pragma unroll
  for (int u = 0; u < U; ++u) v[u] = edge_value<T, HAS_VAL>(values, dinv, drow, e + u * stride, c[u]);
#pragma unroll
  for (int u = 0; u < U; ++u) fma_vec<T>(acc, v[u], x[u]);
}

// Entries e .. end - 1 (fewer than U) of a row in one round: every load is
// issued at an in-bounds index (past the end: the row's last entry again)
// and only the terms of real entries are added, in entry order, so the sum
// is the one that U single steps give.  The add is selected rather than
// scaled by zero, which a non-finite neighbour row would turn into NaN.
template <typename T, bool HAS_VAL, int U>
__device__ __forceinline__ void gather_tail(float* acc, const T* __restrict__ X, int64_t ldx, const int32_t* __restrict__ colidx,
                                            const void* values, const float* dinv, float drow, int64_t e, int64_t end) {
  int32_t c[U];
  uint4 x[U];
  float v[U];
#pragma unroll
  for (int u = 0; u < U; ++u) c[u] = colidx[e + u < end ? e + u : end - 1];
#pragma unroll
  for (int u = 0; u < U; ++u) x[u] = ldg16(X + (int64_t)c[u] * ldx);
#pragma unroll
  for (int u = 0; u < U; ++u) v[u] = edge_value<T, HAS_VAL>(values, dinv, drow, e + u < end ? e + u : end - 1, c[u]);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float xs[Vec<T>::N];
    unpack<T>(x[u], xs);
    const bool live = e + u < end;
#pragma unroll
    for (int i = 0; i < Vec<T>::N; ++i) acc[i] = live ? fmaf(v[u], xs[i], acc[i]) : acc[i];
  }
}

// Entries [e, end) of one row into acc: rounds of 8 gathers, then the tail.
template <typename T, int LPR, bool HAS_VAL>
__device__ __forceinline__ void row_sum(float* acc, const T* __restrict__ X, int64_t ldx,
                                        const int32_t* __restrict__ colidx, const void* values, const float* dinv,
                                        float drow, int64_t e, int64_t end) {
  for (; e + 8 <= end; e += 8) gather_block<T, HAS_VAL, 8>(acc, X, ldx, colidx, values, dinv, drow, e, 1);
  if constexpr (LPR * Vec<T>::N * (int)sizeof(T) <= 256) {
    // neighbour rows of at most 256 bytes: the walk is bound by dependent
    // load latency, so the last 1 .. 7 entries go in one round rather than
    // a round of 4 and single steps (up to 5 dependent rounds); the round
    // is sized to them (1, 4 or 8 gathers), so that rows of a single entry
    // -- the isolated vertices, 41 % of an R-MAT scale-21 graph -- do not
    // issue seven repeated gathers (R-MAT scale 21: F = 128 1.92 -> 1.86 ms,
    // F = 64 1.02 -> 0.99 ms, bit-identical)
    if (e < end) {
      if (end - e == 1) gather_block<T, HAS_VAL, 1>(acc, X, ldx, colidx, values, dinv, drow, e, 1);
      else if (end - e <= 4) gather_tail<T, HAS_VAL, 4>(acc, X, ldx, colidx, values, dinv, drow, e, end);
      else gather_tail<T, HAS_VAL, 8>(acc, X, ldx, colidx, values, dinv, drow, e, end);
    }
  } else {
    // wider rows are bound by the gathered bytes, which the in-bounds
    // repeats of a one-round tail would add to
    if (e + 4 <= end) {
      gather_block<T, HAS_VAL, 4>(acc, X, ldx, colidx, values, dinv, drow, e, 1);
      e += 4;
    }
    for (; e < end; ++e) gather_block<T, HAS_VAL, 1>(acc, X, ldx, colidx, values, dinv, drow, e, 1);
  }
}

__device__ __forceinline__ int64_t desc_beg(uint4 d) { return (int64_t)((uint64_t)d.x | ((uint64_t)d.y << 32)); }

// The bias of the workgroup's column block (LPR * VE columns from
// blockIdx.y * LPR * VE), staged in LDS once per workgroup, zeros where
// there is no bias: a lane then reads its columns from LDS at each row's
// store instead of waiting on eight global loads there (R-MAT scale 21,
// F = 128: bias + ReLU had cost 0.19 ms of a 1.65 ms call).  Every thread
// of the workgroup must call it.
template <typename T, int LPR>
__device__ __forceinline__ void stage_bias(const Epilogue& ep, float* sb) {
  constexpr int W = LPR * Vec<T>::N;
  const bool has = ep.mode == EPI_AGG && ep.bias;
  for (int i = threadIdx.x; i < W; i += 256) {
    const int64_t c = (int64_t)blockIdx.y * W + i;
    sb[i] = has && c < ep.cols ? ep.bias[c] : 0.f;
  }
  __syncthreads();
}

// Lane li's bias columns from the staged block (two 16-byte LDS reads for
// fp16/bf16, one for fp32; no branch, so the row loop keeps no extra
// scalar state).
template <typename T>
__device__ __forceinline__ void staged_bias(const float* sb, int li, float (&bv)[Vec<T>::N]) {
  constexpr int VE = Vec<T>::N;
  const float4* q = reinterpret_cast<const float4*>(sb) + li * (VE / 4);
#pragma unroll
  for (int j = 0; j < VE / 4; ++j) {
    const float4 t = q[j];
    bv[4 * j] = t.x; bv[4 * j + 1] = t.y; bv[4 * j + 2] = t.z; bv[4 * j + 3] = t.w;
  }
}

// Rows of one entry, SINGLE_BUNDLE of them (descriptors k0 .. k0 + cnt - 1)
// at once: descriptors, then column indices and values, then the gathers
// go out together, so the bundle costs the dependent loads of one row.
// Each sum is its single term (bit-identical to the row walk).  Eight rows
// (R-MAT scale 21 against four: F = 128 1.670 -> 1.642 ms, F = 64 0.852 ->
// 0.835 ms, no epilogue); their registers cost no occupancy, which the
// launch holds at four workgroups per compute unit anyway.
constexpr int SINGLE_BUNDLE = 8;

template <typename T, typename IdxT, bool HAS_VAL>
__device__ __forceinline__ void single_bundle(const SpmmParams<IdxT>& p, const T* __restrict__ X, int64_t col0,
                                              const float* sb, int li, int64_t k0, int64_t cnt) {
  constexpr int VE = Vec<T>::N;
  constexpr int B = SINGLE_BUNDLE;
  int64_t beg[B];
  int32_t row[B], c[B];
  float v[B], drow[B];
  uint4 x[B];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    const uint4 d = ldg16(p.row_desc + k0 + (k < cnt ? k : 0));
    beg[k] = desc_beg(d);
    row[k] = (int32_t)d.z;
  }
#pragma unroll
  for (int k = 0; k < B; ++k) c[k] = p.colidx[beg[k]];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    if (HAS_VAL) v[k] = to_f32<T>(reinterpret_cast<const T*>(p.values)[beg[k]]);
    else drow[k] = p.dinv[row[k]];
  }
  // dropout decisions drawn while the index loads are out
  int32_t keep[B];
  const bool draws = epi_draws(p.epi);
#pragma unroll
  for (int k = 0; k < B; ++k) keep[k] = draws ? (int32_t)dropout_bits<VE>(p.epi, row[k], col0) : -1;
#pragma unroll
  for (int k = 0; k < B; ++k) x[k] = ldg16(X + (int64_t)c[k] * p.ldx);
  if (!HAS_VAL) {
#pragma unroll
    for (int k = 0; k < B; ++k) v[k] = drow[k] * p.dinv[c[k]];
  }
#pragma unroll
  for (int k = 0; k < B; ++k) {
    if (k < cnt) {
      float acc[VE];
#pragma unroll
      for (int i = 0; i < VE; ++i) acc[i] = 0.f;
      fma_vec<T>(acc, v[k], x[k]);
      float bv[VE];
      staged_bias<T>(sb, li, bv);
      epi_store_vec_b<T>(p.epi, row[k], col0, acc, bv, keep[k]);
    }
  }
}

// Light rows for workgroup bx of nbx (bx: position among the light-row
// workgroups of the launch).  With the schedule's descriptors a lane group
// walks work units slot, slot + stride, ...: first the rows of several
// entries, loading the next row's descriptor before it gathers the current
// row, so that one dependent load (instead of the permutation and the row
// pointers) stands between two rows; then bundles of SINGLE_BUNDLE rows of
// one entry.
template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__device__ __forceinline__ void spmm_rows_body(const SpmmParams<IdxT>& p, const float* sb, int64_t bx, int64_t nbx) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int64_t col0 = ((int64_t)blockIdx.y * LPR + li) * VE;
  if (col0 >= p.F) return;
  const T* __restrict__ X = reinterpret_cast<const T*>(p.X) + col0;
  const int64_t stride = nbx * 4 * G;
  int64_t slot = (bx * 4 + wave) * G + g;
  if (p.row_desc) {
    const int64_t n_multi = p.n_rows - p.n_single;
    const int64_t units = n_multi + (p.n_single + SINGLE_BUNDLE - 1) / SINGLE_BUNDLE;
    uint4 d = slot < n_multi ? ldg16(p.row_desc + slot) : make_uint4(0, 0, 0, 0);
    while (slot < n_multi) {
      const int64_t beg = desc_beg(d);
      const int64_t row = (int64_t)(int32_t)d.z;
      const int64_t end = beg + (int64_t)(int32_t)d.w;
      const int64_t nslot = slot + stride;
      if (nslot < n_multi) d = ldg16(p.row_desc + nslot);
      const float drow = HAS_VAL ? 0.f : p.dinv[row];
      // the row's dropout decisions are drawn while its first loads are out
      const int32_t keep = epi_draws(p.epi) ? (int32_t)dropout_bits<VE>(p.epi, row, col0) : -1;
      float acc[VE];
#pragma unroll
      for (int i = 0; i < VE; ++i) acc[i] = 0.f;
      row_sum<T, LPR, HAS_VAL>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, beg, end);
      float bv[VE];
      staged_bias<T>(sb, li, bv);
      epi_store_vec_b<T>(p.epi, row, col0, acc, bv, keep);
      slot = nslot;
    }
    for (; slot < units; slot += stride) {
      const int64_t k0 = n_multi + (slot - n_multi) * SINGLE_BUNDLE;
      const int64_t cnt = p.n_rows - k0 < SINGLE_BUNDLE ? p.n_rows - k0 : SINGLE_BUNDLE;
      single_bundle<T, IdxT, HAS_VAL>(p, X, col0, sb, li, k0, cnt);
    }
    return;
  }
  // no schedule: every row, in index order
  for (; slot < p.n_rows; slot += stride) {
    const int64_t row = slot;
    const int64_t beg = (int64_t)p.rowptr[row], end = (int64_t)p.rowptr[row + 1];
    const float drow = HAS_VAL ? 0.f : p.dinv[row];
    float acc[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] = 0.f;
    row_sum<T, LPR, HAS_VAL>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, beg, end);
    float bv[VE];
    staged_bias<T>(sb, li, bv);
    epi_store_vec_b<T>(p.epi, row, col0, acc, bv);
  }
}

template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__global__ __launch_bounds__(256) void spmm_rows_kernel(SpmmParams<IdxT> p) {
  __shared__ __align__(16) float sb[LPR * Vec<T>::N];
  stage_bias<T, LPR>(p.epi, sb);
  spmm_rows_body<T, IdxT, LPR, HAS_VAL>(p, sb, blockIdx.x, gridDim.x);
}

struct PieceParams {
  const RowDesc* desc;          // [n_chunks] in launch (chunk_order) positions
  const int32_t* pos_of;        // [n_chunks] launch position of each piece
  const int32_t* heavy_rows;
  const int32_t* heavy_chunk_off;
  const int64_t* part_off;
  const int32_t* fix_rows;      // [n_fix] heavy-row slots of the rows of > 1 piece, big ones first
  int64_t n_fix, n_fix_big;
  int64_t n_chunks;
  int64_t parts;
  const int32_t* colidx;
  const void* values;
  const float* dinv;
  const void* X;
  int64_t ldx;
  int64_t F;
  int64_t ldp;                  // floats per partial row
  float* partials;              // [n_chunks][ldp], by launch position
  Epilogue epi;
};

// Launch position of the k-th piece of die x's list, or -1: with column
// ranges die x takes the pieces of ranges x, x + XCDS, ... in turn; without,
// there is one list.
__device__ __forceinline__ int64_t piece_at(const PieceParams& p, int64_t x, int64_t k) {
  if (p.parts <= 1) return k < p.n_chunks ? k : -1;
  for (int64_t q = x; q < p.parts; q += XCDS) {
    const int64_t len = p.part_off[q + 1] - p.part_off[q];
    if (k < len) return p.part_off[q] + k;
    k -= len;
  }
  return -1;
}

// Piece workgroup w of nw: its lane groups walk their die's list with the
// next piece's descriptor loaded ahead (nw is a multiple of XCDS when there
// are column ranges, so piece workgroup w runs on die w % XCDS).
template <typename T, int LPR, bool HAS_VAL>
__device__ __forceinline__ void spmm_piece_body(const PieceParams& p, const float* sb, int64_t w, int64_t nw) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int64_t col0 = ((int64_t)blockIdx.y * LPR + li) * VE;
  if (col0 >= p.F) return;
  const bool ranges = p.parts > 1;
  const int64_t x = ranges ? w % XCDS : 0;
  const int64_t j = ranges ? w / XCDS : w;
  const int64_t per = ranges ? nw / XCDS : nw;
  int64_t k = j * (4 * G) + wave * G + g;
  const int64_t stride = per * (4 * G);
  int64_t pos = piece_at(p, x, k);
  uint4 d = pos >= 0 ? ldg16(p.desc + pos) : make_uint4(0, 0, 0, 0);
  const T* __restrict__ X = reinterpret_cast<const T*>(p.X) + col0;
  while (pos >= 0) {
    const int64_t beg = desc_beg(d);
    const int64_t row = (int64_t)(int32_t)d.z;
    const int64_t end = beg + (int64_t)(d.w & 0x7fffffffu);
    const bool single = (d.w & 0x80000000u) != 0;
    k += stride;
    const int64_t npos = piece_at(p, x, k);
    if (npos >= 0) d = ldg16(p.desc + npos);
    const float drow = HAS_VAL ? 0.f : p.dinv[row];
    float acc[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] = 0.f;
    row_sum<T, LPR, HAS_VAL>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, beg, end);
    if (single) {
      // the row's only piece holds its whole sum: the epilogue stores it here
      float bv[VE];
      staged_bias<T>(sb, li, bv);
      epi_store_vec_b<T>(p.epi, row, col0, acc, bv);
    } else {
      float4* out = reinterpret_cast<float4*>(p.partials + pos * p.ldp + col0);
#pragma unroll
      for (int i = 0; i < VE / 4; ++i) out[i] = make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]);
    }
    pos = npos;
  }
}

// Pieces and light rows in one launch: workgroups [0, n_piece_wg) take the
// pieces, the rest walk the light rows.
template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__global__ __launch_bounds__(256) void spmm_main_kernel(SpmmParams<IdxT> p, PieceParams pp, int64_t n_piece_wg) {
  __shared__ __align__(16) float sb[LPR * Vec<T>::N];
  stage_bias<T, LPR>(p.epi, sb);
  const int64_t b = blockIdx.x;
  if (b < n_piece_wg) spmm_piece_body<T, LPR, HAS_VAL>(pp, sb, b, n_piece_wg);
  else spmm_rows_body<T, IdxT, LPR, HAS_VAL>(p, sb, b - n_piece_wg, (int64_t)gridDim.x - n_piece_wg);
}

// Partials of launch positions pos_of[a0 .. a1) (VE columns from col0) into
// acc, in that order: rounds of 4 rows in flight, the last 1 .. 3 in one
// round at clamped in-bounds positions whose surplus terms are dropped.
template <int VE>
__device__ __forceinline__ void add_partials(float* acc, const PieceParams& p, int64_t col0, int64_t a0, int64_t a1) {
  const float* __restrict__ part = p.partials + col0;
  int64_t c = a0;
  for (; c + 4 <= a1; c += 4) {
    int32_t q[4];
    float4 v[4][VE / 4];
#pragma unroll
    for (int u = 0; u < 4; ++u) q[u] = p.pos_of[c + u];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < VE / 4; ++i) v[u][i] = reinterpret_cast<const float4*>(part + (int64_t)q[u] * p.ldp)[i];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < VE / 4; ++i) {
        acc[4 * i] += v[u][i].x; acc[4 * i + 1] += v[u][i].y;
        acc[4 * i + 2] += v[u][i].z; acc[4 * i + 3] += v[u][i].w;
      }
  }
  if (c < a1) {
    int32_t q[3];
    float4 v[3][VE / 4];
#pragma unroll
    for (int u = 0; u < 3; ++u) q[u] = p.pos_of[c + u < a1 ? c + u : a1 - 1];
#pragma unroll
    for (int u = 0; u < 3; ++u)
#pragma unroll
      for (int i = 0; i < VE / 4; ++i) v[u][i] = reinterpret_cast<const float4*>(part + (int64_t)q[u] * p.ldp)[i];
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      const bool live = c + u < a1;
#pragma unroll
      for (int i = 0; i < VE / 4; ++i) {
        acc[4 * i] = live ? acc[4 * i] + v[u][i].x : acc[4 * i];
        acc[4 * i + 1] = live ? acc[4 * i + 1] + v[u][i].y : acc[4 * i + 1];
        acc[4 * i + 2] = live ? acc[4 * i + 2] + v[u][i].z : acc[4 * i + 2];
        acc[4 * i + 3] = live ? acc[4 * i + 3] + v[u][i].w : acc[4 * i + 3];
      }
    }
  }
}

// Fix-up of the heavy rows of more than one piece (fix_rows), the lane
// geometry that of the main kernel (lane li of a group owns VE columns):
//  * workgroups [0, n_fix_big): one row of more than GCN_FIX_BIG_PIECES
//    pieces each; lane group k of the workgroup adds the k-th contiguous run
//    of the row's pieces in piece order, the runs are then added in group
//    order through LDS and the epilogue stores the row;
//  * the other workgroups: one row per lane group, its partials added in
//    piece order.
template <typename T, int LPR>
__global__ __launch_bounds__(256) void spmm_fixup_kernel(PieceParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int NG = 4 * (64 / LPR);              // lane groups per workgroup
  const int gi = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int64_t col0 = ((int64_t)blockIdx.y * LPR + li) * VE;
  const bool live = col0 < p.F;
  const int64_t b = blockIdx.x;
  __shared__ __align__(16) float sb[LPR * VE];
  stage_bias<T, LPR>(p.epi, sb);
  float bv[VE];
  staged_bias<T>(sb, li, bv);
  float acc[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) acc[i] = 0.f;
  if (b < p.n_fix_big) {
    __shared__ float red[NG][LPR * VE];
    const int64_t h = p.fix_rows[b];
    const int64_t c0 = p.heavy_chunk_off[h], c1 = p.heavy_chunk_off[h + 1];
    const int64_t per = (c1 - c0 + NG - 1) / NG;
    const int64_t a0 = c0 + gi * per < c1 ? c0 + gi * per : c1;
    const int64_t a1 = a0 + per < c1 ? a0 + per : c1;
    if (live) add_partials<VE>(acc, p, col0, a0, a1);
#pragma unroll
    for (int i = 0; i < VE; ++i) red[gi][li * VE + i] = acc[i];
    __syncthreads();
    if (gi == 0 && live) {
#pragma unroll
      for (int i = 0; i < VE; ++i) acc[i] = red[0][li * VE + i];
      for (int k = 1; k < NG; ++k)
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[i] += red[k][li * VE + i];
      epi_store_vec_b<T>(p.epi, p.heavy_rows[h], col0, acc, bv);
    }
    return;
  }
  const int64_t slot = p.n_fix_big + (b - p.n_fix_big) * NG + gi;
  if (slot >= p.n_fix || !live) return;
  const int64_t h = p.fix_rows[slot];
  add_partials<VE>(acc, p, col0, p.heavy_chunk_off[h], p.heavy_chunk_off[h + 1]);
  epi_store_vec_b<T>(p.epi, p.heavy_rows[h], col0, acc, bv);
}

// Workgroups of each kind in one launch: enough for every lane group to
// walk several rows (or pieces) with its descriptor loads ahead, and about
// four rounds of workgroups over the chip's 256 compute units.
constexpr int64_t SPMM_WG_CAP = 8192;

// Resident workgroups of the main kernel per compute unit.  Five waves per
// SIMD put more gathers in flight, which evict the reused rows from L2
// (R-MAT scale 21 with bundles of four rows at 82-86 VGPRs: 1.707 against
// 1.674 ms at F = 128, 0.887 against 0.853 ms at F = 64, no epilogue), so
// the launch asks for dynamic LDS that leaves room for four 256-thread
// workgroups in the 160 KB of LDS of a gfx950 compute unit (the static LDS
// of the kernel is at most 2 KB).  With bundles of eight the fp16 variants
// need 108-122 VGPRs and hold four waves per SIMD by their registers too.
constexpr int SPMM_WG_PER_CU = 4;
constexpr unsigned SPMM_LDS_PER_CU = 160u * 1024u;
constexpr unsigned SPMM_OCCUPANCY_LDS = SPMM_LDS_PER_CU / SPMM_WG_PER_CU - 2048u;

template <typename T, typename IdxT, int LPR, bool HAS_VAL>
hipError_t launch_cfg(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                      float* partials, hipStream_t s) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int64_t colblocks = (F + LPR * VE - 1) / (LPR * VE);
  SpmmParams<IdxT> p;
  p.n = A.n;
  p.row_desc = A.row_perm ? A.row_desc : nullptr;
  p.n_rows = A.row_perm ? A.n_light : A.n;
  p.n_single = A.row_perm ? A.n_light_single : 0;
  p.rowptr = reinterpret_cast<const IdxT*>(A.rowptr);
  p.colidx = A.colidx;
  p.values = A.values;
  p.dinv = A.dinv;
  p.X = X; p.ldx = ldx; p.F = F; p.epi = epi;
  const int64_t per_wg = 4 * G;
  const int64_t units = p.n_rows - p.n_single + (p.n_single + SINGLE_BUNDLE - 1) / SINGLE_BUNDLE;
  int64_t lblocks = units > 0 ? std::min<int64_t>((units + per_wg - 1) / per_wg, SPMM_WG_CAP) : 0;
  hipError_t e = hipSuccess;
  if (A.n_heavy <= 0) {
    if (lblocks > 0) {
      hipLaunchKernelGGL((spmm_rows_kernel<T, IdxT, LPR, HAS_VAL>), dim3((unsigned)lblocks, (unsigned)colblocks),
                         dim3(256), 0, s, p);
      e = hipGetLastError();
    }
    return e;
  }
  PieceParams pp;
  pp.desc = A.piece_desc; pp.pos_of = A.piece_pos;
  pp.heavy_rows = A.heavy_rows; pp.heavy_chunk_off = A.heavy_chunk_off; pp.part_off = A.part_off;
  pp.fix_rows = A.fix_rows; pp.n_fix = A.n_fix; pp.n_fix_big = A.n_fix_big;
  pp.n_chunks = A.n_chunks; pp.parts = A.parts;
  pp.colidx = A.colidx; pp.values = A.values; pp.dinv = A.dinv;
  pp.X = X; pp.ldx = ldx; pp.F = F;
  pp.ldp = colblocks * LPR * VE;
  pp.partials = partials; pp.epi = epi;
  int64_t n_piece_wg;
  if (A.parts > 1) {
    n_piece_wg = XCDS * std::min<int64_t>((A.part_slots + per_wg - 1) / per_wg, SPMM_WG_CAP / XCDS);
    // keep the grid's x extent a multiple of XCDS, so that every column
    // block (grid y) deals its piece workgroups to the dies alike
    lblocks = (lblocks + XCDS - 1) / XCDS * XCDS;
  } else {
    n_piece_wg = std::min<int64_t>((A.n_chunks + per_wg - 1) / per_wg, SPMM_WG_CAP);
  }
  hipLaunchKernelGGL((spmm_main_kernel<T, IdxT, LPR, HAS_VAL>),
                     dim3((unsigned)(n_piece_wg + lblocks), (unsigned)colblocks), dim3(256), SPMM_OCCUPANCY_LDS, s,
                     p, pp, n_piece_wg);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (A.n_fix <= 0) return hipSuccess;               // every heavy row is one piece: all stored
  const int64_t fix_wg = A.n_fix_big + (A.n_fix - A.n_fix_big + per_wg - 1) / per_wg;
  hipLaunchKernelGGL((spmm_fixup_kernel<T, LPR>), dim3((unsigned)fix_wg, (unsigned)colblocks), dim3(256), 0, s, pp);
  return hipGetLastError();
}

// Neighbour rows wider than 256 bytes are gathered in 256-byte column
// blocks (grid y; the blocks of the first columns run first) once the
// gathered table exceeds 128 MiB: each pass then keeps twice as many reused
// rows in L2.  R-MAT scale 21, fp32, F = 128 (1 GiB table): 3.63 -> 3.30
// ms; Barabasi-Albert n = 200000, fp32, F = 256 (205 MB): 0.483 -> 0.471
// ms; a 67 MB table (R-MAT scale 17, fp16, F = 256) was 6 % slower split.
constexpr int64_t SPMM_ROW_BLOCK_BYTES = 256;
constexpr int64_t SPMM_SPLIT_TABLE_BYTES = (int64_t)128 << 20;

template <typename T, typename IdxT, bool HAS_VAL>
hipError_t launch_lpr(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                      float* partials, hipStream_t s) {
  constexpr int VE = Vec<T>::N;
  constexpr int64_t LPR_BLOCK = SPMM_ROW_BLOCK_BYTES / (VE * (int64_t)sizeof(T));   // 16 lanes
  int64_t nvec = (F + VE - 1) / VE;
  if (nvec > LPR_BLOCK && A.n * F * (int64_t)sizeof(T) > SPMM_SPLIT_TABLE_BYTES) nvec = LPR_BLOCK;
  if (nvec <= 1) return launch_cfg<T, IdxT, 1, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  if (nvec <= 2) return launch_cfg<T, IdxT, 2, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  if (nvec <= 4) return launch_cfg<T, IdxT, 4, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  if (nvec <= 8) return launch_cfg<T, IdxT, 8, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  if (nvec <= 16) return launch_cfg<T, IdxT, 16, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  if (nvec <= 32) return launch_cfg<T, IdxT, 32, HAS_VAL>(A, X, ldx, F, epi, partials, s);
  return launch_cfg<T, IdxT, 64, HAS_VAL>(A, X, ldx, F, epi, partials, s);
}

template <typename T>
hipError_t launch_t(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                    float* partials, hipStream_t s) {
  if (A.idx64)
    return A.values ? launch_lpr<T, int64_t, true>(A, X, ldx, F, epi, partials, s)
                    : launch_lpr<T, int64_t, false>(A, X, ldx, F, epi, partials, s);
  return A.values ? launch_lpr<T, int32_t, true>(A, X, ldx, F, epi, partials, s)
                  : launch_lpr<T, int32_t, false>(A, X, ldx, F, epi, partials, s);
}

}  // namespace
}  // namespace gcn

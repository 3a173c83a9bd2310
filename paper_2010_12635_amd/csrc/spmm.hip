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
//    wave walk rows of similar length.  fp32 accumulation.
//  * Heavy rows (power-law hubs): split into chunks of chunk_nnz entries;
//    one workgroup per chunk reduces its entries across 256/LPR lane groups
//    through LDS in a fixed order into an fp32 partial row.  Chunks are
//    launched in the schedule's order of their first column, so chunks of
//    different hubs that cover the same columns run at the same time and
//    find those rows of X in cache.  A fixup kernel
//    sums the partials of each heavy row in chunk order and applies the
//    epilogue.  No atomics: results are run-to-run identical.
#include "internal.h"

namespace gcn {

namespace {

template <typename IdxT>
struct SpmmParams {
  int64_t n;
  int64_t n_rows;               // rows to process: n_light with a permutation, else n
  const int32_t* row_perm;      // may be NULL
  const IdxT* rowptr;
  const int32_t* colidx;
  const void* values;
  const float* dinv;
  int64_t heavy_threshold;      // 0: no heavy split
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

// Light rows for workgroup bx of nbx (bx: position among the light-row
// workgroups of the launch).
template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__device__ __forceinline__ void spmm_rows_body(const SpmmParams<IdxT>& p, int64_t bx, int64_t nbx) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int64_t col0 = ((int64_t)blockIdx.y * LPR + li) * VE;
  if (col0 >= p.F) return;
  const T* __restrict__ X = reinterpret_cast<const T*>(p.X) + col0;
  // the grid is capped (at most 2^32 work-items per dispatch dimension):
  // a workgroup takes row slots bx, bx + nbx, ...
  for (int64_t slot = (bx * 4 + wave) * G + g; slot < p.n_rows; slot += nbx * 4 * G) {
    const int64_t row = p.row_perm ? (int64_t)p.row_perm[slot] : slot;
    const int64_t beg = (int64_t)p.rowptr[row], end = (int64_t)p.rowptr[row + 1];
    if (!p.row_perm && p.heavy_threshold > 0 && end - beg > p.heavy_threshold) continue;
    const float drow = HAS_VAL ? 0.f : p.dinv[row];
    float acc[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] = 0.f;
    int64_t e = beg;
    for (; e + 8 <= end; e += 8) gather_block<T, HAS_VAL, 8>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, 1);
    if constexpr (LPR * Vec<T>::N * (int)sizeof(T) <= 256) {
      // neighbour rows of at most 256 bytes: the walk is bound by dependent
      // load latency, so the last 1 .. 7 entries go in one round rather than
      // a round of 4 and single steps (up to 5 dependent rounds)
      if (e < end) gather_tail<T, HAS_VAL, 8>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, end);
    } else {
      // wider rows are bound by the gathered bytes, which the in-bounds
      // repeats of a one-round tail would add to
      if (e + 4 <= end) {
        gather_block<T, HAS_VAL, 4>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, 1);
        e += 4;
      }
      for (; e < end; ++e) gather_block<T, HAS_VAL, 1>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, 1);
    }
    epi_store_vec<T>(p.epi, row, col0, acc);
  }
}

template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__global__ __launch_bounds__(256) void spmm_rows_kernel(SpmmParams<IdxT> p) {
  spmm_rows_body<T, IdxT, LPR, HAS_VAL>(p, blockIdx.x, gridDim.x);
}

template <typename IdxT>
struct HeavyParams {
  const IdxT* rowptr;
  const int32_t* colidx;
  const void* values;
  const float* dinv;
  const int32_t* heavy_rows;
  const int32_t* heavy_chunk_off;
  const int32_t* chunk_heavy;
  const int32_t* chunk_order;   // launch order (may be NULL)
  int64_t chunk_nnz;
  int64_t n_chunks;
  const void* X;
  int64_t ldx;
  int64_t F;
  int64_t ldp;                  // floats per partial row
  float* partials;              // [n_chunks][ldp]
  Epilogue epi;
};

// One workgroup per (chunk, column block): launch position bx of the chunks.
template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__device__ __forceinline__ void spmm_heavy_body(const HeavyParams<IdxT>& p, int64_t bx) {
  constexpr int VE = Vec<T>::N;
  constexpr int NG = 256 / LPR;
  __shared__ float red[4 * LPR * VE];
  const int64_t chunk = p.chunk_order ? (int64_t)p.chunk_order[bx] : bx;
  const int g = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int64_t col0 = ((int64_t)blockIdx.y * LPR + li) * VE;
  const int32_t h = p.chunk_heavy[chunk];
  const int64_t row = p.heavy_rows[h];
  const int64_t rbeg = (int64_t)p.rowptr[row], rend = (int64_t)p.rowptr[row + 1];
  const int64_t cbeg = rbeg + (chunk - p.heavy_chunk_off[h]) * p.chunk_nnz;
  const int64_t cend = min(rend, cbeg + p.chunk_nnz);
  float acc[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) acc[i] = 0.f;
  if (col0 < p.F) {
    const T* __restrict__ X = reinterpret_cast<const T*>(p.X) + col0;
    const float drow = HAS_VAL ? 0.f : p.dinv[row];
    int64_t e = cbeg + g;
    for (; e + 7 * NG < cend; e += 8 * NG)
      gather_block<T, HAS_VAL, 8>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, NG);
    for (; e < cend; e += NG)
      gather_block<T, HAS_VAL, 1>(acc, X, p.ldx, p.colidx, p.values, p.dinv, drow, e, NG);
  }
  // reduce over the lane groups of a wave (xor butterfly over the group
  // bits of the lane id), then over the 4 waves through LDS in wave order
#pragma unroll
  for (int o = 32; o >= LPR; o >>= 1)
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] += __shfl_xor(acc[i], o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < LPR) {
#pragma unroll
    for (int i = 0; i < VE; ++i) red[(wave * LPR + lane) * VE + i] = acc[i];
  }
  __syncthreads();
  if (threadIdx.x < LPR && col0 < p.ldp) {
    float s[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) {
      s[i] = red[(0 * LPR + li) * VE + i] + red[(1 * LPR + li) * VE + i];
      s[i] += red[(2 * LPR + li) * VE + i];
      s[i] += red[(3 * LPR + li) * VE + i];
    }
    if (p.heavy_chunk_off[h + 1] - p.heavy_chunk_off[h] == 1) {
      // the row's only chunk holds its whole sum: the epilogue stores it here
      if (col0 < p.F) epi_store_vec<T>(p.epi, row, col0, s);
    } else {
      float* out = p.partials + chunk * p.ldp + col0;
#pragma unroll
      for (int i = 0; i < VE; ++i)
        if (col0 + i < p.ldp) out[i] = s[i];
    }
  }
}

template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__global__ __launch_bounds__(256) void spmm_heavy_chunk_kernel(HeavyParams<IdxT> p) {
  spmm_heavy_body<T, IdxT, LPR, HAS_VAL>(p, blockIdx.x);
}

// Heavy chunks and light rows in one launch: workgroups [0, n_heavy) take
// the chunks (longest work first), the rest walk the light rows, so that the
// hubs are reduced while the light rows run instead of in a launch of their
// own (on graphs with few hubs that launch leaves most of the chip idle).
// A workgroup is wholly one or the other, so the chunk body's barriers are
// reached by all its threads.
template <typename T, typename IdxT, int LPR, bool HAS_VAL>
__global__ __launch_bounds__(256) void spmm_fused_kernel(SpmmParams<IdxT> p, HeavyParams<IdxT> hp, int64_t n_heavy) {
  const int64_t b = blockIdx.x;
  if (b < n_heavy) spmm_heavy_body<T, IdxT, LPR, HAS_VAL>(hp, b);
  else spmm_rows_body<T, IdxT, LPR, HAS_VAL>(p, b - n_heavy, (int64_t)gridDim.x - n_heavy);
}

// One thread per (heavy row, column): fixed-order sum of the chunk partials
// (rows of a single chunk were stored by their chunk).
template <typename T, typename IdxT>
__global__ __launch_bounds__(256) void spmm_heavy_fixup_kernel(HeavyParams<IdxT> p) {
  const int64_t h = blockIdx.x;
  const int64_t col = (int64_t)blockIdx.y * 256 + threadIdx.x;
  if (col >= p.F) return;
  const int64_t row = p.heavy_rows[h];
  const int64_t c0 = p.heavy_chunk_off[h], c1 = p.heavy_chunk_off[h + 1];
  if (c1 - c0 == 1) return;
  float a = 0.f;
  for (int64_t c = c0; c < c1; ++c) a += p.partials[c * p.ldp + col];
  epi_store1<T>(p.epi, row, col, a);
}

// Chunk workgroups below which the chunks share the light rows' launch
// (8 per compute unit).
constexpr int64_t SPMM_FUSE_CHUNKS = 8 * 256;

template <typename T, typename IdxT, int LPR, bool HAS_VAL>
hipError_t launch_cfg(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                      float* partials, hipStream_t s) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int64_t colblocks = (F + LPR * VE - 1) / (LPR * VE);
  SpmmParams<IdxT> p;
  p.n = A.n;
  p.row_perm = A.row_perm;
  p.n_rows = A.row_perm ? A.n_light : A.n;
  p.rowptr = reinterpret_cast<const IdxT*>(A.rowptr);
  p.colidx = A.colidx;
  p.values = A.values;
  p.dinv = A.dinv;
  p.heavy_threshold = A.n_heavy > 0 ? A.heavy_threshold : 0;
  p.X = X; p.ldx = ldx; p.F = F; p.epi = epi;
  const int64_t rows_per_block = 4 * G;
  const int64_t lblocks = p.n_rows > 0 ? std::min<int64_t>((p.n_rows + rows_per_block - 1) / rows_per_block, 1 << 20) : 0;
  hipError_t e = hipSuccess;
  if (A.n_heavy <= 0) {
    if (lblocks > 0) {
      hipLaunchKernelGGL((spmm_rows_kernel<T, IdxT, LPR, HAS_VAL>), dim3((unsigned)lblocks, (unsigned)colblocks),
                         dim3(256), 0, s, p);
      e = hipGetLastError();
    }
    return e;
  }

  HeavyParams<IdxT> hp;
  hp.rowptr = p.rowptr; hp.colidx = A.colidx; hp.values = A.values; hp.dinv = A.dinv;
  hp.heavy_rows = A.heavy_rows; hp.heavy_chunk_off = A.heavy_chunk_off; hp.chunk_heavy = A.chunk_heavy;
  hp.chunk_order = A.chunk_order;
  hp.chunk_nnz = A.chunk_nnz; hp.n_chunks = A.n_chunks;
  hp.X = X; hp.ldx = ldx; hp.F = F;
  hp.ldp = colblocks * LPR * VE;
  hp.partials = partials; hp.epi = epi;
  if (lblocks > 0 && A.n_chunks * colblocks < SPMM_FUSE_CHUNKS) {
    // few chunks (fewer than 8 workgroups per compute unit on their own):
    // one launch with the light rows (grid below 2^32 work-items)
    dim3 gridf2((unsigned)(A.n_chunks + lblocks), (unsigned)colblocks);
    hipLaunchKernelGGL((spmm_fused_kernel<T, IdxT, LPR, HAS_VAL>), gridf2, dim3(256), 0, s, p, hp, (int64_t)A.n_chunks);
  } else {
    // many chunks fill the chip by themselves and keep their first-column
    // order to themselves (mixed with light rows: +2 % on R-MAT scale 21)
    if (lblocks > 0) {
      hipLaunchKernelGGL((spmm_rows_kernel<T, IdxT, LPR, HAS_VAL>), dim3((unsigned)lblocks, (unsigned)colblocks),
                         dim3(256), 0, s, p);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((spmm_heavy_chunk_kernel<T, IdxT, LPR, HAS_VAL>), dim3((unsigned)A.n_chunks, (unsigned)colblocks),
                       dim3(256), 0, s, hp);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (A.n_chunks == A.n_heavy) return hipSuccess;     // every heavy row is one chunk: all stored
  dim3 gridf((unsigned)A.n_heavy, (unsigned)((F + 255) / 256));
  hipLaunchKernelGGL((spmm_heavy_fixup_kernel<T, IdxT>), gridf, dim3(256), 0, s, hp);
  return hipGetLastError();
}

template <typename T, typename IdxT, bool HAS_VAL>
hipError_t launch_lpr(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                      float* partials, hipStream_t s) {
  constexpr int VE = Vec<T>::N;
  const int64_t nvec = (F + VE - 1) / VE;
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

int lpr_for(int prec, int64_t F) {
  const int VE = prec == 0 ? 4 : 8;
  const int64_t nvec = (F + VE - 1) / VE;
  int l = 1;
  while (l < nvec && l < 64) l <<= 1;
  return l;
}

}  // namespace

int64_t spmm_partials_floats(const CsrView& A, int prec, int64_t F) {
  if (A.n_heavy <= 0) return 0;
  const int VE = prec == 0 ? 4 : 8;
  const int lpr = lpr_for(prec, F);
  const int64_t colblocks = (F + (int64_t)lpr * VE - 1) / ((int64_t)lpr * VE);
  return A.n_chunks * colblocks * lpr * VE;
}

hipError_t spmm_launch(const CsrView& A, int prec, const void* X, int64_t ldx, int64_t F,
                       const Epilogue& epi, float* partials, hipStream_t s) {
  switch (prec) {
    case 0: return launch_t<float>(A, X, ldx, F, epi, partials, s);
    case 1: return launch_t<f16>(A, X, ldx, F, epi, partials, s);
    case 2: return launch_t<bf16>(A, X, ldx, F, epi, partials, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

// Dense-A_hat aggregation Y = epilogue(A_hat X) for A_hat stored as a dense
// n x n matrix (the paper's own storage: every tensor cast to dense,
// Section "Reduced Precision Changes").  With the feature width F <= 64 the
// product is bound by streaming A_hat from HBM (s * n^2 bytes against
// 2 * n^2 * F flops), so the kernel is built around that stream:
//
//  * Operand order.  MFMA 16x16 operands take, in lane l, 16 bytes of row
//    l % 16 at k-group l / 16.  In the tiled layout every 16-row x KC-column
//    piece (KC = 4 x 16 bytes of k) is one contiguous 1 KiB block in exactly
//    that lane order, and the four 16-row pieces of a 64-row block follow
//    each other, so each operand load is one contiguous 1 KiB and a wave's
//    k range is one contiguous stream (row-major rows give 16 short runs per
//    load, which measured far below the stream rate on MI355X).
//    X is transposed into the same tiled layout (Xt) before the product.
//  * A workgroup owns 64 rows and a 64-column block; its 8 waves split the
//    k range in 8 contiguous parts, each keeping its partial 64 x 64 tile in
//    MFMA accumulators, with a 3-deep register ring of loads in flight.
//  * The 8 partial tiles are summed through LDS in a fixed order (wave w
//    adds wave w + 4, then the four sums are added in wave order), then the
//    fused epilogue (bias, ReLU, dropout, cast, overflow flag) stores
//    16-byte vectors row by row.  No global partial sums, one launch.
#include "internal.h"
#include "xpose.h"

namespace gcn {

namespace {

constexpr int DA_BM = 64;     // rows per workgroup
constexpr int DA_BN = 64;     // columns per workgroup (column block of Xt)
constexpr int DA_WAVES = 8;   // waves per workgroup, one k range each

// Tiled offset (elements) of entry (i, j) of an R x K matrix in operand
// order: 64-row blocks, KC-column chunks, 16-row pieces of 1 KiB.
template <typename T>
__host__ __device__ __forceinline__ int64_t tiled_off(int64_t i, int64_t j, int64_t nc) {
  constexpr int VE = Vec<T>::N, KC = 4 * VE;
  return (((i / 64) * nc + j / KC) * 4 + (i % 64) / 16) * (16 * KC) + ((j % KC) / VE * 16 + i % 16) * VE + j % VE;
}
template <typename T> constexpr int tile_kc() { return 4 * Vec<T>::N; }

// Xt = tiled(X^T): X is n x F (ldx); Xt has Fp = ceil(F / 64) * 64 rows
// and kpad = nc * KC columns; entries outside F x n are zero.  Each thread
// turns one VE x VE block (VE vertices x VE features) around in registers:
// VE 16-byte row loads, a register transpose, VE 16-byte stores, each of
// VE consecutive vertices of one feature, i.e. one contiguous piece of the
// tiled layout.  A wave covers 64 features x XB_K vertices, a workgroup four
// waves along the vertices.  With colsum != NULL the kernel also sums each
// feature over the workgroup's vertices (fixed order: block rows, a xor
// butterfly over the wave's vertex blocks, then the four waves in order)
// and writes row blockIdx.x of colsum ([gridDim.x][F] floats).
template <typename T>
struct XpGeom {
  static constexpr int VE = Vec<T>::N;
  static constexpr int FB = 64 / VE;          // feature blocks per wave
  static constexpr int KB = 64 / FB;          // vertex blocks per wave
  static constexpr int WAVE_K = KB * VE;      // vertices per wave
  static constexpr int WG_K = 4 * WAVE_K;     // vertices per workgroup
};

template <typename T>
__global__ __launch_bounds__(256) void transpose_tiled_kernel(const T* __restrict__ X, int64_t ldx, int64_t n, int64_t F,
                                                              T* __restrict__ Xt, int64_t nc, float* __restrict__ colsum) {
  using G = XpGeom<T>;
  constexpr int VE = G::VE, KC = 4 * VE;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fb = lane % G::FB, kb = lane / G::FB;
  const int64_t f0 = (int64_t)blockIdx.y * 64 + fb * VE;
  const int64_t k0 = (int64_t)blockIdx.x * G::WG_K + wave * G::WAVE_K + kb * VE;
  const int64_t kpad = nc * KC;
  // all VE loads go out before any is used: rows >= n and feature blocks
  // >= F read row 0 / column 0 (in bounds) and are zeroed afterwards
  const int64_t nf = F - f0;
  const int vc = nf <= 0 ? 0 : nf >= VE ? VE : (int)nf;
  const T* colp = X + (vc > 0 ? f0 : 0);         // f0 + VE <= round_up(F, 8) <= ldx
  uint4 in[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) in[i] = ldg16(colp + (k0 + i < n ? k0 + i : 0) * ldx);
#pragma unroll
  for (int i = 0; i < VE; ++i) in[i] = keep_first<T>(in[i], k0 + i < n ? vc : 0);
  uint4 out[VE];
  transpose_block(in, out, T());
  if (k0 < kpad) {
#pragma unroll
    for (int j = 0; j < VE; ++j) stg16(Xt + tiled_off<T>(f0 + j, k0, nc), out[j]);
  }
  if (!colsum) return;
  __shared__ float red[4][64];
  float cs[VE];
#pragma unroll
  for (int j = 0; j < VE; ++j) {
    float v[VE];
    unpack<T>(out[j], v);
    float a = v[0];
#pragma unroll
    for (int i = 1; i < VE; ++i) a += v[i];
    cs[j] = a;
  }
#pragma unroll
  for (int off = G::FB; off < 64; off <<= 1)
#pragma unroll
    for (int j = 0; j < VE; ++j) cs[j] += __shfl_xor(cs[j], off);
  if (kb == 0) {
#pragma unroll
    for (int j = 0; j < VE; ++j) red[wave][fb * VE + j] = cs[j];
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int64_t f = (int64_t)blockIdx.y * 64 + threadIdx.x;
    float a = red[0][threadIdx.x] + red[1][threadIdx.x];
    a += red[2][threadIdx.x];
    a += red[3][threadIdx.x];
    if (f < F) colsum[(int64_t)blockIdx.x * F + f] = a;
  }
}

template <typename T> struct DaMfma;
template <> struct DaMfma<f16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
template <> struct DaMfma<bf16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct DaMfma<float> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

struct DaParams {
  const void* A; int64_t lda;     // dense A_hat, n x lda
  const void* Xt; int64_t ldt;    // Fp x ldt
  int64_t n;
  int64_t F;                      // logical output width
  Epilogue epi;
};

// One k chunk (4 lane groups x VE) of operand fragments.
template <int TN>
struct Frag {
  uint4 a[4];
  uint4 b[TN];
};

// In chunk c lane group g (= lane / 16) holds k = c * KC + g * VE + [0, VE)
// of A_hat and of Xt alike, so the MFMA sums over exactly the same k.
template <typename T, int TN, bool TILED>
__global__ __launch_bounds__(64 * DA_WAVES) void dense_agg_kernel(DaParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int KC = 4 * VE;                 // k per chunk: 32 (16-bit) / 16 (fp32)
  constexpr int PIECE = 16 * KC;             // elements of one 16-row piece (1 KiB)
  constexpr int LDR = DA_BN + 4;             // LDS row stride (floats)
  __shared__ float red[4][DA_BM * LDR];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t m0 = (int64_t)blockIdx.x * DA_BM;
  const int64_t c0 = (int64_t)blockIdx.y * DA_BN;
  const int64_t nc = (p.n + KC - 1) / KC;
  const T* __restrict__ A = reinterpret_cast<const T*>(p.A);
  const T* __restrict__ Xt = reinterpret_cast<const T*>(p.Xt);

  // Operand base pointers; fragment (chunk c, tile t) is at base + c * step + t * tstep.
  const T* abase[4];
  int64_t astep;
  if (TILED) {
    const T* blk = A + (int64_t)blockIdx.x * nc * 4 * PIECE + lane * VE;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) abase[tm] = blk + tm * PIECE;
    astep = 4 * PIECE;
  } else {
    // rows beyond n read row n-1 (their results are never stored)
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
      int64_t r = m0 + tm * 16 + (lane & 15);
      if (r >= p.n) r = p.n - 1;
      abase[tm] = A + r * p.lda + (lane >> 4) * VE;
    }
    astep = KC;
  }
  const T* bbase = Xt + (int64_t)blockIdx.y * nc * 4 * PIECE + lane * VE;

  const int64_t cb = nc * wave / DA_WAVES, ce = nc * (wave + 1) / DA_WAVES;
  const int64_t full_end = TILED ? ce : min(ce, p.n / KC);   // chunks needing no mask

  f32x4 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](Frag<TN>& f, int64_t c) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) f.a[tm] = ldg16(abase[tm] + c * astep);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) f.b[tn] = ldg16(bbase + c * 4 * PIECE + tn * PIECE);
  };
  auto compute = [&](const Frag<TN>& f) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = DaMfma<T>::run(f.a[tm], f.b[tn], acc[tm][tn]);
  };
  // keep the scheduler from moving MFMAs ahead of the loads issued before them
#define DA_FENCE() __builtin_amdgcn_sched_barrier(0)

  // full chunks: 4-deep ring of fragments (3 chunks in flight while computing)
  Frag<TN> f0, f1, f2, f3;
  int64_t c = cb;
  if (c + 3 <= full_end) {
    load(f0, c);
    load(f1, c + 1);
    load(f2, c + 2);
    DA_FENCE();
    for (; c + 7 <= full_end; c += 4) {
      load(f3, c + 3); DA_FENCE(); compute(f0); DA_FENCE();
      load(f0, c + 4); DA_FENCE(); compute(f1); DA_FENCE();
      load(f1, c + 5); DA_FENCE(); compute(f2); DA_FENCE();
      load(f2, c + 6); DA_FENCE(); compute(f3); DA_FENCE();
    }
    // drain: f0, f1, f2 hold chunks c, c+1, c+2
    compute(f0);
    compute(f1);
    compute(f2);
    c += 3;
  }
  for (; c < full_end; ++c) {
    load(f0, c);
    compute(f0);
  }
#undef DA_FENCE
  // row-major A_hat only: the chunk that straddles n (last wave): mask k >= n
  if (!TILED && c < ce) {
    const int64_t kl = c * KC + (lane >> 4) * VE;   // first k of this lane's vector
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) f0.b[tn] = ldg16(bbase + c * 4 * PIECE + tn * PIECE);   // Xt is zero-padded
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
      // a vector starting below n ends inside the row (lda >= n rounded up
      // to 8); one starting at or beyond n is not loaded at all
      f0.a[tm] = kl < p.n ? ldg16(abase[tm] + c * astep) : make_uint4(0, 0, 0, 0);
      T* e = reinterpret_cast<T*>(&f0.a[tm]);
#pragma unroll
      for (int j = 0; j < VE; ++j)
        if (kl + j >= p.n) e[j] = T(0);
    }
    compute(f0);
  }

  // partial tiles -> LDS (MFMA layout: lane holds rows 4*(lane/16)+v of
  // column lane%16).  Stage 1: waves 4..7 park their tiles, waves 0..3 add
  // them; stage 2: waves 0..3 park the sums.
  auto lds_at = [&](int w, int tm, int tn, int v) -> float& {
    return red[w][(tm * 16 + (lane >> 4) * 4 + v) * LDR + tn * 16 + (lane & 15)];
  };
  if (wave >= 4) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int v = 0; v < 4; ++v) lds_at(wave - 4, tm, tn, v) = acc[tm][tn][v];
  }
  __syncthreads();
  if (wave < 4) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[tm][tn][v] += lds_at(wave, tm, tn, v);
  }
  __syncthreads();
  if (wave < 4) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int v = 0; v < 4; ++v) lds_at(wave, tm, tn, v) = acc[tm][tn][v];
  }
  __syncthreads();

  // fixed-order sum of the 4 partials, fused epilogue, 16-byte stores
  constexpr int OV = Vec<T>::N;              // output elements per vector
  constexpr int VPR = DA_BN / OV;            // vectors per row of the block
  for (int idx = threadIdx.x; idx < DA_BM * VPR; idx += 64 * DA_WAVES) {
    const int r = idx / VPR, cv = idx % VPR;
    const int64_t row = m0 + r, col = c0 + cv * OV;
    if (row >= p.n || col >= p.F || cv * OV >= TN * 16) continue;
    float v[OV];
#pragma unroll
    for (int j = 0; j < OV; ++j) {
      const int cc = cv * OV + j;
      v[j] = red[0][r * LDR + cc] + red[1][r * LDR + cc];
      v[j] += red[2][r * LDR + cc];
      v[j] += red[3][r * LDR + cc];
    }
    epi_store_vec<T>(p.epi, row, col, v);
  }
}

int64_t xt_elems(int prec, int64_t n, int64_t F) {
  const int64_t kc = prec == 0 ? 16 : 32;
  const int64_t nc = (n + kc - 1) / kc;
  return ((F + 63) / 64) * 64 * nc * kc;
}

template <typename T>
hipError_t launch_t(const void* A, int64_t lda, bool tiled, int64_t n, const void* X, int64_t ldx, int64_t F,
                    const Epilogue& epi, void* ws, float* colsum, hipStream_t s) {
  constexpr int KC = tile_kc<T>();
  const int64_t nc = (n + KC - 1) / KC;
  const int64_t fblocks = (F + 63) / 64;
  T* Xt = reinterpret_cast<T*>(ws);
  dim3 tg((unsigned)((nc * KC + XpGeom<T>::WG_K - 1) / XpGeom<T>::WG_K), (unsigned)fblocks);
  hipLaunchKernelGGL(transpose_tiled_kernel<T>, tg, dim3(256), 0, s, reinterpret_cast<const T*>(X), ldx, n, F, Xt, nc,
                     colsum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DaParams p;
  p.A = A; p.lda = lda; p.Xt = Xt; p.ldt = 0; p.n = n; p.F = F; p.epi = epi;
  dim3 grid((unsigned)((n + DA_BM - 1) / DA_BM), (unsigned)fblocks);
  const int tn = F > 48 ? 4 : (int)((F + 15) / 16);
  const dim3 blk(64 * DA_WAVES);
#define DA_LAUNCH(TN_)                                                                          \
  if (tiled) hipLaunchKernelGGL((dense_agg_kernel<T, TN_, true>), grid, blk, 0, s, p);          \
  else hipLaunchKernelGGL((dense_agg_kernel<T, TN_, false>), grid, blk, 0, s, p);
  switch (tn) {
    case 1: DA_LAUNCH(1) break;
    case 2: DA_LAUNCH(2) break;
    case 3: DA_LAUNCH(3) break;
    default: DA_LAUNCH(4) break;
  }
#undef DA_LAUNCH
  return hipGetLastError();
}

// Dense form of a CSR A_hat: one wave per row scatters its entries.
template <typename T, typename IdxT, bool TILED>
__global__ __launch_bounds__(256) void densify_kernel(int64_t n, const IdxT* __restrict__ rowptr,
                                                      const int32_t* __restrict__ colidx, const T* __restrict__ values,
                                                      const float* __restrict__ dinv, T* __restrict__ dense,
                                                      int64_t ld, int64_t nc) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += (int64_t)gridDim.x * 4) {
    const float dr = values ? 0.f : dinv[r];
    for (int64_t k = (int64_t)rowptr[r] + lane; k < (int64_t)rowptr[r + 1]; k += 64) {
      const int32_t c = colidx[k];
      const T v = values ? values[k] : from_f32<T>(dr * dinv[c]);
      dense[TILED ? tiled_off<T>(r, c, nc) : r * ld + c] = v;
    }
  }
}

template <typename T>
hipError_t densify_t(const CsrView& A, bool tiled, void* dense, int64_t ld, hipStream_t s) {
  constexpr int KC = tile_kc<T>();
  const int64_t nc = (A.n + KC - 1) / KC;
  const size_t bytes = tiled ? (size_t)((A.n + 63) / 64) * 64 * nc * KC * sizeof(T) : (size_t)A.n * ld * sizeof(T);
  hipError_t e = fill_zero(dense, bytes, s);
  if (e != hipSuccess) return e;
  const dim3 g((unsigned)std::min<int64_t>((A.n + 3) / 4, 1 << 20));   // the kernel loops over rows
  const T* vals = reinterpret_cast<const T*>(A.values);
  T* d = reinterpret_cast<T*>(dense);
  if (A.idx64) {
    const int64_t* rp = reinterpret_cast<const int64_t*>(A.rowptr);
    if (tiled) hipLaunchKernelGGL((densify_kernel<T, int64_t, true>), g, dim3(256), 0, s, A.n, rp, A.colidx, vals, A.dinv, d, ld, nc);
    else hipLaunchKernelGGL((densify_kernel<T, int64_t, false>), g, dim3(256), 0, s, A.n, rp, A.colidx, vals, A.dinv, d, ld, nc);
  } else {
    const int32_t* rp = reinterpret_cast<const int32_t*>(A.rowptr);
    if (tiled) hipLaunchKernelGGL((densify_kernel<T, int32_t, true>), g, dim3(256), 0, s, A.n, rp, A.colidx, vals, A.dinv, d, ld, nc);
    else hipLaunchKernelGGL((densify_kernel<T, int32_t, false>), g, dim3(256), 0, s, A.n, rp, A.colidx, vals, A.dinv, d, ld, nc);
  }
  return hipGetLastError();
}

}  // namespace

size_t dense_agg_workspace_bytes(int prec, int64_t n, int64_t F) {
  return (size_t)xt_elems(prec, n, F) * (prec == 0 ? 4 : 2);
}

int64_t dense_tiled_elems(int prec, int64_t n) {
  const int64_t kc = prec == 0 ? 16 : 32;
  return ((n + 63) / 64) * 64 * ((n + kc - 1) / kc) * kc;
}

hipError_t dense_agg_launch(int prec, const void* A, int64_t lda, bool tiled, int64_t n, const void* X, int64_t ldx,
                            int64_t F, const Epilogue& epi, void* ws, float* colsum, hipStream_t s) {
  switch (prec) {
    case 0: return launch_t<float>(A, lda, tiled, n, X, ldx, F, epi, ws, colsum, s);
    case 1: return launch_t<f16>(A, lda, tiled, n, X, ldx, F, epi, ws, colsum, s);
    case 2: return launch_t<bf16>(A, lda, tiled, n, X, ldx, F, epi, ws, colsum, s);
  }
  return hipErrorInvalidValue;
}

int64_t dense_agg_colsum_rows(int prec, int64_t n) {
  const int64_t kc = prec == 0 ? 16 : 32;
  const int64_t wg_k = prec == 0 ? XpGeom<float>::WG_K : XpGeom<f16>::WG_K;
  return ((n + kc - 1) / kc * kc + wg_k - 1) / wg_k;
}

hipError_t densify_launch(const CsrView& A, int prec, bool tiled, void* dense, int64_t ld, hipStream_t s) {
  switch (prec) {
    case 0: return densify_t<float>(A, tiled, dense, ld, s);
    case 1: return densify_t<f16>(A, tiled, dense, ld, s);
    case 2: return densify_t<bf16>(A, tiled, dense, ld, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

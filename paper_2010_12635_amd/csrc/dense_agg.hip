// Dense-A_hat aggregation Y = epilogue(A_hat X) for A_hat stored as a dense
// n x n matrix (the paper's own storage: every tensor cast to dense,
// Section "Reduced Precision Changes").  With the feature width F <= 64 the
// product is bound by streaming A_hat from HBM (s * n^2 bytes against
// 2 * n^2 * F flops), so the kernel is built around that stream:
//
//  * X is first transposed into Xt (Fp x ldt, Fp = F rounded up to 16,
//    zero-padded), so that both MFMA operands are k-contiguous and every
//    operand fragment is one 16-byte global load: A_hat rows come straight
//    from HBM into registers, Xt (a few MB) is served from L2.
//  * A workgroup owns 64 rows and all (up to 64) columns; its 8 waves split
//    the k range in 8 contiguous parts, each keeping its partial 64 x Fp
//    tile in MFMA accumulators, with a 3-deep register ring of loads in
//    flight.  No global partial sums, one launch.
//  * The 8 partial tiles are summed through LDS in a fixed order (wave w
//    adds wave w + 4, then the four sums are added in wave order), then the
//    fused epilogue (bias, ReLU, dropout, cast, overflow flag) stores
//    16-byte vectors row by row.
#include "internal.h"

namespace gcn {

namespace {

constexpr int DA_BM = 64;     // rows per workgroup
constexpr int DA_BN = 64;     // columns per workgroup (column block of Xt)
constexpr int DA_WAVES = 8;   // waves per workgroup, one k range each

// Xt[f][k] = X[k][f] for f < F, k < n; zero for F <= f < Fp or n <= k < ldt.
template <typename T>
__global__ __launch_bounds__(256) void transpose_pad_kernel(const T* __restrict__ X, int64_t ldx, int64_t n, int64_t F,
                                                            T* __restrict__ Xt, int64_t ldt, int64_t Fp) {
  __shared__ T tile[64][65];
  const int64_t k0 = (int64_t)blockIdx.x * 64, f0 = (int64_t)blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;   // 64 x 4
  for (int r = ty; r < 64; r += 4) {
    const int64_t k = k0 + r, f = f0 + tx;
    tile[r][tx] = (k < n && f < F) ? X[k * ldx + f] : T(0);
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {
    const int64_t f = f0 + r, k = k0 + tx;
    if (f < Fp && k < ldt) Xt[f * ldt + k] = tile[tx][r];
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

template <typename T, int TN>
__global__ __launch_bounds__(64 * DA_WAVES) void dense_agg_kernel(DaParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int KC = 4 * VE;                 // k per chunk: 32 (16-bit) / 16 (fp32)
  constexpr int LDR = DA_BN + 4;             // LDS row stride (floats)
  __shared__ float red[4][DA_BM * LDR];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * DA_BM;
  const int64_t c0 = (int64_t)blockIdx.y * DA_BN;
  const T* __restrict__ A = reinterpret_cast<const T*>(p.A);
  const T* __restrict__ Xt = reinterpret_cast<const T*>(p.Xt);

  // rows beyond n read row n-1 (their results are never stored)
  const T* arow[4];
#pragma unroll
  for (int tm = 0; tm < 4; ++tm) {
    int64_t r = m0 + tm * 16 + (lane & 15);
    if (r >= p.n) r = p.n - 1;
    arow[tm] = A + r * p.lda + (lane >> 4) * VE;
  }
  const T* brow[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) brow[tn] = Xt + (c0 + tn * 16 + (lane & 15)) * p.ldt + (lane >> 4) * VE;

  const int64_t chunks = (p.n + KC - 1) / KC;
  const int64_t cb = chunks * wave / DA_WAVES, ce = chunks * (wave + 1) / DA_WAVES;
  const int64_t full_end = min(ce, p.n / KC);   // chunks entirely below n

  f32x4 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](Frag<TN>& f, int64_t c) {
    const int64_t k = c * KC;
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) f.a[tm] = ldg16(arow[tm] + k);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) f.b[tn] = ldg16(brow[tn] + k);
  };
  auto compute = [&](const Frag<TN>& f) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = DaMfma<T>::run(f.a[tm], f.b[tn], acc[tm][tn]);
  };

  // full chunks: 4-deep ring of fragments (3 loads in flight while computing)
  Frag<TN> f0, f1, f2, f3;
  int64_t c = cb;
  if (c + 3 <= full_end) {
    load(f0, c);
    load(f1, c + 1);
    load(f2, c + 2);
    for (; c + 7 <= full_end; c += 4) {
      load(f3, c + 3); compute(f0);
      load(f0, c + 4); compute(f1);
      load(f1, c + 5); compute(f2);
      load(f2, c + 6); compute(f3);
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
  // the chunk that straddles n (only in the last wave's range): mask k >= n
  if (c < ce) {
    const int64_t k = c * KC;
    const int64_t kl = k + (lane >> 4) * VE;   // first k of this lane's vector
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) f0.b[tn] = ldg16(brow[tn] + k);   // Xt is zero-padded to ldt
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
      // a vector starting below n ends inside the row (lda >= n rounded up to 8);
      // one starting at or beyond n is not loaded at all
      f0.a[tm] = kl < p.n ? ldg16(arow[tm] + k) : make_uint4(0, 0, 0, 0);
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

template <typename T>
hipError_t launch_t(const void* A, int64_t lda, int64_t n, const void* X, int64_t ldx, int64_t F,
                    const Epilogue& epi, void* ws, hipStream_t s) {
  const int64_t Fp = F <= DA_BN ? (F + 15) / 16 * 16 : (F + DA_BN - 1) / DA_BN * DA_BN;
  const int64_t ldt = (n + 63) / 64 * 64;
  T* Xt = reinterpret_cast<T*>(ws);
  dim3 tg((unsigned)(ldt / 64), (unsigned)((Fp + 63) / 64));
  hipLaunchKernelGGL(transpose_pad_kernel<T>, tg, dim3(256), 0, s, reinterpret_cast<const T*>(X), ldx, n, F, Xt,
                     ldt, Fp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DaParams p;
  p.A = A; p.lda = lda; p.Xt = Xt; p.ldt = ldt; p.n = n; p.F = F; p.epi = epi;
  dim3 grid((unsigned)((n + DA_BM - 1) / DA_BM), (unsigned)((Fp + DA_BN - 1) / DA_BN));
  const int tn = Fp >= 64 ? 4 : (int)(Fp / 16);
  switch (tn) {
    case 1: hipLaunchKernelGGL((dense_agg_kernel<T, 1>), grid, dim3(64 * DA_WAVES), 0, s, p); break;
    case 2: hipLaunchKernelGGL((dense_agg_kernel<T, 2>), grid, dim3(64 * DA_WAVES), 0, s, p); break;
    case 3: hipLaunchKernelGGL((dense_agg_kernel<T, 3>), grid, dim3(64 * DA_WAVES), 0, s, p); break;
    default: hipLaunchKernelGGL((dense_agg_kernel<T, 4>), grid, dim3(64 * DA_WAVES), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace

size_t dense_agg_workspace_bytes(int prec, int64_t n, int64_t F) {
  const int64_t Fp = F <= DA_BN ? (F + 15) / 16 * 16 : (F + DA_BN - 1) / DA_BN * DA_BN;
  const int64_t ldt = (n + 63) / 64 * 64;
  return (size_t)Fp * (size_t)ldt * (prec == 0 ? 4 : 2);
}

hipError_t dense_agg_launch(int prec, const void* A, int64_t lda, int64_t n, const void* X, int64_t ldx, int64_t F,
                            const Epilogue& epi, void* ws, hipStream_t s) {
  switch (prec) {
    case 0: return launch_t<float>(A, lda, n, X, ldx, F, epi, ws, s);
    case 1: return launch_t<f16>(A, lda, n, X, ldx, F, epi, ws, s);
    case 2: return launch_t<bf16>(A, lda, n, X, ldx, F, epi, ws, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

// Dense contractions of the GCN layer on gfx950 matrix cores:
//   S = H W, dH = G_S W^T (epilogue: ReLU / dropout derivative), dW = H^T G_S
//   (split over the vertex dimension), and the dense-A_hat aggregation.
//
// One templated kernel covers every operand orientation.  Tiles of A and B
// are staged through LDS in "k-contiguous" form (each row of the LDS tile
// holds consecutive k of one output row / column), so that every MFMA
// operand fragment is one 16-byte LDS read:
//   16-bit storage: v_mfma_f32_16x16x32_{f16,bf16}, 8 k per lane;
//   fp32 storage:   four v_mfma_f32_16x16x4_f32, 4 k per lane.
// Within an MFMA, lane l supplies row (l % 16) of A and column (l % 16) of
// B; which k a lane group supplies only has to agree between A and B, so
// the fp32 path assigns k = 4 * (l / 16) + step to keep 16-byte reads.
// Operands stored with k as the slow axis (H^T, G_S in dW; W in S = H W)
// are transposed while being written to LDS.
#include "internal.h"

#include <algorithm>

namespace gcn {

namespace {

template <typename T> struct Mfma;

template <> struct Mfma<f16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                   __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mfma<bf16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

template <typename T> constexpr int k_tile() { return 8 * Vec<T>::N; }   // 64 (16-bit) / 32 (fp32)

struct GemmParams {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  int64_t M, N, K;
  int64_t k_per_split;
  int splits;
  float* partials;
  Epilogue epi;
};

// Loads a (R x BK) operand tile (R = output rows or columns) from global
// memory into registers, then writes it k-contiguous into LDS.
//   KC:  element (r, k) at base[r * ld + k]
//   !KC: element (r, k) at base[k * ld + r]
// Elements outside [0, Rtot) x [k0, kend) are zero.  16-byte loads stay in
// bounds because ld >= round_up(width, 8) and ld % 8 == 0.
template <typename T, bool KC, int R, int BK>
struct TileLoader {
  static constexpr int VE = Vec<T>::N;
  static constexpr int LDK = BK + VE;
  static constexpr int NVEC = R * BK / VE;
  static constexpr int PER = (NVEC + 255) / 256;
  uint4 reg[PER];

  __device__ __forceinline__ void load(const T* __restrict__ base, int64_t ld, int64_t r0, int64_t Rtot,
                                       int64_t k0, int64_t kend, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = tid + i * 256;
      uint4 x = make_uint4(0, 0, 0, 0);
      if (v < NVEC) {
        if (KC) {
          const int r = v / (BK / VE), kv = v % (BK / VE);
          const int64_t gr = r0 + r, gk = k0 + (int64_t)kv * VE;
          if (gr < Rtot && gk < kend) {
            x = ldg16(base + gr * ld + gk);
            if (gk + VE > kend) {
              T* e = reinterpret_cast<T*>(&x);
#pragma unroll
              for (int j = 0; j < VE; ++j)
                if (gk + j >= kend) e[j] = T(0);
            }
          }
        } else {
          const int k = v / (R / VE), rv = v % (R / VE);
          const int64_t gk = k0 + k, gr = r0 + (int64_t)rv * VE;
          if (gk < kend && gr < Rtot) {
            x = ldg16(base + gk * ld + gr);
            if (gr + VE > Rtot) {
              T* e = reinterpret_cast<T*>(&x);
#pragma unroll
              for (int j = 0; j < VE; ++j)
                if (gr + j >= Rtot) e[j] = T(0);
            }
          }
        }
      }
      reg[i] = x;
    }
  }

  __device__ __forceinline__ void store(T* __restrict__ s, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = tid + i * 256;
      if (v < NVEC) {
        if (KC) {
          const int r = v / (BK / VE), kv = v % (BK / VE);
          *reinterpret_cast<uint4*>(s + r * LDK + kv * VE) = reg[i];
        } else {
          const int k = v / (R / VE), rv = v % (R / VE);
          const T* e = reinterpret_cast<const T*>(&reg[i]);
#pragma unroll
          for (int j = 0; j < VE; ++j) s[(rv * VE + j) * LDK + k] = e[j];
        }
      }
    }
  }
};

template <typename T, bool AKC, bool BKC, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int BK = k_tile<T>();
  constexpr int LDK = BK + VE;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  static_assert(WM * WN == 4, "four waves per workgroup");
  static_assert(TM >= 1 && TN >= 1, "wave tile at least 16 x 16");

  __shared__ __align__(16) T sA[2][BM * LDK];
  __shared__ __align__(16) T sB[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int64_t m0 = (int64_t)blockIdx.x * BM, n0 = (int64_t)blockIdx.y * BN;
  const int64_t kb = (int64_t)blockIdx.z * p.k_per_split;
  const int64_t ke = min(p.K, kb + p.k_per_split);
  const T* __restrict__ A = reinterpret_cast<const T*>(p.A);
  const T* __restrict__ B = reinterpret_cast<const T*>(p.B);

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  TileLoader<T, AKC, BM, BK> la;
  TileLoader<T, BKC, BN, BK> lb;
  const int64_t nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
  if (nk > 0) {
    la.load(A, p.lda, m0, p.M, kb, ke, tid);
    lb.load(B, p.ldb, n0, p.N, kb, ke, tid);
  }
  for (int64_t t = 0; t < nk; ++t) {
    const int st = (int)(t & 1);
    la.store(sA[st], tid);
    lb.store(sB[st], tid);
    __syncthreads();
    if (t + 1 < nk) {
      const int64_t k0 = kb + (t + 1) * BK;
      la.load(A, p.lda, m0, p.M, k0, ke, tid);
      lb.load(B, p.ldb, n0, p.N, k0, ke, tid);
    }
    const T* a_s = sA[st] + (wm * WTM + (lane & 15)) * LDK + (lane >> 4) * VE;
    const T* b_s = sB[st] + (wn * WTN + (lane & 15)) * LDK + (lane >> 4) * VE;
#pragma unroll
    for (int ks = 0; ks < BK / (4 * VE); ++ks) {
      uint4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const uint4*>(a_s + i * 16 * LDK + ks * 4 * VE);
#pragma unroll
      for (int j = 0; j < TN; ++j) bf[j] = *reinterpret_cast<const uint4*>(b_s + j * 16 * LDK + ks * 4 * VE);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = Mfma<T>::run(af[i], bf[j], acc[i][j]);
    }
  }

  // Accumulator layout of a 16 x 16 MFMA tile: lane l holds rows
  // 4 * (l / 16) + v, v = 0..3, of column l % 16.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = m0 + wm * WTM + i * 16 + (lane >> 4) * 4 + v;
        const int64_t col = n0 + wn * WTN + j * 16 + (lane & 15);
        if (row < p.M && col < p.N) {
          if (p.partials)
            p.partials[((int64_t)blockIdx.z * p.M + row) * p.N + col] = acc[i][j][v];
          else
            epi_store1<T>(p.epi, row, col, acc[i][j][v]);
        }
      }
}

template <typename T, bool AKC, bool BKC>
hipError_t launch_layout(const GemmParams& p, hipStream_t s) {
  const dim3 block(256);
  const int64_t BM = 128;
  if (p.N <= 16) {
    dim3 grid((unsigned)((p.M + BM - 1) / BM), (unsigned)((p.N + 15) / 16), (unsigned)p.splits);
    hipLaunchKernelGGL((gemm_kernel<T, AKC, BKC, 128, 16, 4, 1>), grid, block, 0, s, p);
  } else if (p.N <= 32) {
    dim3 grid((unsigned)((p.M + BM - 1) / BM), (unsigned)((p.N + 31) / 32), (unsigned)p.splits);
    hipLaunchKernelGGL((gemm_kernel<T, AKC, BKC, 128, 32, 4, 1>), grid, block, 0, s, p);
  } else if (p.N <= 64) {
    dim3 grid((unsigned)((p.M + BM - 1) / BM), (unsigned)((p.N + 63) / 64), (unsigned)p.splits);
    hipLaunchKernelGGL((gemm_kernel<T, AKC, BKC, 128, 64, 4, 1>), grid, block, 0, s, p);
  } else {
    dim3 grid((unsigned)((p.M + BM - 1) / BM), (unsigned)((p.N + 127) / 128), (unsigned)p.splits);
    hipLaunchKernelGGL((gemm_kernel<T, AKC, BKC, 128, 128, 2, 2>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_typed(const GemmCall& c, const GemmParams& p, hipStream_t s) {
  if (c.a_kc && !c.b_kc) return launch_layout<T, true, false>(p, s);
  if (c.a_kc && c.b_kc) return launch_layout<T, true, true>(p, s);
  if (!c.a_kc && !c.b_kc) return launch_layout<T, false, false>(p, s);
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------ reductions ----

// One reduction: OPW outputs per workgroup and NG = 256 / OPW groups of
// splits; group g walks splits g, g + NG, ... in order, then the group sums
// are added in group order.  Few outputs with many splits (the column sums
// of a long matrix) take small OPW, so that no thread walks a long chain of
// dependent loads.
template <typename T, int OPW>
__device__ __forceinline__ void reduce_body_t(const RedJob& j, int64_t blk) {
  constexpr int NG = 256 / OPW;
  __shared__ float red[NG][OPW];
  const int64_t total = j.M * j.width;
  const int t = threadIdx.x % OPW, g = threadIdx.x / OPW;
  const int64_t idx = blk * OPW + t;
  const int64_t r = idx / j.width, c = idx % j.width;
  const bool live = idx < total && c < j.N;
  float a = 0.f;
  if (live) {
    const float* q = j.part + r * j.ld + c;
    const int64_t stride = j.M * j.ld;
#pragma unroll 8
    for (int sidx = g; sidx < j.splits; sidx += NG) a += q[(int64_t)sidx * stride];
  }
  red[g][t] = a;
  __syncthreads();
  if (g != 0 || idx >= total) return;
  if (c >= j.N) {   // EPI_F32 padding columns
    reinterpret_cast<float*>(j.ep.out)[r * j.ep.ldo + c] = 0.f;
    return;
  }
  float sum = red[0][t];
  for (int k = 1; k < NG; ++k) sum += red[k][t];
  epi_store1<T>(j.ep, r, c, sum);
}

template <typename T>
__device__ __forceinline__ void reduce_body(const RedJob& j, int64_t blk) {
  if (j.opw == 1) reduce_body_t<T, 1>(j, blk);
  else if (j.opw == 4) reduce_body_t<T, 4>(j, blk);
  else if (j.opw == 16) reduce_body_t<T, 16>(j, blk);
  else reduce_body_t<T, 64>(j, blk);
}

// Up to two independent reductions in one launch: blocks [0, j0.blocks)
// take j0, the rest j1.
template <typename T>
__global__ __launch_bounds__(256) void reduce_partials_kernel(RedJob j0, RedJob j1) {
  if ((int64_t)blockIdx.x < j0.blocks) reduce_body<T>(j0, blockIdx.x);
  else reduce_body<T>(j1, (int64_t)blockIdx.x - j0.blocks);
}

// Column sums: a workgroup sums `rows_per_block` consecutive rows of the
// lpr * VE columns from blockIdx.y * lpr * VE.  Lane li of a row slot owns
// VE columns (one 16-byte load per row); the 256 / lpr slots walk rows
// r0 + slot, r0 + slot + slots, ... in that order with eight rows in flight,
// then the slots are added in slot order through LDS.
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const T* __restrict__ X, int64_t rows, int64_t cols,
                                                             int64_t ld, int64_t ldp, int64_t rows_per_block,
                                                             int lpr_log2, float* __restrict__ part) {
  constexpr int VE = Vec<T>::N;
  __shared__ float red[256 * VE];
  const int lpr = 1 << lpr_log2, slots = 256 >> lpr_log2, width = lpr * VE;
  const int li = threadIdx.x & (lpr - 1), slot = threadIdx.x >> lpr_log2;
  const int64_t c0 = ((int64_t)blockIdx.y * lpr + li) * VE;
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = min(rows, r0 + rows_per_block);
  float a[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) a[i] = 0.f;
  if (c0 < ldp) {                 // c0 + VE <= ldp <= ld: ldp is a multiple of 8
    const T* __restrict__ x = X + c0;
    int64_t r = r0 + slot;
    for (; r + 7 * slots < r1; r += 8 * slots) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = ldg16(x + (r + u * slots) * ld);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float f[VE];
        unpack<T>(v[u], f);
#pragma unroll
        for (int i = 0; i < VE; ++i) a[i] += f[i];
      }
    }
    for (; r < r1; r += slots) {
      float f[VE];
      unpack<T>(ldg16(x + r * ld), f);
#pragma unroll
      for (int i = 0; i < VE; ++i) a[i] += f[i];
    }
  }
#pragma unroll
  for (int i = 0; i < VE; ++i) red[slot * width + li * VE + i] = a[i];
  __syncthreads();
  for (int t = threadIdx.x; t < width; t += 256) {
    const int64_t c = (int64_t)blockIdx.y * width + t;
    if (c < ldp) {
      float sum = red[t];
      for (int k = 1; k < slots; ++k) sum += red[k * width + t];
      part[(int64_t)blockIdx.x * ldp + c] = c < cols ? sum : 0.f;
    }
  }
}

int64_t colsum_rows_per_block(int64_t rows) {
  int64_t r = (rows + 2047) / 2048;
  return r < 64 ? 64 : r;
}

}  // namespace

int gemm_choose_splits(int prec, int64_t M, int64_t N, int64_t K) {
  const int64_t BK = prec == 0 ? 32 : 64;
  const int64_t BN = N <= 16 ? 16 : N <= 32 ? 32 : N <= 64 ? 64 : 128;
  const int64_t tiles = ((M + 127) / 128) * ((N + BN - 1) / BN);
  const int64_t ktiles = (K + BK - 1) / BK;
  const int64_t target = 512;
  if (tiles >= target / 2 || ktiles < 8) return 1;
  int64_t splits = (target + tiles - 1) / tiles;
  splits = std::min(splits, ktiles / 4);
  return (int)std::max<int64_t>(splits, 1);
}

hipError_t gemm_launch(const GemmCall& c, hipStream_t s) {
  GemmParams p;
  p.A = c.A; p.lda = c.lda; p.B = c.B; p.ldb = c.ldb;
  p.M = c.M; p.N = c.N; p.K = c.K;
  p.splits = c.splits < 1 ? 1 : c.splits;
  p.partials = c.partials;
  p.epi = c.epi;
  const int64_t BK = c.prec == 0 ? 32 : 64;
  const int64_t ktiles = (c.K + BK - 1) / BK;
  p.k_per_split = ((ktiles + p.splits - 1) / p.splits) * BK;
  if (p.k_per_split <= 0) p.k_per_split = BK;
  switch (c.prec) {
    case 0: return launch_typed<float>(c, p, s);
    case 1: return launch_typed<f16>(c, p, s);
    case 2: return launch_typed<bf16>(c, p, s);
  }
  return hipErrorInvalidValue;
}

RedJob make_job(const float* partials, int splits, int64_t M, int64_t N, const Epilogue& epi) {
  return make_job_ld(partials, splits, M, N, N, epi);
}

RedJob make_job_ld(const float* partials, int splits, int64_t M, int64_t N, int64_t ld, const Epilogue& epi) {
  RedJob j;
  j.part = partials; j.splits = splits; j.M = M; j.N = N; j.ld = ld; j.ep = epi;
  j.width = epi.mode == EPI_F32 ? epi.ldo : N;
  // about 32 splits per thread at most where the outputs allow it (one
  // output per workgroup, 64 splits per thread, beyond 4096 splits)
  j.opw = splits > 4096 ? 1 : splits > 512 ? 4 : splits > 128 ? 16 : 64;
  j.blocks = (M * j.width + j.opw - 1) / j.opw;
  return j;
}

hipError_t reduce_partials2(int prec, const RedJob& a, const RedJob* b, hipStream_t s) {
  RedJob j1 = b ? *b : a;
  if (!b) j1.blocks = 0;
  const int64_t blocks = a.blocks + j1.blocks;
  if (blocks <= 0) return hipSuccess;
  switch (prec) {
    case 0: hipLaunchKernelGGL(reduce_partials_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, s, a, j1); break;
    case 1: hipLaunchKernelGGL(reduce_partials_kernel<f16>, dim3((unsigned)blocks), dim3(256), 0, s, a, j1); break;
    case 2: hipLaunchKernelGGL(reduce_partials_kernel<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, a, j1); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t reduce_partials(int prec, const float* partials, int splits, int64_t M, int64_t N,
                           const Epilogue& epi, hipStream_t s) {
  return reduce_partials2(prec, make_job(partials, splits, M, N, epi), nullptr, s);
}

int64_t colsum_partials_floats(int64_t rows, int64_t ld) {
  const int64_t rpb = colsum_rows_per_block(rows);
  return ((rows + rpb - 1) / rpb) * ld;
}

hipError_t colsum_partial_launch(int prec, const void* X, int64_t rows, int64_t cols, int64_t ld, float* partials,
                                 int64_t ldp, int* splits, hipStream_t s) {
  if (ldp % 8 || ld < ldp || (reinterpret_cast<uintptr_t>(X) & 15u)) return hipErrorInvalidValue;
  const int64_t rpb = colsum_rows_per_block(rows);
  const int64_t nb = (rows + rpb - 1) / rpb;
  const int ve = prec == 0 ? 4 : 8;
  int lg = 0;
  while ((int64_t)(1 << lg) * ve < ldp && lg < 6) ++lg;
  const int64_t width = (int64_t)ve << lg;
  dim3 grid((unsigned)nb, (unsigned)((ldp + width - 1) / width));
  switch (prec) {
    case 0: hipLaunchKernelGGL(colsum_partial_kernel<float>, grid, dim3(256), 0, s, (const float*)X, rows, cols, ld, ldp, rpb, lg, partials); break;
    case 1: hipLaunchKernelGGL(colsum_partial_kernel<f16>, grid, dim3(256), 0, s, (const f16*)X, rows, cols, ld, ldp, rpb, lg, partials); break;
    case 2: hipLaunchKernelGGL(colsum_partial_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)X, rows, cols, ld, ldp, rpb, lg, partials); break;
    default: return hipErrorInvalidValue;
  }
  *splits = (int)nb;
  return hipGetLastError();
}

}  // namespace gcn

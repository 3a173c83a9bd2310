// Tall-skinny products of the layer, C (n x N) = A (n x K) . B (K x N) with
// n large and K, N <= a few hundred:
//   S = H W                        (B(k, n) = W[k][n])
//   dZ_below = (G_S W^T) * mask    (B(k, n) = W[n][k])
// Both are bound by streaming A and C through HBM (arithmetic intensity
// <= 64 flop/byte in 16-bit storage), so the kernel is organised around the
// stream:
//  * a workgroup stages its block of B (up to 128 columns x K, k-contiguous,
//    zero-padded to the MFMA k chunk) in LDS once;
//  * each of its 4 waves owns TM x 16 consecutive rows of A and reads their
//    MFMA operand fragments straight from global memory (rows are adjacent,
//    so a wave's loads stay inside one compact region), with a 3-deep
//    register ring of chunks in flight; B fragments come from LDS;
//  * the output of each 16-row tile is staged through a per-wave LDS buffer
//    and written as 16-byte row-contiguous vectors after the epilogue
//    (plain store, or the ReLU/dropout derivative read from H).
#include "internal.h"
#include "xpose.h"

#include <algorithm>

namespace gcn {

namespace {

template <typename T> struct TsMfma;
template <> struct TsMfma<f16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
template <> struct TsMfma<bf16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct TsMfma<float> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

constexpr int TS_LDS_B_BYTES = 80 * 1024;   // cap of the B block in LDS

struct TsParams {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  int64_t M, N, K;
  int64_t kpad;            // K rounded up to the k chunk
  int nblk;                // columns per workgroup (multiple of 16)
  Epilogue epi;
  float* colsum;           // CS: [gridDim.x][N] column sums of the stored C, one row per workgroup
};

// Dynamic LDS: B block [nblk][kpad + VE] (T), then 4 per-wave staging
// buffers [16][nblk + 4] (fp32).
// DM: epilogue multiplies by the ReLU/dropout derivative read from H
// (EPI_DMASK with relu); otherwise a plain store.
// CS: the workgroup also sums the stored values (as stored, i.e. rounded to
// T) of each of its columns: the store pass writes them back to its staging
// buffer, a lane adds the tile's 16 rows of its columns (tiles in order),
// and at the end the four waves' sums are added in wave order into the
// workgroup's row of p.colsum (bias gradient of the layer below, without a
// pass of its own over C).
template <typename T, bool BKC, bool DM, int CSM, int TM, int TNW>
__global__ __launch_bounds__(256) void tsgemm_kernel(TsParams p) {
  constexpr bool CS = CSM != 0;
  constexpr int VE = Vec<T>::N;
  constexpr int KC = 4 * VE;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nblk = p.nblk;
  const int64_t ldsb = p.kpad + VE;                 // LDS row stride of B (elements)
  T* sB = reinterpret_cast<T*>(smem);
  float* sC = reinterpret_cast<float*>(smem + ((size_t)nblk * ldsb * sizeof(T) + 15) / 16 * 16);
  const int ldc = nblk + 4;
  float* myC = sC + wave * 16 * ldc;
  const int64_t n0 = (int64_t)blockIdx.y * nblk;
  const T* __restrict__ Bg = reinterpret_cast<const T*>(p.B);

  // ---- B block -> LDS, k-contiguous: sB[c][k] = B(k, n0 + c), zero outside.
  // Every load of a batch is issued (at an in-bounds address) before any is
  // used; out-of-range elements are zeroed afterwards with dword masks.
  if (BKC) {   // B(k, n) = Bg[n * ldb + k]: copy 16-byte vectors
    constexpr int TS_STAGE = 8;
    const int vpr = (int)(p.kpad / VE);
    const int total = nblk * vpr;
    for (int base = 0; base < total; base += 256 * TS_STAGE) {
      uint4 x[TS_STAGE];
#pragma unroll
      for (int u = 0; u < TS_STAGE; ++u) {
        const int v = base + u * 256 + (int)threadIdx.x;
        const int64_t n = n0 + v / vpr, k = (int64_t)(v % vpr) * VE;
        const bool ok = v < total && n < p.N && k < p.K;
        x[u] = ldg16(Bg + (ok ? n * p.ldb + k : 0));
      }
#pragma unroll
      for (int u = 0; u < TS_STAGE; ++u) {
        const int v = base + u * 256 + (int)threadIdx.x;
        if (v >= total) break;
        const int c = v / vpr;
        const int64_t n = n0 + c, k = (int64_t)(v % vpr) * VE;
        const int64_t nk = p.K - k;
        const int vk = (n >= p.N || nk <= 0) ? 0 : nk >= VE ? VE : (int)nk;
        *reinterpret_cast<uint4*>(sB + c * ldsb + k) = keep_first<T>(x[u], vk);
      }
    }
  } else {     // B(k, n) = Bg[k * ldb + n]: VE x VE blocks (VE k rows x VE columns) turned around in registers
    const int cpb = nblk / VE;                        // column blocks
    const int kpb = (int)(p.kpad / VE);               // k blocks
    const int total = cpb * kpb;
    for (int blk = threadIdx.x; blk < total; blk += 256) {
      const int kb = blk % kpb, cb = blk / kpb;       // consecutive threads: consecutive k blocks (LDS banks)
      const int64_t k0 = (int64_t)kb * VE, n = n0 + (int64_t)cb * VE;
      const int64_t nn = p.N - n;
      const int vc = nn <= 0 ? 0 : nn >= VE ? VE : (int)nn;
      const T* colp = Bg + (vc > 0 ? n : 0);         // n + VE <= round_up(N, 8) <= ldb
      uint4 in[VE], out[VE];
#pragma unroll
      for (int i = 0; i < VE; ++i) in[i] = ldg16(colp + (k0 + i < p.K ? k0 + i : 0) * p.ldb);
#pragma unroll
      for (int i = 0; i < VE; ++i) in[i] = keep_first<T>(in[i], k0 + i < p.K ? vc : 0);
      transpose_block(in, out, T());
#pragma unroll
      for (int j = 0; j < VE; ++j) *reinterpret_cast<uint4*>(sB + (cb * VE + j) * ldsb + k0) = out[j];
    }
  }
  __syncthreads();

  // ---- stream row tiles of A (4 waves x TM x 16 rows per tile), B stays in LDS
  const int64_t tile_rows = 4 * TM * 16;
  const int64_t ntiles = (p.M + tile_rows - 1) / tile_rows;
  const T* __restrict__ Ag = reinterpret_cast<const T*>(p.A);
  const T* bfrag = sB + (lane & 15) * ldsb + (lane >> 4) * VE;
  const int64_t nch = p.kpad / KC;
  const int64_t full = p.K / KC;                    // chunks with no k >= K
  const int tnw = min(TNW, nblk / 16);              // live column tiles of this block
  constexpr int OV = Vec<T>::N;
  const int vpr = nblk / OV;
  // CSM == 1 (vpr divides 64): a lane always stores the same column vector
  // and sums it in registers (creg); CSM == 2: the tile's stored values go
  // back to LDS and a lane sums columns lane and lane + 64 (csum)
  constexpr bool cs_reg = CSM == 1;
  float csum[2] = {0.f, 0.f};
  float creg[OV];
#pragma unroll
  for (int j = 0; j < OV; ++j) creg[j] = 0.f;

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t r0 = tile * tile_rows + (int64_t)wave * (TM * 16);
    const T* arow[TM];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      int64_t r = r0 + tm * 16 + (lane & 15);
      if (r >= p.M) r = p.M - 1;                     // clamped rows are never stored
      arow[tm] = Ag + r * p.lda + (lane >> 4) * VE;
    }
    f32x4 acc[TM][TNW];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto loadA = [&](uint4* a, int64_t c) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) a[tm] = ldg16(arow[tm] + c * KC);
    };
    auto compute = [&](const uint4* a, int64_t c) {
#pragma unroll
      for (int tn = 0; tn < TNW; ++tn) {
        if (tn < tnw) {
          const uint4 b = *reinterpret_cast<const uint4*>(bfrag + tn * 16 * ldsb + c * KC);
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) acc[tm][tn] = TsMfma<T>::run(a[tm], b, acc[tm][tn]);
        }
      }
    };
    // The ReLU/dropout derivative of the epilogue reads H: for 16-bit types
    // the wave's H vectors are requested together with its A fragments, so
    // the tile costs one memory latency.
    constexpr bool dmask = DM;
    constexpr bool HPRE = DM && sizeof(T) == 2;          // H prefetched into registers
    constexpr int EIT = HPRE ? 4 : 1;                    // vectors per lane per 16 rows (nblk <= 128)
    uint4 hv[TM][EIT];
    auto prefetch_h = [&]() {
      if constexpr (HPRE) {
        const T* hm = reinterpret_cast<const T*>(p.epi.hmask);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int it = 0; it < EIT; ++it) {
            const int idx = lane + 64 * it;
            const int rr = idx / vpr, cv = idx % vpr;
            const int64_t row = r0 + tm * 16 + rr, col = n0 + cv * OV;
            const bool ok = idx < 16 * vpr && row < p.M && col < p.N;
            hv[tm][it] = ldg16(hm + (ok ? row * p.epi.ldh + col : 0));
          }
      }
    };
#define TS_FENCE() __builtin_amdgcn_sched_barrier(0)
    uint4 a0[TM], a1[TM], a2[TM], a3[TM];
    if (nch <= 4) {
      // The whole K range fits the four fragment sets: every load of the
      // tile is issued before the first is used (one memory latency per
      // tile).  Vectors at or past K read the row start and are zeroed.
      const int64_t kl0 = (lane >> 4) * VE;
      auto loadw = [&](uint4* a, int64_t c) {
        const int64_t off = c * KC + kl0 < p.K ? c * KC : -kl0;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) a[tm] = ldg16(arow[tm] + off);
      };
      auto maskw = [&](uint4* a, int64_t c) {
        const int64_t nk = p.K - (c * KC + kl0);
        const int vk = nk <= 0 ? 0 : nk >= VE ? VE : (int)nk;
        if (vk < VE) {
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) a[tm] = keep_first<T>(a[tm], vk);
        }
      };
      loadw(a0, 0);
      if (nch > 1) loadw(a1, 1);
      if (nch > 2) loadw(a2, 2);
      if (nch > 3) loadw(a3, 3);
      prefetch_h();   // after the A loads: waiting for A does not wait for H
      TS_FENCE();
      maskw(a0, 0); compute(a0, 0);
      if (nch > 1) { maskw(a1, 1); compute(a1, 1); }
      if (nch > 2) { maskw(a2, 2); compute(a2, 2); }
      if (nch > 3) { maskw(a3, 3); compute(a3, 3); }
    } else {
      prefetch_h();
      int64_t c = 0;
      if (full >= 3) {
        loadA(a0, 0); loadA(a1, 1); loadA(a2, 2);
        TS_FENCE();
        for (; c + 7 <= full; c += 4) {
          loadA(a3, c + 3); TS_FENCE(); compute(a0, c); TS_FENCE();
          loadA(a0, c + 4); TS_FENCE(); compute(a1, c + 1); TS_FENCE();
          loadA(a1, c + 5); TS_FENCE(); compute(a2, c + 2); TS_FENCE();
          loadA(a2, c + 6); TS_FENCE(); compute(a3, c + 3); TS_FENCE();
        }
        compute(a0, c); compute(a1, c + 1); compute(a2, c + 2);
        c += 3;
      }
      for (; c < full; ++c) { loadA(a0, c); compute(a0, c); }
      if (c < nch) {   // the chunk that straddles K: mask k >= K (B rows there are zero too)
        const int64_t kl = c * KC + (lane >> 4) * VE;
        // a vector starting below K ends inside the row (lda >= K rounded up to 8)
        const int64_t nk = p.K - kl;
        const int vk = nk <= 0 ? 0 : nk >= VE ? VE : (int)nk;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) a0[tm] = ldg16(arow[tm] + (vk > 0 ? c * KC : -(lane >> 4) * VE));
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) a0[tm] = keep_first<T>(a0[tm], vk);
        compute(a0, c);
      }
    }
#undef TS_FENCE

    // ---- epilogue: per 16-row tile, MFMA layout -> LDS -> row vectors
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
      for (int tn = 0; tn < TNW; ++tn)
        if (tn < tnw) {
#pragma unroll
          for (int v = 0; v < 4; ++v) myC[((lane >> 4) * 4 + v) * ldc + tn * 16 + (lane & 15)] = acc[tm][tn][v];
        }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      constexpr int NIT = 16 * 128 / Vec<T>::N / 64;   // iterations covering nblk <= 128
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int idx = lane + 64 * it;
        if (idx >= 16 * vpr) break;
        const int rr = idx / vpr, cv = idx % vpr;
        const int64_t row = r0 + tm * 16 + rr, col = n0 + cv * OV;
        if (row >= p.M || col >= p.N) {
          if constexpr (CS && !cs_reg) {
#pragma unroll
            for (int j = 0; j < OV; ++j) myC[rr * ldc + cv * OV + j] = 0.f;
          }
          continue;
        }
        float v[OV];
#pragma unroll
        for (int j = 0; j < OV; ++j) v[j] = myC[rr * ldc + cv * OV + j];
        if constexpr (dmask) {
          float h[OV];
          if constexpr (HPRE) unpack<T>(hv[tm][it], h);
          else unpack<T>(ldg16(reinterpret_cast<const T*>(p.epi.hmask) + row * p.epi.ldh + col), h);
#pragma unroll
          for (int j = 0; j < OV; ++j) v[j] = h[j] > 0.f ? v[j] * p.epi.keep_scale : 0.f;
        }
        if constexpr (CS) {
          if constexpr (cs_reg) {
#pragma unroll
            for (int j = 0; j < OV; ++j) creg[j] += col + j < p.N ? to_f32<T>(from_f32<T>(v[j])) : 0.f;
          } else {
#pragma unroll
            for (int j = 0; j < OV; ++j)
              myC[rr * ldc + cv * OV + j] = col + j < p.N ? to_f32<T>(from_f32<T>(v[j])) : 0.f;
          }
        }
        Epilogue plain = p.epi;
        plain.mode = EPI_STORE;
        epi_store_vec<T>(plain, row, col, v);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if constexpr (CS && !cs_reg) {
        // the tile's stored values are in myC: rows in order per column
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int c = lane + 64 * h;
          if (c < nblk) {
            float a = myC[c];
#pragma unroll
            for (int r = 1; r < 16; ++r) a += myC[r * ldc + c];
            csum[h] += a;
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
  }
  if constexpr (CS) {
    if constexpr (cs_reg) {
      // lanes l, l + vpr, l + 2 vpr, ... hold the same columns: butterfly
#pragma unroll
      for (int off = 32; off > 0; off >>= 1)
        if (off >= vpr)
#pragma unroll
          for (int j = 0; j < OV; ++j) creg[j] += __shfl_xor(creg[j], off);
    }
    __syncthreads();
    if constexpr (cs_reg) {
      if (lane < vpr)
#pragma unroll
        for (int j = 0; j < OV; ++j) myC[lane * OV + j] = creg[j];
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (lane + 64 * h < nblk) myC[lane + 64 * h] = csum[h];
    }
    __syncthreads();
    for (int c = threadIdx.x; c < nblk; c += 256) {
      if (n0 + c < p.N) {
        float a = sC[c];
        a += sC[1 * 16 * ldc + c];
        a += sC[2 * 16 * ldc + c];
        a += sC[3 * 16 * ldc + c];
        p.colsum[(int64_t)blockIdx.x * p.N + n0 + c] = a;
      }
    }
  }
}

// Dynamic LDS of one workgroup: the B block, then the four staging buffers.
template <typename T>
size_t ts_lds_bytes(int64_t nblk, int64_t kpad) {
  return ((size_t)nblk * (kpad + Vec<T>::N) * sizeof(T) + 15) / 16 * 16 + (size_t)4 * 16 * (nblk + 4) * sizeof(float);
}

// Half of a gfx950 compute unit's 160 KB of LDS.
constexpr size_t TS_LDS_TWO_WG = 80 * 1024;

template <typename T>
int ts_nblk(int64_t N, int64_t kpad) {
  int64_t nb = std::min<int64_t>(128, (N + 15) / 16 * 16);
  const int64_t cap = (TS_LDS_B_BYTES / ((kpad + Vec<T>::N) * (int64_t)sizeof(T))) / 16 * 16;
  nb = std::min<int64_t>(nb, std::max<int64_t>(cap, 16));
  // fp32: equal narrower column blocks rather than one workgroup (one wave
  // per SIMD) per compute unit: a 128 x 128 fp32 block of W with its
  // staging needs 101 KB, and the 16x16x4 fp32 matrix instructions then
  // wait on each B read from LDS with no other wave to issue
  if (sizeof(T) == 4) {
    for (int64_t parts = 2; nb > 16 && ts_lds_bytes<T>(nb, kpad) > TS_LDS_TWO_WG; ++parts)
      nb = std::min<int64_t>(nb, ((N + parts - 1) / parts + 15) / 16 * 16);
  }
  return (int)nb;
}

template <typename T, bool BKC, bool DM, int CSM, int TM>
hipError_t launch_tm(const TsParams& p, int* grid_rows, hipStream_t s) {
  const int tnw = p.nblk / 16;
  const size_t lds = ts_lds_bytes<T>(p.nblk, p.kpad);
  // persistent workgroups: enough to fill every CU twice, each looping over row tiles
  const int64_t nb = (p.N + p.nblk - 1) / p.nblk;
  const int64_t ntiles = (p.M + 64 * TM - 1) / (64 * TM);
  const int64_t per_col = std::max<int64_t>(1, 512 / nb);
  dim3 grid((unsigned)std::min<int64_t>(ntiles, per_col), (unsigned)nb);
  if (grid_rows) *grid_rows = (int)grid.x;
#define TS_L(TNW_)                                                                                          \
  do {                                                                                                      \
    if (lds > 65536) {                                                                                      \
      hipError_t ea = hipFuncSetAttribute(reinterpret_cast<const void*>(&tsgemm_kernel<T, BKC, DM, CSM, TM, TNW_>),\
                                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);           \
      if (ea != hipSuccess) return ea;                                                                      \
    }                                                                                                       \
    hipLaunchKernelGGL((tsgemm_kernel<T, BKC, DM, CSM, TM, TNW_>), grid, dim3(256), lds, s, p);                \
  } while (0)
  if (tnw <= 1) TS_L(1);
  else if (tnw <= 2) TS_L(2);
  else if (tnw <= 4) TS_L(4);
  else TS_L(8);
#undef TS_L
  return hipGetLastError();
}

template <typename T, bool BKC, bool DM, bool CS>
hipError_t launch_b(TsParams p, int* grid_rows, hipStream_t s) {
  constexpr int OV = Vec<T>::N;
  constexpr int KC = 4 * Vec<T>::N;
  p.kpad = (p.K + KC - 1) / KC * KC;
  p.nblk = ts_nblk<T>(p.N, p.kpad);
  // rows per wave: 32 when there are enough rows to fill the GPU, else 16
  const int64_t tiles64 = (p.M + 255) / 256 * ((p.N + p.nblk - 1) / p.nblk);
  // (TM = 4 would need more than 256 registers per lane with the whole-K
  // fragment sets, i.e. one wave per SIMD; TM = 2 keeps two)
  // (the H-mask epilogue with 128-column blocks holds another 32 registers:
  // one row tile per wave keeps two waves per SIMD there)
  const bool two = tiles64 >= 256 && !(DM && p.nblk > 64);
  if constexpr (CS) {
    if (64 % (p.nblk / OV) == 0)
      return two ? launch_tm<T, BKC, DM, 1, 2>(p, grid_rows, s) : launch_tm<T, BKC, DM, 1, 1>(p, grid_rows, s);
    return two ? launch_tm<T, BKC, DM, 2, 2>(p, grid_rows, s) : launch_tm<T, BKC, DM, 2, 1>(p, grid_rows, s);
  }
  return two ? launch_tm<T, BKC, DM, 0, 2>(p, grid_rows, s) : launch_tm<T, BKC, DM, 0, 1>(p, grid_rows, s);
}

// Column sums (CS) are only asked of dZ_below = (G_S W^T) * mask, whose B
// is k-contiguous.
template <typename T>
hipError_t launch_t(const TsParams& p, bool bkc, int* grid_rows, hipStream_t s) {
  const bool dm = p.epi.mode == EPI_DMASK && p.epi.relu;
  if (p.colsum) {
    if (!bkc) return hipErrorInvalidValue;
    return dm ? launch_b<T, true, true, true>(p, grid_rows, s) : launch_b<T, true, false, true>(p, grid_rows, s);
  }
  if (!bkc && !dm) return launch_b<T, false, false, false>(p, grid_rows, s);
  if (!dm) return launch_b<T, true, false, false>(p, grid_rows, s);
  return bkc ? launch_b<T, true, true, false>(p, grid_rows, s) : launch_b<T, false, true, false>(p, grid_rows, s);
}

}  // namespace

bool tsgemm_supported(int prec, int64_t K) {
  const int64_t kc = prec == 0 ? 16 : 32;
  const int64_t kpad = (K + kc - 1) / kc * kc;
  const int64_t s = prec == 0 ? 4 : 2;
  return (kpad + 16 / s) * s * 16 <= TS_LDS_B_BYTES;   // at least one 16-column block fits
}

int tsgemm_colsum_rows_max() { return 512; }

hipError_t tsgemm_launch(int prec, const void* A, int64_t lda, const void* B, int64_t ldb, bool b_kc, int64_t M,
                         int64_t N, int64_t K, const Epilogue& epi, hipStream_t s, float* colsum, int* colsum_rows) {
  TsParams p;
  p.A = A; p.lda = lda; p.B = B; p.ldb = ldb; p.M = M; p.N = N; p.K = K; p.kpad = 0; p.nblk = 0; p.epi = epi;
  p.colsum = colsum;
  switch (prec) {
    case 0: return launch_t<float>(p, b_kc, colsum_rows, s);
    case 1: return launch_t<f16>(p, b_kc, colsum_rows, s);
    case 2: return launch_t<bf16>(p, b_kc, colsum_rows, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

// Weight gradient dW = H^T G_S (f_in x f_out) summed over all n vertices.
// Both operands are stored vertex-major (rows of H and of G_S are
// contiguous), so the contraction index k is the slow axis of both.
//  * The vertex range is cut into contiguous spans, one per workgroup; each
//    workgroup owns a whole (up to) 128 x 128 output block and writes its
//    fp32 partial sum; reduce_partials adds the spans in span order.
//  * Per k tile (KT = 8 * VE vertices) the workgroup loads KT x 128 of H
//    and of G_S with 16-byte row-contiguous loads, two tiles ahead in
//    registers.  Each thread holds VE x VE blocks, transposes them in
//    registers (v_perm_b32 for 16-bit) and writes 16-byte k-contiguous
//    columns into a double-buffered LDS tile, from which MFMA fragments are
//    16-byte reads.
#include "internal.h"
#include "xpose.h"

#include <algorithm>

namespace gcn {

namespace {

template <typename T> struct WgMfma;
template <> struct WgMfma<f16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
template <> struct WgMfma<bf16> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct WgMfma<float> {
  static __device__ __forceinline__ f32x4 run(uint4 a, uint4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

constexpr int WG_B = 128;                 // output block edge (rows of dW and columns)

struct WgParams {
  const void* H; int64_t ldh;             // n x M
  const void* G; int64_t ldg;             // n x N
  int64_t n, M, N;
  int64_t span;                           // vertices per workgroup (multiple of KT)
  float* partials;                        // [splits][M][N]
};

// One k tile of H and G_S (KT vertices x 128 columns each) cut into VE x VE
// blocks; thread t holds block(s) of VE rows x 16 bytes in registers.
//   16-bit: 8 x 16 blocks per operand, threads 0..127 take H, 128..255 G_S.
//   fp32:   8 x 32 blocks per operand, every thread takes one of each.
template <typename T>
struct Tile {
  static constexpr int VE = Vec<T>::N;
  static constexpr int KT = 8 * VE;                // 64 (16-bit) / 32 (fp32)
  static constexpr int CB = WG_B / VE;             // column blocks per operand
  static constexpr int NBLK = VE == 8 ? 1 : 2;     // blocks per thread
  uint4 r[NBLK][VE];
  int vrows[NBLK];                                 // rows of the block inside the span
  int vcols[NBLK];                                 // columns of the block inside the operand

  // Issue the block's VE row loads without waiting for any of them: rows
  // beyond the span and blocks beyond the operand read row kfirst / column 0
  // instead (always in bounds) and are zeroed in store(), so the loads are
  // unconditional and stay in flight while the previous tile is multiplied.
  __device__ __forceinline__ void load_block(int b, const T* __restrict__ base, int64_t ld, int64_t c0, int64_t cols,
                                             int64_t k0, int64_t kend, int64_t kfirst, int blk) {
    const int rb = blk / CB, cb = blk % CB;
    const int64_t gc = c0 + (int64_t)cb * VE;
    const int64_t r0 = k0 + rb * VE;
    const int64_t nr = kend - r0, ncol = cols - gc;
    vrows[b] = nr <= 0 ? 0 : nr >= VE ? VE : (int)nr;
    vcols[b] = ncol <= 0 ? 0 : ncol >= VE ? VE : (int)ncol;
    const T* colp = base + (gc < cols ? gc : 0);   // gc + VE <= round_up(cols, 8) <= ld
#pragma unroll
    for (int i = 0; i < VE; ++i) {
      const int64_t gk = r0 + i < kend ? r0 + i : kfirst;
      r[b][i] = ldg16(colp + gk * ld);
    }
  }
  __device__ __forceinline__ void load(const WgParams& p, const T* H, const T* G, int64_t m0, int64_t n0,
                                       int64_t k0, int64_t kend, int64_t kfirst, int tid) {
    if (VE == 8) {
      if (tid < 128) load_block(0, H, p.ldh, m0, p.M, k0, kend, kfirst, tid);
      else load_block(0, G, p.ldg, n0, p.N, k0, kend, kfirst, tid - 128);
    } else {
      load_block(0, H, p.ldh, m0, p.M, k0, kend, kfirst, tid);
      load_block(NBLK - 1, G, p.ldg, n0, p.N, k0, kend, kfirst, tid);
    }
  }
  // Zero the rows and columns outside the operand (first use of the data),
  // with whole-dword masks so the data is never split into 16-bit pieces.
  __device__ __forceinline__ void mask(int b) {
    const int vc = vcols[b];
    uint32_t m[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (VE == 8)
        m[w] = (2 * w < vc ? 0x0000ffffu : 0u) | (2 * w + 1 < vc ? 0xffff0000u : 0u);
      else
        m[w] = w < vc ? 0xffffffffu : 0u;
    }
#pragma unroll
    for (int i = 0; i < VE; ++i) {
      const uint32_t rm = i < vrows[b] ? 0xffffffffu : 0u;
      r[b][i].x &= m[0] & rm;
      r[b][i].y &= m[1] & rm;
      r[b][i].z &= m[2] & rm;
      r[b][i].w &= m[3] & rm;
    }
  }
  // LDS tiles [column][KT + VE], k-contiguous: one 16-byte store per column
  __device__ __forceinline__ void store(T* __restrict__ sA, T* __restrict__ sB, int tid) {
#pragma unroll
    for (int b = 0; b < NBLK; ++b) {
      mask(b);
      const bool isB = VE == 8 ? tid >= 128 : b == 1;
      const int blk = VE == 8 ? (tid & 127) : tid;
      const int rb = blk / CB, cb = blk % CB;
      uint4 t[VE];
      transpose_block(r[b], t, T());
      T* dst = (isB ? sB : sA) + (cb * VE) * (KT + VE) + rb * VE;
#pragma unroll
      for (int j = 0; j < VE; ++j) *reinterpret_cast<uint4*>(dst + j * (KT + VE)) = t[j];
    }
  }
};

// NARROW (N <= 64, one column block): the four waves take 32 rows x 64
// columns each instead of 2 x 2 tiles of 64 x 64, so that no wave
// multiplies the zero columns 64 .. 127 (fp32 dW of a 64-column layer had
// half of its matrix instructions on zeros).
template <typename T, bool NARROW>
__global__ __launch_bounds__(256) void wgrad_kernel(WgParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int KT = Tile<T>::KT;
  constexpr int LDK = KT + VE;
  constexpr int TM = NARROW ? 2 : 4, TN = 4;       // wave tile 32 x 64 (4 x 1 waves) or 64 x 64 (2 x 2)
  __shared__ __align__(16) T sA[2][WG_B * LDK];
  __shared__ __align__(16) T sB[2][WG_B * LDK];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = NARROW ? wave * 32 : (wave >> 1) * 64;   // first row and column of the wave's tile
  const int wc = NARROW ? 0 : (wave & 1) * 64;
  const int64_t split = blockIdx.x;
  const int64_t m0 = (int64_t)blockIdx.y * WG_B, n0 = (int64_t)blockIdx.z * WG_B;
  const int64_t kb = split * p.span, ke = std::min(p.n, kb + p.span);
  const T* __restrict__ Hg = reinterpret_cast<const T*>(p.H);
  const T* __restrict__ Gg = reinterpret_cast<const T*>(p.G);

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nt = ke > kb ? (ke - kb + KT - 1) / KT : 0;
  Tile<T> t0, t1;
  auto load = [&](Tile<T>& x, int64_t t) { x.load(p, Hg, Gg, m0, n0, kb + t * KT, ke, kb, tid); };
  auto compute = [&](int st) {
    const T* as = sA[st] + (wr + (lane & 15)) * LDK + (lane >> 4) * VE;
    const T* bs = sB[st] + (wc + (lane & 15)) * LDK + (lane >> 4) * VE;
#pragma unroll
    for (int ks = 0; ks < KT / (4 * VE); ++ks) {
      uint4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const uint4*>(as + i * 16 * LDK + ks * 4 * VE);
#pragma unroll
      for (int j = 0; j < TN; ++j) bf[j] = *reinterpret_cast<const uint4*>(bs + j * 16 * LDK + ks * 4 * VE);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = WgMfma<T>::run(af[i], bf[j], acc[i][j]);
    }
  };
  // one step: park tile t (registers x) in LDS buffer t % 2, refill x with
  // tile t + 2, multiply tile t
  auto step = [&](Tile<T>& x, int64_t t) {
    const int st = (int)(t & 1);
    x.store(sA[st], sB[st], tid);
    __syncthreads();
    if (t + 2 < nt) load(x, t + 2);
    compute(st);
  };
  if (nt > 0) load(t0, 0);
  if (nt > 1) load(t1, 1);
  int64_t t = 0;
  for (; t + 2 <= nt; t += 2) {
    step(t0, t);
    step(t1, t + 1);
  }
  if (t < nt) step(t0, t);

  // partial block -> partials[split] (MFMA layout: rows 4*(lane/16)+v, column lane%16)
  float* out = p.partials + split * p.M * p.N;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t m = m0 + wr + i * 16 + (lane >> 4) * 4 + v;
        const int64_t nn = n0 + wc + j * 16 + (lane & 15);
        if (m < p.M && nn < p.N) out[m * p.N + nn] = acc[i][j][v];
      }
}

template <typename T>
hipError_t launch_t(const WgParams& p, int splits, hipStream_t s) {
  dim3 grid((unsigned)splits, (unsigned)((p.M + WG_B - 1) / WG_B), (unsigned)((p.N + WG_B - 1) / WG_B));
  if (p.N <= 64) hipLaunchKernelGGL((wgrad_kernel<T, true>), grid, dim3(256), 0, s, p);
  else hipLaunchKernelGGL((wgrad_kernel<T, false>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

int64_t wgrad_kt(int prec) { return prec == 0 ? 32 : 64; }

}  // namespace

// Vertices per span: about 512 workgroups over the M x N blocks, at least
// 4 k tiles each.
int wgrad_splits(int prec, int64_t n, int64_t M, int64_t N) {
  const int64_t kt = wgrad_kt(prec);
  const int64_t blocks = ((M + WG_B - 1) / WG_B) * ((N + WG_B - 1) / WG_B);
  int64_t splits = std::max<int64_t>(1, 512 / blocks);
  const int64_t max_splits = std::max<int64_t>(1, (n + 4 * kt - 1) / (4 * kt));
  splits = std::min(splits, max_splits);
  return (int)splits;
}

hipError_t wgrad_launch(int prec, const void* H, int64_t ldh, const void* G, int64_t ldg, int64_t n, int64_t M,
                        int64_t N, int splits, float* partials, hipStream_t s) {
  const int64_t kt = wgrad_kt(prec);
  WgParams p;
  p.H = H; p.ldh = ldh; p.G = G; p.ldg = ldg; p.n = n; p.M = M; p.N = N; p.partials = partials;
  p.span = ((n + splits - 1) / splits + kt - 1) / kt * kt;
  switch (prec) {
    case 0: return launch_t<float>(p, splits, s);
    case 1: return launch_t<f16>(p, splits, s);
    case 2: return launch_t<bf16>(p, splits, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

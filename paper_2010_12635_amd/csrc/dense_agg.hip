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
//    load, which measured far below the stream rate on MI355X).  Tiled
//    A_hat is read once per call, with non-temporal loads (measured 7-13 %
//    faster at n = 16384, F = 64 and 32; Xt, which every workgroup re-reads,
//    keeps ordinary loads).  Row-major A_hat does not: each of its 128-byte
//    lines serves two consecutive chunks, and with non-temporal loads the
//    line is gone before the second (O1 training 23 % slower).
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
    for (int tm = 0; tm < 4; ++tm)
      f.a[tm] = TILED ? ldg16_nt(abase[tm] + c * astep) : ldg16(abase[tm] + c * astep);
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
    // A step issues the 4 + TN loads of one chunk spread among the MFMAs of
    // another, one load before every NM / NL MFMAs, so that the matrix pipe
    // and the loads overlap (fp32, where the MFMAs dominate: 375 -> 274 us at
    // n = 16384, F = 64, 201 -> 170 us at F = 32; 16-bit unchanged, bound by
    // the stream).  With fewer MFMAs than loads the loads go first.
    constexpr int NL = 4 + TN, NM = 4 * TN * (sizeof(T) == 4 ? 4 : 1), PER = NM / NL;
#define DA_STEP(FL, CL, FC)                                                            \
    if (PER >= 1) {                                                                    \
      load(FL, CL); compute(FC);                                                       \
      _Pragma("unroll") for (int q_ = 0; q_ < NL; ++q_) {                              \
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   /* vector-memory read */  \
        __builtin_amdgcn_sched_group_barrier(0x008, PER >= 1 ? PER : 1, 0); /* MFMA */ \
      }                                                                                \
    } else {                                                                           \
      load(FL, CL); DA_FENCE(); compute(FC);                                           \
    }                                                                                  \
    DA_FENCE();
    for (; c + 7 <= full_end; c += 4) {
      DA_STEP(f3, c + 3, f0)
      DA_STEP(f0, c + 4, f1)
      DA_STEP(f1, c + 5, f2)
      DA_STEP(f2, c + 6, f3)
    }
#undef DA_STEP
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

// ---------------------------------------------------------------------------
// Wide features (F >= 128, the large model sizes of the paper's Table 1):
// 2 n^2 F flops against s n^2 bytes of A_hat put the product far above the
// ridge point, so this kernel is built around the matrix cores.
//  * A workgroup of 4 waves owns a 256 x 256 output tile, each wave a
//    128 x 128 quarter (8 x 8 MFMA 16x16 tiles, 256 fp32 accumulators per
//    lane, one wave per SIMD).
//  * Both operands come straight from global memory in MFMA operand order
//    (tiled A_hat, tiled X^T): a fragment is one contiguous 1 KiB, 16 per
//    k chunk per wave, with MM_DEPTH - 1 chunks in flight.  The two waves
//    that share the rows (or the columns) of the tile read the same lines.
//    (Staging the chunk through LDS, each fragment loaded once per
//    workgroup, measured slower: 41 % against 54 % of the MFMA peak.)
//  * Tiles are dealt out XCD by XCD: workgroup b runs on XCD b % 8, and each
//    XCD takes a contiguous range of tiles in row-major order, so the column
//    tiles of a row block run together and share A_hat in that XCD's L2
//    (measured at n = 32768: 1-2 % over plain order, 4 % over column-major).
//  * The epilogue stages each 16-row strip of the wave's quarter through
//    LDS and stores rows as 16-byte vectors through the fused epilogue
//    (with the bias of a lane's columns loaded once per tile).
// ---------------------------------------------------------------------------
constexpr int MM_LDR = 128 + 4;   // LDS stride (floats) of a staged strip
// Each wave stages through its own LDS area, so a strip needs no workgroup
// barrier: the wave's own LDS operations complete in order, and waiting for
// them (with a compiler memory fence) orders the writes of one lane before
// the reads of another (measured 2-5 % faster at F = 512 and 1024).
#define MM_SYNC() asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory")

struct MmParams {
  const void* A;      // tiled A_hat
  const void* Xt;     // tiled X^T
  int64_t n, F, nc;   // vertices, features, k chunks
  int64_t rblocks;    // 64-row blocks of A_hat
  int64_t fblocks;    // 64-row blocks of X^T
  int64_t tiles, cb, per_xcd;
  int64_t ksplit, kc; // k ranges of kc chunks (the last one shorter), one per workgroup of a tile
  float* part;        // ksplit > 1: fp32 partial products [ksplit][n][ldp]
  int64_t ldp;        // F rounded up to a whole output vector
  Epilogue epi;
};

// Rows row0 .. row0 + 15, columns col0 .. col0 + W - 1 of the output from a
// staged strip (16 x W fp32, stride MM_LDR), through the fused epilogue.  A
// lane stores the same vector of columns in every row it takes (64 is a
// multiple of W / Vec<T>::N), whose bias bv the caller loads once per tile.
template <typename T, int W>
__device__ __forceinline__ void mm_store_strip(const MmParams& p, const float* st, int lane, int64_t row0, int64_t col0,
                                               const float (&bv)[Vec<T>::N]) {
  constexpr int OV = Vec<T>::N;
  constexpr int VPR = W / OV;                      // vectors per strip row
#pragma unroll 1
  for (int k = 0; k < 16 * VPR / 64; ++k) {
    const int idx = k * 64 + lane;
    const int r = idx / VPR, cv = idx % VPR;
    const int64_t row = row0 + r, col = col0 + cv * OV;
    if (row >= p.n || col >= p.F) continue;
    float v[OV];
#pragma unroll
    for (int e = 0; e < OV; ++e) v[e] = st[r * MM_LDR + cv * OV + e];
    epi_store_vec_b<T>(p.epi, row, col, v, bv);
  }
}

// A wave owns WR x WC 64 x 64 blocks of the output (WR, WC in {1, 2}); the
// workgroup's 2 x 2 waves own (128 WR) x (128 WC).
// The same strip as fp32 partial products of k range `split`, for the
// fixed-order reduction that applies the epilogue.
template <int W, int OV>
__device__ __forceinline__ void mm_store_strip_part(const MmParams& p, const float* st, int lane, int64_t row0,
                                                    int64_t col0, int64_t split) {
  constexpr int VPR = W / OV;
  float* part = p.part + split * p.n * p.ldp;
#pragma unroll 1
  for (int k = 0; k < 16 * VPR / 64; ++k) {
    const int idx = k * 64 + lane;
    const int r = idx / VPR, cv = idx % VPR;
    const int64_t row = row0 + r, col = col0 + cv * OV;
    if (row >= p.n || col >= p.F) continue;
    float4* o = reinterpret_cast<float4*>(part + row * p.ldp + col);
#pragma unroll
    for (int e = 0; e < OV / 4; ++e)
      o[e] = make_float4(st[r * MM_LDR + cv * OV + 4 * e], st[r * MM_LDR + cv * OV + 4 * e + 1],
                         st[r * MM_LDR + cv * OV + 4 * e + 2], st[r * MM_LDR + cv * OV + 4 * e + 3]);
  }
}

// Sum of the k ranges' partials in range order, one output vector per
// thread, through the vector epilogue (one Philox block per 8 outputs).
template <typename T>
__global__ __launch_bounds__(256) void mm_reduce_kernel(const float* __restrict__ part, int64_t ksplit, int64_t n,
                                                        int64_t F, int64_t ldp, Epilogue epi) {
  constexpr int VE = Vec<T>::N;
  const int64_t vpr = ldp / VE;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n * vpr) return;
  const int64_t row = idx / vpr, col0 = (idx - row * vpr) * VE;
  float acc[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) acc[i] = 0.f;
  for (int64_t k = 0; k < ksplit; ++k) {
    const float4* q = reinterpret_cast<const float4*>(part + (k * n + row) * ldp + col0);
#pragma unroll
    for (int e = 0; e < VE / 4; ++e) {
      const float4 v = q[e];
      acc[4 * e] += v.x; acc[4 * e + 1] += v.y; acc[4 * e + 2] += v.z; acc[4 * e + 3] += v.w;
    }
  }
  epi_store_vec<T>(epi, row, col0, acc);
}

template <typename T, int WR, int WC, int DEPTH>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void dense_mm_kernel(MmParams p) {
  constexpr int VE = Vec<T>::N, KC = 4 * VE, PIECE = 16 * KC;
  constexpr int TM = 4 * WR, TN = 4 * WC;          // 16 x 16 MFMA tiles per wave
  __shared__ float stage[4][16 * MM_LDR];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t b = blockIdx.x;
  // units are (k range, tile), k range outermost, so that the workgroups of
  // one die (consecutive units) share rows of A_hat as before
  const int64_t u = (b & 7) * p.per_xcd + (b >> 3);
  if (u >= p.tiles * p.ksplit) return;
  const int64_t split = u / p.tiles;
  const int64_t t = u - split * p.tiles;
  const int64_t tr = t / p.cb, tc = t - (t / p.cb) * p.cb;
  const int64_t rb0 = (tr * 2 + (wave >> 1)) * WR;   // this wave's first 64-row block
  const int64_t fb0 = (tc * 2 + (wave & 1)) * WC;    // and first 64-column block
  const int64_t c_lo = split * p.kc;                  // this workgroup's k chunks: [c_lo, c_lo + nc)
  const int64_t nc = min(p.nc, c_lo + p.kc) - c_lo;   // >= 8 (the launch sizes the ranges so)
  const int64_t blk = p.nc * 4 * PIECE;               // elements of one 64-row block
  const T* __restrict__ A = reinterpret_cast<const T*>(p.A);
  const T* __restrict__ Xt = reinterpret_cast<const T*>(p.Xt);
  // blocks past the padded extent read the last one (never stored)
  const T* abase[WR];
  const T* bbase[WC];
#pragma unroll
  for (int i = 0; i < WR; ++i) abase[i] = A + min(rb0 + i, p.rblocks - 1) * blk + c_lo * 4 * PIECE + lane * VE;
#pragma unroll
  for (int i = 0; i < WC; ++i) bbase[i] = Xt + min(fb0 + i, p.fblocks - 1) * blk + c_lo * 4 * PIECE + lane * VE;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct Fr { uint4 a[TM]; uint4 b[TN]; };
  auto load = [&](Fr& f, int64_t c) {
    c = c < nc ? c : nc - 1;                      // past the end: in bounds, unused
    const int64_t off = c * 4 * PIECE;
#pragma unroll
    for (int i = 0; i < WR; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) f.a[i * 4 + q] = ldg16(abase[i] + off + q * PIECE);
#pragma unroll
    for (int i = 0; i < WC; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) f.b[i * 4 + q] = ldg16(bbase[i] + off + q * PIECE);
  };
  auto compute = [&](const Fr& f) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = DaMfma<T>::run(f.a[i], f.b[j], acc[i][j]);
  };
#define MM_FENCE() __builtin_amdgcn_sched_barrier(0)
  // Loop steps of the 3-deep ring: the 4 (WR + WC) loads of one chunk are
  // spread among the MFMAs of another, one load before every NM / NL MFMAs
  // (the rest after the last load), instead of all loads first: the matrix
  // pipe keeps issuing while the loads go out (measured 3.20 -> 2.99 ms at
  // n = 32768, F = 2048, 1.60 -> 1.57 ms at F = 1024; for the 2-deep ring of
  // the 256 x 128 tiles it was 2-4 % slower, so that loop keeps plain fences).
  constexpr int NL = 4 * (WR + WC), NM = TM * TN * (sizeof(T) == 4 ? 4 : 1), PER = NM / NL;   // fp32: 4 MFMAs per pair
#define MM_SCHED()                                                                   \
  do {                                                                               \
    _Pragma("unroll") for (int q_ = 0; q_ < NL; ++q_) {                              \
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   /* vector-memory read */  \
      __builtin_amdgcn_sched_group_barrier(0x008, PER, 0); /* MFMA */                \
    }                                                                                \
    __builtin_amdgcn_sched_group_barrier(0x008, NM - PER * NL, 0);                   \
  } while (0)
  // The chunks that do not fill a whole trip of the unrolled loop are done
  // first, so that nothing follows the loop: with a compute after it the
  // register allocator rotates the accumulators on every trip.
  // The launch guarantees n >= 256, i.e. nc >= 8 chunks, so each loop below
  // runs at least once; written as do-while, it has no path that skips it
  // (where such a path meets the loop exit the register allocator spills
  // accumulators, and the reloads before the loop make the compiler wait
  // for a whole chunk of loads more than the ring needs at the loop head).
  if (DEPTH == 2) {
    Fr f0, f1;
    int64_t c = 0;
    if (nc & 1) { load(f0, 0); compute(f0); c = 1; }
    load(f0, c);
    do {
      load(f1, c + 1); MM_FENCE(); compute(f0); MM_FENCE();
      load(f0, c + 2); MM_FENCE(); compute(f1); MM_FENCE();
      c += 2;
    } while (c + 2 <= nc);
  } else {
    Fr f0, f1, f2;
    int64_t c = 0;
    const int64_t r3 = nc % 3;
    if (r3 >= 1) { load(f0, 0); compute(f0); }
    if (r3 >= 2) { load(f0, 1); compute(f0); }
    c = r3;
    load(f0, c);
    load(f1, c + 1);
    do {
      load(f2, c + 2); compute(f0); MM_SCHED(); MM_FENCE();
      load(f0, c + 3); compute(f1); MM_SCHED(); MM_FENCE();
      load(f1, c + 4); compute(f2); MM_SCHED(); MM_FENCE();
      c += 3;
    } while (c + 3 <= nc);
  }
#undef MM_FENCE
#undef MM_SCHED

  // epilogue: one 16-row strip of the wave's block at a time (the strip
  // index is spelled out so that every accumulator index is static); with
  // k ranges the strips go out as fp32 partials instead
  float* st = stage[wave];
  float bv[VE];
  epi_load_bias<T>(p.epi, fb0 * 64 + (lane % (16 * TN / VE)) * VE, bv);
  const bool partial = p.ksplit > 1;
#define MM_STRIP(S)                                                                             \
  if ((S) < TM) {                                                                               \
    MM_SYNC();                                                                            \
    _Pragma("unroll") for (int j = 0; j < TN; ++j)                                              \
      _Pragma("unroll") for (int v = 0; v < 4; ++v)                                             \
        st[((lane >> 4) * 4 + v) * MM_LDR + j * 16 + (lane & 15)] = acc[(S) < TM ? (S) : 0][j][v]; \
    MM_SYNC();                                                                            \
    if (partial) mm_store_strip_part<16 * TN, VE>(p, st, lane, (rb0 + (S) / 4) * 64 + ((S) % 4) * 16, fb0 * 64, split); \
    else mm_store_strip<T, 16 * TN>(p, st, lane, (rb0 + (S) / 4) * 64 + ((S) % 4) * 16, fb0 * 64, bv); \
  }
  MM_STRIP(0) MM_STRIP(1) MM_STRIP(2) MM_STRIP(3) MM_STRIP(4) MM_STRIP(5) MM_STRIP(6) MM_STRIP(7)
#undef MM_STRIP
}

int64_t xt_elems(int prec, int64_t n, int64_t F) {
  const int64_t kc = prec == 0 ? 16 : 32;
  const int64_t nc = (n + kc - 1) / kc;
  return ((F + 63) / 64) * 64 * nc * kc;
}

// Bytes of the transposed X, rounded up to 256 (the partials follow it).
size_t xt_bytes(int prec, int64_t n, int64_t F) {
  return ((size_t)xt_elems(prec, n, F) * (prec == 0 ? 4 : 2) + 255) / 256 * 256;
}

#ifndef MM_MIN_F
#define MM_MIN_F 192
#endif
#ifndef MM_DEPTH
#define MM_DEPTH 3
#endif
#ifndef MM_SMALL_TILES
#define MM_SMALL_TILES 256
#endif
// The wide-feature kernel takes over from F >= MM_MIN_F (tiled A_hat):
// 128 x 64 per wave up to F = 384, 128 x 128 above (measured on MI355X at
// n = 32768: F = 256 0.72 ms against 0.92 ms, F = 2048 3.3 ms against
// 4.8 ms; the streaming kernel takes 0.77 ms at F = 128, 1.5 ms at 256).
bool use_dense_mm(int64_t n, int64_t F) { return F >= MM_MIN_F && n >= 256; }

// Tile shape and k ranges of the wide kernel.  Fewer tiles than compute
// units, 16-bit: first cut the k loop of every tile into 2, 4 or 8 ranges of
// at least MM_SPLIT_MIN chunks each (their fp32 partials are added in range
// order by a reduction that applies the epilogue), keeping the 128 x 128
// accumulator tile per wave.  Where the k loop is too short for that, step
// down to 256 x 128 or 128 x 128 workgroup tiles if that alone fills the
// compute units, else cut the k loop into ranges of at least 8 chunks.
// Measured in 16-bit: n = 16384, F = 512 (128 tiles): two ranges 0.29 ms,
// 256 x 128 tiles 0.36 ms; n = 4096, F = 2048 (k loop of 128 chunks): two
// ranges 0.108 ms, 256 x 128 tiles 0.10 ms; n = 4096, F = 512 (32 tiles):
// eight ranges 0.054 ms, 128 x 128 tiles 0.061 ms.
#ifndef MM_SPLIT_MIN
#define MM_SPLIT_MIN 128
#endif
struct MmPlan { int wr, wc; int64_t ksplit, kc; };

MmPlan mm_plan(int prec, int64_t n, int64_t F) {
  const int64_t kcw = prec == 0 ? 16 : 32;
  const int64_t nc = (n + kcw - 1) / kcw;
  MmPlan pl{2, F > 384 ? 2 : 1, 1, nc};
  auto tiles_of = [&](int wr, int wc) { return (n + 128 * wr - 1) / (128 * wr) * ((F + 128 * wc - 1) / (128 * wc)); };
  auto split = [&](int64_t min_chunks) {
    while (tiles_of(pl.wr, pl.wc) * pl.ksplit < MM_SMALL_TILES && pl.ksplit < 8) {
      const int64_t k2 = pl.ksplit * 2, kc = (nc + k2 - 1) / k2;
      if (kc < min_chunks || nc - (k2 - 1) * kc < 8) break;
      pl.ksplit = k2;
    }
  };
  if (prec == 0) {
    // fp32 is bound by the matrix units at these widths, where smaller
    // tiles cost only re-reads: step down first, then cut the k loop
    // (n = 4096, F = 512: 885 epochs/s cutting the k loop of 256 x 256
    // tiles, 1481 with 128 x 128 tiles)
    if (tiles_of(pl.wr, pl.wc) < MM_SMALL_TILES) {
      if (pl.wc == 2 && tiles_of(2, 1) >= MM_SMALL_TILES) pl.wc = 1;
      else pl.wr = pl.wc = 1;
    }
    split(8);
  } else {
    split(MM_SPLIT_MIN);
    if (pl.ksplit == 1 && tiles_of(pl.wr, pl.wc) < MM_SMALL_TILES) {
      if (pl.wc == 2 && tiles_of(2, 1) >= MM_SMALL_TILES) pl.wc = 1;
      else if (tiles_of(1, 1) >= MM_SMALL_TILES) pl.wr = pl.wc = 1;
      else split(8);
    }
  }
  pl.kc = (nc + pl.ksplit - 1) / pl.ksplit;
  return pl;
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
  if (tiled && use_dense_mm(n, F)) {
    const MmPlan pl = mm_plan(sizeof(T) == 4 ? 0 : 1, n, F);
    const int WR = pl.wr, WC = pl.wc;
    MmParams q;
    q.A = A; q.Xt = Xt; q.n = n; q.F = F; q.nc = nc;
    q.rblocks = (n + 63) / 64;
    q.fblocks = fblocks;
    const int64_t rt = (n + 128 * WR - 1) / (128 * WR);
    q.cb = (F + 128 * WC - 1) / (128 * WC);
    q.tiles = rt * q.cb;
    q.ksplit = pl.ksplit;
    q.kc = pl.kc;
    q.part = pl.ksplit > 1 ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + xt_bytes(sizeof(T) == 4 ? 0 : 1, n, F))
                           : nullptr;
    q.ldp = (F + Vec<T>::N - 1) / Vec<T>::N * Vec<T>::N;
    q.per_xcd = (q.tiles * q.ksplit + 7) / 8;
    q.epi = epi;
    const dim3 g((unsigned)(8 * q.per_xcd));
    if (WR == 1) hipLaunchKernelGGL((dense_mm_kernel<T, 1, 1, MM_DEPTH>), g, dim3(256), 0, s, q);
    else if (WC == 2) hipLaunchKernelGGL((dense_mm_kernel<T, 2, 2, MM_DEPTH>), g, dim3(256), 0, s, q);
    else hipLaunchKernelGGL((dense_mm_kernel<T, 2, 1, 2>), g, dim3(256), 0, s, q);
    e = hipGetLastError();
    if (e != hipSuccess || pl.ksplit == 1) return e;
    // the k ranges' partials, added in range order, through the epilogue
    const int64_t vecs = n * (q.ldp / Vec<T>::N);
    hipLaunchKernelGGL(mm_reduce_kernel<T>, dim3((unsigned)((vecs + 255) / 256)), dim3(256), 0, s, q.part, pl.ksplit,
                       n, F, q.ldp, epi);
    return hipGetLastError();
  }
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

size_t dense_agg_workspace_bytes(int prec, int64_t n, int64_t F, bool tiled) {
  size_t b = xt_bytes(prec, n, F);
  if (tiled && use_dense_mm(n, F)) {
    const MmPlan pl = mm_plan(prec, n, F);
    const int64_t ve = prec == 0 ? 4 : 8;
    if (pl.ksplit > 1) b += (size_t)pl.ksplit * (size_t)n * (size_t)((F + ve - 1) / ve * ve) * sizeof(float);
  }
  return b;
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

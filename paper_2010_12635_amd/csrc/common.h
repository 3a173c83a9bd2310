// Device-side helpers shared by the libgcn kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gcn {

typedef _Float16 f16;
typedef __bf16 bf16;

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte vector of storage elements: 8 x 16-bit or 4 x fp32.
template <typename T> struct Vec;
template <> struct Vec<float> { static constexpr int N = 4; typedef f32x4 type; };
template <> struct Vec<f16>   { static constexpr int N = 8; typedef f16x8 type; };
template <> struct Vec<bf16>  { static constexpr int N = 8; typedef bf16x8 type; };

template <typename T> __device__ __forceinline__ float to_f32(T x) { return (float)x; }
// Round-to-nearest-even conversions (v_cvt_f16_f32 / bf16 RNE), never the
// round-toward-zero packed forms.
template <typename T> __device__ __forceinline__ T from_f32(float x) { return (T)x; }

__device__ __forceinline__ uint4 ldg16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}
// Non-temporal 16-byte load, for data read once (a stream that should not
// displace reused lines from the caches).  Measured on MI355X: a read-only
// stream of 512 MiB reaches 6.7-7.2 TB/s this way against 6.0-6.5 TB/s with
// ordinary loads.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stg16(void* p, uint4 v) {
  *reinterpret_cast<uint4*>(p) = v;
}

// Unpack a 16-byte vector of storage elements into fp32.
template <typename T>
__device__ __forceinline__ void unpack(uint4 raw, float* out) {
  const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) out[i] = to_f32<T>(e[i]);
}
template <typename T>
__device__ __forceinline__ uint4 pack(const float* in) {
  uint4 raw;
  T* e = reinterpret_cast<T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) e[i] = from_f32<T>(in[i]);
  return raw;
}

__device__ __forceinline__ bool finite_f32(float x) {
  return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u;
}

// ---------------------------------------------------------------------------
// Philox-4x64-10 (Salmon, Moraes, Dror & Shaw, SC'11): ten rounds of two
// 64x64->128-bit multiplies; the key is bumped by two Weyl constants between
// rounds.
// ---------------------------------------------------------------------------
struct Philox8 { uint64_t w[4]; };

// Full 128-bit product a * m from four 32 x 32 -> 64-bit multiply-adds
// (schoolbook: no partial sum exceeds 64 bits, and the high word of the
// exact product is below 2^64).  The compiler maps each step to one
// v_mad_u64_u32; the 64-bit product and the 64-bit high product written
// as such cost about a third more multiplies.
__device__ __forceinline__ void mul_64x64_128(uint64_t a, uint64_t m, uint64_t& lo, uint64_t& hi) {
  const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32), m0 = (uint32_t)m, m1 = (uint32_t)(m >> 32);
  const uint64_t p00 = (uint64_t)a0 * m0;
  const uint64_t p01 = (uint64_t)a0 * m1 + (p00 >> 32);
  const uint64_t p10 = (uint64_t)a1 * m0 + (uint32_t)p01;
  hi = (uint64_t)a1 * m1 + (p01 >> 32) + (p10 >> 32);
  lo = (p10 << 32) | (uint32_t)p00;
}

__device__ __forceinline__ Philox8 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                  uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    uint64_t lo0, hi0, lo1, hi1;
    mul_64x64_128(c0, M0, lo0, hi0);
    mul_64x64_128(c2, M1, lo1, hi1);
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += W0; k1 += W1;
  }
  Philox8 o; o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
  return o;
}

// Word w (0..7) of a Philox block: low half of output w/2 for even w, high
// half for odd w.  Selected without indexing so the block stays in registers.
__device__ __forceinline__ uint32_t philox_word(const Philox8& o, uint32_t w) {
  const uint32_t h = w >> 1;
  const uint64_t x = h == 0 ? o.w[0] : h == 1 ? o.w[1] : h == 2 ? o.w[2] : o.w[3];
  return (w & 1) ? (uint32_t)(x >> 32) : (uint32_t)x;
}

// ---------------------------------------------------------------------------
// Output epilogue shared by the aggregation and GEMM kernels.
// ---------------------------------------------------------------------------
enum EpiMode : int {
  EPI_STORE = 0,   // out = cvt(acc)
  EPI_AGG = 1,     // out = cvt(dropout(act(acc + bias)))
  EPI_DMASK = 2,   // out = cvt(acc * [H > 0] * keep_scale)  (or acc if !relu_below)
  EPI_F32 = 3,     // out(fp32) = acc
};

struct Epilogue {
  void* out;             // output base (T or fp32 for EPI_F32)
  int64_t ldo;
  int64_t rows, cols;    // logical output size
  int mode;
  // EPI_AGG
  const float* bias;
  int relu;
  int dropout;           // training && p > 0
  uint32_t thr;          // floor(p * 2^32)
  float keep_scale;      // 1 / (1 - p)
  uint64_t seed;
  uint64_t layer;
  uint64_t epoch;
  const int32_t* epoch_ctr;  // if set, two int32 counters added to epoch when the kernel runs
  // EPI_DMASK
  const void* hmask;     // H (T), same shape as output
  int64_t ldh;
  // overflow flag (may be NULL)
  int32_t* flag;
};

// Dropout counter word: the epoch argument, plus, when the layer names a
// device-resident loss-scale state, its applied and skipped optimiser steps
// as the kernel finds them (so that a captured and replayed epoch draws a
// new mask each time).
__device__ __forceinline__ uint64_t dropout_epoch(const Epilogue& ep) {
  if (!ep.epoch_ctr) return ep.epoch;
  return ep.epoch + (uint64_t)(uint32_t)ep.epoch_ctr[0] + (uint64_t)(uint32_t)ep.epoch_ctr[1];
}

// Philox-4x32-10 (same paper): ten rounds of two 32x32->64-bit multiplies
// (one v_mad_u64_u32 each), the key bumped by two Weyl constants between
// rounds.  The dropout stream: four words per block, about half the
// arithmetic per word of the 4x64 variant.
struct Philox4 { uint32_t w[4]; };

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                 uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)c0 * 0xD2511F53u, p1 = (uint64_t)c2 * 0xCD9E8D57u;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  Philox4 o;
  o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
  return o;
}

// Dropout block b (elements 4b .. 4b + 3): counter (b mod 2^32, b div 2^32,
// epoch mod 2^32, layer), key (seed mod 2^32, seed div 2^32).
__device__ __forceinline__ Philox4 dropout_block(const Epilogue& ep, uint64_t b) {
  return philox4x32_10((uint32_t)b, (uint32_t)(b >> 32), (uint32_t)dropout_epoch(ep), (uint32_t)ep.layer,
                       (uint32_t)ep.seed, (uint32_t)(ep.seed >> 32));
}

__device__ __forceinline__ uint32_t philox4_word(const Philox4& o, uint32_t w) {
  return w == 0 ? o.w[0] : w == 1 ? o.w[1] : w == 2 ? o.w[2] : o.w[3];
}

// Keep decision for element linear index e = row * cols + col: word e mod 4
// of block e div 4 at or above floor(p 2^32).
__device__ __forceinline__ bool dropout_keep(const Epilogue& ep, uint64_t e) {
  return philox4_word(dropout_block(ep, e >> 2), (uint32_t)(e & 3)) >= ep.thr;
}

// Called by the lanes that saw a non-finite value: the lowest of them
// reports for its wave, and only if the flag is not set yet, so that a
// tensor full of NaN or infinity costs one store per wave at most.
__device__ __forceinline__ void raise_flag(int32_t* flag) {
  if (!flag) return;
  const uint64_t active = __ballot(1);
  if ((threadIdx.x & 63) == (unsigned)(__ffsll((unsigned long long)active) - 1)) {
    volatile int32_t* f = flag;
    if (*f == 0) *f = 1;
  }
}

// Scalar epilogue for one element (row < rows, col < cols).
template <typename T>
__device__ __forceinline__ void epi_store1(const Epilogue& ep, int64_t row, int64_t col, float acc) {
  if (ep.mode == EPI_F32) {
    reinterpret_cast<float*>(ep.out)[row * ep.ldo + col] = acc;
    if (!finite_f32(acc)) raise_flag(ep.flag);
    return;
  }
  float z = acc;
  if (ep.mode == EPI_AGG) {
    if (ep.bias) z += ep.bias[col];
    if (ep.relu) {
      z = z > 0.f ? z : 0.f;
      if (ep.dropout) z = dropout_keep(ep, (uint64_t)row * (uint64_t)ep.cols + (uint64_t)col) ? z * ep.keep_scale : 0.f;
    }
  } else if (ep.mode == EPI_DMASK) {
    if (ep.relu) {
      float h = to_f32<T>(reinterpret_cast<const T*>(ep.hmask)[row * ep.ldh + col]);
      z = h > 0.f ? z * ep.keep_scale : 0.f;
    }
  }
  T o = from_f32<T>(z);
  reinterpret_cast<T*>(ep.out)[row * ep.ldo + col] = o;
  if (!finite_f32(to_f32<T>(o))) raise_flag(ep.flag);
}

// Bias of the Vec<T>::N columns from col0 (any col0 >= 0; entries past cols
// re-read column 0 and are never added), for a caller that stores the same
// columns of many rows and loads them once.
template <typename T>
__device__ __forceinline__ void epi_load_bias(const Epilogue& ep, int64_t col0, float (&bv)[Vec<T>::N]) {
  constexpr int VE = Vec<T>::N;
#pragma unroll
  for (int i = 0; i < VE; ++i) bv[i] = 0.f;
  if (!ep.bias || ep.mode != EPI_AGG) return;
#pragma unroll
  for (int i = 0; i < VE; ++i) bv[i] = ep.bias[col0 + i < ep.cols ? col0 + i : 0];
}

// Keep bits of the VE elements from e0 = row * cols + col0 (bit i: element
// e0 + i kept): VE / 4 whole blocks when e0 is a multiple of 4 (cols a
// multiple of 4), else up to VE / 4 + 1 blocks, each element taking its word.
template <int VE>
__device__ __forceinline__ uint32_t dropout_bits(const Epilogue& ep, int64_t row, int64_t col0) {
  const uint64_t e0 = (uint64_t)row * (uint64_t)ep.cols + (uint64_t)col0;
  uint32_t bits = 0;
  if ((e0 & 3) == 0) {
#pragma unroll
    for (int j = 0; j < VE / 4; ++j) {
      const Philox4 o = dropout_block(ep, (e0 >> 2) + j);
#pragma unroll
      for (int q = 0; q < 4; ++q) bits |= (o.w[q] >= ep.thr ? 1u : 0u) << (4 * j + q);
    }
  } else {
    const uint64_t b0 = e0 >> 2, bl = (e0 + VE - 1) >> 2;
#pragma unroll
    for (int j = 0; j <= VE / 4; ++j) {
      if (b0 + j <= bl) {
        const Philox4 o = dropout_block(ep, b0 + j);
#pragma unroll
        for (int i = 0; i < VE; ++i)
          if (((e0 + i) >> 2) == b0 + j) bits |= (philox4_word(o, (uint32_t)((e0 + i) & 3)) >= ep.thr ? 1u : 0u) << i;
      }
    }
  }
  return bits;
}

// Whether an epilogue draws dropout decisions (a caller may draw them with
// dropout_bits ahead of time, while its loads are in flight).
__device__ __forceinline__ bool epi_draws(const Epilogue& ep) { return ep.mode == EPI_AGG && ep.relu && ep.dropout; }

// Vector epilogue: Vec<T>::N consecutive columns starting at col0 (col0 is a
// multiple of the vector width, col0 < cols).  Columns >= cols are written 0.
// bv holds the bias of these columns (epi_load_bias); keep, when >= 0, the
// dropout_bits of these columns drawn earlier.
template <typename T>
__device__ __forceinline__ void epi_store_vec_b(const Epilogue& ep, int64_t row, int64_t col0, float* acc,
                                                const float (&bv)[Vec<T>::N], int32_t keep = -1) {
  constexpr int VE = Vec<T>::N;
  const int64_t cols = ep.cols;
  if (ep.mode == EPI_AGG) {
    if (ep.bias) {
#pragma unroll
      for (int i = 0; i < VE; ++i)
        if (col0 + i < cols) acc[i] += bv[i];
    }
    if (ep.relu) {
#pragma unroll
      for (int i = 0; i < VE; ++i) acc[i] = acc[i] > 0.f ? acc[i] : 0.f;
      if (ep.dropout) {
        const uint32_t kb = keep >= 0 ? (uint32_t)keep : dropout_bits<VE>(ep, row, col0);
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[i] = (kb >> i) & 1u ? acc[i] * ep.keep_scale : 0.f;
      }
    }
  }
  bool bad = false;
  uint4 raw;
  T* e = reinterpret_cast<T*>(&raw);
#pragma unroll
  for (int i = 0; i < VE; ++i) {
    float z = (col0 + i < cols) ? acc[i] : 0.f;
    e[i] = from_f32<T>(z);
    bad |= !finite_f32(to_f32<T>(e[i]));
  }
  stg16(reinterpret_cast<T*>(ep.out) + row * ep.ldo + col0, raw);
  if (bad) raise_flag(ep.flag);
}

// The same, loading the bias of these columns itself.
template <typename T>
__device__ __forceinline__ void epi_store_vec(const Epilogue& ep, int64_t row, int64_t col0, float* acc,
                                              int32_t keep = -1) {
  float bv[Vec<T>::N];
  epi_load_bias<T>(ep, col0, bv);
  epi_store_vec_b<T>(ep, row, col0, acc, bv, keep);
}

}  // namespace gcn

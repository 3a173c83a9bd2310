// Precision levels of Section "Background and Motivation" beyond the O2
// path of the layer kernels:
//
//  * cast_kernel: conversion of a strided block between storage types, the
//    per-operation casts of the O1 cast lists (GEMM-class operations take
//    16-bit copies of their fp32 operands, the loss takes an fp32 copy of
//    16-bit logits).  Eight elements per work-item, 16-byte loads and
//    stores, round-to-nearest-even; HBM-bound.
//  * adam_half_kernel: level O3, Adam with the parameters and both moments
//    held in 16 bits, no master copy and no loss scale.  Every elementwise
//    operation is evaluated in fp32 (one rounding per arithmetic operation,
//    no fused multiply-add) from 16-bit operands and rounded back, so the
//    moments and the update underflow and overflow exactly where 16-bit
//    tensors would.
#include "internal.h"

namespace gcn {

namespace {

template <typename S, typename D>
__global__ __launch_bounds__(256) void cast_kernel(int64_t rows, int64_t cols, const S* __restrict__ src,
                                                   int64_t lds, D* __restrict__ dst, int64_t ldd,
                                                   int32_t* flag, int64_t zcols) {
  const int64_t cpr = (zcols + 7) >> 3;  // 8-element chunks per row
  const int64_t total = rows * cpr;
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = rows == 1 ? 0 : i / cpr;
    const int64_t c0 = (i - r * cpr) << 3;
    const S* sp = src + r * lds + c0;
    D* dp = dst + r * ldd + c0;
    float x[8];
    if (c0 >= cols) {                    // zero padding [cols, zcols)
      const int m = (int)min<int64_t>(8, zcols - c0);
      for (int k = 0; k < m; ++k) dp[k] = from_f32<D>(0.f);
    } else if (c0 + 8 <= cols) {
      if constexpr (sizeof(S) == 4) {
        unpack<float>(ldg16(sp), x);
        unpack<float>(ldg16(sp + 4), x + 4);
      } else {
        unpack<S>(ldg16(sp), x);
      }
      D y[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        y[k] = from_f32<D>(x[k]);
        bad |= !finite_f32(to_f32<D>(y[k]));
      }
      if constexpr (sizeof(D) == 4) {
        stg16(dp, *reinterpret_cast<const uint4*>(y));
        stg16(dp + 4, *reinterpret_cast<const uint4*>(y + 4));
      } else {
        stg16(dp, *reinterpret_cast<const uint4*>(y));
      }
    } else {
      const int m = (int)(cols - c0);
      for (int k = 0; k < m; ++k) {
        const D y = from_f32<D>(to_f32<S>(sp[k]));
        dp[k] = y;
        bad |= !finite_f32(to_f32<D>(y));
      }
      const int mz = (int)min<int64_t>(8, zcols - c0);
      for (int k = m; k < mz; ++k) dp[k] = from_f32<D>(0.f);
    }
  }
  if (bad) raise_flag(flag);
}

template <typename S, typename D>
hipError_t cast_t(int64_t rows, int64_t cols, const void* src, int64_t lds, void* dst, int64_t ldd, int32_t* flag,
                  hipStream_t s, int64_t zcols) {
  const int64_t chunks = rows * ((zcols + 7) >> 3);
  int64_t blocks = (chunks + 255) / 256;
  if (blocks > (int64_t)1 << 16) blocks = (int64_t)1 << 16;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((cast_kernel<S, D>), dim3((unsigned)blocks), dim3(256), 0, s, rows, cols,
                     reinterpret_cast<const S*>(src), lds, reinterpret_cast<D*>(dst), ldd, flag, zcols);
  return hipGetLastError();
}

template <typename S>
hipError_t cast_from(int dst_prec, int64_t rows, int64_t cols, const void* src, int64_t lds, void* dst, int64_t ldd,
                     int32_t* flag, hipStream_t s, int64_t zcols) {
  switch (dst_prec) {
    case 0: return cast_t<S, float>(rows, cols, src, lds, dst, ldd, flag, s, zcols);
    case 1: return cast_t<S, f16>(rows, cols, src, lds, dst, ldd, flag, s, zcols);
    case 2: return cast_t<S, bf16>(rows, cols, src, lds, dst, ldd, flag, s, zcols);
  }
  return hipErrorInvalidValue;
}

// r(): one elementwise result rounded to the storage type T.
template <typename T>
__device__ __forceinline__ float rnd(float x) { return to_f32<T>(from_f32<T>(x)); }

template <typename T>
__global__ __launch_bounds__(256) void adam_half_kernel(int64_t count, T* __restrict__ w, const float* __restrict__ g,
                                                        T* __restrict__ m, T* __restrict__ v,
                                                        float* __restrict__ widened, AdamHyper hp,
                                                        const ScalerState* __restrict__ st) {
  // one fp32 rounding per arithmetic operation: no fused multiply-add
#pragma clang fp contract(off)
  const double t = (double)(st->step + 1);
  const float bc1 = (float)(1.0 - pow((double)hp.beta1, t));   // 1 - b^t, then rounded once
  const float bc2 = (float)(1.0 - pow((double)hp.beta2, t));
  const float c1 = 1.f - hp.beta1, c2 = 1.f - hp.beta2;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
    const float gi = rnd<T>(g[i]);
    const float mi = rnd<T>(hp.beta1 * to_f32<T>(m[i]) + c1 * gi);
    const float vi = rnd<T>(hp.beta2 * to_f32<T>(v[i]) + (c2 * gi) * gi);
    const float mh = rnd<T>(mi / bc1);
    const float vh = rnd<T>(vi / bc2);
    const float d = rnd<T>(rnd<T>(sqrtf(vh)) + hp.eps);
    const T wi = from_f32<T>(to_f32<T>(w[i]) - rnd<T>((hp.lr * mh) / d));
    m[i] = from_f32<T>(mi);
    v[i] = from_f32<T>(vi);
    w[i] = wi;
    if (widened) widened[i] = to_f32<T>(wi);
  }
}

// Step count and the flag: the step always applies; a step that carried a
// non-finite gradient is counted in `skipped` (as a diagnostic only).
__global__ void half_state_kernel(ScalerState* st, int32_t* flag) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  ScalerState s = *st;
  s.step += 1;
  if (*flag) s.skipped += 1;
  *st = s;
  *flag = 0;
}

__global__ __launch_bounds__(256) void nonfinite_kernel(int64_t count, const float* __restrict__ g, int32_t* flag) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
    bad |= !finite_f32(g[i]);
  if (bad) raise_flag(flag);
}

}  // namespace

hipError_t cast_launch(int src_prec, int dst_prec, int64_t rows, int64_t cols, const void* src, int64_t lds,
                       void* dst, int64_t ldd, int32_t* flag, hipStream_t s, int64_t zcols) {
  if (zcols < cols) zcols = cols;
  switch (src_prec) {
    case 0: return cast_from<float>(dst_prec, rows, cols, src, lds, dst, ldd, flag, s, zcols);
    case 1: return cast_from<f16>(dst_prec, rows, cols, src, lds, dst, ldd, flag, s, zcols);
    case 2: return cast_from<bf16>(dst_prec, rows, cols, src, lds, dst, ldd, flag, s, zcols);
  }
  return hipErrorInvalidValue;
}

hipError_t adam_half_launch(int64_t count, void* w, const float* grad, void* m, void* v, float* widened, int prec,
                            const AdamHyper& hp, ScalerState* state, int32_t* flag, hipStream_t s) {
  int64_t blocks = (count + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(nonfinite_kernel, dim3((unsigned)blocks), dim3(256), 0, s, count, grad, flag);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (prec) {
    case 1:
      hipLaunchKernelGGL(adam_half_kernel<f16>, dim3((unsigned)blocks), dim3(256), 0, s, count, (f16*)w, grad,
                         (f16*)m, (f16*)v, widened, hp, state);
      break;
    case 2:
      hipLaunchKernelGGL(adam_half_kernel<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, count, (bf16*)w, grad,
                         (bf16*)m, (bf16*)v, widened, hp, state);
      break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(half_state_kernel, dim3(1), dim3(64), 0, s, state, flag);
  return hipGetLastError();
}

}  // namespace gcn

// Optimiser step with fp32 master weights and dynamic loss scaling, the O2
// scheme of the paper's Section "Background and Motivation": gradients of
// the scaled loss are checked for overflow, unscaled, and applied by Adam
// (Kingma & Ba) to fp32 masters, whose 16-bit copies feed the next forward
// pass.  All state stays on the device: three launches, no host sync.
#include "internal.h"

namespace gcn {

namespace {

__global__ __launch_bounds__(256) void grad_check_kernel(int64_t count, const float* __restrict__ g, int32_t* flag) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
    bad |= !finite_f32(g[i]);
  if (bad) raise_flag(flag);
}

template <typename T>
__global__ __launch_bounds__(256) void adam_kernel(int64_t count, float* __restrict__ w, const float* __restrict__ g,
                                                   float* __restrict__ m, float* __restrict__ v, T* __restrict__ working,
                                                   AdamHyper hp, const ScalerState* __restrict__ st,
                                                   const int32_t* __restrict__ flag) {
  if (*flag) return;
  const float inv_scale = 1.f / st->scale;
  const float t = (float)(st->step + 1);
  const float bc1 = 1.f - powf(hp.beta1, t);
  const float bc2 = 1.f - powf(hp.beta2, t);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
    const float gi = g[i] * inv_scale;
    const float mi = hp.beta1 * m[i] + (1.f - hp.beta1) * gi;
    const float vi = hp.beta2 * v[i] + (1.f - hp.beta2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    const float wi = w[i] - hp.lr * (mi / bc1) / (sqrtf(vi / bc2) + hp.eps);
    w[i] = wi;
    if (working) working[i] = from_f32<T>(wi);
  }
}

__global__ void scaler_kernel(AdamHyper hp, ScalerState* st, int32_t* flag) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  ScalerState s = *st;
  if (*flag) {
    s.scale = fmaxf(s.scale * hp.backoff, hp.min_scale);
    s.good_steps = 0;
    s.skipped += 1;
  } else {
    s.step += 1;
    s.good_steps += 1;
    if (s.good_steps >= hp.interval) {
      s.scale = fminf(s.scale * hp.growth, hp.max_scale);
      s.good_steps = 0;
    }
  }
  *st = s;
  *flag = 0;
}

}  // namespace

hipError_t optimizer_launch(int64_t count, float* master, const float* grad, float* m, float* v, void* working,
                            int prec, const AdamHyper& hp, ScalerState* state, int32_t* flag, hipStream_t s) {
  int64_t blocks = (count + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(grad_check_kernel, dim3((unsigned)blocks), dim3(256), 0, s, count, grad, flag);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (prec) {
    case 0: hipLaunchKernelGGL(adam_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, s, count, master, grad, m, v, (float*)working, hp, state, flag); break;
    case 1: hipLaunchKernelGGL(adam_kernel<f16>, dim3((unsigned)blocks), dim3(256), 0, s, count, master, grad, m, v, (f16*)working, hp, state, flag); break;
    case 2: hipLaunchKernelGGL(adam_kernel<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, count, master, grad, m, v, (bf16*)working, hp, state, flag); break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scaler_kernel, dim3(1), dim3(64), 0, s, hp, state, flag);
  return hipGetLastError();
}

}  // namespace gcn

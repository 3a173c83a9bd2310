// Masked softmax cross-entropy for vertex classification, fused with the
// scaled gradient: one read of the logits, one write of dlogits, one
// exponential per element (exp(z - max) serves the sum and, times the
// reciprocal of the sum, the softmax).  A group of
// LPR lanes owns one row (16 bytes of classes per lane); max, sum of
// exponentials, label logit and arg-max are reduced with lane shuffles
// inside the group.  Per-row losses are summed per workgroup in row order
// and the workgroup sums in a second fixed-order pass (deterministic).
#include "internal.h"

namespace gcn {

namespace {

struct LossParams {
  int64_t n, C, ld;
  const void* logits;
  const int32_t* labels;
  const uint8_t* mask;
  float inv_count;
  const float* loss_scale;
  void* dlogits;
  float* part_loss;     // [blocks]
  int32_t* part_corr;   // [blocks]
  int32_t* flag;
};

template <int LPR>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
template <int LPR>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Rows handled per lane group and iteration (R): all their loads go out
// before any is used (one memory latency per iteration instead of one per
// row).  R = 4 when one row per iteration would give more than
// LOSS_R4_GROUPS workgroups, else R = 1 (fewer rows keep more workgroups).
constexpr int64_t LOSS_R4_GROUPS = 16384;

template <typename T, int LPR, int LOSS_R>
__global__ __launch_bounds__(256) void softmax_ce_kernel(LossParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  constexpr int RG = 4 * G;                          // rows per workgroup and sub-step
  __shared__ float s_loss[RG];
  __shared__ int32_t s_corr[RG];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int slot = wave * G + g;
  const int64_t col0 = (int64_t)li * VE;
  const bool col_ok = col0 < p.C;
  const T* __restrict__ logits = reinterpret_cast<const T*>(p.logits);
  // the workgroup walks blocks of LOSS_R * RG rows: blockIdx.x, blockIdx.x
  // + gridDim.x, ...; a slot takes rows base + r * RG + slot, r = 0 .. LOSS_R - 1
  // (in that order for the per-slot sums)
  float acc_loss = 0.f;
  int32_t acc_corr = 0;
  const float sc = (p.loss_scale ? *p.loss_scale : 1.f) * p.inv_count;
  for (int64_t base = (int64_t)blockIdx.x * (LOSS_R * RG); base < p.n; base += (int64_t)gridDim.x * (LOSS_R * RG)) {
    uint4 raw[LOSS_R];
    int32_t lab[LOSS_R];
    uint8_t msk[LOSS_R];
#pragma unroll
    for (int r = 0; r < LOSS_R; ++r) {
      int64_t row = base + r * RG + slot;
      row = row < p.n ? row : p.n - 1;               // in bounds; not counted below
      raw[r] = ldg16(logits + row * p.ld + (col_ok ? col0 : 0));
      lab[r] = p.labels[row];
      msk[r] = p.mask ? p.mask[row] : (uint8_t)1;
    }
#pragma unroll
    for (int r = 0; r < LOSS_R; ++r) {
      const int64_t row = base + r * RG + slot;
      const bool row_ok = row < p.n;
      float x[VE], z[VE];
      unpack<T>(raw[r], x);
#pragma unroll
      for (int i = 0; i < VE; ++i) z[i] = (row_ok && col0 + i < p.C) ? x[i] : -INFINITY;
      // row maximum and arg-max (lowest index on ties)
      float mx = -INFINITY;
      int am = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < VE; ++i)
        if (col0 + i < p.C && (z[i] > mx || am == 0x7fffffff)) { mx = z[i]; am = (int)(col0 + i); }
#pragma unroll
      for (int o = LPR / 2; o > 0; o >>= 1) {
        const float om = __shfl_xor(mx, o);
        const int oa = __shfl_xor(am, o);
        if (om > mx || (om == mx && oa < am)) { mx = om; am = oa; }
      }
      const float rmax = mx;
      // exp(z - max) once per element: the sum of exponentials and, scaled
      // by its reciprocal, the softmax of the gradient
      float ez[VE];
      float se = 0.f;
#pragma unroll
      for (int i = 0; i < VE; ++i) {
        ez[i] = (col0 + i < p.C) ? expf(z[i] - rmax) : 0.f;
        se += ez[i];
      }
      se = group_sum<LPR>(se);
      const float lse = rmax + logf(se);
      const float inv_se = 1.f / se;
      const int32_t y = row_ok ? lab[r] : 0;
      float zy = 0.f;
#pragma unroll
      for (int i = 0; i < VE; ++i)
        if (col0 + i == y) zy = z[i];
      zy = group_sum<LPR>(zy);
      const bool in_mask = row_ok && msk[r] != 0;
      if (row_ok && col_ok) {
        float d[VE];
#pragma unroll
        for (int i = 0; i < VE; ++i) {
          const int64_t c = col0 + i;
          if (c < p.C && in_mask) d[i] = (ez[i] * inv_se - (c == y ? 1.f : 0.f)) * sc;
          else d[i] = 0.f;
        }
        uint4 o = pack<T>(d);
        stg16(reinterpret_cast<T*>(p.dlogits) + row * p.ld + col0, o);
        bool bad = false;
        const T* e = reinterpret_cast<const T*>(&o);
#pragma unroll
        for (int i = 0; i < VE; ++i) bad |= !finite_f32(to_f32<T>(e[i]));
        if (bad) raise_flag(p.flag);
      }
      acc_loss += in_mask ? (lse - zy) : 0.f;
      acc_corr += (in_mask && am == y) ? 1 : 0;
    }
  }
  if (li == 0) {
    s_loss[slot] = acc_loss;
    s_corr[slot] = acc_corr;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.f;
    int32_t c = 0;
    for (int i = 0; i < RG; ++i) { a += s_loss[i]; c += s_corr[i]; }
    p.part_loss[blockIdx.x] = a;
    p.part_corr[blockIdx.x] = c;
  }
}

__global__ __launch_bounds__(256) void loss_final_kernel(const float* __restrict__ part, const int32_t* __restrict__ corr,
                                                         int64_t nb, float inv_count, float* loss, int32_t* n_correct,
                                                         int32_t* flag) {
  __shared__ float sl[256];
  __shared__ int32_t sc[256];
  float a = 0.f;
  int32_t c = 0;
  for (int64_t i = threadIdx.x; i < nb; i += 256) { a += part[i]; c += corr[i]; }
  sl[threadIdx.x] = a;
  sc[threadIdx.x] = c;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) { sl[threadIdx.x] += sl[threadIdx.x + s]; sc[threadIdx.x] += sc[threadIdx.x + s]; }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float l = sl[0] * inv_count;
    *loss = l;
    if (n_correct) *n_correct = sc[0];
    if (!finite_f32(l)) raise_flag(flag);
  }
}

// Workgroups of the loss kernel: one per row group up to 65536 (each then
// walks several groups).
int64_t loss_blocks(int64_t n, int64_t rows_per_group) {
  const int64_t nb = (n + rows_per_group - 1) / rows_per_group;
  return nb < 65536 ? nb : 65536;
}

int loss_rows_per_iter(int64_t n, int64_t rows_per_group) {
  return (n + rows_per_group - 1) / rows_per_group > LOSS_R4_GROUPS ? 4 : 1;
}

template <typename T, int LPR>
hipError_t launch_cfg(const LossParams& p, hipStream_t s) {
  constexpr int64_t RG = 4 * (64 / LPR);
  if (loss_rows_per_iter(p.n, RG) == 4)
    hipLaunchKernelGGL((softmax_ce_kernel<T, LPR, 4>), dim3((unsigned)loss_blocks(p.n, 4 * RG)), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((softmax_ce_kernel<T, LPR, 1>), dim3((unsigned)loss_blocks(p.n, RG)), dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_t(const LossParams& p, hipStream_t s) {
  constexpr int VE = Vec<T>::N;
  const int64_t nvec = (p.C + VE - 1) / VE;
  if (nvec <= 1) return launch_cfg<T, 1>(p, s);
  if (nvec <= 2) return launch_cfg<T, 2>(p, s);
  if (nvec <= 4) return launch_cfg<T, 4>(p, s);
  if (nvec <= 8) return launch_cfg<T, 8>(p, s);
  if (nvec <= 16) return launch_cfg<T, 16>(p, s);
  if (nvec <= 32) return launch_cfg<T, 32>(p, s);
  return launch_cfg<T, 64>(p, s);
}

// Rows per workgroup iteration for n rows (as the launch chooses).
int64_t rows_per_block(int prec, int64_t C, int64_t n) {
  const int VE = prec == 0 ? 4 : 8;
  const int64_t nvec = (C + VE - 1) / VE;
  int l = 1;
  while (l < nvec && l < 64) l <<= 1;
  const int64_t rg = 4 * (64 / l);
  return loss_rows_per_iter(n, rg) * rg;
}

}  // namespace

size_t loss_workspace_bytes(int64_t n, int64_t C) {
  const int64_t nb = (n + rows_per_block(0, C, n) - 1) / rows_per_block(0, C, n) + 1;   // fp32 needs the most blocks
  const int64_t nb16 = (n + rows_per_block(1, C, n) - 1) / rows_per_block(1, C, n) + 1;
  const int64_t m = nb > nb16 ? nb : nb16;
  return (size_t)m * (sizeof(float) + sizeof(int32_t)) + 256;
}

hipError_t loss_launch(int prec, int64_t n, int64_t C, int64_t ld, const void* logits, const int32_t* labels,
                       const uint8_t* mask, int64_t n_mask, const float* loss_scale, float* loss, void* dlogits,
                       int32_t* n_correct, int32_t* flag, void* ws, hipStream_t s) {
  const int64_t nb = loss_blocks(n, rows_per_block(prec, C, n));
  LossParams p;
  p.n = n; p.C = C; p.ld = ld; p.logits = logits; p.labels = labels; p.mask = mask;
  p.inv_count = 1.f / (float)n_mask;
  p.loss_scale = loss_scale; p.dlogits = dlogits;
  p.part_loss = reinterpret_cast<float*>(ws);
  p.part_corr = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(ws) + ((nb * sizeof(float) + 255) & ~size_t(255)));
  p.flag = flag;
  hipError_t e;
  switch (prec) {
    case 0: e = launch_t<float>(p, s); break;
    case 1: e = launch_t<f16>(p, s); break;
    case 2: e = launch_t<bf16>(p, s); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(256), 0, s, p.part_loss, p.part_corr, nb, p.inv_count, loss,
                     n_correct, flag);
  return hipGetLastError();
}

}  // namespace gcn

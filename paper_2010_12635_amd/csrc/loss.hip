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
  float* part_cs;       // [blocks][ldcs] column sums of the stored dlogits, or NULL
  int64_t ldcs;         // row stride of part_cs: C rounded up to 8
  int32_t* flag;
};

// Reductions over a lane group of LPR lanes (aligned, a power of two),
// every lane ending with the result: lanes exchange values through DPP
// moves inside rows of 16 lanes (quad permutations, then the half-row and
// row mirrors, each pairing a lane with one of the other half once the
// halves agree), across rows through lane shuffles.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}
constexpr int DPP_XOR1 = 0xB1;         // quad_perm [1, 0, 3, 2]
constexpr int DPP_XOR2 = 0x4E;         // quad_perm [2, 3, 0, 1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <-> 7 - i of each 8
constexpr int DPP_MIRROR = 0x140;      // lane i <-> 15 - i of each 16

template <int LPR>
__device__ __forceinline__ float group_sum(float v) {
  if (LPR >= 2) v += dpp_f<DPP_XOR1>(v);
  if (LPR >= 4) v += dpp_f<DPP_XOR2>(v);
  if (LPR >= 8) v += dpp_f<DPP_HALF_MIRROR>(v);
  if (LPR >= 16) v += dpp_f<DPP_MIRROR>(v);
  if (LPR >= 32) v += __shfl_xor(v, 16);
  if (LPR >= 64) v += __shfl_xor(v, 32);
  return v;
}

// (maximum, lowest index among the maxima) over the group
__device__ __forceinline__ void argmax_step(float& mx, int& am, float om, int oa) {
  const bool take = om > mx || (om == mx && oa < am);
  mx = take ? om : mx;
  am = take ? oa : am;
}
template <int LPR>
__device__ __forceinline__ void group_argmax(float& mx, int& am) {
  if (LPR >= 2) argmax_step(mx, am, dpp_f<DPP_XOR1>(mx), dpp_i<DPP_XOR1>(am));
  if (LPR >= 4) argmax_step(mx, am, dpp_f<DPP_XOR2>(mx), dpp_i<DPP_XOR2>(am));
  if (LPR >= 8) argmax_step(mx, am, dpp_f<DPP_HALF_MIRROR>(mx), dpp_i<DPP_HALF_MIRROR>(am));
  if (LPR >= 16) argmax_step(mx, am, dpp_f<DPP_MIRROR>(mx), dpp_i<DPP_MIRROR>(am));
  if (LPR >= 32) argmax_step(mx, am, __shfl_xor(mx, 16), __shfl_xor(am, 16));
  if (LPR >= 64) argmax_step(mx, am, __shfl_xor(mx, 32), __shfl_xor(am, 32));
}

// Rows handled per lane group and iteration (R): all their loads go out
// before any is used (one memory latency per iteration instead of one per
// row).  R = 4 when one row per iteration would give more than
// LOSS_R4_GROUPS workgroups, else R = 1 (fewer rows keep more workgroups).
constexpr int64_t LOSS_R4_GROUPS = 16384;

template <typename T> __device__ __forceinline__ float max_finite();
template <> __device__ __forceinline__ float max_finite<float>() { return 3.40282347e38f; }
template <> __device__ __forceinline__ float max_finite<f16>() { return 65504.f; }
template <> __device__ __forceinline__ float max_finite<bf16>() { return 3.38953139e38f; }

// Any non-finite element among the VE packed values (exponent field all ones).
template <typename T> __device__ __forceinline__ bool packed_nonfinite(uint4 o);
template <> __device__ __forceinline__ bool packed_nonfinite<float>(uint4 o) {
  const uint32_t e = 0x7f800000u;
  return (o.x & e) == e || (o.y & e) == e || (o.z & e) == e || (o.w & e) == e;
}
template <uint32_t E>
__device__ __forceinline__ bool half_pair_nonfinite(uint32_t w) {
  return (w & E) == E || (w & (E << 16)) == (E << 16);
}
template <> __device__ __forceinline__ bool packed_nonfinite<f16>(uint4 o) {
  return half_pair_nonfinite<0x7c00u>(o.x) || half_pair_nonfinite<0x7c00u>(o.y) ||
         half_pair_nonfinite<0x7c00u>(o.z) || half_pair_nonfinite<0x7c00u>(o.w);
}
template <> __device__ __forceinline__ bool packed_nonfinite<bf16>(uint4 o) {
  return half_pair_nonfinite<0x7f80u>(o.x) || half_pair_nonfinite<0x7f80u>(o.y) ||
         half_pair_nonfinite<0x7f80u>(o.z) || half_pair_nonfinite<0x7f80u>(o.w);
}

// FULL: C = LPR * VE, so every lane holds VE classes and no element needs
// a bounds test.  The exponentials use the hardware
// base-2 exponential of (z - max) log2(e) (relative error a few 1e-7 for the
// arguments <= 0 that occur here).
template <typename T, int LPR, int LOSS_R, bool FULL>
__global__ __launch_bounds__(256) void softmax_ce_kernel(LossParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  constexpr int RG = 4 * G;                          // rows per workgroup and sub-step
  __shared__ float s_loss[RG];
  __shared__ int32_t s_corr[RG];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int slot = wave * G + g;
  const int col0 = li * VE;
  const bool col_ok = FULL || col0 < p.C;
  const int nv = FULL ? VE : (int)(p.C - col0 < VE ? (p.C - col0 > 0 ? p.C - col0 : 0) : VE);   // classes of this lane
  const T* __restrict__ logits = reinterpret_cast<const T*>(p.logits);
  // the workgroup walks blocks of LOSS_R * RG rows: blockIdx.x, blockIdx.x
  // + gridDim.x, ...; a slot takes rows base + r * RG + slot, r = 0 .. LOSS_R - 1
  // (in that order for the per-slot sums)
  float acc_loss = 0.f;
  int32_t acc_corr = 0;
  float acc_cs[VE];                                 // this lane's classes over its rows (as stored)
#pragma unroll
  for (int i = 0; i < VE; ++i) acc_cs[i] = 0.f;
  const bool want_cs = p.part_cs != nullptr;
  const float sc = (p.loss_scale ? *p.loss_scale : 1.f) * p.inv_count;
  constexpr float LOG2E = 1.4426950408889634f;
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
      float z[VE];
      unpack<T>(raw[r], z);
      if (!FULL) {
#pragma unroll
        for (int i = 0; i < VE; ++i) z[i] = i < nv ? z[i] : -INFINITY;
      }
      // row maximum and arg-max (lowest index on ties; a lane without
      // classes offers -inf at an index past every class)
      float mx = z[0];
      int am = col_ok ? col0 : 0x7fffffff;
#pragma unroll
      for (int i = 1; i < VE; ++i) {
        const bool gt = z[i] > mx;
        mx = gt ? z[i] : mx;
        am = gt ? col0 + i : am;
      }
      group_argmax<LPR>(mx, am);
      const float mlog = mx * LOG2E;
      // exp(z - max) once per element: the sum of exponentials and, scaled
      // by its reciprocal, the softmax of the gradient
      float ez[VE];
      float se = 0.f;
#pragma unroll
      for (int i = 0; i < VE; ++i) {
        ez[i] = __builtin_amdgcn_exp2f(fmaf(z[i], LOG2E, -mlog));
        if (!FULL) ez[i] = i < nv ? ez[i] : 0.f;
        se += ez[i];
      }
      se = group_sum<LPR>(se);
      const float lse = mx + logf(se);
      const float inv_se = 1.f / se;
      const int32_t y = row_ok ? lab[r] : 0;
      const int ky = y - col0;                       // the label's element in this lane, if in [0, VE)
      float zy = 0.f;
#pragma unroll
      for (int i = 0; i < VE; ++i) zy = i == ky ? z[i] : zy;
      zy = group_sum<LPR>(zy);
      const bool in_mask = row_ok && msk[r] != 0;
      if (row_ok && col_ok) {
        float d[VE];
        const float s_in = in_mask ? sc : 0.f;
#pragma unroll
        for (int i = 0; i < VE; ++i) d[i] = (ez[i] * inv_se - (i == ky ? 1.f : 0.f)) * s_in;
        if (!FULL) {
#pragma unroll
          for (int i = 0; i < VE; ++i) d[i] = i < nv ? d[i] : 0.f;
        }
        const uint4 o = pack<T>(d);
        stg16(reinterpret_cast<T*>(p.dlogits) + row * p.ld + col0, o);
        if (want_cs) {
          float st[VE];
          unpack<T>(o, st);
#pragma unroll
          for (int i = 0; i < VE; ++i) acc_cs[i] += st[i];
        }
        // |d| <= |s_in| (softmax values lie in [0, 1]): with finite logits
        // (lse finite) and |s_in| at most the largest finite value of T no
        // element can overflow; otherwise every element is checked
        if (!(finite_f32(lse) && fabsf(s_in) <= max_finite<T>()) && packed_nonfinite<T>(o)) raise_flag(p.flag);
      }
      acc_loss += in_mask ? (lse - zy) : 0.f;
      acc_corr += (in_mask && am == y) ? 1 : 0;
    }
  }
  if (li == 0) {
    s_loss[slot] = acc_loss;
    s_corr[slot] = acc_corr;
  }
  __shared__ float s_cs[RG][LPR * VE];
  if (want_cs) {
#pragma unroll
    for (int i = 0; i < VE; ++i) s_cs[slot][li * VE + i] = acc_cs[i];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.f;
    int32_t c = 0;
    for (int i = 0; i < RG; ++i) { a += s_loss[i]; c += s_corr[i]; }
    p.part_loss[blockIdx.x] = a;
    p.part_corr[blockIdx.x] = c;
  }
  if (want_cs) {
    // the workgroup's column sums: its row slots added in slot order
    for (int cidx = threadIdx.x; cidx < p.C; cidx += 256) {
      float a = s_cs[0][cidx];
      for (int k = 1; k < RG; ++k) a += s_cs[k][cidx];
      p.part_cs[(int64_t)blockIdx.x * p.ldcs + cidx] = a;
    }
  }
}

// Thread t adds partials t, t + 256, ... in that order (eight loads in
// flight), then the 256 sums are added by a fixed tree.
__global__ __launch_bounds__(256) void loss_final_kernel(const float* __restrict__ part, const int32_t* __restrict__ corr,
                                                         int64_t nb, float inv_count, float* loss, int32_t* n_correct,
                                                         int32_t* flag) {
  __shared__ float sl[256];
  __shared__ int32_t sc[256];
  float a = 0.f;
  int32_t c = 0;
  int64_t i = threadIdx.x;
  for (; i + 7 * 256 < nb; i += 8 * 256) {
    float v[8];
    int32_t k[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { v[u] = part[i + u * 256]; k[u] = corr[i + u * 256]; }
#pragma unroll
    for (int u = 0; u < 8; ++u) { a += v[u]; c += k[u]; }
  }
  for (; i < nb; i += 256) { a += part[i]; c += corr[i]; }
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
// walks several groups).  Capping them at 2048 to bound the column-sum
// partials made the kernel slower on R-MAT scale 21 (105 -> 118 us) than
// the wider reduction of 16384 partials costs.
constexpr int64_t LOSS_MAX_BLOCKS = 65536;
int64_t loss_blocks(int64_t n, int64_t rows_per_group) {
  const int64_t nb = (n + rows_per_group - 1) / rows_per_group;
  return nb < LOSS_MAX_BLOCKS ? nb : LOSS_MAX_BLOCKS;
}

int loss_rows_per_iter(int64_t n, int64_t rows_per_group) {
  return (n + rows_per_group - 1) / rows_per_group > LOSS_R4_GROUPS ? 4 : 1;
}

template <typename T, int LPR, bool FULL>
hipError_t launch_full(const LossParams& p, hipStream_t s) {
  constexpr int64_t RG = 4 * (64 / LPR);
  if (loss_rows_per_iter(p.n, RG) == 4)
    hipLaunchKernelGGL((softmax_ce_kernel<T, LPR, 4, FULL>), dim3((unsigned)loss_blocks(p.n, 4 * RG)), dim3(256), 0, s,
                       p);
  else
    hipLaunchKernelGGL((softmax_ce_kernel<T, LPR, 1, FULL>), dim3((unsigned)loss_blocks(p.n, RG)), dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename T, int LPR>
hipError_t launch_cfg(const LossParams& p, hipStream_t s) {
  return p.C == LPR * Vec<T>::N ? launch_full<T, LPR, true>(p, s) : launch_full<T, LPR, false>(p, s);
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

// Workgroups of the softmax launch at most (fp32 needs the most).
int64_t loss_max_blocks(int64_t n, int64_t C) {
  const int64_t nb = loss_blocks(n, rows_per_block(0, C, n));
  const int64_t nb16 = loss_blocks(n, rows_per_block(1, C, n));
  return nb > nb16 ? nb : nb16;
}

// More column-sum partial rows than this are first summed in blocks of
// consecutive rows (one launch), then the blocks' rows (a second).
constexpr int64_t LOSS_CS_ONE_STAGE = 4096;

int64_t loss_cs_ld(int64_t C) { return (C + 7) / 8 * 8; }

// [loss partials][correct-count partials][column-sum partials (blocks x
// ldcs)][their block sums]
size_t loss_workspace_bytes(int64_t n, int64_t C) {
  const int64_t m = loss_max_blocks(n, C) + 1;
  const int64_t ldcs = loss_cs_ld(C);
  const size_t a = ((size_t)m * sizeof(float) + 255) & ~size_t(255);
  const size_t b = ((size_t)m * sizeof(int32_t) + 255) & ~size_t(255);
  const size_t c = ((size_t)m * (size_t)ldcs * sizeof(float) + 255) & ~size_t(255);
  return a + b + c + (size_t)colsum_partials_floats(m, ldcs) * sizeof(float) + 256;
}

hipError_t loss_launch(int prec, int64_t n, int64_t C, int64_t ld, const void* logits, const int32_t* labels,
                       const uint8_t* mask, int64_t n_mask, const float* loss_scale, float* loss, void* dlogits,
                       float* dlogits_colsum, int32_t* n_correct, int32_t* flag, void* ws, hipStream_t s) {
  const int64_t nb = loss_blocks(n, rows_per_block(prec, C, n));
  const int64_t m = loss_max_blocks(n, C) + 1;
  LossParams p;
  p.n = n; p.C = C; p.ld = ld; p.logits = logits; p.labels = labels; p.mask = mask;
  p.inv_count = 1.f / (float)n_mask;
  p.loss_scale = loss_scale; p.dlogits = dlogits;
  char* w = reinterpret_cast<char*>(ws);
  p.part_loss = reinterpret_cast<float*>(w);
  w += ((size_t)m * sizeof(float) + 255) & ~size_t(255);
  p.part_corr = reinterpret_cast<int32_t*>(w);
  w += ((size_t)m * sizeof(int32_t) + 255) & ~size_t(255);
  p.part_cs = dlogits_colsum ? reinterpret_cast<float*>(w) : nullptr;
  p.ldcs = loss_cs_ld(C);
  w += ((size_t)m * (size_t)p.ldcs * sizeof(float) + 255) & ~size_t(255);
  float* cs_blocks = reinterpret_cast<float*>(w);
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
  e = hipGetLastError();
  if (e != hipSuccess || !dlogits_colsum) return e;
  // the workgroups' column sums added in a fixed order; classes [C, ld) get 0
  Epilogue eb{};
  eb.out = dlogits_colsum; eb.ldo = ld; eb.rows = 1; eb.cols = C; eb.mode = EPI_F32; eb.flag = flag;
  eb.keep_scale = 1.f;
  if (nb <= LOSS_CS_ONE_STAGE)
    return reduce_partials2(prec, make_job_ld(p.part_cs, (int)nb, 1, C, p.ldcs, eb), nullptr, s);
  // many workgroups (R-MAT scale 21: 16384): blocks of consecutive partial
  // rows first, with coalesced row reads over the whole chip, then the
  // blocks' sums (one launch of one output per workgroup reading a column
  // each took 24 us in fp16 and 41 us in fp32)
  int blocks = 0;
  e = colsum_partial_launch(0, p.part_cs, nb, C, p.ldcs, cs_blocks, p.ldcs, &blocks, s);
  if (e != hipSuccess) return e;
  return reduce_partials2(prec, make_job_ld(cs_blocks, blocks, 1, C, p.ldcs, eb), nullptr, s);
}

}  // namespace gcn

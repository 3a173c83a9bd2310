// Link prediction with the graph auto-encoder of Section "Graph
// Auto-Encoders", Eq. (2): A' = sigmoid(Z Z^T), evaluated on sampled vertex
// pairs rather than on all n^2 entries.
//
//  * sample_pairs_kernel: one Philox-4x64-10 block per pair (key (seed,
//    PAIR_STREAM), counter (k, epoch, 0, 0)); positives are training edges,
//    negatives uniform pairs of distinct vertices.
//  * pair_loss_kernel: a group of LPR lanes per pair gathers the two rows of
//    Z as 16-byte slices, reduces their inner product with shuffles, and
//    takes the logistic loss and its gradient g_k in fp32.  Per-pair losses
//    are summed per workgroup in a fixed order, then across workgroups.
//  * pair backward: the pairs are bucketed by endpoint (count, scan,
//    scatter, per-row sort by pair index), then a lane group per row sums
//    g_k Z[other endpoint] in increasing k: dZ is run-to-run identical
//    without floating-point atomics.
//  * pair_metrics_kernel: exact AUC and AP of held-out pairs by counting,
//    for every positive, the scores below / equal / above it (O(P (P + N))
//    comparisons through LDS tiles), then fixed-order sums.
#include "internal.h"

namespace gcn {

namespace {

constexpr uint64_t PAIR_STREAM = 0x50414952ull;   // second key word of the pair sampler

__global__ __launch_bounds__(256) void sample_pairs_kernel(int64_t n, const int32_t* __restrict__ edge_u,
                                                           const int32_t* __restrict__ edge_v, int64_t n_edges,
                                                           int64_t n_pos, int64_t total, uint64_t seed, uint64_t epoch,
                                                           int32_t* __restrict__ pu, int32_t* __restrict__ pv) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += (int64_t)gridDim.x * blockDim.x) {
    const Philox8 o = philox4x64_10((uint64_t)k, epoch, 0, 0, seed, PAIR_STREAM);
    if (k < n_pos) {
      const int64_t e = (int64_t)(o.w[0] % (uint64_t)n_edges);
      pu[k] = edge_u[e];
      pv[k] = edge_v[e];
    } else {
      const uint64_t u = o.w[0] % (uint64_t)n;
      const uint64_t v = (u + 1 + o.w[1] % (uint64_t)(n - 1)) % (uint64_t)n;
      pu[k] = (int32_t)u;
      pv[k] = (int32_t)v;
    }
  }
}

__device__ __forceinline__ float softplus_f(float x) { return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x))); }
__device__ __forceinline__ float sigmoid_f(float x) {
  if (x >= 0.f) return 1.f / (1.f + expf(-x));
  const float e = expf(x);
  return e / (1.f + e);
}

struct PairLossParams {
  int64_t n, F, ld;
  const void* Z;
  const int32_t* pu;
  const int32_t* pv;
  int64_t n_pos, total;
  float inv_total;
  const float* loss_scale;
  float* scores;
  float* g;
  float* part;          // [gridDim.x]
  int32_t* flag;
};

template <typename T, int LPR>
__global__ __launch_bounds__(256) void pair_loss_kernel(PairLossParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  __shared__ float s_loss[4 * G];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / LPR, li = lane % LPR;
  const int slot = wave * G + g;
  const int64_t col0 = (int64_t)li * VE;
  const int64_t nf = p.F - col0;
  const int vc = nf <= 0 ? 0 : nf >= VE ? VE : (int)nf;   // live elements of this lane's slice
  const float scale = (p.loss_scale ? *p.loss_scale : 1.f) * p.inv_total;
  const T* Z = reinterpret_cast<const T*>(p.Z);
  float acc_loss = 0.f;
  for (int64_t base = (int64_t)blockIdx.x * (4 * G); base < p.total; base += (int64_t)gridDim.x * (4 * G)) {
    const int64_t k = base + slot;
    const bool live = k < p.total;
    const int32_t u = live ? p.pu[k] : 0, v = live ? p.pv[k] : 0;
    const bool ok = live && u >= 0 && v >= 0 && u < p.n && v < p.n;
    float dot = 0.f;
    if (ok && vc > 0) {
      float a[VE], b[VE];
      unpack<T>(ldg16(Z + (int64_t)u * p.ld + col0), a);
      unpack<T>(ldg16(Z + (int64_t)v * p.ld + col0), b);
#pragma unroll
      for (int i = 0; i < VE; ++i)
        if (i < vc) dot = fmaf(a[i], b[i], dot);
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
    if (li == 0 && live) {
      const float y = k < p.n_pos ? 1.f : 0.f;
      if (ok) {
        const float gk = (sigmoid_f(dot) - y) * scale;
        acc_loss += softplus_f(dot) - y * dot;
        if (p.scores) p.scores[k] = dot;
        p.g[k] = gk;
        if (!finite_f32(gk) || !finite_f32(dot)) raise_flag(p.flag);
      } else {   // vertex id outside [0, n): the pair is skipped
        if (p.scores) p.scores[k] = __int_as_float(0x7fc00000);
        p.g[k] = 0.f;
        raise_flag(p.flag);
      }
    }
  }
  if (li == 0) s_loss[slot] = acc_loss;
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.f;
    for (int i = 0; i < 4 * G; ++i) a += s_loss[i];
    p.part[blockIdx.x] = a;
  }
}

__global__ __launch_bounds__(256) void pair_loss_final_kernel(const float* __restrict__ part, int64_t nb, float inv_total,
                                                              float* loss, int32_t* flag) {
  __shared__ float sl[256];
  float a = 0.f;
  for (int64_t i = threadIdx.x; i < nb; i += 256) a += part[i];
  sl[threadIdx.x] = a;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) sl[threadIdx.x] += sl[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float l = sl[0] * inv_total;
    *loss = l;
    if (!finite_f32(l)) raise_flag(flag);
  }
}

int lpr_for(int prec, int64_t F) {
  const int VE = prec == 0 ? 4 : 8;
  const int64_t nvec = (F + VE - 1) / VE;
  int l = 1;
  while (l < nvec && l < 64) l <<= 1;
  return l;
}

int64_t capped_blocks(int64_t items, int64_t per_block) {
  const int64_t b = (items + per_block - 1) / per_block;
  return b < 1 ? 1 : b < 65536 ? b : 65536;
}

template <typename T>
hipError_t pair_loss_t(PairLossParams p, int lpr, hipStream_t s, int64_t* nb_out) {
  const int64_t nb = capped_blocks(p.total, 4 * (64 / lpr));
  *nb_out = nb;
#define PL(L) hipLaunchKernelGGL((pair_loss_kernel<T, L>), dim3((unsigned)nb), dim3(256), 0, s, p); break;
  switch (lpr) {
    case 1: PL(1)
    case 2: PL(2)
    case 4: PL(4)
    case 8: PL(8)
    case 16: PL(16)
    case 32: PL(32)
    default: PL(64)
  }
#undef PL
  return hipGetLastError();
}

// ---- backward: pairs bucketed by endpoint
__global__ void pair_count_kernel(int64_t n, int64_t total, const int32_t* __restrict__ pu, const int32_t* __restrict__ pv,
                                  int32_t* __restrict__ cnt) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = pu[k], v = pv[k];
    if (u < 0 || v < 0 || u >= n || v >= n) continue;
    atomicAdd(&cnt[u], 1);
    atomicAdd(&cnt[v], 1);
  }
}

__global__ void pair_widen_kernel(int64_t n, const int32_t* __restrict__ in, int64_t* __restrict__ out) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r <= n; r += (int64_t)gridDim.x * blockDim.x)
    out[r] = r < n ? (int64_t)in[r] : 0;
}

__global__ void pair_scatter_kernel(int64_t n, int64_t total, const int32_t* __restrict__ pu,
                                    const int32_t* __restrict__ pv, const int64_t* __restrict__ off,
                                    int32_t* __restrict__ cur, int32_t* __restrict__ entries) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = pu[k], v = pv[k];
    if (u < 0 || v < 0 || u >= n || v >= n) continue;
    entries[off[u] + atomicAdd(&cur[u], 1)] = (int32_t)k;
    entries[off[v] + atomicAdd(&cur[v], 1)] = (int32_t)k;
  }
}

// dZ[r] = sum over the (sorted) entries k of row r of g_k Z[other endpoint].
template <typename T, int LPR>
__global__ __launch_bounds__(256) void pair_gather_kernel(int64_t n, int64_t F, int64_t ld, const T* __restrict__ Z,
                                                          const int32_t* __restrict__ pu, const int32_t* __restrict__ pv,
                                                          const float* __restrict__ g, const int64_t* __restrict__ off,
                                                          const int32_t* __restrict__ entries, Epilogue ep) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gi = lane / LPR, li = lane % LPR;
  const int64_t col0 = (int64_t)li * VE;
  if (col0 >= ep.ldo) return;
  const bool zero_slice = col0 >= F;   // padding columns [F, ldz): written 0
  constexpr int U = 4;
  for (int64_t r = ((int64_t)blockIdx.x * 4 + wave) * G + gi; r < n; r += (int64_t)gridDim.x * 4 * G) {
    float acc[VE];
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] = 0.f;
    const int64_t beg = off[r], end = zero_slice ? off[r] : off[r + 1];
    for (int64_t e = beg; e < end; e += U) {
      int32_t k[U];
#pragma unroll
      for (int u = 0; u < U; ++u) k[u] = entries[e + u < end ? e + u : end - 1];
      int32_t other[U];
      float w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int32_t a = pu[k[u]], b = pv[k[u]];
        other[u] = a == (int32_t)r ? b : a;
        w[u] = e + u < end ? g[k[u]] : 0.f;
      }
      uint4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = ldg16(Z + (int64_t)other[u] * ld + col0);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (e + u >= end) break;
        float xv[VE];
        unpack<T>(x[u], xv);
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[i] = fmaf(w[u], xv[i], acc[i]);
      }
    }
    epi_store_vec<T>(ep, r, col0, acc);
  }
}

template <typename T>
hipError_t pair_gather_t(int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pu, const int32_t* pv,
                         const float* g, const int64_t* off, const int32_t* entries, const Epilogue& ep, int lpr,
                         hipStream_t s) {
  const T* z = reinterpret_cast<const T*>(Z);
  const int64_t rows_per_block = 4 * (64 / lpr);
  const unsigned blocks = (unsigned)capped_blocks(n, rows_per_block);
  const int64_t colblocks = (F + (int64_t)lpr * Vec<T>::N - 1) / ((int64_t)lpr * Vec<T>::N);
  (void)colblocks;   // lpr covers F (lpr * VE >= F for F <= 64 * VE)
#define PG(L) hipLaunchKernelGGL((pair_gather_kernel<T, L>), dim3(blocks), dim3(256), 0, s, n, F, ld, z, pu, pv, g, off, entries, ep); break;
  switch (lpr) {
    case 1: PG(1)
    case 2: PG(2)
    case 4: PG(4)
    case 8: PG(8)
    case 16: PG(16)
    case 32: PG(32)
    default: PG(64)
  }
#undef PG
  return hipGetLastError();
}

// ---- metrics
constexpr int MT_TILE = 2048;

__global__ __launch_bounds__(256) void pair_metrics_kernel(const float* __restrict__ scores, int64_t P, int64_t N,
                                                           unsigned long long* __restrict__ auc_part,
                                                           double* __restrict__ ap_part) {
  __shared__ float tile[MT_TILE];
  __shared__ double sd[256];
  __shared__ unsigned long long su[256];
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const float si = i < P ? scores[i] : 0.f;
  unsigned long long pos_ge = 0, neg_ge = 0, auc2 = 0;   // auc2 = 2 * #{neg < s_i} + #{neg == s_i}
  const int64_t total = P + N;
  for (int64_t t0 = 0; t0 < total; t0 += MT_TILE) {
    const int64_t len = total - t0 < MT_TILE ? total - t0 : MT_TILE;
    __syncthreads();
    for (int j = threadIdx.x; j < len; j += 256) tile[j] = scores[t0 + j];
    __syncthreads();
    const int64_t npos = P - t0 <= 0 ? 0 : (P - t0 < len ? P - t0 : len);   // tile entries that are positives
    for (int j = 0; j < npos; ++j) pos_ge += tile[j] >= si ? 1ull : 0ull;
    for (int j = (int)npos; j < len; ++j) {
      const float sj = tile[j];
      neg_ge += sj >= si ? 1ull : 0ull;
      auc2 += sj < si ? 2ull : (sj == si ? 1ull : 0ull);
    }
  }
  double ap = 0.0;
  if (i < P) ap = (double)pos_ge / (double)(pos_ge + neg_ge);
  else auc2 = 0;
  sd[threadIdx.x] = ap;
  su[threadIdx.x] = auc2;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      sd[threadIdx.x] += sd[threadIdx.x + s];
      su[threadIdx.x] += su[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    ap_part[blockIdx.x] = sd[0];
    auc_part[blockIdx.x] = su[0];
  }
}

__global__ __launch_bounds__(256) void pair_metrics_final_kernel(const unsigned long long* __restrict__ auc_part,
                                                                 const double* __restrict__ ap_part, int64_t nb,
                                                                 int64_t P, int64_t N, double* out) {
  __shared__ double sd[256];
  __shared__ unsigned long long su[256];
  double a = 0.0;
  unsigned long long c = 0;
  for (int64_t b = threadIdx.x; b < nb; b += 256) { a += ap_part[b]; c += auc_part[b]; }
  sd[threadIdx.x] = a;
  su[threadIdx.x] = c;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      sd[threadIdx.x] += sd[threadIdx.x + s];
      su[threadIdx.x] += su[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[0] = (double)su[0] / (2.0 * (double)P * (double)N);
    out[1] = sd[0] / (double)P;
  }
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

hipError_t sample_pairs_launch(int64_t n, const int32_t* edge_u, const int32_t* edge_v, int64_t n_edges, int64_t n_pos,
                               int64_t n_neg, uint64_t seed, uint64_t epoch, int32_t* pair_u, int32_t* pair_v,
                               hipStream_t s) {
  const int64_t total = n_pos + n_neg;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(sample_pairs_kernel, dim3((unsigned)capped_blocks(total, 256)), dim3(256), 0, s, n, edge_u, edge_v,
                     n_edges, n_pos, total, seed, epoch, pair_u, pair_v);
  return hipGetLastError();
}

size_t pair_loss_workspace_bytes(int64_t n_pairs) {
  (void)n_pairs;
  return 65536 * sizeof(float) + 256;
}

hipError_t pair_loss_launch(int prec, int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pair_u,
                            const int32_t* pair_v, int64_t n_pos, int64_t n_neg, const float* loss_scale, float* loss,
                            float* scores, float* g, int32_t* flag, void* ws, hipStream_t s) {
  PairLossParams p;
  p.n = n; p.F = F; p.ld = ld; p.Z = Z; p.pu = pair_u; p.pv = pair_v;
  p.n_pos = n_pos; p.total = n_pos + n_neg; p.inv_total = 1.f / (float)p.total;
  p.loss_scale = loss_scale; p.scores = scores; p.g = g;
  p.part = reinterpret_cast<float*>(ws);
  p.flag = flag;
  const int lpr = lpr_for(prec, F);
  int64_t nb = 0;
  hipError_t e;
  switch (prec) {
    case 0: e = pair_loss_t<float>(p, lpr, s, &nb); break;
    case 1: e = pair_loss_t<f16>(p, lpr, s, &nb); break;
    case 2: e = pair_loss_t<bf16>(p, lpr, s, &nb); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pair_loss_final_kernel, dim3(1), dim3(256), 0, s, p.part, nb, p.inv_total, loss, flag);
  return hipGetLastError();
}

size_t pair_backward_workspace_bytes(int64_t n, int64_t n_pairs) {
  size_t b = 0;
  b += align256(sizeof(int32_t) * n);                                     // counts, then distinct counts
  b += align256(sizeof(int32_t) * n);                                     // cursors
  b += align256(sizeof(int64_t) * (n + 1));                               // row offsets
  b += align256(sizeof(int32_t) * 2 * n_pairs);                           // entries (pair ids)
  b += align256(sizeof(int64_t) * segment_scan_scratch_elems(n + 1));     // scan scratch
  return b;
}

hipError_t pair_backward_launch(int prec, int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pair_u,
                                const int32_t* pair_v, int64_t n_pairs, const float* g, void* dZ, int64_t ldz,
                                int32_t* flag, void* ws, hipStream_t s) {
  char* w = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* q = w; w += align256(bytes); return q; };
  int32_t* cnt = (int32_t*)take(sizeof(int32_t) * n);
  int32_t* cur = (int32_t*)take(sizeof(int32_t) * n);
  int64_t* off = (int64_t*)take(sizeof(int64_t) * (n + 1));
  int32_t* entries = (int32_t*)take(sizeof(int32_t) * 2 * n_pairs);
  int64_t* scr = (int64_t*)take(sizeof(int64_t) * segment_scan_scratch_elems(n + 1));
  hipError_t e;
#define GCN_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  GCN_TRY(fill_zero(cnt, sizeof(int32_t) * n, s));
  GCN_TRY(fill_zero(cur, sizeof(int32_t) * n, s));
  const unsigned gp = (unsigned)capped_blocks(n_pairs, 256);
  if (n_pairs > 0) {
    hipLaunchKernelGGL(pair_count_kernel, dim3(gp), dim3(256), 0, s, n, n_pairs, pair_u, pair_v, cnt);
    GCN_TRY(hipGetLastError());
  }
  hipLaunchKernelGGL(pair_widen_kernel, dim3((unsigned)capped_blocks(n + 1, 256)), dim3(256), 0, s, n, cnt, off);
  GCN_TRY(hipGetLastError());
  GCN_TRY(segment_scan_exclusive(off, n + 1, scr, s));
  if (n_pairs > 0) {
    hipLaunchKernelGGL(pair_scatter_kernel, dim3(gp), dim3(256), 0, s, n, n_pairs, pair_u, pair_v, off, cur, entries);
    GCN_TRY(hipGetLastError());
  }
  GCN_TRY(sort_segments(n, off, entries, cnt, s));
  Epilogue ep{};
  ep.out = dZ; ep.ldo = ldz; ep.rows = n; ep.cols = F; ep.mode = EPI_STORE; ep.flag = flag; ep.keep_scale = 1.f;
  const int lpr = lpr_for(prec, F);
  switch (prec) {
    case 0: GCN_TRY(pair_gather_t<float>(n, F, ld, Z, pair_u, pair_v, g, off, entries, ep, lpr, s)); break;
    case 1: GCN_TRY(pair_gather_t<f16>(n, F, ld, Z, pair_u, pair_v, g, off, entries, ep, lpr, s)); break;
    case 2: GCN_TRY(pair_gather_t<bf16>(n, F, ld, Z, pair_u, pair_v, g, off, entries, ep, lpr, s)); break;
    default: return hipErrorInvalidValue;
  }
#undef GCN_TRY
  return hipSuccess;
}

size_t pair_metrics_workspace_bytes(int64_t n_pos) {
  const int64_t nb = (n_pos + 255) / 256;
  return align256(sizeof(double) * nb) + align256(sizeof(unsigned long long) * nb);
}

hipError_t pair_metrics_launch(const float* scores, int64_t n_pos, int64_t n_neg, double* auc_ap, void* ws,
                               hipStream_t s) {
  const int64_t nb = (n_pos + 255) / 256;
  double* ap_part = reinterpret_cast<double*>(ws);
  unsigned long long* auc_part =
      reinterpret_cast<unsigned long long*>(static_cast<char*>(ws) + align256(sizeof(double) * nb));
  hipLaunchKernelGGL(pair_metrics_kernel, dim3((unsigned)nb), dim3(256), 0, s, scores, n_pos, n_neg, auc_part, ap_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pair_metrics_final_kernel, dim3(1), dim3(256), 0, s, auc_part, ap_part, nb, n_pos, n_neg, auc_ap);
  return hipGetLastError();
}

}  // namespace gcn

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
//  * pair backward: the pair endpoints are sorted by vertex with a stable
//    radix sort (so each row's entries stay in increasing k), then cut into
//    equal segments of entries; a lane group per segment sums the rows
//    inside it and a fix-up pass adds the partial sums of rows that cross
//    segment ends, in segment order: dZ is run-to-run identical without
//    floating-point atomics, and hub rows no longer serialise on one group.
//  * pair metrics: exact AUC and AP of held-out pairs.  The scores are
//    sorted once (the same stable radix sort, on order-preserving 32-bit
//    keys), the negatives before every position are counted by a scan, and
//    every positive finds the ends of its run of equal scores by binary
//    search: negatives below / equal and all scores >= it follow from the
//    counts at those ends, O((P + N) log(P + N)) in all.  Fixed-order sums.
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
  // at most 4096 workgroups (each loops over pairs), so that the final
  // fixed-order sum over their partials is short
  int64_t nb = capped_blocks(p.total, 4 * (64 / lpr));
  if (nb > 4096) nb = 4096;
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

// ---- backward: pair entries sorted by endpoint, then a balanced gather
//
// Entry i of the 2K entries is endpoint (i even ? u : v) of pair k = i / 2;
// its key is that endpoint (n for a pair with an id outside [0, n)).  A
// stable LSD radix sort by key (8-bit digits: per-tile digit histograms,
// one exclusive scan, a stable scatter that ranks equal digits by ballots)
// puts each row's entries together in increasing k without atomics.  The
// sorted entries are cut into segments of SEG entries; a lane group per
// segment sums the rows that lie inside it and leaves partial sums for the
// rows that cross its ends, which a fix-up pass adds in segment order.
constexpr int RS_MAX_BITS = 8;                      // digit width
constexpr int RS_IPT = 8;                           // items per thread per tile
constexpr int RS_TILE = 256 * RS_IPT;
constexpr int SEG = 64;                             // sorted entries per gather segment

__device__ __forceinline__ int32_t entry_key(int64_t n, const int32_t* __restrict__ pu, const int32_t* __restrict__ pv,
                                             int64_t i) {
  const int32_t u = pu[i >> 1], v = pv[i >> 1];
  const bool ok = u >= 0 && v >= 0 && u < n && v < n;
  return ok ? ((i & 1) ? v : u) : (int32_t)n;
}

// Digit histogram of one tile: hist[d * nblk + blockIdx.x] (digit-major).
template <int BITS>
__global__ __launch_bounds__(256) void rs_hist_kernel(int64_t n, const int32_t* __restrict__ pu,
                                                      const int32_t* __restrict__ pv, const int32_t* __restrict__ keys,
                                                      int64_t total, int shift, int64_t nblk,
                                                      int64_t* __restrict__ hist) {
  constexpr int DIGITS = 1 << BITS;
  __shared__ int cnt[DIGITS];
  for (int d = threadIdx.x; d < DIGITS; d += 256) cnt[d] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
  int32_t ks[RS_IPT];                               // all loads first (clamped indices)
#pragma unroll
  for (int r = 0; r < RS_IPT; ++r) {
    int64_t i = base + r * 256 + threadIdx.x;
    i = i < total ? i : total - 1;
    ks[r] = keys ? keys[i] : entry_key(n, pu, pv, i);
  }
#pragma unroll
  for (int r = 0; r < RS_IPT; ++r)
    if (base + r * 256 + threadIdx.x < total) atomicAdd(&cnt[(ks[r] >> shift) & (DIGITS - 1)], 1);
  __syncthreads();
  for (int d = threadIdx.x; d < DIGITS; d += 256) hist[(int64_t)d * nblk + blockIdx.x] = cnt[d];
}

// Stable scatter of one tile: items are ranked round by round (256
// consecutive items per round, thread order = item order); inside a wave
// the lanes with the same digit are found with 8 ballots, across the four
// waves through per-wave counts in LDS stamped with the round.  The ranked
// items are first placed in LDS in the tile's own digit order, then written
// out digit run by digit run, so that neighbouring lanes store to
// neighbouring addresses (placed straight at their global positions, every
// lane of a store would hit another cache line).
// Each item carries the gradient g_k of its pair (as bits) and the other
// endpoint: the segment sums then read g_k with the entry instead of
// gathering it by pair index.
template <int BITS>
__global__ __launch_bounds__(256) void rs_scatter_kernel(int64_t n, const int32_t* __restrict__ pu,
                                                         const int32_t* __restrict__ pv,
                                                         const int32_t* __restrict__ kin, const int32_t* __restrict__ vin,
                                                         const int32_t* __restrict__ oin, const float* __restrict__ g,
                                                         int64_t total, int shift, int64_t nblk,
                                                         const int64_t* __restrict__ off, int32_t* __restrict__ kout,
                                                         int32_t* __restrict__ vout, int32_t* __restrict__ oout) {
  constexpr int DIGITS = 1 << BITS;
  static_assert(DIGITS == 256, "one digit per thread");
  __shared__ int cnt[4][DIGITS];                    // (round << 16) | count
  __shared__ int run[DIGITS];
  __shared__ int toff[DIGITS];                      // first slot of each digit in the tile
  __shared__ int wsum[4];
  __shared__ int64_t dbase[DIGITS];
  __shared__ int32_t lk[RS_TILE], lv[RS_TILE], lo[RS_TILE];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
  // every item of the tile is requested before the first round: the rounds
  // are separated by barriers, and loads issued round by round would cost a
  // memory latency each (indices past the end read the last item, unused)
  int32_t ks[RS_IPT], vs[RS_IPT], os[RS_IPT];
#pragma unroll
  for (int r = 0; r < RS_IPT; ++r) {
    int64_t i = base + r * 256 + threadIdx.x;
    i = i < total ? i : total - 1;
    if (kin) {
      ks[r] = kin[i];
      vs[r] = vin[i];
      os[r] = oin[i];
    } else {                                        // first pass: items in pair order
      ks[r] = entry_key(n, pu, pv, i);
      vs[r] = __float_as_int(g[i >> 1]);
      os[r] = (i & 1) ? pu[i >> 1] : pv[i >> 1];
    }
  }
  {
    // thread d: the global start of digit d for this tile, and the tile's
    // count of digit d (difference of consecutive entries of the scanned
    // digit-major histogram); an exclusive scan of the counts gives toff
    const int d = threadIdx.x;
    const int64_t L = (int64_t)d * nblk + blockIdx.x;
    const int64_t b0 = off[L];
    const int64_t b1 = L + 1 < (int64_t)DIGITS * nblk ? off[L + 1] : total;
    const int c = (int)(b1 - b0);
    run[d] = 0;
    dbase[d] = b0;
#pragma unroll
    for (int w = 0; w < 4; ++w) cnt[w][d] = -1;     // stamp -1: no round yet
    int x = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    toff[d] = before + x - c;
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int r = 0; r < RS_IPT; ++r) {
    const int64_t i = base + r * 256 + threadIdx.x;
    const bool valid = i < total;
    const int32_t k = valid ? ks[r] : 0, val = vs[r], oth = os[r];
    const int d = (k >> shift) & (DIGITS - 1);
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < BITS; ++bit) {
      const uint64_t bb = __ballot((d >> bit) & 1);
      m &= ((d >> bit) & 1) ? bb : ~bb;
    }
    const int rank = __popcll(m & lt);
    if (valid && rank == 0) cnt[wave][d] = (r << 16) | __popcll(m);
    __syncthreads();
    if (valid) {
      int before = 0;
      for (int w = 0; w < wave; ++w) {
        const int c = cnt[w][d];
        if ((c >> 16) == r) before += c & 0xFFFF;
      }
      const int slot = toff[d] + run[d] + before + rank;
      lk[slot] = k;
      lv[slot] = val;
      lo[slot] = oth;
    }
    __syncthreads();
    {
      const int dd = threadIdx.x;
      int add = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int c = cnt[w][dd];
        if ((c >> 16) == r) add += c & 0xFFFF;
      }
      run[dd] += add;
    }
    __syncthreads();
  }
  // slot j of the tile holds the (j - toff[d])-th item of digit d
  const int64_t rest = total - base;
  const int tile_n = rest < RS_TILE ? (int)rest : RS_TILE;
  for (int j = threadIdx.x; j < tile_n; j += 256) {
    const int32_t k = lk[j];
    const int d = (k >> shift) & (DIGITS - 1);
    const int64_t pos = dbase[d] + (j - toff[d]);
    kout[pos] = k;
    vout[pos] = lv[j];
    oout[pos] = lo[j];
  }
}

// Row offsets from sorted keys: off[r] = first position with key >= r,
// r = 0 .. n (keys equal to n, the skipped pairs, lie past off[n]).
__global__ void rs_bounds_kernel(int64_t n, const int32_t* __restrict__ keys, int64_t total,
                                 int64_t* __restrict__ off) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j <= total; j += (int64_t)gridDim.x * blockDim.x) {
    const int64_t lo = j == 0 ? -1 : keys[j - 1];
    const int64_t hi = j == total ? n : min<int64_t>(keys[j], n);
    for (int64_t r = lo + 1; r <= hi; ++r) off[r] = j;
  }
}

__device__ __forceinline__ int64_t lower_row(const int64_t* __restrict__ off, int64_t n, int64_t x) {
  int64_t lo = 0, hi = n;                           // first r in [0, n] with off[r] >= x
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (off[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

struct SegParams {
  int64_t n, F, ld;
  const void* Z;
  const int32_t* pu;
  const int32_t* pv;
  const int64_t* off;                               // [n + 1]
  const int32_t* pg;                                // sorted entries: the pair's gradient g_k (bits)
  const int32_t* po;                                // sorted entries: other endpoint
  int64_t nseg;
  float* head;                                      // [nseg][ldp]
  float* tail;                                      // [nseg][ldp]
  int32_t* tail_row;                                // [nseg]
  int64_t ldp;
  Epilogue ep;
};

// Sum of g_k Z[other endpoint] over sorted entries [e0, e1) into acc.
template <typename T>
__device__ __forceinline__ void seg_sum(const SegParams& p, int64_t e0, int64_t e1, int64_t col0, float* acc) {
  constexpr int VE = Vec<T>::N, U = 8;
  const T* __restrict__ Z = reinterpret_cast<const T*>(p.Z);
  for (int64_t e = e0; e < e1; e += U) {
    int32_t other[U];
    float w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t ee = e + u < e1 ? e + u : e1 - 1;
      w[u] = __int_as_float(p.pg[ee]);
      other[u] = p.po[ee];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = e + u < e1 ? w[u] : 0.f;
    uint4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = ldg16(Z + (int64_t)other[u] * p.ld + col0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float xv[VE];
      unpack<T>(x[u], xv);
#pragma unroll
      for (int q = 0; q < VE; ++q) acc[q] = fmaf(w[u], xv[q], acc[q]);
    }
  }
}

template <typename T, int LPR>
__global__ __launch_bounds__(256) void pair_segment_kernel(SegParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gi = lane / LPR, li = lane % LPR;
  const int64_t col0 = (int64_t)li * VE;
  if (col0 >= p.ep.ldo) return;
  const bool live = col0 < p.F;                     // padding slices only write zeros
  const int64_t total = p.off[p.n];                 // entries of valid pairs
  const int64_t nuse = total > 0 ? (total + SEG - 1) / SEG : 1;
  for (int64_t sgi = ((int64_t)blockIdx.x * 4 + wave) * G + gi; sgi < p.nseg; sgi += (int64_t)gridDim.x * 4 * G) {
    if (sgi >= nuse) {                              // past the valid entries
      if (li == 0) p.tail_row[sgi] = -1;
      continue;
    }
    // rows starting in [a, b) belong to this segment; the last one also
    // takes the empty rows that start at the end
    const int64_t a = sgi * SEG, b = min(a + SEG, total);
    const int64_t r0 = lower_row(p.off, p.n, a);
    const int64_t r1 = sgi == nuse - 1 ? p.n : lower_row(p.off, p.n, b);
    float acc[VE];
    // head: the row that started before this segment
    if (r0 > 0 && p.off[r0] > a && a < b) {
#pragma unroll
      for (int q = 0; q < VE; ++q) acc[q] = 0.f;
      if (live) seg_sum<T>(p, a, min(p.off[r0], b), col0, acc);
      if (col0 < p.ldp) {
#pragma unroll
        for (int q = 0; q < VE; ++q) p.head[sgi * p.ldp + col0 + q] = acc[q];
      }
    }
    int32_t trow = -1;
    for (int64_t r = r0; r < r1; ++r) {
      const int64_t rs = p.off[r], re = p.off[r + 1];
#pragma unroll
      for (int q = 0; q < VE; ++q) acc[q] = 0.f;
      if (re <= b) {
        if (live) seg_sum<T>(p, rs, re, col0, acc);
        epi_store_vec<T>(p.ep, r, col0, acc);
      } else {                                      // crosses the end: partial, fixed up later
        if (live) seg_sum<T>(p, rs, b, col0, acc);
        if (col0 < p.ldp) {
#pragma unroll
          for (int q = 0; q < VE; ++q) p.tail[sgi * p.ldp + col0 + q] = acc[q];
        }
        trow = (int32_t)r;
      }
    }
    if (li == 0) p.tail_row[sgi] = trow;
  }
}

// Rows that cross segment ends: the tail partial of the segment where the
// row starts plus the head partials of the following segments, in order.
template <typename T, int LPR>
__global__ __launch_bounds__(256) void pair_fixup_kernel(SegParams p) {
  constexpr int VE = Vec<T>::N;
  constexpr int G = 64 / LPR;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gi = lane / LPR, li = lane % LPR;
  const int64_t col0 = (int64_t)li * VE;
  if (col0 >= p.ep.ldo) return;
  for (int64_t sgi = ((int64_t)blockIdx.x * 4 + wave) * G + gi; sgi < p.nseg; sgi += (int64_t)gridDim.x * 4 * G) {
    const int32_t r = p.tail_row[sgi];
    if (r < 0) continue;
    float acc[VE];
#pragma unroll
    for (int q = 0; q < VE; ++q) acc[q] = 0.f;
    if (col0 < p.F) {
      const int64_t last = (p.off[r + 1] - 1) / SEG;
#pragma unroll
      for (int q = 0; q < VE; ++q) acc[q] = p.tail[sgi * p.ldp + col0 + q];
      for (int64_t t = sgi + 1; t <= last; ++t) {
#pragma unroll
        for (int q = 0; q < VE; ++q) acc[q] += p.head[t * p.ldp + col0 + q];
      }
    }
    epi_store_vec<T>(p.ep, r, col0, acc);
  }
}

template <typename T>
hipError_t pair_segments_t(SegParams p, int lpr, hipStream_t s) {
  const int64_t per_block = 4 * (64 / lpr);
  const unsigned blocks = (unsigned)capped_blocks(p.nseg, per_block);
#define PG(L)                                                                                   \
  hipLaunchKernelGGL((pair_segment_kernel<T, L>), dim3(blocks), dim3(256), 0, s, p);            \
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;                            \
  hipLaunchKernelGGL((pair_fixup_kernel<T, L>), dim3(blocks), dim3(256), 0, s, p);              \
  break;
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

// Order-preserving key of a finite score: unsigned comparison of the keys
// agrees with < on the floats; -0 is taken as +0 (the two compare equal).
__device__ __forceinline__ uint32_t score_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Sort input: key, positive flag and index of each of the P + N scores.
__global__ __launch_bounds__(256) void metrics_prep_kernel(const float* __restrict__ scores, int64_t P, int64_t total,
                                                           int32_t* __restrict__ key, int32_t* __restrict__ pos,
                                                           int32_t* __restrict__ idx) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    key[i] = (int32_t)score_key(scores[i]);
    pos[i] = i < P ? 1 : 0;
    idx[i] = (int32_t)i;
  }
}

// cnt[j] = 1 for a negative at sorted position j, cnt[total] = 0; an
// exclusive scan then gives the negatives before every position.
__global__ __launch_bounds__(256) void metrics_negflag_kernel(const int32_t* __restrict__ pos, int64_t total,
                                                              int64_t* __restrict__ cnt) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j <= total; j += (int64_t)gridDim.x * blockDim.x)
    cnt[j] = j < total ? 1 - pos[j] : 0;
}

// For the positive at sorted position j with key k: lo = first position
// with key k, hi = first position past them (binary searches).  Negatives
// below: neg[lo]; equal: neg[hi] - neg[lo]; scores >= s: total - lo, of
// which positives: P - (lo - neg[lo]).  Sums per workgroup in position order.
__global__ __launch_bounds__(256) void metrics_count_kernel(const int32_t* __restrict__ key,
                                                            const int32_t* __restrict__ pos,
                                                            const int64_t* __restrict__ neg, int64_t P, int64_t total,
                                                            unsigned long long* __restrict__ auc_part,
                                                            double* __restrict__ ap_part) {
  __shared__ double sd[256];
  __shared__ unsigned long long su[256];
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double ap = 0.0;
  unsigned long long auc2 = 0;
  if (j < total && pos[j]) {
    const uint32_t k = (uint32_t)key[j];
    int64_t a = 0, b = j;                           // first position in [0, j] with key >= k
    while (a < b) {
      const int64_t m = a + (b - a) / 2;
      if ((uint32_t)key[m] < k) a = m + 1; else b = m;
    }
    const int64_t lo = a;
    a = j + 1; b = total;                           // first position in [j + 1, total) with key > k
    while (a < b) {
      const int64_t m = a + (b - a) / 2;
      if ((uint32_t)key[m] <= k) a = m + 1; else b = m;
    }
    const int64_t hi = a;
    const int64_t nlo = neg[lo], nhi = neg[hi];
    auc2 = 2ull * (unsigned long long)nlo + (unsigned long long)(nhi - nlo);
    ap = (double)(P - (lo - nlo)) / (double)(total - lo);
  }
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

// Passes for keys in [0, n] with 8-bit digits (wider digits measured no
// faster: the 9-bit scatter took as long as the pass it saved).
void rs_plan(int64_t n, int* passes, int* width) {
  int bits = 1;
  while (((int64_t)1 << bits) <= n) ++bits;
  *width = 8;
  *passes = (bits + 7) / 8;
}

int64_t pair_seg_count(int64_t n_pairs) {
  const int64_t t = (2 * n_pairs + SEG - 1) / SEG;
  return t < 1 ? 1 : t;
}

int64_t pair_partial_ld(int prec, int64_t F) {
  const int64_t ve = prec == 0 ? 4 : 8;
  return (F + ve - 1) / ve * ve;
}

size_t pair_backward_workspace_bytes(int64_t n, int64_t n_pairs, int64_t F) {
  const int64_t total = 2 * n_pairs;
  const int64_t nblk = (total + RS_TILE - 1) / RS_TILE;
  const int64_t nh = ((int64_t)1 << RS_MAX_BITS) * (nblk < 1 ? 1 : nblk);
  const int64_t nseg = pair_seg_count(n_pairs);
  const int64_t ldp = pair_partial_ld(1, F) > pair_partial_ld(0, F) ? pair_partial_ld(1, F) : pair_partial_ld(0, F);
  size_t b = 0;
  b += 6 * align256(sizeof(int32_t) * (total > 0 ? total : 1));          // key, pair, other: two buffers each
  b += align256(sizeof(int64_t) * nh);                                    // digit histograms / offsets
  b += align256(sizeof(int64_t) * segment_scan_scratch_elems(nh));        // scan scratch
  b += align256(sizeof(int64_t) * (n + 1));                               // row offsets
  b += 2 * align256(sizeof(float) * nseg * ldp);                          // head and tail partials
  b += align256(sizeof(int32_t) * nseg);                                  // tail rows
  return b;
}

hipError_t pair_backward_launch(int prec, int64_t n, int64_t F, int64_t ld, const void* Z, const int32_t* pair_u,
                                const int32_t* pair_v, int64_t n_pairs, const float* g, void* dZ, int64_t ldz,
                                int32_t* flag, void* ws, hipStream_t s) {
  const int64_t total = 2 * n_pairs;
  const int64_t nblk = (total + RS_TILE - 1) / RS_TILE;
  const int64_t nh = ((int64_t)1 << RS_MAX_BITS) * (nblk < 1 ? 1 : nblk);
  const int64_t nseg = pair_seg_count(n_pairs);
  const int64_t ldp = pair_partial_ld(prec, F);
  char* w = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* q = w; w += align256(bytes); return q; };
  const size_t tb = sizeof(int32_t) * (total > 0 ? total : 1);
  int32_t* kA = (int32_t*)take(tb);
  int32_t* vA = (int32_t*)take(tb);
  int32_t* oA = (int32_t*)take(tb);
  int32_t* kB = (int32_t*)take(tb);
  int32_t* vB = (int32_t*)take(tb);
  int32_t* oB = (int32_t*)take(tb);
  int64_t* hist = (int64_t*)take(sizeof(int64_t) * nh);
  int64_t* scr = (int64_t*)take(sizeof(int64_t) * segment_scan_scratch_elems(nh));
  int64_t* off = (int64_t*)take(sizeof(int64_t) * (n + 1));
  const size_t pbytes = sizeof(float) * nseg * (pair_partial_ld(1, F) > pair_partial_ld(0, F) ? pair_partial_ld(1, F)
                                                                                               : pair_partial_ld(0, F));
  float* head = (float*)take(pbytes);
  float* tail = (float*)take(pbytes);
  int32_t* trow = (int32_t*)take(sizeof(int32_t) * nseg);
  hipError_t e;
#define GCN_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  const int32_t* kin = nullptr;
  const int32_t* vin = nullptr;
  const int32_t* oin = nullptr;
  int32_t* kout = kA;
  int32_t* vout = vA;
  int32_t* oout = oA;
  if (total > 0) {
    int passes = 0, width = 8;
    rs_plan(n, &passes, &width);
    const int64_t nhw = ((int64_t)1 << width) * nblk;
    for (int ps = 0; ps < passes; ++ps) {
      const int shift = ps * width;
#define RS_PASS(B)                                                                                          \
  hipLaunchKernelGGL(rs_hist_kernel<B>, dim3((unsigned)nblk), dim3(256), 0, s, n, pair_u, pair_v, kin, total, \
                     shift, nblk, hist);                                                                    \
  GCN_TRY(hipGetLastError());                                                                               \
  GCN_TRY(segment_scan_exclusive(hist, nhw, scr, s));                                                       \
  hipLaunchKernelGGL(rs_scatter_kernel<B>, dim3((unsigned)nblk), dim3(256), 0, s, n, pair_u, pair_v, kin, vin, \
                     oin, g, total, shift, nblk, hist, kout, vout, oout);                                      \
  GCN_TRY(hipGetLastError());
      RS_PASS(8)
#undef RS_PASS
      kin = kout;
      vin = vout;
      oin = oout;
      kout = kout == kA ? kB : kA;
      vout = vout == vA ? vB : vA;
      oout = oout == oA ? oB : oA;
    }
  }
  const unsigned bb = (unsigned)capped_blocks(total + 1, 256);
  hipLaunchKernelGGL(rs_bounds_kernel, dim3(bb), dim3(256), 0, s, n, kin ? kin : kA, total, off);
  GCN_TRY(hipGetLastError());
  SegParams p;
  p.n = n; p.F = F; p.ld = ld; p.Z = Z; p.pu = pair_u; p.pv = pair_v; p.off = off;
  p.pg = vin ? vin : vA;
  p.po = oin ? oin : oA;
  p.nseg = nseg; p.head = head; p.tail = tail; p.tail_row = trow; p.ldp = ldp;
  Epilogue ep{};
  ep.out = dZ; ep.ldo = ldz; ep.rows = n; ep.cols = F; ep.mode = EPI_STORE; ep.flag = flag; ep.keep_scale = 1.f;
  p.ep = ep;
  const int lpr = lpr_for(prec, F);
  switch (prec) {
    case 0: GCN_TRY(pair_segments_t<float>(p, lpr, s)); break;
    case 1: GCN_TRY(pair_segments_t<f16>(p, lpr, s)); break;
    case 2: GCN_TRY(pair_segments_t<bf16>(p, lpr, s)); break;
    default: return hipErrorInvalidValue;
  }
#undef GCN_TRY
  return hipSuccess;
}

namespace {
struct MetricsLayout {
  int32_t *kA, *pA, *iA, *kB, *pB, *iB;
  int64_t *hist, *scr, *neg;
  double* ap_part;
  unsigned long long* auc_part;
  size_t bytes;
};
// Carves the workspace (ws may be NULL to size it).
MetricsLayout metrics_layout(int64_t total, void* ws) {
  const int64_t nblk = (total + RS_TILE - 1) / RS_TILE;
  const int64_t nh = ((int64_t)1 << RS_MAX_BITS) * (nblk < 1 ? 1 : nblk);
  const int64_t nb = (total + 255) / 256;
  const int64_t scan_n = nh > total + 1 ? nh : total + 1;
  MetricsLayout L;
  char* base = static_cast<char*>(ws);
  size_t o = 0;
  auto take = [&](size_t bytes) { char* q = base ? base + o : nullptr; o += align256(bytes); return q; };
  const size_t tb = sizeof(int32_t) * total;
  L.kA = (int32_t*)take(tb); L.pA = (int32_t*)take(tb); L.iA = (int32_t*)take(tb);
  L.kB = (int32_t*)take(tb); L.pB = (int32_t*)take(tb); L.iB = (int32_t*)take(tb);
  L.hist = (int64_t*)take(sizeof(int64_t) * nh);
  L.scr = (int64_t*)take(sizeof(int64_t) * segment_scan_scratch_elems(scan_n));
  L.neg = (int64_t*)take(sizeof(int64_t) * (total + 1));
  L.ap_part = (double*)take(sizeof(double) * nb);
  L.auc_part = (unsigned long long*)take(sizeof(unsigned long long) * nb);
  L.bytes = o;
  return L;
}
}  // namespace

size_t pair_metrics_workspace_bytes(int64_t n_pos, int64_t n_neg) {
  return metrics_layout(n_pos + n_neg, nullptr).bytes;
}

hipError_t pair_metrics_launch(const float* scores, int64_t n_pos, int64_t n_neg, double* auc_ap, void* ws,
                               hipStream_t s) {
  const int64_t total = n_pos + n_neg;
  const MetricsLayout L = metrics_layout(total, ws);
  const int64_t nblk = (total + RS_TILE - 1) / RS_TILE;
  const int64_t nb = (total + 255) / 256;
  const unsigned gb = (unsigned)capped_blocks(total + 1, 256);
  hipError_t e;
#define GCN_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  hipLaunchKernelGGL(metrics_prep_kernel, dim3(gb), dim3(256), 0, s, scores, n_pos, total, L.kA, L.pA, L.iA);
  GCN_TRY(hipGetLastError());
  // four stable 8-bit passes over the 32-bit keys: A -> B -> A -> B -> A
  int32_t *kin = L.kA, *pin = L.pA, *iin = L.iA, *kout = L.kB, *pout = L.pB, *iout = L.iB;
  for (int shift = 0; shift < 32; shift += RS_MAX_BITS) {
    hipLaunchKernelGGL(rs_hist_kernel<RS_MAX_BITS>, dim3((unsigned)nblk), dim3(256), 0, s, (int64_t)0, nullptr, nullptr,
                       kin, total, shift, nblk, L.hist);
    GCN_TRY(hipGetLastError());
    GCN_TRY(segment_scan_exclusive(L.hist, ((int64_t)1 << RS_MAX_BITS) * nblk, L.scr, s));
    hipLaunchKernelGGL(rs_scatter_kernel<RS_MAX_BITS>, dim3((unsigned)nblk), dim3(256), 0, s, (int64_t)0, nullptr,
                       nullptr, kin, pin, iin, nullptr, total, shift, nblk, L.hist, kout, pout, iout);
    GCN_TRY(hipGetLastError());
    int32_t* t;
    t = kin; kin = kout; kout = t;
    t = pin; pin = pout; pout = t;
    t = iin; iin = iout; iout = t;
  }
  hipLaunchKernelGGL(metrics_negflag_kernel, dim3(gb), dim3(256), 0, s, pin, total, L.neg);
  GCN_TRY(hipGetLastError());
  GCN_TRY(segment_scan_exclusive(L.neg, total + 1, L.scr, s));
  hipLaunchKernelGGL(metrics_count_kernel, dim3((unsigned)nb), dim3(256), 0, s, kin, pin, L.neg, n_pos, total,
                     L.auc_part, L.ap_part);
  GCN_TRY(hipGetLastError());
  hipLaunchKernelGGL(pair_metrics_final_kernel, dim3(1), dim3(256), 0, s, L.auc_part, L.ap_part, nb, n_pos, n_neg,
                     auc_ap);
#undef GCN_TRY
  return hipGetLastError();
}

}  // namespace gcn

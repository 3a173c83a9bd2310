// A_hat = D^-1/2 (A + I) D^-1/2 from an undirected edge list, as canonical
// CSR (rows ascending, columns ascending and unique), plus the heavy-row
// schedule used by the sparse aggregation.
//
// Steps (all integer work is order-independent, so the CSR is bit-identical
// from run to run even though the scatter uses atomics):
//   count    per-row counts of both directions of every u != v pair
//   scan     segment offsets (count + 1 slot for the self-loop)
//   scatter  neighbour ids into per-row segments (+ the self-loop)
//   sort     each segment: wave bitonic (<= 64), LDS bitonic (<= 4096),
//            global-memory bitonic (larger hubs)
//   unique   per-row count of distinct neighbours -> degree
//   scan     row pointers; compact; dinv = fp32(1 / sqrt(fp64(deg)))
//   values   dinv[row] * dinv[col] in the value precision; optional dense
#include "internal.h"

#include <algorithm>
#include <vector>

namespace gcn {

namespace {

constexpr int SCAN_BLOCK = 1024;   // elements per scan block (256 threads x 4)
constexpr int64_t SORT_LDS_MAX = 4096;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int64_t scan_scratch_elems(int64_t count) {
  int64_t total = 0;
  while (count > SCAN_BLOCK) {
    count = (count + SCAN_BLOCK - 1) / SCAN_BLOCK;
    total += count;
  }
  return total + 1;
}

// ------------------------------------------------------------------ scan ----
__global__ __launch_bounds__(256) void scan_block_kernel(int64_t* __restrict__ data, int64_t count,
                                                         int64_t* __restrict__ block_sums) {
  __shared__ int64_t s[256];
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + threadIdx.x * 4;
  int64_t v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = base + i < count ? data[base + i] : 0;
  const int64_t tsum = v[0] + v[1] + v[2] + v[3];
  s[threadIdx.x] = tsum;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int64_t add = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
    __syncthreads();
    s[threadIdx.x] += add;
    __syncthreads();
  }
  int64_t run = s[threadIdx.x] - tsum;   // exclusive prefix of this thread
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (base + i < count) data[base + i] = run;
    run += v[i];
  }
  if (threadIdx.x == 255 && block_sums) block_sums[blockIdx.x] = s[255];
}

__global__ __launch_bounds__(256) void scan_add_kernel(int64_t* __restrict__ data, int64_t count,
                                                       const int64_t* __restrict__ block_off) {
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + threadIdx.x * 4;
  const int64_t add = block_off[blockIdx.x];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (base + i < count) data[base + i] += add;
}

// In-place exclusive scan of data[0..count); scratch holds scan_scratch_elems(count).
hipError_t scan_exclusive(int64_t* data, int64_t count, int64_t* scratch, hipStream_t s) {
  const int64_t nb = (count + SCAN_BLOCK - 1) / SCAN_BLOCK;
  hipLaunchKernelGGL(scan_block_kernel, dim3((unsigned)nb), dim3(256), 0, s, data, count, nb > 1 ? scratch : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nb <= 1) return e;
  e = scan_exclusive(scratch, nb, scratch + nb, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scan_add_kernel, dim3((unsigned)nb), dim3(256), 0, s, data, count, scratch);
  return hipGetLastError();
}

// ---------------------------------------------------------------- helpers ----
__global__ void fill_zero_kernel(uint32_t* p, int64_t words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// Workgroups for one wave per row, 4 rows per workgroup of 256 threads; the
// kernels loop over rows, so the grid is capped (a dispatch may not exceed
// 2^32 work-items per dimension).
unsigned wave_rows_grid(int64_t rows) {
  int64_t g = (rows + 3) / 4;
  if (g < 1) g = 1;
  if (g > (1 << 20)) g = 1 << 20;
  return (unsigned)g;
}

unsigned grid_for(int64_t items, int per_block = 256, int64_t cap = 65536) {
  int64_t g = (items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

// ---------------------------------------------------------------- kernels ----
__global__ void count_kernel(int64_t n, int64_t E, const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                             int32_t* __restrict__ cnt, int32_t* __restrict__ bad) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < E; k += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = src[k], v = dst[k];
    if (u < 0 || v < 0 || u >= n || v >= n) { *reinterpret_cast<volatile int32_t*>(bad) = 1; continue; }
    if (u == v) continue;
    atomicAdd(&cnt[u], 1);
    atomicAdd(&cnt[v], 1);
  }
}

// seg[r] = cnt[r] + 1 (self-loop slot), seg[n] = 0
__global__ void seglen_kernel(int64_t n, const int32_t* __restrict__ cnt, int64_t* __restrict__ seg) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r <= n; r += (int64_t)gridDim.x * blockDim.x)
    seg[r] = r < n ? (int64_t)cnt[r] + 1 : 0;
}

// out[r] = in[r], out[n] = 0
__global__ void widen_kernel(int64_t n, const int32_t* __restrict__ in, int64_t* __restrict__ out) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r <= n; r += (int64_t)gridDim.x * blockDim.x)
    out[r] = r < n ? (int64_t)in[r] : 0;
}

__global__ void scatter_kernel(int64_t n, int64_t E, const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                               const int64_t* __restrict__ off, int32_t* __restrict__ cur, int32_t* __restrict__ tmp) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < E; k += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = src[k], v = dst[k];
    if (u < 0 || v < 0 || u >= n || v >= n || u == v) continue;
    const int32_t pu = atomicAdd(&cur[u], 1);
    tmp[off[u] + pu] = v;
    const int32_t pv = atomicAdd(&cur[v], 1);
    tmp[off[v] + pv] = u;
  }
}

__global__ void selfloop_kernel(int64_t n, const int64_t* __restrict__ off, const int32_t* __restrict__ cnt,
                                int32_t* __restrict__ tmp) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x)
    tmp[off[r] + cnt[r]] = (int32_t)r;
}

// Segments of at most 64 entries: one wave, register bitonic sort.
__global__ __launch_bounds__(256) void sort_small_kernel(int64_t n, const int64_t* __restrict__ off,
                                                         int32_t* __restrict__ tmp, int32_t* __restrict__ ucnt) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += (int64_t)gridDim.x * 4) {
    const int64_t b = off[r], len = off[r + 1] - b;
    if (len > 64) continue;
    int x = lane < len ? tmp[b + lane] : INT32_MAX;
    for (int k = 2; k <= 64; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        const int y = __shfl_xor(x, j);
        const bool asc = (lane & k) == 0;
        const bool lower = (lane & j) == 0;
        x = (lower == asc) ? min(x, y) : max(x, y);
      }
    }
    const int prev = __shfl(x, lane == 0 ? 0 : lane - 1);
    const bool flag = lane < len && (lane == 0 || x != prev);
    const uint64_t bal = __ballot(flag);
    if (lane < len) tmp[b + lane] = x;
    if (lane == 0) ucnt[r] = __popcll(bal);
  }
}

__device__ int block_sum_int(int v, int* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const int out = red[0];
  __syncthreads();
  return out;
}

// Segments of 65..4096 entries: one workgroup, bitonic sort in LDS.
__global__ __launch_bounds__(256) void sort_medium_kernel(int64_t n, const int64_t* __restrict__ off,
                                                          int32_t* __restrict__ tmp, int32_t* __restrict__ ucnt) {
  __shared__ int s[SORT_LDS_MAX];
  __shared__ int red[256];
  for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
    const int64_t b = off[r], len = off[r + 1] - b;
    if (len <= 64 || len > SORT_LDS_MAX) continue;
    int P = 128;
    while (P < len) P <<= 1;
    for (int i = threadIdx.x; i < P; i += 256) s[i] = i < len ? tmp[b + i] : INT32_MAX;
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = threadIdx.x; i < P; i += 256) {
          const int ixj = i ^ j;
          if (ixj > i) {
            const int a = s[i], c = s[ixj];
            const bool asc = (i & k) == 0;
            if ((a > c) == asc) { s[i] = c; s[ixj] = a; }
          }
        }
        __syncthreads();
      }
    }
    int cntu = 0;
    for (int i = threadIdx.x; i < len; i += 256) {
      tmp[b + i] = s[i];
      cntu += (i == 0 || s[i] != s[i - 1]) ? 1 : 0;
    }
    const int tot = block_sum_int(cntu, red);
    if (threadIdx.x == 0) ucnt[r] = tot;
    __syncthreads();
  }
}

// Segments above 4096 entries: one workgroup, bitonic network in global
// memory in its "always ascending" form (the first step of each merge
// compares i with its mirror in the block), so positions >= len act as +inf
// and are never touched.
__global__ __launch_bounds__(256) void sort_large_kernel(int64_t n, const int64_t* __restrict__ off,
                                                         int32_t* __restrict__ tmp, int32_t* __restrict__ ucnt) {
  __shared__ int red[256];
  for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
    const int64_t b = off[r], len = off[r + 1] - b;
    if (len <= SORT_LDS_MAX) continue;
    int32_t* a = tmp + b;
    int64_t P = 1;
    while (P < len) P <<= 1;
    for (int64_t k = 2; k <= P; k <<= 1) {
      // mirror step
      for (int64_t t = threadIdx.x; t < P / 2; t += 256) {
        const int64_t blk = t / (k / 2), w = t % (k / 2);
        const int64_t i = blk * k + w, p = blk * k + (k - 1 - w);
        if (p < len) {
          const int32_t x = a[i], y = a[p];
          if (x > y) { a[i] = y; a[p] = x; }
        }
      }
      __syncthreads();
      for (int64_t j = k / 4; j > 0; j >>= 1) {
        for (int64_t t = threadIdx.x; t < P / 2; t += 256) {
          const int64_t blk = t / j, w = t % j;
          const int64_t i = blk * 2 * j + w, p = i + j;
          if (p < len) {
            const int32_t x = a[i], y = a[p];
            if (x > y) { a[i] = y; a[p] = x; }
          }
        }
        __syncthreads();
      }
    }
    int cntu = 0;
    for (int64_t i = threadIdx.x; i < len; i += 256) cntu += (i == 0 || a[i] != a[i - 1]) ? 1 : 0;
    const int tot = block_sum_int(cntu, red);
    if (threadIdx.x == 0) ucnt[r] = tot;
    __syncthreads();
  }
}

// Compact sorted segments to unique columns; write rowptr, deg, dinv.
template <typename IdxT>
__global__ __launch_bounds__(256) void compact_kernel(int64_t n, const int64_t* __restrict__ off,
                                                      const int32_t* __restrict__ tmp, const int64_t* __restrict__ rp64,
                                                      const int32_t* __restrict__ ucnt, IdxT* __restrict__ rowptr,
                                                      int32_t* __restrict__ colidx, int32_t* __restrict__ deg,
                                                      float* __restrict__ dinv) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r <= n; r += (int64_t)gridDim.x * 4) {
    if (r == n) {
      if (lane == 0) rowptr[n] = (IdxT)rp64[n];
      continue;
    }
    const int64_t b = off[r], len = off[r + 1] - b;
    const int64_t o = rp64[r];
    int64_t run = 0;
    for (int64_t base = 0; base < len; base += 64) {
      const int64_t i = base + lane;
      const int x = i < len ? tmp[b + i] : 0;
      const bool flag = i < len && (i == 0 || x != tmp[b + i - 1]);
      const uint64_t bal = __ballot(flag);
      const int pre = __popcll(bal & __lanemask_lt());
      if (flag) colidx[o + run + pre] = x;
      run += __popcll(bal);
    }
    if (lane == 0) {
      rowptr[r] = (IdxT)o;
      const int32_t d = ucnt[r];
      if (deg) deg[r] = d;
      dinv[r] = (float)(1.0 / sqrt((double)d));
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void values_kernel(int64_t n, const int64_t* __restrict__ rp64,
                                                     const int32_t* __restrict__ colidx, const float* __restrict__ dinv,
                                                     T* __restrict__ values, T* __restrict__ dense, int64_t ld_dense) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += (int64_t)gridDim.x * 4) {
    const float dr = dinv[r];
    for (int64_t k = rp64[r] + lane; k < rp64[r + 1]; k += 64) {
      const int32_t c = colidx[k];
      const T v = from_f32<T>(dr * dinv[c]);
      if (values) values[k] = v;
      if (dense) dense[r * ld_dense + c] = v;
    }
  }
}

// ---------------------------------------------------------------- schedule ----
// Heavy rows are cut into pieces: at the boundaries of the P column ranges
// (column c lies in range floor(c P / n)) and then every `seg` entries.
// Range q ends at the first entry of the (sorted) row whose column c has
// c P >= (q + 1) n, i.e. c >= ceil((q + 1) n / P).
// First column of range q: ceil(q n / P).
__device__ __forceinline__ int64_t range_first(int64_t q, int64_t n, int64_t parts) {
  return (q * n + parts - 1) / parts;
}

__device__ __forceinline__ int64_t range_end(const int32_t* __restrict__ colidx, int64_t lo, int64_t hi, int64_t bound) {
  while (lo < hi) {                       // first k in [lo, hi) with colidx[k] >= bound
    const int64_t mid = lo + ((hi - lo) >> 1);
    if ((int64_t)colidx[mid] < bound) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

template <typename IdxT>
__global__ void piece_count_kernel(int64_t n, const IdxT* __restrict__ rowptr, const int32_t* __restrict__ colidx,
                                   int64_t thr, int64_t seg, int64_t parts, int64_t* __restrict__ flag,
                                   int64_t* __restrict__ npieces) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r <= n; r += (int64_t)gridDim.x * blockDim.x) {
    if (r == n) { flag[n] = 0; npieces[n] = 0; continue; }
    const int64_t beg = (int64_t)rowptr[r], end = (int64_t)rowptr[r + 1];
    if (end - beg <= thr) { flag[r] = 0; npieces[r] = 0; continue; }
    int64_t cnt = 0, a = beg;
    for (int64_t q = 0; q < parts; ++q) {
      const int64_t b = q + 1 == parts ? end : range_end(colidx, a, end, range_first(q + 1, n, parts));
      cnt += (b - a + seg - 1) / seg;
      a = b;
    }
    flag[r] = 1;
    npieces[r] = cnt;
  }
}

template <typename IdxT>
__global__ void piece_fill_kernel(int64_t n, int64_t nnz, const IdxT* __restrict__ rowptr,
                                  const int32_t* __restrict__ colidx, int64_t thr, int64_t seg, int64_t parts,
                                  const int64_t* __restrict__ hidx, const int64_t* __restrict__ poff,
                                  int32_t* __restrict__ heavy_rows, int32_t* __restrict__ heavy_chunk_off,
                                  int32_t* __restrict__ chunk_heavy, int64_t* __restrict__ chunk_beg) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r <= n; r += (int64_t)gridDim.x * blockDim.x) {
    if (r == n) {
      heavy_chunk_off[hidx[n]] = (int32_t)poff[n];
      chunk_beg[poff[n]] = nnz;
      continue;
    }
    const int64_t beg = (int64_t)rowptr[r], end = (int64_t)rowptr[r + 1];
    if (end - beg <= thr) continue;
    const int64_t h = hidx[r];
    heavy_rows[h] = (int32_t)r;
    heavy_chunk_off[h] = (int32_t)poff[r];
    int64_t c = poff[r], a = beg;
    for (int64_t q = 0; q < parts; ++q) {
      const int64_t b = q + 1 == parts ? end : range_end(colidx, a, end, range_first(q + 1, n, parts));
      for (int64_t k = a; k < b; k += seg) {
        chunk_heavy[c] = (int32_t)h;
        chunk_beg[c] = k;
        ++c;
      }
      a = b;
    }
  }
}

// Light rows, block by block of `blk` consecutive row ids, by decreasing
// degree inside a block: a counting sort over the buckets
// (r / blk) (thr + 1) + thr - deg (deg <= thr), except the rows of exactly
// one entry, which all go to one last bucket so that the product can take
// them in bundles (on R-MAT scale 21 they are 42 % of the light rows).  Rows of similar length
// share a wave, and on large graphs rows whose ids are close -- whose
// neighbours overlap more in an R-MAT graph -- run together (R-MAT scale 21:
// 5 % faster than one global degree order).  Below 2^20 rows one block (a
// global decreasing-degree order) is kept: there the longest rows must
// start first or they form the tail (R-MAT scale 17, F = 256: 23 % slower
// with blocks of 4096).  A workgroup owns a contiguous range of rows and
// first counts them per bucket in LDS, so the global atomics are one per
// bucket and workgroup; buckets beyond LIGHT_LDS_BINS of the workgroup's
// first bucket use global atomics.
constexpr int LIGHT_LDS_BINS = 1024;

int64_t light_block(int64_t n) { return n >= ((int64_t)1 << 20) ? 4096 : (n > 0 ? n : 1); }
int64_t light_buckets(int64_t n, int64_t thr) {
  const int64_t blk = light_block(n);
  return (n + blk - 1) / blk * (thr + 1) + 1;
}

// Bucket of a light row r of degree d (nb buckets, the last for one-entry
// rows) and its LDS slot in a workgroup whose first block bucket is base
// (LIGHT_LDS_BINS for the last bucket; -1: no slot, global atomics).
__device__ __forceinline__ int64_t light_bucket(int64_t r, int64_t d, int64_t thr, int64_t blk, int64_t nb) {
  return d == 1 ? nb - 1 : (r / blk) * (thr + 1) + thr - d;
}
__device__ __forceinline__ int light_slot(int64_t b, int64_t base, int64_t nb) {
  if (b == nb - 1) return LIGHT_LDS_BINS;
  return b - base < LIGHT_LDS_BINS ? (int)(b - base) : -1;
}
// Bucket of LDS slot k (or -1 when the slot maps to no bucket of the block range).
__device__ __forceinline__ int64_t slot_bucket(int k, int64_t base, int64_t nb) {
  if (k == LIGHT_LDS_BINS) return nb - 1;
  return base + k < nb - 1 ? base + k : -1;
}

__device__ __forceinline__ void row_range(int64_t n, int64_t* r0, int64_t* r1) {
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  *r0 = (int64_t)blockIdx.x * per;
  *r1 = *r0 + per < n ? *r0 + per : n;
}

template <typename IdxT>
__global__ __launch_bounds__(256) void light_hist_kernel(int64_t n, const IdxT* __restrict__ rowptr, int64_t thr,
                                                         int64_t blk, int64_t nb, int32_t* __restrict__ hist) {
  __shared__ int32_t lh[LIGHT_LDS_BINS + 1];
  for (int b = threadIdx.x; b <= LIGHT_LDS_BINS; b += 256) lh[b] = 0;
  __syncthreads();
  int64_t r0, r1;
  row_range(n, &r0, &r1);
  const int64_t base = (r0 / blk) * (thr + 1);
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) {
    const int64_t d = (int64_t)rowptr[r + 1] - (int64_t)rowptr[r];
    if (d > thr) continue;
    const int64_t b = light_bucket(r, d, thr, blk, nb);
    const int k = light_slot(b, base, nb);
    if (k >= 0) atomicAdd(&lh[k], 1);
    else atomicAdd(&hist[b], 1);
  }
  __syncthreads();
  for (int k = threadIdx.x; k <= LIGHT_LDS_BINS; k += 256) {
    const int64_t b = slot_bucket(k, base, nb);
    if (b >= 0 && lh[k]) atomicAdd(&hist[b], lh[k]);
  }
}

template <typename IdxT>
__global__ __launch_bounds__(256) void light_scatter_kernel(int64_t n, const IdxT* __restrict__ rowptr, int64_t thr,
                                                            int64_t blk, int64_t nb, const int64_t* __restrict__ boff,
                                                            int32_t* __restrict__ cur, int32_t* __restrict__ perm) {
  __shared__ int32_t lh[LIGHT_LDS_BINS + 1];     // count, then this workgroup's base within the bucket
  __shared__ int32_t lc[LIGHT_LDS_BINS + 1];     // local cursor
  for (int b = threadIdx.x; b <= LIGHT_LDS_BINS; b += 256) { lh[b] = 0; lc[b] = 0; }
  __syncthreads();
  int64_t r0, r1;
  row_range(n, &r0, &r1);
  const int64_t base = (r0 / blk) * (thr + 1);
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) {
    const int64_t d = (int64_t)rowptr[r + 1] - (int64_t)rowptr[r];
    if (d > thr) continue;
    const int k = light_slot(light_bucket(r, d, thr, blk, nb), base, nb);
    if (k >= 0) atomicAdd(&lh[k], 1);
  }
  __syncthreads();
  for (int k = threadIdx.x; k <= LIGHT_LDS_BINS; k += 256) {
    const int64_t b = slot_bucket(k, base, nb);
    if (b >= 0 && lh[k]) lh[k] = atomicAdd(&cur[b], lh[k]);
  }
  __syncthreads();
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) {
    const int64_t d = (int64_t)rowptr[r + 1] - (int64_t)rowptr[r];
    if (d > thr) continue;
    const int64_t b = light_bucket(r, d, thr, blk, nb);
    const int k = light_slot(b, base, nb);
    const int64_t pos = k >= 0 ? (int64_t)lh[k] + atomicAdd(&lc[k], 1) : (int64_t)atomicAdd(&cur[b], 1);
    perm[boff[b] + pos] = (int32_t)r;
  }
}

// Piece launch order: counting sort of the pieces by the column bucket of
// their first entry (CHUNK_BUCKETS buckets over [0, n)).  The bucket of a
// column, c * 4096 / n, nests in its column range c * P / n for every P
// that divides 4096, so the sorted pieces of range p are one run, starting
// at the offset of bucket p * 4096 / P.
constexpr int64_t CHUNK_BUCKETS = 4096;

__global__ void part_off_kernel(int64_t parts, const int64_t* __restrict__ boff, int64_t* __restrict__ part_off) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q <= parts) part_off[q] = boff[q * (CHUNK_BUCKETS / parts)];
}

// 16-byte descriptors in launch order, so that a lane group learns where a
// row or piece lies with one load: light rows {first entry, row, length};
// pieces {first entry, row, length | 2^31 if the row has no other piece},
// plus the launch position of every piece (its partial row's slot).
template <typename IdxT>
__global__ void light_desc_kernel(int64_t n_light, const IdxT* __restrict__ rowptr, const int32_t* __restrict__ perm,
                                  RowDesc* __restrict__ desc) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_light; i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t r = perm[i];
    const int64_t b = (int64_t)rowptr[r];
    desc[i] = RowDesc{b, r, (int32_t)((int64_t)rowptr[r + 1] - b)};
  }
}

template <typename IdxT>
__global__ void piece_desc_kernel(int64_t n_chunks, const IdxT* __restrict__ rowptr, const int32_t* __restrict__ order,
                                  const int32_t* __restrict__ chunk_heavy, const int32_t* __restrict__ heavy_rows,
                                  const int32_t* __restrict__ heavy_chunk_off, const int64_t* __restrict__ chunk_beg,
                                  RowDesc* __restrict__ desc, int32_t* __restrict__ pos_of) {
  for (int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; pos < n_chunks; pos += (int64_t)gridDim.x * blockDim.x) {
    const int32_t c = order[pos];
    const int32_t h = chunk_heavy[c];
    const int32_t r = heavy_rows[h];
    const int64_t b = chunk_beg[c];
    const int64_t rend = (int64_t)rowptr[r + 1];
    const int64_t e = chunk_beg[c + 1] < rend ? chunk_beg[c + 1] : rend;
    const bool single = heavy_chunk_off[h + 1] - heavy_chunk_off[h] == 1;
    desc[pos] = RowDesc{b, r, (int32_t)((uint32_t)(e - b) | (single ? 0x80000000u : 0u))};
    pos_of[c] = (int32_t)pos;
  }
}

// Heavy rows whose partials the fix-up adds (more than one piece), flagged
// for two stable compactions: big[h] for more than GCN_FIX_BIG_PIECES
// pieces, small[h] for 2 .. GCN_FIX_BIG_PIECES; entry n_heavy is 0.
__global__ void fix_flag_kernel(int64_t n_heavy, const int32_t* __restrict__ heavy_chunk_off, int64_t* __restrict__ big,
                                int64_t* __restrict__ small) {
  for (int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; h <= n_heavy; h += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = h < n_heavy ? heavy_chunk_off[h + 1] - heavy_chunk_off[h] : 0;
    big[h] = m > GCN_FIX_BIG_PIECES ? 1 : 0;
    small[h] = m >= 2 && m <= GCN_FIX_BIG_PIECES ? 1 : 0;
  }
}

// fix_rows = [big rows ascending, small rows ascending] from the exclusive
// scans of the flags.
__global__ void fix_scatter_kernel(int64_t n_heavy, const int32_t* __restrict__ heavy_chunk_off,
                                   const int64_t* __restrict__ big_off, const int64_t* __restrict__ small_off,
                                   int32_t* __restrict__ fix_rows) {
  const int64_t n_big = big_off[n_heavy];
  for (int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; h < n_heavy; h += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = heavy_chunk_off[h + 1] - heavy_chunk_off[h];
    if (m > GCN_FIX_BIG_PIECES) fix_rows[big_off[h]] = (int32_t)h;
    else if (m >= 2) fix_rows[n_big + small_off[h]] = (int32_t)h;
  }
}

__global__ void chunk_key_kernel(int64_t n, int64_t n_chunks, const int32_t* __restrict__ colidx,
                                 const int64_t* __restrict__ chunk_beg, int32_t* __restrict__ key,
                                 int32_t* __restrict__ hist) {
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < n_chunks; c += (int64_t)gridDim.x * blockDim.x) {
    const int32_t b = (int32_t)((int64_t)colidx[chunk_beg[c]] * CHUNK_BUCKETS / n);
    key[c] = b;
    atomicAdd(&hist[b], 1);
  }
}

__global__ void chunk_scatter_kernel(int64_t n_chunks, const int32_t* __restrict__ key, const int64_t* __restrict__ boff,
                                     int32_t* __restrict__ cur, int32_t* __restrict__ order) {
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < n_chunks; c += (int64_t)gridDim.x * blockDim.x) {
    const int32_t b = key[c];
    order[boff[b] + atomicAdd(&cur[b], 1)] = (int32_t)c;
  }
}

}  // namespace

int64_t segment_scan_scratch_elems(int64_t count) { return scan_scratch_elems(count); }

hipError_t segment_scan_exclusive(int64_t* data, int64_t count, int64_t* scratch, hipStream_t s) {
  return scan_exclusive(data, count, scratch, s);
}

hipError_t fill_zero(void* p, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  // callers pass 4-byte multiples
  const int64_t words = (int64_t)(bytes / 4);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(words, 256, 16384)), dim3(256), 0, s, (uint32_t*)p, words);
  return hipGetLastError();
}

size_t normalize_workspace_bytes(int64_t n, int64_t E) {
  size_t b = 0;
  b += align256(sizeof(int32_t) * n);                         // cnt / ucnt
  b += align256(sizeof(int32_t) * n);                         // cur
  b += align256(sizeof(int64_t) * (n + 1));                   // off
  b += align256(sizeof(int64_t) * (n + 1));                   // rp64
  b += align256(sizeof(int32_t) * (2 * E + n));               // tmp
  b += align256(sizeof(int64_t) * scan_scratch_elems(n + 1)); // scan scratch
  b += align256(sizeof(int64_t) * 4);                         // misc
  return b;
}

hipError_t normalize_run(int64_t n, int64_t E, const int32_t* src, const int32_t* dst, bool idx64,
                         void* rowptr, int32_t* colidx, int32_t* deg, float* dinv, int value_prec,
                         void* values, void* dense, int64_t ld_dense, int64_t* nnz_out, int32_t* bad_ids,
                         void* ws, size_t ws_bytes, hipStream_t s) {
  char* w = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* p = w; w += align256(bytes); return p; };
  int32_t* cnt = (int32_t*)take(sizeof(int32_t) * n);
  int32_t* cur = (int32_t*)take(sizeof(int32_t) * n);
  int64_t* off = (int64_t*)take(sizeof(int64_t) * (n + 1));
  int64_t* rp64 = (int64_t*)take(sizeof(int64_t) * (n + 1));
  int32_t* tmp = (int32_t*)take(sizeof(int32_t) * (2 * E + n));
  int64_t* scr = (int64_t*)take(sizeof(int64_t) * scan_scratch_elems(n + 1));
  int64_t* misc = (int64_t*)take(sizeof(int64_t) * 4);
  if ((size_t)(w - static_cast<char*>(ws)) > ws_bytes) return hipErrorInvalidValue;

  hipError_t e;
#define GCN_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  GCN_TRY(fill_zero(cnt, sizeof(int32_t) * n, s));
  GCN_TRY(fill_zero(cur, sizeof(int32_t) * n, s));
  GCN_TRY(fill_zero(misc, sizeof(int64_t) * 4, s));
  int32_t* bad = reinterpret_cast<int32_t*>(misc + 1);
  if (E > 0) {
    hipLaunchKernelGGL(count_kernel, dim3(grid_for(E)), dim3(256), 0, s, n, E, src, dst, cnt, bad);
    GCN_TRY(hipGetLastError());
  }
  hipLaunchKernelGGL(seglen_kernel, dim3(grid_for(n + 1)), dim3(256), 0, s, n, cnt, off);
  GCN_TRY(hipGetLastError());
  GCN_TRY(scan_exclusive(off, n + 1, scr, s));
  if (E > 0) {
    hipLaunchKernelGGL(scatter_kernel, dim3(grid_for(E)), dim3(256), 0, s, n, E, src, dst, off, cur, tmp);
    GCN_TRY(hipGetLastError());
  }
  hipLaunchKernelGGL(selfloop_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, off, cnt, tmp);
  GCN_TRY(hipGetLastError());
  int32_t* ucnt = cnt;   // counts are no longer needed after the self-loop slots are placed
  hipLaunchKernelGGL(sort_small_kernel, dim3(wave_rows_grid(n)), dim3(256), 0, s, n, off, tmp, ucnt);
  GCN_TRY(hipGetLastError());
  hipLaunchKernelGGL(sort_medium_kernel, dim3(grid_for(n, 1, 4096)), dim3(256), 0, s, n, off, tmp, ucnt);
  GCN_TRY(hipGetLastError());
  hipLaunchKernelGGL(sort_large_kernel, dim3(grid_for(n, 1, 1024)), dim3(256), 0, s, n, off, tmp, ucnt);
  GCN_TRY(hipGetLastError());
  hipLaunchKernelGGL(widen_kernel, dim3(grid_for(n + 1)), dim3(256), 0, s, n, ucnt, rp64);
  GCN_TRY(hipGetLastError());
  GCN_TRY(scan_exclusive(rp64, n + 1, scr, s));
  if (idx64)
    hipLaunchKernelGGL(compact_kernel<int64_t>, dim3(wave_rows_grid(n + 1)), dim3(256), 0, s, n, off, tmp, rp64,
                       ucnt, (int64_t*)rowptr, colidx, deg, dinv);
  else
    hipLaunchKernelGGL(compact_kernel<int32_t>, dim3(wave_rows_grid(n + 1)), dim3(256), 0, s, n, off, tmp, rp64,
                       ucnt, (int32_t*)rowptr, colidx, deg, dinv);
  GCN_TRY(hipGetLastError());
  if (dense) GCN_TRY(fill_zero(dense, (size_t)n * (size_t)ld_dense * (value_prec == 0 ? 4 : 2), s));
  if (values || dense) {
    const dim3 g(wave_rows_grid(n));
    switch (value_prec) {
      case 0: hipLaunchKernelGGL(values_kernel<float>, g, dim3(256), 0, s, n, rp64, colidx, dinv, (float*)values, (float*)dense, ld_dense); break;
      case 1: hipLaunchKernelGGL(values_kernel<f16>, g, dim3(256), 0, s, n, rp64, colidx, dinv, (f16*)values, (f16*)dense, ld_dense); break;
      case 2: hipLaunchKernelGGL(values_kernel<bf16>, g, dim3(256), 0, s, n, rp64, colidx, dinv, (bf16*)values, (bf16*)dense, ld_dense); break;
      default: return hipErrorInvalidValue;
    }
    GCN_TRY(hipGetLastError());
  }
  // the one synchronisation: nnz and the bad-id flag back to the host
  int64_t host[2] = {0, 0};
  GCN_TRY(hipMemcpyAsync(&host[0], rp64 + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  int32_t hbad = 0;
  GCN_TRY(hipMemcpyAsync(&hbad, bad, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  GCN_TRY(hipStreamSynchronize(s));
  *nnz_out = host[0];
  *bad_ids = hbad;
#undef GCN_TRY
  return hipSuccess;
}

// Most pieces a schedule can hold: every heavy row (more than thr entries,
// so at most nnz / (thr + 1) of them) has at most one piece per column range
// plus one per chunk_nnz entries.
int64_t max_pieces(int64_t n, int64_t nnz, int64_t thr, int64_t chunk_nnz, int64_t parts) {
  const int64_t rows = std::min<int64_t>(n, nnz / (thr + 1));
  return nnz / chunk_nnz + rows * parts + 1;
}

size_t schedule_bytes(int64_t n, int64_t nnz, int64_t thr, int64_t chunk_nnz, int64_t parts) {
  const int64_t max_chunks = max_pieces(n, nnz, thr, chunk_nnz, parts);
  const int64_t nb = light_buckets(n, thr);
  int64_t scan_n = (n + 1 > nb + 1) ? n + 1 : nb + 1;
  if (scan_n < CHUNK_BUCKETS + 1) scan_n = CHUNK_BUCKETS + 1;
  size_t b = 0;
  b += align256(sizeof(int32_t) * max_chunks);                  // chunk_order
  b += align256(sizeof(int32_t) * max_chunks);                  // chunk keys
  b += align256(sizeof(int32_t) * CHUNK_BUCKETS);               // chunk bucket histogram
  b += align256(sizeof(int32_t) * CHUNK_BUCKETS);               // chunk bucket cursors
  b += align256(sizeof(int64_t) * (CHUNK_BUCKETS + 1));         // chunk bucket offsets
  b += align256(sizeof(int32_t) * n);                           // heavy_rows
  b += align256(sizeof(int32_t) * (n + 1));                     // heavy_chunk_off
  b += align256(sizeof(int32_t) * max_chunks);                  // chunk_heavy
  b += align256(sizeof(int64_t) * (max_chunks + 1));            // chunk_beg
  b += align256(sizeof(int64_t) * (parts + 1));                 // part_off
  b += align256(sizeof(RowDesc) * max_chunks);                  // piece descriptors
  b += align256(sizeof(int32_t) * max_chunks);                  // launch position of each piece
  b += align256(sizeof(int32_t) * n);                           // fix_rows
  b += align256(sizeof(RowDesc) * n);                           // light-row descriptors
  b += align256(sizeof(int32_t) * n);                           // row_perm
  b += align256(sizeof(int64_t) * (n + 1));                     // flags -> heavy index
  b += align256(sizeof(int64_t) * (n + 1));                     // pieces per row -> piece offsets
  b += align256(sizeof(int32_t) * nb);                          // (block, degree) histogram
  b += align256(sizeof(int32_t) * nb);                          // bucket cursors
  b += align256(sizeof(int64_t) * (nb + 1));                    // bucket offsets
  b += align256(sizeof(int64_t) * scan_scratch_elems(scan_n));  // scan scratch
  return b;
}

hipError_t schedule_run(int64_t n, int64_t nnz, bool idx64, const void* rowptr, const int32_t* colidx, int64_t thr,
                        int64_t chunk, int64_t parts, void* sched, size_t sched_bytes, SchedOut* out, hipStream_t s) {
  char* w = static_cast<char*>(sched);
  auto take = [&](size_t bytes) { char* p = w; w += align256(bytes); return p; };
  const int64_t max_chunks = max_pieces(n, nnz, thr, chunk, parts);
  const int64_t nb = light_buckets(n, thr);
  int64_t scan_n = (n + 1 > nb + 1) ? n + 1 : nb + 1;
  if (scan_n < CHUNK_BUCKETS + 1) scan_n = CHUNK_BUCKETS + 1;
  int32_t* corder = (int32_t*)take(sizeof(int32_t) * max_chunks);
  int32_t* ckey = (int32_t*)take(sizeof(int32_t) * max_chunks);
  int32_t* chist = (int32_t*)take(sizeof(int32_t) * CHUNK_BUCKETS);
  int32_t* ccur = (int32_t*)take(sizeof(int32_t) * CHUNK_BUCKETS);
  int64_t* cboff = (int64_t*)take(sizeof(int64_t) * (CHUNK_BUCKETS + 1));
  int32_t* hr = (int32_t*)take(sizeof(int32_t) * n);
  int32_t* hco = (int32_t*)take(sizeof(int32_t) * (n + 1));
  int32_t* ch = (int32_t*)take(sizeof(int32_t) * max_chunks);
  int64_t* cbeg = (int64_t*)take(sizeof(int64_t) * (max_chunks + 1));
  int64_t* poff = (int64_t*)take(sizeof(int64_t) * (parts + 1));
  RowDesc* pdesc = (RowDesc*)take(sizeof(RowDesc) * max_chunks);
  int32_t* ppos = (int32_t*)take(sizeof(int32_t) * max_chunks);
  int32_t* fixr = (int32_t*)take(sizeof(int32_t) * n);
  RowDesc* ldesc = (RowDesc*)take(sizeof(RowDesc) * n);
  int32_t* perm = (int32_t*)take(sizeof(int32_t) * n);
  int64_t* hidx = (int64_t*)take(sizeof(int64_t) * (n + 1));
  int64_t* choff = (int64_t*)take(sizeof(int64_t) * (n + 1));
  int32_t* hist = (int32_t*)take(sizeof(int32_t) * nb);
  int32_t* cur = (int32_t*)take(sizeof(int32_t) * nb);
  int64_t* boff = (int64_t*)take(sizeof(int64_t) * (nb + 1));
  int64_t* scr = (int64_t*)take(sizeof(int64_t) * scan_scratch_elems(scan_n));
  if ((size_t)(w - static_cast<char*>(sched)) > sched_bytes) return hipErrorInvalidValue;
  hipError_t e;
#define GCN_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  if (idx64)
    hipLaunchKernelGGL(piece_count_kernel<int64_t>, dim3(grid_for(n + 1)), dim3(256), 0, s, n, (const int64_t*)rowptr, colidx, thr, chunk, parts, hidx, choff);
  else
    hipLaunchKernelGGL(piece_count_kernel<int32_t>, dim3(grid_for(n + 1)), dim3(256), 0, s, n, (const int32_t*)rowptr, colidx, thr, chunk, parts, hidx, choff);
  GCN_TRY(hipGetLastError());
  GCN_TRY(scan_exclusive(hidx, n + 1, scr, s));
  GCN_TRY(scan_exclusive(choff, n + 1, scr, s));
  if (idx64)
    hipLaunchKernelGGL(piece_fill_kernel<int64_t>, dim3(grid_for(n + 1)), dim3(256), 0, s, n, nnz, (const int64_t*)rowptr, colidx, thr, chunk, parts, hidx, choff, hr, hco, ch, cbeg);
  else
    hipLaunchKernelGGL(piece_fill_kernel<int32_t>, dim3(grid_for(n + 1)), dim3(256), 0, s, n, nnz, (const int32_t*)rowptr, colidx, thr, chunk, parts, hidx, choff, hr, hco, ch, cbeg);
  GCN_TRY(hipGetLastError());
  // light rows, block by block, by decreasing degree inside a block
  GCN_TRY(fill_zero(hist, sizeof(int32_t) * nb, s));
  GCN_TRY(fill_zero(cur, sizeof(int32_t) * nb, s));
  if (idx64)
    hipLaunchKernelGGL(light_hist_kernel<int64_t>, dim3(grid_for(n)), dim3(256), 0, s, n, (const int64_t*)rowptr, thr, light_block(n), nb, hist);
  else
    hipLaunchKernelGGL(light_hist_kernel<int32_t>, dim3(grid_for(n)), dim3(256), 0, s, n, (const int32_t*)rowptr, thr, light_block(n), nb, hist);
  GCN_TRY(hipGetLastError());
  hipLaunchKernelGGL(widen_kernel, dim3(grid_for(nb + 1)), dim3(256), 0, s, nb, hist, boff);
  GCN_TRY(hipGetLastError());
  GCN_TRY(scan_exclusive(boff, nb + 1, scr, s));
  if (idx64)
    hipLaunchKernelGGL(light_scatter_kernel<int64_t>, dim3(grid_for(n)), dim3(256), 0, s, n, (const int64_t*)rowptr, thr, light_block(n), nb, boff, cur, perm);
  else
    hipLaunchKernelGGL(light_scatter_kernel<int32_t>, dim3(grid_for(n)), dim3(256), 0, s, n, (const int32_t*)rowptr, thr, light_block(n), nb, boff, cur, perm);
  GCN_TRY(hipGetLastError());
  int64_t host[4] = {0, 0, 0, 0};
  GCN_TRY(hipMemcpyAsync(&host[0], hidx + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  GCN_TRY(hipMemcpyAsync(&host[1], choff + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  GCN_TRY(hipMemcpyAsync(&host[2], boff + nb, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  GCN_TRY(hipMemcpyAsync(&host[3], boff + nb - 1, sizeof(int64_t), hipMemcpyDeviceToHost, s));
  GCN_TRY(hipStreamSynchronize(s));
  // light-row descriptors in row_perm order
  if (host[2] > 0) {
    if (idx64)
      hipLaunchKernelGGL(light_desc_kernel<int64_t>, dim3(grid_for(host[2])), dim3(256), 0, s, host[2], (const int64_t*)rowptr, perm, ldesc);
    else
      hipLaunchKernelGGL(light_desc_kernel<int32_t>, dim3(grid_for(host[2])), dim3(256), 0, s, host[2], (const int32_t*)rowptr, perm, ldesc);
    GCN_TRY(hipGetLastError());
  }
  // pieces in order of the column bucket of their first entry, which groups
  // them by column range
  const int64_t nch = host[1];
  if (nch > max_chunks) return hipErrorInvalidValue;
  int64_t slots = 0, n_fix = 0, n_fix_big = 0;
  if (nch > 0) {
    GCN_TRY(fill_zero(chist, sizeof(int32_t) * CHUNK_BUCKETS, s));
    GCN_TRY(fill_zero(ccur, sizeof(int32_t) * CHUNK_BUCKETS, s));
    hipLaunchKernelGGL(chunk_key_kernel, dim3(grid_for(nch)), dim3(256), 0, s, n, nch, colidx, cbeg, ckey, chist);
    GCN_TRY(hipGetLastError());
    hipLaunchKernelGGL(widen_kernel, dim3(grid_for(CHUNK_BUCKETS + 1)), dim3(256), 0, s, CHUNK_BUCKETS, chist, cboff);
    GCN_TRY(hipGetLastError());
    GCN_TRY(scan_exclusive(cboff, CHUNK_BUCKETS + 1, scr, s));
    hipLaunchKernelGGL(chunk_scatter_kernel, dim3(grid_for(nch)), dim3(256), 0, s, nch, ckey, cboff, ccur, corder);
    GCN_TRY(hipGetLastError());
    hipLaunchKernelGGL(part_off_kernel, dim3(grid_for(parts + 1)), dim3(256), 0, s, parts, cboff, poff);
    GCN_TRY(hipGetLastError());
    if (idx64)
      hipLaunchKernelGGL(piece_desc_kernel<int64_t>, dim3(grid_for(nch)), dim3(256), 0, s, nch, (const int64_t*)rowptr, corder, ch, hr, hco, cbeg, pdesc, ppos);
    else
      hipLaunchKernelGGL(piece_desc_kernel<int32_t>, dim3(grid_for(nch)), dim3(256), 0, s, nch, (const int32_t*)rowptr, corder, ch, hr, hco, cbeg, pdesc, ppos);
    GCN_TRY(hipGetLastError());
    // rows for the fix-up; hidx and choff (free again) hold the flag scans
    const int64_t nh = host[0];
    hipLaunchKernelGGL(fix_flag_kernel, dim3(grid_for(nh + 1)), dim3(256), 0, s, nh, hco, hidx, choff);
    GCN_TRY(hipGetLastError());
    GCN_TRY(scan_exclusive(hidx, nh + 1, scr, s));
    GCN_TRY(scan_exclusive(choff, nh + 1, scr, s));
    hipLaunchKernelGGL(fix_scatter_kernel, dim3(grid_for(nh)), dim3(256), 0, s, nh, hco, hidx, choff, fixr);
    GCN_TRY(hipGetLastError());
    int64_t nfix[2] = {0, 0};
    GCN_TRY(hipMemcpyAsync(&nfix[0], hidx + nh, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    GCN_TRY(hipMemcpyAsync(&nfix[1], choff + nh, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    // the most pieces one XCD takes: ranges x, x + 8, ... run on XCD x
    std::vector<int64_t> hp((size_t)parts + 1);
    GCN_TRY(hipMemcpyAsync(hp.data(), poff, sizeof(int64_t) * (parts + 1), hipMemcpyDeviceToHost, s));
    GCN_TRY(hipStreamSynchronize(s));
    n_fix_big = nfix[0];
    n_fix = nfix[0] + nfix[1];
    if (parts > 1) {
      for (int64_t x = 0; x < XCDS; ++x) {
        int64_t t = 0;
        for (int64_t q = x; q < parts; q += XCDS) t += hp[q + 1] - hp[q];
        slots = std::max(slots, t);
      }
    } else {
      slots = nch;
    }
  }
#undef GCN_TRY
  out->heavy_rows = hr; out->heavy_chunk_off = hco; out->chunk_heavy = ch; out->row_perm = perm;
  out->chunk_order = nch > 0 ? corder : nullptr;
  out->chunk_beg = cbeg; out->part_off = poff; out->part_slots = slots;
  out->piece_desc = pdesc; out->piece_pos = ppos; out->row_desc = ldesc;
  out->fix_rows = fixr; out->n_fix = n_fix; out->n_fix_big = n_fix_big;
  out->n_heavy = host[0]; out->n_chunks = nch; out->n_light = host[2]; out->n_light_single = host[2] - host[3];
  return hipSuccess;
}

}  // namespace gcn

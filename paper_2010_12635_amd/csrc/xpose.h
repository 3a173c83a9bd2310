// In-register transposes of small square blocks held as 16-byte rows, used
// where an operand stored vertex-major must become k-contiguous for MFMA.
#pragma once

#include "common.h"

namespace gcn {

// VE x VE block: in[i] is row i (VE consecutive elements of one row), out[j]
// is column j (element i = row i).  VE = 8 for 16-bit types, 4 for fp32.
__device__ __forceinline__ void transpose_block(const uint4* in, uint4* out, f16) {
  // 8 x 8 halves: output dword e of column c packs rows 2e and 2e+1
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    uint32_t d[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = (&in[2 * e].x)[c >> 1], hi = (&in[2 * e + 1].x)[c >> 1];
      // v_perm_b32: bytes {hi, lo} selected; low half for even c, high half for odd c
      d[e] = (c & 1) ? __builtin_amdgcn_perm(hi, lo, 0x07060302u) : __builtin_amdgcn_perm(hi, lo, 0x05040100u);
    }
    out[c] = make_uint4(d[0], d[1], d[2], d[3]);
  }
}
__device__ __forceinline__ void transpose_block(const uint4* in, uint4* out, bf16) {
  transpose_block(in, out, f16());
}
__device__ __forceinline__ void transpose_block(const uint4* in, uint4* out, float) {
  out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
  out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
  out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
  out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
}

// Keep the first vc (0..VE) elements of a 16-byte vector and zero the rest,
// with dword masks (the vector is never split into 16-bit pieces).
template <typename T>
__device__ __forceinline__ uint4 keep_first(uint4 x, int vc) {
  uint32_t m[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (Vec<T>::N == 8)
      m[w] = (2 * w < vc ? 0x0000ffffu : 0u) | (2 * w + 1 < vc ? 0xffff0000u : 0u);
    else
      m[w] = w < vc ? 0xffffffffu : 0u;
  }
  return make_uint4(x.x & m[0], x.y & m[1], x.z & m[2], x.w & m[3]);
}

}  // namespace gcn

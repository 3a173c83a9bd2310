// Dispatch of the CSR aggregation (kernels in spmm_impl.h, instantiated per
// storage type in spmm_f32.hip, spmm_f16.hip and spmm_bf16.hip) and the size
// of its partial-row buffer.
#include "internal.h"

namespace gcn {

hipError_t spmm_launch_f32(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                           float* partials, hipStream_t s);
hipError_t spmm_launch_f16(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                           float* partials, hipStream_t s);
hipError_t spmm_launch_bf16(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                            float* partials, hipStream_t s);

namespace {

int lpr_for(int prec, int64_t F) {
  const int VE = prec == 0 ? 4 : 8;
  const int64_t nvec = (F + VE - 1) / VE;
  int l = 1;
  while (l < nvec && l < 64) l <<= 1;
  return l;
}

}  // namespace

// Floats of the heavy-row partials: enough for the widest lane groups, and
// so also when the launch gathers in narrower column blocks.
int64_t spmm_partials_floats(const CsrView& A, int prec, int64_t F) {
  if (A.n_heavy <= 0) return 0;
  const int VE = prec == 0 ? 4 : 8;
  const int lpr = lpr_for(prec, F);
  const int64_t colblocks = (F + (int64_t)lpr * VE - 1) / ((int64_t)lpr * VE);
  return A.n_chunks * colblocks * lpr * VE;
}

hipError_t spmm_launch(const CsrView& A, int prec, const void* X, int64_t ldx, int64_t F,
                       const Epilogue& epi, float* partials, hipStream_t s) {
  switch (prec) {
    case 0: return spmm_launch_f32(A, X, ldx, F, epi, partials, s);
    case 1: return spmm_launch_f16(A, X, ldx, F, epi, partials, s);
    case 2: return spmm_launch_bf16(A, X, ldx, F, epi, partials, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace gcn

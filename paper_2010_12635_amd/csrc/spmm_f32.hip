// CSR aggregation kernels instantiated for f32 storage (one translation
// unit per storage type keeps the build parallel).
#include "spmm_impl.h"

namespace gcn {

hipError_t spmm_launch_f32(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                           float* partials, hipStream_t s) {
  return launch_t<float>(A, X, ldx, F, epi, partials, s);
}

}  // namespace gcn

// CSR aggregation kernels instantiated for f16 storage (one translation
// unit per storage type keeps the build parallel).
#include "spmm_impl.h"

namespace gcn {

hipError_t spmm_launch_f16(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                           float* partials, hipStream_t s) {
  return launch_t<f16>(A, X, ldx, F, epi, partials, s);
}

}  // namespace gcn

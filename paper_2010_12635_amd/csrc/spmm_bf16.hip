// CSR aggregation kernels instantiated for bf16 storage (one translation
// unit per storage type keeps the build parallel).
#include "spmm_impl.h"

namespace gcn {

hipError_t spmm_launch_bf16(const CsrView& A, const void* X, int64_t ldx, int64_t F, const Epilogue& epi,
                           float* partials, hipStream_t s) {
  return launch_t<bf16>(A, X, ldx, F, epi, partials, s);
}

}  // namespace gcn

// GEMM kernels instantiated for bf16 operands (see gemm_kernels.h).
#include "gemm_kernels.h"

namespace mpx {

hipError_t run_gemm_bf16(const GemmArgs& g, bool ak, bool bk, int64_t nbatch, hipStream_t s,
                         bool* db_fused) {
  return run_gemm<MPX_BF16>(g, ak, bk, nbatch, s, db_fused);
}

}  // namespace mpx

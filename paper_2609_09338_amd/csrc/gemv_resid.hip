// Instantiations of the weight-streaming products for one input/epilogue kind
// (one file per kind so that they compile in parallel): the wavefront GEMV for
// one row or fp32 weights, the matrix-core GEMM for several rows of bf16 weights.
#include "gemm_mfma.h"
#include "gemv_kernel.h"

namespace osp {

void launch_gemv_resid(int wdtype, const GemvArgs& a, hipStream_t st) {
  if (gemm_use_mfma(wdtype, a.max_rows)) launch_gemm_mfma_t<SRC_PLAIN, EPI_RESID>(a, st);
  else launch_gemv_kind<SRC_PLAIN, EPI_RESID>(wdtype, a, st);
}

}  // namespace osp

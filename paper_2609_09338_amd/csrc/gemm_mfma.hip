// Instantiations and dispatch of the matrix-core GEMM (kernel in gemm_mfma.h).
#include "gemm_mfma.h"

namespace osp {

// Passes of two or more rows of bf16 weights take the matrix-core path.
bool gemm_use_mfma(int wdtype, int rows) { return wdtype == 1 && rows >= 2; }

int gemm_rows_per_block(EpiKind epi) { return gemm_mfma_rows_per_block(epi); }

int launch_gemm(SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st) {
  if (src == SRC_TAPS && epi == EPI_STORE) return launch_gemm_mfma_t<SRC_TAPS, EPI_STORE>(a, st);
  if (src == SRC_PREP && epi == EPI_STORE) return launch_gemm_mfma_t<SRC_PREP, EPI_STORE>(a, st);
  if (src == SRC_PREP && epi == EPI_SWIGLU) return launch_gemm_mfma_t<SRC_PREP, EPI_SWIGLU>(a, st);
  if (src == SRC_PREP && epi == EPI_LOGITS) return launch_gemm_mfma_t<SRC_PREP, EPI_LOGITS>(a, st);
  return 0;
}

}  // namespace osp

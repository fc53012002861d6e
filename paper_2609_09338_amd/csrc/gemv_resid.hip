// Instantiations of the wavefront GEMV for one input/epilogue kind (one file per
// kind so that they compile in parallel).
#include "gemv_kernel.h"

namespace osp {

void launch_gemv_resid(int wdtype, const GemvArgs& a, hipStream_t st) {
  launch_gemv_kind<SRC_PLAIN, EPI_RESID>(wdtype, a, st);
}

bool gemv_attn_supported(int wdtype, int rows, int Kd, int hd, int n_split) {
  return wdtype == 1 && rows == 1 && hd > 0 && hd % 8 == 0 && Kd % hd == 0 && Kd <= 8 * kGemvThreads &&
         Kd / hd <= kGemvAttnMaxHeads && n_split >= 1 && n_split <= kGemvAttnMaxSplit;
}

// O projection + residual of one row whose input is merged from the attention's
// context splits (SRC_ATTN); the caller has checked gemv_attn_supported.  One output
// row per wavefront, as the plain projection (fewer, wider blocks measured slower).
void launch_gemv_attn_resid(const GemvArgs& a, hipStream_t st) {
  const GemvPlan p = gemv_plan(1, EPI_RESID, 1, a.N, a.Kd);
  if (p.xv == 4) return launch_gemv_nw<bf16_t, SRC_ATTN, EPI_RESID, 1, 4>(p, a, st);
  if (p.xv == 2) return launch_gemv_nw<bf16_t, SRC_ATTN, EPI_RESID, 1, 2>(p, a, st);
  return launch_gemv_nw<bf16_t, SRC_ATTN, EPI_RESID, 1, 1>(p, a, st);
}

}  // namespace osp

// Instantiations of the wavefront GEMV for the expanded-QKV input (one file per kind so
// that they compile in parallel), with the single-sequence form that draws its token.
#include "gemv_kernel.h"

namespace osp {

void launch_gemv_qkv(int wdtype, const GemvArgs& a, hipStream_t st) {
  launch_gemv_kind<SRC_QKV, EPI_STORE>(wdtype, a, st);
}

bool gemv_pick_supported(int wdtype, int rows, int nblk) {
  return wdtype == 1 && rows == 1 && nblk >= 1 && nblk <= kPickMaxRecords;
}

// The caller has checked gemv_pick_supported; the shape is the plain single-row QKV's.
void launch_gemv_qkv_pick(const GemvArgs& a, hipStream_t st) {
  const GemvPlan p = gemv_plan(1, EPI_STORE, 1, a.N, a.Kd);
  launch_gemv_xv<bf16_t, SRC_QKV_PICK, EPI_STORE, 1>(p, a, st);
}

}  // namespace osp

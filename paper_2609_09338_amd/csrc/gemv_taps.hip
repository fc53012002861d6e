// Instantiations of the wavefront GEMV for one input/epilogue kind (one file per
// kind so that they compile in parallel).
#include "gemv_kernel.h"

namespace osp {

void launch_gemv_taps(int wdtype, const GemvArgs& a, hipStream_t st) {
  launch_gemv_kind<SRC_TAPS, EPI_STORE>(wdtype, a, st);
}

}  // namespace osp

// Dispatch of the weight-streaming GEMV kinds (kernel in gemv_kernel.h).
#include "gemv_kernel.h"

namespace osp {

void launch_gemv_taps(int wdtype, const GemvArgs& a, hipStream_t st);
void launch_gemv_qkv(int wdtype, const GemvArgs& a, hipStream_t st);
void launch_gemv_resid(int wdtype, const GemvArgs& a, hipStream_t st);
void launch_gemv_swiglu(int wdtype, const GemvArgs& a, hipStream_t st);
void launch_gemv_logits(int wdtype, const GemvArgs& a, hipStream_t st);

void launch_gemv(int wdtype, SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st) {
  if (src == SRC_TAPS && epi == EPI_STORE) return launch_gemv_taps(wdtype, a, st);
  if (src == SRC_QKV && epi == EPI_STORE) return launch_gemv_qkv(wdtype, a, st);
  if (src == SRC_PLAIN && epi == EPI_RESID) return launch_gemv_resid(wdtype, a, st);
  if (src == SRC_NORM && epi == EPI_SWIGLU) return launch_gemv_swiglu(wdtype, a, st);
  if (src == SRC_NORM && epi == EPI_LOGITS) return launch_gemv_logits(wdtype, a, st);
}

GemvShape gemv_shape(int wdtype, EpiKind epi, int rows, int N, int Kd) {
  if (gemm_use_mfma(wdtype, rows)) {
    GemvShape s;
    s.rows_per_wave = gemm_rows_per_block(epi);
    s.waves = (N + s.rows_per_wave - 1) / s.rows_per_wave;
    return s;
  }
  const GemvPlan p = gemv_plan(wdtype, epi, rows, N, Kd);
  GemvShape s;
  s.rows_per_wave = p.rpw;
  s.waves = p.waves;
  return s;
}

}  // namespace osp

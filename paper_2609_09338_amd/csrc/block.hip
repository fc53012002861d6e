// Block drafting (the EAGLE-style interface of the DFlash ablation, appendix): the rows
// of the block pass.  Sequence b's rows b K + j are its anchor (j = 0: the last ingested
// token, at committed - 1, its keys/values already cached) and K - 1 mask rows at the
// positions after it; all take the anchor's conditioning input (the target feature is
// taken once at the anchor and broadcast over the block) and the sequence's drafter
// temperature.
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kBlockThreads = 256;

__global__ void __launch_bounds__(kBlockThreads) k_block_rows(BlockArgs a) {
  const int b = blockIdx.x, tid = threadIdx.x;
  const int K = a.K;
  const int lr = a.last_row[b];
  const int L = a.committed[b];
  for (int j = tid; j < K; j += kBlockThreads) {
    const int r = b * K + j;
    a.r_seq[r] = b;
    a.r_tok[r] = j == 0 ? a.ing_tok[lr] : a.mask;
    a.r_pos[r] = L - 1 + j;
    a.r_skip[r] = j == 0 ? 1 : 0;
    a.r_temp[r] = a.temp[b];
  }
  if (tid == 0) {
    a.r_cu[b] = b * K;
    if (b == a.B - 1) a.r_cu[a.B] = a.B * K;
  }
  const float4* src = reinterpret_cast<const float4*>(a.s + (long)lr * a.d);
  for (int j = 0; j < K; ++j) {
    float4* dst = reinterpret_cast<float4*>(a.r_s + (long)(b * K + j) * a.d);
    for (int i = tid; i < a.d / 4; i += kBlockThreads) dst[i] = src[i];
  }
}

void launch_block_rows(const BlockArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_block_rows, dim3(a.B), dim3(kBlockThreads), 0, st, a);
}

}  // namespace osp

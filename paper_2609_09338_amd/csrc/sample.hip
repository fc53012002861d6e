// Draft-token selection from the LM-head statistics (the pick itself: pick.h).
//
// One block per sequence: the pick of its row, then the token, its position and the
// last-layer hidden state (fed back as the next step's conditioning input) are written
// for the next autoregressive step, and the row's (S, M, lowest argmax) for the
// verification of the chain.
#include "common.h"
#include "internal.h"
#include "pick.h"

namespace osp {

// (threads per sequence: 64 / 128 / 256 / 512 / 1024 measured 1009 / 939 / 913 / 904 / 909 us
// per c2 draft call: the records' per-thread serial work outweighs the barriers)
constexpr int kSampleThreads = 512;
constexpr int kPer = (kGemvMaxWaves + kSampleThreads - 1) / kSampleThreads;  // records per thread

__global__ void __launch_bounds__(kSampleThreads) k_sample(SampleArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int k = a.block ? (int)blockIdx.y : a.k;  // (block drafting: proposal k of sequence b)
  const int prow = a.block ? b * a.K + k : b;     // its records' and logits' row
  const float* part = a.part + (long)prow * a.nblk * 4;
  PickRecs<kPer> rec;
  pick_request<kSampleThreads, kPer>(rec, part, a.nblk);
  // the hidden state fed back to the next step does not depend on the pick: read it
  // now, with the records, so its load is not one more round trip at the end
  constexpr int kFbPer = 4096 / (kSampleThreads * 4);   // d <= 4096 = kSampleThreads * 4 * kFbPer
  const int xr = a.gather ? a.gather[b] : b;
  float4 fb[kFbPer];
#pragma unroll
  for (int q = 0; q < kFbPer; ++q) {
    const int c = (tid + q * kSampleThreads) * 4;
    fb[q] = c < a.d ? *reinterpret_cast<const float4*>(a.x + (long)xr * a.d + c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const float* lg = a.logits + (long)b * a.ld_logits + (a.block ? (long)k * a.V : 0L);
  const Pick p = pick_draft<kSampleThreads, kPer>(rec, a.nblk, a.blk_rows, lg, a.V, a.d2t, a.temp[b],
                                                  a.u[(long)b * a.K + k]);
  if (tid == 0) {
    a.drafts[(long)b * a.ld_drafts + k] = p.tok;
    if (a.drafts_out) a.drafts_out[(long)b * a.K + k] = p.tok;
    if (!a.block) {
      a.ar_tok[b] = p.tok;
      a.ar_pos[b] = a.committed[b] + k;
    }
    // the row's statistics, for the verification of this draft
    if (a.qstat) a.qstat[(long)b * a.ld_qstat + k] = QStat{p.S, p.M, p.am};
  }
#pragma unroll
  for (int q = 0; q < kFbPer; ++q) {
    const int c = (tid + q * kSampleThreads) * 4;
    if (c < a.d) *reinterpret_cast<float4*>(a.gfb + (long)b * a.d + c) = fb[q];
  }
}

void launch_sample(const SampleArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_sample, dim3(a.B, a.block ? a.K : 1), dim3(kSampleThreads), 0, st, a);
}

}  // namespace osp

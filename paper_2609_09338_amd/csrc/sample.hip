// Draft-token selection from the LM-head block statistics.
//
// One block per sequence.  The LM-head kernel left, for every block of TN
// logits, (max, sum exp((l - max)/T), lowest argmax).  Here they are merged in
// block order: at T = 0 the draft is the lowest-index argmax; at T > 0 the
// inverse CDF of softmax(l / T) over drafter rows in ascending order picks the
// smallest row whose running sum exceeds u * S -- the block holding that point
// is found from the block sums, then that block's logits are scanned.  The row
// is mapped to a target id through d2t; the token, its position and the
// last-layer hidden state (fed back as the next step's conditioning input) are
// written for the next autoregressive step.
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kSampleThreads = 256;

__global__ void __launch_bounds__(kSampleThreads) k_sample(SampleArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float s_wm[4];
  __shared__ int s_wi[4];
  __shared__ double s_scan[4];
  __shared__ double s_before, s_target;
  __shared__ int s_blk, s_row;

  const float* part = a.part + (long)b * a.nblk * 4;
  // ---- global max and lowest argmax -------------------------------------------------
  float m = -INFINITY;
  int am = 0x7fffffff;
  for (int i = tid; i < a.nblk; i += kSampleThreads) {
    const float v = part[i * 4 + 0];
    const int ai = __float_as_int(part[i * 4 + 2]);
    if (v > m || (v == m && v > -INFINITY && ai < am)) { m = v; am = ai; }
  }
  {
    const float wm = wave_max(m);
    const int wi = wave_min_i((m == wm && m > -INFINITY) ? am : 0x7fffffff);
    if (lane == 0) { s_wm[wave] = wm; s_wi[wave] = wi; }
    __syncthreads();
    float bm = -INFINITY;
    int bi = 0x7fffffff;
    for (int w = 0; w < 4; ++w) {
      if (s_wm[w] > bm) { bm = s_wm[w]; bi = s_wi[w]; }
      else if (s_wm[w] == bm && s_wi[w] < bi) bi = s_wi[w];
    }
    m = bm;
    am = bi;
    __syncthreads();
  }
  const float M = m;
  const int amax = am;
  const float T = a.temp[b];
  int row;
  if (T <= 0.f || M == -INFINITY) {
    row = amax;
  } else {
    // ---- block sums rescaled to the global max; thread t owns a contiguous range ----
    const int per = (a.nblk + kSampleThreads - 1) / kSampleThreads;
    const int i0 = min(a.nblk, tid * per), i1 = min(a.nblk, i0 + per);
    // sums in float64: the breakpoints of a 10^5-entry CDF are ~1e-5 of the total apart
    double loc = 0.0;
    for (int i = i0; i < i1; ++i) {
      const float bm = part[i * 4 + 0];
      if (bm > -INFINITY) loc += (double)part[i * 4 + 1] * (double)__expf((bm - M) / T);
    }
    double incl, tot;
    const double excl = block_scan<kSampleThreads, double>(loc, s_scan, incl, tot);
    const double target = (double)a.u[(long)b * a.K + a.k] * tot;
    if (tid == 0) { s_blk = -1; s_row = -1; }
    __syncthreads();
    if (i0 < i1 && excl <= target && incl > target) {
      double run = excl;
      for (int i = i0; i < i1; ++i) {
        const float bm = part[i * 4 + 0];
        const double bs = bm > -INFINITY ? (double)part[i * 4 + 1] * (double)__expf((bm - M) / T) : 0.0;
        if (run + bs > target || i == i1 - 1) { s_blk = i; s_before = run; break; }
        run += bs;
      }
    }
    __syncthreads();
    if (tid == 0 && s_blk < 0) {        // rounding pushed the target past the last block
      int last = a.nblk - 1;
      while (last > 0 && !(part[last * 4 + 0] > -INFINITY)) --last;
      s_blk = last;
      s_before = 0.0;
    }
    if (tid == 0) s_target = target;
    __syncthreads();
    // ---- scan the chosen block's logits with one wavefront ----------------------------
    if (wave == 0) {
      const int r0 = s_blk * a.blk_rows;
      const int r1 = min(r0 + a.blk_rows, a.V);
      const float* lg = a.logits + (long)b * a.ld_logits;
      double run = s_before;
      const double tg = s_target;
      int last_pos = -1, found = -1;
      for (int c0 = r0; c0 < r1; c0 += OSP_WAVE) {
        const int i = c0 + lane;
        const float li = i < r1 ? lg[i] : -INFINITY;
        const float w = li > -INFINITY ? __expf((li - M) / T) : 0.f;
        const float inc = wave_incl_scan<float>(w);
        const unsigned long long hit = __ballot(w > 0.f && run + (double)inc > tg);
        const unsigned long long pos = __ballot(w > 0.f);
        if (pos) last_pos = c0 + 63 - __builtin_clzll(pos);
        if (hit) { found = c0 + __builtin_ctzll(hit); break; }
        run += (double)__shfl(inc, 63, OSP_WAVE);
      }
      if (lane == 0) s_row = found >= 0 ? found : (last_pos >= 0 ? last_pos : amax);
    }
    __syncthreads();
    row = s_row;
  }
  row = min(max(row, 0), a.V - 1);
  const int d = a.d2t[row];
  if (tid == 0) {
    a.drafts[(long)b * a.ld_drafts + a.k] = d;
    if (a.drafts_out) a.drafts_out[(long)b * a.K + a.k] = d;
    a.ar_tok[b] = d;
    a.ar_pos[b] = a.committed[b] + a.k;
  }
  const int xr = a.gather ? a.gather[b] : b;
  for (int c = tid; c < a.d; c += kSampleThreads) a.gfb[(long)b * a.d + c] = a.x[(long)xr * a.d + c];
}

void launch_sample(const SampleArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_sample, dim3(a.B), dim3(kSampleThreads), 0, st, a);
}

}  // namespace osp

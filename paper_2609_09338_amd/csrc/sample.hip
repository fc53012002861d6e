// Draft-token selection from the LM-head statistics.
//
// One block per sequence.  The LM-head kernel left one record per wavefront
// range of logits: (max, sum exp((l - max)/T), lowest argmax).  Here they are
// merged in range order: at T = 0 the draft is the lowest-index argmax; at
// T > 0 the inverse CDF of softmax(l / T) over drafter rows in ascending order
// picks the smallest row whose running sum exceeds u * S -- the range holding
// that point is found from the range sums (float64 prefix), then that range's
// logits are scanned.  The row is mapped to a target id through d2t; the token,
// its position and the last-layer hidden state (fed back as the next step's
// conditioning input) are written for the next autoregressive step, and the row's
// (S, M, lowest argmax) for the verification of the chain.
#include "common.h"
#include "internal.h"

namespace osp {

// (threads per sequence: 64 / 128 / 256 / 512 / 1024 measured 1009 / 939 / 913 / 904 / 909 us
// per c2 draft call: the records' per-thread serial work outweighs the barriers)
constexpr int kSampleThreads = 512;
constexpr int kSampleWaves = kSampleThreads / OSP_WAVE;
constexpr int kPer = (kGemvMaxWaves + kSampleThreads - 1) / kSampleThreads;  // records per thread

__global__ void __launch_bounds__(kSampleThreads) k_sample(SampleArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float s_wm[kSampleWaves];
  __shared__ int s_wi[kSampleWaves];
  __shared__ double s_scan[kSampleWaves];
  __shared__ double s_before;
  __shared__ int s_blk, s_row, s_map;

  const int k = a.block ? (int)blockIdx.y : a.k;  // (block drafting: proposal k of sequence b)
  const int prow = a.block ? b * a.K + k : b;     // its records' and logits' row
  const float* part = a.part + (long)prow * a.nblk * 4;
  const float T = a.temp[b];
  const float u = a.u[(long)b * a.K + k];
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
  // ---- this thread's contiguous records, all loads issued together ----------------
  const int i0 = tid * kPer;
  float bm[kPer], bs[kPer];
  int ba[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = i0 + q;
    if (i < a.nblk) {
      const float4 r = *reinterpret_cast<const float4*>(part + i * 4);
      bm[q] = r.x;
      bs[q] = r.y;
      ba[q] = __float_as_int(r.z);
    } else {
      bm[q] = -INFINITY;
      bs[q] = 0.f;
      ba[q] = -1;
    }
  }
  // ---- global max and lowest argmax ------------------------------------------------
  float m = -INFINITY;
  int am = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < kPer; ++q)
    if (bm[q] > m) { m = bm[q]; am = ba[q]; }   // ascending records: first hit has the lowest id
  {
    const float wm = wave_max(m);
    const int wi = wave_min_i((m == wm && m > -INFINITY) ? am : 0x7fffffff);
    if (lane == 0) { s_wm[wave] = wm; s_wi[wave] = wi; }
    __syncthreads();
    float gm = -INFINITY;
    int gi = 0x7fffffff;
    for (int w = 0; w < kSampleWaves; ++w) {
      if (s_wm[w] > gm) { gm = s_wm[w]; gi = s_wi[w]; }
      else if (s_wm[w] == gm && s_wi[w] < gi) gi = s_wi[w];
    }
    m = gm;
    am = gi;
  }
  const float M = m;
  int row;
  double S = 0.0;
  if (T <= 0.f || M == -INFINITY) {
    row = am;
  } else {
    // range sums rescaled to the global max, prefix in float64 (the breakpoints of a
    // 10^5-entry CDF are ~1e-5 of the total apart)
    double bsum[kPer];
    double loc = 0.0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      bsum[q] = bm[q] > -INFINITY ? (double)bs[q] * (double)__expf((bm[q] - M) / T) : 0.0;
      loc += bsum[q];
    }
    double incl, tot;
    const double excl = block_scan<kSampleThreads, double>(loc, s_scan, incl, tot);
    S = tot;
    const double target = (double)u * tot;
    if (tid == 0) { s_blk = -1; s_row = -1; }
    __syncthreads();
    if (excl <= target && incl > target) {
      double run = excl;
      int hit = -1;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        if (hit < 0 && i0 + q < a.nblk) {
          if (run + bsum[q] > target) { hit = q; } else { run += bsum[q]; }
        }
      }
      if (hit < 0) {   // rounding: the last non-empty record of this thread
        run = excl;
        for (int q = 0; q < kPer; ++q)
          if (i0 + q < a.nblk && bsum[q] > 0.0) { hit = q; }
        for (int q = 0; q < hit; ++q) run += bsum[q];
      }
      if (hit >= 0) { s_blk = i0 + hit; s_before = run; }
    }
    __syncthreads();
    if (tid == 0 && s_blk < 0) {        // rounding pushed the target past the last record
      int last = a.nblk - 1;
      while (last > 0 && !(part[last * 4 + 0] > -INFINITY)) --last;
      s_blk = last;
      double run = 0.0;
      for (int i = 0; i < last; ++i) {
        const float mm = part[i * 4 + 0];
        if (mm > -INFINITY) run += (double)part[i * 4 + 1] * (double)__expf((mm - M) / T);
      }
      s_before = run;
    }
    __syncthreads();
    // ---- scan the chosen range's logits with one wavefront; the first kScanPre x 64 of
    //      them are requested at once (a range holds 16 T <= 128 logits) -------------------
    if (wave == 0) {
      constexpr int kScanPre = 2;
      const int r0 = s_blk * a.blk_rows;
      const int r1 = min(r0 + a.blk_rows, a.V);
      const float* lg = a.logits + (long)b * a.ld_logits + (a.block ? (long)k * a.V : 0L);
      float pre[kScanPre];
      int pmap[kScanPre];   // the range's vocabulary map, requested with its logits
#pragma unroll
      for (int q = 0; q < kScanPre; ++q) {
        const int i = r0 + q * OSP_WAVE + lane;
        pre[q] = i < r1 ? lg[i] : -INFINITY;
        pmap[q] = a.d2t[min(i, a.V - 1)];
      }
      double run = s_before;
      int last_pos = -1, found = -1;
      for (int c0 = r0, q = 0; c0 < r1; c0 += OSP_WAVE, ++q) {
        const int i = c0 + lane;
        float li = -INFINITY;
#pragma unroll
        for (int p = 0; p < kScanPre; ++p)
          if (p == q) li = pre[p];
        if (q >= kScanPre) li = i < r1 ? lg[i] : -INFINITY;
        const float w = li > -INFINITY ? __expf((li - M) / T) : 0.f;
        const float inc = wave_incl_scan<float>(w);
        const unsigned long long hit = __ballot(w > 0.f && run + (double)inc > target);
        const unsigned long long pos = __ballot(w > 0.f);
        if (pos) last_pos = c0 + 63 - __builtin_clzll(pos);
        if (hit) { found = c0 + __builtin_ctzll(hit); break; }
        run += (double)lane_f(inc, 63);
      }
      const int pick = found >= 0 ? found : (last_pos >= 0 ? last_pos : am);
      // its target id from the prefetched map when it lies in the prefetched part
      int dmap = -2;
#pragma unroll
      for (int q = 0; q < kScanPre; ++q) {
        const int l = pick - r0 - q * OSP_WAVE;
        if (l >= 0 && l < OSP_WAVE) dmap = lane_i(pmap[q], l);
      }
      if (lane == 0) { s_row = pick; s_map = dmap; }
    }
    __syncthreads();
    row = s_row;
  }
  row = min(max(row, 0), a.V - 1);
  const int d = (T > 0.f && M > -INFINITY && s_map != -2 && s_row == row) ? s_map : a.d2t[row];
  if (tid == 0) {
    a.drafts[(long)b * a.ld_drafts + k] = d;
    if (a.drafts_out) a.drafts_out[(long)b * a.K + k] = d;
    if (!a.block) {
      a.ar_tok[b] = d;
      a.ar_pos[b] = a.committed[b] + k;
    }
    // the row's statistics, for the verification of this draft
    if (a.qstat) a.qstat[(long)b * a.ld_qstat + k] = QStat{S, M, am == 0x7fffffff ? -1 : am};
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

// The draft pick of one LM-head row, by one block (Section 3.4: the drafter proposes
// its tokens autoregressively; the pick itself is plain temperature sampling).
//
// The LM-head kernel left one record per range of blk_rows consecutive logits:
// (max, sum exp((l - max)/T), lowest argmax).  They are merged in range order: at
// T = 0 the pick is the lowest-index argmax; at T > 0 the inverse CDF of softmax(l / T)
// over drafter rows in ascending order picks the smallest row whose running sum exceeds
// u * S -- the range holding that point is found from the range sums (float64 prefix),
// then that range's logits are scanned.  The row is mapped to a target id through d2t.
//
// Used by the sampling kernel and, where the next draft step consumes the draft, by that
// step's first kernel (a single sequence's layer-0 QKV GEMV, a batch's row preparation),
// which then needs no sampling launch before it.
#pragma once

#include "common.h"
#include "internal.h"

namespace osp {

struct Pick {
  int row;    // drafter row drawn
  int tok;    // its target id (d2t)
  double S;   // sum over the row of exp((l - M)/T) (T > 0; else 0)
  float M;    // row max
  int am;     // lowest argmax (-1: no mapped entry)
};

// The records a thread merges: records [t PER, t PER + PER) of the row, raw.
template <int PER> struct PickRecs {
  float4 r[PER];
};

// Requests this thread's records (1 <= nblk <= NT * PER), all at once, from clamped
// addresses with no condition: a load under a condition makes the wavefront wait for
// every load issued before it, so the records would arrive one at a time.  Nothing
// reads them until pick_draft, so a caller can request its own data in between.
// (Strided records -- each wavefront load reading 64 adjacent records, the prefix then
// taken per round of NT records -- measured slower: the sampling kernel 6.5 -> 7.4 us.)
template <int NT, int PER>
OSP_DEV void pick_request(PickRecs<PER>& rec, const float* part, int nblk) {
  const int i0 = threadIdx.x * PER;
#pragma unroll
  for (int q = 0; q < PER; ++q) rec.r[q] = *reinterpret_cast<const float4*>(part + min(i0 + q, nblk - 1) * 4);
}

// Every thread of the NT-thread block calls this (it holds block barriers) and gets
// the same result.  rec: what pick_request loaded, the row's nblk records; lg: the
// row's logits.  T and u are the row's temperature and uniform.
template <int NT, int PER>
OSP_DEV Pick pick_draft(const PickRecs<PER>& rec, int nblk, int blk_rows, const float* lg, int V,
                        const int32_t* d2t, float T, float u) {
  constexpr int NW = NT / OSP_WAVE;
  __shared__ float s_wm[NW];
  __shared__ int s_wi[NW];
  __shared__ double s_scan[NW];
  __shared__ double s_before;
  __shared__ int s_blk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = tid * PER;
  float bm[PER], bs[PER];
  int ba[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const bool live = i0 + q < nblk;
    bm[q] = live ? rec.r[q].x : -INFINITY;
    bs[q] = live ? rec.r[q].y : 0.f;
    ba[q] = live ? __float_as_int(rec.r[q].z) : -1;
  }
  // ---- global max and lowest argmax ------------------------------------------------
  // (selects, not branches: a record field read under a branch would be loaded there)
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < PER; ++q) m = fmaxf(m, bm[q]);
  int am = 0x7fffffff;   // ascending ranges: the lowest argmax among the maximal records
#pragma unroll
  for (int q = 0; q < PER; ++q) am = bm[q] == m ? min(am, ba[q]) : am;
  {
    const float wm = wave_max(m);
    const int wi = wave_min_i((m == wm && m > -INFINITY) ? am : 0x7fffffff);
    if (lane == 0) { s_wm[wave] = wm; s_wi[wave] = wi; }
    __syncthreads();
    float gm = -INFINITY;
    int gi = 0x7fffffff;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (s_wm[w] > gm) { gm = s_wm[w]; gi = s_wi[w]; }
      else if (s_wm[w] == gm && s_wi[w] < gi) gi = s_wi[w];
    }
    m = gm;
    am = gi;
  }
  Pick p;
  p.M = m;
  p.am = am == 0x7fffffff ? -1 : am;
  p.S = 0.0;
  int row, dmap = -2;
  if (T <= 0.f || m == -INFINITY) {
    row = am;
  } else {
    const float M = m;
    // range sums rescaled to the global max, prefix in float64 (the breakpoints of a
    // 10^5-entry CDF are ~1e-5 of the total apart)
    double bsum[PER];
    double loc = 0.0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      bsum[q] = bm[q] > -INFINITY ? (double)bs[q] * (double)__expf((bm[q] - M) / T) : 0.0;
      loc += bsum[q];
    }
    double incl, tot;
    const double excl = block_scan<NT, double>(loc, s_scan, incl, tot);
    p.S = tot;
    const double target = (double)u * tot;
    if (tid == 0) s_blk = -1;
    __syncthreads();
    if (excl <= target && incl > target) {
      double run = excl;
      int hit = -1;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        if (hit < 0 && i0 + q < nblk) {
          if (run + bsum[q] > target) { hit = q; } else { run += bsum[q]; }
        }
      }
      if (hit < 0) {   // rounding: the last non-empty record of this thread
        run = excl;
        for (int q = 0; q < PER; ++q)
          if (i0 + q < nblk && bsum[q] > 0.0) { hit = q; }
        for (int q = 0; q < hit; ++q) run += bsum[q];
      }
      if (hit >= 0) { s_blk = i0 + hit; s_before = run; }
    }
    __syncthreads();
    if (s_blk < 0) {   // (uniform) rounding pushed the target past the last record with weight
      int li = -1;
      double lb = 0.0, run = excl;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        if (i0 + q < nblk && bsum[q] > 0.0) { li = i0 + q; lb = run; }
        run += bsum[q];
      }
      const int wl = wave_max_i(li);
      if (lane == 0) s_wi[wave] = wl;
      __syncthreads();
      int last = -1;
#pragma unroll
      for (int w = 0; w < NW; ++w) last = max(last, s_wi[w]);
      if (li >= 0 && li == last) { s_blk = li; s_before = lb; }
      if (last < 0 && tid == 0) { s_blk = 0; s_before = 0.0; }   // (no weight at all: not reached)
      __syncthreads();
    }
    // ---- every wavefront scans the chosen range's logits (no barrier after); the
    //      first kScanPre x 64 are requested at once (a head range holds 16 T <= 80) ----
    constexpr int kScanPre = 2;
    const int r0 = s_blk * blk_rows;
    const int r1 = min(r0 + blk_rows, V);
    float pre[kScanPre];
    int pmap[kScanPre];   // the range's vocabulary map, requested with its logits
#pragma unroll
    for (int q = 0; q < kScanPre; ++q) {
      const int i = r0 + q * OSP_WAVE + lane;
      const float v = lg[min(i, r1 - 1)];
      pmap[q] = d2t[min(i, V - 1)];
      pre[q] = i < r1 ? v : -INFINITY;
    }
    double run = s_before;
    int last_pos = -1, found = -1;
    for (int c0 = r0, q = 0; c0 < r1; c0 += OSP_WAVE, ++q) {
      const int i = c0 + lane;
      float li = -INFINITY;
#pragma unroll
      for (int pq = 0; pq < kScanPre; ++pq)
        if (pq == q) li = pre[pq];
      if (q >= kScanPre) li = i < r1 ? lg[i] : -INFINITY;
      const float w = li > -INFINITY ? __expf((li - M) / T) : 0.f;
      const float inc = wave_incl_scan<float>(w);
      const unsigned long long hit = __ballot(w > 0.f && run + (double)inc > target);
      const unsigned long long pos = __ballot(w > 0.f);
      if (pos) last_pos = c0 + 63 - __builtin_clzll(pos);
      if (hit) { found = c0 + __builtin_ctzll(hit); break; }
      run += (double)lane_f(inc, 63);
    }
    row = found >= 0 ? found : (last_pos >= 0 ? last_pos : am);
    // its target id from the prefetched map when it lies in the prefetched part
#pragma unroll
    for (int q = 0; q < kScanPre; ++q) {
      const int l = row - r0 - q * OSP_WAVE;
      if (l >= 0 && l < OSP_WAVE) dmap = lane_i(pmap[q], l);
    }
  }
  const int rc = min(max(row, 0), V - 1);
  p.row = rc;
  p.tok = (dmap != -2 && rc == row) ? dmap : d2t[rc];
  return p;
}

}  // namespace osp

// Growing a draft tree (top-k > 1; the paper serves chains, top-k 1, Section 4):
// every node of the frontier runs through the drafter, its k most likely rows become
// candidates scored by the cumulative log-probability of their path (temperature 1),
// the k best candidates of a depth form the next frontier, and the n best candidates
// of all depths form the tree.
//
//   k_tree_topk  (rows x 64)  the k best (logit, row) pairs of each 1/64 of an LM-head
//                             row (larger logit first, lower row on ties)
//   k_tree_step  (B)          per sequence: the rows' k best pairs and log-normalisers
//                             (LM-head records at temperature 1), the new candidates,
//                             the next frontier and the next pass's rows: token, position,
//                             node slot, ancestors' slots and conditioning row (the
//                             parent's hidden state)
//   k_tree_final (B)          the n best candidates in generation order, parents
//                             re-indexed
// A frontier row's attention over its ancestors' and its own keys/values (the tree
// cache) is one more split of the context attention, added by the split combine.
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kTkThreads = 256;
constexpr int kTkPer = 16;        // logits per thread and block: a row of up to 64 x 4096
constexpr int kTkRecLane = kTkMaxRecords / OSP_WAVE;   // LM-head records per lane

OSP_DEV bool tk_better(float v1, int r1, float v2, int r2) { return v1 > v2 || (v1 == v2 && r1 < r2); }

// Wavefront-wide best (value, row) pair.
OSP_DEV void wave_best(float& v, int& r) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = xor_lane_c(v, m);
    const int orow = xor_lane_ci(r, m);
    if (tk_better(ov, orow, v, r)) { v = ov; r = orow; }
  }
}

__global__ void __launch_bounds__(kTkThreads) k_tree_topk(TreeArgs a) {
  __shared__ float s_v[kTkThreads / OSP_WAVE][kMaxTopk];
  __shared__ int s_r[kTkThreads / OSP_WAVE][kMaxTopk];
  const int row = blockIdx.x, blk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.k;
  const int chunk = (a.V + kTkBlocks - 1) / kTkBlocks;
  const int i0 = blk * chunk, i1 = min(a.V, i0 + chunk);
  const float* lg = a.logits + (long)row * a.ld_logits;
  float v[kTkPer];
  int idx[kTkPer];
#pragma unroll
  for (int q = 0; q < kTkPer; ++q) {
    const int i = i0 + tid + q * kTkThreads;
    const float l = lg[min(i, a.V - 1)];          // clamped address, masked below
    v[q] = i < i1 ? l : -INFINITY;
    idx[q] = i < i1 ? i : 0x7fffffff;
  }
  // the wavefront's K best: K rounds of a wavefront arg-best, the winner removed
  for (int t = 0; t < K; ++t) {
    float bv = -INFINITY;
    int br = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < kTkPer; ++q)
      if (tk_better(v[q], idx[q], bv, br)) { bv = v[q]; br = idx[q]; }
    float wv = bv;
    int wr = br;
    wave_best(wv, wr);
#pragma unroll
    for (int q = 0; q < kTkPer; ++q)
      if (idx[q] == wr && wr != 0x7fffffff) { v[q] = -INFINITY; idx[q] = 0x7fffffff; }
    if (lane == 0) { s_v[wave][t] = wv; s_r[wave][t] = wr; }
  }
  __syncthreads();
  if (wave == 0) {
    const int nc = (kTkThreads / OSP_WAVE) * K;
    float cv = lane < nc ? s_v[lane / K][lane % K] : -INFINITY;
    int cr = lane < nc ? s_r[lane / K][lane % K] : 0x7fffffff;
    const long o = ((long)row * kTkBlocks + blk) * kMaxTopk;
    for (int t = 0; t < K; ++t) {
      float wv = cv;
      int wr = cr;
      wave_best(wv, wr);
      if (cr == wr && wr != 0x7fffffff) { cv = -INFINITY; cr = 0x7fffffff; }
      if (lane == 0) { a.cand_v[o + t] = wv; a.cand_r[o + t] = wr; }
    }
  }
}

// Candidate c is better than candidate e: larger score, lower index on ties.
OSP_DEV bool cand_better(double s1, int i1, double s2, int i2) { return s1 > s2 || (s1 == s2 && i1 < i2); }

constexpr int kTkRanges = 16;     // record ranges a record-guided selection reads (else the row)

// This lane's kMaxTopk best (value, index) pairs, best first: insert one.
OSP_DEV void top_insert(float (&bv)[kMaxTopk], int (&br)[kMaxTopk], float v, int r) {
  if (!tk_better(v, r, bv[kMaxTopk - 1], br[kMaxTopk - 1])) return;
#pragma unroll
  for (int i = 0; i < kMaxTopk; ++i) {
    if (tk_better(v, r, bv[i], br[i])) {
      const float tv = bv[i];
      const int tr = br[i];
      bv[i] = v;
      br[i] = r;
      v = tv;
      r = tr;
    }
  }
}

// The wavefront's best pair over the lanes' lists (wv, wr); the lane holding it drops it.
OSP_DEV void wave_pop_best(float (&bv)[kMaxTopk], int (&br)[kMaxTopk], float& wv, int& wr) {
  wv = bv[0];
  wr = br[0];
  wave_best(wv, wr);
  if (br[0] == wr && bv[0] == wv && wr != 0x7fffffff) {
#pragma unroll
    for (int i = 0; i + 1 < kMaxTopk; ++i) { bv[i] = bv[i + 1]; br[i] = br[i + 1]; }
    bv[kMaxTopk - 1] = -INFINITY;
    br[kMaxTopk - 1] = 0x7fffffff;
  }
}

// K rounds of the wavefront's best (value, index) pair over the lanes' N pairs, each
// winner dropped by its lane; lane 0 writes the winners to ov / orr when given.  Returns
// the K-th winner's value.
template <int N>
OSP_DEV float wave_topk(const float (&v)[N], const int (&ix)[N], int K, float* ov, int* orr) {
  unsigned long long gone = 0ull;
  float last = -INFINITY;
  for (int t = 0; t < K; ++t) {
    float bv = -INFINITY;
    int br = 0x7fffffff, bq = -1;
#pragma unroll
    for (int q = 0; q < N; ++q)
      if (!((gone >> q) & 1ull) && tk_better(v[q], ix[q], bv, br)) { bv = v[q]; br = ix[q]; bq = q; }
    float wv = bv;
    int wr = br;
    wave_best(wv, wr);
    if (bq >= 0 && br == wr && wr != 0x7fffffff) gone |= 1ull << bq;
    if (ov && (threadIdx.x & 63) == 0) { ov[t] = wv; orr[t] = wr; }
    last = wv;
  }
  return last;
}

__global__ void __launch_bounds__(kTkThreads) k_tree_step(TreeArgs a) {
  __shared__ float s_cv[kMaxTopk][kMaxTopk];
  __shared__ int s_cr[kMaxTopk][kMaxTopk];
  __shared__ double s_lse[kMaxTopk];
  __shared__ double s_sc[kMaxTopk * kMaxTopk];
  __shared__ int s_sel[kMaxTopk];
  __shared__ int s_src[kMaxTopk];
  __shared__ int s_prev[kMaxTopk];
  __shared__ int s_ntok[kMaxTopk * kMaxTopk], s_ndep[kMaxTopk * kMaxTopk];
  __shared__ int s_rank[kMaxTopk * kMaxTopk];
  __shared__ int s_rng[kMaxTopk][kTkRanges];
  __shared__ int s_n0;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.k, p = a.pass;
  const int nfr = p == 0 ? 1 : K;                 // rows of this pass that are sequence b's
  const int row0 = p == 0 ? b : b * K;
  const long cb = (long)b * kMaxCand;
  // this pass's rows' ancestor lists (read before the next pass's replace them)
  __shared__ int s_anc[kMaxTopk][kMaxTreeDepth];
  if (p > 0 && tid < K * kMaxTreeDepth)
    s_anc[tid / kMaxTreeDepth][tid % kMaxTreeDepth] = a.r_anc[(long)b * K * kMaxTreeDepth + tid];
  if (tid < K) s_prev[tid] = p == 0 ? -1 : a.front[b * kMaxTopk + tid];
  if (tid == 0) s_n0 = p == 0 ? 0 : a.n_cand[b];   // (read before anyone writes it below)
  if (tid < K) { s_sel[tid] = tid; s_src[tid] = p == 0 ? 0 : tid; }   // (overwritten below)
  // ---- each row's K best (logit, row) pairs and its log-normaliser M + log S --------------
  for (int j = wave; j < nfr; j += kTkThreads / OSP_WAVE) {
    const int r = row0 + j;
    // LM-head records of the row (temperature 1): max and rescaled sums, every record
    // of the lane requested at once (clamped addresses; lane l: records l, l + 64, ...)
    const float* rec = a.rec + (long)r * a.nblk * 4;
    float2 rs[kTkRecLane];
#pragma unroll
    for (int q = 0; q < kTkRecLane; ++q)
      rs[q] = *reinterpret_cast<const float2*>(rec + (long)min(lane + q * OSP_WAVE, a.nblk - 1) * 4);
    float m = -INFINITY;
#pragma unroll
    for (int q = 0; q < kTkRecLane; ++q)
      if (lane + q * OSP_WAVE < a.nblk) m = fmaxf(m, rs[q].x);
    const float M = wave_max(m);
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < kTkRecLane; ++q)
      if (lane + q * OSP_WAVE < a.nblk && rs[q].x > -INFINITY) s += (double)rs[q].y * (double)__expf(rs[q].x - M);
    const double S = wave_sum_d(s);
    if (!a.cand_v) {
      // record-guided (passes of many rows): the K best logits lie in ranges whose max
      // reaches Mk, the K-th largest range max (the K ranges of largest max hold K values
      // >= Mk, so the K-th best value is >= Mk); only those ranges are read
      float mv[kTkRecLane];
      int mi[kTkRecLane];
#pragma unroll
      for (int q = 0; q < kTkRecLane; ++q) {
        const bool in = lane + q * OSP_WAVE < a.nblk;
        mv[q] = in ? rs[q].x : -INFINITY;
        mi[q] = in ? lane + q * OSP_WAVE : 0x7fffffff;
      }
      const float Mk = wave_topk(mv, mi, K, nullptr, nullptr);
      int n = 0;
#pragma unroll
      for (int q = 0; q < kTkRecLane; ++q) {
        const int c = lane + q * OSP_WAVE;
        const bool in = c < a.nblk && rs[q].x >= Mk;
        const unsigned long long bal = __ballot(in);
        const int at = n + __popcll(bal & ((1ull << lane) - 1ull));
        if (in && at < kTkRanges) s_rng[j][at] = c;
        n += __popcll(bal);
      }
      __builtin_amdgcn_wave_barrier();
      const float* lg = a.logits + (long)r * a.ld_logits;
      if (n <= kTkRanges) {
        // every listed range's logits requested at once: lane l reads entries l and l + 64
        float lv[2 * kTkRanges];
        int li[2 * kTkRanges];
#pragma unroll
        for (int i = 0; i < kTkRanges; ++i) {
          const int e0 = (i < n ? s_rng[j][i] : 0) * a.blk_rows + lane, e1 = e0 + OSP_WAVE;
          const float l0 = lg[min(e0, a.V - 1)], l1 = lg[min(e1, a.V - 1)];   // clamped, masked below
          const bool in0 = i < n && lane < a.blk_rows && e0 < a.V;
          const bool in1 = i < n && lane + OSP_WAVE < a.blk_rows && e1 < a.V;
          lv[2 * i] = in0 ? l0 : -INFINITY;
          li[2 * i] = in0 ? e0 : 0x7fffffff;
          lv[2 * i + 1] = in1 ? l1 : -INFINITY;
          li[2 * i + 1] = in1 ? e1 : 0x7fffffff;
        }
        wave_topk(lv, li, K, s_cv[j], s_cr[j]);
      } else {
        // ties or masked rows put more ranges at Mk: the whole row
        float bv[kMaxTopk];
        int br[kMaxTopk];
#pragma unroll
        for (int i = 0; i < kMaxTopk; ++i) { bv[i] = -INFINITY; br[i] = 0x7fffffff; }
        for (int i = lane; i < a.V; i += OSP_WAVE) top_insert(bv, br, lg[i], i);
        for (int t = 0; t < K; ++t) {
          float wv;
          int wr;
          wave_pop_best(bv, br, wv, wr);
          if (lane == 0) { s_cv[j][t] = wv; s_cr[j][t] = wr; }
        }
      }
    } else {
      // the blocks' candidates: kTkBlocks x K pairs, lane l holds pairs l, l + 64, ...
      constexpr int NPL = kTkBlocks * kMaxTopk / OSP_WAVE;
      float cv[NPL];
      int cr[NPL];
#pragma unroll
      for (int q = 0; q < NPL; ++q) {
        const int e = lane + q * OSP_WAVE;            // pair e = block e / kMaxTopk, rank e % kMaxTopk
        const bool in = e % kMaxTopk < K;
        const long o = ((long)r * kTkBlocks) * kMaxTopk + e;
        cv[q] = in ? a.cand_v[o] : -INFINITY;
        cr[q] = in ? a.cand_r[o] : 0x7fffffff;
      }
      for (int t = 0; t < K; ++t) {
        float bv = -INFINITY;
        int br = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < NPL; ++q)
          if (tk_better(cv[q], cr[q], bv, br)) { bv = cv[q]; br = cr[q]; }
        float wv = bv;
        int wr = br;
        wave_best(wv, wr);
#pragma unroll
        for (int q = 0; q < NPL; ++q)
          if (cr[q] == wr && wr != 0x7fffffff) { cv[q] = -INFINITY; cr[q] = 0x7fffffff; }
        if (lane == 0) { s_cv[j][t] = wv; s_cr[j][t] = wr; }
      }
    }
    if (lane == 0) s_lse[j] = (double)M + log(S);
  }
  __syncthreads();
  // ---- the new candidates (row j, rank t) in generation order -----------------------------
  const int n0 = s_n0;
  const int nnew = nfr * K;
  if (tid < nnew) {
    const int j = tid / K, t = tid % K;
    const int par = s_prev[j];
    const int c = n0 + tid;
    const int rr = s_cr[j][t];
    const bool ok = rr >= 0 && rr < a.V;
    const double sc = (par >= 0 ? a.c_score[cb + par] : 0.0) + ((double)s_cv[j][t] - s_lse[j]);
    const int tok = ok ? a.d2t[rr] : -1;
    const int dep = (par >= 0 ? a.c_depth[cb + par] : 0) + 1;
    a.c_tok[cb + c] = tok;
    a.c_par[cb + c] = par;
    a.c_score[cb + c] = sc;
    a.c_depth[cb + c] = dep;
    s_sc[tid] = sc;
    s_ntok[tid] = tok;                              // (read back below from LDS: another
    s_ndep[tid] = dep;                              // wavefront's global writes may not be)
  }
  if (tid == 0) a.n_cand[b] = n0 + nnew;
  __syncthreads();
  if (p + 1 >= a.depth) {                         // the last pass: no next frontier
    if (tid < nnew) a.c_slot[cb + n0 + tid] = -1;
    return;
  }
  // ---- the next frontier: the K best new candidates, then in generation order -------------
  if (tid < nnew) {
    int rank = 0;
    for (int e = 0; e < nnew; ++e) rank += cand_better(s_sc[e], e, s_sc[tid], tid) ? 1 : 0;
    s_rank[tid] = rank;
  }
  __syncthreads();
  if (tid < nnew) {
    int pos = K;
    if (s_rank[tid] < K) {
      pos = 0;            // place among the selected, by generation order
      for (int e = 0; e < tid; ++e) pos += s_rank[e] < K ? 1 : 0;
    }
    if (pos < K) {        // (scores that are not numbers could put more than K below rank K)
      s_sel[pos] = tid;                             // (new candidate n0 + tid)
      s_src[pos] = tid / K;                         // the frontier row of its parent
      // (each new candidate's slot is written once, by its own thread)
      a.c_slot[cb + n0 + tid] = b * kMaxTreeProc + p * K + pos;
    } else {
      a.c_slot[cb + n0 + tid] = -1;
    }
  }
  __syncthreads();
  // ---- the next pass's rows ---------------------------------------------------------------
  if (tid < K) {
    const int j = tid;
    const int e0 = s_sel[j];                        // index among the new candidates
    const int c = n0 + e0;
    const int slot = b * kMaxTreeProc + p * K + j;  // run through the drafter in pass p + 1
    a.front[b * kMaxTopk + j] = c;
    const int r = b * K + j;
    const int L = a.committed[b];
    a.r_tok[r] = max(s_ntok[e0], 0);
    a.r_pos[r] = L + s_ndep[e0] - 1;
    a.r_attpos[r] = L - 1;
    a.r_node[r] = slot;
    if (j == 0) {                                   // the next pass's rows of sequence b
      a.r_cu[b] = b * K;
      if (b == a.B - 1) a.r_cu[a.B] = a.B * K;
    }
    // ancestors' slots, the root's child first, then the node itself: the parent's list
    // (a row of this pass; root children: none) followed by the node's slot
    const int pr = s_src[j];
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < kMaxTreeDepth; ++i)
      if (p > 0 && cnt == i && s_anc[pr][i] >= 0) cnt = i + 1;
#pragma unroll
    for (int i = 0; i < kMaxTreeDepth; ++i)
      a.r_anc[r * kMaxTreeDepth + i] = i < cnt ? s_anc[pr][i] : (i == cnt ? slot : -1);
  }
  // ---- conditioning rows: the parent's hidden state (root: the last ingest row); the
  //      buffers do not overlap, so the loads of several iterations go out together -------
  const int d4 = a.d / 4, nv = K * d4;
  const float4* __restrict__ x4 = reinterpret_cast<const float4*>(a.x);
  float4* __restrict__ s4 = reinterpret_cast<float4*>(a.r_s) + (long)b * K * d4;
#pragma unroll 4
  for (int i = tid; i < nv; i += kTkThreads) {
    const int j = i / d4;
    const int src = p == 0 ? a.last_row[b] : b * K + s_src[j];
    s4[i] = x4[(long)src * d4 + (i - j * d4)];
  }
}

__global__ void __launch_bounds__(kTkThreads) k_tree_final(TreeArgs a) {
  __shared__ double s_sc[kMaxCand];
  __shared__ int s_keep[kMaxCand];
  __shared__ int s_pos[kMaxCand];
  const int b = blockIdx.x, tid = threadIdx.x;
  const long cb = (long)b * kMaxCand;
  const int n = min(a.n_cand[b], kMaxCand);
  const int N = min(a.n_nodes, n);
  for (int c = tid; c < n; c += kTkThreads) s_sc[c] = a.c_score[cb + c];
  __syncthreads();
  for (int c = tid; c < n; c += kTkThreads) {
    int rank = 0;
    for (int e = 0; e < n; ++e) rank += cand_better(s_sc[e], e, s_sc[c], c) ? 1 : 0;
    s_keep[c] = rank < N ? 1 : 0;
  }
  __syncthreads();
  for (int c = tid; c < n; c += kTkThreads) {
    int pos = 0;
    for (int e = 0; e < c; ++e) pos += s_keep[e];
    s_pos[c] = pos;
  }
  __syncthreads();
  for (int c = tid; c < n; c += kTkThreads) {
    if (!s_keep[c] || s_pos[c] >= a.n_nodes) continue;
    const int i = s_pos[c];
    const int par = a.c_par[cb + c];
    a.out_tok[(long)b * a.n_nodes + i] = a.c_tok[cb + c];
    // (the parent scores at least as high and comes earlier: it is kept too)
    a.out_par[(long)b * a.n_nodes + i] = par >= 0 ? (s_keep[par] ? s_pos[par] : -2) : -1;
    if (a.out_score) a.out_score[(long)b * a.n_nodes + i] = s_sc[c];
  }
  for (int i = N + tid; i < a.n_nodes; i += kTkThreads) {
    a.out_tok[(long)b * a.n_nodes + i] = -1;
    a.out_par[(long)b * a.n_nodes + i] = -2;
    if (a.out_score) a.out_score[(long)b * a.n_nodes + i] = -INFINITY;
  }
}

void launch_tree_topk(const TreeArgs& a, int rows, hipStream_t st) {
  hipLaunchKernelGGL(k_tree_topk, dim3(rows, kTkBlocks), dim3(kTkThreads), 0, st, a);
}

void launch_tree_step(const TreeArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_tree_step, dim3(a.B), dim3(kTkThreads), 0, st, a);
}

void launch_tree_final(const TreeArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_tree_final, dim3(a.B), dim3(kTkThreads), 0, st, a);
}

}  // namespace osp

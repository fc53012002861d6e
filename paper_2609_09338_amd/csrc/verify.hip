// Lossless verification of the drafted chain (the standard speculative
// decoding acceptance rule, unchanged by the paper).
//
// Row convention per sequence: drafts d_0..d_{K-1} with drafter logit rows
// q_0..q_{K-1} (over drafter rows, mapped to target ids by d2t / t2d); target
// logit rows p_0..p_K over target ids.  p is the softmax of the target row at the
// request's temperature T, q that of the drafter row at the temperature the drafts
// were drawn at (T_d; T_d = 0: one-hot at the drafter row's lowest argmax, which
// reduces acceptance to u_k < p_k(d_k) and the residual to p_a without d_a).
//
//   k_vstats  (B x jobs)   per chunk of every target and drafter row: max,
//                          lowest argmax and sum exp((l - max)/T) (stateful
//                          verify: target rows only; the drafter rows' were kept
//                          by the draft step's sampling kernel)
//   k_vaccept (B)          merges chunks in order; accepts d_k while
//                          u_k < min(1, p_k(d_k)/q_k(d_k)) (T = 0: d_k equals
//                          the target argmax); writes a, the mask and d_0..d_{a-1};
//                          at T = 0 also the token at index a (the argmax of p_a)
//   k_vresid  (B x chunks) per chunk of target row a (T > 0): sums of the residual
//                          max(0, p_a - q_a) (q = 0 when a = K) and of p_a, per
//                          64-id sub-range and per chunk
//   k_vfinal  (B, one wavefront) inverse CDF over the residual (or p_a if it is
//                          empty) in ascending target ids: chunk, sub-range, id
//                          -> the token at index a
//
// Either way the stateful verify records the a + 1 committed tokens as the slot's
// pending ingest.  Draft trees (deterministic top-k children, accepted in turn with
// the target's probability renormalised over the children not yet rejected; the bonus
// from the target without the rejected tokens) replace k_vaccept by k_tree_walk (B),
// which walks the tree from the root; the last node's row and rejected tokens go to
// k_vresid / k_vfinal.
//
// (Finishing a sequence in the last block of the statistics or residual kernel to
// arrive, instead of in the small kernels, needs an agent-scope release before the
// arrival count -- an L2 write-back per block -- and measured slower: 48.6 against
// 45.4 us at batch 1, 1031 against 118 us at batch 64.)
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kVThreads = 256;

constexpr int kVPer = 16;   // elements per thread of a 4096-element chunk

// Block-wide (max, lowest index) and float64 sum; results broadcast to every thread.
OSP_DEV void block_stats(float& m, int& am, double& s, float* sm, int* si, double* sd) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float wm = wave_max(m);
  const int wi = wave_min_i((m == wm && m > -INFINITY) ? am : 0x7fffffff);
  const double ws = wave_sum_d(s);
  if (lane == 0) { sm[wave] = wm; si[wave] = wi; sd[wave] = ws; }
  __syncthreads();
  float gm = -INFINITY;
  int gi = 0x7fffffff;
  double gs = 0.0;
  for (int w = 0; w < kVThreads / 64; ++w) {
    if (sm[w] > gm) { gm = sm[w]; gi = si[w]; }
    else if (sm[w] == gm && si[w] < gi) gi = si[w];
    gs += sd[w];
  }
  __syncthreads();
  m = gm;
  am = gi;
  s = gs;
}

// One wavefront per chunk (job): lane l reads ids l, l + 64, ... of the chunk (every
// load is 256 contiguous bytes), keeps them in registers for the max and the float64
// sum, and the chunk needs no block barrier.  Four jobs per block.
constexpr int kVWaveElems = 4096 / 64;   // elements per lane (chunk / 64)

// STREAM: the rows are read with non-temporal loads (a verification whose rows outsize
// the last-level cache: read once, faster, and the drafter's weights stay cached).
typedef float vf_f32x4 __attribute__((ext_vector_type(4)));
template <bool STREAM>
OSP_DEV float4 ld4(const float* p) {
  if constexpr (STREAM) {
    const vf_f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const vf_f32x4*>(p));
    return make_float4(x[0], x[1], x[2], x[3]);
  } else {
    return *reinterpret_cast<const float4*>(p);
  }
}
template <bool STREAM>
OSP_DEV float ld1(const float* p) {
  if constexpr (STREAM) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool STREAM>
OSP_DEV void chunk_stats(const VerifyArgs& a, int b, int j, int nt, int nj) {
  const int lane = threadIdx.x & 63;
  const float* row;
  int V, c;
  if (j < nt) {
    const int k = j / a.nchunk_t;
    c = j - k * a.nchunk_t;
    row = a.target + ((long)b * (a.K + 1) + k) * a.V_T;
    V = a.V_T;
  } else {
    const int jj = j - nt;
    const int k = jj / a.nchunk_d;
    c = jj - k * a.nchunk_d;
    row = a.draft + ((long)b * a.ld_draft_b + k) * a.V_d;
    V = a.V_d;
  }
  const int i0 = c * a.chunk, i1 = min(V, i0 + a.chunk);
  float v[kVWaveElems];
  float m = -INFINITY;
  int am = 0x7fffffff;
  // 16-byte loads (lane l: ids 4 l .. 4 l + 3 of every 256) when the row allows them: a
  // vocabulary that is a multiple of 4 never splits a load at a chunk or row end
  const bool vec = (V & 3) == 0 && (reinterpret_cast<uintptr_t>(row) & 15) == 0;
  if (vec) {
#pragma unroll
    for (int q = 0; q < kVWaveElems / 4; ++q) {
      const int i = i0 + q * 256 + 4 * lane;
      const float4 t = ld4<STREAM>(row + min(i, V - 4));   // clamped, masked below
      const bool in = i < i1;
      v[4 * q + 0] = in ? t.x : -INFINITY;
      v[4 * q + 1] = in ? t.y : -INFINITY;
      v[4 * q + 2] = in ? t.z : -INFINITY;
      v[4 * q + 3] = in ? t.w : -INFINITY;
    }
#pragma unroll
    for (int q = 0; q < kVWaveElems; ++q)   // ascending ids: first hit is lowest
      if (v[q] > m) { m = v[q]; am = i0 + (q >> 2) * 256 + 4 * lane + (q & 3); }
  } else {
#pragma unroll
    for (int q = 0; q < kVWaveElems; ++q) {
      const int i = i0 + lane + q * 64;
      v[q] = i < i1 ? ld1<STREAM>(row + i) : -INFINITY;
    }
#pragma unroll
    for (int q = 0; q < kVWaveElems; ++q)
      if (v[q] > m) { m = v[q]; am = i0 + lane + q * 64; }   // ascending ids: first hit is lowest
  }
  const float M = wave_max(m);
  const int A = wave_min_i((m == M && m > -INFINITY) ? am : 0x7fffffff);
  const float T = j < nt ? a.temp[b] : a.temp_d[b];
  // (a reciprocal, not 64 divisions: 136 instead of 158 registers, one more wavefront
  // per SIMD; verify at c5 111 -> 104 us)
  const float iT = 1.0f / T;
  double se = 0.0;   // float64 sums: exactness of the 10^5-entry CDFs that follow
  if (T > 0.f && M > -INFINITY) {
#pragma unroll
    for (int q = 0; q < kVWaveElems; ++q)
      if (v[q] > -INFINITY) se += (double)__expf((v[q] - M) * iT);
  }
  se = wave_sum_d(se);
  if (lane == 0) {
    float* p = a.part + ((long)b * nj + j) * 4;
    p[0] = M;
    p[1] = (float)se;
    p[2] = __int_as_float(M > -INFINITY ? A : -1);
    p[3] = 0.f;
  }
}

// Merge the chunk statistics of one row with one wavefront: max M, lowest
// argmax, S = sum exp((l - M)/T).  Fixed summation order.
constexpr int kMergeLane = 2;   // chunk records per lane held in registers by merge_row

OSP_DEV void merge_row(const float* p, int n, float T, float& M, double& S, int& am) {
  const int lane = threadIdx.x & 63;
  // the lane's first kMergeLane records requested at once and kept for both passes
  // (clamped addresses; vocabularies up to kMergeLane x 64 chunks), any further ones
  // read in a loop
  float4 rq[kMergeLane];
#pragma unroll
  for (int q = 0; q < kMergeLane; ++q)
    rq[q] = *reinterpret_cast<const float4*>(p + (long)min(lane + q * 64, n - 1) * 4);
  float m = -INFINITY;
  int ai = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < kMergeLane; ++q) {
    const float mc = rq[q].x;
    const int ac = __float_as_int(rq[q].z);
    if (lane + q * 64 < n && (mc > m || (mc == m && mc > -INFINITY && ac < ai))) { m = mc; ai = ac; }
  }
  for (int c = lane + kMergeLane * 64; c < n; c += 64) {
    const float mc = p[c * 4];
    const int ac = __float_as_int(p[c * 4 + 2]);
    if (mc > m || (mc == m && mc > -INFINITY && ac < ai)) { m = mc; ai = ac; }
  }
  M = wave_max(m);
  am = wave_min_i((m == M && m > -INFINITY) ? ai : 0x7fffffff);
  if (am == 0x7fffffff) am = -1;
  double s = 0.0;
  if (T > 0.f && M > -INFINITY) {
#pragma unroll
    for (int q = 0; q < kMergeLane; ++q)
      if (lane + q * 64 < n && rq[q].x > -INFINITY) s += (double)rq[q].y * (double)__expf((rq[q].x - M) / T);
    for (int c = lane + kMergeLane * 64; c < n; c += 64) {
      const float mc = p[c * 4];
      if (mc > -INFINITY) s += (double)p[c * 4 + 1] * (double)__expf((mc - M) / T);
    }
  }
  S = wave_sum_d(s);
}

// The token at index idx of sequence b's output, and (stateful verify) the slot's
// pending ingest: d_0 .. d_{A-1}, then `tok`.  One thread.
OSP_DEV void finalize(const VerifyArgs& a, int b, int idx, int A, int tok) {
  a.out_tokens[(long)b * (a.K + 1) + idx] = tok;
  if (a.bslot) {
    const int slot = a.bslot[b];
    const int32_t* dr = a.drafts + (long)b * a.ld_drafts;
    a.pend_n[slot] = A + 1;
    for (int k = 0; k < A; ++k) a.pend_tok[(long)slot * a.pend_ld + k] = dr[k];
    a.pend_tok[(long)slot * a.pend_ld + A] = tok;
  }
}

// Acceptance of sequence b's chain (one block): the chunk records of every row are
// merged in parallel (one wavefront per row), thread k decides draft k, and the
// accepted length is the first rejection.  At T = 0 the sequence is finished here (the
// next token is the argmax of row a).
OSP_DEV void accept_tail(const VerifyArgs& a, int b) {
  __shared__ float s_M[2 * 64 + 1];
  __shared__ double s_S[2 * 64 + 1];
  __shared__ int s_am[2 * 64 + 1];
  __shared__ int s_ok[64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.K;
  const int nt = (K + 1) * a.nchunk_t;
  const int nj = nt + (a.qstat ? 0 : K * a.nchunk_d);
  const float* part = a.part + (long)b * nj * 4;
  const float T = a.temp[b], Td = a.temp_d[b];
  // drafter rows: the statistics the sampling kernel kept, or merged chunks
  const bool kept = a.qstat != nullptr;
  if (kept && T > 0.f && tid < K) {
    const QStat qs = a.qstat[(long)b * a.ld_qstat + tid];
    s_M[K + 1 + tid] = qs.M;
    s_S[K + 1 + tid] = qs.S;
    s_am[K + 1 + tid] = qs.am;
  }
  const int nrows = (K + 1) + (T > 0.f && !kept ? K : 0);
  for (int q = wave; q < nrows; q += kVThreads / 64) {
    float M;
    double S;
    int am;
    if (q <= K) merge_row(part + (long)q * a.nchunk_t * 4, a.nchunk_t, T, M, S, am);
    else merge_row(part + ((long)nt + (long)(q - K - 1) * a.nchunk_d) * 4, a.nchunk_d, Td, M, S, am);
    if (lane == 0) { s_M[q] = M; s_S[q] = S; s_am[q] = am; }
  }
  __syncthreads();
  const int32_t* dr = a.drafts + (long)b * a.ld_drafts;
  if (tid < K) {
    const int k = tid;
    const int d = dr[k];
    int ok = 0;
    if (d < 0 || d >= a.V_T) {
      atomicOr(a.err, 1u << 4);
    } else if (T <= 0.f) {
      ok = d == s_am[k];
    } else {
      const float* tl = a.target + ((long)b * (K + 1) + k) * a.V_T;
      const int s = a.t2d[d];
      const float tv = tl[d];
      double qd = 0.0;
      if (s >= 0) {
        if (Td > 0.f) {
          const float ls = a.draft[((long)b * a.ld_draft_b + k) * a.V_d + s];
          if (ls > -INFINITY) qd = (double)__expf((ls - s_M[K + 1 + k]) / Td) / s_S[K + 1 + k];
        } else {
          qd = s == s_am[K + 1 + k] ? 1.0 : 0.0;   // greedy drafting: q one-hot
        }
      }
      const double pd = (double)__expf((tv - s_M[k]) / T) / s_S[k];
      const double r = qd > 0.0 ? fmin(1.0, pd / qd) : (pd > 0.0 ? 1.0 : 0.0);
      ok = (double)a.u_acc[(long)b * K + k] < r;
    }
    s_ok[k] = ok;
  }
  __syncthreads();
  int A = 0;
  while (A < K && s_ok[A]) ++A;
  if (tid < K) {
    a.accept_mask[(long)b * K + tid] = tid < A ? 1 : 0;
    a.out_tokens[(long)b * (K + 1) + tid] = tid < A ? dr[tid] : -1;
  }
  if (tid == 0) {
    a.out_tokens[(long)b * (K + 1) + K] = -1;
    a.accept_len[b] = A;
    // statistics of row A for the residual pass
    a.vstate[b * 4 + 0] = A;
    a.vstate[b * 4 + 1] = s_am[A];
    a.vstat[b * 4 + 0] = s_M[A];
    a.vstat[b * 4 + 1] = s_S[A];
    const bool dq = A < K && T > 0.f;
    a.vstat[b * 4 + 2] = dq ? s_M[K + 1 + A] : 0.0;
    a.vstat[b * 4 + 3] = (dq && Td > 0.f) ? s_S[K + 1 + A] : 1.0;
    // greedy drafting: the drafter row q_a is one-hot at (-1: no drafter row / a = K)
    a.vstate[b * 4 + 2] = (dq && !(Td > 0.f)) ? s_am[K + 1 + A] : -1;
  }
  __syncthreads();   // (the token at index A is written after the -1 above)
  if (tid == 0 && !(T > 0.f)) finalize(a, b, A, A, s_am[A]);
}

// Residual weight max(0, p(v) - q(v)) and p(v) of target id v in row a.  The
// normalisers are float64 so that p and q carry no common fp32 scale error.
struct ResidRow {
  const float* tl;   // target row a
  const float* dl;   // drafter row a (nullptr when a = K)
  const int32_t* t2d;
  float Mt, Md, T, Td;
  float iT;          // 1 / T
  double iSt, iSd;   // 1 / normalisers
  int onehot;        // Td = 0: the drafter row q_a is one-hot at (else -1)
  const int32_t* rem;   // draft trees: tokens removed from p (nrem of them); chains: nrem < 0
  int nrem;
  OSP_DEV bool removed(int v) const {
    bool r = false;
    for (int i = 0; i < nrem; ++i) r |= rem[i] == v;
    return r;
  }
  // residual weight of target id v with target probability p (drafter row entry s, logit l)
  OSP_DEV double resid(double p, int v, int s, float l) const {
    if (nrem >= 0) return removed(v) ? 0.0 : p;
    return fmax(p - q_of(s, l), 0.0);
  }
  // q_a(v) from the drafter row entry s = t2d[v] (-1: none) and its logit l
  OSP_DEV double q_of(int s, float l) const {
    if (!dl || s < 0) return 0.0;
    if (!(Td > 0.f)) return s == onehot ? 1.0 : 0.0;
    return l > -INFINITY ? (double)__expf((l - Md) / Td) * iSd : 0.0;
  }
  // Residual weight (which = 0) or target probability (which = 1) of id v (0 at or past V).
  OSP_DEV double eval_one(int v, int V, int which) const {
    const bool in = v < V;
    const float t = in ? tl[v] : -INFINITY;
    const int s = (in && dl && !which) ? t2d[v] : -1;
    const float d = (s >= 0 && Td > 0.f) ? dl[s] : -INFINITY;
    const double p = t > -INFINITY ? (double)__expf((t - Mt) * iT) * iSt : 0.0;
    return which ? p : resid(p, v, s, d);
  }
};

OSP_DEV ResidRow resid_row(const VerifyArgs& a, int b) {
  ResidRow r;
  const int A = a.vstate[b * 4 + 0];
  r.tl = a.target + ((long)b * (a.K + 1) + A) * a.V_T;
  r.dl = (A < a.K && !a.tree_par) ? a.draft + ((long)b * a.ld_draft_b + A) * a.V_d : nullptr;
  r.rem = a.tree_par ? a.tree_removed + (long)b * kMaxTreeNodes : nullptr;
  r.nrem = a.tree_par ? a.vstate[b * 4 + 3] : -1;
  r.t2d = a.t2d;
  r.Mt = (float)a.vstat[b * 4 + 0];
  r.iSt = 1.0 / a.vstat[b * 4 + 1];
  r.Md = (float)a.vstat[b * 4 + 2];
  r.iSd = 1.0 / a.vstat[b * 4 + 3];
  r.T = a.temp[b];
  r.iT = 1.0f / r.T;
  r.Td = a.temp_d[b];
  r.onehot = a.vstate[b * 4 + 2];
  return r;
}

// Sums of 16 float64 values per lane over the 64 lanes at once: on return v[0] of lane l
// holds the total of value index l >> 2 (21 shuffle steps instead of 6 x 16).  Fixed
// order.  Every step is a template with compile-time indices, so the values stay in
// registers (a loop whose bounds the compiler cannot resolve indexes them by runtime
// selects).
template <int H, int M>
OSP_DEV void tr_step(double* v, int lane) {
  const bool hi = (lane & M) != 0;
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const double mine = hi ? v[i + H] : v[i];
    const double other = hi ? v[i] : v[i + H];
    v[i] = mine + xor_lane_d<M>(other, lane);
  }
}
OSP_DEV double transpose_reduce16_d(double* v, int lane) {
  tr_step<8, 32>(v, lane);
  tr_step<4, 16>(v, lane);
  tr_step<2, 8>(v, lane);
  tr_step<1, 4>(v, lane);
  v[0] += xor_lane_d<2>(v[0], lane);
  v[0] += xor_lane_d<1>(v[0], lane);
  return v[0];
}
static_assert(kVPer == 16 && kVSub == 4 * kVPer, "one sub-range per (id group q, wavefront)");

// The draw of sequence b (one wavefront): the inverse CDF over the residual (or over
// p_a if the residual is empty) in ascending target ids, in three steps -- the chunk (totals in order), the 64-id
// sub-range within it (its kVSub sums), the id (one id per lane) -- each falling back,
// where rounding leaves the draw point past the last positive entry, to the last
// positive entry of that level.
OSP_DEV void final_tail(const VerifyArgs& a, int b, const ResidRow& rr) {
  const int lane = threadIdx.x & 63;
  if (threadIdx.x >= 64) return;
  const int n = a.nchunk_t;
  const double* rp = a.res_part + (long)b * n * 2;
  double W = 0.0;
  for (int c0 = 0; c0 < n; c0 += 64) {
    const int c = c0 + lane;
    W += wave_sum_d(c < n ? rp[c * 2] : 0.0);
  }
  const int which = W > 0.0 ? 0 : 1;
  double tot = W;
  if (which) {
    tot = 0.0;
    for (int c0 = 0; c0 < n; c0 += 64) {
      const int c = c0 + lane;
      tot += wave_sum_d(c < n ? rp[c * 2 + 1] : 0.0);
    }
  }
  const double target = (double)a.u_bonus[b] * tot;
  // 1. the chunk
  double run = 0.0, before = 0.0, before_last = 0.0;
  int ch = -1, last = -1;
  for (int c0 = 0; c0 < n && ch < 0; c0 += 64) {
    const int c = c0 + lane;
    const double v = c < n ? rp[c * 2 + which] : 0.0;
    const double inc = wave_incl_scan<double>(v);
    const unsigned long long pos = __ballot(c < n && v > 0.0);
    if (pos) {
      const int l = 63 - __builtin_clzll(pos);
      last = c0 + l;
      before_last = run + lane_d(inc, l) - lane_d(v, l);
    }
    const unsigned long long hit = __ballot(c < n && v > 0.0 && run + inc > target);
    if (hit) {
      const int l = __builtin_ctzll(hit);
      ch = c0 + l;
      before = run + lane_d(inc, l) - lane_d(v, l);
    }
    run += lane_d(inc, 63);
  }
  int tok = -1;
  if (ch < 0 && last >= 0) { ch = last; before = before_last; }
  if (ch >= 0) {
    // 2. the 64-id sub-range (j covers ids ch * chunk + (j / 4) * 256 + (j % 4) * 64 ..)
    const double* sub = a.res_sub + ((long)b * n + ch) * kVSub * 2;
    const double v = sub[lane * 2 + which];
    const double inc = wave_incl_scan<double>(v);
    const unsigned long long pos = __ballot(v > 0.0);
    const unsigned long long hit = __ballot(v > 0.0 && before + inc > target);
    int j = -1;
    if (hit) j = __builtin_ctzll(hit);
    else if (pos) j = 63 - __builtin_clzll(pos);
    if (j >= 0) {
      const double before2 = before + lane_d(inc, j) - lane_d(v, j);
      // 3. the id
      const int i1 = min(a.V_T, ch * a.chunk + a.chunk);
      const int id = ch * a.chunk + (j >> 2) * kVThreads + (j & 3) * 64 + lane;
      const double x = rr.eval_one(id, i1, which);
      const double inc2 = wave_incl_scan<double>(x);
      const unsigned long long pos2 = __ballot(x > 0.0);
      const unsigned long long hit2 = __ballot(x > 0.0 && before2 + inc2 > target);
      if (hit2) tok = lane_i(id, __builtin_ctzll(hit2));
      else if (pos2) tok = lane_i(id, 63 - __builtin_clzll(pos2));
    }
  }
  if (tok < 0) tok = a.vstate[b * 4 + 1];   // nothing positive at all: the argmax
  if (lane == 0)
    finalize(a, b, a.tree_par ? a.accept_len[b] : a.vstate[b * 4 + 0], a.vstate[b * 4 + 0], tok);
}

// Per chunk of target row a: the sums of the residual weights and of p, per 64-id
// sub-range and per chunk (the chunk total is the sum of its sub-ranges).
// Thread t takes ids t, t + 256, ... of the chunk: every wavefront load is 256
// contiguous bytes, and both sums come from one pass over the row.  Greedy sequences
// (T = 0) were finished by the acceptance.
__global__ void __launch_bounds__(kVThreads) k_vresid(VerifyArgs a) {
  __shared__ double s_sub[kVSub][2];
  const int b = blockIdx.x, c = blockIdx.y;
  if (!(a.temp[b] > 0.f)) return;
  const ResidRow rr = resid_row(a, b);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = c * a.chunk + tid;
  const int i1 = min(a.V_T, c * a.chunk + a.chunk);
  float tv[kVPer];
  int sidx[kVPer];
#pragma unroll
  for (int q = 0; q < kVPer; ++q) {
    const int v = i0 + q * kVThreads;
    const bool in = v < i1;
    tv[q] = in ? rr.tl[v] : -INFINITY;
    sidx[q] = (in && rr.dl) ? rr.t2d[v] : -1;
  }
  float dv[kVPer];
#pragma unroll
  for (int q = 0; q < kVPer; ++q) dv[q] = (sidx[q] >= 0 && rr.Td > 0.f) ? rr.dl[sidx[q]] : -INFINITY;
  double sw[kVPer], sp[kVPer];
#pragma unroll
  for (int q = 0; q < kVPer; ++q) {
    const double p = tv[q] > -INFINITY ? (double)__expf((tv[q] - rr.Mt) * rr.iT) * rr.iSt : 0.0;
    sw[q] = rr.resid(p, i0 + q * kVThreads, sidx[q], dv[q]);
    sp[q] = p;
  }
  // the 64 ids of (q, this wavefront) are consecutive: one sub-range each
  const double tw = transpose_reduce16_d(sw, lane);
  const double tp = transpose_reduce16_d(sp, lane);
  if ((lane & 3) == 0) {
    s_sub[(lane >> 2) * 4 + wave][0] = tw;
    s_sub[(lane >> 2) * 4 + wave][1] = tp;
  }
  __syncthreads();
  // wavefront 0: the sub-range sums out, and the chunk's totals (a fixed butterfly
  // order over the 64 sub-ranges)
  if (tid < kVSub) {
    double* sub = a.res_sub + ((long)b * a.nchunk_t + c) * kVSub * 2;
    const double w = s_sub[tid][0], pp = s_sub[tid][1];
    sub[tid * 2 + 0] = w;
    sub[tid * 2 + 1] = pp;
    const double tw2 = wave_sum_d(w), tp2 = wave_sum_d(pp);
    if (tid == 0) {
      a.res_part[((long)b * a.nchunk_t + c) * 2 + 0] = tw2;
      a.res_part[((long)b * a.nchunk_t + c) * 2 + 1] = tp2;
    }
  }
}

// One wavefront per sequence: the draw (final_tail) over the residual kernel's sums.
__global__ void __launch_bounds__(64) k_vfinal(VerifyArgs a) {
  const int b = blockIdx.x;
  if (!(a.temp[b] > 0.f)) return;
  final_tail(a, b, resid_row(a, b));
}

// Walk of sequence b's draft tree (one block).  Every node's token, parent, uniform and target logit in its parent's row are read at
// once (thread c: node c), the K + 1 row statistics merged in parallel (one wavefront
// per row); one thread then walks the tree from the root: the children of a node
// follow it in index order, so the walk ends within K steps.  At T = 0 the bonus (the
// argmax of the last node's row) is written here.
OSP_DEV void walk_tail(const VerifyArgs& a, int b) {
  __shared__ float s_M[kMaxTreeNodes + 1];
  __shared__ double s_S[kMaxTreeNodes + 1];
  __shared__ int s_am[kMaxTreeNodes + 1];
  __shared__ int s_tok[kMaxTreeNodes], s_par[kMaxTreeNodes], s_path[kMaxTreeNodes];
  __shared__ float s_lt[kMaxTreeNodes], s_u[kMaxTreeNodes];
  __shared__ int s_rem[kMaxTreeNodes];
  __shared__ int s_A, s_nrem, s_row;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.K;
  const float T = a.temp[b];
  if (tid < N) {
    int t = a.tree_tok[(long)b * N + tid];
    int p = a.tree_par[(long)b * N + tid];
    if (p < -1 || p >= tid) { atomicOr(a.err, 1u << 5); p = -2; }      // unreachable
    if (t < 0 || t >= a.V_T) { atomicOr(a.err, 1u << 4); t = 0; p = -2; }
    s_tok[tid] = t;
    s_par[tid] = p;
    s_u[tid] = a.u_acc[(long)b * N + tid];
    s_lt[tid] = a.target[((long)b * (N + 1) + max(p, -1) + 1) * a.V_T + t];
  }
  const float* part = a.part + (long)b * (N + 1) * a.nchunk_t * 4;
  for (int q = wave; q <= N; q += kVThreads / 64) {
    float M;
    double S;
    int am;
    merge_row(part + (long)q * a.nchunk_t * 4, a.nchunk_t, T, M, S, am);
    if (lane == 0) { s_M[q] = M; s_S[q] = S; s_am[q] = am; }
  }
  __syncthreads();
  if (tid == 0) {
    int* rem = s_rem;
    int cur = -1, A = 0, nrem = 0;
    for (;;) {
      const int row = cur + 1;
      int nxt = -1;
      double left = 1.0;                 // target mass not yet removed at this node
      nrem = 0;
      for (int c = cur + 1; c < N && nxt < 0; ++c) {
        if (s_par[c] != cur) continue;
        const int t = s_tok[c];
        if (!(T > 0.f)) {
          if (t == s_am[row]) nxt = c;
          continue;
        }
        bool dup = false;
        for (int r = 0; r < nrem; ++r) dup |= rem[r] == t;
        if (dup) continue;               // already rejected here: p'(t) = 0
        const double pt = s_lt[c] > -INFINITY ? (double)__expf((s_lt[c] - s_M[row]) / T) / s_S[row] : 0.0;
        if (left > 0.0 && (double)s_u[c] < pt / left) {
          nxt = c;
        } else {
          rem[nrem++] = t;
          left -= pt;
        }
      }
      if (nxt < 0) break;
      s_path[A++] = nxt;
      cur = nxt;
    }
    s_A = A;
    s_nrem = T > 0.f ? nrem : 0;
    const int row = cur + 1;
    s_row = row;
    a.accept_len[b] = A;
    a.vstate[b * 4 + 0] = row;
    a.vstate[b * 4 + 1] = s_am[row];
    a.vstate[b * 4 + 2] = -1;
    a.vstate[b * 4 + 3] = T > 0.f ? nrem : 0;
    a.vstat[b * 4 + 0] = s_M[row];
    a.vstat[b * 4 + 1] = s_S[row];
    a.vstat[b * 4 + 2] = 0.0;
    a.vstat[b * 4 + 3] = 1.0;
  }
  __syncthreads();
  const int A = s_A;
  if (tid < s_nrem) a.tree_removed[(long)b * kMaxTreeNodes + tid] = s_rem[tid];
  for (int i = tid; i < N; i += kVThreads) a.tree_path[(long)b * N + i] = i < A ? s_path[i] : -1;
  for (int i = tid; i <= N; i += kVThreads)
    if (i != A) a.out_tokens[(long)b * (N + 1) + i] = i < A ? s_tok[s_path[i]] : -1;
  if (tid == 0 && !(T > 0.f)) finalize(a, b, A, A, s_am[s_row]);
}

// Chunk statistics of every target row (and, for verify_rows, drafter row), one
// wavefront per 4096-id chunk.
template <bool STREAM>
__global__ void __launch_bounds__(kVThreads) k_vstats(VerifyArgs a) {
  const int b = blockIdx.x;
  const int j = blockIdx.y * (kVThreads / 64) + (threadIdx.x >> 6);
  const int nt = (a.K + 1) * a.nchunk_t;
  const int nj = nt + (a.qstat || a.tree_par ? 0 : a.K * a.nchunk_d);
  if (j < nj) chunk_stats<STREAM>(a, b, j, nt, nj);
}

// Rows of more than 128 MB in all are streamed (k_vstats<true>).
constexpr long kVStreamBytes = 128L << 20;
static void launch_vstats(const VerifyArgs& a, int nj, bool drafts, hipStream_t st) {
  const long bytes = 4L * a.B * ((a.K + 1) * (long)a.V_T + (drafts ? (long)a.K * a.V_d : 0L));
  const dim3 grid(a.B, (nj + kVThreads / 64 - 1) / (kVThreads / 64));
  if (bytes > kVStreamBytes) hipLaunchKernelGGL(k_vstats<true>, grid, dim3(kVThreads), 0, st, a);
  else hipLaunchKernelGGL(k_vstats<false>, grid, dim3(kVThreads), 0, st, a);
}

__global__ void __launch_bounds__(kVThreads) k_vaccept(VerifyArgs a) { accept_tail(a, blockIdx.x); }
__global__ void __launch_bounds__(kVThreads) k_tree_walk(VerifyArgs a) { walk_tail(a, blockIdx.x); }

void launch_verify_tree(const VerifyArgs& a, hipStream_t st) {
  const int nj = (a.K + 1) * a.nchunk_t;
  launch_vstats(a, nj, false, st);
  hipLaunchKernelGGL(k_tree_walk, dim3(a.B), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vresid, dim3(a.B, a.nchunk_t), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vfinal, dim3(a.B), dim3(64), 0, st, a);
}

void launch_verify(const VerifyArgs& a, hipStream_t st) {
  const int nj = (a.K + 1) * a.nchunk_t + (a.qstat ? 0 : a.K * a.nchunk_d);
  launch_vstats(a, nj, !a.qstat, st);
  hipLaunchKernelGGL(k_vaccept, dim3(a.B), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vresid, dim3(a.B, a.nchunk_t), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vfinal, dim3(a.B), dim3(64), 0, st, a);
}

}  // namespace osp

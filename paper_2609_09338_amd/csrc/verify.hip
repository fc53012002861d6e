// Lossless verification of the drafted chain (the standard speculative
// decoding acceptance rule, unchanged by the paper).
//
// Row convention per sequence: drafts d_0..d_{K-1} with drafter logit rows
// q_0..q_{K-1} (over drafter rows, mapped to target ids by d2t / t2d); target
// logit rows p_0..p_K over target ids.
//
//   k_vstats  (B x jobs)   per chunk of every target and drafter row: max,
//                          lowest argmax and sum exp((l - max)/T)
//   k_vaccept (B)          merges chunks in order; accepts d_k while
//                          u_k < min(1, p_k(d_k)/q_k(d_k)) (T = 0: d_k equals
//                          the target argmax); writes a, the mask and d_0..d_{a-1}
//   k_vresid  (B x chunks) per chunk of target row a: sum of the residual
//                          max(0, p_a - q_a) (q = 0 when a = K) and of p_a
//   k_vfinal  (B)          inverse CDF over the residual (or p_a if it is empty)
//                          in ascending target ids -> the token at index a;
//                          stateful verify also records the a + 1 committed
//                          tokens as the slot's pending ingest
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kVThreads = 256;

OSP_DEV void block_max_argmax(float& m, int& am, float* sm, int* si) {
  const int tid = threadIdx.x;
  sm[tid] = m;
  si[tid] = am;
  __syncthreads();
  for (int s = kVThreads / 2; s > 0; s >>= 1) {
    if (tid < s) {
      const float o = sm[tid + s];
      const int oi = si[tid + s];
      if (o > sm[tid] || (o == sm[tid] && oi < si[tid])) { sm[tid] = o; si[tid] = oi; }
    }
    __syncthreads();
  }
  m = sm[0];
  am = si[0];
  __syncthreads();
}

OSP_DEV double block_sum(double v, double* sm) {
  const int tid = threadIdx.x;
  sm[tid] = v;
  __syncthreads();
  for (int s = kVThreads / 2; s > 0; s >>= 1) {
    if (tid < s) sm[tid] += sm[tid + s];
    __syncthreads();
  }
  const double r = sm[0];
  __syncthreads();
  return r;
}

__global__ void __launch_bounds__(kVThreads) k_vstats(VerifyArgs a) {
  __shared__ float sm[kVThreads];
  __shared__ int si[kVThreads];
  __shared__ double sd[kVThreads];
  const int b = blockIdx.x, j = blockIdx.y;
  const int tid = threadIdx.x;
  const int nt = (a.K + 1) * a.nchunk_t;
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
  float m = -INFINITY;
  int am = 0x7fffffff;
  for (int i = i0 + tid; i < i1; i += kVThreads) {
    const float v = row[i];
    if (v > m) { m = v; am = i; }
  }
  block_max_argmax(m, am, sm, si);
  const float T = a.temp[b];
  double se = 0.0;   // float64 sums: exactness of the 10^5-entry CDFs that follow
  if (T > 0.f && m > -INFINITY)
    for (int i = i0 + tid; i < i1; i += kVThreads) se += (double)__expf((row[i] - m) / T);
  se = block_sum(se, sd);
  if (tid == 0) {
    float* p = a.part + ((long)b * gridDim.y + j) * 4;
    p[0] = m;
    p[1] = (float)se;
    p[2] = __int_as_float(m > -INFINITY ? am : -1);
    p[3] = 0.f;
  }
}

// Merge the chunk statistics of one row with one wavefront: max M, lowest
// argmax, S = sum exp((l - M)/T).  Fixed summation order.
OSP_DEV void merge_row(const float* p, int n, float T, float& M, double& S, int& am) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY;
  int ai = 0x7fffffff;
  for (int c = lane; c < n; c += 64) {
    const float mc = p[c * 4];
    const int ac = __float_as_int(p[c * 4 + 2]);
    if (mc > m || (mc == m && mc > -INFINITY && ac < ai)) { m = mc; ai = ac; }
  }
  M = wave_max(m);
  am = wave_min_i((m == M && m > -INFINITY) ? ai : 0x7fffffff);
  if (am == 0x7fffffff) am = -1;
  double s = 0.0;
  if (T > 0.f && M > -INFINITY)
    for (int c = lane; c < n; c += 64) {
      const float mc = p[c * 4];
      if (mc > -INFINITY) s += (double)p[c * 4 + 1] * (double)__expf((mc - M) / T);
    }
  S = wave_sum_d(s);
}

__global__ void __launch_bounds__(64) k_vaccept(VerifyArgs a) {
  const int b = blockIdx.x;
  const bool lead = threadIdx.x == 0;
  const int nt = (a.K + 1) * a.nchunk_t;
  const int nj = nt + a.K * a.nchunk_d;
  const float* part = a.part + (long)b * nj * 4;
  const float T = a.temp[b];
  const int32_t* dr = a.drafts + (long)b * a.ld_drafts;
  int acc = 0;
  for (; acc < a.K; ++acc) {
    const int k = acc;
    float Mt, Md;
    double St, Sd;
    int at, ad;
    merge_row(part + (long)k * a.nchunk_t * 4, a.nchunk_t, T, Mt, St, at);
    int d = dr[k];
    if (d < 0 || d >= a.V_T) { if (lead) atomicOr(a.err, 1u << 4); break; }
    bool ok;
    if (T <= 0.f) {
      ok = (d == at);
    } else {
      merge_row(part + ((long)nt + (long)k * a.nchunk_d) * 4, a.nchunk_d, T, Md, Sd, ad);
      const float* tl = a.target + ((long)b * (a.K + 1) + k) * a.V_T;
      const double pd = (double)__expf((tl[d] - Mt) / T) / St;
      const int s = a.t2d[d];
      double qd = 0.0;
      if (s >= 0) {
        const float* dl = a.draft + ((long)b * a.ld_draft_b + k) * a.V_d;
        const float ls = dl[s];
        qd = ls > -INFINITY ? (double)__expf((ls - Md) / T) / Sd : 0.0;
      }
      const double r = qd > 0.0 ? fmin(1.0, pd / qd) : (pd > 0.0 ? 1.0 : 0.0);
      ok = (double)a.u_acc[(long)b * a.K + k] < r;
    }
    if (!ok) break;
  }
  const int A = acc;
  if (lead) for (int k = 0; k < a.K; ++k) {
    a.accept_mask[(long)b * a.K + k] = k < A ? 1 : 0;
    a.out_tokens[(long)b * (a.K + 1) + k] = k < A ? dr[k] : -1;
  }
  if (lead) {
    a.out_tokens[(long)b * (a.K + 1) + a.K] = -1;
    a.accept_len[b] = A;
  }
  // statistics of row A for the residual pass
  float Mt, Md = 0.f;
  double St, Sd = 1.0;
  int at, ad = -1;
  merge_row(part + (long)A * a.nchunk_t * 4, a.nchunk_t, T, Mt, St, at);
  if (A < a.K && T > 0.f)
    merge_row(part + ((long)nt + (long)A * a.nchunk_d) * 4, a.nchunk_d, T, Md, Sd, ad);
  if (lead) {
    a.vstate[b * 4 + 0] = A;
    a.vstate[b * 4 + 1] = at;
    a.vstat[b * 4 + 0] = Mt;
    a.vstat[b * 4 + 1] = St;
    a.vstat[b * 4 + 2] = Md;
    a.vstat[b * 4 + 3] = Sd;
  }
}

// Residual weight max(0, p(v) - q(v)) and p(v) of target id v in row a.  The
// normalisers are float64 so that p and q carry no common fp32 scale error.
struct ResidRow {
  const float* tl;   // target row a
  const float* dl;   // drafter row a (nullptr when a = K)
  const int32_t* t2d;
  float Mt, Md, T;
  double iSt, iSd;   // 1 / normalisers
  OSP_DEV void eval(int v, double& w, double& p) const {
    p = (double)__expf((tl[v] - Mt) / T) * iSt;
    double q = 0.0;
    if (dl) {
      const int s = t2d[v];
      if (s >= 0) {
        const float l = dl[s];
        if (l > -INFINITY) q = (double)__expf((l - Md) / T) * iSd;
      }
    }
    w = fmax(p - q, 0.0);
  }
};

OSP_DEV ResidRow resid_row(const VerifyArgs& a, int b) {
  ResidRow r;
  const int A = a.vstate[b * 4 + 0];
  r.tl = a.target + ((long)b * (a.K + 1) + A) * a.V_T;
  r.dl = A < a.K ? a.draft + ((long)b * a.ld_draft_b + A) * a.V_d : nullptr;
  r.t2d = a.t2d;
  r.Mt = (float)a.vstat[b * 4 + 0];
  r.iSt = 1.0 / a.vstat[b * 4 + 1];
  r.Md = (float)a.vstat[b * 4 + 2];
  r.iSd = 1.0 / a.vstat[b * 4 + 3];
  r.T = a.temp[b];
  return r;
}

__global__ void __launch_bounds__(kVThreads) k_vresid(VerifyArgs a) {
  __shared__ double sm[4];
  const int b = blockIdx.x, c = blockIdx.y;
  if (!(a.temp[b] > 0.f)) return;
  const ResidRow rr = resid_row(a, b);
  const int i0 = c * a.chunk, i1 = min(a.V_T, i0 + a.chunk);
  // thread t owns a contiguous run of the chunk (the same split as the final scan)
  const int per = (a.chunk + kVThreads - 1) / kVThreads;
  const int t0 = min(i1, i0 + (int)threadIdx.x * per), t1 = min(i1, t0 + per);
  double sw = 0.0, sp = 0.0;
  for (int v = t0; v < t1; ++v) { double w, p; rr.eval(v, w, p); sw += w; sp += p; }
  // fixed-order block sums in float64
  double incl, tw, tp;
  block_scan<kVThreads, double>(sw, sm, incl, tw);
  block_scan<kVThreads, double>(sp, sm, incl, tp);
  if (threadIdx.x == 0) {
    a.res_part[((long)b * a.nchunk_t + c) * 2 + 0] = tw;
    a.res_part[((long)b * a.nchunk_t + c) * 2 + 1] = tp;
  }
}

__global__ void __launch_bounds__(kVThreads) k_vfinal(VerifyArgs a) {
  __shared__ double sm[4];
  __shared__ int s_chunk, s_tok;
  __shared__ double s_before, s_target;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int A = a.vstate[b * 4 + 0];
  const float T = a.temp[b];
  int tok;
  if (!(T > 0.f)) {
    tok = a.vstate[b * 4 + 1];
  } else {
    const ResidRow rr = resid_row(a, b);
    if (wave == 0) {
      // chunk totals in order: which = 0 residual, 1 = p (when the residual is empty)
      const double* rp = a.res_part + (long)b * a.nchunk_t * 2;
      double W = 0.0;
      for (int c0 = 0; c0 < a.nchunk_t; c0 += 64) {
        const int c = c0 + lane;
        W += wave_sum_d(c < a.nchunk_t ? rp[c * 2] : 0.0);
      }
      const int which = W > 0.0 ? 0 : 1;
      double tot = W;
      if (which) {
        tot = 0.0;
        for (int c0 = 0; c0 < a.nchunk_t; c0 += 64) {
          const int c = c0 + lane;
          tot += wave_sum_d(c < a.nchunk_t ? rp[c * 2 + 1] : 0.0);
        }
      }
      const double target = (double)a.u_bonus[b] * tot;
      double run = 0.0;
      int ch = -1;
      double before = 0.0;
      for (int c0 = 0; c0 < a.nchunk_t; c0 += 64) {
        const int c = c0 + lane;
        const double v = c < a.nchunk_t ? rp[c * 2 + which] : 0.0;
        const double inc = wave_incl_scan<double>(v);
        const unsigned long long hit = __ballot(c < a.nchunk_t && v > 0.0 && run + inc > target);
        if (hit) {
          const int l = __builtin_ctzll(hit);
          ch = c0 + l;
          before = run + __shfl(inc, l, OSP_WAVE) - __shfl(v, l, OSP_WAVE);
          break;
        }
        run += __shfl(inc, 63, OSP_WAVE);
      }
      if (ch < 0) {                      // rounding: the last chunk
        ch = a.nchunk_t - 1;
        before = run - rp[(long)ch * 2 + which];
      }
      if (lane == 0) {
        s_chunk = ch * 2 + which;
        s_before = before;
        s_target = target;
        s_tok = -1;
      }
    }
    __syncthreads();
    const int ch = s_chunk >> 1, which = s_chunk & 1;
    const int i0 = ch * a.chunk, i1 = min(a.V_T, i0 + a.chunk);
    const int per = (a.chunk + kVThreads - 1) / kVThreads;
    const int t0 = min(i1, i0 + tid * per), t1 = min(i1, t0 + per);
    double loc = 0.0;
    for (int v = t0; v < t1; ++v) { double w, p; rr.eval(v, w, p); loc += which ? p : w; }
    double incl_l, tot_l;
    const double excl_l = block_scan<kVThreads, double>(loc, sm, incl_l, tot_l);
    const double target = s_target;
    const double excl = s_before + excl_l;
    if (t0 < t1 && excl <= target && s_before + incl_l > target) {
      double run = excl;
      for (int v = t0; v < t1; ++v) {
        double w, p;
        rr.eval(v, w, p);
        const double x = which ? p : w;
        if (x > 0.0 && run + x > target) { s_tok = v; break; }
        run += x;
      }
    }
    __syncthreads();
    if (tid == 0 && s_tok < 0) {       // rounding: take the last positive id of the chunk
      for (int v = i1 - 1; v >= i0; --v) {
        double w, p;
        rr.eval(v, w, p);
        if ((which ? p : w) > 0.0) { s_tok = v; break; }
      }
      if (s_tok < 0) s_tok = a.vstate[b * 4 + 1];
    }
    __syncthreads();
    tok = s_tok;
  }
  if (tid == 0) {
    a.out_tokens[(long)b * (a.K + 1) + A] = tok;
    if (a.bslot) {
      const int slot = a.bslot[b];
      a.pend_n[slot] = A + 1;
      for (int k = 0; k <= A; ++k)
        a.pend_tok[(long)slot * a.pend_ld + k] = a.out_tokens[(long)b * (a.K + 1) + k];
    }
  }
}

void launch_verify(const VerifyArgs& a, hipStream_t st) {
  const int nj = (a.K + 1) * a.nchunk_t + a.K * a.nchunk_d;
  hipLaunchKernelGGL(k_vstats, dim3(a.B, nj), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vaccept, dim3(a.B), dim3(64), 0, st, a);
  hipLaunchKernelGGL(k_vresid, dim3(a.B, a.nchunk_t), dim3(kVThreads), 0, st, a);
  hipLaunchKernelGGL(k_vfinal, dim3(a.B), dim3(kVThreads), 0, st, a);
}

}  // namespace osp

// Weight-streaming matrix-vector products of the drafter (few rows at a time).
//
// Y[r][n] = sum_c X[r][c] * W[n][c] for the rows r of one forward pass.  Every
// weight byte is read from HBM once per block of RB rows.  Each wavefront is
// independent (no LDS, no barriers): it owns a contiguous range of weight rows
// and walks it NW rows at a time; lane l reads the 16-byte column vectors
// l, l+64, ..., l+64(XV-1) of those rows, i.e. NW*XV fully coalesced 1 KB
// wavefront loads in flight per step.  The lane's matching input values are
// loaded once per wavefront and kept in registers when the row fits
// (Kd <= 64*XV*VEC; otherwise they are re-read per step, chunk by chunk).  The
// NW*RB partial sums are reduced across the 64 lanes with one transposed
// butterfly.
//
// The virtual input X is formed on the fly (the norm prologues of the body):
//   SRC_PLAIN  fp32 rows (attention output, FFN hidden)
//   SRC_NORM   RMSNorm(x) * gain (post-attention norm, final norm)
//   SRC_QKV    [s ; RMSNorm(x) * gain] -- the expanded-QKV input of Eq. 2-3, read
//              from its two segments with no concatenated copy; in layer 0 x is
//              the embedding row of the token (one wavefront materialises it)
//   SRC_TAPS   target hidden-state taps (Eq. 1)
//   SRC_ATTN   one row's attention output, merged from its context splits by the
//              block into LDS before the products (single rows, Kd <= 2048)
//   SRC_QKV_PICK  SRC_QKV of layer 0 for one sequence: every block draws the step's
//              token itself from the LM head's records (pick.h) while its first
//              weights are in flight, so that no sampling kernel runs in between
// and the epilogue writes, accumulates into the residual, applies SwiGLU, or
// writes masked logits plus, per wavefront range, the (max, sum exp((l-max)/T),
// lowest argmax) statistics that sampling merges.
#pragma once

#include "common.h"
#include "internal.h"
#include "pick.h"

namespace osp {

constexpr int kGemvThreads = 256;
constexpr int kGemvWavesPerBlock = kGemvThreads / OSP_WAVE;

// Expanded-QKV input kinds (the token's own draw aside, the same input).
constexpr bool src_qkv(int src) { return src == SRC_QKV || src == SRC_QKV_PICK; }

template <int N> struct Log2 { static constexpr int v = 1 + Log2<N / 2>::v; };
template <> struct Log2<1> { static constexpr int v = 0; };

// Raw 16-byte weight vector and its widening.
template <typename TW> struct WRaw;
template <> struct WRaw<bf16_t> {
  uint4 v;
  OSP_DEV void load(const bf16_t* p) { v = *reinterpret_cast<const uint4*>(p); }
  OSP_DEV void zero() { v = make_uint4(0u, 0u, 0u, 0u); }
  OSP_DEV float get(int e) const {
    const uint32_t w = e < 2 ? v.x : e < 4 ? v.y : e < 6 ? v.z : v.w;
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  }
  OSP_DEV float dot(const float* x, float s) const {
    s = fmaf(bf16_lo(v.x), x[0], s); s = fmaf(bf16_hi(v.x), x[1], s);
    s = fmaf(bf16_lo(v.y), x[2], s); s = fmaf(bf16_hi(v.y), x[3], s);
    s = fmaf(bf16_lo(v.z), x[4], s); s = fmaf(bf16_hi(v.z), x[5], s);
    s = fmaf(bf16_lo(v.w), x[6], s); s = fmaf(bf16_hi(v.w), x[7], s);
    return s;
  }
};
template <> struct WRaw<float> {
  float4 v;
  OSP_DEV void load(const float* p) { v = *reinterpret_cast<const float4*>(p); }
  OSP_DEV void zero() { v = make_float4(0.f, 0.f, 0.f, 0.f); }
  OSP_DEV float get(int e) const { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; }
  OSP_DEV float dot(const float* x, float s) const {
    s = fmaf(v.x, x[0], s); s = fmaf(v.y, x[1], s); s = fmaf(v.z, x[2], s); s = fmaf(v.w, x[3], s);
    return s;
  }
};

OSP_DEV void load_f4s(const float* p, float* out, int n) {
  for (int e = 0; e < n; e += 4) {
    const float4 v = *reinterpret_cast<const float4*>(p + e);
    out[e] = v.x; out[e + 1] = v.y; out[e + 2] = v.z; out[e + 3] = v.w;
  }
}

// Raw input values X[rr][col .. col+VEC) before normalisation, and whether they
// belong to the normalised segment (norm factor still to be applied).
// (SRC_QKV_PICK: `tok` is the token the block drew; the other kinds ignore it.)
template <typename TW, int SRC, int VEC>
OSP_DEV bool load_x_raw(const GemvArgs& a, int rr, int col, float* out, int tok = 0) {
  if constexpr (SRC == SRC_PLAIN) {
    load_f4s(a.xin + (long)rr * a.ldx + col, out, VEC);
    return false;
  } else if constexpr (SRC == SRC_TAPS) {
    load_vec<TW>(reinterpret_cast<const TW*>(a.taps) + (long)a.tap_row[rr] * a.ldt + col, out);
    return false;
  } else {
    int c = col;
    if constexpr (src_qkv(SRC)) {
      if (col < a.d_norm) {   // conditioning segment, used as is
        const int sr = a.s_gather ? a.s_gather[rr] : rr;
        load_f4s(a.s + (long)sr * a.lds + col, out, VEC);
        return false;
      }
      c = col - a.d_norm;
      if (a.embed) {
        int t = SRC == SRC_QKV_PICK ? tok : a.tok[rr];
        t = min(max(t, 0), a.vocab_embed - 1);
        load_vec<TW>(reinterpret_cast<const TW*>(a.embed) + (long)t * a.d_norm + c, out);
        return true;
      }
    }
    const int xr = a.gather ? a.gather[rr] : rr;
    load_f4s(a.xin + (long)xr * a.ldx + c, out, VEC);
    return true;
  }
}

// Apply RMSNorm factor and gain to a normalised-segment vector.
template <typename TW, int SRC, int VEC>
OSP_DEV void norm_x(const GemvArgs& a, int col, float inv_rms, float* v) {
  const int c = src_qkv(SRC) ? col - a.d_norm : col;
  float g[VEC];
  load_vec<TW>(reinterpret_cast<const TW*>(a.gamma) + c, g);
#pragma unroll
  for (int e = 0; e < VEC; ++e) v[e] = v[e] * inv_rms * g[e];
}

// Column of the gain vector that input column `col` uses (negative: not normalised).
template <int SRC>
OSP_DEV int gain_col(const GemvArgs& a, int col) { return src_qkv(SRC) ? col - a.d_norm : col; }

// 1 / sqrt(mean(x^2) + eps) of the normalised segment of row rr, by one wavefront.
template <typename TW, int SRC>
OSP_DEV float row_inv_rms(const GemvArgs& a, int rr, int lane, int tok) {
  constexpr int VEC = Vec<TW>::N;
  const int d = a.d_norm;
  const int base = src_qkv(SRC) ? d : 0;
  float ss = 0.f;
  for (int c = lane * VEC; c < d; c += OSP_WAVE * VEC) {
    float v[VEC];
    load_x_raw<TW, SRC, VEC>(a, rr, base + c, v, tok);
#pragma unroll
    for (int e = 0; e < VEC; ++e) ss += v[e] * v[e];
  }
  ss = wave_sum(ss);
  return 1.0f / sqrtf(ss / (float)d + a.eps);
}

// Register budget: the streaming kernels want >= 4 wavefronts per SIMD (<= 128 VGPRs)
// so that enough loads are in flight; small-row variants fit that budget.  Normalised
// inputs also hold the first step's weights and the gains across the norm: they get
// 2 wavefronts per SIMD (their grids never place more there).
template <int RB, int NW, int XV, bool NORMED> struct GemvOcc {
  static constexpr int value = (RB * NW * XV <= 8 && RB * XV <= 4) ? (NORMED ? 2 : 4) : 1;
};

// SRC_ATTN: every thread holds its segment of every split's output (one block per CU).
constexpr int kGemvAttnMaxSplit = 20;   // splits merged in the input stage (bound)
constexpr int kGemvAttnMaxHeads = 16;   // heads of the merged row (bound)

template <typename TW, int SRC, int EPI, int RB, int NW, int XV, bool CACHED>
__global__ void __launch_bounds__(kGemvThreads,
                                  (SRC == SRC_ATTN ? 1 : GemvOcc<RB, NW, XV, (SRC == SRC_NORM || src_qkv(SRC))>::value))
k_gemv(GemvArgs a, int rows_per_wave) {
  constexpr int VEC = Vec<TW>::N;
  constexpr int NWV = (EPI == EPI_SWIGLU) ? 2 * NW : NW;
  constexpr int V = NWV * RB;
  constexpr int LOGV = Log2<V>::v;
  constexpr int SH = 6 - LOGV;
  constexpr bool NORMED = (SRC == SRC_NORM || src_qkv(SRC));
  static_assert((1 << LOGV) == V && V <= 64, "values per lane must be a power of two <= 64");

  const int lane = threadIdx.x & (OSP_WAVE - 1);
  const int gw = blockIdx.x * kGemvWavesPerBlock + (threadIdx.x >> 6);
  const int n_lo = gw * rows_per_wave;
  // (the split merge of SRC_ATTN and the pick of SRC_QKV_PICK need every wavefront of
  // the block at their barriers)
  if (SRC != SRC_ATTN && SRC != SRC_QKV_PICK && n_lo >= a.N) return;
  const int n_hi = min(a.N, n_lo + rows_per_wave);
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  const TW* __restrict__ w0 = reinterpret_cast<const TW*>(a.w0);
  const TW* __restrict__ w1 = reinterpret_cast<const TW*>(a.w1);
  const int nvec = a.Kd / VEC;                 // 16-byte vectors per weight row
  constexpr bool cached = CACHED;              // the whole input row fits in registers

  // Weights of one step: rows n0 .. n0 + NW (gate and up for SwiGLU), vectors jb + lane + 64 u.
  auto load_w = [&](WRaw<TW> (&wr)[NWV][XV], int n0, int jb) {
#pragma unroll
    for (int i = 0; i < NWV; ++i) {
      const int n = n0 + (i % NW);
#pragma unroll
      for (int u = 0; u < XV; ++u) {
        const int j = jb + lane + OSP_WAVE * u;
        if constexpr (SRC == SRC_QKV_PICK) {
          // clamped addresses, no condition: the compiler must count these loads exactly
          // for the pick's waits not to cover them (rows past n_hi are never stored;
          // columns past Kd meet zero inputs, and the clamped weights are finite)
          wr[i][u].load(w0 + (long)min(n, a.N - 1) * a.Kd + min(j, nvec - 1) * VEC);
        } else if (n < n_hi && j < nvec) {
          wr[i][u].load(((EPI == EPI_SWIGLU && i >= NW) ? w1 : w0) + (long)n * a.Kd + j * VEC);
        } else {
          wr[i][u].zero();
        }
      }
    }
  };
  // SRC_QKV_PICK: the LM head's records are requested first.  The wavefront's memory
  // counter is in order, so whatever is requested after the weights arrives no earlier
  // than they do; the pick's chain (records, then the chosen range's logits, then the
  // token's embedding row) would otherwise start only once the weights are in.
  constexpr int kPickPer = kPickMaxRecords / kGemvThreads;
  PickRecs<SRC == SRC_QKV_PICK ? kPickPer : 1> rec;
  int pk_pos = 0;   // the step's position (block 0, thread 0 writes it out at its end)
  if constexpr (SRC == SRC_QKV_PICK) {
    pick_request<kGemvThreads, kPickPer>(rec, a.pick.part, a.pick.nblk);
    pk_pos = a.pick.committed[0] + a.pick.k;
  }

  // The first step's weights do not depend on the input rows: they are requested
  // before the rows, their norm and the gains, so that those latencies overlap.
  WRaw<TW> wr[NWV][XV];
  load_w(wr, n_lo, 0);
  bool have_w = true;

  // SRC_QKV_PICK (one row, held in registers): this lane's conditioning values (row 0
  // of s) and gains do not depend on the token, so they are requested with the
  // weights, like the embedding values after the pick from clamped addresses with no
  // condition (the row's loads then wait on one another only once)
  static_assert(SRC != SRC_QKV_PICK || RB == 1, "the drawing projection takes one row");
  constexpr bool PK = SRC == SRC_QKV_PICK && CACHED;
  float xs_pk[PK ? XV : 1][VEC];
  WRaw<TW> g_pk[PK ? XV : 1];
  if constexpr (PK) {
#pragma unroll
    for (int u = 0; u < XV; ++u) {
      const int col = (lane + OSP_WAVE * u) * VEC;
      load_f4s(a.s + min(col, a.d_norm - VEC), xs_pk[u], VEC);
      g_pk[u].load(reinterpret_cast<const TW*>(a.gamma) + min(max(col - a.d_norm, 0), a.d_norm - VEC));
    }
  }

  // (nothing that reads the records may be scheduled above this point: every request
  // above is issued before the first wait)
  if constexpr (SRC == SRC_QKV_PICK) __builtin_amdgcn_sched_barrier(0);

  // SRC_QKV_PICK: the step's token, drawn by the whole block (every block draws the same
  // one); block 0 writes the draft, the next position and the row statistics out at its
  // end, after its own products
  int tok = 0;
  Pick pk_res{};
  if constexpr (SRC == SRC_QKV_PICK) {
    const PickArgs& pk = a.pick;
    pk_res = pick_draft<kGemvThreads, kPickPer>(rec, pk.nblk, pk.blk_rows, pk.logits, pk.V, pk.d2t,
                                                pk.temp[0], pk.u[0]);
    tok = pk_res.tok;
    if (n_lo >= a.N) return;
  }

  // SRC_ATTN (one row, Kd <= 8 kGemvThreads): thread t merges columns [8t, 8t + 8) of
  // head h = 8t / hd.  Split s of head h holds (max m, sum l, unnormalised output o) at
  // attn_part + (h n_split + s)(hd + 2); splits past pos / split_len hold nothing for the
  // row and are dropped by selection (their words are stale).  x = sum_s f_s o_s with
  // f_s = exp(m_s - M) / sum_s' exp(m_s' - M) l_s', M the head's largest m_s.
  __shared__ float s_x[SRC == SRC_ATTN ? 8 * kGemvThreads : 1];
  if constexpr (SRC == SRC_ATTN) {
    __shared__ float s_f[kGemvAttnMaxHeads * 2 * 16];
    const int tid = threadIdx.x;
    const int hd = a.attn_hd, nsp = a.attn_nsplit, rec = a.attn_hd + 2;
    const int c0 = 8 * tid;
    const bool seg = c0 < a.Kd;
    const int h = seg ? c0 / hd : 0;
    // every split's segment requested at once, before the row position is known
    const float* po = a.attn_part + (long)h * nsp * rec + 2 + (seg ? c0 - h * hd : 0);
    float2 ov[kGemvAttnMaxSplit][4];
#pragma unroll
    for (int sp = 0; sp < kGemvAttnMaxSplit; ++sp)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        ov[sp][q] = (seg && sp < nsp) ? *reinterpret_cast<const float2*>(po + (long)sp * rec + 2 * q)
                                      : make_float2(0.f, 0.f);
    // merge weights: 16 threads per head, splits i and i + 16
    const int hh = tid >> 4, i = tid & 15;
    const int nh = a.Kd / hd;
    const float* pm = a.attn_part + (long)hh * nsp * rec;
    float m0 = -INFINITY, l0 = 0.f, m1 = -INFINITY, l1 = 0.f;
    if (hh < nh && i < nsp) { m0 = pm[(long)i * rec]; l0 = pm[(long)i * rec + 1]; }
    if (hh < nh && i + 16 < nsp) { m1 = pm[(long)(i + 16) * rec]; l1 = pm[(long)(i + 16) * rec + 1]; }
    const int ns = min(nsp, a.attn_pos[0] / a.attn_split_len + 1);
    if (i >= ns) { m0 = -INFINITY; l0 = 0.f; }
    if (i + 16 >= ns) { m1 = -INFINITY; l1 = 0.f; }
    float M = fmaxf(m0, m1);
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) M = fmaxf(M, xor_lane_c(M, o));
    const float f0 = m0 > -INFINITY ? __expf(m0 - M) : 0.f;
    const float f1 = m1 > -INFINITY ? __expf(m1 - M) : 0.f;
    float L = l0 * f0 + l1 * f1;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) L += xor_lane_c(L, o);
    if (hh < kGemvAttnMaxHeads) {
      s_f[hh * 32 + i] = L > 0.f ? f0 / L : 0.f;
      s_f[hh * 32 + i + 16] = L > 0.f ? f1 / L : 0.f;
    }
    __syncthreads();
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = 0.f;
#pragma unroll
    for (int sp = 0; sp < kGemvAttnMaxSplit; ++sp) {
      if (sp < ns) {
        const float f = s_f[h * 32 + sp];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          x[2 * q] = fmaf(f, ov[sp][q].x, x[2 * q]);
          x[2 * q + 1] = fmaf(f, ov[sp][q].y, x[2 * q + 1]);
        }
      }
    }
    if (seg) {
      *reinterpret_cast<float4*>(s_x + c0) = make_float4(x[0], x[1], x[2], x[3]);
      *reinterpret_cast<float4*>(s_x + c0 + 4) = make_float4(x[4], x[5], x[6], x[7]);
    }
    __syncthreads();
    if (n_lo >= a.N) return;
  }

  for (int r0 = 0; r0 < rows; r0 += RB) {
    float xc[RB][XV][VEC];                     // this lane's input values (cached mode)
    float inv_rms[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) inv_rms[r] = 1.f;
    if constexpr (PK) {
      // the embedding row of the drawn token, then the RMS of that segment
      const int t = min(max(tok, 0), a.vocab_embed - 1);
      const TW* er = reinterpret_cast<const TW*>(a.embed) + (long)t * a.d_norm;
      float ev[XV][VEC];
#pragma unroll
      for (int u = 0; u < XV; ++u)   // every vector requested before any is used
        load_vec<TW>(er + min(max((lane + OSP_WAVE * u) * VEC - a.d_norm, 0), a.d_norm - VEC), ev[u]);
      bool isn[XV];
      float ss = 0.f;
#pragma unroll
      for (int u = 0; u < XV; ++u) {
        const int j = lane + OSP_WAVE * u;
        const bool live = j < nvec;
        isn[u] = live && j * VEC >= a.d_norm;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          xc[0][u][e] = !live ? 0.f : isn[u] ? ev[u][e] : xs_pk[u][e];
          ss += isn[u] ? ev[u][e] * ev[u][e] : 0.f;
        }
      }
      ss = wave_sum(ss);
      inv_rms[0] = 1.0f / sqrtf(ss / (float)a.d_norm + a.eps);
#pragma unroll
      for (int u = 0; u < XV; ++u) {
        if (isn[u]) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) xc[0][u][e] = xc[0][u][e] * inv_rms[0] * g_pk[u].get(e);
        }
        // x = embed[token] for the residual, each vector written by one wavefront
        const int jn = lane + OSP_WAVE * u - a.d_norm / VEC;
        if (a.x_out && isn[u] && jn % ((a.N + rows_per_wave - 1) / rows_per_wave) == gw) {
          float* xo = a.x_out + jn * VEC;
#pragma unroll
          for (int e = 0; e < VEC; e += 4)
            *reinterpret_cast<float4*>(xo + e) = make_float4(ev[u][e], ev[u][e + 1], ev[u][e + 2], ev[u][e + 3]);
        }
      }
    } else if constexpr (cached) {
      // gains of this lane's columns, requested with the rows
      WRaw<TW> gr[XV];
      if constexpr (NORMED) {
#pragma unroll
        for (int u = 0; u < XV; ++u) {
          const int gc = gain_col<SRC>(a, (lane + OSP_WAVE * u) * VEC);
          if (gc >= 0 && gc < a.d_norm) gr[u].load(reinterpret_cast<const TW*>(a.gamma) + gc);
          else gr[u].zero();
        }
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        bool isn[XV];
        float ss = 0.f;
#pragma unroll
        for (int u = 0; u < XV; ++u) {
          const int j = lane + OSP_WAVE * u;
          isn[u] = false;
          if (r0 + r < rows && j < nvec) {
            if constexpr (SRC == SRC_ATTN) {
#pragma unroll
              for (int e = 0; e < VEC; ++e) xc[r][u][e] = s_x[j * VEC + e];
              isn[u] = false;
            } else {
              isn[u] = load_x_raw<TW, SRC, VEC>(a, r0 + r, j * VEC, xc[r][u], tok);
            }
            if (isn[u]) {
#pragma unroll
              for (int e = 0; e < VEC; ++e) ss += xc[r][u][e] * xc[r][u][e];
            }
            if constexpr (src_qkv(SRC)) {
              // layer 0: x = embed[token] for the residual, each vector written by one
              // wavefront (the one whose index matches it modulo the working wavefronts)
              if (a.embed && a.x_out && isn[u]) {
                const int jn = j - a.d_norm / VEC;
                if (jn % ((a.N + rows_per_wave - 1) / rows_per_wave) == gw) {
                  float* xo = a.x_out + (long)(r0 + r) * a.ldx + jn * VEC;
#pragma unroll
                  for (int e = 0; e < VEC; e += 4)
                    *reinterpret_cast<float4*>(xo + e) =
                        make_float4(xc[r][u][e], xc[r][u][e + 1], xc[r][u][e + 2], xc[r][u][e + 3]);
                }
              }
            }
          } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) xc[r][u][e] = 0.f;
          }
        }
        if constexpr (NORMED) {
          ss = wave_sum(ss);
          inv_rms[r] = 1.0f / sqrtf(ss / (float)a.d_norm + a.eps);
#pragma unroll
          for (int u = 0; u < XV; ++u)
            if (isn[u]) {
#pragma unroll
              for (int e = 0; e < VEC; ++e) xc[r][u][e] = xc[r][u][e] * inv_rms[r] * gr[u].get(e);
            }
        }
      }
    } else if constexpr (NORMED) {
#pragma unroll
      for (int r = 0; r < RB; ++r)
        if (r0 + r < rows) inv_rms[r] = row_inv_rms<TW, SRC>(a, r0 + r, lane, tok);
    }
    // layer 0 of the expanded QKV (rows not held in registers): one wavefront writes
    // x = embed[token] for the residual
    if constexpr (src_qkv(SRC) && !cached) {
      if (a.embed && a.x_out && gw == 0) {
        for (int r = 0; r < RB && r0 + r < rows; ++r) {
          int t = SRC == SRC_QKV_PICK ? tok : a.tok[r0 + r];
          t = min(max(t, 0), a.vocab_embed - 1);
          const TW* e = reinterpret_cast<const TW*>(a.embed) + (long)t * a.d_norm;
          for (int c = lane; c < a.d_norm; c += OSP_WAVE)
            a.x_out[(long)(r0 + r) * a.ldx + c] = load_f32(e, c);
        }
      }
    }
    // logits: temperature of each row; running (max, sum exp, argmax) of owner lanes
    float st_m[RB], st_s[RB], temp[RB];
    int st_a[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      st_m[r] = -INFINITY;
      st_s[r] = 0.f;
      st_a[r] = 0x7fffffff;
      temp[r] = 0.f;
      if constexpr (EPI == EPI_LOGITS)
        if (r0 + r < rows) temp[r] = a.temp[a.row_seq ? a.row_seq[r0 + r] : r0 + r];
    }

    for (int n0 = n_lo; n0 < n_hi; n0 += NW) {
      const int idx = lane >> SH;
      const int vi = idx / RB, rsel = idx - vi * RB;
      const bool owner = (lane & ((1 << SH) - 1)) == 0;
      const int rr = r0 + rsel;
      const int n = n0 + vi;
      int mapped = 1;
      if constexpr (EPI == EPI_LOGITS)   // prefetch the vocabulary map of this step's rows
        mapped = (n0 + vi < n_hi) ? a.d2t[n0 + vi] : -1;
      float y_old = 0.f;                 // the residual value this lane updates, read early
      if constexpr (EPI == EPI_RESID)
        if (owner && rr < rows && n < n_hi) y_old = a.y[(long)rr * a.ldy + n];
      float acc[V];
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] = 0.f;
      for (int jb = 0; jb < nvec; jb += OSP_WAVE * XV) {
        if (!have_w) load_w(wr, n0, jb);
        have_w = false;
        if constexpr (!cached) {
#pragma unroll
          for (int r = 0; r < RB; ++r)
#pragma unroll
            for (int u = 0; u < XV; ++u) {
              const int j = jb + lane + OSP_WAVE * u;
              if (r0 + r < rows && j < nvec) {
                const bool isn = load_x_raw<TW, SRC, VEC>(a, r0 + r, j * VEC, xc[r][u], tok);
                if constexpr (NORMED)
                  if (isn) norm_x<TW, SRC, VEC>(a, j * VEC, inv_rms[r], xc[r][u]);
              } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e) xc[r][u][e] = 0.f;
              }
            }
        }
#pragma unroll
        for (int i = 0; i < NWV; ++i)
#pragma unroll
          for (int r = 0; r < RB; ++r) {
            float s = acc[i * RB + r];
#pragma unroll
            for (int u = 0; u < XV; ++u) s = wr[i][u].dot(xc[r][u], s);
            acc[i * RB + r] = s;
          }
      }
      // ---- reduce across lanes: lane l ends with value index l >> SH --------------------
      const float tot = transpose_reduce<LOGV>(acc, lane);
      if constexpr (EPI == EPI_SWIGLU) {
        // gate rows are values [0, NW), up rows [NW, 2 NW)
        // (the up value of a gate lane sits 32 lanes on: V << SH = 64, up = gate index + V / 2)
        const float up = xor_lane_c(tot, 32);
        if (owner && vi < NW && rr < rows && n < n_hi)
          a.y[(long)rr * a.ldy + n] = tot / (1.0f + __expf(-tot)) * up;
      } else if constexpr (EPI == EPI_LOGITS) {
        const bool live = owner && rr < rows && n < n_hi;
        const float lv = (live && mapped >= 0) ? tot : -INFINITY;
        if (live) a.y[(long)rr * a.ld_logits + n] = lv;
#pragma unroll
        for (int q = 0; q < RB; ++q) {
          if (q == rsel && lv > -INFINITY) {
            const float T = temp[q];
            if (lv > st_m[q]) {
              st_s[q] = (T > 0.f && st_m[q] > -INFINITY) ? st_s[q] * __expf((st_m[q] - lv) / T) : 0.f;
              st_m[q] = lv;
              st_a[q] = n;
            }
            if (T > 0.f) st_s[q] += __expf((lv - st_m[q]) / T);
          }
        }
      } else {
        if (owner && rr < rows && n < n_hi) a.y[(long)rr * a.ldy + n] = y_old + tot;
      }
    }
    if constexpr (EPI == EPI_LOGITS) {
      // merge the lanes' statistics of each row and write this wavefront's record
#pragma unroll
      for (int q = 0; q < RB; ++q) {
        const int rr = r0 + q;
        if (rr >= rows) continue;
        const float M = wave_max(st_m[q]);
        int am = (st_m[q] == M && M > -INFINITY) ? st_a[q] : 0x7fffffff;
        am = wave_min_i(am);
        const float T = temp[q];
        float s = (T > 0.f && st_m[q] > -INFINITY) ? st_s[q] * __expf((st_m[q] - M) / T) : 0.f;
        s = wave_sum(s);
        if (lane == 0) {
          float* p = a.part + ((long)rr * a.nblk + gw) * 4;
          p[0] = M;
          p[1] = s;
          p[2] = __int_as_float(am == 0x7fffffff ? -1 : am);
          p[3] = 0.f;
        }
      }
    }
  }
  if constexpr (SRC == SRC_QKV_PICK) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      const PickArgs& pk = a.pick;
      pk.draft[0] = pk_res.tok;
      if (pk.draft_out) pk.draft_out[0] = pk_res.tok;
      pk.ar_tok[0] = pk_res.tok;
      pk.ar_pos[0] = pk_pos;
      if (pk.qstat) pk.qstat[0] = QStat{pk_res.S, pk_res.M, pk_res.am};
    }
  }
}

// ---------------------------------------------------------------------------------------
// Launch shape.  RB rows per pass in {1, 2, 4, 8}; XV = 16-byte vectors per lane and
// row in one step ({1, 2, 4, 8}, RB * XV <= 8 so the cached input is <= 64 values);
// NW weight rows per step with NW * XV * RB <= 8 vectors in flight per lane (SwiGLU
// counts gate and up) so that 4 wavefronts fit per SIMD; NW shrinks further until
// the grid has enough wavefronts.
struct GemvPlan {
  int rb, xv, nw, rpw, waves;
};

inline GemvPlan gemv_plan(int wdtype, EpiKind epi, int rows, int N, int Kd) {
  GemvPlan p;
  const int vec = wdtype == 1 ? 8 : 4;
  p.rb = rows <= 1 ? 1 : rows <= 2 ? 2 : rows <= 4 ? 4 : 8;
  const int per_lane = (Kd / vec + OSP_WAVE - 1) / OSP_WAVE;
  int xv = 1;
  while (xv < per_lane && xv * 2 * p.rb <= 8) xv *= 2;
  p.xv = xv;
  const int f = epi == EPI_SWIGLU ? 2 : 1;
  int nw = 8;
  while (nw > 1 && nw * xv * p.rb * f > 8) nw /= 2;
  const int min_waves = epi == EPI_LOGITS ? 1024 : 2048;
  while (nw > 1 && (N + nw - 1) / nw < min_waves) nw /= 2;
  p.nw = nw;
  int rpw = (N + kGemvMaxWaves - 1) / kGemvMaxWaves;
  rpw = (rpw + nw - 1) / nw * nw;
  p.rpw = rpw < nw ? nw : rpw;
  p.waves = (N + p.rpw - 1) / p.rpw;
  return p;
}

template <typename TW, int SRC, int EPI, int RB, int NW, int XV>
void launch_gemv_t(const GemvArgs& a, int rpw, hipStream_t st) {
  const int waves = (a.N + rpw - 1) / rpw;
  const int grid = (waves + kGemvWavesPerBlock - 1) / kGemvWavesPerBlock;
  const bool cached = a.Kd / Vec<TW>::N <= OSP_WAVE * XV;
  if constexpr (SRC == SRC_ATTN) {
    // (only the cached form exists: gemv_attn_supported bounds Kd)
    hipLaunchKernelGGL((k_gemv<TW, SRC, EPI, RB, NW, XV, true>), dim3(grid), dim3(kGemvThreads), 0, st, a, rpw);
  } else {
    if (cached)
      hipLaunchKernelGGL((k_gemv<TW, SRC, EPI, RB, NW, XV, true>), dim3(grid), dim3(kGemvThreads), 0,
                         st, a, rpw);
    else
      hipLaunchKernelGGL((k_gemv<TW, SRC, EPI, RB, NW, XV, false>), dim3(grid), dim3(kGemvThreads), 0,
                         st, a, rpw);
  }
}

template <typename TW, int SRC, int EPI, int RB, int XV>
void launch_gemv_nw(const GemvPlan& p, const GemvArgs& a, hipStream_t st) {
  constexpr int F = (EPI == EPI_SWIGLU) ? 2 : 1;
  if constexpr (8 * XV * RB * F <= 8) { if (p.nw == 8) return launch_gemv_t<TW, SRC, EPI, RB, 8, XV>(a, p.rpw, st); }
  if constexpr (4 * XV * RB * F <= 8) { if (p.nw == 4) return launch_gemv_t<TW, SRC, EPI, RB, 4, XV>(a, p.rpw, st); }
  if constexpr (2 * XV * RB * F <= 8) { if (p.nw == 2) return launch_gemv_t<TW, SRC, EPI, RB, 2, XV>(a, p.rpw, st); }
  return launch_gemv_t<TW, SRC, EPI, RB, 1, XV>(a, p.rpw, st);
}

template <typename TW, int SRC, int EPI, int RB>
void launch_gemv_xv(const GemvPlan& p, const GemvArgs& a, hipStream_t st) {
  if constexpr (RB * 8 <= 8) { if (p.xv == 8) return launch_gemv_nw<TW, SRC, EPI, RB, 8>(p, a, st); }
  if constexpr (RB * 4 <= 8) { if (p.xv == 4) return launch_gemv_nw<TW, SRC, EPI, RB, 4>(p, a, st); }
  if constexpr (RB * 2 <= 8) { if (p.xv == 2) return launch_gemv_nw<TW, SRC, EPI, RB, 2>(p, a, st); }
  return launch_gemv_nw<TW, SRC, EPI, RB, 1>(p, a, st);
}

template <int SRC, int EPI>
void launch_gemv_kind(int wdtype, const GemvArgs& a, hipStream_t st) {
  const GemvPlan p = gemv_plan(wdtype, (EpiKind)EPI, a.max_rows, a.N, a.Kd);
  if (wdtype == 1) {
    switch (p.rb) {
      case 1: return launch_gemv_xv<bf16_t, SRC, EPI, 1>(p, a, st);
      case 2: return launch_gemv_xv<bf16_t, SRC, EPI, 2>(p, a, st);
      case 4: return launch_gemv_xv<bf16_t, SRC, EPI, 4>(p, a, st);
      default: return launch_gemv_xv<bf16_t, SRC, EPI, 8>(p, a, st);
    }
  } else {
    switch (p.rb) {
      case 1: return launch_gemv_xv<float, SRC, EPI, 1>(p, a, st);
      case 2: return launch_gemv_xv<float, SRC, EPI, 2>(p, a, st);
      case 4: return launch_gemv_xv<float, SRC, EPI, 4>(p, a, st);
      default: return launch_gemv_xv<float, SRC, EPI, 8>(p, a, st);
    }
  }
}

}  // namespace osp

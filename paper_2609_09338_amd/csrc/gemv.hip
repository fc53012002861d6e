// Weight-streaming matrix-vector products of the drafter (few rows at a time).
//
// Y[r][n] = sum_c X[r][c] * W[n][c] for the rows r of one forward pass.  Every
// weight byte is read from HBM once per pass (per block of RB rows); the input
// rows are staged in LDS one column chunk at a time and each lane keeps the 64
// input values it needs in registers.  A wavefront owns NW weight rows; lane l
// reads 16-byte vectors l, l+64, ... of a row (fully coalesced), and the NW*RB
// partial sums are reduced across the 64 lanes with one transposed butterfly.
//
// The virtual input X is formed on the fly (the norm prologues of the body):
//   SRC_PLAIN  fp32 rows (attention output, FFN hidden)
//   SRC_NORM   RMSNorm(x) * gain (post-attention norm, final norm)
//   SRC_QKV    [s ; RMSNorm(x) * gain] -- the expanded-QKV input of Eq. 2-3, read
//              from its two segments with no concatenated copy; in layer 0 x is
//              the embedding row of the token and block 0 materialises it
//   SRC_TAPS   target hidden-state taps (Eq. 1)
// and the epilogue writes, accumulates into the residual, applies SwiGLU, or
// writes masked logits plus per-block softmax statistics for sampling.
#include "common.h"
#include "internal.h"

namespace osp {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / OSP_WAVE;

template <int N> struct Log2 { static constexpr int v = 1 + Log2<N / 2>::v; };
template <> struct Log2<1> { static constexpr int v = 0; };

template <typename TW, int SRC, int EPI, int RB, int NW>
__global__ void __launch_bounds__(kThreads) k_gemv(GemvArgs a) {
  constexpr int VEC = Vec<TW>::N;
  constexpr int KC = 4096 / RB;               // input columns staged per chunk
  constexpr int PER_LANE = KC / OSP_WAVE;      // input values per lane per row (64 / RB)
  constexpr int JV = PER_LANE / VEC;           // 16-byte weight vectors per lane per row
  constexpr int NWV = (EPI == EPI_SWIGLU) ? 2 * NW : NW;
  constexpr int V = NWV * RB;
  constexpr int LOGV = Log2<V>::v;
  constexpr int TN = kWaves * NW;              // weight rows (outputs) per block
  static_assert((1 << LOGV) == V && V <= 64, "values per lane must be a power of two <= 64");
  static_assert(JV >= 1, "chunk too small");

  __shared__ float xs[RB * KC];
  __shared__ float inv_rms[RB];
  __shared__ float lg[(EPI == EPI_LOGITS) ? RB * TN : 1];

  const int tid = threadIdx.x;
  const int lane = tid & (OSP_WAVE - 1);
  const int wave = tid >> 6;
  const int n_base = blockIdx.x * TN + wave * NW;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  const TW* __restrict__ w0 = reinterpret_cast<const TW*>(a.w0);
  const TW* __restrict__ w1 = reinterpret_cast<const TW*>(a.w1);
  const TW* __restrict__ gamma = reinterpret_cast<const TW*>(a.gamma);
  const int d = a.d_norm;

  for (int r0 = 0; r0 < rows; r0 += RB) {
    // ---- per-row prologue: RMS of the normalised segment -------------------------
    if constexpr (SRC == SRC_NORM || SRC == SRC_QKV) {
      for (int r = wave; r < RB; r += kWaves) {
        const int rr = r0 + r;
        float ss = 0.f;
        if (rr < rows) {
          if constexpr (SRC == SRC_QKV) {
            if (a.embed) {
              int t = a.tok[rr];
              t = min(max(t, 0), a.vocab_embed - 1);
              const TW* e = reinterpret_cast<const TW*>(a.embed) + (long)t * d;
              for (int c = lane; c < d; c += OSP_WAVE) { float v = load_f32(e, c); ss += v * v; }
            } else {
              const int xr = a.gather ? a.gather[rr] : rr;
              const float* xp = a.xin + (long)xr * a.ldx;
              for (int c = lane; c < d; c += OSP_WAVE) { float v = xp[c]; ss += v * v; }
            }
          } else {
            const int xr = a.gather ? a.gather[rr] : rr;
            const float* xp = a.xin + (long)xr * a.ldx;
            for (int c = lane; c < d; c += OSP_WAVE) { float v = xp[c]; ss += v * v; }
          }
        }
        ss = wave_sum(ss);
        if (lane == 0) inv_rms[r] = 1.0f / sqrtf(ss / (float)d + a.eps);
      }
      __syncthreads();
    }

    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;

    for (int k0 = 0; k0 < a.Kd; k0 += KC) {
      const int kc = min(KC, a.Kd - k0);
      // ---- stage X[r0 .. r0+RB)[k0 .. k0+kc) into LDS --------------------------------
      for (int i = tid; i < RB * KC; i += kThreads) {
        const int r = i / KC, c = i - r * KC;
        const int rr = r0 + r, col = k0 + c;
        float v = 0.f;
        if (rr < rows && c < kc) {
          if constexpr (SRC == SRC_PLAIN) {
            v = a.xin[(long)rr * a.ldx + col];
          } else if constexpr (SRC == SRC_NORM) {
            const int xr = a.gather ? a.gather[rr] : rr;
            v = a.xin[(long)xr * a.ldx + col] * inv_rms[r] * load_f32(gamma, col);
          } else if constexpr (SRC == SRC_TAPS) {
            const TW* tp = reinterpret_cast<const TW*>(a.taps);
            v = load_f32(tp, (long)a.tap_row[rr] * a.ldt + col);
          } else {  // SRC_QKV
            if (col < d) {
              const int sr = a.s_gather ? a.s_gather[rr] : rr;
              v = a.s[(long)sr * a.lds + col];
            } else {
              const int cc = col - d;
              float xv;
              if (a.embed) {
                int t = a.tok[rr];
                t = min(max(t, 0), a.vocab_embed - 1);
                xv = load_f32(reinterpret_cast<const TW*>(a.embed), (long)t * d + cc);
                if (blockIdx.x == 0 && a.x_out) a.x_out[(long)rr * a.ldx + cc] = xv;
              } else {
                const int xr = a.gather ? a.gather[rr] : rr;
                xv = a.xin[(long)xr * a.ldx + cc];
              }
              v = xv * inv_rms[r] * load_f32(gamma, cc);
            }
          }
        }
        xs[i] = v;
      }
      __syncthreads();
      // ---- this lane's input values ----------------------------------------------------
      float xr[RB][PER_LANE];
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int j = 0; j < JV; ++j)
#pragma unroll
          for (int e = 0; e < VEC; ++e) xr[r][j * VEC + e] = xs[r * KC + (j * OSP_WAVE + lane) * VEC + e];
      __syncthreads();
      // ---- stream the weight rows ------------------------------------------------------
#pragma unroll
      for (int i = 0; i < NWV; ++i) {
        const int n = n_base + (i % NW);
        if (n >= a.N) continue;
        const TW* wrow = ((EPI == EPI_SWIGLU && i >= NW) ? w1 : w0) + (long)n * a.Kd + k0;
#pragma unroll
        for (int j = 0; j < JV; ++j) {
          const int c = (j * OSP_WAVE + lane) * VEC;
          if (c < kc) {
            float wv[VEC];
            load_vec<TW>(wrow + c, wv);
#pragma unroll
            for (int r = 0; r < RB; ++r) {
              float s = acc[i * RB + r];
#pragma unroll
              for (int e = 0; e < VEC; ++e) s = fmaf(wv[e], xr[r][j * VEC + e], s);
              acc[i * RB + r] = s;
            }
          }
        }
      }
    }

    // ---- reduce across lanes: lane l ends with value index l >> (6 - LOGV) ------------
    const float tot = transpose_reduce<LOGV>(acc, lane);
    const int idx = lane >> (6 - LOGV);
    const bool owner = (lane & ((1 << (6 - LOGV)) - 1)) == 0;
    const int vi = idx / RB, r = idx - vi * RB;
    const int rr = r0 + r;

    if constexpr (EPI == EPI_SWIGLU) {
      // gate rows are value rows [0, NW), up rows [NW, 2 NW)
      const int up_lane = ((vi + NW) * RB + r) << (6 - LOGV);
      const float up = __shfl(tot, up_lane < OSP_WAVE ? up_lane : 0, OSP_WAVE);
      const int n = n_base + vi;
      if (owner && vi < NW && rr < rows && n < a.N) {
        const float g = tot;
        a.y[(long)rr * a.ldy + n] = g / (1.0f + __expf(-g)) * up;
      }
    } else if constexpr (EPI == EPI_LOGITS) {
      const int n_local = wave * NW + vi;
      const int n = n_base + vi;
      float lv = -INFINITY;
      if (n < a.N && a.d2t[n] >= 0) lv = tot;
      if (owner) {
        lg[r * TN + n_local] = lv;
        if (rr < rows && n < a.N) a.y[(long)rr * a.ld_logits + n] = lv;
      }
      __syncthreads();
      // per-row statistics of this block's TN logits: max, lowest argmax, sum exp((l-max)/T)
      for (int r2 = wave; r2 < RB; r2 += kWaves) {
        const int rr2 = r0 + r2;
        if (rr2 >= rows) continue;
        float m = -INFINITY;
        int am = 0x7fffffff;
        for (int t = lane; t < TN; t += OSP_WAVE) {
          const float v = lg[r2 * TN + t];
          if (v > m) { m = v; am = t; }
        }
        const float mw = wave_max(m);
        int cand = (m == mw && m > -INFINITY) ? am : 0x7fffffff;
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) cand = min(cand, __shfl_xor(cand, s, OSP_WAVE));
        const int b = a.row_seq ? a.row_seq[rr2] : rr2;
        const float T = a.temp[b];
        float se = 0.f;
        if (T > 0.f && mw > -INFINITY)
          for (int t = lane; t < TN; t += OSP_WAVE) se += __expf((lg[r2 * TN + t] - mw) / T);
        se = wave_sum(se);
        if (lane == 0) {
          float* p = a.part + ((long)rr2 * a.nblk + blockIdx.x) * 4;
          p[0] = mw;
          p[1] = se;
          p[2] = __int_as_float(cand == 0x7fffffff ? -1 : blockIdx.x * TN + cand);
          p[3] = 0.f;
        }
      }
      __syncthreads();
    } else {
      const int n = n_base + vi;
      if (owner && rr < rows && n < a.N) {
        float* yp = a.y + (long)rr * a.ldy + n;
        if constexpr (EPI == EPI_RESID) *yp += tot; else *yp = tot;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------------------
// Launch-shape selection: rows per pass RB in {1, 2, 4, 8}; weight rows per wave NW in
// {1, 4, 16} (fewer for small N so that the grid still covers the chip).
static int pick_rb(int rows) { return rows <= 1 ? 1 : rows <= 2 ? 2 : rows <= 4 ? 4 : 8; }

static int pick_nw(EpiKind epi, int rb, int N) {
  const int vmax = 64 / (rb * (epi == EPI_SWIGLU ? 2 : 1));
  int nw = 16;
  while (nw > vmax) nw /= 4;
  if (epi == EPI_LOGITS) return nw;            // large N: many blocks regardless
  while (nw > 1 && (N + kWaves * nw - 1) / (kWaves * nw) < 512) nw /= 4;
  return nw;
}

int gemv_rows_per_block(int /*wdtype*/, EpiKind epi, int rows) {
  const int rb = pick_rb(rows);
  // only the logits epilogue needs the block size (for the statistics layout)
  return kWaves * pick_nw(epi, rb, 1 << 30);
}

template <typename TW, int SRC, int EPI, int RB, int NW>
static void launch_t(const GemvArgs& a, hipStream_t st) {
  constexpr int TN = kWaves * NW;
  const int grid = (a.N + TN - 1) / TN;
  hipLaunchKernelGGL((k_gemv<TW, SRC, EPI, RB, NW>), dim3(grid), dim3(kThreads), 0, st, a);
}

template <typename TW, int SRC, int EPI, int RB>
static void launch_nw(int nw, const GemvArgs& a, hipStream_t st) {
  constexpr int F = (EPI == EPI_SWIGLU) ? 2 : 1;
  if constexpr (16 * RB * F <= 64) { if (nw == 16) return launch_t<TW, SRC, EPI, RB, 16>(a, st); }
  if constexpr (4 * RB * F <= 64) { if (nw == 4) return launch_t<TW, SRC, EPI, RB, 4>(a, st); }
  return launch_t<TW, SRC, EPI, RB, 1>(a, st);
}

template <typename TW, int SRC, int EPI>
static void launch_rb(const GemvArgs& a, hipStream_t st) {
  const int rb = pick_rb(a.max_rows);
  const int nw = pick_nw((EpiKind)EPI, rb, a.N);
  switch (rb) {
    case 1: return launch_nw<TW, SRC, EPI, 1>(nw, a, st);
    case 2: return launch_nw<TW, SRC, EPI, 2>(nw, a, st);
    case 4: return launch_nw<TW, SRC, EPI, 4>(nw, a, st);
    default: return launch_nw<TW, SRC, EPI, 8>(nw, a, st);
  }
}

template <typename TW>
static void launch_kind(SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st) {
  if (src == SRC_TAPS && epi == EPI_STORE) return launch_rb<TW, SRC_TAPS, EPI_STORE>(a, st);
  if (src == SRC_QKV && epi == EPI_STORE) return launch_rb<TW, SRC_QKV, EPI_STORE>(a, st);
  if (src == SRC_PLAIN && epi == EPI_RESID) return launch_rb<TW, SRC_PLAIN, EPI_RESID>(a, st);
  if (src == SRC_NORM && epi == EPI_SWIGLU) return launch_rb<TW, SRC_NORM, EPI_SWIGLU>(a, st);
  if (src == SRC_NORM && epi == EPI_LOGITS) return launch_rb<TW, SRC_NORM, EPI_LOGITS>(a, st);
}

void launch_gemv(int wdtype, SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st) {
  if (wdtype == 1) launch_kind<bf16_t>(src, epi, a, st);
  else launch_kind<float>(src, epi, a, st);
}

}  // namespace osp

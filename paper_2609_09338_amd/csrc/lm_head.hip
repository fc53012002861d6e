// Vocabulary-aligned LM head on the matrix cores (Section 3.3, Eq. 4: the head's
// rows are indexed by the drafter vocabulary and mapped to target ids through
// d2t; rows without a target id are masked).
//
//   logits[r][n] = RMSNorm_final(x_r) . W_head[n]      (n mapped by d2t, else -inf)
//
// plus, for every wavefront's contiguous range of vocabulary rows, a softmax
// record (max, sum exp((l - max) / T), lowest argmax) per input row, which the
// sampling kernel merges.
//
// One block per CU (8 wavefronts).  The block copies the inputs (RMSNorm output as
// bf16 hi / lo pairs, all R <= 16 MT rows, KC columns per phase; either prepared by
// the row kernels or normalised here from the fp32 rows) into LDS once per phase; after that every wavefront works alone, with no further
// block barrier: it streams its T tiles of 16 weight rows in units of 16 rows x
// 256 columns (8 KB) through a ring of three register buffers (two units in
// flight while it multiplies the third), each unit feeding 8 K steps of
// v_mfma_f32_16x16x32_bf16 for every M tile, hi and lo.  A wavefront's T tiles
// are consecutive vocabulary rows, so its record covers 16 T consecutive logits.
//
// HBM traffic: the weights once (N x K bf16) plus the logits (R x N fp32); the
// inputs come from L2 (R x K x 4 bytes per block and phase).
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace osp {

typedef __bf16 lm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float lm_f32x4 __attribute__((ext_vector_type(4)));

constexpr int kLmWaves = 8;
constexpr int kLmThreads = kLmWaves * 64;
constexpr int kLmUnit = 256;              // weight columns per streamed unit
constexpr int kLmDepth = 3;               // register ring of units

// Input columns resident per phase and tiles per wavefront: 8 wavefronts x 5 tiles
// x 16 rows per CU cover a 152k vocabulary on 256 CUs in one wave of blocks (the
// register budget, 2 wavefronts per SIMD, allows one block per CU).
template <int MT> struct LmCfg { static constexpr int KC = MT == 4 ? 512 : 1024, TMAX = 5; };

// NORM: the inputs are the fp32 rows xin (gathered), normalised here (RMSNorm with
// gain gamma) while they are staged; otherwise they arrive prepared as bf16 pairs.
template <int MT, bool NORM>
__global__ void __launch_bounds__(kLmThreads) k_lm_head(GemvArgs a, int T) {
  constexpr int KC = LmCfg<MT>::KC;       // input columns resident per phase
  constexpr int TMAX = LmCfg<MT>::TMAX;   // tiles per wavefront (bound)
  constexpr int ROWS = 16 * MT;
  constexpr int PITCH = KC + 8;           // bf16 per LDS row (16-byte skew per row)
  constexpr int NCH = KC / kLmUnit;       // units per tile and phase
  constexpr int NU = TMAX * NCH;          // units per phase (bound)
  __shared__ __attribute__((aligned(16))) bf16_t xh[ROWS * PITCH];
  __shared__ __attribute__((aligned(16))) bf16_t xl[ROWS * PITCH];
  __shared__ float s_inv[NORM ? ROWS : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wrow = lane & 15, grp = lane >> 4;
  const int R = min(a.max_rows, ROWS);
  const int wg = blockIdx.x * kLmWaves + wave;          // record index
  const int nt16 = (a.N + 15) >> 4;
  const int t0 = wg * T;
  const int ntiles = max(0, min(T, nt16 - t0));
  const bf16_t* __restrict__ W = reinterpret_cast<const bf16_t*>(a.w0);

  lm_f32x4 acc[TMAX][MT];
#pragma unroll
  for (int j = 0; j < TMAX; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = lm_f32x4{0.f, 0.f, 0.f, 0.f};

  // Addresses are clamped into the matrix instead of masking the loaded values: a
  // select on a loaded register would wait for that load and serialise the ring.
  // Rows past N only produce logits that the epilogue drops; columns past Kd meet
  // zero inputs in LDS (the clamped weights are finite).
  auto load_unit = [&](uint4* w, int k0, int u) {
    const int n = min((t0 + u / NCH) * 16 + wrow, a.N - 1);
    const int kb = k0 + (u % NCH) * kLmUnit + 8 * grp;
    const bf16_t* wr = W + (long)n * a.Kd;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      w[ks] = *reinterpret_cast<const uint4*>(wr + min(kb + 32 * ks, a.Kd - 8));
  };
  const int nphase = (a.Kd + KC - 1) / KC;
  const int nu = ntiles * NCH;                          // units per phase
  uint4 ring[kLmDepth][8];
  // the first units of a phase are requested before its inputs are staged
  auto prefetch_phase = [&](int k0) {
#pragma unroll
    for (int u = 0; u + 1 < kLmDepth; ++u)
      if (u < nu) load_unit(ring[u], k0, u);
  };
  prefetch_phase(0);
  if constexpr (NORM) {
    // RMS of every input row (one wavefront per row)
    for (int r = wave; r < R; r += kLmWaves) {
      const float* xr = a.xin + (long)(a.gather ? a.gather[r] : r) * a.ldx;
      float ss = 0.f;
      for (int c = lane * 4; c < a.Kd; c += 64 * 4) {
        const float4 v = *reinterpret_cast<const float4*>(xr + c);
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
      ss = wave_sum(ss);
      if (lane == 0) s_inv[r] = 1.0f / sqrtf(ss / (float)a.Kd + a.eps);
    }
    __syncthreads();
  }
  for (int ph = 0; ph < nphase; ++ph) {
    const int k0 = ph * KC;
    if (ph > 0) __syncthreads();
    // ---- inputs of this phase into LDS (rows past R and columns past Kd are zero) ----
    for (int i = tid; i < ROWS * (KC / 8); i += kLmThreads) {
      const int r = i / (KC / 8), col = (i - r * (KC / 8)) * 8;
      uint4 h = make_uint4(0u, 0u, 0u, 0u), l = h;
      if (r < R && k0 + col < a.Kd) {
        if constexpr (NORM) {
          const float* xr = a.xin + (long)(a.gather ? a.gather[r] : r) * a.ldx + k0 + col;
          const float4 v0 = *reinterpret_cast<const float4*>(xr);
          const float4 v1 = *reinterpret_cast<const float4*>(xr + 4);
          const uint4 g = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16_t*>(a.gamma) + k0 + col);
          const float inv = s_inv[r];
          split_bf16x2(v0.x * inv * bf16_lo(g.x), v0.y * inv * bf16_hi(g.x), h.x, l.x);
          split_bf16x2(v0.z * inv * bf16_lo(g.y), v0.w * inv * bf16_hi(g.y), h.y, l.y);
          split_bf16x2(v1.x * inv * bf16_lo(g.z), v1.y * inv * bf16_hi(g.z), h.z, l.z);
          split_bf16x2(v1.z * inv * bf16_lo(g.w), v1.w * inv * bf16_hi(g.w), h.w, l.w);
        } else {
          const long o = (long)(a.gather ? a.gather[r] : r) * a.ld_xa + k0 + col;
          h = *reinterpret_cast<const uint4*>(a.xa_hi + o);
          l = *reinterpret_cast<const uint4*>(a.xa_lo + o);
        }
      }
      *reinterpret_cast<uint4*>(xh + r * PITCH + col) = h;
      *reinterpret_cast<uint4*>(xl + r * PITCH + col) = l;
    }
    __syncthreads();

    // ---- stream this wavefront's units: tile j = u / NCH, columns (u % NCH) * 256 ----
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      if (u < nu) {
        if (u + kLmDepth - 1 < nu) load_unit(ring[(u + kLmDepth - 1) % kLmDepth], k0, u + kLmDepth - 1);
        // keep each unit's work in place: hoisting later units' LDS reads or loads
        // above this point only raises register pressure
        __builtin_amdgcn_sched_barrier(0);
        const uint4* w = ring[u % kLmDepth];
        const int j = u / NCH;
        const int kl = (u % NCH) * kLmUnit + 8 * grp;   // column within the phase
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const lm_bf16x8 bw = *reinterpret_cast<const lm_bf16x8*>(&w[ks]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int off = (mt * 16 + wrow) * PITCH + kl + 32 * ks;
            const lm_bf16x8 ah = *reinterpret_cast<const lm_bf16x8*>(xh + off);
            const lm_bf16x8 al = *reinterpret_cast<const lm_bf16x8*>(xl + off);
            acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw, acc[j][mt], 0, 0, 0);
            acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw, acc[j][mt], 0, 0, 0);
          }
        }
      }
    }
    if (ph + 1 < nphase) prefetch_phase(k0 + KC);
  }
  if (ntiles == 0) return;

  // ---- epilogue: lane holds logits of rows 16 mt + 4 grp + e, columns tile + wrow -------
  float mx[MT][4];
  int am[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 4; ++e) { mx[mt][e] = -INFINITY; am[mt][e] = 0x7fffffff; }
#pragma unroll
  for (int j = 0; j < TMAX; ++j) {
    if (j < ntiles) {
      const int n = (t0 + j) * 16 + wrow;
      const bool live = n < a.N && a.d2t[n] >= 0;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * grp + e;
          const float lv = live ? acc[j][mt][e] : -INFINITY;
          acc[j][mt][e] = lv;
          if (m < R && n < a.N) a.y[(long)m * a.ld_logits + n] = lv;
          if (lv > mx[mt][e]) { mx[mt][e] = lv; am[mt][e] = n; }
        }
    }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float M = mx[mt][e];
      int A = am[mt][e];
#pragma unroll
      for (int s = 1; s < 16; s <<= 1) {
        const float om = __shfl_xor(M, s, OSP_WAVE);
        const int oa = __shfl_xor(A, s, OSP_WAVE);
        if (om > M || (om == M && oa < A)) { M = om; A = oa; }
      }
      mx[mt][e] = M;
      am[mt][e] = A;
    }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = mt * 16 + 4 * grp + e;
      const float Tm = m < R ? a.temp[a.row_seq ? a.row_seq[m] : m] : 0.f;
      float s = 0.f;
      if (Tm > 0.f && mx[mt][e] > -INFINITY) {
#pragma unroll
        for (int j = 0; j < TMAX; ++j)
          if (j < ntiles && acc[j][mt][e] > -INFINITY) s += __expf((acc[j][mt][e] - mx[mt][e]) / Tm);
      }
#pragma unroll
      for (int sft = 1; sft < 16; sft <<= 1) s += __shfl_xor(s, sft, OSP_WAVE);
      if (wrow == 0 && m < R) {
        float* p = a.part + ((long)m * a.nblk + wg) * 4;
        p[0] = mx[mt][e];
        p[1] = s;
        p[2] = __int_as_float(mx[mt][e] > -INFINITY ? am[mt][e] : -1);
        p[3] = 0.f;
      }
    }
}

LmPlan lm_head_plan(int rows, int N, int n_cu) {
  LmPlan p;
  p.mt = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
  const int tmax = LmCfg<1>::TMAX;
  const int nt16 = (N + 15) / 16;
  p.grid = std::min(n_cu, kGemvMaxWaves / kLmWaves);
  p.T = (nt16 + p.grid * kLmWaves - 1) / (p.grid * kLmWaves);
  if (p.T > tmax) {
    p.T = tmax;
    p.grid = (nt16 + tmax * kLmWaves - 1) / (tmax * kLmWaves);
  }
  p.nblk = (nt16 + p.T - 1) / p.T;
  p.blk_rows = 16 * p.T;
  return p;
}

void launch_lm_head(const GemvArgs& a, const LmPlan& p, bool norm_in, hipStream_t st) {
  const dim3 g(p.grid), b(kLmThreads);
  if (norm_in) {
    if (p.mt == 1) hipLaunchKernelGGL((k_lm_head<1, true>), g, b, 0, st, a, p.T);
    else if (p.mt == 2) hipLaunchKernelGGL((k_lm_head<2, true>), g, b, 0, st, a, p.T);
    else hipLaunchKernelGGL((k_lm_head<4, true>), g, b, 0, st, a, p.T);
  } else {
    if (p.mt == 1) hipLaunchKernelGGL((k_lm_head<1, false>), g, b, 0, st, a, p.T);
    else if (p.mt == 2) hipLaunchKernelGGL((k_lm_head<2, false>), g, b, 0, st, a, p.T);
    else hipLaunchKernelGGL((k_lm_head<4, false>), g, b, 0, st, a, p.T);
  }
}

}  // namespace osp

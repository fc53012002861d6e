// Skinny GEMM on the matrix cores for passes with several rows (ingest, batch > 1).
//
// Y[r][n] = sum_c X[r][c] * W[n][c] with bf16 weights, for R rows (up to 64 per
// pass; more rows loop).  v_mfma_f32_16x16x32_bf16 computes a 16 x 16 tile per
// 32-wide K step; the weight tile is the B operand, read straight from the
// row-major weights: lane l loads 16 bytes of weight row (l % 16) at column
// offset 8 (l / 16), so four lanes cover 64 contiguous bytes of a row.  Every
// weight byte is read once per 64 rows.
//
// The input rows are formed exactly as in the GEMV kinds (conditioning segment,
// RMSNorm prologue, embedding for layer 0, taps) and staged in LDS as a pair of
// bf16 values per element, hi = bf16(x) and lo = bf16(x - hi); two MFMAs (hi and
// lo) keep about 16 significant bits of every activation, so the products stay
// close to fp32 (weights are exact bf16; accumulation is fp32).  Taps are bf16
// already and use the hi part only.
//
// Inputs arrive prepared: the row kernels that precede each product (norms,
// residual, SwiGLU, attention combine) write every input element once as bf16
// hi / lo pairs, so a block only copies its input chunk into LDS.  The
// expanded-QKV input [c ; RMSNorm(x)] of Eq. 2-3 is read from its two segments.
//
// This kernel serves passes of more than 64 rows (ingest of large batches); it
// covers them in 64-row passes spread over blockIdx.z.  Block: 8 wavefronts with
// two 16-row weight tiles each (SwiGLU: a gate tile and its up tile) sharing one
// staged input chunk of 256 columns, so one chunk serves 256 (SwiGLU 128) output
// columns.  K is split across blocks (a block walks its chunks one after another);
// every block writes its partial sums to [split][row][N] (SwiGLU: gate then up, 2 N
// wide) and the row kernel that follows adds the splits in a fixed order.  The
// logits kind (never split) writes masked logits and one (max, sum exp((l - max)/T),
// lowest argmax) record per block of consecutive rows.
#pragma once

#include "common.h"
#include "internal.h"

namespace osp {

typedef __bf16 mfma_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

constexpr int kMmRows = 64;          // input rows per pass (4 M tiles)
constexpr int kMmKc = 256;           // K columns per chunk
constexpr int kMmPitch = kMmKc + 16;  // LDS row pitch in bf16: a 32-byte skew per row (16 bytes left bank conflicts)

// Block shape: 8 wavefronts, two weight tiles each.
template <int EPI> struct MmShape {
  static constexpr int WAVES = 8;
  static constexpr int WT = 2;
  static constexpr int NT = EPI == EPI_SWIGLU ? 1 : WT;   // output tiles per wavefront
  static constexpr int THREADS = WAVES * 64;
  static constexpr int ROWS = WAVES * NT * 16;            // output rows per block
};

template <int SRC, int EPI>
__global__ void __launch_bounds__(MmShape<EPI>::THREADS) k_gemm_mfma(GemvArgs a, int chunks_per_split) {
  constexpr bool EXACT_X = (SRC == SRC_TAPS);          // inputs already bf16: no lo part
  constexpr int kMmWaves = MmShape<EPI>::WAVES;
  constexpr int kMmThreads = MmShape<EPI>::THREADS;
  constexpr int kMmWT = MmShape<EPI>::WT;
  constexpr int NT = MmShape<EPI>::NT;
  __shared__ __attribute__((aligned(16))) bf16_t xs_hi[kMmRows * kMmPitch];
  __shared__ __attribute__((aligned(16))) bf16_t xs_lo[EXACT_X ? 8 : kMmRows * kMmPitch];
  constexpr int SW = EPI == EPI_LOGITS ? kMmWaves : 1;
  __shared__ float s_m[SW][kMmRows];
  __shared__ float s_s[SW][kMmRows];
  __shared__ int s_a[SW][kMmRows];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  const bf16_t* __restrict__ w0 = reinterpret_cast<const bf16_t*>(a.w0);
  const bf16_t* __restrict__ w1 = reinterpret_cast<const bf16_t*>(a.w1);
  const int rows_per_block = kMmWaves * NT * 16;
  const int nb0 = blockIdx.x * rows_per_block;          // first output row of the block
  const int nw0 = nb0 + wave * NT * 16;                 // first output row of this wavefront
  const int wrow = lane & 15, kg = lane >> 4;           // B operand: weight row, 8-column group
  const int k_begin = blockIdx.y * chunks_per_split * kMmKc;
  const int k_end = min(a.Kd, k_begin + chunks_per_split * kMmKc);

  // passes of 64 rows are spread over blockIdx.z (each block: one pass)
  for (int r0 = blockIdx.z * kMmRows; r0 < rows && r0 < (int)(blockIdx.z + 1) * kMmRows; r0 += kMmRows) {
    const int rcount = min(kMmRows, rows - r0);
    const int mt_n = (rcount + 15) >> 4;                // M tiles in use
    mfma_f32x4 acc[4][kMmWT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int wt = 0; wt < kMmWT; ++wt) acc[mt][wt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = k_begin; k0 < k_end; k0 += kMmKc) {
      // ---- request this chunk's weights (8 K steps x kMmWT tiles) ----------------------
      uint4 wb[kMmWT][kMmKc / 32];
#pragma unroll
      for (int wt = 0; wt < kMmWT; ++wt) {
        const int n = (EPI == EPI_SWIGLU) ? nw0 + wrow : nw0 + wt * 16 + wrow;
        const bf16_t* base = (EPI == EPI_SWIGLU && wt == 1) ? w1 : w0;
#pragma unroll
        for (int t = 0; t < kMmKc / 32; ++t) {
          const int col = k0 + 32 * t + 8 * kg;
          if (n < a.N && col < a.Kd)
            wb[wt][t] = *reinterpret_cast<const uint4*>(base + (long)n * a.Kd + col);
          else
            wb[wt][t] = make_uint4(0u, 0u, 0u, 0u);
        }
      }
      // ---- stage the input chunk (bf16 hi / lo, 16-byte copies) ---------------------------
      for (int i = tid; i < kMmRows * (kMmKc / 8); i += kMmThreads) {
        const int r = i / (kMmKc / 8), cv = i - r * (kMmKc / 8);
        const int col = k0 + cv * 8;
        uint4 ph = make_uint4(0u, 0u, 0u, 0u), pl = ph;
        if (r < rcount && col < a.Kd) {
          const int rr = r0 + r;
          if constexpr (SRC == SRC_TAPS) {
            ph = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16_t*>(a.taps) +
                                                 (long)a.tap_row[rr] * a.ldt + col);
          } else if (col < a.seg) {
            const long o = (long)rr * a.ld_xs + col;
            ph = *reinterpret_cast<const uint4*>(a.xs_hi + o);
            pl = *reinterpret_cast<const uint4*>(a.xs_lo + o);
          } else {
            const long o = (long)(a.gather ? a.gather[rr] : rr) * a.ld_xa + (col - a.seg);
            ph = *reinterpret_cast<const uint4*>(a.xa_hi + o);
            pl = *reinterpret_cast<const uint4*>(a.xa_lo + o);
          }
        }
        *reinterpret_cast<uint4*>(xs_hi + r * kMmPitch + cv * 8) = ph;
        if constexpr (!EXACT_X) *reinterpret_cast<uint4*>(xs_lo + r * kMmPitch + cv * 8) = pl;
      }
      __syncthreads();
      // ---- MFMAs --------------------------------------------------------------------------
#pragma unroll
      for (int t = 0; t < kMmKc / 32; ++t) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          if (mt < mt_n) {
            const int off = (mt * 16 + wrow) * kMmPitch + 32 * t + 8 * kg;
            const mfma_bf16x8 ah = *reinterpret_cast<const mfma_bf16x8*>(xs_hi + off);
#pragma unroll
            for (int wt = 0; wt < kMmWT; ++wt) {
              const mfma_bf16x8 bv = *reinterpret_cast<const mfma_bf16x8*>(&wb[wt][t]);
              acc[mt][wt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bv, acc[mt][wt], 0, 0, 0);
            }
            if constexpr (!EXACT_X) {
              const mfma_bf16x8 al = *reinterpret_cast<const mfma_bf16x8*>(xs_lo + off);
#pragma unroll
              for (int wt = 0; wt < kMmWT; ++wt) {
                const mfma_bf16x8 bv = *reinterpret_cast<const mfma_bf16x8*>(&wb[wt][t]);
                acc[mt][wt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bv, acc[mt][wt], 0, 0, 0);
              }
            }
          }
        }
      }
      __syncthreads();
    }

    // ---- epilogue: lane l holds C[m = 16 mt + 4 (l/16) + e][n = tile + l % 16] -------------
    const int ncol = lane & 15;
    if constexpr (EPI == EPI_LOGITS) {
      // masked logits and per-row statistics of this wavefront's 32 rows
      float T[4][4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * kg + e;
          T[mt][e] = (m < rcount) ? a.temp[a.row_seq ? a.row_seq[r0 + m] : r0 + m] : 0.f;
        }
      int mapped[kMmWT];
#pragma unroll
      for (int wt = 0; wt < kMmWT; ++wt) {
        const int n = nw0 + wt * 16 + ncol;
        mapped[wt] = n < a.N ? a.d2t[n] : -1;
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_n) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * kg + e;
          float mx = -INFINITY;
          int am = 0x7fffffff;
          float lv[kMmWT];
#pragma unroll
          for (int wt = 0; wt < kMmWT; ++wt) {
            const int n = nw0 + wt * 16 + ncol;
            lv[wt] = (m < rcount && n < a.N && mapped[wt] >= 0) ? acc[mt][wt][e] : -INFINITY;
            if (m < rcount && n < a.N) a.y[(long)(r0 + m) * a.ld_logits + n] = lv[wt];
            if (lv[wt] > mx) { mx = lv[wt]; am = n; }
          }
          // reduce over the 16 lanes holding row m (xor 1, 2, 4, 8)
#pragma unroll
          for (int sft = 1; sft < 16; sft <<= 1) {
            const float om = xor_lane_c(mx, sft);
            const int oa = xor_lane_ci(am, sft);
            if (om > mx || (om == mx && oa < am)) { mx = om; am = oa; }
          }
          float se = 0.f;
          if (T[mt][e] > 0.f && mx > -INFINITY)
#pragma unroll
            for (int wt = 0; wt < kMmWT; ++wt)
              if (lv[wt] > -INFINITY) se += __expf((lv[wt] - mx) / T[mt][e]);
#pragma unroll
          for (int sft = 1; sft < 16; sft <<= 1) se += xor_lane_c(se, sft);
          if (ncol == 0 && m < rcount) { s_m[wave][m] = mx; s_s[wave][m] = se; s_a[wave][m] = am; }
        }
      }
      __syncthreads();
      // merge the block's wavefronts (ascending rows) into one record per row
      for (int m = tid; m < rcount; m += kMmThreads) {
        float M = -INFINITY;
        int A = 0x7fffffff;
        for (int w = 0; w < kMmWaves; ++w)
          if (s_m[w][m] > M) { M = s_m[w][m]; A = s_a[w][m]; }
        const float Tm = a.temp[a.row_seq ? a.row_seq[r0 + m] : r0 + m];
        float S = 0.f;
        if (Tm > 0.f && M > -INFINITY)
          for (int w = 0; w < kMmWaves; ++w)
            if (s_m[w][m] > -INFINITY) S += s_s[w][m] * __expf((s_m[w][m] - M) / Tm);
        float* p = a.part + ((long)(r0 + m) * a.nblk + blockIdx.x) * 4;
        p[0] = M;
        p[1] = S;
        p[2] = __int_as_float(M > -INFINITY ? A : -1);
        p[3] = 0.f;
      }
      __syncthreads();
    } else {
      // partial sums of this K split: [split][row][N] (SwiGLU: gate then up, 2 N wide)
      const int W = (EPI == EPI_SWIGLU) ? 2 * a.N : a.N;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_n) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * kg + e;
          if (m >= rcount) continue;
          float* pr = a.split_buf + ((long)blockIdx.y * a.max_rows + r0 + m) * W;
#pragma unroll
          for (int wt = 0; wt < kMmWT; ++wt) {
            const int n = (EPI == EPI_SWIGLU) ? nw0 + ncol : nw0 + wt * 16 + ncol;
            if (n < a.N) pr[(EPI == EPI_SWIGLU ? wt * a.N : 0) + n] = acc[mt][wt][e];
          }
        }
      }
    }
    __syncthreads();
  }
}

inline int gemm_mfma_rows_per_block(EpiKind epi) {
  return epi == EPI_LOGITS ? MmShape<EPI_LOGITS>::ROWS
                           : (epi == EPI_SWIGLU ? MmShape<EPI_SWIGLU>::ROWS : MmShape<EPI_STORE>::ROWS);
}

// K splits: a block walks its chunks one after another (load, stage, multiply), so
// the K range is split as finely as the partial buffer allows (one chunk per block
// up to kMaxKSplit splits); never for logits.  Returns the chunks per split; *ks
// receives the splits actually used.
inline int gemm_mfma_split_plan(EpiKind epi, int N, int Kd, int passes, int* ks_out) {
  (void)N;
  (void)passes;
  const int chunks = (Kd + kMmKc - 1) / kMmKc;
  int ks = 1;
  if (epi != EPI_LOGITS) ks = chunks > kMaxKSplit ? kMaxKSplit : chunks;
  const int cps = (chunks + ks - 1) / ks;
  *ks_out = (chunks + cps - 1) / cps;
  return cps;
}

template <int SRC, int EPI>
int launch_gemm_mfma_t(const GemvArgs& a, hipStream_t st) {
  const int rpb = gemm_mfma_rows_per_block((EpiKind)EPI);
  const int nb = (a.N + rpb - 1) / rpb;
  const int passes = (a.max_rows + kMmRows - 1) / kMmRows;
  int ks = 1;
  const int cps = gemm_mfma_split_plan((EpiKind)EPI, a.N, a.Kd, passes, &ks);
  hipLaunchKernelGGL((k_gemm_mfma<SRC, EPI>), dim3(nb, ks, passes), dim3(MmShape<EPI>::THREADS), 0, st, a, cps);
  return ks;
}

}  // namespace osp

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
// Block: 8 wavefronts sharing one input stage; wavefront w owns WT = 2 tiles of
// 16 weight rows (SwiGLU: a gate tile and the matching up tile).  K is walked in
// chunks of 256 columns: the weights of a chunk are requested before the input
// chunk is staged, so both transfers overlap.
#pragma once

#include "common.h"
#include "internal.h"

namespace osp {

typedef __bf16 mfma_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

constexpr int kMmRows = 64;          // input rows per pass (4 M tiles)
constexpr int kMmKc = 256;           // K columns per chunk
constexpr int kMmPitch = kMmKc + 8;  // LDS row pitch in bf16 (pads banks)

// Block shape per kind: the logits kind (large N, no split) uses 8 wavefronts with
// two weight tiles each; the others 4 wavefronts with one tile (SwiGLU: a gate
// tile and its up tile) and split K across blocks when N alone gives too few.
template <int EPI> struct MmShape {
  static constexpr int WAVES = EPI == EPI_LOGITS ? 8 : 4;
  static constexpr int WT = EPI == EPI_LOGITS ? 2 : (EPI == EPI_SWIGLU ? 2 : 1);
  static constexpr int NT = EPI == EPI_SWIGLU ? 1 : WT;   // output tiles per wavefront
  static constexpr int THREADS = WAVES * 64;
  static constexpr int ROWS = WAVES * NT * 16;            // output rows per block
};

OSP_DEV uint32_t pack_bf16x2(bf16_t lo, bf16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

// Input values X[rr][col .. col+8) (fp32) of the pass; the normalised segment is
// scaled by inv_rms * gain.
template <int SRC>
OSP_DEV void mm_load_x8(const GemvArgs& a, int rr, int col, float inv_rms, float* out) {
  if constexpr (SRC == SRC_PLAIN) {
    const float* p = a.xin + (long)rr * a.ldx + col;
    const float4 v0 = *reinterpret_cast<const float4*>(p);
    const float4 v1 = *reinterpret_cast<const float4*>(p + 4);
    out[0] = v0.x; out[1] = v0.y; out[2] = v0.z; out[3] = v0.w;
    out[4] = v1.x; out[5] = v1.y; out[6] = v1.z; out[7] = v1.w;
  } else if constexpr (SRC == SRC_TAPS) {
    load_vec<bf16_t>(reinterpret_cast<const bf16_t*>(a.taps) + (long)a.tap_row[rr] * a.ldt + col, out);
  } else {
    int c = col;
    if constexpr (SRC == SRC_QKV) {
      if (col < a.d_norm) {
        const int sr = a.s_gather ? a.s_gather[rr] : rr;
        const float* p = a.s + (long)sr * a.lds + col;
        const float4 v0 = *reinterpret_cast<const float4*>(p);
        const float4 v1 = *reinterpret_cast<const float4*>(p + 4);
        out[0] = v0.x; out[1] = v0.y; out[2] = v0.z; out[3] = v0.w;
        out[4] = v1.x; out[5] = v1.y; out[6] = v1.z; out[7] = v1.w;
        return;
      }
      c = col - a.d_norm;
    }
    if (SRC == SRC_QKV && a.embed) {
      int t = a.tok[rr];
      t = min(max(t, 0), a.vocab_embed - 1);
      load_vec<bf16_t>(reinterpret_cast<const bf16_t*>(a.embed) + (long)t * a.d_norm + c, out);
    } else {
      const int xr = a.gather ? a.gather[rr] : rr;
      const float* p = a.xin + (long)xr * a.ldx + c;
      const float4 v0 = *reinterpret_cast<const float4*>(p);
      const float4 v1 = *reinterpret_cast<const float4*>(p + 4);
      out[0] = v0.x; out[1] = v0.y; out[2] = v0.z; out[3] = v0.w;
      out[4] = v1.x; out[5] = v1.y; out[6] = v1.z; out[7] = v1.w;
    }
    float g[8];
    load_vec<bf16_t>(reinterpret_cast<const bf16_t*>(a.gamma) + c, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = out[e] * inv_rms * g[e];
  }
}

template <int SRC, int EPI>
__global__ void __launch_bounds__(MmShape<EPI>::THREADS) k_gemm_mfma(GemvArgs a, float* split_out,
                                                                      int chunks_per_split) {
  constexpr bool NORMED = (SRC == SRC_NORM || SRC == SRC_QKV);
  constexpr bool EXACT_X = (SRC == SRC_TAPS);          // inputs already bf16: no lo part
  constexpr int kMmWaves = MmShape<EPI>::WAVES;
  constexpr int kMmThreads = MmShape<EPI>::THREADS;
  constexpr int kMmWT = MmShape<EPI>::WT;
  constexpr int NT = MmShape<EPI>::NT;
  __shared__ __attribute__((aligned(16))) bf16_t xs_hi[kMmRows * kMmPitch];
  __shared__ __attribute__((aligned(16))) bf16_t xs_lo[EXACT_X ? 8 : kMmRows * kMmPitch];
  __shared__ float s_inv[kMmRows];
  __shared__ float s_m[kMmWaves][kMmRows];
  __shared__ float s_s[kMmWaves][kMmRows];
  __shared__ int s_a[kMmWaves][kMmRows];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  const bf16_t* __restrict__ w0 = reinterpret_cast<const bf16_t*>(a.w0);
  const bf16_t* __restrict__ w1 = reinterpret_cast<const bf16_t*>(a.w1);
  const int rows_per_block = kMmWaves * NT * 16;
  const int nb0 = blockIdx.x * rows_per_block;          // first output row of the block
  const int nw0 = nb0 + wave * NT * 16;                 // first output row of this wavefront
  const int wrow = lane & 15, kg = lane >> 4;           // B operand: weight row, 8-column group

  for (int r0 = 0; r0 < rows; r0 += kMmRows) {
    const int rcount = min(kMmRows, rows - r0);
    const int mt_n = (rcount + 15) >> 4;                // M tiles in use
    // ---- RMSNorm factors of the rows of this pass ------------------------------------
    if constexpr (NORMED) {
      for (int r = wave; r < rcount; r += kMmWaves) {
        const int rr = r0 + r;
        float ss = 0.f;
        // sum of squares of the raw (un-normalised) segment
        if (SRC == SRC_QKV && a.embed) {
          int t = a.tok[rr];
          t = min(max(t, 0), a.vocab_embed - 1);
          const bf16_t* e = reinterpret_cast<const bf16_t*>(a.embed) + (long)t * a.d_norm;
          for (int c = lane * 8; c < a.d_norm; c += OSP_WAVE * 8) {
            float v[8];
            load_vec<bf16_t>(e + c, v);
#pragma unroll
            for (int q = 0; q < 8; ++q) ss += v[q] * v[q];
          }
        } else {
          const int xr = a.gather ? a.gather[rr] : rr;
          const float* xp = a.xin + (long)xr * a.ldx;
          for (int c = lane * 4; c < a.d_norm; c += OSP_WAVE * 4) {
            const float4 v = *reinterpret_cast<const float4*>(xp + c);
            ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
          }
        }
        ss = wave_sum(ss);
        if (lane == 0) s_inv[r] = 1.0f / sqrtf(ss / (float)a.d_norm + a.eps);
      }
    }
    // layer 0 of the expanded QKV: block 0 writes x = embed[token] for the residual
    if constexpr (SRC == SRC_QKV) {
      if (a.embed && a.x_out && blockIdx.x == 0 && blockIdx.y == 0) {
        for (int i = tid; i < rcount * a.d_norm; i += kMmThreads) {
          const int r = i / a.d_norm, c = i - r * a.d_norm;
          int t = a.tok[r0 + r];
          t = min(max(t, 0), a.vocab_embed - 1);
          a.x_out[(long)(r0 + r) * a.ldx + c] =
              load_f32(reinterpret_cast<const bf16_t*>(a.embed), (long)t * a.d_norm + c);
        }
      }
    }
    __syncthreads();

    mfma_f32x4 acc[4][kMmWT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int wt = 0; wt < kMmWT; ++wt) acc[mt][wt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};

    const int k_begin = blockIdx.y * chunks_per_split * kMmKc;
    const int k_end = min(a.Kd, k_begin + chunks_per_split * kMmKc);
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
      // ---- stage the input chunk as bf16 hi / lo ----------------------------------------
      for (int i = tid; i < kMmRows * (kMmKc / 8); i += kMmThreads) {
        const int r = i / (kMmKc / 8), cv = i - r * (kMmKc / 8);
        const int col = k0 + cv * 8;
        float v[8];
        if (r < rcount && col < a.Kd) {
          float inv = 1.f;
          if constexpr (NORMED) inv = s_inv[r];
          mm_load_x8<SRC>(a, r0 + r, col, inv, v);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = 0.f;
        }
        bf16_t hi[8], lo[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          hi[e] = f32_to_bf16(v[e]);
          lo[e] = f32_to_bf16(v[e] - bf16_to_f32(hi[e]));
        }
        uint4 ph = make_uint4(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]),
                              pack_bf16x2(hi[4], hi[5]), pack_bf16x2(hi[6], hi[7]));
        *reinterpret_cast<uint4*>(xs_hi + r * kMmPitch + cv * 8) = ph;
        if constexpr (!EXACT_X) {
          uint4 pl = make_uint4(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]),
                                pack_bf16x2(lo[4], lo[5]), pack_bf16x2(lo[6], lo[7]));
          *reinterpret_cast<uint4*>(xs_lo + r * kMmPitch + cv * 8) = pl;
        }
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
            const float om = __shfl_xor(mx, sft, OSP_WAVE);
            const int oa = __shfl_xor(am, sft, OSP_WAVE);
            if (om > mx || (om == mx && oa < am)) { mx = om; am = oa; }
          }
          float se = 0.f;
          if (T[mt][e] > 0.f && mx > -INFINITY)
#pragma unroll
            for (int wt = 0; wt < kMmWT; ++wt)
              if (lv[wt] > -INFINITY) se += __expf((lv[wt] - mx) / T[mt][e]);
#pragma unroll
          for (int sft = 1; sft < 16; sft <<= 1) se += __shfl_xor(se, sft, OSP_WAVE);
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
    } else if (split_out) {
      // split K: this block's partial sums, [split][row][N] (SwiGLU: gate then up, 2N)
      const int W = (EPI == EPI_SWIGLU) ? 2 * a.N : a.N;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_n) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * kg + e;
          if (m >= rcount) continue;
          float* pr = split_out + ((long)blockIdx.y * a.max_rows + r0 + m) * W;
#pragma unroll
          for (int wt = 0; wt < kMmWT; ++wt) {
            const int n = (EPI == EPI_SWIGLU) ? nw0 + ncol : nw0 + wt * 16 + ncol;
            if (n < a.N) pr[(EPI == EPI_SWIGLU ? wt * a.N : 0) + n] = acc[mt][wt][e];
          }
        }
      }
    } else {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_n) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = mt * 16 + 4 * kg + e;
          if (m >= rcount) continue;
          float* yr = a.y + (long)(r0 + m) * a.ldy;
          if constexpr (EPI == EPI_SWIGLU) {
            const int n = nw0 + ncol;
            if (n < a.N) {
              const float g = acc[mt][0][e], u = acc[mt][1][e];
              yr[n] = g / (1.0f + __expf(-g)) * u;
            }
          } else {
#pragma unroll
            for (int wt = 0; wt < kMmWT; ++wt) {
              const int n = nw0 + wt * 16 + ncol;
              if (n < a.N) {
                if constexpr (EPI == EPI_RESID) yr[n] += acc[mt][wt][e]; else yr[n] = acc[mt][wt][e];
              }
            }
          }
        }
      }
    }
    __syncthreads();
  }
}

// The matrix-core path serves passes of two or more rows of bf16 weights.
inline bool gemm_use_mfma(int wdtype, int rows) { return wdtype == 1 && rows >= 2; }

inline int gemm_mfma_rows_per_block(EpiKind epi) {
  return epi == EPI_LOGITS ? MmShape<EPI_LOGITS>::ROWS
                           : (epi == EPI_SWIGLU ? MmShape<EPI_SWIGLU>::ROWS : MmShape<EPI_STORE>::ROWS);
}

// K splits: enough blocks to cover the chip (about 2 per CU), never for logits.
inline int gemm_mfma_splits(EpiKind epi, int N, int Kd) {
  if (epi == EPI_LOGITS) return 1;
  const int nb = (N + gemm_mfma_rows_per_block(epi) - 1) / gemm_mfma_rows_per_block(epi);
  const int chunks = (Kd + kMmKc - 1) / kMmKc;
  int ks = (512 + nb - 1) / nb;
  ks = ks < 1 ? 1 : (ks > chunks ? chunks : ks);
  return ks > kMaxKSplit ? kMaxKSplit : ks;
}

// Sum of the K-split partials in split order, then the kind's epilogue.
template <int EPI>
__global__ void __launch_bounds__(256) k_splitk_reduce(GemvArgs a, const float* split_out, int ks) {
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  const long total = (long)rows * a.N;
  const int W = (EPI == EPI_SWIGLU) ? 2 * a.N : a.N;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const int m = (int)(i / a.N), n = (int)(i - (long)m * a.N);
    float s0 = 0.f, s1 = 0.f;
    for (int k = 0; k < ks; ++k) {
      const float* pr = split_out + ((long)k * a.max_rows + m) * W;
      s0 += pr[n];
      if constexpr (EPI == EPI_SWIGLU) s1 += pr[a.N + n];
    }
    float* yp = a.y + (long)m * a.ldy + n;
    if constexpr (EPI == EPI_SWIGLU) *yp = s0 / (1.0f + __expf(-s0)) * s1;
    else if constexpr (EPI == EPI_RESID) *yp += s0;
    else *yp = s0;
  }
}

template <int SRC, int EPI>
void launch_gemm_mfma_t(const GemvArgs& a, hipStream_t st) {
  const int rpb = gemm_mfma_rows_per_block((EpiKind)EPI);
  const int nb = (a.N + rpb - 1) / rpb;
  const int ks = gemm_mfma_splits((EpiKind)EPI, a.N, a.Kd);
  const int chunks = (a.Kd + kMmKc - 1) / kMmKc;
  const int cps = (chunks + ks - 1) / ks;
  const int ks_used = (chunks + cps - 1) / cps;
  float* split = ks_used > 1 ? a.split_buf : nullptr;
  hipLaunchKernelGGL((k_gemm_mfma<SRC, EPI>), dim3(nb, ks_used), dim3(MmShape<EPI>::THREADS), 0, st,
                     a, split, cps);
  if (split) {
    const long total = (long)a.max_rows * a.N;
    const int grid = (int)((total + 255) / 256 < 2048 ? (total + 255) / 256 : 2048);
    hipLaunchKernelGGL((k_splitk_reduce<EPI>), dim3(grid), dim3(256), 0, st, a, split, ks_used);
  }
}

}  // namespace osp

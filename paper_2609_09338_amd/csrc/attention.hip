// Attention of the drafter over its paged KV cache.
//
// k_rope_kvwrite: per row and head, the Qwen3 per-head RMSNorm of q and k,
//   rotate-half RoPE at the row's absolute position (cos/sin table built on the
//   host in float64), then k and v are stored (rounded to bf16 in bf16 pools)
//   into the row's cache slot; q is kept in fp32.
// k_attn: one block per (sequence, kv head, context split).  Each wavefront
//   walks 16-token cache blocks of the split (one KV page per step): 4 lanes per
//   token, each lane holding a quarter of the head dimension, so a page of K or V
//   is one fully coalesced 4 KB read.  Every query vector of the sequence that
//   reads this kv head (all new rows x the GQA group) is scored against the page,
//   with a causal mask at the row's position and an online softmax; the four
//   wavefronts' partial results are merged in LDS and written per split.
// k_attn_combine: merges the splits of each (row, head) with their log-sum-exp
//   weights (flash-decoding) and normalises.
#include "common.h"
#include "internal.h"

namespace osp {

template <typename TKV>
__global__ void __launch_bounds__(64) k_rope_kvwrite(AttnArgs a) {
  const int r = blockIdx.x;
  const int hh = blockIdx.y;
  const int rows = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  if (r >= rows) return;
  const int lane = threadIdx.x;
  const int hd = a.hd, half = hd >> 1;
  const int pos = a.rows.pos[r];
  const int b = a.rows.seq ? a.rows.seq[r] : r;
  const bool is_q = hh < a.nq;
  const int g = is_q ? 0 : hh - a.nq;
  const float* src = a.qkv + (long)r * a.qkv_w + (is_q ? hh * hd : (a.nq + g) * hd);
  const bool act = lane < half;
  float x1 = act ? src[lane] : 0.f, x2 = act ? src[lane + half] : 0.f;
  if (a.qk_norm) {
    const float ss = wave_sum(x1 * x1 + x2 * x2);
    const float inv = 1.0f / sqrtf(ss / (float)hd + a.eps);
    const TKV* gn = reinterpret_cast<const TKV*>(is_q ? a.q_norm : a.k_norm);
    if (act) {
      x1 = x1 * inv * load_f32(gn, lane);
      x2 = x2 * inv * load_f32(gn, lane + half);
    }
  }
  const int p = min(max(pos, 0), a.max_seq - 1);
  const float c = act ? a.rope_cos[(long)p * half + lane] : 0.f;
  const float s = act ? a.rope_sin[(long)p * half + lane] : 0.f;
  const float y1 = x1 * c - x2 * s;
  const float y2 = x2 * c + x1 * s;
  if (is_q) {
    if (act) {
      float* q = a.q + (long)r * (a.nq * hd) + hh * hd;
      q[lane] = y1;
      q[lane + half] = y2;
    }
    return;
  }
  const int slot = a.bslot[b];
  const int blk = pos / a.kv_block, within = pos - blk * a.kv_block;
  if (pos < 0 || blk >= a.slot_nblocks[slot]) {
    if (lane == 0) atomicOr(a.err, 1u << 3);
    return;
  }
  const long phys = a.block_table[(long)slot * a.max_blocks + blk];
  TKV* base = reinterpret_cast<TKV*>(a.kv) +
              phys * kv_block_elems(a.n_layers, a.nkv, a.kv_block, hd);
  TKV* kp = base + (((long)a.layer * 2 + 0) * a.nkv + g) * a.kv_block * hd + (long)within * hd;
  TKV* vp = base + (((long)a.layer * 2 + 1) * a.nkv + g) * a.kv_block * hd + (long)within * hd;
  const float* vs = a.qkv + (long)r * a.qkv_w + (a.nq + a.nkv + g) * hd;
  if (act) {
    store_from_f32(kp, lane, y1);
    store_from_f32(kp, lane + half, y2);
    store_from_f32(vp, lane, vs[lane]);
    store_from_f32(vp, lane + half, vs[lane + half]);
  }
}

// Load DPL consecutive cache elements as floats.
template <typename TKV, int DPL>
OSP_DEV void load_seg(const TKV* p, float* out) {
  constexpr int VEC = Vec<TKV>::N;
#pragma unroll
  for (int j = 0; j < DPL / VEC; ++j) load_vec<TKV>(p + j * VEC, out + j * VEC);
}

template <typename TKV, int HD>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int LPT = 4;               // lanes per token
  constexpr int DPL = HD / LPT;        // head dims per lane
  constexpr int QV = 256 / HD;         // query vectors per pass (q + o = 2*QV*DPL = 128 regs)
  constexpr int TPW = OSP_WAVE / LPT;  // tokens per wavefront step (= KV page size 16)
  __shared__ float sm_m[4][QV];
  __shared__ float sm_l[4][QV];
  __shared__ float sm_o[4][QV][HD];

  const int b = blockIdx.x, g = blockIdx.y, sp = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tok = lane / LPT, seg = lane % LPT;
  int r_beg, r_end;
  if (a.cu) { r_beg = a.cu[b]; r_end = a.cu[b + 1]; } else { r_beg = b; r_end = b + 1; }
  const int rows_total = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  r_end = min(r_end, rows_total);
  if (r_beg >= r_end) return;
  const int G = a.nq / a.nkv;
  const int nvec = (r_end - r_beg) * G;
  const int n_ctx = a.rows.pos[r_end - 1] + 1;
  int ts = (n_ctx + a.n_split - 1) / a.n_split;
  ts = (ts + TPW - 1) / TPW * TPW;
  const int p_lo = sp * ts;
  const int p_hi = min(n_ctx, p_lo + ts);
  const int slot = a.bslot[b];
  const int nblocks = a.slot_nblocks[slot];
  const int32_t* bt = a.block_table + (long)slot * a.max_blocks;
  const TKV* kvb = reinterpret_cast<const TKV*>(a.kv);
  const long blk_elems = kv_block_elems(a.n_layers, a.nkv, a.kv_block, HD);
  const long k_off = (((long)a.layer * 2 + 0) * a.nkv + g) * a.kv_block * HD;
  const long v_off = (((long)a.layer * 2 + 1) * a.nkv + g) * a.kv_block * HD;
  const int nq_hd = a.nq * HD;

  for (int j0 = 0; j0 < nvec; j0 += QV) {
    float q[QV][DPL], o[QV][DPL], m[QV], l[QV];
    int qpos[QV];
#pragma unroll
    for (int j = 0; j < QV; ++j) {
      const int jj = j0 + j;
      m[j] = -INFINITY;
      l[j] = 0.f;
      qpos[j] = -1;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
      if (jj < nvec) {
        const int r = r_beg + jj / G, h = g * G + jj % G;
        qpos[j] = a.rows.pos[r];
        const float* qp = a.q + (long)r * nq_hd + h * HD + seg * DPL;
#pragma unroll
        for (int e = 0; e < DPL; ++e) q[j][e] = qp[e] * a.scale;
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) q[j][e] = 0.f;
      }
    }
    for (int t0 = p_lo + wave * TPW; t0 < p_hi; t0 += 4 * TPW) {
      const int p = t0 + tok;
      const int blk = t0 / a.kv_block;
      const bool valid = p < p_hi && blk < nblocks;
      float kf[DPL], vf[DPL];
      if (valid) {
        const long phys = bt[blk];
        const TKV* kp = kvb + phys * blk_elems + k_off + (long)(p - blk * a.kv_block) * HD + seg * DPL;
        const TKV* vp = kvb + phys * blk_elems + v_off + (long)(p - blk * a.kv_block) * HD + seg * DPL;
        load_seg<TKV, DPL>(kp, kf);
        load_seg<TKV, DPL>(vp, vf);
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) { kf[e] = 0.f; vf[e] = 0.f; }
      }
#pragma unroll
      for (int j = 0; j < QV; ++j) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) s = fmaf(q[j][e], kf[e], s);
        s += __shfl_xor(s, 1, OSP_WAVE);
        s += __shfl_xor(s, 2, OSP_WAVE);
        if (!valid || p > qpos[j]) s = -INFINITY;
        float bm = s;
        bm = fmaxf(bm, __shfl_xor(bm, 4, OSP_WAVE));
        bm = fmaxf(bm, __shfl_xor(bm, 8, OSP_WAVE));
        bm = fmaxf(bm, __shfl_xor(bm, 16, OSP_WAVE));
        bm = fmaxf(bm, __shfl_xor(bm, 32, OSP_WAVE));
        const float mn = fmaxf(m[j], bm);
        if (mn == -INFINITY) continue;
        const float so = __expf(m[j] - mn);
        const float pe = __expf(s - mn);
        l[j] = l[j] * so + pe;
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(pe, vf[e], o[j][e] * so);
        m[j] = mn;
      }
    }
    // ---- merge lanes of one wave: sum over the 16 token lanes of each segment ---------
#pragma unroll
    for (int j = 0; j < QV; ++j) {
#pragma unroll
      for (int sft = 4; sft < 64; sft <<= 1) {
        l[j] += __shfl_xor(l[j], sft, OSP_WAVE);
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] += __shfl_xor(o[j][e], sft, OSP_WAVE);
      }
      if (lane < LPT) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) sm_o[wave][j][seg * DPL + e] = o[j][e];
      }
      if (lane == 0) { sm_m[wave][j] = m[j]; sm_l[wave][j] = l[j]; }
    }
    __syncthreads();
    // ---- merge the four wavefronts and write this split's partial --------------------
    for (int i = tid; i < QV * HD; i += 256) {
      const int j = i / HD, e = i - j * HD;
      const int jj = j0 + j;
      if (jj >= nvec) continue;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, sm_m[w][j]);
      float L = 0.f, O = 0.f;
      if (M > -INFINITY) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float f = __expf(sm_m[w][j] - M);
          L += sm_l[w][j] * f;
          O += sm_o[w][j][e] * f;
        }
      }
      const int r = r_beg + jj / G, h = g * G + jj % G;
      float* pp = a.part + (((long)r * a.nq + h) * a.n_split + sp) * (HD + 2);
      pp[2 + e] = O;
      if (e == 0) { pp[0] = M; pp[1] = L; }
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(128) k_attn_combine(AttnArgs a) {
  const int r = blockIdx.x, h = blockIdx.y;
  const int rows = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  if (r >= rows) return;
  const int hd = a.hd;
  const float* pp = a.part + ((long)r * a.nq + h) * a.n_split * (hd + 2);
  float M = -INFINITY;
  for (int sp = 0; sp < a.n_split; ++sp) M = fmaxf(M, pp[sp * (hd + 2)]);
  for (int e = threadIdx.x; e < hd; e += blockDim.x) {
    float L = 0.f, O = 0.f;
    for (int sp = 0; sp < a.n_split; ++sp) {
      const float m = pp[sp * (hd + 2)];
      if (m == -INFINITY) continue;
      const float f = __expf(m - M);
      L += pp[sp * (hd + 2) + 1] * f;
      O += pp[sp * (hd + 2) + 2 + e] * f;
    }
    a.o[(long)r * a.nq * hd + h * hd + e] = L > 0.f ? O / L : 0.f;
  }
}

void launch_rope_kvwrite(int kvdtype, const AttnArgs& a, hipStream_t st) {
  dim3 grid(a.rows.max_rows, a.nq + a.nkv);
  if (kvdtype == 1) hipLaunchKernelGGL(k_rope_kvwrite<bf16_t>, grid, dim3(64), 0, st, a);
  else hipLaunchKernelGGL(k_rope_kvwrite<float>, grid, dim3(64), 0, st, a);
}

void launch_attention(int kvdtype, const AttnArgs& a, hipStream_t st) {
  dim3 grid(a.B, a.nkv, a.n_split);
  if (kvdtype == 1) {
    if (a.hd == 128) hipLaunchKernelGGL((k_attn<bf16_t, 128>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((k_attn<bf16_t, 64>), grid, dim3(256), 0, st, a);
  } else {
    if (a.hd == 128) hipLaunchKernelGGL((k_attn<float, 128>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((k_attn<float, 64>), grid, dim3(256), 0, st, a);
  }
}

void launch_attn_combine(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_attn_combine, dim3(a.rows.max_rows, a.nq), dim3(128), 0, st, a);
}

}  // namespace osp

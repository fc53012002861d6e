// Attention of the drafter over its paged KV cache (flash-decoding: each block
// covers one context split of one (sequence, kv head); k_attn_combine merges the
// splits with their log-sum-exp weights and normalises).
//
// Both kernels first do the row work of the pass:
//   * new rows whose position falls in the block's split: Qwen3 per-head RMSNorm
//     of k, rotate-half RoPE at the row's absolute position (cos/sin table built
//     on the host in float64), then k and v go into the row's cache page
//     (rounded to bf16 in bf16 pools).  Every position belongs to exactly one
//     split, so each new key/value is written once, by the block that reads it;
//   * the query vectors that read this kv head (new rows x GQA group) are
//     normalised, rotated and scaled by 1/sqrt(hd) into LDS.
// Projections come either as plain rows or as K-split partial sums (matrix-core
// path), which are added on load in split order.
//
// Blocks are (kv head, work item): the head varies fastest, so the setup kernel's
// longest-first order of (sequence, split) items holds across heads.
//
// k_attn_mfma (bf16 pools): up to 16 query vectors per pass.  Each wavefront
// walks 16-token pages of the split:
//   S^T = K Q^T   (tokens x queries; 16x16x32 bf16 MFMA over the head dimension,
//                  queries as bf16 hi + lo pairs),
//   online softmax per query (a lane owns one query, 4 tokens),
//   O^T += V^T P^T (head dims x queries; 16x16x16 bf16 MFMA over the page's
//                  tokens, P as bf16 hi + lo pairs),
// with the next pages already requested.
// The transposed value page gives V^T tiles as 8-byte loads, and the score
// tile's register layout is exactly the B operand of the second product, so no
// data moves between lanes except the per-query max/sum reductions.
// k_attn (fp32 pools): 16 lanes per token, online softmax on the vector units.
#include "common.h"
#include "internal.h"

namespace osp {

// DPL consecutive cache elements kept in their storage form (bf16 pairs or fp32).
template <typename TKV, int DPL> struct Seg;
template <int DPL> struct Seg<bf16_t, DPL> {
  static_assert(DPL == 4 || DPL == 8, "bf16 segments of 4 or 8 elements");
  uint32_t raw[DPL / 2];
  OSP_DEV void load(const bf16_t* p) {
    if constexpr (DPL == 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(p);
      raw[0] = v.x; raw[1] = v.y; raw[2] = v.z; raw[3] = v.w;
    } else {
      const uint2 v = *reinterpret_cast<const uint2*>(p);
      raw[0] = v.x; raw[1] = v.y;
    }
  }
  OSP_DEV void zero() {
#pragma unroll
    for (int i = 0; i < DPL / 2; ++i) raw[i] = 0u;
  }
  OSP_DEV float get(int e) const { return (e & 1) ? bf16_hi(raw[e >> 1]) : bf16_lo(raw[e >> 1]); }
};
template <int DPL> struct Seg<float, DPL> {
  float raw[DPL];
  OSP_DEV void load_t(const float* p, int stride) {
#pragma unroll
    for (int i = 0; i < DPL; ++i) raw[i] = p[(long)i * stride];
  }
  OSP_DEV void load(const float* p) {
#pragma unroll
    for (int j = 0; j < DPL / 4; ++j) {
      const float4 v = *reinterpret_cast<const float4*>(p + j * 4);
      raw[4 * j] = v.x; raw[4 * j + 1] = v.y; raw[4 * j + 2] = v.z; raw[4 * j + 3] = v.w;
    }
  }
  OSP_DEV void zero() {
#pragma unroll
    for (int i = 0; i < DPL; ++i) raw[i] = 0.f;
  }
  OSP_DEV float get(int e) const { return raw[e]; }
};

// Per-head RMSNorm (optional) + rotate-half RoPE of one head vector held as
// (x1 = element lane, x2 = element lane + HD/2) by lanes < HD/2 of a wavefront.
template <typename TKV, int HD>
OSP_DEV void norm_rope(const AttnArgs& a, const void* gain, int pos, int lane, float& x1,
                       float& x2) {
  constexpr int HALF = HD / 2;
  const bool act = lane < HALF;
  if (a.qk_norm) {
    const float ss = wave_sum(act ? x1 * x1 + x2 * x2 : 0.f);
    const float inv = 1.0f / sqrtf(ss / (float)HD + a.eps);
    if (act) {
      const TKV* gn = reinterpret_cast<const TKV*>(gain);
      x1 = x1 * inv * load_f32(gn, lane);
      x2 = x2 * inv * load_f32(gn, lane + HALF);
    }
  }
  const int p = min(max(pos, 0), a.max_seq - 1);
  const float c = act ? a.rope_cos[(long)p * HALF + lane] : 0.f;
  const float s = act ? a.rope_sin[(long)p * HALF + lane] : 0.f;
  const float y1 = x1 * c - x2 * s;
  const float y2 = x2 * c + x1 * s;
  x1 = y1;
  x2 = y2;
}

// One 16-token page of one kv head (fp32): lane l holds head dims [DPL*(l%16), +DPL)
// of tokens 4u + l/16, u = 0..3 (each of the 4 key loads is one coalesced
// wavefront read of 4 consecutive tokens; values come from the transposed page).
template <typename TKV, int HD>
struct Page {
  static constexpr int DPL = HD / 16;
  Seg<TKV, DPL> k[4], v[4];
  OSP_DEV void load(const TKV* kbase, const TKV* vbase, int lane) {
    const int off = (lane >> 4) * HD + (lane & 15) * DPL;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      k[u].load(kbase + u * 4 * HD + off);
      v[u].load_t(vbase + kv_v_at(4 * u + (lane >> 4), (lane & 15) * DPL, 16), 16);
    }
  }
  OSP_DEV void zero() {
#pragma unroll
    for (int u = 0; u < 4; ++u) { k[u].zero(); v[u].zero(); }
  }
};

constexpr int kMaxSplitAttn = 64;   // context splits per row (bound; the host keeps to it)

// Elements off[j] (j < N) of the projections: the sums of the K-split partials
// (in split order) on the matrix-core path, else the plain row.  Every split's load of
// every element is requested at once, from a clamped address (loads past the last
// split re-read it and add zero), so no load waits on a condition.
template <int N>
OSP_DEV void qkv_get(const AttnArgs& a, const long (&off)[N], float (&out)[N]) {
  if (a.qkv_ks <= 1) {
#pragma unroll
    for (int j = 0; j < N; ++j) out[j] = a.qkv[off[j]];
    return;
  }
  float v[N][kMaxKSplit];
#pragma unroll
  for (int k = 0; k < kMaxKSplit; ++k)
#pragma unroll
    for (int j = 0; j < N; ++j) v[j][k] = a.qkv[min(k, a.qkv_ks - 1) * a.qkv_split + off[j]];
#pragma unroll
  for (int j = 0; j < N; ++j) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxKSplit; ++k) s += k < a.qkv_ks ? v[j][k] : 0.f;
    out[j] = s;
  }
}

// Element `off` of the projections, as qkv_get does, one element per request: the
// loads of its splits are issued back to back under uniform branches (no wait between
// them), with fewer registers held than a batched request needs.
OSP_DEV float qkv_at(const AttnArgs& a, long off) {
  if (a.qkv_ks <= 1) return a.qkv[off];
  float v[kMaxKSplit];
#pragma unroll
  for (int k = 0; k < kMaxKSplit; ++k) v[k] = k < a.qkv_ks ? a.qkv[k * a.qkv_split + off] : 0.f;
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kMaxKSplit; ++k) s += v[k];
  return s;
}

// The projection elements a wavefront's lanes < hd / 2 need: columns base + lane and
// base + lane + hd / 2 of each base in `base`.  The matrix-core attention with bf16
// pages requests all of them at once (its register count allows it: two waves per SIMD
// either way); the other attention kernels request one element at a time.
template <typename TKV, int HD>
constexpr bool kBatchQkv = HD == 128 && sizeof(TKV) == 2;

template <int HD, bool BATCH, int N>
OSP_DEV void qkv_lanes(const AttnArgs& a, const long (&base)[N], int lane, float (&out)[2 * N]) {
  constexpr int HALF = HD / 2;
#pragma unroll
  for (int j = 0; j < 2 * N; ++j) out[j] = 0.f;
  if (lane >= HALF) return;
  if constexpr (BATCH) {
    long off[2 * N];
#pragma unroll
    for (int j = 0; j < N; ++j) { off[2 * j] = base[j] + lane; off[2 * j + 1] = base[j] + lane + HALF; }
    qkv_get<2 * N>(a, off, out);
  } else {
#pragma unroll
    for (int j = 0; j < N; ++j) { out[2 * j] = qkv_at(a, base[j] + lane); out[2 * j + 1] = qkv_at(a, base[j] + lane + HALF); }
  }
}

// Block (kv head blockIdx.x, work item blockIdx.y) -> (sequence, split, cache slot):
// from the setup kernel's longest-first list (which carries the slot), or split-major
// when there is none.  False for grid slots past the list.
OSP_DEV bool attn_block(const AttnArgs& a, int& b, int& sp, int& slot) {
  const int it = blockIdx.y;
  if (a.items) {
    if (it >= *a.n_items) return false;
    const int v = a.items[it];
    b = v & 0xff;
    slot = (v >> 8) & 0xff;
    sp = v >> 16;
  } else {
    b = it % a.B;
    sp = it / a.B;
    slot = a.slot0 >= 0 ? a.slot0 : a.bslot[b];
  }
  return true;
}

// New keys/values of rows r_beg..r_end whose position lies in [p_lo, p_hi):
// k normalised and rotated, both stored into the row's cache page.
template <typename TKV, int HD>
OSP_DEV void append_new_kv(const AttnArgs& a, int r_beg, int r_end, int p_lo, int p_hi,
                           const int32_t* bt, int nblocks, TKV* kvb, long blk_elems, long k_off,
                           long v_off, int g, int wave, int lane) {
  constexpr int HALF = HD / 2;
  bool wrote = false;
  for (int r = r_beg + (3 - wave); r < r_end; r += 4) {
    const int pos = a.rows.pos[r];
    if (pos < p_lo || pos >= p_hi) continue;
    const int blk = pos / a.kv_block;
    if (blk >= nblocks) { if (lane == 0) atomicOr(a.err, 1u << 3); continue; }
    const long ko = (long)r * a.qkv_w + (a.nq + g) * HD;
    const long vo = (long)r * a.qkv_w + (a.nq + a.nkv + g) * HD;
    float kv[4];
    qkv_lanes<HD, kBatchQkv<TKV, HD>>(a, {ko, vo}, lane, kv);
    float k1 = kv[0], k2 = kv[1];
    const float v1 = kv[2], v2 = kv[3];
    norm_rope<TKV, HD>(a, a.k_norm, pos, lane, k1, k2);
    const long base = (long)bt[blk] * blk_elems;
    const int w = pos - blk * a.kv_block;
    if (lane < HALF) {
      store_from_f32(kvb, base + k_off + kv_k_at(w, lane, HD), k1);
      store_from_f32(kvb, base + k_off + kv_k_at(w, lane + HALF, HD), k2);
      store_from_f32(kvb, base + v_off + kv_v_at(w, lane, a.kv_block), v1);
      store_from_f32(kvb, base + v_off + kv_v_at(w, lane + HALF, a.kv_block), v2);
    }
    wrote = true;
  }
  if (wrote) __threadfence_block();
}

// Query vectors j0 .. j0+NV of the block (vector j: row r_beg + j / G, head
// g G + j % G): per-head norm + RoPE, scaled by 1/sqrt(hd), into sm_q; vectors
// past nvec are zero.
template <typename TKV, int HD, int NV>
OSP_DEV void stage_queries(const AttnArgs& a, float (*sm_q)[HD], int j0, int nvec, int r_beg, int G,
                           int g, int wave, int lane) {
  constexpr int HALF = HD / 2;
  for (int j = wave; j < NV; j += 4) {
    const int jj = j0 + j;
    if (jj < nvec && a.q_prep) {
      const int r = r_beg + jj / G, h = g * G + jj % G;
      const float* qp = a.q_prep + ((long)r * a.nq + h) * HD;
      if (lane < HALF) { sm_q[j][lane] = qp[lane]; sm_q[j][lane + HALF] = qp[lane + HALF]; }
    } else if (jj < nvec) {
      const int r = r_beg + jj / G, h = g * G + jj % G;
      const long qo = (long)r * a.qkv_w + h * HD;
      float qv[2];
      qkv_lanes<HD, kBatchQkv<TKV, HD>>(a, {qo}, lane, qv);
      float q1 = qv[0], q2 = qv[1];
      norm_rope<TKV, HD>(a, a.q_norm, a.rows.pos[r], lane, q1, q2);
      if (lane < HALF) { sm_q[j][lane] = q1 * a.scale; sm_q[j][lane + HALF] = q2 * a.scale; }
    } else if (lane < HALF) {
      sm_q[j][lane] = 0.f;
      sm_q[j][lane + HALF] = 0.f;
    }
  }
}

template <typename TKV, int HD, int QV>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int DPL = HD / 16;         // head dims per lane (QV query vectors per pass)
  constexpr int PG = 16;               // tokens per KV page
  constexpr int HALF = HD / 2;
  __shared__ float sm_q[QV][HD];
  __shared__ float sm_m[4][QV];
  __shared__ float sm_l[4][QV];
  __shared__ float sm_o[4][QV][HD];

  int b, sp, slot;
  if (!attn_block(a, b, sp, slot)) return;
  const int g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int dseg = (lane & 15) * DPL;  // this lane's head dims
  const int tsub = lane >> 4;          // token within each group of 4
  int r_beg, r_end;
  if (a.cu) { r_beg = a.cu[b]; r_end = a.cu[b + 1]; } else { r_beg = b; r_end = b + 1; }
  const int rows_total = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  r_end = min(r_end, rows_total);
  if (r_beg >= r_end) return;
  const int G = a.nq / a.nkv;
  const int nvec = (r_end - r_beg) * G;
  const int first_new = a.rows.pos[r_beg];
  const int n_ctx = a.rows.pos[r_end - 1] + 1;
  const int p_lo = sp * a.split_len;
  if (p_lo >= n_ctx) return;           // beyond this sequence: the combine reads no partial here
  const int p_hi = min(n_ctx, p_lo + a.split_len);
  const int nblocks = a.slot_nblocks[slot];
  const int32_t* bt = a.block_table + (long)slot * a.max_blocks;
  TKV* kvb = reinterpret_cast<TKV*>(a.kv);
  const long blk_elems = kv_block_elems(a.n_layers, a.nkv, a.kv_block, HD);
  const long k_off = (((long)a.layer * 2 + 0) * a.nkv + g) * a.kv_block * HD;
  const long v_off = (((long)a.layer * 2 + 1) * a.nkv + g) * a.kv_block * HD;

  // ---- 0. prefetch this wavefront's first page if it holds only older positions -------
  Page<TKV, HD> pre;
  const int t_first = p_lo + wave * PG;
  const bool prefetched = t_first < p_hi && (a.q_prep || t_first + PG <= first_new) && t_first / PG < nblocks;
  if (prefetched) {
    const long base = (long)bt[t_first / PG] * blk_elems;
    pre.load(kvb + base + k_off, kvb + base + v_off, lane);
  }

  // ---- 1. keys/values of the new rows that fall in this split ------------------------
  if (!a.q_prep)
    append_new_kv<TKV, HD>(a, r_beg, r_end, p_lo, p_hi, bt, nblocks, kvb, blk_elems, k_off, v_off, g,
                           wave, lane);

  for (int j0 = 0; j0 < nvec; j0 += QV) {
    // ---- 2. this pass's query vectors: norm + RoPE into LDS (scaled by 1/sqrt(hd)) ----
    stage_queries<TKV, HD, QV>(a, sm_q, j0, nvec, r_beg, G, g, wave, lane);
    __syncthreads();
    float q[QV][DPL], o[QV][DPL], m[QV], l[QV];
    int qpos[QV];
#pragma unroll
    for (int j = 0; j < QV; ++j) {
      const int jj = j0 + j;
      m[j] = -INFINITY;
      l[j] = 0.f;
      qpos[j] = jj < nvec ? a.rows.pos[r_beg + jj / G] : -1;
#pragma unroll
      for (int e = 0; e < DPL; ++e) { o[j][e] = 0.f; q[j][e] = sm_q[j][dseg + e]; }
    }
    // ---- 3. walk the split's pages -------------------------------------------------------
    for (int t0 = t_first; t0 < p_hi; t0 += 4 * PG) {
      const int blk = t0 / PG;
      Page<TKV, HD> pg;
      if (j0 == 0 && t0 == t_first && prefetched) {
        pg = pre;
      } else if (blk < nblocks) {
        const long base = (long)bt[blk] * blk_elems;
        pg.load(kvb + base + k_off, kvb + base + v_off, lane);
      } else {
        pg.zero();
      }
#pragma unroll
      for (int j = 0; j < QV; ++j) {
        float sc[4];
        float bm = -INFINITY;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float s = 0.f;
#pragma unroll
          for (int e = 0; e < DPL; ++e) s = fmaf(q[j][e], pg.k[u].get(e), s);
          s += xor_lane_c(s, 1);
          s += xor_lane_c(s, 2);
          s += xor_lane_c(s, 4);
          s += xor_lane_c(s, 8);
          const int p = t0 + 4 * u + tsub;
          if (p >= p_hi || p > qpos[j] || blk >= nblocks) s = -INFINITY;
          sc[u] = s;
          bm = fmaxf(bm, s);
        }
        bm = fmaxf(bm, xor_lane_c(bm, 16));
        bm = fmaxf(bm, xor_lane_c(bm, 32));
        const float mn = fmaxf(m[j], bm);
        if (mn == -INFINITY) continue;
        const float so = __expf(m[j] - mn);
        l[j] *= so;
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] *= so;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          // masked tokens (past the sequence end: unwritten cache memory) contribute
          // nothing, not even 0 * NaN
          if (sc[u] > -INFINITY) {
            const float pe = __expf(sc[u] - mn);
            l[j] += pe;
#pragma unroll
            for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(pe, pg.v[u].get(e), o[j][e]);
          }
        }
        m[j] = mn;
      }
    }
    // ---- merge the 4 token groups of each wave (lanes l, l^16, l^32, l^48) -------------
#pragma unroll
    for (int j = 0; j < QV; ++j) {
#pragma unroll
      for (int sft = 16; sft < 64; sft <<= 1) {
        l[j] += xor_lane_c(l[j], sft);
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] += xor_lane_c(o[j][e], sft);
      }
      if (lane < 16) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) sm_o[wave][j][dseg + e] = o[j][e];
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

// Pages held in registers by each wavefront of k_attn_mfma (DEPTH - 1 in flight).
#ifndef OSP_ATTN_DEPTH
#define OSP_ATTN_DEPTH 2
#endif
constexpr int kAttnDepth = OSP_ATTN_DEPTH;

typedef __bf16 att_bf16x8 __attribute__((ext_vector_type(8)));
typedef short att_i16x4 __attribute__((ext_vector_type(4)));
typedef float att_f32x4 __attribute__((ext_vector_type(4)));

// One 16-token page as matrix-core operands: lane l holds
//   k[c] = K[token l%16][32 c + 8 (l/16) .. +8]          (A of S^T = K Q^T)
//   v[n] = V^T[16 n + l%16][tokens 4 (l/16) .. +4]       (A of O^T = V^T P^T)
typedef unsigned att_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned att_u32x2 __attribute__((ext_vector_type(2)));
// STREAM: non-temporal loads, for passes whose context outsizes the last-level cache
// (they read faster and leave the drafter's weights in that cache).
template <int HD> struct MPage {
  uint4 k[HD / 32];
  uint2 v[HD / 16];
  bool ok;   // a page of the sequence (else its words come from page 0 and are dropped)
  template <bool STREAM>
  OSP_DEV void load(const bf16_t* kb, const bf16_t* vb, int lane) {
    const int row = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) {
      const bf16_t* p = kb + kv_k_at(row, 32 * c + 8 * grp, HD);
      if constexpr (STREAM) {
        const att_u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const att_u32x4*>(p));
        k[c] = make_uint4(x[0], x[1], x[2], x[3]);
      } else {
        k[c] = *reinterpret_cast<const uint4*>(p);
      }
    }
#pragma unroll
    for (int n = 0; n < HD / 16; ++n) {
      const bf16_t* p = vb + kv_v_at(4 * grp, 16 * n + row, 16);
      if constexpr (STREAM) {
        const att_u32x2 x = __builtin_nontemporal_load(reinterpret_cast<const att_u32x2*>(p));
        v[n] = make_uint2(x[0], x[1]);
      } else {
        v[n] = *reinterpret_cast<const uint2*>(p);
      }
    }
  }
  OSP_DEV void zero() {
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) k[c] = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int n = 0; n < HD / 16; ++n) v[n] = make_uint2(0u, 0u);
  }
};

template <int HD, int DEPTH, bool STREAM>
__global__ void __launch_bounds__(256) k_attn_mfma(AttnArgs a) {
  constexpr int PG = 16;               // tokens per KV page
  constexpr int NV = 16;               // query vectors per pass
  constexpr int KC = HD / 32;          // 32-wide head-dim chunks of Q K^T
  constexpr int NT = HD / 16;          // 16-dim output tiles
  constexpr int OP = HD + 4;           // LDS pitch of the output merge
  __shared__ float sm_q[NV][HD];
  __shared__ float sm_m[4][NV];
  __shared__ float sm_l[4][NV];
  __shared__ __attribute__((aligned(16))) float sm_o[4][NV][OP];
  // Q^T fragments (hi, lo) in lane order; read from LDS at every page instead of
  // being held in registers, which leaves room for a deeper page ring
  __shared__ __attribute__((aligned(16))) uint4 sm_qf[KC][2][64];

  int b, sp, slot;
  if (!attn_block(a, b, sp, slot)) return;
  const int g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = lane & 15, grp = lane >> 4;
  // The slot comes with the work item (an argument for a batch of one), so that the
  // page-table entries of a whole split, the slot's page count and the row positions
  // are requested together and the first page follows after one round trip.
  const int32_t* bt = a.block_table + (long)slot * a.max_blocks;
  const int pg_lo = sp * a.split_len / PG;   // split_len is a multiple of a page
  // this wavefront's pages: split pages wave, wave + 4, ... (at most 64: the host keeps
  // split_len <= 4096), their page-table entries one per lane
  const int pid = pg_lo + wave + 4 * lane;
  const int n_pg_full = a.split_len / PG;
  const int n_mine_full = min(64, n_pg_full > wave ? (n_pg_full - wave + 3) / 4 : 0);
  const int bt_any = (lane < n_mine_full && pid < a.max_blocks) ? bt[pid] : -1;
  const int nblocks = a.slot_nblocks[slot];
  int r_beg, r_end;
  if (a.cu) { r_beg = a.cu[b]; r_end = a.cu[b + 1]; } else { r_beg = b; r_end = b + 1; }
  const int rows_total = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  r_end = min(r_end, rows_total);
  if (r_beg >= r_end) return;
  const int G = a.nq / a.nkv;
  const int nvec = (r_end - r_beg) * G;
  const int first_new = a.rows.pos[r_beg];
  const int n_ctx = a.rows.pos[r_end - 1] + 1;
  const int p_lo = sp * a.split_len;
  if (p_lo >= n_ctx) return;           // beyond this sequence: the combine reads no partial here
  const int p_hi = min(n_ctx, p_lo + a.split_len);
  bf16_t* kvb = reinterpret_cast<bf16_t*>(a.kv);
  const long blk_elems = kv_block_elems(a.n_layers, a.nkv, a.kv_block, HD);
  const long k_off = (((long)a.layer * 2 + 0) * a.nkv + g) * a.kv_block * HD;
  const long v_off = (((long)a.layer * 2 + 1) * a.nkv + g) * a.kv_block * HD;

  // the pages that hold positions of this split (-1: beyond the slot's pages)
  const int n_pg = p_hi > p_lo ? (p_hi - p_lo + PG - 1) / PG : 0;
  const int n_mine = min(64, n_pg > wave ? (n_pg - wave + 3) / 4 : 0);
  const int bt_reg = (lane < n_mine && pid < nblocks) ? bt_any : -1;
  // Every page is requested with no condition on its index or its table entry: with a
  // load under a condition the compiler cannot count the loads in flight, and it then
  // waits for all of them -- the pages requested ahead included -- before using one.
  // A missing table entry, or an index past the wavefront's pages (i >= n_mine: a
  // request the ring makes at its end), reads page 0 (always in the pool, and cached
  // after the first such read) and is dropped in page_step or never used.
  auto load_page = [&](MPage<HD>& pg, int i) {
    const int e = lane_i(bt_reg, min(i, OSP_WAVE - 1));
    const int phys = i < n_mine ? e : -1;
    pg.ok = phys >= 0;
    const long base = (long)max(phys, 0) * blk_elems;
    pg.template load<STREAM>(kvb + base + k_off, kvb + base + v_off, lane);
  };

  // ---- 0. the first page early when it holds only older positions ---------------------
  MPage<HD> ring[DEPTH];
  const bool early = n_mine > 0 && (a.q_prep || (pg_lo + wave + 1) * PG <= first_new);
  if (early) load_page(ring[0], 0);

  // ---- 1. keys/values of the new rows that fall in this split ------------------------
  if (!a.q_prep)
    append_new_kv<bf16_t, HD>(a, r_beg, r_end, p_lo, p_hi, bt, nblocks, kvb, blk_elems, k_off, v_off,
                              g, wave, lane);

  for (int j0 = 0; j0 < nvec; j0 += NV) {
    // ---- 2. queries: norm + RoPE into LDS, then Q^T fragments as bf16 hi / lo ---------
    stage_queries<bf16_t, HD, NV>(a, sm_q, j0, nvec, r_beg, G, g, wave, lane);
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        uint32_t h[4], l[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          split_bf16x2(sm_q[row][32 * c + 8 * grp + 2 * e], sm_q[row][32 * c + 8 * grp + 2 * e + 1], h[e], l[e]);
        sm_qf[c][0][lane] = make_uint4(h[0], h[1], h[2], h[3]);
        sm_qf[c][1][lane] = make_uint4(l[0], l[1], l[2], l[3]);
      }
    }
    __syncthreads();
    const int qj = j0 + row;
    const int qpos = qj < nvec ? a.rows.pos[r_beg + qj / G] : -1;
    // consume qpos here: a first use inside the page loop would make every iteration
    // wait for all outstanding loads, the page prefetches included
    asm volatile("" ::"v"(qpos));
    float m = -INFINITY, lsum = 0.f;
    att_f32x4 acc[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] = att_f32x4{0.f, 0.f, 0.f, 0.f};

    // ---- 3. pages: a ring of DEPTH register pages, DEPTH - 1 requested ahead; the
    //      ring is unrolled so that no page is copied between registers (a copy would
    //      wait for its load and stall the pipeline) ------------------------------------
    auto page_step = [&](MPage<HD>& pg, int i) {
      const int t0 = (pg_lo + wave + 4 * i) * PG;
      // S^T[token][query]: lane holds tokens 4 grp + e of query `row`
      att_f32x4 sc = att_f32x4{0.f, 0.f, 0.f, 0.f};
      // (the opaque lane index keeps the compiler from hoisting these reads out of the
      // page loop into registers)
      int ql_ = lane;
      asm volatile("" : "+v"(ql_));
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const att_bf16x8 ka = *reinterpret_cast<const att_bf16x8*>(&pg.k[c]);
        const uint4 qh = sm_qf[c][0][ql_], qlo = sm_qf[c][1][ql_];
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, *reinterpret_cast<const att_bf16x8*>(&qh), sc, 0, 0, 0);
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, *reinterpret_cast<const att_bf16x8*>(&qlo), sc, 0, 0, 0);
      }
      // causal / sequence-end mask; value entries past the sequence end are cleared so
      // that unwritten cache memory cannot reach the products (0 * NaN)
      float s4[4];
      float bm = -INFINITY;
      uint32_t keep[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int p = t0 + 4 * grp + e;
        const bool in = pg.ok && p < p_hi;
        s4[e] = (in && p <= qpos) ? sc[e] : -INFINITY;
        bm = fmaxf(bm, s4[e]);
        if (in) keep[e >> 1] |= (e & 1) ? 0xffff0000u : 0x0000ffffu;
      }
#pragma unroll
      for (int n = 0; n < NT; ++n) { pg.v[n].x &= keep[0]; pg.v[n].y &= keep[1]; }
      bm = fmaxf(bm, xor_lane_c(bm, 16));
      bm = fmaxf(bm, xor_lane_c(bm, 32));
      const float mn = fmaxf(m, bm);
      const float f = (mn == -INFINITY) ? 1.f : __expf(m - mn);
      float pe[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) pe[e] = (s4[e] == -INFINITY) ? 0.f : __expf(s4[e] - mn);
      lsum = lsum * f + ((pe[0] + pe[1]) + (pe[2] + pe[3]));
      m = mn;
      uint2 ph2, pl2;
      split_bf16x2(pe[0], pe[1], ph2.x, pl2.x);
      split_bf16x2(pe[2], pe[3], ph2.y, pl2.y);
      const att_i16x4 ph = *reinterpret_cast<const att_i16x4*>(&ph2);
      const att_i16x4 pl = *reinterpret_cast<const att_i16x4*>(&pl2);
      // O^T[dim][query] += V^T P^T
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        acc[n] *= f;
        const att_i16x4 va = *reinterpret_cast<const att_i16x4*>(&pg.v[n]);
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, ph, acc[n], 0, 0, 0);
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pl, acc[n], 0, 0, 0);
      }
    };
    if (n_mine > 0) {
      if (!(early && j0 == 0)) load_page(ring[0], 0);
#pragma unroll
      for (int u = 1; u + 1 < DEPTH; ++u) load_page(ring[u], u);
    }
    for (int i0 = 0; i0 < n_mine; i0 += DEPTH) {
#pragma unroll
      for (int u = 0; u < DEPTH; ++u) {
        const int i = i0 + u;
        if (i < n_mine) {
          load_page(ring[(u + DEPTH - 1) % DEPTH], i + DEPTH - 1);
          page_step(ring[u], i);
        }
      }
    }
    // ---- merge the wavefronts: lane holds O^T[16 n + 4 grp + e][row] ------------------
    lsum += xor_lane_c(lsum, 16);
    lsum += xor_lane_c(lsum, 32);
    if (grp == 0) { sm_m[wave][row] = m; sm_l[wave][row] = lsum; }
#pragma unroll
    for (int n = 0; n < NT; ++n)
      *reinterpret_cast<float4*>(&sm_o[wave][row][16 * n + 4 * grp]) =
          make_float4(acc[n][0], acc[n][1], acc[n][2], acc[n][3]);
    __syncthreads();
    for (int i = tid; i < NV * HD; i += 256) {
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
          const float fw = __expf(sm_m[w][j] - M);
          L += sm_l[w][j] * fw;
          O += sm_o[w][j][e] * fw;
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

// Matrix-core path, once per row: the QKV split partials are added, q and k
// normalised (per head) and rotated, q scaled by 1/sqrt(hd) into q_out and the
// new key/value stored in the row's cache page.  Block (row, group of 4 heads);
// wavefront w handles head 4 y + w of the nq query heads followed by the nkv
// key/value heads.
template <typename TKV, int HD>
__global__ void __launch_bounds__(256) k_rows_qkv(AttnArgs a, float* q_out) {
  constexpr int HALF = HD / 2;
  const int r = blockIdx.x;
  const int rows = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  if (r >= rows) return;
  const int lane = threadIdx.x & 63;
  const int hh = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (hh >= a.nq + a.nkv) return;
  // (a draft-tree row: its own position for RoPE; rows.pos bounds the context read)
  const int pos = a.tree_pos ? a.tree_pos[r] : a.rows.pos[r];
  if (hh < a.nq) {
    const long qo = (long)r * a.qkv_w + (long)hh * HD;
    float qv[2];
    qkv_lanes<HD, true>(a, {qo}, lane, qv);
    float q1 = qv[0], q2 = qv[1];
    norm_rope<TKV, HD>(a, a.q_norm, pos, lane, q1, q2);
    if (lane < HALF) {
      float* qp = q_out + ((long)r * a.nq + hh) * HD;
      qp[lane] = q1 * a.scale;
      qp[lane + HALF] = q2 * a.scale;
    }
    return;
  }
  const int g = hh - a.nq;
  const long ko = (long)r * a.qkv_w + (long)(a.nq + g) * HD;
  const long vo = (long)r * a.qkv_w + (long)(a.nq + a.nkv + g) * HD;
  float kv[4];
  qkv_lanes<HD, true>(a, {ko, vo}, lane, kv);
  float k1 = kv[0], k2 = kv[1];
  const float v1 = kv[2], v2 = kv[3];
  norm_rope<TKV, HD>(a, a.k_norm, pos, lane, k1, k2);
  if (a.tree_node) {
    // draft tree: into the tree cache at the node's slot, [layer][k | v][kv head][dim]
    if (a.tree_node[r] < 0 || a.tree_node[r] >= a.tree_slots) { if (lane == 0) atomicOr(a.err, 1u << 3); return; }
    TKV* tk = reinterpret_cast<TKV*>(a.tree_kv);
    const long kb = ((((long)a.tree_node[r] * a.n_layers + a.layer) * 2 + 0) * a.nkv + g) * HD;
    const long vb = kb + (long)a.nkv * HD;
    if (lane < HALF) {
      store_from_f32(tk, kb + lane, k1);
      store_from_f32(tk, kb + lane + HALF, k2);
      store_from_f32(tk, vb + lane, v1);
      store_from_f32(tk, vb + lane + HALF, v2);
    }
    return;
  }
  const int b = a.rows.seq ? a.rows.seq[r] : r;
  const int slot = a.slot0 >= 0 ? a.slot0 : a.bslot[b];
  const int blk = pos / a.kv_block;
  if (blk >= a.slot_nblocks[slot]) { if (lane == 0) atomicOr(a.err, 1u << 3); return; }
  TKV* kvb = reinterpret_cast<TKV*>(a.kv);
  const long base = (long)a.block_table[(long)slot * a.max_blocks + blk] *
                    kv_block_elems(a.n_layers, a.nkv, a.kv_block, HD);
  const long k_off = (((long)a.layer * 2 + 0) * a.nkv + g) * a.kv_block * HD;
  const long v_off = (((long)a.layer * 2 + 1) * a.nkv + g) * a.kv_block * HD;
  const int w = pos - blk * a.kv_block;
  if (lane < HALF) {
    store_from_f32(kvb, base + k_off + kv_k_at(w, lane, HD), k1);
    store_from_f32(kvb, base + k_off + kv_k_at(w, lane + HALF, HD), k2);
    store_from_f32(kvb, base + v_off + kv_v_at(w, lane, a.kv_block), v1);
    store_from_f32(kvb, base + v_off + kv_v_at(w, lane + HALF, a.kv_block), v2);
  }
}

// One block per (row, head).  Every thread requests its share of the split outputs
// at once (dimension tid % hd, splits tid / hd, + 256 / hd, ...) while wavefront 0
// reads the splits' (max, sum); the weights exp(m_s - M) / L come through LDS and the
// thread groups are added in LDS, in a fixed order.
// A draft-tree row's attention over its ancestors' and its own keys/values in the tree
// cache (one wavefront): the (max, sum, unnormalised output) of one more split.  Every
// ancestor's key and value are requested at once (slots clamped into the cache; the
// -1 padding masked afterwards), then scored and summed.
template <int HD>
OSP_DEV void tree_partial(const AttnArgs& a, int r, int h, int lane, float& m, float& l, float* s_o) {
  constexpr int DPL = HD / OSP_WAVE;              // head dims per lane
  const int g = h / (a.nq / a.nkv);
  const float* q = a.q_prep + ((long)r * a.nq + h) * HD;
  const bf16_t* kv = reinterpret_cast<const bf16_t*>(a.tree_kv);
  const int my = lane < kMaxTreeDepth ? a.tree_anc[r * kMaxTreeDepth + lane] : -1;
  float qv[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) qv[e] = q[lane * DPL + e];
  float kx[kMaxTreeDepth][DPL], vx[kMaxTreeDepth][DPL];
  bool ok[kMaxTreeDepth];
  bool run = true;                                // leading valid slots only
#pragma unroll
  for (int i = 0; i < kMaxTreeDepth; ++i) {
    const int slot = lane_i(my, i);
    run = run && slot >= 0 && slot < a.tree_slots;
    ok[i] = run;
    const long kb = ((((long)(run ? slot : 0) * a.n_layers + a.layer) * 2 + 0) * a.nkv + g) * HD + lane * DPL;
    const long vb = kb + (long)a.nkv * HD;
#pragma unroll
    for (int e = 0; e < DPL; ++e) { kx[i][e] = load_f32(kv, kb + e); vx[i][e] = load_f32(kv, vb + e); }
  }
  float sc[kMaxTreeDepth];
  m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxTreeDepth; ++i) {
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) d += qv[e] * kx[i][e];
    d = wave_sum(d);
    sc[i] = ok[i] ? d : -INFINITY;
    m = fmaxf(m, sc[i]);
  }
  float o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  l = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxTreeDepth; ++i) {
    const float w = ok[i] ? __expf(sc[i] - m) : 0.f;
    l += w;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] += w * vx[i][e];
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) s_o[lane * DPL + e] = o[e];
}

template <int HD>
__global__ void __launch_bounds__(256) k_attn_combine(AttnArgs a) {
  constexpr int G = 256 / HD;              // thread groups (splits interleaved)
  constexpr int PER = kMaxSplitAttn / G;   // splits per thread (bound)
  __shared__ float s_f[kMaxSplitAttn];
  __shared__ float s_part[G][HD];
  __shared__ float s_to[HD];               // a draft-tree row's partial over its ancestors
  const int r = blockIdx.x, h = blockIdx.y;
  const int rows = a.rows.count ? min(*a.rows.count, a.rows.max_rows) : a.rows.max_rows;
  if (r >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int e = tid % HD, grp = tid / HD;
  // splits that hold any position visible to this row (later ones were not written)
  const int ns = min(a.n_split, a.rows.pos[r] / a.split_len + 1);
  const float* pp = a.part + ((long)r * a.nq + h) * a.n_split * (HD + 2);
  // every split's values are requested before the row position arrives; those of
  // splits past ns (not written for this row) are discarded by selection
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int sp = grp + G * i;
    v[i] = sp < a.n_split ? pp[(long)sp * (HD + 2) + 2 + e] : 0.f;
  }
  // (a draft-tree row: one more split after the context's, its attention over its
  // ancestors and itself)
  const bool tree = a.tree_node != nullptr;
  const int extra = tree ? a.n_split : -1;
  if (tid < 64) {
    float m_any = lane < a.n_split ? pp[(long)lane * (HD + 2)] : -INFINITY;
    float l_any = lane < a.n_split ? pp[(long)lane * (HD + 2) + 1] : 0.f;
    if (tree) {
      float tm, tl;
      tree_partial<HD>(a, r, h, lane, tm, tl, s_to);
      if (lane == extra) { m_any = tm; l_any = tl; }
    }
    const bool use = lane < ns || lane == extra;
    const float m = use ? m_any : -INFINITY;
    const float lsum = use ? l_any : 0.f;
    const float M = wave_max(m);
    const float f = (m > -INFINITY) ? __expf(m - M) : 0.f;
    const float L = wave_sum(lsum * f);
    s_f[lane] = L > 0.f ? f / L : 0.f;
  }
  __syncthreads();
  float O = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int sp = grp + G * i;
    if (sp < ns) O += v[i] * s_f[sp];
  }
  if (tree && grp == 0) O += s_to[e] * s_f[extra];
  s_part[grp][e] = O;
  __syncthreads();
  if (tid < HD) {
    float y = 0.f;
#pragma unroll
    for (int g2 = 0; g2 < G; ++g2) y += s_part[g2][tid];
    const long o = (long)r * a.nq * HD + h * HD + tid;
    if (a.o_hi) {
      const bf16_t yh = f32_to_bf16(y);
      a.o_hi[o] = yh;
      a.o_lo[o] = f32_to_bf16(y - bf16_to_f32(yh));
    } else {
      a.o[o] = y;
    }
  }
}

// Query vectors per pass: enough for every row of a sequence times its GQA group,
// at most 8 (head_dim 128) or 16 (head_dim 64) so q + o stay within 128 registers.
template <typename TKV, int HD>
static void launch_hd(const AttnArgs& a, hipStream_t st) {
  dim3 grid(a.nkv, a.B * a.n_split);
  const int need = a.rows_per_seq * (a.nq / a.nkv);
  constexpr int QMAX = 1024 / HD;
  if (need <= 1) hipLaunchKernelGGL((k_attn<TKV, HD, 1>), grid, dim3(256), 0, st, a);
  else if (need <= 2) hipLaunchKernelGGL((k_attn<TKV, HD, 2>), grid, dim3(256), 0, st, a);
  else if (need <= 4 || QMAX == 4) hipLaunchKernelGGL((k_attn<TKV, HD, 4>), grid, dim3(256), 0, st, a);
  else if (need <= 8 || QMAX == 8) hipLaunchKernelGGL((k_attn<TKV, HD, (QMAX >= 8 ? 8 : 4)>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((k_attn<TKV, HD, QMAX>), grid, dim3(256), 0, st, a);
}

void launch_attention(int kvdtype, const AttnArgs& a, hipStream_t st) {
  if (kvdtype == 1) {
    dim3 grid(a.nkv, a.B * a.n_split);
    if (a.kv_stream) {
      if (a.hd == 128) hipLaunchKernelGGL((k_attn_mfma<128, kAttnDepth, true>), grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL((k_attn_mfma<64, kAttnDepth, true>), grid, dim3(256), 0, st, a);
    } else {
      if (a.hd == 128) hipLaunchKernelGGL((k_attn_mfma<128, kAttnDepth, false>), grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL((k_attn_mfma<64, kAttnDepth, false>), grid, dim3(256), 0, st, a);
    }
  } else {
    if (a.hd == 128) launch_hd<float, 128>(a, st); else launch_hd<float, 64>(a, st);
  }
}

void launch_rows_qkv(int kvdtype, const AttnArgs& a, float* q_out, hipStream_t st) {
  dim3 grid(a.rows.max_rows, (a.nq + a.nkv + 3) / 4);
  if (kvdtype == 1) {
    if (a.hd == 128) hipLaunchKernelGGL((k_rows_qkv<bf16_t, 128>), grid, dim3(256), 0, st, a, q_out);
    else hipLaunchKernelGGL((k_rows_qkv<bf16_t, 64>), grid, dim3(256), 0, st, a, q_out);
  } else {
    if (a.hd == 128) hipLaunchKernelGGL((k_rows_qkv<float, 128>), grid, dim3(256), 0, st, a, q_out);
    else hipLaunchKernelGGL((k_rows_qkv<float, 64>), grid, dim3(256), 0, st, a, q_out);
  }
}

void launch_attn_combine(const AttnArgs& a, hipStream_t st) {
  if (a.hd == 128) hipLaunchKernelGGL(k_attn_combine<128>, dim3(a.rows.max_rows, a.nq), dim3(256), 0, st, a);
  else hipLaunchKernelGGL(k_attn_combine<64>, dim3(a.rows.max_rows, a.nq), dim3(256), 0, st, a);
}

}  // namespace osp

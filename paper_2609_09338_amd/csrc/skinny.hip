// Weight-streaming products on the matrix cores for passes of 1..64 input rows:
// the vocabulary-aligned LM head and the drafter's projections.
//
//   Y[r][n] = X[r] . W[n]        (W row-major [N][K] bf16, fp32 accumulation)
//
// LM head (Section 3.3, Eq. 4: head rows indexed by the drafter vocabulary and
// mapped to target ids through d2t; rows without a target id are masked): the
// epilogue writes the masked logits and, for every wavefront's contiguous range
// of vocabulary rows, a softmax record (max, sum exp((l - max) / T), lowest
// argmax) per input row, which the sampling kernel merges.
// Projections (tap projection of Eq. 1, expanded QKV of Eq. 2-3, O, gate/up, down):
// K is split across blocks (blockIdx.y) and every block writes its partial sums
// to [split][row][N] for the row kernel that follows (gate/up: the up matrix as
// rows [N, 2N)).
//
// A block (8 wavefronts) copies its input columns (all R <= 16 MT rows, as bf16
// hi / lo pairs) into LDS; after that every wavefront works alone, with no further
// block barrier: it streams its T tiles of 16 weight rows in units of 16 rows x
// 256 columns (8 KB) through a ring of three register buffers (two units in
// flight while it multiplies the third), each unit feeding 8 K steps of
// v_mfma_f32_16x16x32_bf16 for every M tile, hi and lo (taps are exact bf16: hi
// only).  Two MFMAs per product keep about 16 significant bits of every input,
// so the result stays close to fp32.
//
// Inputs: prepared pairs (two segments [xs ; xa] for the expanded QKV), one fp32
// row normalised here (LM head after the batch-1 vector body), or bf16 taps rows.
// The single normalised row is staged whole, once, before the stream starts: its
// loads are issued ahead of the first weight units (a load waits for every load
// issued before it), and the K phases then follow one another with no barrier or
// input copy.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace osp {

typedef __bf16 sk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float sk_f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned sk_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSkWaves = 8;
constexpr int kSkThreads = kSkWaves * 64;
constexpr int kSkUnit = 256;              // weight columns per streamed unit
constexpr int kSkDepthMax = 3;            // register ring of units (64 rows: 2)
constexpr int kSkTmaxHead = 5;            // tiles per wavefront (bound): LM head
constexpr int kSkTmaxProj = 1;            // projections: one tile, K split across blocks

enum SkSrc { SK_PREP = 0, SK_NORM = 1, SK_TAPS = 2, SK_SWIGLU = 3, SK_ATTN = 4 };
enum SkEpi { SK_LOGITS = 0, SK_PART = 1 };

// Input columns resident per block and phase: 64 rows x 512 or 32 rows x 1024
// columns of hi / lo pairs fill 132 KB of LDS.
template <int MT> struct SkCfg { static constexpr int KC = MT == 4 ? 512 : 1024; };

// T: tiles per wavefront (LM head); kc: K columns per block (projections, a multiple
// of 256 up to KC).
template <int MT, int SRC, int EPI>
__global__ void __launch_bounds__(kSkThreads) k_skinny(GemvArgs a, int T, int kc) {
  constexpr int KC = SkCfg<MT>::KC;
  constexpr int ROWS = 16 * MT;
  // bf16 per LDS row: a 32-byte skew per row.  (A 16-byte skew -- or 48, 80 -- left the
  // A-fragment reads about 3.7 bank-conflict cycles per instruction; 32 bytes leaves
  // none, rocprofv3 SQ_LDS_BANK_CONFLICT.)
  constexpr int PITCH = KC + 16;
  constexpr int NCH = KC / kSkUnit;       // units per tile and phase
  constexpr int TMAX = EPI == SK_LOGITS ? kSkTmaxHead : kSkTmaxProj;
  constexpr int NU = TMAX * NCH;          // units per phase (bound)
  constexpr bool EXACT = SRC == SK_TAPS;  // bf16 inputs: no lo part
  // ring depth: 64-row passes hold 80 accumulators and need the registers
  constexpr int kSkDepth = MT == 4 ? 2 : kSkDepthMax;
  __shared__ __attribute__((aligned(16))) bf16_t xh[ROWS * PITCH];
  __shared__ __attribute__((aligned(16))) bf16_t xl[EXACT ? 8 : ROWS * PITCH];

  // (the LM head takes the wavefront index through readfirstlane: the compiler then
  // knows that its tile range and every condition on it are uniform, and tests them
  // with scalar branches instead of masking each unit and store; the projections,
  // one tile per wavefront, measured slower that way)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = EPI == SK_LOGITS ? __builtin_amdgcn_readfirstlane(tid >> 6) : tid >> 6;
  const int wrow = lane & 15, grp = lane >> 4;
  // rows of this pass: the device-side count when there is one (the host bound may
  // exceed it, and index rows past it, such as tap_row entries, are stale)
  const int R = min(a.count ? min(*a.count, a.max_rows) : a.max_rows, ROWS);
  const int wg = blockIdx.x * kSkWaves + wave;          // record index (LM head)
  const int NR = (EPI == SK_PART && a.w1) ? 2 * a.N : a.N;   // weight rows
  const int nt16 = (NR + 15) >> 4;
  const int t0 = wg * T;
  const int ntiles = max(0, min(min(T, TMAX), nt16 - t0));
  const int k_lo = EPI == SK_PART ? blockIdx.y * kc : 0;
  const int k_hi = EPI == SK_PART ? min(a.Kd, k_lo + kc) : a.Kd;
  // units per tile and phase (attention outputs: one 256-column unit, a constant, so that
  // the prefetch below is known to be a single unit)
  const int nch = EPI == SK_PART ? (SRC == SK_ATTN ? 1 : kc / kSkUnit) : NCH;
  // LM head blocks with no tile at all leave at once (block-uniform, before any barrier)
  if (EPI == SK_LOGITS && blockIdx.x * kSkWaves * T >= nt16) return;

  sk_f32x4 acc[TMAX][MT];
#pragma unroll
  for (int j = 0; j < TMAX; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = sk_f32x4{0.f, 0.f, 0.f, 0.f};

  // Addresses are clamped into the matrix instead of masking the loaded values: a
  // select on a loaded register would wait for that load and serialise the ring.
  // Rows past the matrix only produce outputs that the epilogue drops; columns
  // past Kd meet zero inputs in LDS (the clamped weights are finite).
  auto load_unit = [&](uint4* w, int k0, int u) {
    const int n = min((t0 + u / nch) * 16 + wrow, NR - 1);
    const int kb = k0 + (u % nch) * kSkUnit + 8 * grp;
    const bf16_t* wr = (n < a.N) ? reinterpret_cast<const bf16_t*>(a.w0) + (long)n * a.Kd
                                 : reinterpret_cast<const bf16_t*>(a.w1) + (long)(n - a.N) * a.Kd;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      w[ks] = *reinterpret_cast<const uint4*>(wr + min(kb + 32 * ks, a.Kd - 8));
  };
  // LM head: the packed copy (pack_head_index), one contiguous kilobyte per load of the
  // wavefront.  The head is read once per pass and outsizes the last-level cache, so
  // its loads are non-temporal: they leave the drafter body's weights and the KV cache,
  // which every draft step reads again, in that cache.  Tiles past the head and units
  // past Kd are clamped into the copy (their products are dropped, or meet zero inputs).
  auto load_unit_packed = [&](uint4* w, int k0, int u) {
    const int nu_row = (a.Kd + kSkUnit - 1) / kSkUnit;
    const int t = min(t0 + u / nch, nt16 - 1);
    const int uu = min(k0 / kSkUnit + u % nch, nu_row - 1);
    const sk_u32x4* p = reinterpret_cast<const sk_u32x4*>(a.w0) + (long)(t * nu_row + uu) * 8 * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const sk_u32x4 v = __builtin_nontemporal_load(p + 64 * ks);
      w[ks] = make_uint4(v[0], v[1], v[2], v[3]);
    }
  };
  auto load = [&](uint4* w, int k0, int u) {
    if constexpr (EPI == SK_LOGITS) load_unit_packed(w, k0, u);
    else load_unit(w, k0, u);
  };
  // (attention outputs: one 256-column unit, one phase; a constant, so that nothing of
  // the merge is hoisted out of a phase loop ahead of the loads it should follow)
  const int nphase = SRC == SK_ATTN ? 1 : (k_hi - k_lo + KC - 1) / KC;
  const int nu = ntiles * nch;                          // units per phase
  // single normalised row: thread t stages columns [8t, 8t + 8) (Kd <= 8 x 512), read
  // before the weights are requested (addresses clamped into the row; pieces past Kd
  // are neither summed nor stored)
  float4 nx0, nx1;
  uint4 ng;
  if constexpr (SRC == SK_NORM) {
    const float* xr = a.xin + (long)(a.gather ? a.gather[0] : 0) * a.ldx;
    const int c = min(tid * 8, a.Kd - 8);
    nx0 = *reinterpret_cast<const float4*>(xr + c);
    nx1 = *reinterpret_cast<const float4*>(xr + c + 4);
    ng = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16_t*>(a.gamma) + c);
  }
  uint4 ring[kSkDepth][8];
  // units whose columns start at or past k_hi (the last phase of a K that is not a
  // multiple of KC) are neither loaded nor multiplied
  auto real = [&](int k0, int u) { return u < nu && k0 + (u % nch) * kSkUnit < k_hi; };
  // the first units of a phase are requested before its inputs are staged.  The
  // single normalised row, and the attention outputs' one unit, request them with no
  // condition (the addresses are clamped; a unit that is not real is never used), so
  // that the waits on the input loads need not assume an unknown number of loads in
  // between; elsewhere a unit past the block's range could be a whole unit of another
  // block's weights
  auto prefetch_phase = [&](int k0) {
#pragma unroll
    for (int u = 0; u + 1 < kSkDepth; ++u)
      if (SRC == SK_NORM || (SRC == SK_ATTN && u == 0) || real(k0, u)) load(ring[u], k0, u);
  };
  // attention outputs: the merge records of item t = (row, head of the K range) and the
  // item's row position, requested first (the merge weights wait for these alone)
  constexpr int kSkAttnHeads = 4;   // heads of at least 64 columns in a 256-column K range
  const int t_r = tid / kSkAttnHeads, t_hh = tid % kSkAttnHeads;
  float2 ml[SRC == SK_ATTN ? kAttnMergeMaxSplit : 1];
  int t_pos = 0;
  if constexpr (SRC == SK_ATTN) {
    const int hd = a.attn_hd, nh = a.Kd / hd, ns_all = a.attn_nsplit;
    const int t_h = min(k_lo / hd + t_hh, nh - 1), t_rc = min(t_r, min(a.max_rows, ROWS) - 1);
    const float* pm = a.attn_part + ((long)t_rc * nh + t_h) * ns_all * (hd + 2);
#pragma unroll
    for (int sp = 0; sp < kAttnMergeMaxSplit; ++sp)
      ml[sp] = *reinterpret_cast<const float2*>(pm + (long)min(sp, ns_all - 1) * (hd + 2));
    t_pos = a.attn_pos[t_rc];
  }
  prefetch_phase(k_lo);
  // LM head: the map entries of this lane's columns (one per tile), read from a clamped
  // address with no condition: a value tested where it is loaded would make the
  // wavefront wait there for every load issued before it (the weights)
  int dmap[TMAX];
#pragma unroll
  for (int j = 0; j < TMAX; ++j)
    dmap[j] = EPI == SK_LOGITS ? a.d2t[min((t0 + j) * 16 + wrow, a.N - 1)] : 0;
  // ... and the temperatures of the lane's output rows 16 mt + 4 grp + e (row r of the
  // pass is sequence r), requested now so that the epilogue does not wait for them
  constexpr int NTK = EPI == SK_LOGITS ? 4 * MT : 1;
  float tk[NTK];
#pragma unroll
  for (int k = 0; k < NTK; ++k)
    tk[k] = EPI == SK_LOGITS ? a.temp[min((k / 4) * 16 + 4 * grp + (k % 4), R - 1)] : 0.f;
  if constexpr (SRC == SK_NORM) {
    // RMS of the row (wavefront sums, then the block's in a fixed order), then the
    // normalised row as hi / lo pairs at LDS columns [0, Kd)
    __shared__ float s_ss[kSkWaves];
    const int c = tid * 8;
    const bool in = c < a.Kd;
    float ss = 0.f;
    if (in)
      ss = nx0.x * nx0.x + nx0.y * nx0.y + nx0.z * nx0.z + nx0.w * nx0.w +
           nx1.x * nx1.x + nx1.y * nx1.y + nx1.z * nx1.z + nx1.w * nx1.w;
    ss = wave_sum(ss);
    if (lane == 0) s_ss[wave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kSkWaves; ++w) tot += s_ss[w];
    const float inv = 1.0f / sqrtf(tot / (float)a.Kd + a.eps);
    if (!in && c < nphase * KC) {   // columns of the last phase past Kd meet zeros
      *reinterpret_cast<uint4*>(xh + c) = make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(xl + c) = make_uint4(0u, 0u, 0u, 0u);
    }
    if (in) {
      uint4 h, l;
      split_bf16x2(nx0.x * inv * bf16_lo(ng.x), nx0.y * inv * bf16_hi(ng.x), h.x, l.x);
      split_bf16x2(nx0.z * inv * bf16_lo(ng.y), nx0.w * inv * bf16_hi(ng.y), h.y, l.y);
      split_bf16x2(nx1.x * inv * bf16_lo(ng.z), nx1.y * inv * bf16_hi(ng.z), h.z, l.z);
      split_bf16x2(nx1.z * inv * bf16_lo(ng.w), nx1.w * inv * bf16_hi(ng.w), h.w, l.w);
      *reinterpret_cast<uint4*>(xh + c) = h;
      *reinterpret_cast<uint4*>(xl + c) = l;
      // the fp32 row is also the next draft step's conditioning input: block 0 copies it
      if (a.fb_out && blockIdx.x == 0) {
        *reinterpret_cast<float4*>(a.fb_out + c) = nx0;
        *reinterpret_cast<float4*>(a.fb_out + c + 4) = nx1;
      }
    }
    __syncthreads();
  }
  __shared__ float s_af[SRC == SK_ATTN ? ROWS * kSkAttnHeads * kAttnMergeMaxSplit : 1];
  for (int ph = 0; ph < nphase; ++ph) {
    const int k0 = k_lo + ph * KC;
    if constexpr (SRC != SK_NORM) {
    if (ph > 0) __syncthreads();
    // ---- inputs of this phase into LDS: rows r < R and the columns this block reads
    //      (the projections' K range, or the whole phase); columns past k_hi are zero.
    //      Rows past R are left as they are: they only feed outputs that are dropped.
    //      Each thread requests a batch of 16-byte pieces before storing any, so the
    //      copy costs a round trip or two instead of one per piece ------------------------
    const int span8 = (EPI == SK_PART ? kc : KC) / 8;      // 16-byte pieces per row
    const int nitems = R * span8;
    // (the LM head holds 20 MT accumulators: smaller batches for more rows)
    // (SwiGLU inputs, at most 16 rows: one piece per thread at the usual K range, each
    // piece kSwRound splits' loads)
    constexpr int BATCH = EPI == SK_LOGITS ? (MT == 4 ? 1 : (MT == 2 ? 2 : 4)) : (SRC == SK_SWIGLU ? 1 : 4);
    constexpr int kSwRound = 4;
    if constexpr (SRC == SK_ATTN) {
      // Attention outputs (K range of one 256-column unit: 32 pieces per row, MT pieces
      // per thread).  Piece (row r, columns c .. c + 7 = dims e .. e + 7 of head hq) is
      // the splits' unnormalised outputs weighted by f_s / L (the merge of max-rescaled
      // splits, M the largest max of the row's splits), added in split order.  Thread t
      // also computes the weights of item t = (row, head of the range).  Everything is
      // requested at once with the unit of weights: the items' positions and split
      // records, then the first AS splits' outputs of the pieces (32 float2 per thread:
      // 1 x 8 at 16 rows, 2 x 4 at 32, 4 x 2 at 64), from clamped addresses below the
      // host's row bound, so that no load waits on the device row count or a position.
      // A split past the row's own count (weight 0) is dropped by selection, never
      // multiplied (its record may be stale); rows past the count are not stored.  (The
      // items' records were requested before the weights, above.)
      constexpr int AB = MT, AS = kAttnMergeMaxSplit / MT;
      const int hd = a.attn_hd, nh = a.Kd / hd, ns_all = a.attn_nsplit, rec = hd + 2;
      const int rb = min(a.max_rows, ROWS);
      const int h0 = k_lo / hd;
      // the pieces' outputs, first round
      const float* pp[AB];
      int pr[AB], pc[AB];
#pragma unroll
      for (int q = 0; q < AB; ++q) {
        const int i = tid + q * kSkThreads;
        pr[q] = i / span8;
        pc[q] = (i - pr[q] * span8) * 8;
        const int c = min(k0 + pc[q], k_hi - 8), hq = c / hd;
        pp[q] = a.attn_part + ((long)min(pr[q], rb - 1) * nh + hq) * ns_all * rec + 2 + (c - hq * hd);
      }
      float2 v[AB][AS][4];
      auto load_round = [&](int s0) {
#pragma unroll
        for (int q = 0; q < AB; ++q)
#pragma unroll
          for (int sp = 0; sp < AS; ++sp)
#pragma unroll
            for (int t = 0; t < 4; ++t)
              v[q][sp][t] = *reinterpret_cast<const float2*>(pp[q] + (long)min(s0 + sp, ns_all - 1) * rec + 2 * t);
      };
      load_round(0);
      // (the first round is consumed here, ahead of the barrier below: left to itself the
      // compiler requests it after the barrier, one round trip later)
#pragma unroll
      for (int q = 0; q < AB; ++q)
#pragma unroll
        for (int sp = 0; sp < AS; ++sp)
#pragma unroll
          for (int t = 0; t < 4; ++t) asm volatile("" ::"v"(v[q][sp][t].x), "v"(v[q][sp][t].y));
      // weights of item t into LDS (rows past the bound and heads past the range get 0)
      if (tid < ROWS * kSkAttnHeads) {
        const bool t_ok = t_r < rb && h0 + t_hh < nh && (h0 + t_hh) * hd < k_hi;
        const int ns = min(ns_all, t_pos / a.attn_split_len + 1);
        float M = -INFINITY;
#pragma unroll
        for (int sp = 0; sp < kAttnMergeMaxSplit; ++sp) M = sp < ns ? fmaxf(M, ml[sp].x) : M;
        float f[kAttnMergeMaxSplit], L = 0.f;
#pragma unroll
        for (int sp = 0; sp < kAttnMergeMaxSplit; ++sp) {
          f[sp] = (sp < ns && ml[sp].x > -INFINITY) ? __expf(ml[sp].x - M) : 0.f;
          L = f[sp] > 0.f ? L + ml[sp].y * f[sp] : L;
        }
#pragma unroll
        for (int sp = 0; sp < kAttnMergeMaxSplit; ++sp)
          s_af[(t_r * kSkAttnHeads + t_hh) * kAttnMergeMaxSplit + sp] = (t_ok && L > 0.f) ? f[sp] / L : 0.f;
      }
      __syncthreads();
      float y[AB][8];
#pragma unroll
      for (int q = 0; q < AB; ++q)
#pragma unroll
        for (int t = 0; t < 8; ++t) y[q][t] = 0.f;
      for (int s0 = 0; s0 < ns_all; s0 += AS) {
        if (s0 > 0) load_round(s0);
#pragma unroll
        for (int q = 0; q < AB; ++q) {
          const int c = min(k0 + pc[q], k_hi - 8), hq = c / hd;
          const float* fw = s_af + (min(pr[q], ROWS - 1) * kSkAttnHeads + (hq - h0)) * kAttnMergeMaxSplit;
#pragma unroll
          for (int sp = 0; sp < AS; ++sp) {
            const float w = s0 + sp < ns_all ? fw[min(s0 + sp, kAttnMergeMaxSplit - 1)] : 0.f;
            const bool in = w != 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              y[q][2 * t] = in ? y[q][2 * t] + w * v[q][sp][t].x : y[q][2 * t];
              y[q][2 * t + 1] = in ? y[q][2 * t + 1] + w * v[q][sp][t].y : y[q][2 * t + 1];
            }
          }
        }
      }
#pragma unroll
      for (int q = 0; q < AB; ++q) {
        if (pr[q] < R && k0 + pc[q] < k_hi) {
          uint4 h, l;
          split_bf16x2(y[q][0], y[q][1], h.x, l.x);
          split_bf16x2(y[q][2], y[q][3], h.y, l.y);
          split_bf16x2(y[q][4], y[q][5], h.z, l.z);
          split_bf16x2(y[q][6], y[q][7], h.w, l.w);
          *reinterpret_cast<uint4*>(xh + pr[q] * PITCH + pc[q]) = h;
          *reinterpret_cast<uint4*>(xl + pr[q] * PITCH + pc[q]) = l;
        }
      }
    } else {
#pragma unroll 1
    for (int b0 = 0; b0 < nitems; b0 += BATCH * kSkThreads) {
      uint4 hv[BATCH], lv[BATCH];
#pragma unroll
      for (int q = 0; q < BATCH; ++q) {
        const int i = b0 + tid + q * kSkThreads;
        const int r = i / span8, col = (i - r * span8) * 8;
        const int c = k0 + col;
        uint4 h = make_uint4(0u, 0u, 0u, 0u), l = h;
        if (i < nitems && c < k_hi) {
          if constexpr (SRC == SK_TAPS) {
            h = *reinterpret_cast<const uint4*>(reinterpret_cast<const bf16_t*>(a.taps) +
                                                (long)a.tap_row[r] * a.ldt + c);
          } else if constexpr (SRC == SK_SWIGLU) {
            // SwiGLU of the gate/up products: their K-split partials added in split order.
            // The loads of kSwRound splits are requested at once, from clamped addresses
            // (a round's loads past the last split re-read it and add zero), so that none
            // waits on a condition: one round trip for the usual 4 splits.
            const float* pr = a.part_in + (long)r * a.ld_in + c;
            float g[8], u[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) { g[e] = 0.f; u[e] = 0.f; }
            auto sw_round = [&](int k0) {
              float4 gv[kSwRound][2], uv[kSwRound][2];
#pragma unroll
              for (int q = 0; q < kSwRound; ++q) {
                const float* pk = pr + (long)min(k0 + q, a.ks_in - 1) * a.part_in_split;
                gv[q][0] = *reinterpret_cast<const float4*>(pk);
                gv[q][1] = *reinterpret_cast<const float4*>(pk + 4);
                uv[q][0] = *reinterpret_cast<const float4*>(pk + a.Kd);
                uv[q][1] = *reinterpret_cast<const float4*>(pk + a.Kd + 4);
              }
#pragma unroll
              for (int q = 0; q < kSwRound; ++q) {
                const bool in = k0 + q < a.ks_in;
                const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
                const float4 g0 = in ? gv[q][0] : z, g1 = in ? gv[q][1] : z;
                const float4 u0 = in ? uv[q][0] : z, u1 = in ? uv[q][1] : z;
                g[0] += g0.x; g[1] += g0.y; g[2] += g0.z; g[3] += g0.w;
                g[4] += g1.x; g[5] += g1.y; g[6] += g1.z; g[7] += g1.w;
                u[0] += u0.x; u[1] += u0.y; u[2] += u0.z; u[3] += u0.w;
                u[4] += u1.x; u[5] += u1.y; u[6] += u1.z; u[7] += u1.w;
              }
            };
            __builtin_assume(a.ks_in >= 1);   // (the gate/up product wrote at least one split)
            sw_round(0);
            for (int k0 = kSwRound; k0 < a.ks_in; k0 += kSwRound) sw_round(k0);
            float y[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) y[e] = g[e] / (1.0f + __expf(-g[e])) * u[e];
            split_bf16x2(y[0], y[1], h.x, l.x);
            split_bf16x2(y[2], y[3], h.y, l.y);
            split_bf16x2(y[4], y[5], h.z, l.z);
            split_bf16x2(y[6], y[7], h.w, l.w);
          } else if (c < a.seg) {
            const long o = (long)r * a.ld_xs + c;
            h = *reinterpret_cast<const uint4*>(a.xs_hi + o);
            l = *reinterpret_cast<const uint4*>(a.xs_lo + o);
          } else {
            const long o = (long)(a.gather ? a.gather[r] : r) * a.ld_xa + (c - a.seg);
            h = *reinterpret_cast<const uint4*>(a.xa_hi + o);
            l = *reinterpret_cast<const uint4*>(a.xa_lo + o);
          }
        }
        hv[q] = h;
        lv[q] = l;
      }
#pragma unroll
      for (int q = 0; q < BATCH; ++q) {
        const int i = b0 + tid + q * kSkThreads;
        const int r = i / span8, col = (i - r * span8) * 8;
        if (i < nitems) {
          *reinterpret_cast<uint4*>(xh + r * PITCH + col) = hv[q];
          if constexpr (!EXACT) *reinterpret_cast<uint4*>(xl + r * PITCH + col) = lv[q];
        }
      }
    }
    }
    __syncthreads();
    }

    // ---- stream this wavefront's units: tile j = u / NCH, columns (u % NCH) * 256 ----
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      // (a unit that is not real still requests the one kSkDepth - 1 places ahead, which
      // may be)
      if (real(k0, u + kSkDepth - 1)) load(ring[(u + kSkDepth - 1) % kSkDepth], k0, u + kSkDepth - 1);
      if (real(k0, u)) {
        // keep each unit's work in place: hoisting later units' LDS reads or loads
        // above this point only raises register pressure
        __builtin_amdgcn_sched_barrier(0);
        const uint4* w = ring[u % kSkDepth];
        const int j = u / NCH;                        // (projections: one tile, j = 0)
        const int kl = (u % NCH) * kSkUnit + 8 * grp;   // column within the phase
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const sk_bf16x8 bw = *reinterpret_cast<const sk_bf16x8*>(&w[ks]);
          // all A fragments of this K step are requested before the first product, so
          // one LDS latency covers the step's 2 MT products instead of one each
          sk_bf16x8 ah[MT], al[MT];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            // (the single normalised row: every lane reads row 0 at its column in the
            // whole row; the outputs of rows 1..15 are dropped)
            const int off = SRC == SK_NORM ? k0 + kl + 32 * ks : (mt * 16 + wrow) * PITCH + kl + 32 * ks;
            ah[mt] = *reinterpret_cast<const sk_bf16x8*>(xh + off);
            if constexpr (!EXACT) al[mt] = *reinterpret_cast<const sk_bf16x8*>(xl + off);
          }
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[mt], bw, acc[j][mt], 0, 0, 0);
            if constexpr (!EXACT) acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[mt], bw, acc[j][mt], 0, 0, 0);
          }
          // keep that order: the scheduler, near the register limit, would otherwise
          // put a wait on each read right before its product
          __builtin_amdgcn_sched_group_barrier(0x100, EXACT ? MT : 2 * MT, 0);   // LDS reads
          __builtin_amdgcn_sched_group_barrier(0x008, EXACT ? MT : 2 * MT, 0);   // MFMAs
        }
      }
    }
    if (ph + 1 < nphase) prefetch_phase(k0 + KC);
  }
  if (ntiles == 0) return;

  // ---- epilogue: lane holds outputs of rows 16 mt + 4 grp + e, columns tile + wrow ------
  if constexpr (EPI == SK_PART) {
    float* pb = a.split_buf + (long)blockIdx.y * a.max_rows * NR;
#pragma unroll
    for (int j = 0; j < TMAX; ++j) {
      if (j < ntiles) {
        const int n = (t0 + j) * 16 + wrow;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int m = mt * 16 + 4 * grp + e;
            if (m < R && n < NR) pb[(long)m * NR + n] = acc[j][mt][e];
          }
      }
    }
    return;
  } else {
    // softmax record of every row over this wavefront's 16 T columns.  Lane (wrow, grp)
    // holds V = 4 MT rows (k = 4 mt + e) of its column in every tile.  The 16 lanes of
    // a row group are reduced by halving exchanges: at each step a lane keeps half of
    // its rows and merges the partner's copies of them, so V rows cost about V
    // shuffles instead of 4 V.
    constexpr int V = 4 * MT;
    constexpr int NH = V == 16 ? 4 : (V == 8 ? 3 : 2);    // halving steps (then plain)
    // masked logits (written here, after the stream: stores issued between the ring's
    // loads would lengthen every wait on them).  Conditions that hold for the whole
    // wavefront (every row of the pass present, a tile inside the vocabulary) are taken
    // once per tile, and per-element ones are selects: tested per element, the compiler
    // gave every store and update a branch of its own (about 500 at 64 rows).
    const bool all_rows = R == ROWS;
#pragma unroll
    for (int j = 0; j < TMAX; ++j) {
      if (j < ntiles) {
        const int n = (t0 + j) * 16 + wrow;
        const bool keep = n < a.N && dmap[j] >= 0;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[j][mt][e] = keep ? acc[j][mt][e] : -INFINITY;
        float* yc = a.y + (long)(4 * grp) * a.ld_logits + n;
        // (64-row passes write 39 MB of logits per launch, read back only at a few
        // entries: non-temporal stores keep them out of the last-level cache)
        if (all_rows && (t0 + j + 1) * 16 <= a.N) {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float* dst = yc + (long)(mt * 16 + e) * a.ld_logits;
              if constexpr (MT == 4) __builtin_nontemporal_store(acc[j][mt][e], dst);
              else *dst = acc[j][mt][e];
            }
        } else {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float* dst = yc + (long)(mt * 16 + e) * a.ld_logits;
              if (mt * 16 + 4 * grp + e < R && n < a.N) {
                if constexpr (MT == 4) __builtin_nontemporal_store(acc[j][mt][e], dst);
                else *dst = acc[j][mt][e];
              }
            }
        }
      }
    }
    float rv[V];
    int ri[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
      rv[k] = -INFINITY;
      ri[k] = 0x7fffffff;
#pragma unroll
      for (int j = 0; j < TMAX; ++j) {
        const float v = acc[j][k / 4][k % 4];
        const bool up = j < ntiles && v > rv[k];
        rv[k] = up ? v : rv[k];
        ri[k] = up ? (t0 + j) * 16 + wrow : ri[k];
      }
    }
    // (1) max and lowest argmax
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int mask = 8 >> st;
      if (st < NH) {
        const int half = V >> (st + 1);
        const bool up = (lane & mask) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
          const float mv = up ? rv[i + half] : rv[i], ov = up ? rv[i] : rv[i + half];
          const int mi = up ? ri[i + half] : ri[i], oi = up ? ri[i] : ri[i + half];
          const float pv = xor_lane_c(ov, mask);
          const int pi = xor_lane_ci(oi, mask);
          const bool take = pv > mv || (pv == mv && pi < mi);
          rv[i] = take ? pv : mv;
          ri[i] = take ? pi : mi;
        }
      } else {
        const float pv = xor_lane_c(rv[0], mask);
        const int pi = xor_lane_ci(ri[0], mask);
        if (pv > rv[0] || (pv == rv[0] && pi < ri[0])) { rv[0] = pv; ri[0] = pi; }
      }
    }
    // lane p of the group now holds row k(p) = its top NH bits, read as a number
    auto row_of_lane = [&](int p) {
      int k = 0;
#pragma unroll
      for (int st = 0; st < NH; ++st) k |= ((p >> (3 - st)) & 1) << (NH - 1 - st);
      return k;
    };
    auto lane_of_row = [&](int k) {
      int p = 0;
#pragma unroll
      for (int st = 0; st < NH; ++st) p |= ((k >> (NH - 1 - st)) & 1) << (3 - st);
      return p;
    };
    // (2) every lane fetches the maxima of its V rows and sums its own columns
    float sv[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const float Mk = row_lane_c(rv[0], lane_of_row(k));
      const int m = (k / 4) * 16 + 4 * grp + (k % 4);
      const float Tk = m < R ? tk[k] : 0.f;
      // (masked entries add exp(-inf) = 0; a row with no sum -- T = 0, or every entry
      // masked, where the terms are NaN -- is selected to 0 after the loop)
      const bool live = Tk > 0.f && Mk > -INFINITY;
      const float iT = 1.0f / (live ? Tk : 1.0f);
      float sum = 0.f;
#pragma unroll
      for (int j = 0; j < TMAX; ++j) {
        const float t = __expf((acc[j][k / 4][k % 4] - Mk) * iT);
        sum += j < ntiles ? t : 0.f;
      }
      sv[k] = live ? sum : 0.f;
    }
    // (3) sums, reduced like the maxima
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int mask = 8 >> st;
      if (st < NH) {
        const int half = V >> (st + 1);
        const bool up = (lane & mask) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
          const float mv = up ? sv[i + half] : sv[i], ov = up ? sv[i] : sv[i + half];
          sv[i] = mv + xor_lane_c(ov, mask);
        }
      } else {
        sv[0] += xor_lane_c(sv[0], mask);
      }
    }
    if ((lane & ((16 >> NH) - 1)) == 0) {
      const int k = row_of_lane(lane & 15);
      const int m = (k / 4) * 16 + 4 * grp + (k % 4);
      if (m < R) {
        float* p = a.part + ((long)m * a.nblk + wg) * 4;
        p[0] = rv[0];
        p[1] = sv[0];
        p[2] = __int_as_float(rv[0] > -INFINITY ? ri[0] : -1);
        p[3] = 0.f;
      }
    }
  }
}

static int sk_mt(int rows) { return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4); }

// ---- LM head ----------------------------------------------------------------------------
LmPlan lm_head_plan(int rows, int N, int n_cu) {
  LmPlan p;
  p.mt = sk_mt(rows);
  const int nt16 = (N + 15) / 16;
  // one block per CU (the register budget allows 2 wavefronts per SIMD)
  p.grid = std::min(n_cu, kGemvMaxWaves / kSkWaves);
  p.T = (nt16 + p.grid * kSkWaves - 1) / (p.grid * kSkWaves);
  if (p.T > kSkTmaxHead) {
    p.T = kSkTmaxHead;
    p.grid = (nt16 + kSkTmaxHead * kSkWaves - 1) / (kSkTmaxHead * kSkWaves);
  }
  p.nblk = (nt16 + p.T - 1) / p.T;
  p.blk_rows = 16 * p.T;
  return p;
}

template <int SRC, int EPI>
static void sk_launch(int mt, dim3 grid, const GemvArgs& a, int T, int kc, hipStream_t st) {
  if (mt == 1) hipLaunchKernelGGL((k_skinny<1, SRC, EPI>), grid, dim3(kSkThreads), 0, st, a, T, kc);
  else if (mt == 2) hipLaunchKernelGGL((k_skinny<2, SRC, EPI>), grid, dim3(kSkThreads), 0, st, a, T, kc);
  else hipLaunchKernelGGL((k_skinny<4, SRC, EPI>), grid, dim3(kSkThreads), 0, st, a, T, kc);
}

bool lm_head_norm_in_supported(int rows, int Kd) { return rows == 1 && Kd <= 8 * kSkThreads; }

bool launch_lm_head(const GemvArgs& a, const LmPlan& p, bool norm_in, hipStream_t st) {
  // the fp32 input is normalised in the head for one row only (batch 1), of at most
  // 8 x kSkThreads columns; anything else is refused (nothing launched)
  if (norm_in && !lm_head_norm_in_supported(a.max_rows, a.Kd)) return false;
  if (norm_in) sk_launch<SK_NORM, SK_LOGITS>(1, dim3(p.grid), a, p.T, 0, st);
  else sk_launch<SK_PREP, SK_LOGITS>(p.mt, dim3(p.grid), a, p.T, 0, st);
  return true;
}

// ---- projections --------------------------------------------------------------------------
// One 16-row tile per wavefront; the K columns per block shrink (down to one 256-column
// unit) until the grid holds about 256 blocks: each wavefront then waits on few loads,
// and the launch costs about one load round trip instead of a per-wavefront stream.
static int skinny_kc(int rows, int N2, int Kd) {
  const int KC = rows > 32 ? SkCfg<4>::KC : SkCfg<1>::KC;
  const int nb = (((N2 + 15) / 16) + kSkWaves - 1) / kSkWaves;   // blocks per K range
  int kc = KC;
  // (the expanded QKV's partials are summed on load by the attention row kernel, which
  // takes at most kMaxKSplit of them)
  while (kc > kSkUnit && (long)nb * ((Kd + kc - 1) / kc) < 256 && (Kd + kc / 2 - 1) / (kc / 2) <= kMaxKSplit)
    kc /= 2;
  return kc;
}

long packed_head_bytes(int N, int Kd) {
  return 2L * ((N + 15) / 16) * 16 * ((Kd + kSkUnit - 1) / kSkUnit) * kSkUnit;
}

// One thread per 16-byte piece of the packed copy.
__global__ void k_pack_head(const bf16_t* __restrict__ w, int N, int Kd, long pieces, uint4* __restrict__ out) {
  const long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= pieces) return;
  const int nu_row = (Kd + kSkUnit - 1) / kSkUnit;
  const int lane = (int)(i & 63), s = (int)((i >> 6) & 7);
  const long tu = i >> 9;                       // tile * nu_row + unit
  const int u = (int)(tu % nu_row), t = (int)(tu / nu_row);
  const int row = 16 * t + (lane & 15);
  const int col = kSkUnit * u + 8 * (lane >> 4) + 32 * s;
  out[i] = (row < N && col < Kd) ? *reinterpret_cast<const uint4*>(w + (long)row * Kd + col)
                                 : make_uint4(0u, 0u, 0u, 0u);
}

void launch_pack_head(const void* w, int N, int Kd, void* packed, hipStream_t st) {
  const long pieces = packed_head_bytes(N, Kd) / 16;
  hipLaunchKernelGGL(k_pack_head, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, st,
                     reinterpret_cast<const bf16_t*>(w), N, Kd, pieces, reinterpret_cast<uint4*>(packed));
}

int skinny_splits(int rows, int Kd) {
  // upper bound over the products of a layer (workspace sizing): the smallest K range
  return (Kd + kSkUnit - 1) / kSkUnit;
}

int launch_skinny(SrcKind src, const GemvArgs& a, hipStream_t st) {
  const int mt = sk_mt(a.max_rows);
  const int NR = a.w1 ? 2 * a.N : a.N;
  // (attention outputs: K ranges of one unit, so that a block's range holds at most 4
  // heads)
  const int kc = src == SRC_ATTN ? kSkUnit : skinny_kc(a.max_rows, NR, a.Kd);
  const int ks = (a.Kd + kc - 1) / kc;
  const dim3 grid((((NR + 15) / 16) + kSkWaves - 1) / kSkWaves, ks);
  if (src == SRC_TAPS) sk_launch<SK_TAPS, SK_PART>(mt, grid, a, 1, kc, st);
  else if (src == SRC_SWIGLU) sk_launch<SK_SWIGLU, SK_PART>(mt, grid, a, 1, kc, st);
  else if (src == SRC_ATTN) sk_launch<SK_ATTN, SK_PART>(mt, grid, a, 1, kc, st);
  else sk_launch<SK_PREP, SK_PART>(mt, grid, a, 1, kc, st);
  return ks;
}

}  // namespace osp

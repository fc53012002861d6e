// Row kernels of the matrix-core path (passes of several rows): they close one
// product and prepare the next one's input.  One block per row (SwiGLU, which is
// elementwise: a row's columns spread over several blocks):
//   * add the K-split partial sums of the product in split order (fixed order,
//     so results do not depend on scheduling),
//   * apply the residual, RMSNorm with gain, or SwiGLU in fp32,
//   * write the next product's input once as a bf16 pair hi = bf16(v),
//     lo = bf16(v - hi), so that every GEMM block only copies its input chunk.
// Widths are multiples of 64 (checked at init); each thread handles 4
// consecutive columns per step.
#include "common.h"
#include "internal.h"
#include "pick.h"

namespace osp {

constexpr int kRowThreads = 256;

OSP_DEV void store_pair4(uint16_t* hi, uint16_t* lo, long o, float4 v) {
  uint32_t h[2], l[2];
  split_bf16x2(v.x, v.y, h[0], l[0]);
  split_bf16x2(v.z, v.w, h[1], l[1]);
  *reinterpret_cast<uint2*>(hi + o) = make_uint2(h[0], h[1]);
  *reinterpret_cast<uint2*>(lo + o) = make_uint2(l[0], l[1]);
}

// Sum over the K splits of columns [col, col + 4) of row r, in split order.  The loads
// of a round of kMaxKSplit splits are requested at once, from clamped addresses: a
// round's loads past the last split read that split again (a cache hit) and add zero,
// so no load waits on a condition.  One round covers the projections (at most
// kMaxKSplit splits); the tap projection over n_taps x target_hidden columns can take
// more (24 at 3 x 8192), hence the further rounds.
template <int N>
OSP_DEV void add_round4(const float* const (&p)[N], long stride, int k0, int ks, float4 (&s)[N]) {
  float4 v[N][kMaxKSplit];
#pragma unroll
  for (int q = 0; q < kMaxKSplit; ++q)
#pragma unroll
    for (int j = 0; j < N; ++j) v[j][q] = *reinterpret_cast<const float4*>(p[j] + min(k0 + q, ks - 1) * stride);
#pragma unroll
  for (int j = 0; j < N; ++j)
#pragma unroll
    for (int q = 0; q < kMaxKSplit; ++q) {
      const bool in = k0 + q < ks;
      s[j].x += in ? v[j][q].x : 0.f; s[j].y += in ? v[j][q].y : 0.f;
      s[j].z += in ? v[j][q].z : 0.f; s[j].w += in ? v[j][q].w : 0.f;
    }
}

// Columns [col[j], col[j] + 4) of row r for each j < N (all requested together).
template <int N>
OSP_DEV void sum_parts(const RowArgs& a, int r, const int (&col)[N], float4 (&s)[N]) {
  const float* p[N];
#pragma unroll
  for (int j = 0; j < N; ++j) {
    p[j] = a.part + (long)r * a.ldp + col[j];
    s[j] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const long stride = (long)a.max_rows * a.ldp;
  __builtin_assume(a.ks >= 1);   // (every producer writes at least one split)
  add_round4<N>(p, stride, 0, a.ks, s);
  for (int k0 = kMaxKSplit; k0 < a.ks; k0 += kMaxKSplit) add_round4<N>(p, stride, k0, a.ks, s);
}

OSP_DEV float4 sum_parts4(const RowArgs& a, int r, int col) {
  float4 s[1];
  sum_parts<1>(a, r, {col}, s);
  return s[0];
}

OSP_DEV float block_sum(float v, float* sm) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) sm[wave] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kRowThreads / 64; ++w) t += sm[w];
  return t;
}

// Column groups of a row per thread: W <= 4 kRowThreads kRowGroups (= 4096, the largest
// d_model the library accepts).
constexpr int kRowGroups = 4;

// Row r's final values are v (column group i at (threadIdx.x + i kRowThreads) 4) and its
// gain gr: out = rmsnorm(x[r]) * gamma as hi / lo, from registers.
OSP_DEV void norm_out(const RowArgs& a, int r, const float4 (&v)[kRowGroups], const uint2 (&gr)[kRowGroups],
                      float ss, float* sm) {
  const float inv = 1.0f / sqrtf(block_sum(ss, sm) / (float)a.W + a.eps);
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    if (c < a.W) {
      const float4 y = make_float4(v[i].x * inv * bf16_lo(gr[i].x), v[i].y * inv * bf16_hi(gr[i].x),
                                   v[i].z * inv * bf16_lo(gr[i].y), v[i].w * inv * bf16_hi(gr[i].y));
      store_pair4(a.out_hi, a.out_lo, (long)r * a.W + c, y);
    }
  }
}

// The gain of this thread's column groups (requested early, used by norm_out).
OSP_DEV void load_gain(const RowArgs& a, uint2 (&gr)[kRowGroups]) {
  const bf16_t* g = reinterpret_cast<const bf16_t*>(a.gamma);
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    gr[i] = *reinterpret_cast<const uint2*>(g + min(c, a.W - 4));
  }
}

// DRAW: row r's token is drawn here from the LM head's records and logits (a.pick), and
// the conditioning rows s_src may be the rows x that this block overwrites (each thread
// reads its columns of row r before it writes them).
template <bool DRAW>
__global__ void __launch_bounds__(kRowThreads) k_rows_prep(RowArgs a) {
  __shared__ float sm[kRowThreads / 64];
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  uint2 gr[kRowGroups], er[kRowGroups];
  int t;
  float4 sv[DRAW ? kRowGroups : 1];
  Pick pk_res{};
  int pk_pos = 0;
  if constexpr (DRAW) {
    // the records first (the memory counter is in order: whatever is requested after
    // them arrives no earlier), then the conditioning row and the gain, whose loads do
    // not depend on the token
    constexpr int PER = kPickMaxRecords / kRowThreads;
    const PickArgs& pk = a.pick;
    const float* part = pk.part + r * pk.ld_part;
    PickRecs<PER> rec;
    pick_request<kRowThreads, PER>(rec, part, pk.nblk);
#pragma unroll
    for (int i = 0; i < kRowGroups; ++i)
      sv[i] = *reinterpret_cast<const float4*>(a.s_src + (long)r * a.W +
                                               min(((int)threadIdx.x + i * kRowThreads) * 4, a.W - 4));
    load_gain(a, gr);
    pk_pos = pk.committed[r] + pk.k;
    // (nothing that reads the records may be scheduled above this point)
    __builtin_amdgcn_sched_barrier(0);
    pk_res = pick_draft<kRowThreads, PER>(rec, pk.nblk, pk.blk_rows, pk.logits + r * pk.ld_logits, pk.V,
                                          pk.d2t, pk.temp[r], pk.u[(long)r * pk.ld_u]);
    t = pk_res.tok;
  } else {
    // the token row and the gain are requested first, ahead of the conditioning segment
    t = a.tok[r];
  }
  t = min(max(t, 0), a.vocab_embed - 1);
  const bf16_t* e = reinterpret_cast<const bf16_t*>(a.embed) + (long)t * a.W;
  if constexpr (!DRAW) load_gain(a, gr);
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i)
    er[i] = *reinterpret_cast<const uint2*>(e + min(((int)threadIdx.x + i * kRowThreads) * 4, a.W - 4));
  // conditioning segment: tap projection (sum of its splits) or the fed-back state
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    if (c < a.W) {
      float4 v;
      if constexpr (DRAW) v = sv[i];
      else v = a.s_src ? *reinterpret_cast<const float4*>(a.s_src + (long)r * a.W + c) : sum_parts4(a, r, c);
      store_pair4(a.s_hi, a.s_lo, (long)r * a.W + c, v);
    }
  }
  // token segment: x = embed[tok], then its normalised copy
  float4 v[kRowGroups];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    v[i] = make_float4(bf16_lo(er[i].x), bf16_hi(er[i].x), bf16_lo(er[i].y), bf16_hi(er[i].y));
    if (c < a.W) {
      *reinterpret_cast<float4*>(a.x + (long)r * a.W + c) = v[i];
      ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
  }
  norm_out(a, r, v, gr, ss, sm);
  // the draft, its position and the row statistics, written once the row is done
  if constexpr (DRAW) {
    if (threadIdx.x == 0) {
      const PickArgs& pk = a.pick;
      pk.draft[(long)r * pk.ld_draft] = pk_res.tok;
      if (pk.draft_out) pk.draft_out[(long)r * pk.ld_draft_out] = pk_res.tok;
      pk.ar_tok[r] = pk_res.tok;
      pk.ar_pos[r] = pk_pos;
      if (pk.qstat) pk.qstat[(long)r * pk.ld_qstat] = QStat{pk_res.S, pk_res.M, pk_res.am};
    }
  }
}

__global__ void __launch_bounds__(kRowThreads) k_rows_resid_norm(RowArgs a) {
  __shared__ float sm[kRowThreads / 64];
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  // the residual and the gain are requested before the partials, in the same round trip
  uint2 gr[kRowGroups];
  load_gain(a, gr);
  float4 v[kRowGroups];
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    v[i] = *reinterpret_cast<const float4*>(a.x + (long)r * a.W + min(c, a.W - 4));
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kRowGroups; ++i) {
    const int c = (threadIdx.x + i * kRowThreads) * 4;
    if (c < a.W) {
      const float4 p = sum_parts4(a, r, c);
      v[i].x += p.x; v[i].y += p.y; v[i].z += p.z; v[i].w += p.w;
      *reinterpret_cast<float4*>(a.x + (long)r * a.W + c) = v[i];
      ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
  }
  norm_out(a, r, v, gr, ss, sm);
}

// Elementwise: the columns of a row are spread over gridDim.y blocks.
__global__ void __launch_bounds__(kRowThreads) k_rows_swiglu(RowArgs a) {
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  for (int c = (blockIdx.y * kRowThreads + threadIdx.x) * 4; c < a.W; c += gridDim.y * kRowThreads * 4) {
    float4 gu[2];
    sum_parts<2>(a, r, {c, a.W + c}, gu);
    const float4 g = gu[0], u = gu[1];
    const float4 h = make_float4(g.x / (1.0f + __expf(-g.x)) * u.x, g.y / (1.0f + __expf(-g.y)) * u.y,
                                 g.z / (1.0f + __expf(-g.z)) * u.z, g.w / (1.0f + __expf(-g.w)) * u.w);
    store_pair4(a.out_hi, a.out_lo, (long)r * a.W + c, h);
  }
}

void launch_rows_prep(const RowArgs& a, hipStream_t st) {
  if (a.pick.part) hipLaunchKernelGGL(k_rows_prep<true>, dim3(a.max_rows), dim3(kRowThreads), 0, st, a);
  else hipLaunchKernelGGL(k_rows_prep<false>, dim3(a.max_rows), dim3(kRowThreads), 0, st, a);
}
void launch_rows_resid_norm(const RowArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_rows_resid_norm, dim3(a.max_rows), dim3(kRowThreads), 0, st, a);
}
void launch_rows_swiglu(const RowArgs& a, hipStream_t st) {
  const int per_row = (a.W + kRowThreads * 4 - 1) / (kRowThreads * 4);   // one column group per block
  hipLaunchKernelGGL(k_rows_swiglu, dim3(a.max_rows, per_row), dim3(kRowThreads), 0, st, a);
}

}  // namespace osp

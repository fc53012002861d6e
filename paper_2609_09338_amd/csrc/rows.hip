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

namespace osp {

constexpr int kRowThreads = 256;

OSP_DEV void store_pair4(uint16_t* hi, uint16_t* lo, long o, float4 v) {
  uint32_t h[2], l[2];
  split_bf16x2(v.x, v.y, h[0], l[0]);
  split_bf16x2(v.z, v.w, h[1], l[1]);
  *reinterpret_cast<uint2*>(hi + o) = make_uint2(h[0], h[1]);
  *reinterpret_cast<uint2*>(lo + o) = make_uint2(l[0], l[1]);
}

// Sum over the K splits of columns [col, col + 4) of row r, in split order; the loads
// of four splits are requested together.
OSP_DEV float4 sum_parts4(const RowArgs& a, int r, int col) {
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  const float* p = a.part + (long)r * a.ldp + col;
  const long stride = (long)a.max_rows * a.ldp;
  for (int k0 = 0; k0 < a.ks; k0 += 4) {
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = k0 + q < a.ks ? *reinterpret_cast<const float4*>(p + (k0 + q) * stride) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q) { s.x += v[q].x; s.y += v[q].y; s.z += v[q].z; s.w += v[q].w; }
  }
  return s;
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

// x[r] is final: out = rmsnorm(x[r]) * gamma as hi / lo.
OSP_DEV void norm_out(const RowArgs& a, int r, float ss, float* sm) {
  const float inv = 1.0f / sqrtf(block_sum(ss, sm) / (float)a.W + a.eps);
  const bf16_t* g = reinterpret_cast<const bf16_t*>(a.gamma);
  for (int c = threadIdx.x * 4; c < a.W; c += kRowThreads * 4) {
    const float4 v = *reinterpret_cast<const float4*>(a.x + (long)r * a.W + c);
    const uint2 gr = *reinterpret_cast<const uint2*>(g + c);
    const float4 y = make_float4(v.x * inv * bf16_lo(gr.x), v.y * inv * bf16_hi(gr.x),
                                 v.z * inv * bf16_lo(gr.y), v.w * inv * bf16_hi(gr.y));
    store_pair4(a.out_hi, a.out_lo, (long)r * a.W + c, y);
  }
}

__global__ void __launch_bounds__(kRowThreads) k_rows_prep(RowArgs a) {
  __shared__ float sm[kRowThreads / 64];
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  // conditioning segment: tap projection (sum of its splits) or the fed-back state
  for (int c = threadIdx.x * 4; c < a.W; c += kRowThreads * 4) {
    const float4 v = a.s_src ? *reinterpret_cast<const float4*>(a.s_src + (long)r * a.W + c)
                             : sum_parts4(a, r, c);
    store_pair4(a.s_hi, a.s_lo, (long)r * a.W + c, v);
  }
  // token segment: x = embed[tok], then its normalised copy
  int t = a.tok[r];
  t = min(max(t, 0), a.vocab_embed - 1);
  const bf16_t* e = reinterpret_cast<const bf16_t*>(a.embed) + (long)t * a.W;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < a.W; c += kRowThreads * 4) {
    const uint2 er = *reinterpret_cast<const uint2*>(e + c);
    const float4 v = make_float4(bf16_lo(er.x), bf16_hi(er.x), bf16_lo(er.y), bf16_hi(er.y));
    *reinterpret_cast<float4*>(a.x + (long)r * a.W + c) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  norm_out(a, r, ss, sm);
}

__global__ void __launch_bounds__(kRowThreads) k_rows_resid_norm(RowArgs a) {
  __shared__ float sm[kRowThreads / 64];
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < a.W; c += kRowThreads * 4) {
    float4* xp = reinterpret_cast<float4*>(a.x + (long)r * a.W + c);
    const float4 p = sum_parts4(a, r, c);
    float4 v = *xp;
    v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    *xp = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  norm_out(a, r, ss, sm);
}

// Elementwise: the columns of a row are spread over gridDim.y blocks.
__global__ void __launch_bounds__(kRowThreads) k_rows_swiglu(RowArgs a) {
  const int r = blockIdx.x;
  const int rows = a.count ? min(*a.count, a.max_rows) : a.max_rows;
  if (r >= rows) return;
  for (int c = (blockIdx.y * kRowThreads + threadIdx.x) * 4; c < a.W; c += gridDim.y * kRowThreads * 4) {
    const float4 g = sum_parts4(a, r, c);
    const float4 u = sum_parts4(a, r, a.W + c);
    const float4 h = make_float4(g.x / (1.0f + __expf(-g.x)) * u.x, g.y / (1.0f + __expf(-g.y)) * u.y,
                                 g.z / (1.0f + __expf(-g.z)) * u.z, g.w / (1.0f + __expf(-g.w)) * u.w);
    store_pair4(a.out_hi, a.out_lo, (long)r * a.W + c, h);
  }
}

void launch_rows_prep(const RowArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_rows_prep, dim3(a.max_rows), dim3(kRowThreads), 0, st, a);
}
void launch_rows_resid_norm(const RowArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_rows_resid_norm, dim3(a.max_rows), dim3(kRowThreads), 0, st, a);
}
void launch_rows_swiglu(const RowArgs& a, hipStream_t st) {
  const int per_row = (a.W + kRowThreads * 4 - 1) / (kRowThreads * 4);   // one column group per block
  hipLaunchKernelGGL(k_rows_swiglu, dim3(a.max_rows, per_row), dim3(kRowThreads), 0, st, a);
}

}  // namespace osp

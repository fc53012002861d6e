// Device helpers and launch-argument structs shared by the HIP kernels of the
// draft-and-verify step.  gfx950 (CDNA4) only: 64-lane wavefronts.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define OSP_WAVE 64
#define OSP_DEV __device__ __forceinline__

namespace osp {

typedef uint16_t bf16_t;   // raw bfloat16 storage

OSP_DEV float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
OSP_DEV float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
OSP_DEV float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bfloat16, round to nearest, ties to even (NaN stays NaN): one
// v_cvt_pk_bf16_f32 on gfx950.
OSP_DEV bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Two floats -> packed bfloat16 pair (lo in bits 0..15), one conversion instruction.
OSP_DEV uint32_t f32x2_to_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Split two floats into bf16 pairs hi = bf16(x), lo = bf16(x - hi).
OSP_DEV void split_bf16x2(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = f32x2_to_bf16x2(a, b);
  lo = f32x2_to_bf16x2(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}

template <typename T> OSP_DEV float load_f32(const T* p, long i);
template <> OSP_DEV float load_f32<float>(const float* p, long i) { return p[i]; }
template <> OSP_DEV float load_f32<bf16_t>(const bf16_t* p, long i) { return bf16_to_f32(p[i]); }

template <typename T> OSP_DEV void store_from_f32(T* p, long i, float v);
template <> OSP_DEV void store_from_f32<float>(float* p, long i, float v) { p[i] = v; }
template <> OSP_DEV void store_from_f32<bf16_t>(bf16_t* p, long i, float v) { p[i] = f32_to_bf16(v); }

// Elements per 16-byte vector load.
template <typename T> struct Vec;
template <> struct Vec<float> { static constexpr int N = 4; };
template <> struct Vec<bf16_t> { static constexpr int N = 8; };

// Load one 16-byte vector and widen to floats.
template <typename T> OSP_DEV void load_vec(const T* p, float* out);
template <> OSP_DEV void load_vec<float>(const float* p, float* out) {
  float4 v = *reinterpret_cast<const float4*>(p);
  out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
}
template <> OSP_DEV void load_vec<bf16_t>(const bf16_t* p, float* out) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  out[0] = bf16_lo(v.x); out[1] = bf16_hi(v.x);
  out[2] = bf16_lo(v.y); out[3] = bf16_hi(v.y);
  out[4] = bf16_lo(v.z); out[5] = bf16_hi(v.z);
  out[6] = bf16_lo(v.w); out[7] = bf16_hi(v.w);
}

// Reductions over the 64 lanes of a wavefront (every lane active), every lane receiving
// the result.  Each 16-lane row is combined by DPP moves (partners lane ^ 1 and lane ^ 2
// by quad permutation, then lane ^ 7 and lane ^ 15 by the half-row and row mirrors),
// which are VALU operations, instead of shuffles through the LDS crossbar (one ~100-cycle
// round trip per step); the four row results are then read lane by lane and combined
// in row order.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within each half-row
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within each row
template <int CTRL> OSP_DEV int dpp_i(int v) { return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false); }
template <int CTRL> OSP_DEV float dpp_f(float v) { return __int_as_float(dpp_i<CTRL>(__float_as_int(v))); }
template <int CTRL> OSP_DEV double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = dpp_i<CTRL>((int)(b & 0xffffffffll)), hi = dpp_i<CTRL>((int)(b >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
OSP_DEV float lane_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }
OSP_DEV double lane_d(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffffll), l);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// The value of lane l ^ M, for every lane l (all 64 lanes active), by VALU operations:
// DPP within 16-lane rows (quad permutations for 1 and 2; the half-row mirror, lane ^ 7,
// then the quad reversal, lane ^ 3, for 4; the row rotation by 8 for 8) and the gfx950
// swaps across rows (v_permlane16_swap / v_permlane32_swap of a register with itself
// yield rows {0, 0, 2, 2} and {1, 1, 3, 3}, or halves {lo, lo} and {hi, hi}; the lane's
// row or half bit picks the partner's).  Same partners as a shuffle by xor, so results
// are the same bit for bit.
template <int M> OSP_DEV int xor_lane_i(int v, int lane) {
  if constexpr (M == 1) return dpp_i<kDppXor1>(v);
  else if constexpr (M == 2) return dpp_i<kDppXor2>(v);
  else if constexpr (M == 4) return dpp_i<0x1B>(dpp_i<kDppHalfMirror>(v));   // quad_perm [3, 2, 1, 0]
  else if constexpr (M == 8) return dpp_i<0x128>(v);                          // row_ror:8
  else if constexpr (M == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    return (int)((lane & 16) ? p[0] : p[1]);
  } else {
    static_assert(M == 32, "xor mask");
    const auto p = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    return (int)((lane & 32) ? p[0] : p[1]);
  }
}
template <int M> OSP_DEV float xor_lane(float v, int lane) { return __int_as_float(xor_lane_i<M>(__float_as_int(v), lane)); }
template <int M> OSP_DEV double xor_lane_d(double v, int lane) {
  const long long b = __double_as_longlong(v);
  const int lo = xor_lane_i<M>((int)(b & 0xffffffffll), lane), hi = xor_lane_i<M>((int)(b >> 32), lane);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// The same for a mask that is a constant once loops are unrolled.
OSP_DEV int xor_lane_ci(int v, int m) {
  const int lane = __lane_id();
  switch (m) {
    case 1: return xor_lane_i<1>(v, lane);
    case 2: return xor_lane_i<2>(v, lane);
    case 4: return xor_lane_i<4>(v, lane);
    case 8: return xor_lane_i<8>(v, lane);
    case 16: return xor_lane_i<16>(v, lane);
    default: return xor_lane_i<32>(v, lane);
  }
}
OSP_DEV float xor_lane_c(float v, int m) { return __int_as_float(xor_lane_ci(__float_as_int(v), m)); }
// The value of lane c of each lane's 16-lane row (DPP row_newbcast), for c a constant
// once loops are unrolled.
template <int C> OSP_DEV int row_lane_i(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x150 + C, 0xF, 0xF, false); }
OSP_DEV float row_lane_c(float v, int c) {
  const int x = __float_as_int(v);
  int r;
  switch (c) {
    case 0: r = row_lane_i<0>(x); break;    case 1: r = row_lane_i<1>(x); break;
    case 2: r = row_lane_i<2>(x); break;    case 3: r = row_lane_i<3>(x); break;
    case 4: r = row_lane_i<4>(x); break;    case 5: r = row_lane_i<5>(x); break;
    case 6: r = row_lane_i<6>(x); break;    case 7: r = row_lane_i<7>(x); break;
    case 8: r = row_lane_i<8>(x); break;    case 9: r = row_lane_i<9>(x); break;
    case 10: r = row_lane_i<10>(x); break;  case 11: r = row_lane_i<11>(x); break;
    case 12: r = row_lane_i<12>(x); break;  case 13: r = row_lane_i<13>(x); break;
    case 14: r = row_lane_i<14>(x); break;  default: r = row_lane_i<15>(x); break;
  }
  return __int_as_float(r);
}
// The value of lane l (the same l on every lane) on every lane.
OSP_DEV int lane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

OSP_DEV float wave_sum(float v) {
  v += dpp_f<kDppXor1>(v);
  v += dpp_f<kDppXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
OSP_DEV double wave_sum_d(double v) {
  v += dpp_d<kDppXor1>(v);
  v += dpp_d<kDppXor2>(v);
  v += dpp_d<kDppHalfMirror>(v);
  v += dpp_d<kDppMirror>(v);
  return (lane_d(v, 0) + lane_d(v, 16)) + (lane_d(v, 32) + lane_d(v, 48));
}
OSP_DEV float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

// Reduce V = 2^LOGV per-lane values over all 64 lanes at once.  On return
// v[0] of lane l holds the full sum of value index (l >> (6 - LOGV)); every
// lane of that group holds the same total.  Costs about V + 6 shuffles
// instead of 6 V.
template <int S, int LOGV>
OSP_DEV void tr_half(float* v, int lane) {
  if constexpr (S < LOGV) {
    constexpr int m = 32 >> S, h = (1 << LOGV) >> (S + 1);
    const bool hi = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < h; ++i) {
      const float mine = hi ? v[i + h] : v[i];
      const float other = hi ? v[i] : v[i + h];
      v[i] = mine + xor_lane<m>(other, lane);
    }
    tr_half<S + 1, LOGV>(v, lane);
  }
}
template <int M>
OSP_DEV void tr_plain(float* v, int lane) {
  if constexpr (M >= 1) {
    v[0] += xor_lane<M>(v[0], lane);
    tr_plain<M / 2>(v, lane);
  }
}
template <int LOGV>
OSP_DEV float transpose_reduce(float* v, int lane) {
  tr_half<0, LOGV>(v, lane);
  tr_plain<(32 >> LOGV)>(v, lane);
  return v[0];
}

// Order-preserving float <-> uint key (for lowest-index argmax merges).
OSP_DEV uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace osp

namespace osp {

// DPP moves that shift data between lanes (lanes with no source read `zero`): within
// each 16-lane row by n, across the whole wavefront by one, and the broadcast of lane 15
// (31) of a row to the next row (rows 2 and 3) -- the row mask leaves the others at 0.
template <int CTRL, int ROWS> OSP_DEV int dpp_shift_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, true);
}
template <int CTRL, int ROWS> OSP_DEV int dpp_shift(int v) { return dpp_shift_i<CTRL, ROWS>(v); }
template <int CTRL, int ROWS> OSP_DEV float dpp_shift(float v) {
  return __int_as_float(dpp_shift_i<CTRL, ROWS>(__float_as_int(v)));
}
template <int CTRL, int ROWS> OSP_DEV double dpp_shift(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = dpp_shift_i<CTRL, ROWS>((int)(b & 0xffffffffll)), hi = dpp_shift_i<CTRL, ROWS>((int)(b >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
constexpr int kDppRowShr = 0x110;   // + n: row_shr:n
constexpr int kDppWaveShr1 = 0x138; // wave_shr:1
constexpr int kDppBcast15 = 0x142;  // row_bcast:15
constexpr int kDppBcast31 = 0x143;  // row_bcast:31

// Inclusive prefix sum across the 64 lanes of a wavefront (fixed order): a Kogge-Stone
// scan within each row by DPP row shifts 1, 2, 4, 8, then each row adds the totals of the
// rows before it (lane 15 broadcast to rows 1 and 3, lane 31 to rows 2 and 3).
template <typename T>
OSP_DEV T wave_incl_scan(T v) {
  v += dpp_shift<kDppRowShr + 1, 0xF>(v);
  v += dpp_shift<kDppRowShr + 2, 0xF>(v);
  v += dpp_shift<kDppRowShr + 4, 0xF>(v);
  v += dpp_shift<kDppRowShr + 8, 0xF>(v);
  v += dpp_shift<kDppBcast15, 0xA>(v);
  v += dpp_shift<kDppBcast31, 0xC>(v);
  return v;
}

// Prefix sums over a block of NT threads (NT/64 wavefronts), in a fixed order.
// Returns the exclusive prefix of this thread; `incl` receives the inclusive
// prefix and `tot` the block total.  The intervals [excl, incl) of consecutive
// threads tile [0, tot) exactly (no rounding gaps).  `sm` needs NT/64 floats.
template <int NT, typename T>
OSP_DEV T block_scan(T v, T* sm, T& incl, T& tot) {
  constexpr int NW = NT / OSP_WAVE;
  const int lane = threadIdx.x & (OSP_WAVE - 1), wave = threadIdx.x >> 6;
  const T inc = wave_incl_scan<T>(v);
  // (the inclusive prefix of lane - 1, moved as data: [excl, incl) of neighbours meet)
  T prev = dpp_shift<kDppWaveShr1, 0xF>(inc);
  if (lane == 0) prev = T(0);
  if (lane == OSP_WAVE - 1) sm[wave] = inc;
  __syncthreads();
  T before = T(0), all = T(0);
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const T t = sm[w];
    if (w < wave) before += t;
    all += t;
  }
  __syncthreads();
  tot = all;
  incl = before + inc;
  return lane == 0 ? before : before + prev;
}

OSP_DEV int wave_max_i(int v) {
  v = max(v, dpp_i<kDppXor1>(v));
  v = max(v, dpp_i<kDppXor2>(v));
  v = max(v, dpp_i<kDppHalfMirror>(v));
  v = max(v, dpp_i<kDppMirror>(v));
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

OSP_DEV int wave_min_i(int v) {
  v = min(v, dpp_i<kDppXor1>(v));
  v = min(v, dpp_i<kDppXor2>(v));
  v = min(v, dpp_i<kDppHalfMirror>(v));
  v = min(v, dpp_i<kDppMirror>(v));
  return min(min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             min(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

}  // namespace osp

// Device-side helpers shared by the decoding kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdec {

constexpr int kWave = 64;

// bfloat16 storage is a raw 16-bit pattern: the upper half of an IEEE float.
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round-to-nearest-even float -> bfloat16 with gfx950's conversion
// instruction (v_cvt_pk_bf16_f32).  It equals the integer rounding
// (u + 0x7fff + ((u >> 16) & 1)) >> 16 on every non-NaN float (all 2^32
// patterns compared on the GPU) and keeps NaNs NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }
// Two values, low half first, in one conversion.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{lo, hi}, bf16x2_t));
}

// Storage-type traits: load/store one element as float.
template <typename T> struct Elt;
template <> struct Elt<float> {
  static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
  // value as it would be after a store + load (identity for float)
  static __device__ __forceinline__ float round(float v) { return v; }
};
template <> struct Elt<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
  static __device__ __forceinline__ void store(bf16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
  static __device__ __forceinline__ float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
};

// Load 16 bytes of T starting at element i (i aligned to 16/sizeof(T)) as floats.
template <typename T> struct Vec16;
template <> struct Vec16<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void load(const float* p, size_t i, float* out) {
    float4 v = *reinterpret_cast<const float4*>(p + i);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  }
};
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void load(const bf16_t* p, size_t i, float* out) {
    uint4 v = *reinterpret_cast<const uint4*>(p + i);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[2 * j] = __uint_as_float(w[j] << 16);
      out[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
};

// Store 8 consecutive values (aligned to 16 bytes for bf16, 32 for float) in
// the storage type, rounded as Elt::store rounds them.
template <typename T> __device__ __forceinline__ void store8(T* p, size_t i, const float* v);
template <> __device__ __forceinline__ void store8<float>(float* p, size_t i, const float* v) {
  *reinterpret_cast<float4*>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <> __device__ __forceinline__ void store8<bf16_t>(bf16_t* p, size_t i, const float* v) {
  *reinterpret_cast<uint4*>(p + i) =
      make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
}

// Load N consecutive elements of T (N = 4 or 8, aligned) as floats.
template <typename T, int N>
__device__ __forceinline__ void load_n(const T* p, size_t i, float* out) {
  constexpr int V = Vec16<T>::N;
  static_assert(N % V == 0 || V % N == 0, "vector width");
  if constexpr (N >= V) {
#pragma unroll
    for (int j = 0; j < N; j += V) Vec16<T>::load(p, i + j, out + j);
  } else {
#pragma unroll
    for (int j = 0; j < N; ++j) out[j] = Elt<T>::load(p, i + j);
  }
}

// Cross-lane reductions on DPP moves (a few cycles each, against a few
// hundred for an LDS permute).  Inside a row of 16 lanes: exchange with lane
// i^1, then i^2 (quad permutes), then the mirror in each half row (i <-> 7-i)
// and in the row (i <-> 15-i).  Each step adds a lane's value and its partner's,
// which both lanes of a pair compute alike, so after the four steps all 16
// lanes hold the bitwise same total, in a fixed order.
constexpr int kDppXor1 = 0xB1;         // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror

template <int CTRL> __device__ __forceinline__ uint32_t dpp_u(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL> __device__ __forceinline__ float dpp_f(float v) {
  return __uint_as_float(dpp_u<CTRL>(__float_as_uint(v)));
}

__device__ __forceinline__ float group16_sum(float v) {
  v += dpp_f<kDppXor1>(v);
  v += dpp_f<kDppXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return v;
}
__device__ __forceinline__ uint32_t group16_or(uint32_t v) {
  v |= dpp_u<kDppXor1>(v);
  v |= dpp_u<kDppXor2>(v);
  v |= dpp_u<kDppHalfMirror>(v);
  v |= dpp_u<kDppMirror>(v);
  return v;
}

// Best (larger key, then lower index) over each row of 16 lanes.  The
// combination is associative and commutative, so every lane ends with the
// same pair.
__device__ __forceinline__ void best_take(uint32_t& bk, uint32_t& bi, uint32_t ok, uint32_t oi) {
  if (ok > bk || (ok == bk && oi < bi)) { bk = ok; bi = oi; }
}
__device__ __forceinline__ void group16_best(uint32_t& bk, uint32_t& bi) {
  best_take(bk, bi, dpp_u<kDppXor1>(bk), dpp_u<kDppXor1>(bi));
  best_take(bk, bi, dpp_u<kDppXor2>(bk), dpp_u<kDppXor2>(bi));
  best_take(bk, bi, dpp_u<kDppHalfMirror>(bk), dpp_u<kDppHalfMirror>(bi));
  best_take(bk, bi, dpp_u<kDppMirror>(bk), dpp_u<kDppMirror>(bi));
}

// Running log-sum-exp of a row as (m, s): m the largest value seen, s the sum
// of exp(x - m) over the values seen; log-sum-exp = m + log(s).  The empty
// state is (-inf, 0).
__device__ __forceinline__ void lse_take(float& m, float& s, float x) {
  if (x > m) {
    s = s * expf(m - x) + 1.f;
    m = x;
  } else {
    s += expf(x - m);
  }
}
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;   // both empty
  s = s * expf(m - mn) + s2 * expf(m2 - mn);
  m = mn;
}
__device__ __forceinline__ void group16_lse(float& m, float& s) {
  lse_merge(m, s, dpp_f<kDppXor1>(m), dpp_f<kDppXor1>(s));
  lse_merge(m, s, dpp_f<kDppXor2>(m), dpp_f<kDppXor2>(s));
  lse_merge(m, s, dpp_f<kDppHalfMirror>(m), dpp_f<kDppHalfMirror>(s));
  lse_merge(m, s, dpp_f<kDppMirror>(m), dpp_f<kDppMirror>(s));
}

// Whole-wave sum / max: the four row results (lanes 0, 16, 32, 48) are read
// into scalars and combined as (r0 + r1) + (r2 + r3), the same in every lane.
// All 64 lanes must be active.
__device__ __forceinline__ float lane_read(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = group16_sum(v);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
  v = group16_max(v);
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}

template <int M> struct Log2 { static constexpr int v = 1 + Log2<M / 2>::v; };
template <> struct Log2<1> { static constexpr int v = 0; };

// Order-preserving map of a float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// LayerNorm statistics of one row of K elements (K a multiple of 8,
// K <= 128 * NT) computed by a group of 16 consecutive lanes.  Lane j of the
// group holds elements k = 8*j + 128*t + e (t < NT, e < 8, k < K) in v[t][e]
// and sums them in that order (the result does not depend on NT once
// 128 * NT >= K: absent chunks are never added); the 16 lane sums are combined by xor-1, 2, 4, 8 pairings.
// Mean first, then the mean of squared deviations (two passes over the values
// held in registers).  All 64 lanes of the wave must call this (invalid rows
// pass valid = false and contribute zeros).  The matrix-product prologue and
// the row LayerNorm kernel both use it, so a row's statistics are bitwise the
// same wherever they are computed.
// LayerNorm of a row of K elements (K a multiple of 8, K <= 512 * NT) by one
// wave: lane j holds elements k = 8j + 512t + e (slab t < NT, e < 8).  Every
// LayerNorm of the decoder (product and vocabulary prologues, the stand-alone
// kernel) uses this split and order, so a row's normalised values are bitwise
// the same wherever they are computed.
//
// The slabs are always loaded (from a valid address, so no load sits under a
// branch); those outside the row are zeroed by mask() once the data is there.
// bf16 rows stay packed and are widened on use, which is exact.
template <typename XT, int NT> struct LnRow {
  float v[NT][8];
  uint32_t live;
  __device__ __forceinline__ void load_slab(const XT* x, int t, int k0) { load_n<XT, 8>(x, k0, v[t]); }
  __device__ __forceinline__ void mask() {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) v[t][e] = ((live >> t) & 1u) ? v[t][e] : 0.f;
  }
  __device__ __forceinline__ float get(int t, int e) const { return v[t][e]; }
};
template <int NT> struct LnRow<bf16_t, NT> {
  uint32_t w[NT][4];
  uint32_t live;
  __device__ __forceinline__ void load_slab(const bf16_t* x, int t, int k0) {
    const uint4 q = *reinterpret_cast<const uint4*>(x + k0);
    w[t][0] = q.x; w[t][1] = q.y; w[t][2] = q.z; w[t][3] = q.w;
  }
  __device__ __forceinline__ void mask() {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) w[t][i] = ((live >> t) & 1u) ? w[t][i] : 0u;
  }
  __device__ __forceinline__ float get(int t, int e) const {
    const uint32_t u = w[t][e >> 1];
    return __uint_as_float((e & 1) ? (u & 0xffff0000u) : (u << 16));
  }
};

// Issue the loads of row x (valid: the row exists; otherwise zeros).
template <typename XT, int NT>
__device__ __forceinline__ void ln_row_load(LnRow<XT, NT>& h, const XT* x, int K, int lane, bool valid) {
  h.live = 0u;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int k0 = 8 * lane + 512 * t;
    const bool in = valid && k0 < K;
    h.load_slab(x, t, in ? k0 : 0);
    h.live |= (in ? 1u : 0u) << t;
  }
}

// Mean and 1 / sqrt(var + eps) of the row (two-pass variance).  All 64 lanes
// must be active.
template <typename XT, int NT>
__device__ __forceinline__ void ln_row_stats(LnRow<XT, NT>& h, int K, float eps, float& mean, float& rstd) {
  h.mask();
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) s += h.get(t, e);
  mean = wave_sum(s) / static_cast<float>(K);
  float q = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if ((h.live >> t) & 1u) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = h.get(t, e) - mean;
        q = fmaf(d, d, q);
      }
    }
  }
  rstd = 1.0f / sqrtf(wave_sum(q) / static_cast<float>(K) + eps);
}

// LayerNorm of one element given its row statistics (same expression
// everywhere it is evaluated, so the result is bitwise identical).
__device__ __forceinline__ float ln_apply(float x, float mean, float rstd, float g, float b) {
  return fmaf((x - mean) * rstd, g, b);
}

}  // namespace pdec

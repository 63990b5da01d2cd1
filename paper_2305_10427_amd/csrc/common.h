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

// Round-to-nearest-even float -> bfloat16 (NaN kept quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return static_cast<bf16_t>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
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

// Butterfly sum over the 64 lanes of a wave; every lane gets the total.
// The pairing order is fixed, so the result is bitwise reproducible.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// Sum of M values per lane across the 64 lanes of a wave (M a power of two,
// M <= 64).  Halving exchange: after log2(M) steps each lane holds one partial
// of value index j = lane >> (6 - log2 M); the remaining steps finish the sum
// inside groups of 64 / M lanes.  Returns the total of value j in every lane of
// group j.  Fixed pairing order: bitwise reproducible.
template <int M>
__device__ __forceinline__ float wave_reduce_scatter(float (&v)[M], int lane) {
  static_assert(M >= 1 && M <= 64 && (M & (M - 1)) == 0, "M must be a power of two <= 64");
  int off = 32;
#pragma unroll
  for (int half = M / 2; half >= 1; half >>= 1, off >>= 1) {
    const bool upper = (lane & off) != 0;
#pragma unroll
    for (int j = 0; j < half; ++j) {
      float a = v[j], b = v[j + half];
      // opaque copies: the per-lane choice must stay a select of two values,
      // not become a lane-dependent index into v (a long compare/select chain)
      __asm__("" : "+v"(a), "+v"(b));
      const float send = upper ? a : b;
      const float keep = upper ? b : a;
      v[j] = keep + __shfl_xor(send, off);
    }
  }
  float r = v[0];
  for (; off >= 1; off >>= 1) r += __shfl_xor(r, off);
  return r;
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
// Row elements held by one lane of a 16-lane LayerNorm group: eight
// consecutive elements per 128-element slab.  bf16 rows stay packed (four
// words per slab) and are widened on use, which is exact.
template <typename XT, int NT> struct LnHold {
  float v[NT][8];
  __device__ __forceinline__ void load(const XT* x, int t, int k0) { load_n<XT, 8>(x, k0, v[t]); }
  __device__ __forceinline__ void clear(int t) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[t][e] = 0.f;
  }
  __device__ __forceinline__ float get(int t, int e) const { return v[t][e]; }
};
template <int NT> struct LnHold<bf16_t, NT> {
  uint32_t w[NT][4];
  __device__ __forceinline__ void load(const bf16_t* x, int t, int k0) {
    const uint4 q = *reinterpret_cast<const uint4*>(x + k0);
    w[t][0] = q.x; w[t][1] = q.y; w[t][2] = q.z; w[t][3] = q.w;
  }
  __device__ __forceinline__ void clear(int t) {
#pragma unroll
    for (int e = 0; e < 4; ++e) w[t][e] = 0u;
  }
  __device__ __forceinline__ float get(int t, int e) const {
    const uint32_t u = w[t][e >> 1];
    return __uint_as_float((e & 1) ? (u & 0xffff0000u) : (u << 16));
  }
};

template <typename XT, int NT>
__device__ __forceinline__ void ln_load_g16(const XT* x, int K, int j, bool valid, LnHold<XT, NT>& h) {
  static_assert(NT >= 1 && NT <= 8, "at most 1024 elements");
  const XT* xj = x + 8 * j;   // slab t of this lane starts 128 * t elements further on
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (valid && 8 * j + 128 * t < K) h.load(xj, t, 128 * t);
    else h.clear(t);
  }
}

template <typename XT, int NT>
__device__ __forceinline__ void ln_stats_held(const LnHold<XT, NT>& h, int K, int j, float eps, float& mean,
                                              float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) s += h.get(t, e);
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) s += __shfl_xor(s, off);
  mean = s / static_cast<float>(K);
  float q = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (8 * j + 128 * t < K) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = h.get(t, e) - mean;
        q = fmaf(d, d, q);
      }
    }
  }
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) q += __shfl_xor(q, off);
  rstd = 1.0f / sqrtf(q / static_cast<float>(K) + eps);
}

template <typename XT, int NT>
__device__ __forceinline__ void ln_stats_g16(const XT* x, int K, int j, float eps, bool valid,
                                             LnHold<XT, NT>& h, float& mean, float& rstd) {
  ln_load_g16<XT, NT>(x, K, j, valid, h);
  ln_stats_held<XT, NT>(h, K, j, eps, mean, rstd);
}

// LayerNorm of one element given its row statistics (same expression
// everywhere it is evaluated, so the result is bitwise identical).
__device__ __forceinline__ float ln_apply(float x, float mean, float rstd, float g, float b) {
  return fmaf((x - mean) * rstd, g, b);
}

}  // namespace pdec

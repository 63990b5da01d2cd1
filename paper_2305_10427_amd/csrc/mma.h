// MFMA building blocks shared by the matrix-product kernels (gfx950).
#pragma once

#include "common.h"

namespace pdec {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  static constexpr int KS = 32;
  static constexpr int EPL = 8;
  typedef uint4 frag;
  static __device__ __forceinline__ floatx4_t step(frag a, frag b, floatx4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const bf16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  // NT: a non-temporal load (global_load ... nt), for data a launch streams
  // once, such as the weights of a batch-1 product
  template <int NT> static __device__ __forceinline__ frag wload(const bf16_t* p) {
    if constexpr (NT != 0) {
      const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
      return make_uint4(t.x, t.y, t.z, t.w);
    } else {
      return load(p);
    }
  }
  static __device__ __forceinline__ frag zero() { return make_uint4(0, 0, 0, 0); }
  static __device__ __forceinline__ void unpack(frag f, float* v) {
    const uint32_t w[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ frag pack(const float* v) {
    return make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                      pack_bf16x2(v[6], v[7]));
  }
};
template <> struct Mma<float> {
  static constexpr int KS = 16;
  static constexpr int EPL = 4;
  typedef float4 frag;
  static __device__ __forceinline__ floatx4_t step(frag a, frag b, floatx4_t c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ frag load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  template <int NT> static __device__ __forceinline__ frag wload(const float* p) {
    if constexpr (NT != 0) {
      const floatx4_t t = __builtin_nontemporal_load(reinterpret_cast<const floatx4_t*>(p));
      return make_float4(t.x, t.y, t.z, t.w);
    } else {
      return load(p);
    }
  }
  static __device__ __forceinline__ frag zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void unpack(frag f, float* v) { v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w; }
  static __device__ __forceinline__ frag pack(const float* v) { return make_float4(v[0], v[1], v[2], v[3]); }
};

// max(v, 0) that keeps a NaN (fmaxf would return 0 for it and hide a
// non-finite value from the argmax's check).
__device__ __forceinline__ float relu(float v) { return v < 0.f ? 0.f : v; }

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

// Normalised values of a row (statistics from ln_row_stats) rounded to the
// storage type and written to dst (one row; lane j writes elements
// 8j + 512t .. +7) and, when out is non-null, also to out.  g, b: gamma and
// beta, in global memory or LDS.
template <typename WT, typename XT, int NT>
__device__ __forceinline__ void ln_row_apply(const LnRow<XT, NT>& h, int K, float mean, float rstd, const WT* g,
                                             const WT* b, WT* dst, WT* out, int lane) {
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int k0 = 8 * lane + 512 * t;
    if (k0 < K) {
      float gv[8], bv[8], y[8];
      load_n<WT, 8>(g, k0, gv);
      load_n<WT, 8>(b, k0, bv);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = ln_apply(h.get(t, e), mean, rstd, gv[e], bv[e]);
      store8<WT>(dst, k0, y);
      if (out != nullptr) store8<WT>(out, k0, y);
    }
  }
}

// LayerNorm of the 16-row input tile rows m0 .. m0+15 into the LDS tile
// sA[16][lda] in the storage type, by 4 waves: wave w owns tile rows
// w, w + 4, w + 8, w + 12 (one row per pass; NPASS passes, so rows
// m0 .. m0 + 4 NPASS - 1).  load() issues the loads of those rows (rows
// >= R_max read row 0 and are not used), so a caller can issue other loads
// after it; finish() normalises the passes that hold rows below
// R_max (rows of later passes are left unwritten: their products are
// discarded) and also writes rows below R_out to ln_out when it is non-null.
// The caller synchronises the workgroup after finish().
template <typename WT, typename XT, int NT, int NPASS = 4> struct LnTile {
  LnRow<XT, NT> h[NPASS];
  int wave, lane, m0, R_max;
  __device__ __forceinline__ void load(const XT* X, int ldx, int K, int m0_, int R_max_, int wave_, int lane_) {
    wave = wave_;
    lane = lane_;
    m0 = m0_;
    R_max = R_max_;
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int row = m0 + 4 * p + wave;
      const bool ok = row < R_max;
      ln_row_load<XT, NT>(h[p], X + static_cast<size_t>(ok ? row : 0) * ldx, K, lane, ok);
    }
  }
  __device__ __forceinline__ void finish(int K, float eps, const WT* g, const WT* b, WT* sA, int lda, WT* ln_out,
                                         int ldlo, int R_out) {
    const int n_pass = min(NPASS, (R_max - m0 + 3) / 4);
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      if (p < n_pass) {
        const int tr = 4 * p + wave;
        const int row = m0 + tr;
        float mean, rstd;
        ln_row_stats<XT, NT>(h[p], K, eps, mean, rstd);
        WT* out = (ln_out != nullptr && row < R_out) ? ln_out + static_cast<size_t>(row) * ldlo : nullptr;
        ln_row_apply<WT, XT, NT>(h[p], K, mean, rstd, g, b, sA + static_cast<size_t>(tr) * lda, out, lane);
      }
    }
  }
};

}  // namespace pdec

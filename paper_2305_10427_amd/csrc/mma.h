// MFMA building blocks shared by the matrix-product kernels (gfx950).
#pragma once

#include "common.h"

namespace pdec {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

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
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w[j] = static_cast<uint32_t>(f32_to_bf16(v[2 * j])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * j + 1])) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
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
  static __device__ __forceinline__ frag zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void unpack(frag f, float* v) { v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w; }
  static __device__ __forceinline__ frag pack(const float* v) { return make_float4(v[0], v[1], v[2], v[3]); }
};

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

// LayerNorm of the 16-row input tile rows m0 .. m0+15 (rows >= R_max read as
// zeros) into the LDS tile sA[16][lda] in the storage type, by waves 0..3:
// wave w owns tile rows 4w .. 4w+3 with 16 lanes per row (statistics as in
// ln_stats_g16).  load() issues the row loads and finish() computes the
// statistics and writes the normalised rows (also to ln_out, rows below
// R_out, when it is non-null), so a caller can issue other loads in between.
// The caller synchronises the workgroup after finish().
template <typename WT, typename XT, int LNT> struct LnTileRows {
  LnHold<XT, LNT> h;
  int lr, tr, row;
  bool ok;
  __device__ __forceinline__ void load(const XT* X, int ldx, int K, int m0, int R_max, int wave, int lane) {
    lr = lane & 15;
    tr = 4 * wave + (lane >> 4);
    row = m0 + tr;
    ok = row < R_max;
    ln_load_g16<XT, LNT>(X + static_cast<size_t>(ok ? row : 0) * ldx, K, lr, ok, h);
  }
  // g, b: gamma and beta, in global memory or LDS
  __device__ __forceinline__ void finish(int K, float eps, const WT* g, const WT* b, WT* sA, int lda, WT* ln_out,
                                         int ldlo, int R_out) {
    float mean, rstd;
    ln_stats_held<XT, LNT>(h, K, lr, eps, mean, rstd);
    const bool write_out = ln_out != nullptr && row < R_out;
    // per-lane bases; slab t adds the constant 128 * t
    const WT* gj = g + 8 * lr;
    const WT* bj = b + 8 * lr;
    WT* aj = sA + static_cast<size_t>(tr) * lda + 8 * lr;
    WT* oj = write_out ? ln_out + static_cast<size_t>(row) * ldlo + 8 * lr : nullptr;
#pragma unroll
    for (int t = 0; t < LNT; ++t) {
      if (8 * lr + 128 * t < K) {
        float gv[8], bv[8], y[8];
        load_n<WT, 8>(gj, 128 * t, gv);
        load_n<WT, 8>(bj, 128 * t, bv);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = Elt<WT>::round(ln_apply(h.get(t, e), mean, rstd, gv[e], bv[e]));
#pragma unroll
        for (int e = 0; e < 8; ++e) Elt<WT>::store(aj, 128 * t + e, y[e]);
        if (write_out) {
#pragma unroll
          for (int e = 0; e < 8; ++e) Elt<WT>::store(oj, 128 * t + e, y[e]);
        }
      }
    }
  }
};

}  // namespace pdec

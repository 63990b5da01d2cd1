// Scaled dot-product attention of one query row by one wave, in chunks of 64
// keys.
//
// For one chunk (keys key0 .. key0+63 that are < nk):
//   s_k = (q . k_k) * scale          lane k scores key key0 + k
//   m_c = max_k s_k,  p_k = exp(s_k - m_c),  l_c = sum_k p_k     (DPP trees)
//   o_c[d] = sum_k p_k v_k[d]        lane d, four partial sums over the keys
//                                    (p and the V rows staged through LDS)
// and a row's chunks are folded in chunk order:
//   m' = max(m, m_c),  o <- o exp(m - m') + o_c exp(m_c - m'),  l likewise,
// the output being o / l.  Chunk boundaries depend only on the row's own key
// count, never on how many rows a launch holds.
#pragma once

#include "common.h"

namespace pdec {

constexpr int kAttnChunk = kWave;   // keys per chunk

// Running state of one row: m, l wave-uniform; lane d owns output dimensions
// d, d + 64, ...
template <int DH> struct RowState {
  static constexpr int NO = (DH + kWave - 1) / kWave;
  float m, l;
  float o[NO];
  __device__ __forceinline__ void init() {
    m = -INFINITY;
    l = 0.f;
#pragma unroll
    for (int i = 0; i < NO; ++i) o[i] = 0.f;
  }
};

// The K and V rows of the key a lane scores, as raw 16-byte words.  V is held only when it fits comfortably in registers
// (<= 256 bytes per row); otherwise it is read again when staged.
template <typename AT, int DH> struct KeyRows {
  static constexpr int V16 = Vec16<AT>::N;        // elements per 16-byte word
  static constexpr int NW = DH / V16;             // words per row
  static constexpr bool HOLD_V = DH * sizeof(AT) <= 256;
  uint4 k[NW];
  uint4 v[HOLD_V ? NW : 1];
  // always loads (key 0 for an invalid lane): no load under a branch
  __device__ __forceinline__ void load(const AT* Kb, const AT* Vb, int key, bool valid) {
    key = valid ? key : 0;
    const uint4* kr = reinterpret_cast<const uint4*>(Kb + static_cast<size_t>(key) * DH);
#pragma unroll
    for (int i = 0; i < NW; ++i) k[i] = kr[i];
    if constexpr (HOLD_V) {
      const uint4* vr = reinterpret_cast<const uint4*>(Vb + static_cast<size_t>(key) * DH);
#pragma unroll
      for (int i = 0; i < NW; ++i) v[i] = vr[i];
    }
  }
};

// Per-wave LDS staging of one chunk: the weights p_k and DP dimensions of the
// 64 V rows at a time (rows padded by 16 bytes).
template <typename AT, int DH> struct AttnStage {
  static constexpr int DP0 = 8192 / (kAttnChunk * static_cast<int>(sizeof(AT)));
  static constexpr int DP = DH < DP0 ? DH : DP0;  // dimensions per pass: 64 (bf16), 32 (f32)
  static constexpr int LDV = DP + 16 / static_cast<int>(sizeof(AT));
  float p[kAttnChunk];
  AT v[kAttnChunk * LDV];
};

template <typename AT> __device__ __forceinline__ void unpack_word(uint4 w, float* out);
template <> __device__ __forceinline__ void unpack_word<float>(uint4 w, float* out) {
  out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
  out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
}
template <> __device__ __forceinline__ void unpack_word<bf16_t>(uint4 w, float* out) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    out[2 * j] = __uint_as_float(u[j] << 16);
    out[2 * j + 1] = __uint_as_float(u[j] & 0xffff0000u);
  }
}

// Orders the wave's LDS writes before its following reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One chunk folded into the row state.  q: the row's query (DH floats, LDS);
// kr: the lane's key (key0 + lane) when it is < nk; Vb: key 0 of the row's
// [T][DH] V slice.  All 64 lanes must be active.
template <typename AT, int DH>
__device__ __forceinline__ void chunk_fold(const float* q, const KeyRows<AT, DH>& kr, const AT* Vb, int key0, int nk,
                                           float scale, int lane, AttnStage<AT, DH>& sm, RowState<DH>& st) {
  using KR = KeyRows<AT, DH>;
  using SM = AttnStage<AT, DH>;
  constexpr int V16 = KR::V16;
  const int key = key0 + lane;
  const bool valid = key < nk;
  // q . k as four interleaved partial sums (element e of each word to sum e % 4)
  float acc4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < KR::NW; ++i) {
    float kv[V16];
    unpack_word<AT>(kr.k[i], kv);
#pragma unroll
    for (int e = 0; e < V16; ++e) acc4[e & 3] = fmaf(q[i * V16 + e], kv[e], acc4[e & 3]);
  }
  const float acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
  const float sc = valid ? acc * scale : -INFINITY;
  const float mc = wave_max(sc);
  const float p = valid ? expf(sc - mc) : 0.f;
  const float lc = wave_sum(p);
  const float mn = fmaxf(st.m, mc);
  const float a1 = expf(st.m - mn);
  const float a2 = expf(mc - mn);
  sm.p[lane] = p;                                  // zero past the row's keys
#pragma unroll
  for (int p0 = 0; p0 < DH; p0 += SM::DP) {
    // stage dimensions p0 .. p0+DP of the lane's V row (zeros past the row)
    uint4* dst = reinterpret_cast<uint4*>(sm.v + lane * SM::LDV);
#pragma unroll
    for (int i = 0; i < SM::DP / V16; ++i) {
      uint4 w;
      if constexpr (KR::HOLD_V) {
        w = kr.v[p0 / V16 + i];
      } else {
        w = reinterpret_cast<const uint4*>(Vb + static_cast<size_t>(valid ? key : 0) * DH + p0)[i];
      }
      dst[i] = valid ? w : make_uint4(0u, 0u, 0u, 0u);
    }
    wave_lds_sync();
    // lane (p0 + j) % 64 sums dimension p0 + j over all 64 keys of the chunk
    // (keys past the row have p = 0 and zero rows: exact zeros)
    const int j = lane - (p0 % kWave);
    if (j >= 0 && j < SM::DP) {
      float o4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < kAttnChunk; ++k)
        o4[k & 3] = fmaf(sm.p[k], Elt<AT>::load(sm.v, k * SM::LDV + j), o4[k & 3]);
      const float oc = (o4[0] + o4[1]) + (o4[2] + o4[3]);
      float& so = st.o[(p0 + j) / kWave];
      so = so * a1 + oc * a2;
    }
    wave_lds_sync();
  }
  st.l = st.l * a1 + lc * a2;
  st.m = mn;
}

// Final output o / l of a row's head slice.
template <typename AT, int DH>
__device__ __forceinline__ void row_output(const RowState<DH>& st, AT* out, int lane) {
#pragma unroll
  for (int i = 0; i < RowState<DH>::NO; ++i) {
    const int d = lane + kWave * i;
    if (d < DH) Elt<AT>::store(out, d, st.o[i] / st.l);
  }
}

}  // namespace pdec

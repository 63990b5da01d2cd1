// Scaled dot-product attention of one query row, evaluated in chunks of 64
// keys (one key per lane).
//
// For one chunk (keys key0 .. key0+63 that are < nk):
//   s_k = (q . k_k) * scale,  m_c = max_k s_k,  p_k = exp(s_k - m_c),
//   l_c = sum_k p_k,  o_c = sum_k p_k v_k            (fixed lane trees)
// and a row's chunks are folded in chunk order:
//   m' = max(m, m_c),  o <- o exp(m - m') + o_c exp(m_c - m'),  l likewise,
// the output being o / l.  Chunk boundaries depend only on the row's own key
// count, never on how many rows a launch holds or on which wave does a chunk.
#pragma once

#include "common.h"

namespace pdec {

constexpr int kAttnChunk = kWave;   // keys per chunk

template <int DH> struct AttnSlot {
  float m, l;
  float o[DH];
};

// Running state of one row, held by one wave: m, l wave-uniform, lane d owns
// output dimensions d, d + 64, ...
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

// The K and V rows of the key a lane scores, as raw 16-byte words, loaded
// before anything else so that their latency overlaps the query load.  V is
// held only when it fits comfortably in registers (<= 256 bytes per row);
// otherwise it is loaded pass by pass.
template <typename AT, int DH> struct KeyRows {
  static constexpr int V16 = Vec16<AT>::N;        // elements per 16-byte word
  static constexpr int NW = DH / V16;             // words per row
  static constexpr bool HOLD_V = DH * sizeof(AT) <= 256;
  uint4 k[NW];
  uint4 v[HOLD_V ? NW : 1];
  __device__ __forceinline__ void load(const AT* Kb, const AT* Vb, int key, bool valid) {
    if (!valid) return;
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

// Partial of one chunk into *slot.  q is the row's query (DH floats, any
// address space); kr holds the lane's key (key0 + lane) when it is < nk;
// Vb points at key 0 of the row's [T][DH] V slice (used when V is not held).
template <typename AT, int DH>
__device__ __forceinline__ void chunk_partial(const float* q, const KeyRows<AT, DH>& kr, const AT* Vb, int key0,
                                              int nk, float scale, int lane, AttnSlot<DH>* slot) {
  using KR = KeyRows<AT, DH>;
  constexpr int V16 = KR::V16;
  const int key = key0 + lane;
  const bool valid = key < nk;
  float sc = -INFINITY;
  if (valid) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < KR::NW; ++i) {
      float kv[V16];
      unpack_word<AT>(kr.k[i], kv);
#pragma unroll
      for (int e = 0; e < V16; ++e) acc = fmaf(q[i * V16 + e], kv[e], acc);
    }
    sc = acc * scale;
  }
  const float m = wave_max(sc);
  const float p = valid ? expf(sc - m) : 0.f;
  const float l = wave_sum(p);
  constexpr int HB = DH < 16 ? DH : 16;          // output dimensions per reduction pass
  constexpr int SPREAD = kWave / HB;             // lanes holding each reduced value
#pragma unroll
  for (int h0 = 0; h0 < DH; h0 += HB) {
    float pv[HB];
    if (valid) {
#pragma unroll
      for (int d = 0; d < HB; d += V16) {
        float vv[V16];
        if constexpr (KR::HOLD_V) {
          unpack_word<AT>(kr.v[(h0 + d) / V16], vv);
        } else {
          Vec16<AT>::load(Vb + static_cast<size_t>(key) * DH + h0, d, vv);
        }
#pragma unroll
        for (int e = 0; e < V16; ++e) pv[d + e] = p * vv[e];
      }
    } else {
#pragma unroll
      for (int d = 0; d < HB; ++d) pv[d] = 0.f;
    }
    const float r = wave_reduce_scatter<HB>(pv, lane);
    if ((lane & (SPREAD - 1)) == 0) slot->o[h0 + lane / SPREAD] = r;
  }
  if (lane == 0) {
    slot->m = m;
    slot->l = l;
  }
}

// Fold one chunk partial into a row's running state.
template <int DH>
__device__ __forceinline__ void merge_chunk(RowState<DH>& st, const AttnSlot<DH>* c, int lane) {
  const float cm = c->m;
  const float mn = fmaxf(st.m, cm);
  const float a1 = expf(st.m - mn);
  const float a2 = expf(cm - mn);
#pragma unroll
  for (int i = 0; i < RowState<DH>::NO; ++i) {
    const int d = lane + kWave * i;
    const float co = d < DH ? c->o[d] : 0.f;
    st.o[i] = st.o[i] * a1 + co * a2;
  }
  st.l = st.l * a1 + c->l * a2;
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

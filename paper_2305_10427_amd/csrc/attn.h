// Scaled dot-product attention of one query row by one wave, in chunks of 64
// keys.
//
// For one chunk (keys key0 .. key0+63 that are < nk):
//   s_k = (q . k_k) * scale          lane k scores key key0 + k
//   m_c = max_k s_k,  p_k = exp(s_k - m_c),  l_c = sum_k p_k     (DPP trees)
//   o_c[d] = sum_k p_k v_k[d]        two dimensions per lane over a half of the
//                                    keys (V read directly, p through LDS)
// and a row's chunks are folded in chunk order:
//   m' = max(m, m_c),  o <- o exp(m - m') + o_c exp(m_c - m'),  l likewise,
// the output being o / l.  Chunk boundaries depend only on the row's own key
// count, never on how many rows a launch holds.
#pragma once

#include "common.h"

namespace pdec {

constexpr int kAttnChunk = kWave;   // keys per chunk

// Running state of one row: m, l wave-uniform; lane l < 32 owns output
// dimensions 2l, 2l + 1 (+ 64 i).
template <int DH> struct RowState {
  static constexpr int NP = (DH + kWave - 1) / kWave;   // 64-dimension groups
  float m, l;
  float o[NP][2];
  __device__ __forceinline__ void init() {
    m = -INFINITY;
    l = 0.f;
#pragma unroll
    for (int i = 0; i < NP; ++i) o[i][0] = o[i][1] = 0.f;
  }
};

// One chunk of a row's keys, in registers: lane k holds the K row of key
// key0 + k (raw 16-byte words), and lane l the V entries of dimensions
// 2(l mod 32), 2(l mod 32) + 1 (+ 64 i) for the 32 keys key0 + 32(l / 32) + k'.
// Keys past nk are loaded from key 0 (every load unconditional) and dropped.
template <typename AT, int DH> struct KeyChunk {
  static constexpr int V16 = Vec16<AT>::N;        // elements per 16-byte word
  static constexpr int NW = DH / V16;             // K words per row
  static constexpr int NP = (DH + kWave - 1) / kWave;
  using Pair = typename std::conditional<sizeof(AT) == 2, uint32_t, uint2>::type;   // two elements
  uint4 k[NW];
  Pair v[NP][32];
  __device__ __forceinline__ void load(const AT* Kb, const AT* Vb, int key0, int nk, int lane) {
    load_k(Kb, key0, nk, lane);
    load_v(Vb, key0, nk, lane);
  }
  __device__ __forceinline__ void load_k(const AT* Kb, int key0, int nk, int lane) {
    const int key = key0 + lane < nk ? key0 + lane : 0;
    const uint4* kr = reinterpret_cast<const uint4*>(Kb + static_cast<size_t>(key) * DH);
#pragma unroll
    for (int i = 0; i < NW; ++i) k[i] = kr[i];
  }
  __device__ __forceinline__ void load_v(const AT* Vb, int key0, int nk, int lane) {
    const int d0 = 2 * (lane & 31);
    const int kh = key0 + 32 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int d = d0 + kWave * i < DH ? d0 + kWave * i : 0;
#pragma unroll
      for (int k2 = 0; k2 < 32; ++k2) {
        const int kk = kh + k2 < nk ? kh + k2 : 0;
        v[i][k2] = *reinterpret_cast<const Pair*>(Vb + static_cast<size_t>(kk) * DH + d);
      }
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
__device__ __forceinline__ void unpack_pair(uint32_t w, float& a, float& b) {
  a = __uint_as_float(w << 16);
  b = __uint_as_float(w & 0xffff0000u);
}
__device__ __forceinline__ void unpack_pair(uint2 w, float& a, float& b) {
  a = __uint_as_float(w.x);
  b = __uint_as_float(w.y);
}

// Per-wave LDS of the chunk computation: the weights p_k.
struct AttnScratch {
  float p[kAttnChunk];
};

// Lane l < 32 receives v of lane l + 32 (v_permlane32_swap exchanges the
// upper half of its first operand with the lower half of its second).
__device__ __forceinline__ float upper_half(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[1]);
}

// Orders the wave's LDS writes before its following reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One chunk's own softmax statistics and unnormalised output: m_c, l_c and
// o_c (lane l < 32: dimensions 2l, 2l + 1 (+ 64 i)).
template <int DH> struct ChunkOut {
  float m, l;
  float o[RowState<DH>::NP][2];
};

// Evaluates one chunk (keys key0 .. key0+63 below nk) for the query q (DH
// floats, LDS).  All 64 lanes must be active.
template <typename AT, int DH>
__device__ __forceinline__ void chunk_eval(const float* q, const KeyChunk<AT, DH>& kc, int key0, int nk, float scale,
                                           int lane, AttnScratch& sm, ChunkOut<DH>& c) {
  using KC = KeyChunk<AT, DH>;
  constexpr int V16 = KC::V16;
  const bool valid = key0 + lane < nk;
  // q . k as four interleaved partial sums
  float acc4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < KC::NW; ++i) {
    float kv[V16];
    unpack_word<AT>(kc.k[i], kv);
#pragma unroll
    for (int e = 0; e < V16; ++e) acc4[e & 3] = fmaf(q[i * V16 + e], kv[e], acc4[e & 3]);
  }
  const float acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
  const float sc = valid ? acc * scale : -INFINITY;
  const float mc = wave_max(sc);
  const float p = valid ? expf(sc - mc) : 0.f;   // zero past the row's keys
  c.m = mc;
  c.l = wave_sum(p);
  sm.p[lane] = p;
  wave_lds_sync();
  // P.V: each lane sums its two dimensions over its half of the keys.  Keys
  // past nk have p = 0 and hold key 0's V entries (a value every row
  // attends to), so they add exact zeros: fmaf(0, v, acc) = acc for finite v.
  const int kh = 32 * (lane >> 5);
  float o[KC::NP][2];
#pragma unroll
  for (int i = 0; i < KC::NP; ++i) {
    float oa[4] = {0.f, 0.f, 0.f, 0.f}, ob[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k2 = 0; k2 < 32; ++k2) {
      float va, vb;
      unpack_pair(kc.v[i][k2], va, vb);
      const float pk = sm.p[kh + k2];
      oa[k2 & 3] = fmaf(pk, va, oa[k2 & 3]);
      ob[k2 & 3] = fmaf(pk, vb, ob[k2 & 3]);
    }
    o[i][0] = (oa[0] + oa[1]) + (oa[2] + oa[3]);
    o[i][1] = (ob[0] + ob[1]) + (ob[2] + ob[3]);
  }
  // lower key half + upper key half, per dimension group: lane l < 32 takes
  // lane l + 32's partial sums by a swap of the wave's halves (lanes >= 32
  // hold values that are never used)
#pragma unroll
  for (int i = 0; i < KC::NP; ++i) {
    c.o[i][0] = o[i][0] + upper_half(o[i][0]);
    c.o[i][1] = o[i][1] + upper_half(o[i][1]);
  }
}

// Folds an evaluated chunk into the row state (chunks in key order):
//   m' = max(m, m_c),  o <- o exp(m - m') + o_c exp(m_c - m'),  l likewise.
template <int DH>
__device__ __forceinline__ void fold_chunk(const ChunkOut<DH>& c, int lane, RowState<DH>& st) {
  const float mn = fmaxf(st.m, c.m);
  const float a1 = expf(st.m - mn);
  const float a2 = expf(c.m - mn);
#pragma unroll
  for (int i = 0; i < RowState<DH>::NP; ++i) {
    if (lane < 32) {
      st.o[i][0] = st.o[i][0] * a1 + c.o[i][0] * a2;
      st.o[i][1] = st.o[i][1] * a1 + c.o[i][1] * a2;
    }
  }
  st.l = st.l * a1 + c.l * a2;
  st.m = mn;
}

// One chunk folded into the row state.
template <typename AT, int DH>
__device__ __forceinline__ void chunk_fold(const float* q, const KeyChunk<AT, DH>& kc, int key0, int nk, float scale,
                                           int lane, AttnScratch& sm, RowState<DH>& st) {
  ChunkOut<DH> c;
  chunk_eval<AT, DH>(q, kc, key0, nk, scale, lane, sm, c);
  fold_chunk<DH>(c, lane, st);
}

// Final output o / l of a row's head slice: element d goes to out[at(d)]
// (d even: at(d + 1) = at(d) + 1 in every layout used).
template <typename AT, int DH, typename At>
__device__ __forceinline__ void row_output(const RowState<DH>& st, AT* out, At at, int lane) {
#pragma unroll
  for (int i = 0; i < RowState<DH>::NP; ++i) {
    const int d = 2 * lane + kWave * i;
    if (lane < 32 && d < DH) {
      const size_t o = at(d);
      Elt<AT>::store(out, o, st.o[i][0] / st.l);
      Elt<AT>::store(out, o + 1, st.o[i][1] / st.l);
    }
  }
}

}  // namespace pdec

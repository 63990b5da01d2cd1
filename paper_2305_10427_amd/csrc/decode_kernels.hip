// Attention, embedding, LayerNorm, argmax reduction and the on-device
// fixed-point control of the parallel decoding iteration.
#include "common.h"
#include "kernels.h"

namespace pdec {

constexpr int kMaxKeys = 1024;
constexpr int kMaxHeadDim = 128;

__device__ __forceinline__ void row_place(const RowMap& m, int row, int& s, int& p) {
  if (m.sent != nullptr) { s = m.sent[row]; p = m.pos[row]; }
  else { s = row / m.per_sent; p = row - s * m.per_sent; }
}

// ---------------------------------------------------------------------------
// Scaled dot-product attention, one wave per (row, head).
//
// The row at position p attends to keys 0..p of its own sentence (causal,
// decoder self-attention over the KV cache whose block entries were written by
// the QKV product of this iteration) or to keys 0..n_s-1 (encoder memory /
// encoder self-attention, padded keys excluded).  Keys are visited in a fixed
// order that depends only on the row's own key count, never on how many rows
// the iteration has: lane j scores keys j, j+64, ...; the softmax max/sum use
// fixed lane trees; lane d accumulates output dimension d over keys 0..n-1.
template <typename AT, int DH>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  __shared__ float s_p[4][kMaxKeys];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const int idx = blockIdx.x * 4 + wave;
  const int row = idx / a.H;
  const int hh = idx - row * a.H;
  const bool active = row < R;
  constexpr int dh = DH;
  const AT* __restrict__ Kc = static_cast<const AT*>(a.kc);
  const AT* __restrict__ Vc = static_cast<const AT*>(a.vc);
  int nk = 0;
  size_t base = 0;
  float denom = 1.f;
  if (active) {
    int s, p;
    row_place(a.rows, row, s, p);
    nk = a.causal ? p + 1 : a.klen[s];
    base = (static_cast<size_t>(s) * a.H + hh) * a.T * dh;
    const float* q = a.q + static_cast<size_t>(row) * a.ldq + hh * dh;
    float qv[DH];
#pragma unroll
    for (int d = 0; d < DH; ++d) qv[d] = q[d];
    float mx = -INFINITY;
    for (int key = lane; key < nk; key += kWave) {
      const AT* kr = Kc + base + static_cast<size_t>(key) * dh;
      float acc = 0.f;
#pragma unroll
      for (int d = 0; d < DH; d += Vec16<AT>::N) {
        float kv[Vec16<AT>::N];
        Vec16<AT>::load(kr, d, kv);
#pragma unroll
        for (int e = 0; e < Vec16<AT>::N; ++e) acc = fmaf(qv[d + e], kv[e], acc);
      }
      const float sc = acc * a.scale;
      s_p[wave][key] = sc;
      mx = fmaxf(mx, sc);
    }
    mx = wave_max(mx);
    float sum = 0.f;
    for (int key = lane; key < nk; key += kWave) {
      const float e = expf(s_p[wave][key] - mx);
      s_p[wave][key] = e;
      sum += e;
    }
    denom = wave_sum(sum);
  }
  __syncthreads();
  if (active) {
    for (int d = lane; d < dh; d += kWave) {
      float o = 0.f;
      for (int key = 0; key < nk; ++key)
        o = fmaf(s_p[wave][key], Elt<AT>::load(Vc, base + static_cast<size_t>(key) * dh + d), o);
      Elt<AT>::store(static_cast<AT*>(a.out), static_cast<size_t>(row) * a.ldo + hh * dh + d, o / denom);
    }
  }
}

// ---------------------------------------------------------------------------
// Token embedding x = E[tok] * scale + PE(pos), PE the interleaved sinusoid
// (columns 2i, 2i+1 = sin, cos of pos * 10000^(-2i/d)), evaluated in double.
template <typename WT>
__device__ __forceinline__ float embed_elem(const WT* emb, int tok, int p, int c, int d, float scale, int vocab) {
  tok = min(max(tok, 0), vocab - 1);
  const double freq = exp(-log(10000.0) * static_cast<double>(c & ~1) / d);
  const double ang = static_cast<double>(p) * freq;
  const float pe = static_cast<float>((c & 1) ? cos(ang) : sin(ang));
  return Elt<WT>::load(emb, static_cast<size_t>(tok) * d + c) * scale + pe;
}

template <typename WT>
__global__ __launch_bounds__(256) void k_embed(EmbedArgs a) {
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const size_t total = static_cast<size_t>(R) * a.d;
  for (size_t t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int row = static_cast<int>(t / a.d);
    const int c = static_cast<int>(t - static_cast<size_t>(row) * a.d);
    int s, p;
    row_place(a.rows, row, s, p);
    Elt<WT>::store(static_cast<WT*>(a.out), t,
                   embed_elem<WT>(static_cast<const WT*>(a.emb), a.tok[row], p, c, a.d, a.scale, a.vocab));
  }
}

// ---------------------------------------------------------------------------
// Row LayerNorm, 4 rows per wave with 16 lanes per row, statistics by
// ln_stats_g16 (the same lane split and pairing as the LayerNorm prologue of
// the matrix products).
template <typename WT, typename XT, int NT>
__global__ __launch_bounds__(256) void k_ln(LnArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15;
  const int row = (blockIdx.x * 4 + wave) * 4 + (lane >> 4);
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const bool ok = row < R;
  const XT* x = static_cast<const XT*>(a.x) + static_cast<size_t>(ok ? row : 0) * a.d;
  float v[8][8], mean, rstd;
  ln_stats_g16<XT, NT>(x, a.d, j, a.eps, ok, v, mean, rstd);
  if (!ok) return;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int k0 = 8 * j + 128 * t;
    if (k0 < a.d) {
      float g[8], b[8];
      load_n<WT, 8>(static_cast<const WT*>(a.g), k0, g);
      load_n<WT, 8>(static_cast<const WT*>(a.b), k0, b);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        Elt<WT>::store(static_cast<WT*>(a.out), static_cast<size_t>(row) * a.d + k0 + e,
                       ln_apply(v[t][e], mean, rstd, g[e], b[e]));
    }
  }
}

// ---------------------------------------------------------------------------
// On-device control of the fixed-point iteration.
//
// Every mode is a sequence of blocks [i, i+L) solved by Jacobi iterations:
//   ar        : L = 1 (greedy decoding, Eq. (1)), stops after [EOS]
//   jacobi    : one block, L = m (Algorithm 1)
//   gs_jacobi : L = min(b, m - i) (Algorithm 2)
//   hybrid    : L = min(b, h - i) while i < h, then 1 (Algorithm 3), stops at
//               the first [EOS] of a converged block
// After an iteration the block is converged when it is unchanged (StopC,
// Eq. (3)) or after L iterations (then it is exact by the triangular
// structure); a converged block is committed and the next one starts.  The
// next iteration's rows carry the shifted-left inputs: position p reads [BOS]
// for p = 0 and y[p-1] otherwise.
enum { MODE_AR = 0, MODE_JACOBI = 1, MODE_GS_JACOBI = 2, MODE_HYBRID = 3 };
enum { FLAG_CONVERGED = 1, FLAG_EOS = 2, FLAG_MAX_ITERS = 4, FLAG_NONFINITE = 8 };

__device__ __forceinline__ int block_len(const CtrlArgs& a, int i, int m) {
  switch (a.mode) {
    case MODE_AR: return 1;
    case MODE_JACOBI: return m - i;
    case MODE_GS_JACOBI: return min(a.block, m - i);
    default: {
      const int h = min(a.horizon > 0 ? a.horizon : m, m);
      return i < h ? min(a.block, h - i) : 1;
    }
  }
}

// Lay out the rows of the next iteration (sentence order, block order),
// publish the row count and, when the control step owns the embedding,
// write the embedded rows.  Single workgroup.
template <typename WT>
__device__ void emit_rows(const CtrlArgs& a) {
  __shared__ int s_total;
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int s = 0; s < a.B; ++s) {
      a.st[s].row0 = acc;
      acc += a.st[s].done ? 0 : a.st[s].L;
    }
    s_total = acc;
  }
  __syncthreads();
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    const SentState st = a.st[s];
    if (st.done) continue;
    const int* y = a.y + static_cast<size_t>(s) * a.ldy;
    for (int r = 0; r < st.L; ++r) {
      const int row = st.row0 + r;
      const int p = st.i + r;
      a.row_sent[row] = s;
      a.row_pos[row] = p;
      a.row_tok[row] = p == 0 ? a.bos_id : y[p - 1];
    }
  }
  const int total = s_total;
  if (threadIdx.x == 0) {
    *a.n_rows = total;
    if (a.host_done != nullptr)
      __hip_atomic_store(a.host_done, total == 0 ? 1 : 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (a.x_out != nullptr) {
    __syncthreads();
    const size_t n = static_cast<size_t>(total) * a.d;
    for (size_t t = threadIdx.x; t < n; t += blockDim.x) {
      const int row = static_cast<int>(t / a.d);
      const int c = static_cast<int>(t - static_cast<size_t>(row) * a.d);
      Elt<WT>::store(static_cast<WT*>(a.x_out), t,
                     embed_elem<WT>(static_cast<const WT*>(a.emb), a.row_tok[row], a.row_pos[row], c, a.d,
                                    a.emb_scale, a.vocab));
    }
  }
}

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_init(CtrlArgs a) {
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    const int m = a.tgt_m[s];
    SentState st;
    st.m = m;
    st.i = 0;
    st.j = 0;
    st.k = 0;
    st.flags = 0;
    st.done = m <= 0;
    st.L = st.done ? 0 : block_len(a, 0, m);
    st.row0 = 0;
    a.st[s] = st;
    int* y = a.y + static_cast<size_t>(s) * a.ldy;
    for (int t = 0; t < a.ldy; ++t) y[t] = a.pad_id;      // InitT: all [PAD]
  }
  __syncthreads();
  emit_rows<WT>(a);
}

// Argmax of each row over the per-workgroup partials of the fused vocabulary
// kernel (largest logit, lowest index on exact ties), one wave per row.
__device__ __forceinline__ void reduce_row(const uint2* p, int n_parts, int lane, int* tok, int* flag) {
  uint32_t bk = 0;
  uint32_t bi = 0x7fffffffu;
  uint32_t nf = 0;
  for (int t = lane; t < n_parts; t += kWave) {
    const uint2 v = p[t];
    const uint32_t i = v.y & 0x7fffffffu;
    nf |= v.y >> 31;
    if (v.x > bk || (v.x == bk && i < bi)) { bk = v.x; bi = i; }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t ok = __shfl_xor(bk, off);
    const uint32_t oi = __shfl_xor(bi, off);
    nf |= __shfl_xor(nf, off);
    if (ok > bk || (ok == bk && oi < bi)) { bk = ok; bi = oi; }
  }
  if (lane == 0) {
    const bool none = bk == 0;           // no finite logit in the row
    *tok = none ? 0 : static_cast<int>(bi);
    *flag = (nf || none) ? 1 : 0;
  }
}

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_step(CtrlArgs a) {
  const int R = *a.n_rows;
  if (R == 0) return;
  if (a.partials != nullptr) {
    const int lane = threadIdx.x & (kWave - 1);
    for (int row = threadIdx.x / kWave; row < R; row += blockDim.x / kWave)
      reduce_row(a.partials + static_cast<size_t>(row) * a.part_ld, a.n_parts, lane,
                 const_cast<int*>(a.new_tok) + row, const_cast<int*>(a.row_flags) + row);
    __syncthreads();
  }
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    SentState st = a.st[s];
    if (st.done) continue;
    int* y = a.y + static_cast<size_t>(s) * a.ldy;
    bool changed = false;
    int nf = 0;
    for (int r = 0; r < st.L; ++r) {
      const int t = a.new_tok[st.row0 + r];
      nf |= a.row_flags[st.row0 + r];
      if (y[st.i + r] != t) changed = true;
      y[st.i + r] = t;
    }
    if (nf) st.flags |= FLAG_NONFINITE;
    st.k += 1;
    st.j += 1;
    const bool converged = !changed || st.j >= st.L;
    if (converged) {
      if (a.mode == MODE_AR || a.mode == MODE_HYBRID) {
        for (int r = 0; r < st.L; ++r)
          if (y[st.i + r] == a.eos_id) { st.done = 1; st.flags |= FLAG_CONVERGED | FLAG_EOS; break; }
      }
      if (!st.done) {
        st.i += st.L;
        st.j = 0;
        if (st.i >= st.m) { st.done = 1; st.flags |= FLAG_CONVERGED; }
        else st.L = block_len(a, st.i, st.m);
      }
    }
    const int cap = a.max_iters > 0 ? a.max_iters : st.m;
    if (!st.done && st.k >= cap) { st.done = 1; st.flags |= FLAG_MAX_ITERS; }
    if (st.done) st.L = 0;
    a.st[s] = st;
  }
  __syncthreads();
  emit_rows<WT>(a);
}

// Outputs: ids cut after the first [EOS] (inclusive) and [PAD]-filled, the
// output length, the iteration count k and the flags of each sentence.
__global__ __launch_bounds__(256) void k_finalize(CtrlArgs a) {
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    const SentState st = a.st[s];
    const int* y = a.y + static_cast<size_t>(s) * a.ldy;
    int len = st.m;
    for (int t = 0; t < st.m; ++t)
      if (y[t] == a.eos_id) { len = t + 1; break; }
    for (int t = 0; t < a.out_ld; ++t)
      a.out_ids[static_cast<size_t>(s) * a.out_ld + t] = (t < len && t < a.ldy) ? y[t] : a.pad_id;
    a.out_len[s] = len;
    a.out_k[s] = st.k;
    a.out_flags[s] = st.flags;
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_argmax_reduce(ReduceArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + threadIdx.x / kWave;
  if (row >= *a.n_rows_dev) return;
  reduce_row(a.partials + static_cast<size_t>(row) * a.part_ld, a.n_parts, lane, a.new_tok + row, a.row_flags + row);
}

template <typename AT>
static hipError_t launch_attn_t(const AttnArgs& a, int grid, hipStream_t s) {
  switch (a.dh) {
    case 16: hipLaunchKernelGGL((k_attn<AT, 16>), dim3(grid), dim3(256), 0, s, a); break;
    case 32: hipLaunchKernelGGL((k_attn<AT, 32>), dim3(grid), dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((k_attn<AT, 64>), dim3(grid), dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn<AT, 128>), dim3(grid), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn(int dtype, const AttnArgs& a, int R_max, hipStream_t s) {
  if (a.dh > kMaxHeadDim || a.T > kMaxKeys) return hipErrorInvalidValue;
  const int grid = (R_max * a.H + 3) / 4;
  if (grid == 0) return hipSuccess;
  return dtype == DT_BF16 ? launch_attn_t<bf16_t>(a, grid, s) : launch_attn_t<float>(a, grid, s);
}

hipError_t launch_embed(int dtype, const EmbedArgs& a, int R_max, hipStream_t s) {
  const size_t total = static_cast<size_t>(R_max) * a.d;
  const int grid = static_cast<int>(std::min<size_t>((total + 255) / 256, 4096));
  if (grid == 0) return hipSuccess;
  if (dtype == DT_BF16) hipLaunchKernelGGL((k_embed<bf16_t>), dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((k_embed<float>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ln(int dtype, const LnArgs& a, int R_max, hipStream_t s) {
  const int grid = (R_max + 15) / 16;
  if (grid == 0) return hipSuccess;
  if (a.d % 8 != 0 || a.d > 1024) return hipErrorInvalidValue;
  if (dtype == DT_BF16) {
    if (a.d > 512) {
      if (a.x_f32) hipLaunchKernelGGL((k_ln<bf16_t, float, 8>), dim3(grid), dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_ln<bf16_t, bf16_t, 8>), dim3(grid), dim3(256), 0, s, a);
    } else {
      if (a.x_f32) hipLaunchKernelGGL((k_ln<bf16_t, float, 4>), dim3(grid), dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_ln<bf16_t, bf16_t, 4>), dim3(grid), dim3(256), 0, s, a);
    }
  } else {
    if (a.d > 512) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_ln<float, float, 4>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_argmax_reduce(const ReduceArgs& a, int R_max, hipStream_t s) {
  if (R_max <= 0) return hipSuccess;
  const int grid = (R_max + 3) / 4;
  hipLaunchKernelGGL(k_argmax_reduce, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ctrl_init(int dtype, const CtrlArgs& a, hipStream_t s) {
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_init<bf16_t>, dim3(1), dim3(1024), 0, s, a);
  else hipLaunchKernelGGL(k_ctrl_init<float>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ctrl_step(int dtype, const CtrlArgs& a, hipStream_t s) {
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_step<bf16_t>, dim3(1), dim3(1024), 0, s, a);
  else hipLaunchKernelGGL(k_ctrl_step<float>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_finalize(const CtrlArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pdec

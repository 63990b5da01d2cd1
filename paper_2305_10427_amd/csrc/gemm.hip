// Matrix products of the decoder/encoder of p_theta on the MFMA units.
//
// Y[r][n] = sum_k X[r][k] * W[n][k] (+ epilogue), W stored [N][K] row-major.
// A workgroup of 4 waves computes 16 rows x 16 columns (KSPLIT = 4: the waves
// split K and their partial tiles are summed in wave order) or 16 rows x 64
// columns (KSPLIT = 1: each wave owns 16 columns and the whole K).  One MFMA
// step multiplies a 16 x KS slice of X with a KS x 16 slice of W^T:
//   bf16: v_mfma_f32_16x16x32_bf16, KS = 32, a lane feeds 8 consecutive k;
//   f32 : 4 x v_mfma_f32_16x16x4_f32, KS = 16, a lane feeds 4 consecutive k,
//         one per instruction.
// Lane l feeds row / column (l & 15) at k = k0 + EPL * (l >> 4) + e, the same
// assignment for X and W, and reads 16 contiguous bytes of each.  The result
// tile holds C[4 * (l >> 4) + i][l & 15] in element i of lane l.
//
// Decoding at batch 1 has 1..16 rows per iteration: one 16-row tile, so a
// block of L rows costs what one row costs and the bound is streaming W.
// Each output element is accumulated over k in a fixed order (MFMA steps in
// increasing k, then the KSPLIT partials in wave order), independent of how
// many rows the call has and of the tile slot a row occupies: a row's result
// is bitwise the same in a block of L rows and alone, so greedy decoding and
// the Jacobi iterations evaluate exactly the same map.
//
// All loads a wave needs (weights, inputs, bias) are issued before any
// result is needed; the device row count only gates the stores, so its load
// overlaps the rest.  Rows between the device count and the launch bound are
// computed from stale activations and discarded.
//
// Prologue PRO_LN normalises the input rows (LayerNorm, statistics from
// ln_stats16) and rounds them to the storage type before use; workgroup 0
// can write the normalised rows out as the new residual stream.
//
// Epilogue EPI_ARGMAX is the fused vocabulary projection + argmax: logits =
// s * acc + bias are never stored; each workgroup keeps the best (largest
// value, then lowest index) per row and writes one partial per row.
#include <hip/hip_ext.h>

#include "common.h"
#include "kernels.h"
#include "mma.h"

namespace pdec {

constexpr int kDepth = 8;   // MFMA steps per weight batch; two batches are in flight

template <typename WT, int PRO, int EPI, int XF32, int KSPLIT, int LNT>
__global__ __launch_bounds__(KSPLIT == 8 ? 512 : 256) void k_gemm(GemmArgs a) {
  if constexpr (EPI == EPI_QKV) layer_select(a, blockIdx.z);
  using AT = WT;
  using XT = typename std::conditional<XF32 != 0, float, AT>::type;
  using MM = Mma<WT>;
  using frag = typename MM::frag;
  constexpr int KS = MM::KS;
  constexpr int EPL = MM::EPL;
  constexpr int D = kDepth;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int lr = lane & 15;          // row (X) / column (W) fed by this lane
  const int lg = lane >> 4;          // k group of this lane
  const int K = a.K, N = a.N;
  constexpr bool SPLIT = KSPLIT > 1;   // waves split K over one 16-column tile
  const int n0 = (SPLIT ? blockIdx.x * 16 : (blockIdx.x * 4 + wave) * 16);
  const int col = n0 + lr;           // weight row loaded by this lane, and output column it finishes
  const int n_steps = K / KS;
  const int s_begin = SPLIT ? (n_steps * wave) / KSPLIT : 0;
  const int s_end = SPLIT ? (n_steps * (wave + 1)) / KSPLIT : n_steps;
  const WT* __restrict__ W = static_cast<const WT*>(a.w);
  const XT* __restrict__ X = static_cast<const XT*>(a.x);
  const WT* __restrict__ wrow = W + static_cast<size_t>(col < N ? col : 0) * K + EPL * lg;
  const int R_max = a.n_rows;        // rows that may be read (launch bound)
  const int m_first = blockIdx.y * 16 * a.mt_per_wg;
  const int m_last = min(R_max, m_first + 16 * a.mt_per_wg);

  // Loads complete in issue order, so the small loads the prologue and the
  // epilogue need go out before the weight stream: PRO_LN's input rows of the
  // first tile and gamma / beta (staged through LDS, one 16-byte word per
  // thread of the first 256), the bias, the residual of the first tile.
  // Every load is unconditional (clamped to a valid address, unused values
  // dropped later): a load under a branch makes the compiler wait for all
  // earlier loads where the paths join.
  LnTile<WT, XT, LNT / 4> ln;   // LNT: 128-element slabs of a 16-lane row group; 4 per 512
  __shared__ uint4 s_gb[PRO == PRO_LN ? 2 : 1][128];
  uint4 gb = make_uint4(0u, 0u, 0u, 0u);
  const int gw = threadIdx.x & 127;
  if constexpr (PRO == PRO_LN) {
    ln.load(X, a.ldx, K, m_first, R_max, wave & 3, lane);
    const bool gb_word = gw < K * static_cast<int>(sizeof(WT)) / 16;
    gb = static_cast<const uint4*>((threadIdx.x & 128) ? a.ln_b : a.ln_g)[gb_word ? gw : 0];
  }
  const float bias_v = Elt<WT>::load(static_cast<const WT*>(a.bias), col < N ? col : 0);
  constexpr int NE = SPLIT ? 1 : 4;       // output elements finished per lane
  const bool epi_wave = !SPLIT || wave < 4;   // waves that finish outputs
  float rpre[NE];
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int row = m_first + 4 * lg + (SPLIT ? (wave & 3) : e);
      const size_t ri = static_cast<size_t>(row < R_max ? row : 0) * a.ldr + (col < N ? col : 0);
      rpre[e] = Elt<AT>::load(static_cast<const AT*>(a.resid), ri);
    }
  }
  int rs[NE], rp[NE];                     // EPI_QKV: (sentence, position) of the first tile's rows
  if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int row = m_first + 4 * lg + (SPLIT ? (wave & 3) : e);
      row_place(a.rows, row < R_max ? row : 0, rs[e], rp[e]);
    }
  }
  __builtin_amdgcn_sched_barrier(0);   // keep the loads above ahead of the weights

  // the first weight batch
  frag bcur[D];
#pragma unroll
  for (int u = 0; u < D; ++u) bcur[u] = MM::load(wrow + min(s_begin + u, n_steps - 1) * KS);
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;

  __shared__ float s_part[KSPLIT > 1 ? KSPLIT : 1][4][64];
  __shared__ uint32_t s_key[4][16];
  __shared__ int s_idx[4][16];
  __shared__ float2 s_lse[EPI == EPI_ARGMAX ? 4 : 1][16];
  // PRO_LN: the normalised 16-row input tile, rows padded by 16 bytes
  extern __shared__ __align__(16) unsigned char s_dyn[];
  AT* sA = reinterpret_cast<AT*>(s_dyn);
  const int lda = K + 16 / static_cast<int>(sizeof(AT));
  if constexpr (PRO == PRO_LN) {
    s_gb[(threadIdx.x >> 7) & 1][gw] = gb;   // words past the rows are never read
    __syncthreads();
  }

  for (int m0 = m_first; m0 < m_last; m0 += 16) {
    if (m0 > m_first && m0 >= R) break;
    const int arow = m0 + lr;                 // X row fed by this lane
    const bool arow_ok = arow < R_max;
    if (m0 != m_first) {
      if constexpr (PRO == PRO_LN) ln.load(X, a.ldx, K, m0, R_max, wave & 3, lane);
#pragma unroll
      for (int u = 0; u < D; ++u) bcur[u] = MM::load(wrow + min(s_begin + u, n_steps - 1) * KS);
    }
    if constexpr (PRO == PRO_LN) {
      if (wave < 4)
        ln.finish(K, a.ln_eps, reinterpret_cast<const WT*>(s_gb[0]), reinterpret_cast<const WT*>(s_gb[1]), sA, lda,
                  blockIdx.x == 0 ? static_cast<AT*>(a.ln_out) : nullptr, a.ldlo, R);
      __syncthreads();
    }
    floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = s_begin; s0 < s_end; s0 += D) {
      // next weight batch goes out before this batch's products
      frag bnext[D];
      const bool more = s0 + D < s_end;
      if (more) {
#pragma unroll
        for (int u = 0; u < D; ++u) bnext[u] = MM::load(wrow + min(s0 + D + u, n_steps - 1) * KS);
      }
      frag af[D];
#pragma unroll
      for (int u = 0; u < D; ++u) {
        const int k = min(s0 + u, n_steps - 1) * KS + EPL * lg;
        if constexpr (PRO == PRO_LN) {
          af[u] = MM::load(sA + static_cast<size_t>(lr) * lda + k);
        } else if constexpr (std::is_same<XT, AT>::value) {
          af[u] = MM::load(X + static_cast<size_t>(arow_ok ? arow : 0) * a.ldx + k);
        } else {
          float xv[EPL];
          load_n<XT, EPL>(X, static_cast<size_t>(arow_ok ? arow : 0) * a.ldx + k, xv);
          af[u] = MM::pack(xv);
        }
      }
      __builtin_amdgcn_sched_barrier(0);   // all loads of the batch before its products
      // only the steps of the wave's K range (a wave-uniform branch)
#pragma unroll
      for (int u = 0; u < D; ++u)
        if (s0 + u < s_end) acc = MM::step(af[u], bcur[u], acc);
      if (more) {
#pragma unroll
        for (int u = 0; u < D; ++u) bcur[u] = bnext[u];
      }
    }
    if constexpr (PRO == PRO_LN) __syncthreads();   // sA is rewritten by the next tile
    // combine the K-split partials: wave w finishes element i = w of every lane
    float cv[4];
    if constexpr (SPLIT) {
#pragma unroll
      for (int i = 0; i < 4; ++i) s_part[wave][i][lane] = acc[i];
      __syncthreads();
      cv[0] = 0.f;
      if (epi_wave) {
        cv[0] = s_part[0][wave][lane];
#pragma unroll
        for (int w = 1; w < KSPLIT; ++w) cv[0] += s_part[w][wave][lane];   // wave order
      }
      __syncthreads();
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) cv[i] = acc[i];
    }
    uint32_t bk[4] = {0u, 0u, 0u, 0u};
    uint32_t bi[4] = {0x7fffffffu, 0x7fffffffu, 0x7fffffffu, 0x7fffffffu};
    uint32_t nf = 0;
    float lm[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, ls[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int i = SPLIT ? wave : e;
      const int row = m0 + 4 * lg + i;
      const float v = cv[e];
      if (!epi_wave || row >= R || col >= N) continue;
      if constexpr (EPI == EPI_F32) {
        a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v + bias_v;
      } else if constexpr (EPI == EPI_ACT) {
        float t = v + bias_v;
        t = (a.act == 2) ? gelu_erf(t) : relu(t);
        Elt<AT>::store(static_cast<AT*>(a.out), static_cast<size_t>(row) * a.ldo + col, t);
      } else if constexpr (EPI == EPI_RESID) {
        const size_t ri = static_cast<size_t>(row) * a.ldr + col;
        const float rv = m0 == m_first ? rpre[e] : Elt<AT>::load(static_cast<const AT*>(a.resid), ri);
        const float t = (v + bias_v) + rv;
        if (a.out_f32 != nullptr) a.out_f32[static_cast<size_t>(row) * a.ldo + col] = t;
        else Elt<AT>::store(static_cast<AT*>(a.out), static_cast<size_t>(row) * a.ldo + col, t);
      } else if constexpr (EPI == EPI_QKV) {
        const float t = v + bias_v;
        if (col < a.q_cols) {
          a.out_f32[static_cast<size_t>(row) * a.ldo + col] = t;
        } else {
          const int c = col - a.q_cols;
          const int which = c / a.d;
          const int cc = c - which * a.d;
          const int hh = cc / a.dh;
          const int dd = cc - hh * a.dh;
          int s = rs[e], p = rp[e];
          if (m0 != m_first) row_place(a.rows, row, s, p);
          const size_t idx = ((static_cast<size_t>(s) * a.H + hh) * a.T + p) * a.dh + dd;
          Elt<AT>::store(static_cast<AT*>(which == 0 ? a.kc : a.vc), idx, t);
        }
      } else if constexpr (EPI == EPI_LOGITS) {
        a.out_f32[static_cast<size_t>(row) * a.ldo + col] = fmaf(a.logit_scale, v, bias_v);
      } else if constexpr (EPI == EPI_ARGMAX) {
        const float logit = fmaf(a.logit_scale, v, bias_v);   // s * (h . E[col]) + bias[col]
        if (!isfinite(logit)) nf |= 1u << e;   // bit e: a non-finite logit in row 4 lg + e
        else {
          bk[e] = float_key(logit);
          bi[e] = static_cast<uint32_t>(col);
          lm[e] = logit;
          ls[e] = 1.f;
        }
      }
    }
    if constexpr (EPI == EPI_ARGMAX) {
      static_assert(KSPLIT == 1, "the fused argmax runs with whole-K waves");
      // best of each row over the 16 columns held by one 16-lane group
#pragma unroll
      for (int e = 0; e < 4; ++e) group16_best(bk[e], bi[e]);
      nf = group16_or(nf);
      const bool want_lse = a.part_lse != nullptr;
      if (want_lse) {
#pragma unroll
        for (int e = 0; e < 4; ++e) group16_lse(lm[e], ls[e]);
      }
      if (lr == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s_key[wave][4 * lg + e] = bk[e];
          s_idx[wave][4 * lg + e] = static_cast<int>(bi[e] | (((nf >> e) & 1u) << 31));
          if (want_lse) s_lse[wave][4 * lg + e] = make_float2(lm[e], ls[e]);
        }
      }
      __syncthreads();
      if (threadIdx.x < 16) {
        const int r = threadIdx.x;
        uint32_t kk = 0;
        int ii = 0x7fffffff, ff = 0;
        for (int w = 0; w < 4; ++w) {
          const uint32_t k2 = s_key[w][r];
          const int raw = s_idx[w][r];
          const int i2 = raw & 0x7fffffff;
          ff |= (raw >> 31) & 1;
          if (k2 > kk || (k2 == kk && i2 < ii)) { kk = k2; ii = i2; }
        }
        if (m0 + r < R) {
          a.partials[static_cast<size_t>(m0 + r) * a.part_ld + blockIdx.x] =
              make_uint2(kk, static_cast<uint32_t>(ii) | (static_cast<uint32_t>(ff) << 31));
          if (want_lse) {
            float m = s_lse[0][r].x, sm = s_lse[0][r].y;
            for (int w = 1; w < 4; ++w) lse_merge(m, sm, s_lse[w][r].x, s_lse[w][r].y);   // wave order
            a.part_lse[static_cast<size_t>(m0 + r) * a.part_ld + blockIdx.x] = make_float2(m, sm);
          }
        }
      }
      __syncthreads();
    }
  }
}

namespace {

// Launch, through hipExtLaunchKernelGGL when a pair of events is given (the
// events then carry the dispatch's own start and end timestamps).
template <typename K>
void launch_ev(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
               const GemmArgs& a) {
  if (ev0 != nullptr) hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(lds), s, ev0, ev1, 0u, a);
  else hipLaunchKernelGGL(kernel, grid, block, lds, s, a);
}

template <typename WT, int PRO, int EPI, int XF32, int LNT>
hipError_t launch_k(GemmArgs a, int ksplit, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int tiles = (a.n_rows + 15) / 16;
  const int gy = tiles < 64 ? tiles : 64;
  a.mt_per_wg = (tiles + gy - 1) / gy;
  const size_t lds = PRO == PRO_LN ? gemm_ln_lds_bytes(a.K, sizeof(WT)) : 0;
  const int gz = EPI == EPI_QKV && a.n_layers > 1 ? a.n_layers : 1;
  if (EPI == EPI_ARGMAX || ksplit == 1) {
    launch_ev(k_gemm<WT, PRO, EPI, XF32, 1, LNT>, dim3(gemm_grid(EPI, a.N, 1), gy, gz), dim3(256), lds, s, ev0, ev1,
              a);
  } else if constexpr (EPI != EPI_ARGMAX) {
    if (ksplit == 8)
      launch_ev(k_gemm<WT, PRO, EPI, XF32, 8, LNT>, dim3(gemm_grid(EPI, a.N, 8), gy, gz), dim3(512), lds, s, ev0,
                ev1, a);
    else
      launch_ev(k_gemm<WT, PRO, EPI, XF32, 4, LNT>, dim3(gemm_grid(EPI, a.N, 4), gy, gz), dim3(256), lds, s, ev0,
                ev1, a);
  }
  return hipGetLastError();
}

// LayerNorm chunks of 128 elements held per lane: 4 covers d <= 512, 8 covers d <= 1024
template <typename WT, int PRO, int EPI, int XF32>
hipError_t launch_t(const GemmArgs& a, int ksplit, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if constexpr (PRO == PRO_LN && std::is_same<WT, bf16_t>::value) {
    if (a.K > 512) return launch_k<WT, PRO, EPI, XF32, 8>(a, ksplit, s, ev0, ev1);
  }
  return launch_k<WT, PRO, EPI, XF32, 4>(a, ksplit, s, ev0, ev1);
}

template <typename WT, int PRO, int XF32>
hipError_t launch_epi(int epi, const GemmArgs& a, int ksplit, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  switch (epi) {
    case EPI_F32: return launch_t<WT, PRO, EPI_F32, XF32>(a, ksplit, s, ev0, ev1);
    case EPI_ACT: return launch_t<WT, PRO, EPI_ACT, XF32>(a, ksplit, s, ev0, ev1);
    case EPI_RESID: return launch_t<WT, PRO, EPI_RESID, XF32>(a, ksplit, s, ev0, ev1);
    case EPI_QKV: return launch_t<WT, PRO, EPI_QKV, XF32>(a, ksplit, s, ev0, ev1);
    case EPI_ARGMAX: return launch_t<WT, PRO, EPI_ARGMAX, XF32>(a, ksplit, s, ev0, ev1);
    case EPI_LOGITS: return launch_t<WT, PRO, EPI_LOGITS, XF32>(a, ksplit, s, ev0, ev1);
    default: return hipErrorInvalidValue;
  }
}

template <typename WT>
hipError_t launch_dt(int pro, int epi, const GemmArgs& a, int ksplit, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (pro == PRO_LN)
    return a.x_f32 ? launch_epi<WT, PRO_LN, 1>(epi, a, ksplit, s, ev0, ev1)
                   : launch_epi<WT, PRO_LN, 0>(epi, a, ksplit, s, ev0, ev1);
  if (a.x_f32) return hipErrorInvalidValue;
  return launch_epi<WT, PRO_NONE, 0>(epi, a, ksplit, s, ev0, ev1);
}

}  // namespace

size_t gemm_ln_lds_bytes(int K, size_t elt) { return 16 * (static_cast<size_t>(K) * elt + 16); }

int gemm_grid(int epi, int N, int ksplit) {
  if (epi == EPI_ARGMAX || ksplit == 1) return (N + 63) / 64;
  return (N + 15) / 16;
}

hipError_t launch_gemm(int dtype, int pro, int epi, int ksplit, const GemmArgs& a, hipStream_t s, hipEvent_t ev0,
                       hipEvent_t ev1) {
  if (a.n_rows <= 0) return hipSuccess;
  const int ks = dtype == DT_BF16 ? Mma<bf16_t>::KS : Mma<float>::KS;
  if (a.K % ks != 0 || a.K % 32 != 0) return hipErrorInvalidValue;
  if (pro == PRO_LN && (a.K > (dtype == DT_BF16 ? 1024 : 512) || gemm_ln_lds_bytes(a.K, dtype == DT_BF16 ? 2 : 4) > 65536))
    return hipErrorInvalidValue;
  if (dtype == DT_BF16) return launch_dt<bf16_t>(pro, epi, a, ksplit, s, ev0, ev1);
  return launch_dt<float>(pro, epi, a, ksplit, s, ev0, ev1);
}

}  // namespace pdec

// Weight-streaming matrix products for the decoder/encoder of p_theta.
//
// Y[r][n] = sum_k X[r][k] * W[n][k] (+ epilogue), W stored [N][K] row-major.
// The decoder rows of one iteration are few (batch x block), so the product
// is bound by reading W once: every wave streams whole 16-byte vectors of NC
// weight rows across its 64 lanes (coalesced along K), multiplies them with
// RT input rows held in registers and reduces across lanes at the end.
//
// Reduction order per output element is fixed: each lane accumulates its K
// slice in increasing k with FMAs, then a fixed lane-pairing tree sums the 64
// lane partials.  It does not depend on how many rows the call has or on which
// slot of a row tile a row lands in, so a row's result is bitwise the same in
// a block of L rows and alone (greedy decoding and the Jacobi iterations then
// evaluate exactly the same map).
//
// Prologue PRO_LN normalises each input row (LayerNorm with the lane split of
// ln_stats below) before use and rounds it to the storage type; workgroup 0
// can write the normalised rows out as the new residual stream.
//
// Epilogue EPI_ARGMAX turns the product into the fused vocabulary projection
// + argmax: logits = s * acc + bias are never stored, each workgroup keeps the
// best (value, lowest index) per row and writes one partial per row.
#include "common.h"
#include "kernels.h"

namespace pdec {

constexpr int kNC = 4;        // weight rows (output columns) per wave per pass
constexpr int kWavesPerWG = 4;

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

template <typename WT, typename AT, int RT, int PRO, int EPI, int XF32>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  using XT = typename std::conditional<XF32 != 0, float, AT>::type;
  constexpr int EPL = Vec16<WT>::N;
  constexpr int M = kNC * RT;
  constexpr int LGM = Log2<M>::v;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  if (R <= 0) return;
  const int K = a.K, N = a.N;
  const int n_groups = (N + kNC - 1) / kNC;
  const int wave_gid = blockIdx.x * kWavesPerWG + wave;
  const int wave_stride = gridDim.x * kWavesPerWG;
  const WT* __restrict__ W = static_cast<const WT*>(a.w);
  const WT* __restrict__ bias = static_cast<const WT*>(a.bias);
  const XT* __restrict__ X = static_cast<const XT*>(a.x);

  __shared__ uint32_t s_key[kWavesPerWG][M];
  __shared__ int s_idx[kWavesPerWG][M];

  const int j_own = lane >> (6 - LGM);
  const bool owner = (lane & ((1 << (6 - LGM)) - 1)) == 0;
  const int n_own = j_own / RT;
  const int r_own = j_own % RT;

  for (int r0 = 0; r0 < R; r0 += RT) {
    const int nr = min(RT, R - r0);
    float mean[RT], rstd[RT];
    if constexpr (PRO == PRO_LN) {
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        mean[r] = 0.f;
        rstd[r] = 0.f;
        if (r < nr) ln_stats<WT, XT>(X + static_cast<size_t>(r0 + r) * a.ldx, K, lane, a.ln_eps, mean[r], rstd[r]);
      }
    }
    uint32_t best_key = 0;
    int best_idx = 0x7fffffff;
    int nonfinite = 0;
    bool first_pass = true;
    for (int g = wave_gid; g < n_groups; g += wave_stride) {
      float acc[kNC][RT];
#pragma unroll
      for (int n = 0; n < kNC; ++n)
#pragma unroll
        for (int r = 0; r < RT; ++r) acc[n][r] = 0.f;
      for (int k0 = lane * EPL; k0 < K; k0 += kWave * EPL) {
        float xv[RT][EPL];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          if (r < nr) {
            load_n<XT, EPL>(X, static_cast<size_t>(r0 + r) * a.ldx + k0, xv[r]);
            if constexpr (PRO == PRO_LN) {
              float gv[EPL], bv[EPL];
              load_n<WT, EPL>(static_cast<const WT*>(a.ln_g), k0, gv);
              load_n<WT, EPL>(static_cast<const WT*>(a.ln_b), k0, bv);
#pragma unroll
              for (int e = 0; e < EPL; ++e)
                xv[r][e] = Elt<AT>::round(ln_apply(xv[r][e], mean[r], rstd[r], gv[e], bv[e]));
              if (a.ln_out != nullptr && blockIdx.x == 0 && wave == 0 && first_pass) {
#pragma unroll
                for (int e = 0; e < EPL; ++e)
                  Elt<AT>::store(static_cast<AT*>(a.ln_out), static_cast<size_t>(r0 + r) * a.ldlo + k0 + e, xv[r][e]);
              }
            }
          } else {
#pragma unroll
            for (int e = 0; e < EPL; ++e) xv[r][e] = 0.f;
          }
        }
#pragma unroll
        for (int n = 0; n < kNC; ++n) {
          const int col = g * kNC + n;
          float wv[EPL];
          if (col < N) {
            load_n<WT, EPL>(W, static_cast<size_t>(col) * K + k0, wv);
          } else {
#pragma unroll
            for (int e = 0; e < EPL; ++e) wv[e] = 0.f;
          }
#pragma unroll
          for (int r = 0; r < RT; ++r)
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[n][r] = fmaf(wv[e], xv[r][e], acc[n][r]);
        }
      }
      first_pass = false;
      float vals[M];
#pragma unroll
      for (int n = 0; n < kNC; ++n)
#pragma unroll
        for (int r = 0; r < RT; ++r) vals[n * RT + r] = acc[n][r];
      float v = wave_reduce_scatter<M>(vals, lane);
      const int col = g * kNC + n_own;
      const int row = r0 + r_own;
      if (!owner || col >= N || r_own >= nr) continue;
      const float bv = Elt<WT>::load(bias, col);
      if constexpr (EPI == EPI_F32) {
        a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v + bv;
      } else if constexpr (EPI == EPI_ACT) {
        v += bv;
        v = (a.act == 2) ? gelu_erf(v) : fmaxf(v, 0.f);
        Elt<AT>::store(static_cast<AT*>(a.out), static_cast<size_t>(row) * a.ldo + col, v);
      } else if constexpr (EPI == EPI_RESID) {
        v += bv;
        const size_t ri = static_cast<size_t>(row) * a.ldr + col;
        v += a.resid_f32 ? static_cast<const float*>(a.resid)[ri] : Elt<AT>::load(static_cast<const AT*>(a.resid), ri);
        if (a.out_f32 != nullptr) a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v;
        else Elt<AT>::store(static_cast<AT*>(a.out), static_cast<size_t>(row) * a.ldo + col, v);
      } else if constexpr (EPI == EPI_QKV) {
        v += bv;
        if (col < a.q_cols) {
          a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v;
        } else {
          const int c = col - a.q_cols;
          const int which = c / a.d;
          const int cc = c - which * a.d;
          const int hh = cc / a.dh;
          const int dd = cc - hh * a.dh;
          int s, p;
          if (a.rows.sent != nullptr) { s = a.rows.sent[row]; p = a.rows.pos[row]; }
          else { s = row / a.rows.per_sent; p = row - s * a.rows.per_sent; }
          const size_t idx = ((static_cast<size_t>(s) * a.H + hh) * a.T + p) * a.dh + dd;
          Elt<AT>::store(static_cast<AT*>(which == 0 ? a.kc : a.vc), idx, v);
        }
      } else if constexpr (EPI == EPI_LOGITS) {
        a.out_f32[static_cast<size_t>(row) * a.ldo + col] = fmaf(a.logit_scale, v, bv);
      } else if constexpr (EPI == EPI_ARGMAX) {
        const float logit = fmaf(a.logit_scale, v, bv);   // s * (h . E[col]) + bias[col]
        if (!isfinite(logit)) {
          nonfinite = 1;
        } else {
          const uint32_t key = float_key(logit);
          if (key > best_key) { best_key = key; best_idx = col; }   // columns rise: first max kept
        }
      }
    }
    if constexpr (EPI == EPI_ARGMAX) {
      // workgroup-level best per row: (largest key, then lowest index)
      if (owner) {
        s_key[wave][j_own] = best_key;
        s_idx[wave][j_own] = best_idx | (nonfinite << 31);
      }
      __syncthreads();
      if (threadIdx.x < RT && static_cast<int>(threadIdx.x) < nr) {
        const int r = threadIdx.x;
        uint32_t bk = 0;
        int bi = 0x7fffffff, nf = 0;
        for (int w = 0; w < kWavesPerWG; ++w)
          for (int n = 0; n < kNC; ++n) {
            const uint32_t k = s_key[w][n * RT + r];
            const int raw = s_idx[w][n * RT + r];
            const int i = raw & 0x7fffffff;
            nf |= (raw >> 31) & 1;
            if (k > bk || (k == bk && i < bi)) { bk = k; bi = i; }
          }
        a.partials[static_cast<size_t>(r0 + r) * a.part_ld + blockIdx.x] =
            make_uint2(bk, static_cast<uint32_t>(bi) | (static_cast<uint32_t>(nf) << 31));
      }
      __syncthreads();
    }
  }
}

namespace {

template <typename WT, typename AT, int RT, int PRO, int EPI, int XF32>
hipError_t launch_t(const GemmArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((k_gemm<WT, AT, RT, PRO, EPI, XF32>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename WT, typename AT, int PRO, int EPI, int XF32>
hipError_t launch_rt(int row_tile, const GemmArgs& a, int grid, hipStream_t s) {
  switch (row_tile) {
    case 1: return launch_t<WT, AT, 1, PRO, EPI, XF32>(a, grid, s);
    case 2: return launch_t<WT, AT, 2, PRO, EPI, XF32>(a, grid, s);
    case 4: return launch_t<WT, AT, 4, PRO, EPI, XF32>(a, grid, s);
    case 8: return launch_t<WT, AT, 8, PRO, EPI, XF32>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename WT, typename AT>
hipError_t launch_dt(int pro, int epi, int row_tile, const GemmArgs& a, int grid, hipStream_t s) {
  if (pro == PRO_LN) {
    if (a.x_f32) {
      switch (epi) {
        case EPI_F32: return launch_rt<WT, AT, PRO_LN, EPI_F32, 1>(row_tile, a, grid, s);
        case EPI_ACT: return launch_rt<WT, AT, PRO_LN, EPI_ACT, 1>(row_tile, a, grid, s);
        case EPI_QKV: return launch_rt<WT, AT, PRO_LN, EPI_QKV, 1>(row_tile, a, grid, s);
        case EPI_ARGMAX: return launch_rt<WT, AT, PRO_LN, EPI_ARGMAX, 1>(row_tile, a, grid, s);
        case EPI_LOGITS: return launch_rt<WT, AT, PRO_LN, EPI_LOGITS, 1>(row_tile, a, grid, s);
        default: return hipErrorInvalidValue;
      }
    }
    switch (epi) {
      case EPI_F32: return launch_rt<WT, AT, PRO_LN, EPI_F32, 0>(row_tile, a, grid, s);
      case EPI_ACT: return launch_rt<WT, AT, PRO_LN, EPI_ACT, 0>(row_tile, a, grid, s);
      case EPI_QKV: return launch_rt<WT, AT, PRO_LN, EPI_QKV, 0>(row_tile, a, grid, s);
      case EPI_ARGMAX: return launch_rt<WT, AT, PRO_LN, EPI_ARGMAX, 0>(row_tile, a, grid, s);
      case EPI_LOGITS: return launch_rt<WT, AT, PRO_LN, EPI_LOGITS, 0>(row_tile, a, grid, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (a.x_f32) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_F32: return launch_rt<WT, AT, PRO_NONE, EPI_F32, 0>(row_tile, a, grid, s);
    case EPI_ACT: return launch_rt<WT, AT, PRO_NONE, EPI_ACT, 0>(row_tile, a, grid, s);
    case EPI_RESID: return launch_rt<WT, AT, PRO_NONE, EPI_RESID, 0>(row_tile, a, grid, s);
    case EPI_QKV: return launch_rt<WT, AT, PRO_NONE, EPI_QKV, 0>(row_tile, a, grid, s);
    case EPI_ARGMAX: return launch_rt<WT, AT, PRO_NONE, EPI_ARGMAX, 0>(row_tile, a, grid, s);
    case EPI_LOGITS: return launch_rt<WT, AT, PRO_NONE, EPI_LOGITS, 0>(row_tile, a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_gemm(int dtype, int pro, int epi, int row_tile, const GemmArgs& a, int grid, hipStream_t s) {
  if (dtype == DT_BF16) return launch_dt<bf16_t, bf16_t>(pro, epi, row_tile, a, grid, s);
  return launch_dt<float, float>(pro, epi, row_tile, a, grid, s);
}

}  // namespace pdec

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
// computed from stale activations and discarded.  When a wave's K range is
// SPW whole MFMA steps (the decoder's shapes), its SPW weight and input loads
// all go out at once; other shapes stream batches of kDepth steps, the next
// batch in flight during the current one's products.  The whole-range weight
// loads are non-temporal (each launch streams its weights once): measured
// faster than ordinary loads on the decoding iterations (large model,
// GS-Jacobi b = 16: 623 -> 585 µs per iteration together with the
// vocabulary kernel's; MT-base, whose weights fit in the last-level cache:
// hybrid b = 5 206 -> 196 µs).
//
// Weights come row-major, or (a.wp) in the order the MFMA steps consume them:
// block (tile c, step s) of 1 KB holds lane l's 16 bytes at 16 l, i.e.
// W[16 c + (l & 15)][s KS + EPL (l >> 4) ...], so each wave-wide load reads
// 1 KB contiguous instead of 64 bytes from each of 16 weight rows.
//
// Row groups (RG < 16, the K-split kernels of one row tile): a workgroup
// computes RG rows of its column tile, and the row groups of a column tile
// are consecutive workgroups of one XCD (linear id mod 8), so its weights
// come from HBM once and the other groups read them from that XCD's L2.
// This spreads a narrow product over more CUs and cuts the LayerNorm
// prologue to RG / 4 rows per wave; lanes of the tile rows past RG repeat the
// group's rows and their results are dropped.
//
// Prologue PRO_LN normalises the input rows (LayerNorm, statistics from
// ln_stats16) and rounds them to the storage type before use; workgroup 0
// can write the normalised rows out as the new residual stream.
//
// Epilogue EPI_ARGMAX is the fused vocabulary projection + argmax: logits =
// s * acc + bias are never stored; each workgroup keeps the best (largest
// value, then lowest index) per row and writes one partial per row.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "mma.h"

namespace pdec {

constexpr int kDepth = 8;   // MFMA steps per weight batch; two batches are in flight

template <typename WT, int PRO, int EPI, int XF32, int KSPLIT, int LNT, int RG, int SPW>
__global__ __launch_bounds__(KSPLIT == 8 ? 512 : 256) void k_gemm(GemmArgs a) {
  if constexpr (EPI == EPI_QKV) layer_select(a, blockIdx.z);
  using AT = WT;
  using XT = typename std::conditional<XF32 != 0, float, AT>::type;
  using MM = Mma<WT>;
  using frag = typename MM::frag;
  constexpr int KS = MM::KS;
  constexpr int EPL = MM::EPL;
  constexpr int D = SPW > 0 ? SPW : kDepth;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int lr = lane & 15;          // row (X) / column (W) fed by this lane
  const int lg = lane >> 4;          // k group of this lane
  const int K = a.K, N = a.N;
  constexpr bool SPLIT = KSPLIT > 1;   // waves split K over one 16-column tile
  static_assert(RG == 16 || (SPLIT && (RG == 4 || RG == 8)), "row groups of 4 or 8 rows need the K split");
  static_assert(SPW == 0 || SPLIT, "whole-range loads need the K split");
  int ctile = blockIdx.x, grp = 0;     // column tile and row group of this workgroup
  if constexpr (RG < 16) {
    const int ct = (N + 15) / 16;
    const int ng = gridDim.x / ct;
    if ((ct & 7) == 0) {                 // the ng groups of tile c: ids ((c / 8) ng + g) 8 + c % 8
      const int q = blockIdx.x >> 3;
      grp = q % ng;
      ctile = (q / ng) * 8 + (blockIdx.x & 7);
    } else {
      grp = blockIdx.x / ct;
      ctile = blockIdx.x - grp * ct;
    }
  }
  const int n0 = (SPLIT ? ctile * 16 : (blockIdx.x * 4 + wave) * 16);
  const int col = n0 + lr;           // weight row loaded by this lane, and output column it finishes
  const int n_steps = K / KS;
  const int s_begin = SPLIT ? (n_steps * wave) / KSPLIT : 0;
  const int s_end = SPLIT ? (n_steps * (wave + 1)) / KSPLIT : n_steps;
  const WT* __restrict__ W = static_cast<const WT*>(a.w);
  const XT* __restrict__ X = static_cast<const XT*>(a.x);
  // step s of this lane's weights sits at wrow + s * wstep
  const bool packed = a.wp != nullptr;
  const WT* __restrict__ wrow =
      packed ? static_cast<const WT*>(a.wp) + (static_cast<size_t>(n0 / 16) * n_steps * kWave + lane) * EPL
             : W + static_cast<size_t>(col < N ? col : 0) * K + EPL * lg;
  const int wstep = packed ? kWave * EPL : KS;
  const int R_max = a.n_rows;        // rows that may be read (launch bound)
  const int m_first = RG < 16 ? grp * RG : blockIdx.y * 16 * a.mt_per_wg;
  const int m_last = min(R_max, m_first + (RG < 16 ? RG : 16 * a.mt_per_wg));
  const int R_grp = RG < 16 ? m_last : R_max;   // rows this workgroup's LayerNorm reads
  const int lrr = lr & (RG - 1);                // tile row fed by this lane

  // Loads complete in issue order, so the small loads the prologue and the
  // epilogue need go out before the weight stream: PRO_LN's input rows of the
  // first tile and gamma / beta (staged through LDS, one 16-byte word per
  // thread of the first 256), the bias, the residual of the first tile.
  // Every load is unconditional (clamped to a valid address, unused values
  // dropped later): a load under a branch makes the compiler wait for all
  // earlier loads where the paths join.
  // LNT: 128-element slabs of a 16-lane row group (4 per 512); one pass per 4 rows
  LnTile<WT, XT, LNT / 4, RG < 16 ? RG / 4 : 4> ln;
  __shared__ uint4 s_gb[PRO == PRO_LN ? 2 : 1][128];
  uint4 gb = make_uint4(0u, 0u, 0u, 0u);
  const int gw = threadIdx.x & 127;
  if constexpr (PRO == PRO_LN) {
    ln.load(X, a.ldx, K, m_first, R_grp, wave & 3, lane);
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
      const int row = m_first + ((4 * lg + (SPLIT ? (wave & 3) : e)) & (RG - 1));
      const size_t ri = static_cast<size_t>(row < R_max ? row : 0) * a.ldr + (col < N ? col : 0);
      rpre[e] = Elt<AT>::load(static_cast<const AT*>(a.resid), ri);
    }
  }
  int rs[NE], rp[NE];                     // EPI_QKV: (sentence, position) of the first tile's rows
  if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int row = m_first + ((4 * lg + (SPLIT ? (wave & 3) : e)) & (RG - 1));
      row_place(a.rows, row < R_max ? row : 0, rs[e], rp[e]);
    }
  }
  __builtin_amdgcn_sched_barrier(0);   // keep the loads above ahead of the weights

  // the first weight batch
  frag bcur[D];
#pragma unroll
  for (int u = 0; u < D; ++u)
    bcur[u] = MM::template wload<SPW != 0>(wrow + static_cast<size_t>(min(s_begin + u, n_steps - 1)) * wstep);
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
    const int arow = m0 + lrr;                // X row fed by this lane
    const bool arow_ok = arow < R_max;
    if (m0 != m_first) {
      if constexpr (PRO == PRO_LN) ln.load(X, a.ldx, K, m0, R_grp, wave & 3, lane);
#pragma unroll
      for (int u = 0; u < D; ++u)
        bcur[u] = MM::template wload<SPW != 0>(wrow + static_cast<size_t>(min(s_begin + u, n_steps - 1)) * wstep);
    }
    if constexpr (PRO == PRO_LN) {
      if (wave < 4)
        ln.finish(K, a.ln_eps, reinterpret_cast<const WT*>(s_gb[0]), reinterpret_cast<const WT*>(s_gb[1]), sA, lda,
                  ctile == 0 ? static_cast<AT*>(a.ln_out) : nullptr, a.ldlo, R);
      __syncthreads();
    }
    floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
    // the input fragment of step s (LDS tile after the LayerNorm, else X)
    auto a_frag = [&](int s) {
      const int k = s * KS + EPL * lg;
      if constexpr (PRO == PRO_LN) {
        return MM::load(sA + static_cast<size_t>(lrr) * lda + k);
      } else if constexpr (std::is_same<XT, AT>::value) {
        // row-major rows, or the tile's feed-order words (one 1 KB block per step)
        const size_t off = a.x_feed ? (static_cast<size_t>(m0 >> 4) * n_steps + s) * (kWave * EPL) + lane * EPL
                                    : static_cast<size_t>(arow_ok ? arow : 0) * a.ldx + k;
        return MM::load(X + off);
      } else {
        float xv[EPL];
        load_n<XT, EPL>(X, static_cast<size_t>(arow_ok ? arow : 0) * a.ldx + k, xv);
        return MM::pack(xv);
      }
    };
    if constexpr (SPW > 0) {
      // the whole range: bcur holds its SPW weight steps
      frag af[D];
#pragma unroll
      for (int u = 0; u < D; ++u) af[u] = a_frag(s_begin + u);
#pragma unroll
      for (int u = 0; u < D; ++u) acc = MM::step(af[u], bcur[u], acc);
    } else
    for (int s0 = s_begin; s0 < s_end; s0 += D) {
      // next weight batch goes out before this batch's products
      frag bnext[D];
      const bool more = s0 + D < s_end;
      if (more) {
#pragma unroll
        for (int u = 0; u < D; ++u) bnext[u] = MM::load(wrow + static_cast<size_t>(min(s0 + D + u, n_steps - 1)) * wstep);
      }
      frag af[D];
#pragma unroll
      for (int u = 0; u < D; ++u) af[u] = a_frag(min(s0 + u, n_steps - 1));
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
      if (!epi_wave || 4 * lg + i >= RG || row >= R || col >= N) continue;
      if constexpr (EPI == EPI_F32) {
        a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v + bias_v;
      } else if constexpr (EPI == EPI_ACT) {
        float t = v + bias_v;
        t = (a.act == 2) ? gelu_erf(t) : relu(t);
        Elt<AT>::store(static_cast<AT*>(a.out),
                       a.out_feed ? feed_index<KS, EPL>(row, col, N) : static_cast<size_t>(row) * a.ldo + col, t);
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

// Rows per workgroup for a K-split product: groups of 4 rows for the
// LayerNorm-prologue products (a quarter of the prologue per wave, and more
// workgroups for a narrow product) up to 768 workgroups, groups of 8 up to
// 1024, whole 16-row tiles beyond.  Measured on the decoder's shapes (d = 512
// and 1024, 1 / 5 / 16 rows): groups did not help the products that read
// their input rows straight from memory.
int row_group(int pro, int col_tiles, int rows, int layers) {
  if (pro != PRO_LN || layers != 1) return 16;
  if (col_tiles * ((rows + 3) / 4) <= 768) return 4;
  if (col_tiles * ((rows + 7) / 8) <= 1024) return 8;
  return 16;
}

template <typename WT, int PRO, int EPI, int XF32, int LNT, int KSPLIT, int RG>
void launch_rg(const GemmArgs& a, int spw, dim3 grid, size_t lds, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  constexpr int NT = KSPLIT == 8 ? 512 : 256;
  if constexpr (KSPLIT == 8) {
    if (spw == 16) return launch_ev(k_gemm<WT, PRO, EPI, XF32, 8, LNT, RG, 16>, grid, dim3(NT), lds, s, ev0, ev1, a);
    if (spw == 8) return launch_ev(k_gemm<WT, PRO, EPI, XF32, 8, LNT, RG, 8>, grid, dim3(NT), lds, s, ev0, ev1, a);
  } else {
    if (spw == 8) return launch_ev(k_gemm<WT, PRO, EPI, XF32, 4, LNT, RG, 8>, grid, dim3(NT), lds, s, ev0, ev1, a);
    if (spw == 4) return launch_ev(k_gemm<WT, PRO, EPI, XF32, 4, LNT, RG, 4>, grid, dim3(NT), lds, s, ev0, ev1, a);
  }
  launch_ev(k_gemm<WT, PRO, EPI, XF32, KSPLIT, LNT, RG, 0>, grid, dim3(NT), lds, s, ev0, ev1, a);
}

template <typename WT, int PRO, int EPI, int XF32, int LNT, int KSPLIT>
void launch_split(const GemmArgs& a, int gy, int gz, size_t lds, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int ct = gemm_grid(EPI, a.N, KSPLIT);
  const int n_steps = a.K / Mma<WT>::KS;
  const int spw = n_steps % KSPLIT == 0 ? n_steps / KSPLIT : 0;
  const int rg = row_group(PRO, ct, a.n_rows, gz);
  if constexpr (PRO == PRO_LN) {
    if (rg == 4) return launch_rg<WT, PRO, EPI, XF32, LNT, KSPLIT, 4>(a, spw, dim3(ct * ((a.n_rows + 3) / 4)), lds, s, ev0, ev1);
    if (rg == 8) return launch_rg<WT, PRO, EPI, XF32, LNT, KSPLIT, 8>(a, spw, dim3(ct * ((a.n_rows + 7) / 8)), lds, s, ev0, ev1);
  }
  launch_rg<WT, PRO, EPI, XF32, LNT, KSPLIT, 16>(a, spw, dim3(ct, gy, gz), lds, s, ev0, ev1);
}

template <typename WT, int PRO, int EPI, int XF32, int LNT>
hipError_t launch_k(GemmArgs a, int ksplit, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int tiles = (a.n_rows + 15) / 16;
  const int gy = tiles < 64 ? tiles : 64;
  a.mt_per_wg = (tiles + gy - 1) / gy;
  const size_t lds = PRO == PRO_LN ? gemm_ln_lds_bytes(a.K, sizeof(WT)) : 0;
  const int gz = EPI == EPI_QKV && a.n_layers > 1 ? a.n_layers : 1;
  if (gz > 1 || a.N % 16 != 0) a.wp = nullptr;   // the packed copy covers single-layer products with whole tiles
  if (EPI == EPI_ARGMAX || ksplit == 1) {
    a.wp = nullptr;
    launch_ev(k_gemm<WT, PRO, EPI, XF32, 1, LNT, 16, 0>, dim3(gemm_grid(EPI, a.N, 1), gy, gz), dim3(256), lds, s, ev0,
              ev1, a);
  } else if constexpr (EPI != EPI_ARGMAX) {
    if (ksplit == 8) launch_split<WT, PRO, EPI, XF32, LNT, 8>(a, gy, gz, lds, s, ev0, ev1);
    else launch_split<WT, PRO, EPI, XF32, LNT, 4>(a, gy, gz, lds, s, ev0, ev1);
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

// W [N][K] row-major -> the MFMA feed order of k_gemm (K a multiple of the
// MFMA step): ceil(N / 16) column tiles, the rows of a ragged last tile past
// N repeating row N - 1; one 16-byte word per thread.
template <typename WT>
__global__ __launch_bounds__(256) void k_pack_feed(const WT* __restrict__ w, WT* __restrict__ out, int N, int K) {
  using MM = Mma<WT>;
  constexpr int KS = MM::KS, EPL = MM::EPL;
  const int n_steps = K / KS;
  const long long words = static_cast<long long>((N + 15) / 16) * 16 * K / EPL;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < words; i += static_cast<long long>(gridDim.x) * 256) {
    const int lane = static_cast<int>(i % kWave);
    const long long blk = i / kWave;                    // c * n_steps + s
    const int c = static_cast<int>(blk / n_steps);
    const int st = static_cast<int>(blk - static_cast<long long>(c) * n_steps);
    const int row = min(16 * c + (lane & 15), N - 1);
    const size_t src = static_cast<size_t>(row) * K + st * KS + EPL * (lane >> 4);
    *reinterpret_cast<uint4*>(out + static_cast<size_t>(i) * EPL) = *reinterpret_cast<const uint4*>(w + src);
  }
}

hipError_t launch_pack_feed(int dtype, const void* w, void* out, int N, int K, hipStream_t s) {
  const int ks = dtype == DT_BF16 ? Mma<bf16_t>::KS : Mma<float>::KS;
  if (N <= 0 || K <= 0 || K % ks != 0) return hipErrorInvalidValue;
  const long long words = static_cast<long long>((N + 15) / 16) * 16 * K / (dtype == DT_BF16 ? 8 : 4);
  const int grid = static_cast<int>(std::min<long long>((words + 255) / 256, 4096));
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(k_pack_feed<bf16_t>, dim3(grid), dim3(256), 0, s, static_cast<const bf16_t*>(w),
                       static_cast<bf16_t*>(out), N, K);
  else
    hipLaunchKernelGGL(k_pack_feed<float>, dim3(grid), dim3(256), 0, s, static_cast<const float*>(w),
                       static_cast<float*>(out), N, K);
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int pro, int epi, int ksplit, const GemmArgs& a, hipStream_t s, hipEvent_t ev0,
                       hipEvent_t ev1) {
  if (a.n_rows <= 0) return hipSuccess;
  if (a.x_feed && (pro == PRO_LN || a.x_f32 || ksplit == 1)) return hipErrorInvalidValue;
  if (a.out_feed && (epi != EPI_ACT || ksplit == 1 || a.N % 32 != 0)) return hipErrorInvalidValue;
  const int ks = dtype == DT_BF16 ? Mma<bf16_t>::KS : Mma<float>::KS;
  if (a.K % ks != 0 || a.K % 32 != 0) return hipErrorInvalidValue;
  if (pro == PRO_LN && (a.K > (dtype == DT_BF16 ? 1024 : 512) || gemm_ln_lds_bytes(a.K, dtype == DT_BF16 ? 2 : 4) > 65536))
    return hipErrorInvalidValue;
  if (dtype == DT_BF16) return launch_dt<bf16_t>(pro, epi, a, ksplit, s, ev0, ev1);
  return launch_dt<float>(pro, epi, a, ksplit, s, ev0, ev1);
}

}  // namespace pdec

// Fused vocabulary projection + argmax for iterations of at most 16 rows (one
// MFMA row tile), the batch-1 decoding regime.
//
//   logit[r][v] = s * (LN(h_r) . E[v]) + b[v]      (never stored)
//
// Each workgroup returns, per row, the best (largest logit, lowest index) over
// the columns it streamed; the control step reduces those partials.
//
// The V x d weight stream is the whole cost, so the kernel keeps it in flight:
// a fixed grid of workgroups (all resident at once, see VocabShape) whose
// waves walk 16-column tiles t = w, w + W, w + 2W, ... (w the wave's global
// index, W the waves in the grid).  Every lane keeps D 16-byte weight loads
// outstanding in a ring over the flattened (tile, k step) sequence, so the
// next tile's loads leave while the current tile is finished.  E is read from
// its copy in the MFMA feed order when one is given (GemmArgs::wp; a wave's
// word of one (tile, step) is then 1 KB contiguous, where the row-major E
// splits every 128-byte line between two steps), with non-temporal loads
// since E is streamed once per launch (a plain read of 512 MB measured 86 µs
// with them against 93 µs with ordinary loads).
//
// Every logit is accumulated exactly as in the general product kernel with
// whole-K waves (MFMA steps in increasing k from zero, then s * acc + b), so
// both kernels pick the same token for a row.
//
// The LSE variant also keeps, per row, a running log-sum-exp of the logits it
// streams (for the decoding trace's token probabilities), returned beside
// the argmax partials; the logits are still never stored.
#include <hip/hip_ext.h>

#include "common.h"
#include "kernels.h"
#include "mma.h"

namespace pdec {

// Ring depth (weight loads in flight per lane) and waves per SIMD of a
// variant: rows of up to 512 elements leave room for a 12-deep ring at 4
// waves per SIMD (1024 resident workgroups); wider bf16 rows hold twice the
// LayerNorm slabs, so they run at 3 waves per SIMD (768 workgroups) with a
// 16-deep ring (8 when the held rows are float).
template <int LNT, int XF32> struct VocabShape {
  static constexpr int D = LNT > 4 ? (XF32 ? 8 : 16) : 12;
  static constexpr int OCC = LNT > 4 ? 3 : 4;
  static constexpr int MAX_WGS = 256 * OCC;
};

template <typename WT, int XF32, int LNT, int LSE, int D = VocabShape<LNT, XF32>::D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(VocabShape<LNT, XF32>::OCC))) void k_vocab(GemmArgs a) {
  using AT = WT;
  using XT = typename std::conditional<XF32 != 0, float, AT>::type;
  using MM = Mma<WT>;
  using frag = typename MM::frag;
  constexpr int KS = MM::KS;
  constexpr int EPL = MM::EPL;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int lr = lane & 15;          // weight row (column of the logits) fed by this lane
  const int lg = lane >> 4;          // k group of this lane; rows 4 lg .. 4 lg + 3 of the result
  const int K = a.K, N = a.N;
  const int n_steps = K / KS;
  const int n_tiles = (N + 15) / 16;
  const int W = gridDim.x * 4;
  const int w_id = blockIdx.x * 4 + wave;
  const int my_tiles = w_id < n_tiles ? (n_tiles - 1 - w_id) / W + 1 : 0;
  const int total = my_tiles * n_steps;
  const WT* __restrict__ E = static_cast<const WT*>(a.w);
  const WT* __restrict__ Ef = static_cast<const WT*>(a.wp);
  const WT* __restrict__ bias = static_cast<const WT*>(a.bias);
  const bool packed = Ef != nullptr;
  const int wstep = packed ? kWave * EPL : KS;    // elements between a lane's words of consecutive steps

  // this lane's word of step 0 of tile j: E row-major (the last tile's rows
  // beyond N repeat row N - 1; their logits are never used), or E's feed-order
  // copy, where a wave's word of one step is 1 KB contiguous (tiles past the
  // last repeat it; the ring's loads past its tiles are never used)
  auto wrow = [&](int j) -> const WT* {
    const int t = w_id + j * W;
    const int col = min(t * 16 + lr, N - 1);
    return packed ? Ef + (static_cast<size_t>(min(t, n_tiles - 1)) * n_steps * kWave + lane) * EPL
                  : E + static_cast<size_t>(col) * K + EPL * lg;
  };

  // Loads complete in issue order, so everything the LayerNorm prologue reads
  // goes out before the weight ring: the rows (held in registers), then
  // gamma and beta (one 16-byte word per lane, staged through LDS).
  LnTile<WT, XT, LNT / 4> ln;
  ln.load(static_cast<const XT*>(a.x), a.ldx, K, 0, a.n_rows, wave, lane);
  __shared__ uint4 s_gb[2][128];                   // gamma, beta: up to 2 KB each
  const int gb_words = K * static_cast<int>(sizeof(WT)) / 16;
  const int gw = threadIdx.x & 127;
  const uint4 gb = static_cast<const uint4*>(threadIdx.x < 128 ? a.ln_g : a.ln_b)[gw < gb_words ? gw : 0];
  __builtin_amdgcn_sched_barrier(0);   // keep these loads ahead of the weight ring

  // prime the ring: the first D (tile, step) loads.  No load sits under a
  // branch (that would make the compiler wait for every earlier load); a
  // wave with fewer than D steps reads clamped rows it never uses.
  frag ring[D];
  int jn = 0, sn = 0;                // (tile, step) of the next load
  const WT* pn = wrow(0);
#pragma unroll
  for (int u = 0; u < D; ++u) {
    ring[u] = MM::template wload<1>(pn + sn * wstep);
    if (++sn == n_steps) { sn = 0; ++jn; pn = wrow(jn); }
  }
  float bias_v = Elt<WT>::load(bias, min(w_id * 16 + lr, N - 1));

  // LayerNorm of the (at most 16) rows into LDS while the weights arrive
  s_gb[threadIdx.x >> 7][gw] = gb;     // words past the rows are never read
  __syncthreads();
  extern __shared__ __align__(16) unsigned char s_dyn[];
  AT* sA = reinterpret_cast<AT*>(s_dyn);
  const int lda = K + 16 / static_cast<int>(sizeof(AT));
  ln.finish(K, a.ln_eps, reinterpret_cast<const WT*>(s_gb[0]), reinterpret_cast<const WT*>(s_gb[1]), sA, lda,
            nullptr, 0, 0);
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  __syncthreads();

  // stream: consume step g from ring[g % D], refill it with step g + D
  uint32_t bk[4] = {0u, 0u, 0u, 0u};
  uint32_t bi[4] = {0x7fffffffu, 0x7fffffffu, 0x7fffffffu, 0x7fffffffu};
  uint32_t nf = 0;                   // bit i: a non-finite logit in row 4 lg + i
  float lm[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, ls[4] = {0.f, 0.f, 0.f, 0.f};
  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  int j = 0, s = 0;                  // (tile, step) being consumed
  const AT* arow = sA + static_cast<size_t>(lr) * lda + EPL * lg;
  for (int g0 = 0; g0 < total; g0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      if (g0 + u >= total) break;
      const frag b = ring[u];
      if (g0 + u + D < total) {
        ring[u] = MM::template wload<1>(pn + sn * wstep);
        if (++sn == n_steps) { sn = 0; ++jn; pn = wrow(jn); }
      }
      acc = MM::step(MM::load(arow + s * KS), b, acc);
      if (++s == n_steps) {
        const int col = (w_id + j * W) * 16 + lr;
        if (col < N) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (4 * lg + i >= R) continue;
            const float logit = fmaf(a.logit_scale, acc[i], bias_v);   // s * (h . E[col]) + bias[col]
            if (!isfinite(logit)) nf |= 1u << i;
            else {
              best_take(bk[i], bi[i], float_key(logit), static_cast<uint32_t>(col));
              if constexpr (LSE != 0) lse_take(lm[i], ls[i], logit);
            }
          }
        }
        acc = floatx4_t{0.f, 0.f, 0.f, 0.f};
        s = 0;
        ++j;
        if (j < my_tiles) bias_v = Elt<WT>::load(bias, min((w_id + j * W) * 16 + lr, N - 1));
      }
    }
  }

  // best of each row over the 16 columns of a lane group, then over the waves
#pragma unroll
  for (int i = 0; i < 4; ++i) group16_best(bk[i], bi[i]);
  nf = group16_or(nf);
  __shared__ uint32_t s_key[4][16];
  __shared__ int s_idx[4][16];
  __shared__ float2 s_lse[LSE != 0 ? 4 : 1][16];
  if constexpr (LSE != 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) group16_lse(lm[i], ls[i]);
  }
  if (lr == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s_key[wave][4 * lg + i] = bk[i];
      s_idx[wave][4 * lg + i] = static_cast<int>(bi[i] | (((nf >> i) & 1u) << 31));
      if constexpr (LSE != 0) s_lse[wave][4 * lg + i] = make_float2(lm[i], ls[i]);
    }
  }
  __syncthreads();
  if (threadIdx.x < 16 && static_cast<int>(threadIdx.x) < R) {
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
    a.partials[static_cast<size_t>(r) * a.part_ld + blockIdx.x] =
        make_uint2(kk, static_cast<uint32_t>(ii) | (static_cast<uint32_t>(ff) << 31));
    if constexpr (LSE != 0) {
      float m = s_lse[0][r].x, sm = s_lse[0][r].y;
      for (int w = 1; w < 4; ++w) lse_merge(m, sm, s_lse[w][r].x, s_lse[w][r].y);   // wave order
      a.part_lse[static_cast<size_t>(r) * a.part_ld + blockIdx.x] = make_float2(m, sm);
    }
  }
}

int vocab_grid(int dtype, int V, int d) {
  const int max_wgs = dtype == DT_BF16 && d > 512 ? VocabShape<8, 0>::MAX_WGS : VocabShape<4, 0>::MAX_WGS;
  const int tiles = (V + 15) / 16;
  return std::max(1, std::min(max_wgs, (tiles + 3) / 4));
}

namespace {

// With events, the launch records the kernel's own start and end in them
// (hipExtLaunchKernel: timestamps of the dispatch itself, no marker packets).
template <typename K>
hipError_t launch_ev(K kernel, dim3 grid, size_t lds, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                     const GemmArgs& a) {
  if (ev0 != nullptr) hipExtLaunchKernelGGL(kernel, grid, dim3(256), static_cast<uint32_t>(lds), s, ev0, ev1, 0u, a);
  else hipLaunchKernelGGL(kernel, grid, dim3(256), lds, s, a);
  return hipGetLastError();
}

template <typename WT, int XF32, int LSE>
hipError_t launch_x(const GemmArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const size_t lds = gemm_ln_lds_bytes(a.K, sizeof(WT));
  const dim3 grid(vocab_grid(std::is_same<WT, bf16_t>::value ? DT_BF16 : DT_F32, a.N, a.K));
  if constexpr (std::is_same<WT, bf16_t>::value) {
    if (a.K > 512) return launch_ev(k_vocab<WT, XF32, 8, LSE>, grid, lds, s, ev0, ev1, a);
  }
  return launch_ev(k_vocab<WT, XF32, 4, LSE>, grid, lds, s, ev0, ev1, a);
}

template <typename WT>
hipError_t launch_w(const GemmArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (a.part_lse != nullptr)
    return a.x_f32 ? launch_x<WT, 1, 1>(a, s, ev0, ev1) : launch_x<WT, 0, 1>(a, s, ev0, ev1);
  return a.x_f32 ? launch_x<WT, 1, 0>(a, s, ev0, ev1) : launch_x<WT, 0, 0>(a, s, ev0, ev1);
}

}  // namespace

hipError_t launch_vocab_argmax(int dtype, const GemmArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (a.n_rows <= 0) return hipSuccess;
  if (a.n_rows > 16 || a.N <= 0) return hipErrorInvalidValue;
  const int ks = dtype == DT_BF16 ? Mma<bf16_t>::KS : Mma<float>::KS;
  if (a.K % ks != 0 || a.K % 32 != 0 || a.K > (dtype == DT_BF16 ? 1024 : 512) ||
      a.part_ld < vocab_grid(dtype, a.N, a.K))
    return hipErrorInvalidValue;
  return dtype == DT_BF16 ? launch_w<bf16_t>(a, s, ev0, ev1) : launch_w<float>(a, s, ev0, ev1);
}

}  // namespace pdec

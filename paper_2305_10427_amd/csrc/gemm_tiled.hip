// Matrix products of iterations with many rows (batched sentences times
// block positions) on LDS-staged MFMA tiles, bf16 storage.
//
// Y[r][n] = sum_k X[r][k] * W[n][k] (+ the epilogues of k_gemm), W stored
// [N][K] row-major.  A workgroup of 4 waves computes a BM x BN output tile;
// wave (wm, wn) owns the (BM/2) x (BN/2) quarter at (wm, wn), as FM x FN
// subtiles of 16 x 16 on v_mfma_f32_16x16x32_bf16.  X and W tiles of 64 k go
// through a double-buffered LDS stage (one barrier per 64 k): the next tile's
// global loads leave before the current tile's products.
//
// Same arithmetic as the row-streaming product kernel, element for element:
// K is cut into the same KSPLIT ranges of MFMA steps (range w covers steps
// [n_steps w / KSPLIT, n_steps (w + 1) / KSPLIT)), each range accumulates
// from zero in increasing k, and the range sums are added in range order; the
// epilogues evaluate the same expressions.  A row's values therefore do not
// depend on which kernel computed them, on the tile slot the row occupies, or
// on the other rows of the call: greedy decoding and every block size of the
// Jacobi iterations evaluate the same map.
//
// Workgroups are laid out for the eight XCDs (each with its own L2): the
// tiles are ordered with row blocks fastest and cut into eight contiguous
// chunks, chunk x going to the workgroups that the dispatcher places on XCD x
// (linear workgroup id = x mod 8).  The row blocks that share a weight tile
// therefore run on one XCD, close in time, and the weight tile is read from
// HBM once per XCD.
//
// Rows at or above the device row count are not stored; a workgroup whose
// rows all lie there returns at once.
#include "common.h"
#include "kernels.h"
#include "mma.h"

namespace pdec {

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource (32-bit data format, no swizzle, no index).
constexpr int kBufferWord3 = 0x00020000;

constexpr int kBK = 64;            // k per LDS stage (two MFMA steps)
constexpr int kLdsPad = 8;         // bf16 elements of padding per LDS row (rows 144 B apart: conflict-free b128 reads)
constexpr int kLdsRow = kBK + kLdsPad;

// BM x BN output tile, WM x WN waves; each wave owns a TM x TN block of
// FM x FN 16 x 16 subtiles.
template <int BM, int BN, int WM, int WN> struct TileShape {
  static constexpr int NT = 64 * WM * WN;           // threads
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 16, FN = TN / 16;
  static constexpr int LA = BM * kBK / 8 / NT;      // 16-byte loads per thread per stage
  static constexpr int LB = BN * kBK / 8 / NT;
  static constexpr size_t LDS = 2ull * (BM + BN) * kLdsRow * sizeof(bf16_t);
  static_assert(FM >= 1 && FN >= 1 && LA >= 1 && LB >= 1, "tile shape");
};

}  // namespace

template <int EPI, int BM, int BN, int WM, int WN, int NS, int KSPLIT>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_tiled(GemmArgs a, int n_rb, int n_tiles) {
  if constexpr (EPI == EPI_QKV) layer_select(a, blockIdx.y);
  using S = TileShape<BM, BN, WM, WN>;
  using MM = Mma<bf16_t>;
  using frag = MM::frag;
  constexpr int FM = S::FM, FN = S::FN, NT = S::NT;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 15, lg = lane >> 4;

  // XCD-aware tile order (see the header comment)
  const int L = blockIdx.x;
  const int xcd = L & 7, q = n_tiles >> 3, rem = n_tiles & 7;
  const int tile = xcd * q + min(xcd, rem) + (L >> 3);
  const int rb = tile % n_rb, cb = tile / n_rb;
  const int m0 = rb * BM, n0 = cb * BN;
  const int R_max = a.n_rows;
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  if (m0 >= R) return;                                   // workgroup-uniform

  const int K = a.K, N = a.N;
  const bf16_t* __restrict__ X = static_cast<const bf16_t*>(a.x);
  const bf16_t* __restrict__ W = static_cast<const bf16_t*>(a.w);
  extern __shared__ __align__(16) unsigned char s_dyn[];
  bf16_t* sA = reinterpret_cast<bf16_t*>(s_dyn);               // [2][BM][kLdsRow]
  bf16_t* sB = sA + 2 * BM * kLdsRow;                         // [2][BN][kLdsRow]

  // global -> register staging: chunk c = tid + NT i covers row c / 8, k 8 (c % 8).
  // Two register sets: the loads of stage kt + 2 leave while stage kt is
  // multiplied and stage kt + 1 waits in the other set for its LDS store.
  // Stage loads are buffer loads: a fixed 32-bit byte offset per lane plus the
  // stage's k offset in a scalar register, so no per-stage address arithmetic
  // writes a register that an earlier load may still be filling (the compiler
  // would then wait for every outstanding load before issuing the next).
  // Reads past the end of a buffer return zero instead of faulting.
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(X), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(R_max) * a.ldx * 2),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(W), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(N) * K * 2), kBufferWord3);
  uint32_t oa[S::LA], ob[S::LB];
#pragma unroll
  for (int i = 0; i < S::LA; ++i) {
    const int c = tid + NT * i;
    const int row = min(m0 + c / 8, R_max - 1);
    oa[i] = (static_cast<uint32_t>(row) * a.ldx + 8 * (c % 8)) * 2;
  }
#pragma unroll
  for (int i = 0; i < S::LB; ++i) {
    const int c = tid + NT * i;
    const int col = min(n0 + c / 8, N - 1);
    ob[i] = (static_cast<uint32_t>(col) * K + 8 * (c % 8)) * 2;
  }
  struct Staged {
    u32x4_t a[S::LA];
    u32x4_t b[S::LB];
  };
  // NS register sets, used in rotation: the loads of stage kt + NS leave
  // while stage kt is multiplied.  (Sets are named by compile-time indices
  // only; HIP's uint4 struct here would be kept in scratch memory.)
  Staged st[NS];
  auto load_stage = [&](Staged& r, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < S::LA; ++i)
      r.a[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(xr, oa[i], 2 * k0, 0));
#pragma unroll
    for (int i = 0; i < S::LB; ++i)
      r.b[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, ob[i], 2 * k0, 0));
  };
  auto store_stage = [&](const Staged& r, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < S::LA; ++i) {
      const int c = tid + NT * i;
      *reinterpret_cast<u32x4_t*>(sA + (buf * BM + c / 8) * kLdsRow + 8 * (c % 8)) = r.a[i];
    }
#pragma unroll
    for (int i = 0; i < S::LB; ++i) {
      const int c = tid + NT * i;
      *reinterpret_cast<u32x4_t*>(sB + (buf * BN + c / 8) * kLdsRow + 8 * (c % 8)) = r.b[i];
    }
  };

  floatx4_t acc[FM][FN], tot[KSPLIT > 1 ? FM : 1][KSPLIT > 1 ? FN : 1];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  // K-split ranges: w_cur is the range being accumulated, bnd the first step of the next one
  const int n_steps = K / MM::KS;
  int w_cur = 0;
  int bnd = KSPLIT > 1 ? n_steps / KSPLIT : n_steps + 1;
  auto fold = [&]() __attribute__((always_inline)) {
    if constexpr (KSPLIT > 1) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          tot[i][j] = w_cur == 0 ? acc[i][j] : tot[i][j] + acc[i][j];
          acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
        }
    }
    ++w_cur;
  };

  auto compute_stage = [&](int kt) __attribute__((always_inline)) {
    const int buf = kt & 1;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int s = kt * 2 + st;
      if constexpr (KSPLIT > 1) {
        while (w_cur + 1 < KSPLIT && s == bnd) {
          fold();
          bnd = (n_steps * (w_cur + 1)) / KSPLIT;
        }
      }
      frag fa[FM], fb[FN];
      const int kk = st * MM::KS + MM::EPL * lg;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *reinterpret_cast<const uint4*>(sA + (buf * BM + wm * S::TM + i * 16 + lr) * kLdsRow + kk);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *reinterpret_cast<const uint4*>(sB + (buf * BN + wn * S::TN + j * 16 + lr) * kLdsRow + kk);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = MM::step(fa[i], fb[j], acc[i][j]);
    }
  };

  const int n_kt = K / kBK;
  // Every load is issued unconditionally (stages past the end reload the last
  // stage): a load under a branch makes the compiler wait for all outstanding
  // loads where the paths join.
#pragma unroll
  for (int u = 0; u < NS; ++u) load_stage(st[u], min(u, n_kt - 1) * kBK);
  store_stage(st[0], 0);
  __syncthreads();
  int kt0 = 0;
  for (; kt0 + NS <= n_kt; kt0 += NS) {
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      // st[u] held stage kt (already in LDS): refill it with stage kt + NS;
      // st[u + 1] holds stage kt + 1, stored once this stage's products are
      // issued (after the last stage the store fills the idle buffer, unread)
      const int kt = kt0 + u;
      load_stage(st[u], min(kt + NS, n_kt - 1) * kBK);
      compute_stage(kt);
      store_stage(st[(u + 1) % NS], (kt + 1) & 1);
      __syncthreads();
    }
  }
  // the last n_kt mod NS stages: their loads have all been issued
#pragma unroll
  for (int u = 0; u < NS - 1; ++u) {
    const int kt = kt0 + u;
    if (kt < n_kt) {
      compute_stage(kt);
      if (kt + 1 < n_kt) store_stage(st[(u + 1) % NS], (kt + 1) & 1);
      __syncthreads();
    }
  }
  while (w_cur < KSPLIT) fold();   // the last range, then any empty trailing ranges
  auto res = [&](int i, int j) __attribute__((always_inline)) -> const floatx4_t& {
    if constexpr (KSPLIT > 1) return tot[i][j];
    else return acc[i][j];
  };

  // epilogue: lane holds C[4 lg + e][lr] of each subtile
  float bias_v[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j)
    bias_v[j] = Elt<bf16_t>::load(static_cast<const bf16_t*>(a.bias), min(n0 + wn * S::TN + j * 16 + lr, N - 1));

  if constexpr (EPI == EPI_ARGMAX) {
    uint32_t bk[FM][4], bi[FM][4];
    uint32_t nf = 0;   // bit 4 i + e: a non-finite logit in row (i, e)
    const bool want_lse = a.part_lse != nullptr;
    float lm[FM][4], ls[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bk[i][e] = 0u;
        bi[i][e] = 0x7fffffffu;
        lm[i][e] = -INFINITY;
        ls[i][e] = 0.f;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + wn * S::TN + j * 16 + lr;
          const float logit = fmaf(a.logit_scale, res(i, j)[e], bias_v[j]);   // s * (h . E[col]) + bias[col]
          if (col < N) {
            if (!isfinite(logit)) nf |= 1u << (4 * i + e);
            else {
              best_take(bk[i][e], bi[i][e], float_key(logit), static_cast<uint32_t>(col));
              if (want_lse) lse_take(lm[i][e], ls[i][e], logit);
            }
          }
        }
        group16_best(bk[i][e], bi[i][e]);
        if (want_lse) group16_lse(lm[i][e], ls[i][e]);
      }
    nf = group16_or(nf);
    __shared__ uint32_t s_key[WN][BM];
    __shared__ uint32_t s_idx[WN][BM];
    __shared__ float2 s_lse[WN][BM];
    if (lr == 0) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rl = wm * S::TM + i * 16 + 4 * lg + e;
          s_key[wn][rl] = bk[i][e];
          s_idx[wn][rl] = bi[i][e] | (((nf >> (4 * i + e)) & 1u) << 31);
          if (want_lse) s_lse[wn][rl] = make_float2(lm[i][e], ls[i][e]);
        }
    }
    __syncthreads();
    for (int t = tid; t < BM; t += NT) {
      if (m0 + t >= R) break;
      uint32_t kk = s_key[0][t], ii = s_idx[0][t] & 0x7fffffffu, ff = s_idx[0][t] >> 31;
#pragma unroll
      for (int w = 1; w < WN; ++w) {
        best_take(kk, ii, s_key[w][t], s_idx[w][t] & 0x7fffffffu);
        ff |= s_idx[w][t] >> 31;
      }
      a.partials[static_cast<size_t>(m0 + t) * a.part_ld + cb] = make_uint2(kk, ii | (ff << 31));
      if (want_lse) {
        float m = s_lse[0][t].x, sm = s_lse[0][t].y;
#pragma unroll
        for (int w = 1; w < WN; ++w) lse_merge(m, sm, s_lse[w][t].x, s_lse[w][t].y);   // wave order
        a.part_lse[static_cast<size_t>(m0 + t) * a.part_ld + cb] = make_float2(m, sm);
      }
    }
    return;
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = m0 + wm * S::TM + i * 16 + 4 * lg + e;
        if (row >= R) continue;
        int sent = 0, pos = 0;
        if constexpr (EPI == EPI_QKV) row_place(a.rows, row, sent, pos);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + wn * S::TN + j * 16 + lr;
          if (col >= N) continue;
          const float v = res(i, j)[e];
          if constexpr (EPI == EPI_F32) {
            a.out_f32[static_cast<size_t>(row) * a.ldo + col] = v + bias_v[j];
          } else if constexpr (EPI == EPI_ACT) {
            float t = v + bias_v[j];
            t = (a.act == 2) ? gelu_erf(t) : relu(t);
            Elt<bf16_t>::store(static_cast<bf16_t*>(a.out), static_cast<size_t>(row) * a.ldo + col, t);
          } else if constexpr (EPI == EPI_RESID) {
            const float rv = Elt<bf16_t>::load(static_cast<const bf16_t*>(a.resid), static_cast<size_t>(row) * a.ldr + col);
            const float t = (v + bias_v[j]) + rv;
            if (a.out_f32 != nullptr) a.out_f32[static_cast<size_t>(row) * a.ldo + col] = t;
            else Elt<bf16_t>::store(static_cast<bf16_t*>(a.out), static_cast<size_t>(row) * a.ldo + col, t);
          } else if constexpr (EPI == EPI_QKV) {
            const float t = v + bias_v[j];
            if (col < a.q_cols) {
              a.out_f32[static_cast<size_t>(row) * a.ldo + col] = t;
            } else {
              const int c = col - a.q_cols;
              const int which = c / a.d;
              const int cc = c - which * a.d;
              const int hh = cc / a.dh;
              const int dd = cc - hh * a.dh;
              const size_t idx = ((static_cast<size_t>(sent) * a.H + hh) * a.T + pos) * a.dh + dd;
              Elt<bf16_t>::store(static_cast<bf16_t*>(which == 0 ? a.kc : a.vc), idx, t);
            }
          } else if constexpr (EPI == EPI_LOGITS) {
            a.out_f32[static_cast<size_t>(row) * a.ldo + col] = fmaf(a.logit_scale, v, bias_v[j]);
          }
        }
      }
  }
}

namespace {

template <int EPI, int BM, int BN, int WM, int WN, int NS, int KSPLIT>
void allow_lds() {
  // double-buffered stages of the larger tiles exceed 64 KB of LDS (gfx950 has 160 KB per CU)
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_tiled<EPI, BM, BN, WM, WN, NS, KSPLIT>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(TileShape<BM, BN, WM, WN>::LDS));
}

template <int EPI, int BM, int BN, int WM, int WN, int NS, int KSPLIT>
hipError_t launch_shape(const GemmArgs& a, hipStream_t s) {
  const int n_rb = (a.n_rows + BM - 1) / BM;
  const int n_tiles = n_rb * ((a.N + BN - 1) / BN);
  const size_t lds = TileShape<BM, BN, WM, WN>::LDS;
  const int gy = EPI == EPI_QKV && a.n_layers > 1 ? a.n_layers : 1;
  hipLaunchKernelGGL((k_gemm_tiled<EPI, BM, BN, WM, WN, NS, KSPLIT>), dim3(n_tiles, gy), dim3(64 * WM * WN), lds, s, a,
                     n_rb, n_tiles);
  return hipGetLastError();
}

// Tile configurations (rows x columns, waves, register sets in flight),
// chosen by measurement on MI355X: 0: 128 x 128, 2 x 2 waves, 2 sets (the
// vocabulary argmax above 64 rows: 712 TFLOP/s at 1024 rows); 1: 64 x 64,
// 2 x 2 waves, 4 sets (decoder products: many workgroups for N of 1-4 K
// columns); 2: 64 x 128, 2 x 2 waves, 3 sets (the vocabulary argmax of
// 17-64 rows: 94 us for 250,027 x 1024 at 64 rows); 3: 32 x 64 and 4: 32 x 32,
// 2 x 2 waves, 4 sets (decoder products of a few hundred rows); 5: 32 x 128,
// 2 x 2 waves, 3 sets (the vocabulary argmax of 17-32 rows).  Every
// configuration accumulates each output element in the same order, so all
// give bitwise the same products.
constexpr int kTileCfgs = 6;

template <int EPI, int KSPLIT>
hipError_t launch_k(const GemmArgs& a, int cfg, hipStream_t s) {
  switch (cfg) {
    case 0: return launch_shape<EPI, 128, 128, 2, 2, 2, KSPLIT>(a, s);
    case 1: return launch_shape<EPI, 64, 64, 2, 2, 4, KSPLIT>(a, s);
    case 2: return launch_shape<EPI, 64, 128, 2, 2, 3, KSPLIT>(a, s);
    case 3: return launch_shape<EPI, 32, 64, 2, 2, 4, KSPLIT>(a, s);
    case 4: return launch_shape<EPI, 32, 32, 2, 2, 4, KSPLIT>(a, s);
    case 5: return launch_shape<EPI, 32, 128, 2, 2, 3, KSPLIT>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int EPI, int KSPLIT>
void init_k() {
  allow_lds<EPI, 128, 128, 2, 2, 2, KSPLIT>();   // the smaller tiles fit the default LDS limit
  allow_lds<EPI, 64, 64, 2, 2, 4, KSPLIT>();
  allow_lds<EPI, 64, 128, 2, 2, 3, KSPLIT>();
}

template <int EPI>
hipError_t launch_e(const GemmArgs& a, int ksplit, int cfg, hipStream_t s) {
  if constexpr (EPI == EPI_ARGMAX || EPI == EPI_LOGITS) {
    return ksplit == 1 ? launch_k<EPI, 1>(a, cfg, s) : hipErrorInvalidValue;
  } else {
    if (ksplit == 4) return launch_k<EPI, 4>(a, cfg, s);
    if (ksplit == 8) return launch_k<EPI, 8>(a, cfg, s);
    return hipErrorInvalidValue;
  }
}

int tile_bn(int cfg) { return cfg == 1 || cfg == 3 ? 64 : (cfg == 4 ? 32 : 128); }   // 0, 2, 5: 128

}  // namespace

void gemm_tiled_init() {
  init_k<EPI_F32, 4>();
  init_k<EPI_F32, 8>();
  init_k<EPI_ACT, 4>();
  init_k<EPI_ACT, 8>();
  init_k<EPI_RESID, 4>();
  init_k<EPI_RESID, 8>();
  init_k<EPI_QKV, 4>();
  init_k<EPI_QKV, 8>();
  init_k<EPI_ARGMAX, 1>();
  init_k<EPI_LOGITS, 1>();
}

// Tile configuration of a product of `rows` rows and N columns.  The
// vocabulary argmax keeps 128-column tiles (its partial count depends only
// on N).
int gemm_tiled_cfg(int epi, int N, int rows) {
  if (epi == EPI_ARGMAX || epi == EPI_LOGITS) {
    // 128 columns; 32 rows up to 32 rows, then 128- or 64-row tiles,
    // whichever pads the rows less (ties: 128)
    if (rows <= 32) return 5;
    const int pad128 = (rows + 127) / 128 * 128, pad64 = (rows + 63) / 64 * 64;
    return rows > 64 && pad128 <= pad64 ? 0 : 2;
  }
  // decoder products: the largest tile that still gives 1024 workgroups (a
  // few per CU), else 32 x 32 (measured at 100, 200, 631 and 1024 rows, N of
  // 512-4096: the smaller tiles win whenever the larger ones leave CUs idle)
  const auto wgs = [&](int bm, int bn) { return ((rows + bm - 1) / bm) * ((N + bn - 1) / bn); };
  if (wgs(64, 64) >= 1024) return 1;
  if (wgs(32, 64) >= 1024) return 3;
  return 4;
}

int gemm_tiled_bn(int epi, int N, int rows) { return tile_bn(gemm_tiled_cfg(epi, N, rows)); }

bool gemm_tiled_ok(int dtype, int pro, const GemmArgs& a) {
  // byte offsets within the input rows and the weight matrix must fit 31 bits
  const bool off32 = static_cast<uint64_t>(a.n_rows) * a.ldx * 2 < (1ull << 31) &&
                     static_cast<uint64_t>(a.N) * a.K * 2 < (1ull << 31);
  return dtype == DT_BF16 && pro == PRO_NONE && !a.x_f32 && a.K % kBK == 0 && a.K > 0 && a.N > 0 && off32;
}

hipError_t launch_gemm_tiled_cfg(int epi, int ksplit, int cfg, const GemmArgs& a, hipStream_t s) {
  if (a.n_rows <= 0) return hipSuccess;
  if (a.K % kBK != 0 || a.x_f32 || cfg < 0 || cfg >= kTileCfgs) return hipErrorInvalidValue;
  // the argmax partials are laid out per column tile: at most ceil(N / 32) per row
  if (epi == EPI_ARGMAX && a.part_ld < (a.N + tile_bn(cfg) - 1) / tile_bn(cfg)) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_F32: return launch_e<EPI_F32>(a, ksplit, cfg, s);
    case EPI_ACT: return launch_e<EPI_ACT>(a, ksplit, cfg, s);
    case EPI_RESID: return launch_e<EPI_RESID>(a, ksplit, cfg, s);
    case EPI_QKV: return launch_e<EPI_QKV>(a, ksplit, cfg, s);
    case EPI_ARGMAX: return launch_e<EPI_ARGMAX>(a, ksplit, cfg, s);
    case EPI_LOGITS: return launch_e<EPI_LOGITS>(a, ksplit, cfg, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_tiled(int epi, int ksplit, const GemmArgs& a, hipStream_t s) {
  if (a.x_feed || a.out_feed) return hipErrorInvalidValue;   // row-major operands only
  return launch_gemm_tiled_cfg(epi, ksplit, gemm_tiled_cfg(epi, a.N, a.n_rows), a, s);
}

}  // namespace pdec

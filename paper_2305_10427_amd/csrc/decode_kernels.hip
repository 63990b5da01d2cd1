// Attention, embedding, LayerNorm, argmax reduction and the on-device
// fixed-point control of the parallel decoding iteration.
#include "attn.h"
#include "common.h"
#include "kernels.h"
#include "mma.h"

namespace pdec {

constexpr int kMaxKeys = 1024;
static_assert(kAttnChunk == kAttnChunkKeys, "attention chunk of the host-side launch choice");
constexpr int kMaxHeadDim = 128;


// ---------------------------------------------------------------------------
// Scaled dot-product attention, one wave per (row, head); a workgroup holds
// one head of kAttnRows consecutive rows.  One row per workgroup spreads a
// launch over the most CUs; measured per large GS-Jacobi b = 16 iteration:
// 4 heads of one row per workgroup 570 µs, one head of 8 / 4 / 2 / 1 rows
// 597 / 559 / 549 / 544 µs (greedy 485 µs, then 462 µs for every size).
//
// The row at position p attends to keys 0..p of its own sentence (causal,
// decoder self-attention over the KV cache whose block entries were written by
// the QKV product of this iteration) or to keys 0..n_s-1 (encoder memory /
// encoder self-attention, padded keys excluded).  The wave walks the row's
// 64-key chunks in order (chunk_fold); chunk boundaries depend only on the
// row's own key count.
constexpr int kAttnRows = 1;   // rows (waves) per workgroup

// ONE: every row is of sentence 0 and attends to its whole source (a batch
// of one, non-causal): the first chunk's key slots are loaded with the query,
// before the key count klen[0] and the row count arrive.  Slots past the key
// count hold finite values (the caches are zeroed at set-up and only ever
// written with finite ones), whose p = 0 adds exact zeros, as key 0 does
// in the other loads; a row past the count leaves after its loads.
template <typename AT, int DH, int ONE>
__global__ __launch_bounds__(kAttnRows * kWave) void k_attn(AttnArgs a) {
  __shared__ float s_q[kAttnRows][DH];
  __shared__ AttnScratch s_scr[kAttnRows];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  // workgroup g: head g mod H of rows kAttnRows (g div H) + wave, so that the
  // waves of a workgroup read one head's keys (of one sentence, but at a
  // sentence boundary)
  const int hh = static_cast<int>(blockIdx.x) % a.H;
  const int row = (static_cast<int>(blockIdx.x) / a.H) * kAttnRows + wave;
  if (row >= a.rows_max) return;         // padding waves of the last workgroup; no workgroup barrier below
  // the device row count, the query and the row's placement go out together
  // (rows below the launch bound have valid query and placement slots); rows
  // at or past the count leave before touching the keys
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const float* q = a.q + static_cast<size_t>(row) * a.ldq + hh * DH;
  float qv[(DH + kWave - 1) / kWave];
#pragma unroll
  for (int i = 0; i < (DH + kWave - 1) / kWave; ++i) {
    const int d = lane + kWave * i;
    qv[i] = q[d < DH ? d : 0];           // unconditional load
  }
  // two chunk buffers: the loads of the next chunk are issued before the
  // current one is folded (a chunk past the row's keys loads key 0 and is
  // never folded)
  KeyChunk<AT, DH> ka, kb;
  int nk;
  const AT* Kb;
  const AT* Vb;
  if constexpr (ONE != 0) {
    nk = *a.klen;
    const size_t base = static_cast<size_t>(hh) * a.T * DH;
    Kb = static_cast<const AT*>(a.kc) + base;
    Vb = static_cast<const AT*>(a.vc) + base;
    ka.load(Kb, Vb, 0, a.T, lane);       // every slot of the first chunk
    if (row >= R) return;
  } else {
    int s, p;
    row_place(a.rows, row, s, p);
    if (row >= R) return;
    nk = a.causal ? p + 1 : a.klen[s];
    const size_t base = (static_cast<size_t>(s) * a.H + hh) * a.T * DH;
    Kb = static_cast<const AT*>(a.kc) + base;
    Vb = static_cast<const AT*>(a.vc) + base;
    ka.load(Kb, Vb, 0, nk, lane);
  }
#pragma unroll
  for (int i = 0; i < (DH + kWave - 1) / kWave; ++i) {
    const int d = lane + kWave * i;
    if (d < DH) s_q[wave][d] = qv[i];
  }
  wave_lds_sync();
  RowState<DH> st;
  st.init();
  if (nk <= kAttnChunk) {                               // wave-uniform: one chunk
    chunk_fold<AT, DH>(s_q[wave], ka, 0, nk, a.scale, lane, s_scr[wave], st);
  } else {
    // every load below is of a chunk that exists and sits on the straight
    // path of the loop body (a load under a branch would make the compiler
    // wait for all outstanding loads before the next use of any of them)
    for (int key0 = 0;; key0 += 2 * kAttnChunk) {
      kb.load(Kb, Vb, key0 + kAttnChunk, nk, lane);
      __builtin_amdgcn_sched_barrier(0);                 // the next chunk's loads go out first
      chunk_fold<AT, DH>(s_q[wave], ka, key0, nk, a.scale, lane, s_scr[wave], st);
      if (key0 + 2 * kAttnChunk >= nk) {                // kb holds the last chunk
        chunk_fold<AT, DH>(s_q[wave], kb, key0 + kAttnChunk, nk, a.scale, lane, s_scr[wave], st);
        break;
      }
      ka.load(Kb, Vb, key0 + 2 * kAttnChunk, nk, lane);
      __builtin_amdgcn_sched_barrier(0);
      chunk_fold<AT, DH>(s_q[wave], kb, key0 + kAttnChunk, nk, a.scale, lane, s_scr[wave], st);
      if (key0 + 3 * kAttnChunk >= nk) {                // ka holds the last chunk
        chunk_fold<AT, DH>(s_q[wave], ka, key0 + 2 * kAttnChunk, nk, a.scale, lane, s_scr[wave], st);
        break;
      }
    }
  }
  AT* out = static_cast<AT*>(a.out);
  if (a.out_feed) {
    const int K = a.H * DH;
    row_output<AT, DH>(st, out, [&](int d) { return feed_index<Mma<AT>::KS, Mma<AT>::EPL>(row, hh * DH + d, K); },
                       lane);
  } else {
    const size_t base = static_cast<size_t>(row) * a.ldo + hh * DH;
    row_output<AT, DH>(st, out, [&](int d) { return base + d; }, lane);
  }
}

// Attention of rows with several key chunks: one workgroup of W waves per
// (row, head).  Wave w
// evaluates chunks w, w + W, ... of the row (chunk_eval) and leaves each
// chunk's (m_c, l_c, o_c) in LDS; wave 0 then folds them in key order
// (fold_chunk).  That is k_attn's arithmetic in k_attn's order, so a row's
// output is bitwise the same, while the chunks of a long row are evaluated
// side by side instead of one after another.
template <typename AT, int DH, int W, int ONE>
__global__ __launch_bounds__(W * kWave) void k_attn_split(AttnArgs a) {
  constexpr int NQ = (DH + kWave - 1) / kWave;
  constexpr int NP = RowState<DH>::NP;
  constexpr int NC = kMaxKeys / kAttnChunk;
  struct Slot {
    float m, l;
    float o[NP][32][2];
  };
  __shared__ float s_q[W][DH];
  __shared__ AttnScratch s_scr[W];
  __shared__ Slot s_c[NC];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int hh = static_cast<int>(blockIdx.x) % a.H;
  const int row = static_cast<int>(blockIdx.x) / a.H;   // below rows_max (grid)
  // the device row count, the query and the row's placement go out together;
  // a row at or past the count leaves with its whole workgroup
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const float* q = a.q + static_cast<size_t>(row) * a.ldq + hh * DH;
  float qv[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int d = lane + kWave * i;
    qv[i] = q[d < DH ? d : 0];           // unconditional load
  }
  int s = 0, p = 0, nk;
  KeyChunk<AT, DH> kc;
  if constexpr (ONE != 0) {
    // every wave loads its first chunk's slots before the key count arrives
    nk = *a.klen;
    kc.load_k(static_cast<const AT*>(a.kc) + static_cast<size_t>(hh) * a.T * DH, wave * kAttnChunk, a.T, lane);
    __builtin_amdgcn_sched_barrier(0);
    kc.load_v(static_cast<const AT*>(a.vc) + static_cast<size_t>(hh) * a.T * DH, wave * kAttnChunk, a.T, lane);
    __builtin_amdgcn_sched_barrier(0);
    if (row >= R) return;                // the whole workgroup (row is uniform)
  } else {
    row_place(a.rows, row, s, p);
    if (row >= R) return;
    nk = a.causal ? p + 1 : a.klen[s];
  }
  const int nc = (nk + kAttnChunk - 1) / kAttnChunk;    // 1 .. NC
  const size_t base = (static_cast<size_t>(s) * a.H + hh) * a.T * DH;
  const AT* Kb = static_cast<const AT*>(a.kc) + base;
  const AT* Vb = static_cast<const AT*>(a.vc) + base;
  if (nc == 1 && wave != 0) return;     // workgroup-uniform: one chunk, no barrier below
  if constexpr (ONE == 0) {
    // every wave loads its first chunk on the straight path (a wave past the
    // row's chunks loads key 0 and evaluates nothing)
    kc.load_k(Kb, wave * kAttnChunk, nk, lane);
    __builtin_amdgcn_sched_barrier(0);   // the K rows first: the scores start while V arrives
    kc.load_v(Vb, wave * kAttnChunk, nk, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int d = lane + kWave * i;
    if (d < DH) s_q[wave][d] = qv[i];
  }
  wave_lds_sync();
  auto keep = [&](const ChunkOut<DH>& c, int j) {
    if (lane < 32) {
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        s_c[j].o[i][lane][0] = c.o[i][0];
        s_c[j].o[i][lane][1] = c.o[i][1];
      }
    }
    if (lane == 0) {
      s_c[j].m = c.m;
      s_c[j].l = c.l;
    }
  };
  ChunkOut<DH> c0;                        // wave 0's chunk 0 stays in registers
  if (wave < nc) {                        // wave-uniform
    chunk_eval<AT, DH>(s_q[wave], kc, wave * kAttnChunk, nk, a.scale, lane, s_scr[wave], c0);
    if (wave != 0) keep(c0, wave);
    for (int j = wave + W; j < nc; j += W) {   // rows of more than W chunks
      kc.load(Kb, Vb, j * kAttnChunk, nk, lane);
      ChunkOut<DH> c;
      chunk_eval<AT, DH>(s_q[wave], kc, j * kAttnChunk, nk, a.scale, lane, s_scr[wave], c);
      keep(c, j);
    }
  }
  if (nc > 1) __syncthreads();
  if (wave != 0) return;
  RowState<DH> st;
  st.init();
  fold_chunk<DH>(c0, lane, st);
  for (int j = 1; j < nc; ++j) {
    ChunkOut<DH> c;
    c.m = s_c[j].m;
    c.l = s_c[j].l;
    if (lane < 32) {
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        c.o[i][0] = s_c[j].o[i][lane][0];
        c.o[i][1] = s_c[j].o[i][lane][1];
      }
    }
    fold_chunk<DH>(c, lane, st);
  }
  AT* out = static_cast<AT*>(a.out);
  if (a.out_feed) {
    const int K = a.H * DH;
    row_output<AT, DH>(st, out, [&](int d) { return feed_index<Mma<AT>::KS, Mma<AT>::EPL>(row, hh * DH + d, K); },
                       lane);
  } else {
    const size_t ob = static_cast<size_t>(row) * a.ldo + hh * DH;
    row_output<AT, DH>(st, out, [&](int d) { return ob + d; }, lane);
  }
}

// ---------------------------------------------------------------------------
// Token embedding x = E[tok] * scale + PE(pos), PE the interleaved sinusoid
// (columns 2i, 2i+1 = sin, cos of pos * 10000^(-2i/d)), evaluated in double
// and rounded to float once per context into a table (k_pe_table), so that
// embedding a row costs two loads per element instead of double-precision
// transcendentals.
__global__ __launch_bounds__(256) void k_pe_table(float* pe, int n_pos, int d) {
  const size_t total = static_cast<size_t>(n_pos) * d;
  for (size_t t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int p = static_cast<int>(t / d);
    const int c = static_cast<int>(t - static_cast<size_t>(p) * d);
    const double freq = exp(-log(10000.0) * static_cast<double>(c & ~1) / d);
    const double ang = static_cast<double>(p) * freq;
    pe[t] = static_cast<float>((c & 1) ? cos(ang) : sin(ang));
  }
}

template <typename WT>
__device__ __forceinline__ float embed_elem(const WT* emb, const float* pe, int tok, int p, int c, int d, float scale,
                                            int vocab) {
  tok = min(max(tok, 0), vocab - 1);
  return Elt<WT>::load(emb, static_cast<size_t>(tok) * d + c) * scale + pe[static_cast<size_t>(p) * d + c];
}

// Embedding of `total` rows into x_out [total][d] by the threads of one
// workgroup (d a multiple of 8): each item is 8 consecutive columns of a row,
// and a thread issues the loads of up to kEmbItems items before computing any
// (the per-element value is embed_elem's: E[tok] * scale + pe, in that order).
// tok(row) / pos(row) give a row's token and position.
constexpr int kEmbItems = 4;
template <typename WT, typename Tok, typename Pos>
__device__ __forceinline__ void embed_rows_block(const WT* emb, const float* pe, float scale, int d, int vocab,
                                                 int total, Tok tok, Pos pos, WT* x_out) {
  const int per_row = d / 8;
  const int n_items = total * per_row;
  const int nt = blockDim.x;
  for (int base = 0; base < n_items; base += kEmbItems * nt) {
    float ev[kEmbItems][8], pv[kEmbItems][8];
#pragma unroll
    for (int u = 0; u < kEmbItems; ++u) {
      const int it = base + threadIdx.x + u * nt;
      const int itc = it < n_items ? it : 0;
      const int row = itc / per_row;
      const int c = (itc - row * per_row) * 8;
      const int t = min(max(tok(row), 0), vocab - 1);
      load_n<WT, 8>(emb, static_cast<size_t>(t) * d + c, ev[u]);
      load_n<float, 8>(pe, static_cast<size_t>(pos(row)) * d + c, pv[u]);
    }
#pragma unroll
    for (int u = 0; u < kEmbItems; ++u) {
      const int it = base + threadIdx.x + u * nt;
      if (it < n_items) {
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = ev[u][e] * scale + pv[u][e];
        store8<WT>(x_out, static_cast<size_t>(it) * 8, y);
      }
    }
  }
}

template <typename WT>
__global__ __launch_bounds__(256) void k_embed(EmbedArgs a) {
  if (blockIdx.x == 0 && a.len_out != nullptr)
    for (int i = threadIdx.x; i < a.n_len; i += blockDim.x) a.len_out[i] = a.len_in[i];
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  const size_t total = static_cast<size_t>(R) * a.d;
  for (size_t t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int row = static_cast<int>(t / a.d);
    const int c = static_cast<int>(t - static_cast<size_t>(row) * a.d);
    int s, p;
    row_place(a.rows, row, s, p);
    Elt<WT>::store(static_cast<WT*>(a.out), t,
                   embed_elem<WT>(static_cast<const WT*>(a.emb), a.pe, a.tok[row], p, c, a.d, a.scale, a.vocab));
  }
}

// ---------------------------------------------------------------------------
// Row LayerNorm, one wave per row, with the statistics and element split of
// the LayerNorm prologue of the products (ln_row_stats, ln_row_apply), so a
// row is normalised bitwise alike here and there.
template <typename WT, typename XT, int NT>
__global__ __launch_bounds__(256) void k_ln(LnArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + threadIdx.x / kWave;
  const int R = a.n_rows_dev ? *a.n_rows_dev : a.n_rows;
  if (row >= R) return;   // whole wave
  LnRow<XT, NT> h;
  ln_row_load<XT, NT>(h, static_cast<const XT*>(a.x) + static_cast<size_t>(row) * a.d, a.d, lane, true);
  float mean, rstd;
  ln_row_stats<XT, NT>(h, a.d, a.eps, mean, rstd);
  ln_row_apply<WT, XT, NT>(h, a.d, mean, rstd, static_cast<const WT*>(a.g), static_cast<const WT*>(a.b),
                           static_cast<WT*>(a.out) + static_cast<size_t>(row) * a.d, nullptr, lane);
}

// Largest logit and log-sum-exp of each row from the vocabulary kernel's
// per-workgroup (max, sum of exp(logit - max)) pairs: one wave per row, lane
// l merging the pairs l, l + 64, ... in order, then the lanes as a fixed tree.
__global__ __launch_bounds__(256) void k_lse_reduce(const float2* part, int part_ld, int n_parts,
                                                    const int* n_rows_dev, int R_max, float* row_max,
                                                    float* row_lse) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + static_cast<int>(threadIdx.x / kWave);
  const int R = n_rows_dev ? *n_rows_dev : R_max;
  if (row >= R) return;   // wave-uniform
  const float2* p = part + static_cast<size_t>(row) * part_ld;
  float m = -INFINITY, sm = 0.f;
  for (int q = lane; q < n_parts; q += kWave) lse_merge(m, sm, p[q].x, p[q].y);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const float m2 = __shfl_xor(m, off), s2 = __shfl_xor(sm, off);
    lse_merge(m, sm, m2, s2);
  }
  if (lane == 0) {
    row_max[row] = m;
    row_lse[row] = m + logf(sm);
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
// The control step's sequence number (thread 0 only): the context's counter
// of control steps, advanced (k_ctrl_init sets it to the host's count, seq0).
__device__ __forceinline__ int next_seq(const CtrlArgs& a, bool init) {
  if (a.seq == nullptr) return 0;
  const int q = (init ? a.seq0 : *a.seq + 1) & kSeqMask;
  *a.seq = q;
  return q;
}

// Publishes "no rows" for a control step that finds the decode finished.
__device__ __forceinline__ void publish_done(const CtrlArgs& a) {
  if (threadIdx.x == 0 && a.host_rows != nullptr)
    __hip_atomic_store(a.host_rows, host_word(0, false, next_seq(a, false)), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

template <typename WT>
__device__ void emit_rows(const CtrlArgs& a, bool init) {
  __shared__ int s_total, s_near;
  if (threadIdx.x == 0) {
    int acc = 0;
    bool near = true;
    for (int s = 0; s < a.B; ++s) {
      a.st[s].row0 = acc;
      acc += a.st[s].done ? 0 : a.st[s].L;
      near = near && near_end(a.st[s], a.stop_prefix);
    }
    s_total = acc;
    s_near = near ? 1 : 0;
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
    if (a.rows_total != nullptr) *a.rows_total += static_cast<unsigned long long>(total);
    if (a.host_rows != nullptr)
      __hip_atomic_store(a.host_rows, host_word(total, s_near != 0, next_seq(a, init)), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (a.x_out != nullptr) {
    __syncthreads();
    embed_rows_block<WT>(static_cast<const WT*>(a.emb), a.pe, a.emb_scale, a.d, a.vocab, total,
                         [&](int r) { return a.row_tok[r]; }, [&](int r) { return a.row_pos[r]; },
                         static_cast<WT*>(a.x_out));
  }
}

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_init(CtrlArgs a, InlineLens lens) {
  if (a.reset_trace_count && threadIdx.x == 0) *a.trace_count = 0ull;
  const int* tgt_m = lens.n > 0 ? lens.v : a.tgt_m;
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    const int m = tgt_m[s];
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
  }
  // InitT: the caller's draft over the m positions, else all [PAD]; one
  // (sentence, position) item per thread and step
  const long long n_y = static_cast<long long>(a.B) * a.ldy;
  for (long long i = threadIdx.x; i < n_y; i += blockDim.x) {
    const int s = static_cast<int>(i / a.ldy);
    const int t = static_cast<int>(i - static_cast<long long>(s) * a.ldy);
    a.y[i] = (a.init != nullptr && t < tgt_m[s]) ? a.init[static_cast<size_t>(s) * a.init_ld + t] : a.pad_id;
  }
  __syncthreads();
  emit_rows<WT>(a, true);
}

// Best entry of a set of argmax partials.
struct Best {
  uint32_t key;   // float_key of the logit (0: none)
  uint32_t idx;   // token index, bit 31 set if a non-finite logit was seen
};

// (larger key, then lower index) wins; the non-finite bits are or-ed.  The
// order of combination does not change the result.
__device__ __forceinline__ void best_merge(uint32_t& bk, uint32_t& bi, uint32_t& nf, uint32_t k2, uint32_t raw) {
  nf |= raw >> 31;
  best_take(bk, bi, k2, raw & 0x7fffffffu);
}

// Best over partials p[t0 .. t1) by one wave, eight loads per lane in flight.
__device__ __forceinline__ Best reduce_span(const uint2* p, int t0, int t1, int lane) {
  uint32_t bk = 0, bi = 0x7fffffffu, nf = 0;
  for (int t = t0 + lane; t < t1; t += 8 * kWave) {
    uint2 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = t + u * kWave < t1 ? p[t + u * kWave] : make_uint2(0u, 0x7fffffffu);
#pragma unroll
    for (int u = 0; u < 8; ++u) best_merge(bk, bi, nf, v[u].x, v[u].y);
  }
  group16_best(bk, bi);
  nf = group16_or(nf);
  // the four rows of 16 lanes (all lanes are active here)
  uint32_t rk = __builtin_amdgcn_readlane(bk, 0), ri = __builtin_amdgcn_readlane(bi, 0);
  uint32_t rf = __builtin_amdgcn_readlane(nf, 0);
#pragma unroll
  for (int r = 16; r < kWave; r += 16) {
    best_take(rk, ri, __builtin_amdgcn_readlane(bk, r), __builtin_amdgcn_readlane(bi, r));
    rf |= __builtin_amdgcn_readlane(nf, r);
  }
  return Best{rk, ri | (rf << 31)};
}

// Argmax of each of R rows over the per-workgroup partials of the fused
// vocabulary kernel (largest logit, lowest index on exact ties).  All waves of
// the workgroup take part: a row's partials are split into S spans (S waves
// per row, S = waves / R when R < waves), combined through LDS.  Ends with
// the workgroup synchronised.
__device__ void reduce_rows(const uint2* partials, int part_ld, int n_parts, int R, int* new_tok, int* row_flags) {
  __shared__ Best s_best[32];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;                 // <= 32
  const int S = R < nw ? nw / R : 1;                 // spans per row
  const int rows_per_round = nw / S;
  for (int row0 = 0; row0 < R; row0 += rows_per_round) {
    const int row = row0 + wave / S;
    const int span = wave - (wave / S) * S;
    if (wave < rows_per_round * S && row < R) {
      const Best b = reduce_span(partials + static_cast<size_t>(row) * part_ld, (n_parts * span) / S,
                                 (n_parts * (span + 1)) / S, lane);
      if (lane == 0) s_best[wave] = b;
    }
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < rows_per_round && row0 + static_cast<int>(threadIdx.x) < R) {
      uint32_t bk = 0, bi = 0x7fffffffu, nf = 0;
      for (int j = 0; j < S; ++j) best_merge(bk, bi, nf, s_best[threadIdx.x * S + j].key, s_best[threadIdx.x * S + j].idx);
      const bool none = bk == 0;                     // no finite logit in the row
      new_tok[row0 + threadIdx.x] = none ? 0 : static_cast<int>(bi);
      row_flags[row0 + threadIdx.x] = (nf || none) ? 1 : 0;
    }
    __syncthreads();
  }
}

// State transition of a sentence after an iteration of its block: lead =
// the number of leading block positions the iteration left unchanged (L: the
// whole block, so Eq. (3) holds), first_eos = the block position of the first
// [EOS] among the new values (L: none), nf = a non-finite logit was seen.
// Eq. (3) commits the block when it is unchanged or after its L-th iteration
// (then exact); the prefix stopping condition commits, every iteration, the
// positions the iteration proved exact: all L when unchanged, else the lead
// unchanged ones and the next (their inputs were already exact).  An [EOS]
// ends PD_AR / PD_HYBRID decoding once it is among the committed positions.
__device__ __forceinline__ void advance_state(const CtrlArgs& a, SentState& st, int lead, int first_eos, int nf) {
  if (nf) st.flags |= FLAG_NONFINITE;
  st.k += 1;
  st.j += 1;
  int commit = 0;
  if (a.stop_prefix) commit = lead >= st.L ? st.L : lead + 1;
  else if (lead >= st.L || st.j >= st.L) commit = st.L;
  if (commit > 0) {
    if ((a.mode == MODE_AR || a.mode == MODE_HYBRID) && first_eos < commit) {
      st.done = 1;
      st.flags |= FLAG_CONVERGED | FLAG_EOS;
    }
    if (!st.done) {
      st.i += commit;
      st.j = 0;
      if (st.i >= st.m) { st.done = 1; st.flags |= FLAG_CONVERGED; }
      else st.L = block_len(a, st.i, st.m);
    }
  }
  const int cap = a.max_iters > 0 ? a.max_iters : st.m;
  if (!st.done && st.k >= cap) { st.done = 1; st.flags |= FLAG_MAX_ITERS; }
  if (st.done) st.L = 0;
}

// Trace record of row `row` of the iteration (the caller's buffer keeps the
// first trace_cap records; the count keeps growing).
__device__ __forceinline__ void trace_row(const CtrlArgs& a, unsigned long long base, int row, int it, int s, int p,
                                          int tok) {
  const unsigned long long idx = base + static_cast<unsigned long long>(row);
  if (idx < static_cast<unsigned long long>(a.trace_cap))
    a.trace[idx] = TraceRec{it, s, p, tok, a.row_max[row], a.row_lse[row]};
}

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_step(CtrlArgs a) {
  const int R = *a.n_rows;
  if (R == 0) {                          // workgroup-uniform: the decode had already finished
    publish_done(a);
    return;
  }
  if (a.partials != nullptr)
    reduce_rows(a.partials, a.part_ld, a.n_parts, R, const_cast<int*>(a.new_tok), const_cast<int*>(a.row_flags));
  for (int s = threadIdx.x; s < a.B; s += blockDim.x) {
    SentState st = a.st[s];
    if (st.done) continue;
    int* y = a.y + static_cast<size_t>(s) * a.ldy;
    int lead = 0, first_eos = st.L, nf = 0;
    for (int r = 0; r < st.L; ++r) {
      const int t = a.new_tok[st.row0 + r];
      nf |= a.row_flags[st.row0 + r];
      if (lead == r && y[st.i + r] == t) lead = r + 1;
      if (first_eos == st.L && t == a.eos_id) first_eos = r;
      y[st.i + r] = t;
      if (a.trace != nullptr) trace_row(a, *a.trace_count, st.row0 + r, st.k + 1, s, st.i + r, t);
    }
    advance_state(a, st, lead, first_eos, nf);
    a.st[s] = st;
  }
  __syncthreads();
  if (a.trace != nullptr && threadIdx.x == 0) *a.trace_count += static_cast<unsigned long long>(R);
  emit_rows<WT>(a, false);
}

// The control step with one thread per row instead of one per sentence (up
// to 1024 sentences; k_ctrl_step above is the fallback for more): the rows'
// loads go out together rather than one block position after another.  The
// per-sentence results (the first changed block position, the first [EOS],
// a non-finite logit) are gathered with LDS atomic minima / ORs, the states
// advance exactly as in k_ctrl_step
// (advance_state), the next layout's first rows come from a prefix sum over
// the sentences, and the next rows are written one thread per row.
constexpr int kCtrlRowsMaxB = 1024;

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_rows(CtrlArgs a) {
  __shared__ int s_nf[kCtrlRowsMaxB];          // a non-finite logit in the sentence's rows
  __shared__ int s_chg[kCtrlRowsMaxB];         // first changed block position (or a large value)
  __shared__ int s_eos[kCtrlRowsMaxB];         // first [EOS] block position (or a large value)
  __shared__ int s_k[kCtrlRowsMaxB];           // iterations so far (trace)
  __shared__ int s_i[kCtrlRowsMaxB];           // current, then next block start
  __shared__ int s_scan[2][kCtrlRowsMaxB + 1]; // next block lengths -> first rows (exclusive prefix)
  __shared__ int s_far;                        // some live sentence is not near its end (near_end)
  const int tid = threadIdx.x;
  const int R = *a.n_rows;
  if (R == 0) {                                // workgroup-uniform: the decode had already finished
    publish_done(a);
    return;
  }
  if (tid == 0) s_far = 0;
  if (a.partials != nullptr)
    reduce_rows(a.partials, a.part_ld, a.n_parts, R, const_cast<int*>(a.new_tok), const_cast<int*>(a.row_flags));
  SentState st;
  const bool sent = tid < a.B;
  if (sent) {
    st = a.st[tid];
    s_nf[tid] = 0;
    s_chg[tid] = s_eos[tid] = 0x7fffffff;
    s_k[tid] = st.k;
    s_i[tid] = st.i;
  }
  __syncthreads();
  const unsigned long long tbase = a.trace != nullptr ? *a.trace_count : 0ull;
  for (int row = tid; row < R; row += blockDim.x) {
    const int s = a.row_sent[row], p = a.row_pos[row];
    const int t = a.new_tok[row];
    int* yp = a.y + static_cast<size_t>(s) * a.ldy + p;
    const int r = p - s_i[s];                   // block position of the row
    if (*yp != t) atomicMin(&s_chg[s], r);
    if (t == a.eos_id) atomicMin(&s_eos[s], r);
    if (a.row_flags[row] != 0) atomicOr(&s_nf[s], 1);
    *yp = t;
    if (a.trace != nullptr) trace_row(a, tbase, row, s_k[s] + 1, s, p, t);
  }
  __syncthreads();
  int len = 0;
  if (sent) {
    if (!st.done) advance_state(a, st, min(s_chg[tid], st.L), min(s_eos[tid], st.L), s_nf[tid]);
    if (!near_end(st, a.stop_prefix)) s_far = 1;
    len = st.done ? 0 : st.L;
    s_i[tid] = st.i;
    s_scan[0][tid + 1] = len;
  }
  if (tid == 0) s_scan[0][0] = 0;
  __syncthreads();
  // inclusive scan of s_scan[.][1..B] (Hillis-Steele), s_scan[.][0] = 0
  int src = 0;
  for (int off = 1; off < a.B; off <<= 1) {
    if (tid < a.B) {
      const int v = s_scan[src][tid + 1];
      s_scan[src ^ 1][tid + 1] = tid >= off ? v + s_scan[src][tid + 1 - off] : v;
    }
    if (tid == 0) s_scan[src ^ 1][0] = 0;
    __syncthreads();
    src ^= 1;
  }
  const int* first = s_scan[src];               // first[s] = first row of sentence s, first[B] = total
  if (sent) {
    st.row0 = first[tid];
    a.st[tid] = st;
  }
  const int total = first[a.B];
  for (int row = tid; row < total; row += blockDim.x) {
    int lo = 0, hi = a.B - 1;                    // the sentence s with first[s] <= row < first[s + 1]
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (first[mid] <= row) lo = mid;
      else hi = mid - 1;
    }
    const int p = s_i[lo] + (row - first[lo]);
    a.row_sent[row] = lo;
    a.row_pos[row] = p;
    a.row_tok[row] = p == 0 ? a.bos_id : a.y[static_cast<size_t>(lo) * a.ldy + p - 1];
  }
  if (tid == 0) {
    if (a.trace != nullptr) *a.trace_count += static_cast<unsigned long long>(R);
    *a.n_rows = total;
    if (a.rows_total != nullptr) *a.rows_total += static_cast<unsigned long long>(total);
    if (a.host_rows != nullptr)
      __hip_atomic_store(a.host_rows, host_word(total, s_far == 0, next_seq(a, false)), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (a.x_out != nullptr) {
    __syncthreads();
    embed_rows_block<WT>(static_cast<const WT*>(a.emb), a.pe, a.emb_scale, a.d, a.vocab, total,
                         [&](int r) { return a.row_tok[r]; }, [&](int r) { return a.row_pos[r]; },
                         static_cast<WT*>(a.x_out));
  }
}

// The control step of iterations of at most 64 rows (so at most 64
// sentences and blocks of at most 64 positions), with everything that does
// not leave the workgroup kept in LDS: the sentence states, the new tokens,
// a window of each sentence's draft and the next rows.  Its global-memory
// round trips are (1) states and row count, (2) the draft windows together
// with the argmax partials, (3) the embedding rows of the next tokens,
// against about seven in k_ctrl_step; the transitions are the same
// (advance_state).
//
// The window of sentence s is y[i - 1 .. i + 126] around its current block
// [i, i + L): the token before the block, the block's previous values and the
// draft after it.  Every position the next rows read as input lies in it:
// the next block starts at most L <= 64 positions later and holds at most 64.
// All 1024 threads load it, (sentence, offset) items 8 per thread, with every
// load in flight before the first wait.
constexpr int kCtrlSmallMax = 64;
constexpr int kCtrlWindow = 2 * kCtrlSmallMax;
constexpr int kCtrlSmallThreads = 1024;

template <typename WT>
__global__ __launch_bounds__(1024) void k_ctrl_small(CtrlArgs a) {
  __shared__ SentState s_st[kCtrlSmallMax];
  __shared__ int s_tok[kCtrlSmallMax], s_flag[kCtrlSmallMax];
  __shared__ int s_rpos[kCtrlSmallMax], s_rtok[kCtrlSmallMax];
  __shared__ int s_win[kCtrlSmallMax][kCtrlWindow];   // s_win[s][r] = y_s[i_s - 1 + r]
  __shared__ int s_total;
  constexpr int kItems = kCtrlSmallMax * kCtrlWindow / kCtrlSmallThreads;
  const int tid = threadIdx.x;
  const bool sent = tid < a.B;
  // (1) states and the row count (and the running row total, read here so
  // that its update below waits for no load)
  SentState st;
  if (sent) {
    st = a.st[tid];
    s_st[tid] = st;
  }
  const int R = *a.n_rows;
  const unsigned long long rows_done = tid == 0 && a.rows_total != nullptr ? *a.rows_total : 0ull;
  __syncthreads();
  // (2) the draft windows (positions clamped into the row; values outside
  // [0, m) are never used), then the argmax partials of every row the launch
  // may hold (rows past the device count are reduced too and ignored): the
  // reduction's wait covers both
  int wv[kItems];
#pragma unroll
  for (int u = 0; u < kItems; ++u) {
    const int it = tid + kCtrlSmallThreads * u;
    const int s = it / kCtrlWindow < a.B ? it / kCtrlWindow : 0;
    const int p = min(max(s_st[s].i - 1 + it % kCtrlWindow, 0), a.ldy - 1);
    wv[u] = a.y[static_cast<size_t>(s) * a.ldy + p];
  }
  reduce_rows(a.partials, a.part_ld, a.n_parts, a.R_max, s_tok, s_flag);   // ends synchronised
#pragma unroll
  for (int u = 0; u < kItems; ++u) {
    const int it = tid + kCtrlSmallThreads * u;
    if (it / kCtrlWindow < a.B) s_win[it / kCtrlWindow][it % kCtrlWindow] = wv[u];
  }
  __syncthreads();
  if (R == 0) {                                // workgroup-uniform: the decode had already finished
    publish_done(a);
    return;
  }
  int i_old = 0, row0_old = 0, L_old = 0;
  if (sent && !st.done) {
    int* y = a.y + static_cast<size_t>(tid) * a.ldy;
    int lead = 0, first_eos = st.L, nf = 0;
    const unsigned long long tbase = a.trace != nullptr ? *a.trace_count : 0ull;
    for (int r = 0; r < st.L; ++r) {
      const int t = s_tok[st.row0 + r];
      nf |= s_flag[st.row0 + r];
      if (lead == r && s_win[tid][1 + r] == t) lead = r + 1;   // previous value y[i + r]
      if (first_eos == st.L && t == a.eos_id) first_eos = r;
      y[st.i + r] = t;
      if (a.trace != nullptr) trace_row(a, tbase, st.row0 + r, st.k + 1, tid, st.i + r, t);
    }
    i_old = st.i;
    row0_old = st.row0;
    L_old = st.L;
    advance_state(a, st, lead, first_eos, nf);
  }
  if (sent) s_st[tid] = st;
  __syncthreads();
  if (tid == 0) {
    if (a.trace != nullptr) *a.trace_count += static_cast<unsigned long long>(R);
    int acc = 0;
    bool near = true;
    for (int s = 0; s < a.B; ++s) {
      s_st[s].row0 = acc;
      acc += s_st[s].done ? 0 : s_st[s].L;
      near = near && near_end(s_st[s], a.stop_prefix);
    }
    s_total = acc;
    *a.n_rows = acc;
    if (a.rows_total != nullptr) *a.rows_total = rows_done + static_cast<unsigned long long>(acc);
    if (a.host_rows != nullptr)
      __hip_atomic_store(a.host_rows, host_word(acc, near, next_seq(a, false)), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
  }
  __syncthreads();
  // the next rows: sentence order, block order; the shifted-left input of
  // position p is [BOS] at p = 0, else y[p - 1]: the value just written, the
  // token before the old block, or the draft past the old block
  if (sent) {
    st = s_st[tid];
    a.st[tid] = st;
    for (int r = 0; r < st.L; ++r) {
      const int row = st.row0 + r;
      const int p = st.i + r;
      int tok;
      if (p == 0) tok = a.bos_id;
      else if (p - 1 < i_old || p - 1 >= i_old + L_old) tok = s_win[tid][p - i_old];   // y[p - 1], unchanged
      else tok = s_tok[row0_old + (p - 1 - i_old)];
      s_rpos[row] = p;
      s_rtok[row] = tok;
      a.row_sent[row] = tid;
      a.row_pos[row] = p;
      a.row_tok[row] = tok;
    }
  }
  __syncthreads();
  // (3) the embedding of the next rows (tokens and positions from LDS)
  embed_rows_block<WT>(static_cast<const WT*>(a.emb), a.pe, a.emb_scale, a.d, a.vocab, s_total,
                       [&](int r) { return s_rtok[r]; }, [&](int r) { return s_rpos[r]; },
                       static_cast<WT*>(a.x_out));
}

// Outputs: ids cut after the first [EOS] (inclusive) and [PAD]-filled, the
// output length, the iteration count k and the flags of each sentence.
__global__ __launch_bounds__(256) void k_finalize(CtrlArgs a) {
  // one wave per sentence; lanes stride over the positions
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  for (int s = blockIdx.x * 4 + wave; s < a.B; s += gridDim.x * 4) {
    const SentState st = a.st[s];
    const int* y = a.y + static_cast<size_t>(s) * a.ldy;
    int first = st.m;                        // first [EOS] at or after this lane's positions
    for (int t = lane; t < st.m; t += kWave)
      if (y[t] == a.eos_id) { first = t; break; }
    // wave minimum (DPP within rows of 16, then across the four rows)
    first = min(first, __builtin_amdgcn_mov_dpp(first, kDppXor1, 0xF, 0xF, false));
    first = min(first, __builtin_amdgcn_mov_dpp(first, kDppXor2, 0xF, 0xF, false));
    first = min(first, __builtin_amdgcn_mov_dpp(first, kDppHalfMirror, 0xF, 0xF, false));
    first = min(first, __builtin_amdgcn_mov_dpp(first, kDppMirror, 0xF, 0xF, false));
    first = min(min(__builtin_amdgcn_readlane(first, 0), __builtin_amdgcn_readlane(first, 16)),
                min(__builtin_amdgcn_readlane(first, 32), __builtin_amdgcn_readlane(first, 48)));
    const int len = first < st.m ? first + 1 : st.m;
    for (int t = lane; t < a.out_ld; t += kWave)
      a.out_ids[static_cast<size_t>(s) * a.out_ld + t] = (t < len && t < a.ldy) ? y[t] : a.pad_id;
    if (lane == 0) {
      a.out_len[s] = len;
      a.out_k[s] = st.k;
      a.out_flags[s] = st.flags;
    }
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_argmax_reduce(ReduceArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + threadIdx.x / kWave;
  if (row >= *a.n_rows_dev) return;
  const Best b = reduce_span(a.partials + static_cast<size_t>(row) * a.part_ld, 0, a.n_parts, lane);
  if (lane == 0) {
    const bool none = b.key == 0;
    a.new_tok[row] = none ? 0 : static_cast<int>(b.idx & 0x7fffffffu);
    a.row_flags[row] = ((b.idx >> 31) || none) ? 1 : 0;
  }
}

template <typename AT, int W, int ONE>
static hipError_t launch_attn_split(const AttnArgs& a, int grid, hipStream_t s) {
  switch (a.dh) {
    case 16: hipLaunchKernelGGL((k_attn_split<AT, 16, W, ONE>), dim3(grid), dim3(W * kWave), 0, s, a); break;
    case 32: hipLaunchKernelGGL((k_attn_split<AT, 32, W, ONE>), dim3(grid), dim3(W * kWave), 0, s, a); break;
    case 64: hipLaunchKernelGGL((k_attn_split<AT, 64, W, ONE>), dim3(grid), dim3(W * kWave), 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn_split<AT, 128, W, ONE>), dim3(grid), dim3(W * kWave), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Launches whose rows may have more than one chunk of keys (by the host's
// bound) evaluate a row's chunks on kAttnSplitWaves waves side by side
// (k_attn_split); the others keep one wave per (row, head), which is faster
// for rows of one chunk.  Both give bitwise the same rows.  Two waves
// measured best at every row count (four: the same at batch 1, slower above
// 64 rows).
constexpr int kAttnSplitWaves = 2;

template <typename AT, int ONE>
static hipError_t launch_attn_f(const AttnArgs& a, int grid, hipStream_t s) {
  if (a.max_keys > kAttnChunk) return launch_attn_split<AT, kAttnSplitWaves, ONE>(a, a.rows_max * a.H, s);
  switch (a.dh) {
    case 16: hipLaunchKernelGGL((k_attn<AT, 16, ONE>), dim3(grid), dim3(kAttnRows * kWave), 0, s, a); break;
    case 32: hipLaunchKernelGGL((k_attn<AT, 32, ONE>), dim3(grid), dim3(kAttnRows * kWave), 0, s, a); break;
    case 64: hipLaunchKernelGGL((k_attn<AT, 64, ONE>), dim3(grid), dim3(kAttnRows * kWave), 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn<AT, 128, ONE>), dim3(grid), dim3(kAttnRows * kWave), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename AT>
static hipError_t launch_attn_t(const AttnArgs& a, int grid, hipStream_t s) {
  return a.one_source ? launch_attn_f<AT, 1>(a, grid, s) : launch_attn_f<AT, 0>(a, grid, s);
}

hipError_t launch_attn(int dtype, const AttnArgs& args, int R_max, hipStream_t s) {
  if (args.dh > kMaxHeadDim || args.T > kMaxKeys) return hipErrorInvalidValue;
  if (args.one_source && (args.causal || args.klen == nullptr)) return hipErrorInvalidValue;
  const int grid = (R_max + kAttnRows - 1) / kAttnRows * args.H;
  if (grid == 0) return hipSuccess;
  AttnArgs a = args;
  a.rows_max = R_max;
  return dtype == DT_BF16 ? launch_attn_t<bf16_t>(a, grid, s) : launch_attn_t<float>(a, grid, s);
}

hipError_t launch_lse_reduce(const float2* part, int part_ld, int n_parts, const int* n_rows_dev, int R_max,
                             float* row_max, float* row_lse, hipStream_t s) {
  if (R_max <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_lse_reduce, dim3((R_max + 3) / 4), dim3(256), 0, s, part, part_ld, n_parts, n_rows_dev, R_max,
                     row_max, row_lse);
  return hipGetLastError();
}

hipError_t launch_pe_table(float* pe, int n_pos, int d, hipStream_t s) {
  const size_t total = static_cast<size_t>(n_pos) * d;
  const int grid = static_cast<int>(std::min<size_t>((total + 255) / 256, 4096));
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pe_table, dim3(grid), dim3(256), 0, s, pe, n_pos, d);
  return hipGetLastError();
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
  const int grid = (R_max + 3) / 4;
  if (grid == 0) return hipSuccess;
  if (a.d % 8 != 0 || a.d > 1024) return hipErrorInvalidValue;
  if (dtype == DT_BF16) {
    if (a.d > 512) {
      if (a.x_f32) hipLaunchKernelGGL((k_ln<bf16_t, float, 2>), dim3(grid), dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_ln<bf16_t, bf16_t, 2>), dim3(grid), dim3(256), 0, s, a);
    } else {
      if (a.x_f32) hipLaunchKernelGGL((k_ln<bf16_t, float, 1>), dim3(grid), dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_ln<bf16_t, bf16_t, 1>), dim3(grid), dim3(256), 0, s, a);
    }
  } else {
    if (a.d > 512) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_ln<float, float, 1>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_argmax_reduce(const ReduceArgs& a, int R_max, hipStream_t s) {
  if (R_max <= 0) return hipSuccess;
  const int grid = (R_max + 3) / 4;
  hipLaunchKernelGGL(k_argmax_reduce, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ctrl_init(int dtype, const CtrlArgs& a, const InlineLens& lens, hipStream_t s) {
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_init<bf16_t>, dim3(1), dim3(1024), 0, s, a, lens);
  else hipLaunchKernelGGL(k_ctrl_init<float>, dim3(1), dim3(1024), 0, s, a, lens);
  return hipGetLastError();
}

hipError_t launch_ctrl_step(int dtype, const CtrlArgs& a, hipStream_t s) {
  const bool small = a.partials != nullptr && a.x_out != nullptr && a.R_max <= kCtrlSmallMax && a.B <= kCtrlSmallMax;
  if (small) {
    if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_small<bf16_t>, dim3(1), dim3(kCtrlSmallThreads), 0, s, a);
    else hipLaunchKernelGGL(k_ctrl_small<float>, dim3(1), dim3(kCtrlSmallThreads), 0, s, a);
    return hipGetLastError();
  }
  if (a.B <= kCtrlRowsMaxB) {
    if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_rows<bf16_t>, dim3(1), dim3(1024), 0, s, a);
    else hipLaunchKernelGGL(k_ctrl_rows<float>, dim3(1), dim3(1024), 0, s, a);
    return hipGetLastError();
  }
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_ctrl_step<bf16_t>, dim3(1), dim3(1024), 0, s, a);
  else hipLaunchKernelGGL(k_ctrl_step<float>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_finalize(const CtrlArgs& a, hipStream_t s) {
  const int grid = std::max(1, std::min((a.B + 3) / 4, 256));
  hipLaunchKernelGGL(k_finalize, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pdec

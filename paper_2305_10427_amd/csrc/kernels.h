// Internal launch interface between the host runtime and the HIP kernels.
// Nothing here crosses the public C ABI (include/pdec.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdec {

enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Where row r of an activation matrix lives: sentence s and input position p.
// With sent == nullptr the rows are laid out densely, s = r / per_sent, p = r % per_sent.
struct RowMap {
  const int* sent;
  const int* pos;
  int per_sent;
};

// Element offset of x[r][k] in the MFMA feed order of a [rows][K] matrix
// (KS, EPL: the MFMA step and elements per lane of the storage type):
// 16-row tile r / 16, step k / KS, lane (r mod 16) + 16 ((k mod KS) / EPL).
template <int KS, int EPL>
__host__ __device__ __forceinline__ size_t feed_index(int r, int k, int K) {
  const int s = k / KS, kk = k - s * KS;
  return ((static_cast<size_t>(r >> 4) * (K / KS) + s) * 64 + (r & 15) + 16 * (kk / EPL)) * EPL + (kk % EPL);
}

// (sentence, position) of row `row`.
__device__ __forceinline__ void row_place(const RowMap& m, int row, int& s, int& p) {
  if (m.sent != nullptr) { s = m.sent[row]; p = m.pos[row]; }
  else { s = row / m.per_sent; p = row - s * m.per_sent; }
}

enum Prologue { PRO_NONE = 0, PRO_LN = 1 };
enum Epilogue {
  EPI_F32 = 0,     // out_f32 = acc + bias
  EPI_ACT = 1,     // out (storage type) = act(acc + bias)
  EPI_RESID = 2,   // out_f32 or out = acc + bias + resid
  EPI_QKV = 3,     // cols [0,q_cols) -> out_f32; next d -> K cache; next d -> V cache
  EPI_ARGMAX = 4,  // logits = scale * acc + bias, reduced to a per-(row, workgroup) best
  EPI_LOGITS = 5,  // out_f32 = scale * acc + bias (verification only)
};

constexpr int kMaxLayers = 16;   // layers of one multi-layer product launch

struct GemmArgs {
  const int* n_rows_dev;   // row count read on device (nullptr: n_rows is exact)
  int n_rows;              // launch bound on the rows (rows >= the device count are discarded)
  int mt_per_wg;           // 16-row tiles per workgroup row (grid.y = ceil(tiles / mt_per_wg))
  // input rows [R][ldx]; element type float if x_f32 else the storage type
  const void* x;
  int ldx;
  int x_f32;
  // 1: x (storage type, no LayerNorm prologue) is in the MFMA feed order of
  // the K-split kernels instead: 16-row tile t, step s: 64 16-byte words,
  // word l = x[16 t + (l & 15)][s KS + EPL (l >> 4) ...] (see feed_index)
  int x_feed;
  int out_feed;            // EPI_ACT: out (storage type, [rows][N]) written in that feed order
  // LayerNorm prologue (PRO_LN): x <- LN(x) * g + b, rounded to the storage type
  const void* ln_g;
  const void* ln_b;
  float ln_eps;
  void* ln_out;            // optional: workgroup 0 writes the normalised rows here
  int ldlo;
  // weights W[N][K] row-major (storage type), bias[N]
  const void* w;
  const void* bias;
  int N, K;
  // epilogues
  float* out_f32;
  void* out;
  int ldo;
  const void* resid;       // residual, storage type (EPI_RESID)
  int ldr;
  int act;                 // 1 relu, 2 gelu (EPI_ACT)
  int q_cols;              // EPI_QKV
  void* kc;                // EPI_QKV: K / V caches [S][H][T][dh] of one layer
  void* vc;
  int H, dh, T, d;
  RowMap rows;
  float logit_scale;       // EPI_ARGMAX
  uint2* partials;         // [row][part_ld] = (order key of best logit, index | nonfinite << 31)
  int part_ld;
  // argmax epilogues, optional: [row][part_ld] = (max, sum of exp(logit - max))
  // over the same columns as partials (finite logits only)
  float2* part_lse;
  // EPI_QKV of several layers in one launch (n_layers > 1; the last grid
  // dimension indexes the layer): layer z reads lw[z], lb[z] and writes the
  // caches kc / vc + z * kv_stride bytes
  int n_layers;
  long long kv_stride;
  const void* lw[kMaxLayers];
  const void* lb[kMaxLayers];
  // optional (nullptr: row-major w only): the same weights in the MFMA feed
  // order of the K-split product kernels (launch_pack_feed); single-layer
  // launches with N % 16 == 0 only, and the vocabulary kernel (any N)
  const void* wp;
};

// The weights and caches of layer z of a multi-layer EPI_QKV launch.  The
// tables are read with constant indices only (a selection chain on the
// uniform z): indexing them with z would copy the argument block to scratch.
__device__ __forceinline__ void layer_select(GemmArgs& a, int z) {
  if (a.n_layers > 1) {
    const void* w = a.lw[0];
    const void* b = a.lb[0];
#pragma unroll
    for (int i = 1; i < kMaxLayers; ++i) {
      w = z == i ? a.lw[i] : w;
      b = z == i ? a.lb[i] : b;
    }
    a.w = w;
    a.wp = nullptr;
    a.bias = b;
    a.kc = static_cast<char*>(a.kc) + z * a.kv_stride;
    a.vc = static_cast<char*>(a.vc) + z * a.kv_stride;
  }
}

constexpr int kAttnChunkKeys = 64;   // keys per attention chunk (one per lane of a wave)

struct AttnArgs {
  const int* n_rows_dev;
  int n_rows;
  const float* q;          // [R][ldq] float, unscaled
  int ldq;
  const void* kc;          // [S][H][T][dh] storage type
  const void* vc;
  int H, dh, T;
  RowMap rows;
  int causal;              // 1: row at position p sees keys 0..p; 0: keys 0..klen[s]-1
  const int* klen;
  void* out;               // [R][ldo] storage type
  int ldo;
  float scale;             // 1/sqrt(dh)
  int rows_max;            // launch bound on the rows (set by launch_attn)
  int out_feed;            // 1: out ([R][H dh]) written in the MFMA feed order (feed_index), ldo unused
  int max_keys;            // host bound on any row's key count (0: unknown); chooses the launch shape only
  int one_source;          // 1: every row is of sentence 0 and non-causal (a batch of one): key slots are
                           // loaded before klen[0] arrives (the caches must hold finite values throughout)
};

struct EmbedArgs {
  const int* n_rows_dev;
  int n_rows;
  const int* tok;          // [R] token of each row
  RowMap rows;             // position of each row
  const void* emb;         // E[V][d]
  const float* pe;         // positional table [positions][d] (k_pe_table)
  float scale;
  int d;
  int vocab;               // ids outside [0, vocab) are clamped into it
  void* out;               // [R][d] storage type
  // optional: n_len (<= kInlineLens) integers copied from the arguments to
  // len_out by the launch (per-sentence lengths without a staging copy)
  int* len_out;
  int n_len;
  int len_in[64];
};
constexpr int kInlineLens = 64;

// Per-sentence target lengths carried by k_ctrl_init's arguments (n > 0), in
// place of CtrlArgs::tgt_m, for up to kInlineLens sentences.
struct InlineLens {
  int n;
  int v[kInlineLens];
};

struct LnArgs {
  const int* n_rows_dev;
  int n_rows;
  const void* x;
  int x_f32;
  const void* g;
  const void* b;
  float eps;
  int d;
  void* out;               // storage type
};

// One record of the decoding trace: the token an iteration produced at a
// target position, its logit and the log-sum-exp of the row's logits
// (probability exp(top1 - lse)).  Same layout as pd_trace_record.
struct TraceRec {
  int iteration;   // 1-based iteration count of the sentence that produced the token
  int sentence;
  int position;    // 0-based target position
  int token;
  float top1;
  float lse;
};

// Per-sentence decoding state kept on the device.
struct SentState {
  int m;          // target length (number of equations)
  int i;          // first position of the current block
  int L;          // current block length (0 when done)
  int j;          // iterations spent on the current block
  int k;          // total iterations
  int done;
  int flags;
  int row0;       // first row of this sentence in the current iteration
};

struct CtrlArgs {
  SentState* st;
  int B;
  int mode, block, horizon, max_iters;
  int stop_prefix;         // 1: commit each iteration's proven prefix (PD_STOP_PREFIX), 0: Eq. (3)
  const int* tgt_m;        // [B]
  int* y;                  // [B][ldy] draft
  int ldy;
  const int* new_tok;      // [R] argmax of each row of the last iteration
  const int* row_flags;    // [R] nonzero: a non-finite logit was seen
  int* row_sent;           // [R_max] rows of the next iteration
  int* row_pos;
  int* row_tok;
  int* n_rows;             // device scalar
  unsigned long long* rows_total;   // device counter: rows of every iteration laid out (may be null)
  int* host_rows;          // mapped pinned host word (may be null): host_word(rows of the next iteration, near_end, seq)
  int* seq;                // device counter of the context's control steps (mod 64)
  int seq0;                // k_ctrl_init: the value it sets the counter to and publishes
  int pad_id, bos_id, eos_id;
  int R_max;
  const int* init;         // initial draft [B][init_ld] (nullptr: all [PAD])
  int init_ld;
  int reset_trace_count;   // k_ctrl_init zeroes *trace_count first
  // decoding trace (nullptr: off): one record per evaluated row
  TraceRec* trace;
  long long trace_cap;
  unsigned long long* trace_count;
  const float* row_max;    // [R] largest logit of each row of the iteration
  const float* row_lse;    // [R] log-sum-exp of each row
  // fused into the control step when non-null: the argmax over the vocabulary
  // partials of the rows just computed, and the embedding of the next rows
  const uint2* partials;
  int part_ld, n_parts;
  void* x_out;
  const void* emb;
  const float* pe;         // positional table [positions][d]
  float emb_scale;
  int d, vocab;
  // finalize
  int* out_ids; int out_ld; int* out_len; int* out_k; int* out_flags;
};

// The word the control step publishes to the host after laying out the next
// iteration: its row count (0 when every sentence is done) and, in bit 30,
// whether that iteration may be the last one: every live sentence is in its
// last block, the iteration is not the first of a block of several positions
// (which compares with an unrefined draft), and the block's cap of L
// iterations leaves at most kNearEndIters more (under the prefix stopping
// condition, which commits at least one position per iteration: the last
// block holds at most kNearEndIters positions).  The bit only paces the host.
// Bits 24..29 carry the number of control steps run so far (mod 64), so that
// the host recognises the word of the step it waits for without an event
// record after every iteration (each costs a few µs of GPU time); the rows
// take the low 24 bits (every launch has fewer than 2^24 rows).
constexpr int kNearEndBit = 1 << 30;
constexpr int kSeqShift = 24;
constexpr int kSeqMask = 63;
constexpr int kRowsMask = (1 << kSeqShift) - 1;
constexpr int kNearEndIters = 8;
__device__ __forceinline__ bool near_end(const SentState& st, int stop_prefix) {
  if (stop_prefix) return st.done || (st.i + st.L >= st.m && st.L <= kNearEndIters);   // >= 1 position per iteration
  return st.done || (st.i + st.L >= st.m && (st.j >= 1 || st.L == 1) && st.L - st.j <= kNearEndIters);
}
__host__ __device__ __forceinline__ int host_word(int rows, bool near, int seq) {
  return rows | (near && rows > 0 ? kNearEndBit : 0) | ((seq & kSeqMask) << kSeqShift);
}

struct ReduceArgs {
  const int* n_rows_dev;
  const uint2* partials;
  int part_ld;
  int n_parts;
  int* new_tok;
  int* row_flags;
};

// launchers (return hipError_t of the launch)
// With ev0 / ev1, the events receive the kernel dispatch's own start and end times.
hipError_t launch_gemm(int dtype, int pro, int epi, int ksplit, const GemmArgs& a, hipStream_t s,
                       hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
int gemm_grid(int epi, int N, int ksplit);
// W [N][K] (row-major) -> out [ceil(N / 16) 16 K] in the MFMA feed order read
// through GemmArgs::wp: block (c, s) of 64 16-byte words holds, in word l,
// W[min(16 c + (l & 15), N - 1)][s KS + EPL (l >> 4) ... + EPL - 1] (KS, EPL of
// the MFMA step of the type; a ragged last tile repeats row N - 1).
// K % KS == 0, else hipErrorInvalidValue.
hipError_t launch_pack_feed(int dtype, const void* w, void* out, int N, int K, hipStream_t s);
size_t gemm_ln_lds_bytes(int K, size_t elt);
// Products of many rows on LDS-staged MFMA tiles (bf16, no prologue, K a
// multiple of 64); bitwise the same values as launch_gemm.  The vocabulary
// argmax writes ceil(N / gemm_tiled_bn(EPI_ARGMAX, N, rows)) partials per row.
bool gemm_tiled_ok(int dtype, int pro, const GemmArgs& a);
int gemm_tiled_bn(int epi, int N, int rows);
void gemm_tiled_init();
hipError_t launch_gemm_tiled(int epi, int ksplit, const GemmArgs& a, hipStream_t s);
int gemm_tiled_cfg(int epi, int N, int rows);
hipError_t launch_gemm_tiled_cfg(int epi, int ksplit, int cfg, const GemmArgs& a, hipStream_t s);
hipError_t launch_attn(int dtype, const AttnArgs& a, int R_max, hipStream_t s);
// Fused vocabulary projection + argmax for at most 16 rows (streaming kernel);
// writes vocab_grid(dtype, V, d) partials per row (at most ceil(V / 64)).
// Optional events ev0 / ev1 receive the kernel's own start and end times.
int vocab_grid(int dtype, int V, int d);
hipError_t launch_vocab_argmax(int dtype, const GemmArgs& a, hipStream_t s, hipEvent_t ev0 = nullptr,
                               hipEvent_t ev1 = nullptr);
hipError_t launch_embed(int dtype, const EmbedArgs& a, int R_max, hipStream_t s);
// Trace: largest logit and log-sum-exp of each of the iteration's rows (rows
// counted on the device, at most R_max) from the argmax kernels' per-part
// (max, sum of exp(logit - max)) pairs part[row][part_ld], n_parts per row.
hipError_t launch_lse_reduce(const float2* part, int part_ld, int n_parts, const int* n_rows_dev, int R_max,
                             float* row_max, float* row_lse, hipStream_t s);
// Sinusoidal positional table pe[p][c] for p < n_pos (float of the double-precision value).
hipError_t launch_pe_table(float* pe, int n_pos, int d, hipStream_t s);
hipError_t launch_ln(int dtype, const LnArgs& a, int R_max, hipStream_t s);
hipError_t launch_argmax_reduce(const ReduceArgs& a, int R_max, hipStream_t s);
hipError_t launch_ctrl_init(int dtype, const CtrlArgs& a, const InlineLens& lens, hipStream_t s);
hipError_t launch_ctrl_step(int dtype, const CtrlArgs& a, hipStream_t s);
hipError_t launch_finalize(const CtrlArgs& a, hipStream_t s);

}  // namespace pdec

// Traced decode on caller-chosen log-sum-exp scratch (runtime.cpp): pd_decode
// with the decoding trace on, records appended from index 0 (the count is
// zeroed on the stream), iterations launched kernel by kernel (no graph is
// captured or instantiated), the context's own trace setting left as it was.
struct pd_ctx;
namespace pdec {
// Records `msg` as the calling thread's pd_last_error and returns status.
int32_t fail_with(int32_t status, const char* msg);
int32_t decode_traced_on(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                         const int32_t* tgt_m, int32_t* out_ids, int32_t out_ld, int32_t* out_len, int32_t* out_k,
                         int32_t* out_flags, void* records, int64_t capacity, void* scratch, size_t scratch_bytes,
                         const char* scratch_name, void* stream);


}  // namespace pdec

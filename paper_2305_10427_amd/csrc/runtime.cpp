// Host runtime behind the C ABI of include/pdec.h: configuration checks,
// workspace planning, the encoder pass, the decoder pass of one iteration and
// the iteration loop of the four decoding modes.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "../../include/pdec.h"

using namespace pdec;

namespace {

thread_local std::string g_err;

pd_status fail(pd_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

#define PD_HIP(call)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(PD_E_DEVICE, std::string(#call " failed: ") + hipGetErrorString(e_));     \
  } while (0)

// Up to this many rows a product runs on the streaming kernel with the
// LayerNorm in its prologue; above it the LayerNorm runs as its own kernel and
// bf16 products on the LDS-tiled kernel.  Both choices give bitwise the same
// rows.  For d <= 512 the streaming kernel stays ahead up to 128 rows; for
// wider models its per-workgroup LayerNorm costs more than the separate pass
// from 65 rows on.
int stream_max_rows(int d) { return d <= 512 ? 128 : 64; }
constexpr size_t kAlign = 256;
constexpr long long kMaxCtxRows = 1LL << 24;   // rows of the largest launch a context may need

int weight_count(const pd_config& c) {
  return 2 + 12 * c.n_enc + (c.pre_ln ? 2 : 0) + 20 * c.n_dec + (c.pre_ln ? 2 : 0);
}

bool check_config(const pd_config* c, std::string* why) {
  if (c == nullptr) { *why = "null config"; return false; }
  if (c->n_enc < 1 || c->n_dec < 1 || c->d_model < 8 || c->n_heads < 1 || c->d_ff < 8 || c->vocab < 4) {
    *why = "non-positive model size";
    return false;
  }
  if (c->dtype != PD_F32 && c->dtype != PD_BF16) { *why = "dtype must be PD_F32 or PD_BF16"; return false; }
  if (c->d_model % c->n_heads != 0) { *why = "d_model must be a multiple of n_heads"; return false; }
  const int dh = c->d_model / c->n_heads;
  if (dh != 16 && dh != 32 && dh != 64 && dh != 128) { *why = "head dim must be 16, 32, 64 or 128"; return false; }
  if (c->d_model % 32 != 0 || c->d_ff % 32 != 0) { *why = "d_model and d_ff must be multiples of 32"; return false; }
  if (c->d_model > (c->dtype == PD_BF16 ? 1024 : 512)) {
    *why = "d_model must be <= 1024 (bf16) or <= 512 (f32)";
    return false;
  }
  for (int id : {c->pad_id, c->bos_id, c->eos_id})
    if (id < 0 || id >= c->vocab) { *why = "special token id out of vocabulary"; return false; }
  if (!(c->ln_eps > 0.f)) { *why = "ln_eps must be positive"; return false; }
  return true;
}

void shape_of(const pd_config& c, int idx, int64_t* rows, int64_t* cols) {
  const int64_t d = c.d_model, f = c.d_ff, V = c.vocab;
  *cols = 1;
  if (idx == 0) { *rows = V; *cols = d; return; }
  if (idx == 1) { *rows = V; return; }
  int t = idx - 2;
  if (t < 12 * c.n_enc) {
    static const int64_t r_[12] = {3, 3, 1, 1, 1, 1, -1, -1, 1, 1, 1, 1};
    static const int c_[12] = {1, 0, 1, 0, 0, 0, 1, 0, 2, 0, 0, 0};   // 1: d, 2: d_ff, 0: vector
    const int j = t % 12;
    *rows = r_[j] > 0 ? r_[j] * d : f;
    *cols = c_[j] == 1 ? d : (c_[j] == 2 ? f : 1);
    return;
  }
  t -= 12 * c.n_enc;
  if (c.pre_ln) {
    if (t < 2) { *rows = d; return; }
    t -= 2;
  }
  if (t < 20 * c.n_dec) {
    static const int64_t r_[20] = {3, 3, 1, 1, 1, 1, 1, 1, 2, 2, 1, 1, 1, 1, -1, -1, 1, 1, 1, 1};
    static const int c_[20] = {1, 0, 1, 0, 0, 0, 1, 0, 1, 0, 1, 0, 0, 0, 1, 0, 2, 0, 0, 0};
    const int j = t % 20;
    *rows = r_[j] > 0 ? r_[j] * d : f;
    *cols = c_[j] == 1 ? d : (c_[j] == 2 ? f : 1);
    return;
  }
  *rows = d;   // final decoder LayerNorm
}

}  // namespace

struct pd_model {
  pd_config cfg;
  std::vector<const void*> w;
  // per weight: its copy in the MFMA feed order of the K-split product
  // kernels (owned, nullptr for weights that are not such products), made by
  // the first context created on the model (make_feed)
  mutable std::vector<void*> feed;
  mutable std::mutex feed_mu;
  mutable bool feed_ready = false;
  int dt;          // DT_F32 / DT_BF16
  int d, H, dh, dff, V;
  float enc_scale, dec_scale;

  const void* enc(int l, int j) const { return w[2 + 12 * l + j]; }
  const void* enc_feed(int l, int j) const { return feed[2 + 12 * l + j]; }
  const void* enc_ln(int j) const { return w[2 + 12 * cfg.n_enc + j]; }
  int dec_base() const { return 2 + 12 * cfg.n_enc + (cfg.pre_ln ? 2 : 0); }
  const void* dec(int l, int j) const { return w[dec_base() + 20 * l + j]; }
  const void* dec_feed(int l, int j) const { return feed[dec_base() + 20 * l + j]; }
  const void* dec_ln(int j) const { return w[dec_base() + 20 * cfg.n_dec + j]; }
  ~pd_model() {
    for (void* p : feed)
      if (p != nullptr) hipFree(p);
  }
};

namespace {

enum { E_WQKV = 0, E_BQKV, E_WO, E_BO, E_LN1G, E_LN1B, E_W1, E_B1, E_W2, E_B2, E_LN2G, E_LN2B };
enum {
  D_WQKV = 0, D_BQKV, D_WO, D_BO, D_LN1G, D_LN1B, D_CWQ, D_CBQ, D_CWKV, D_CBKV, D_CWO, D_CBO,
  D_LN2G, D_LN2B, D_W1, D_B1, D_W2, D_B2, D_LN3G, D_LN3B
};

struct Layout {
  size_t x_res, s_buf, q_buf, a_buf, h_buf;
  size_t enc_k, enc_v, cross_k, cross_v, self_k, self_v;
  size_t partials, new_tok, row_flags, row_sent, row_pos, row_tok;
  size_t st, y, tgt_m, src_len, n_rows, seq, rows_total, pe, trace_count, row_max, row_lse;
  size_t total;
};

Layout plan(const pd_model& M, int max_batch, int max_src, int max_tgt) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + kAlign - 1) / kAlign * kAlign;
    return at;
  };
  const size_t es = M.dt == DT_BF16 ? 2 : 4;
  const size_t rows_dec = static_cast<size_t>(max_batch) * max_tgt;
  const size_t vocab_wgs = static_cast<size_t>(gemm_grid(EPI_ARGMAX, M.V, 1));
  const size_t rows = std::max(static_cast<size_t>(max_batch) * max_src, rows_dec);
  const size_t rows16 = (rows + 15) / 16 * 16;    // whole 16-row tiles (feed-order activations)
  const size_t d = M.d;
  L.x_res = take(rows * d * es);
  L.s_buf = take(rows * d * 4);
  L.q_buf = take(rows * d * 4);
  L.a_buf = take(rows16 * d * es);
  L.h_buf = take(rows16 * M.dff * es);
  const size_t enc_kv = static_cast<size_t>(max_batch) * max_src * d * es;
  L.enc_k = take(enc_kv);
  L.enc_v = take(enc_kv);
  L.cross_k = take(enc_kv * M.cfg.n_dec);
  L.cross_v = take(enc_kv * M.cfg.n_dec);
  const size_t self_kv = rows_dec * d * es * M.cfg.n_dec;
  L.self_k = take(self_kv);
  L.self_v = take(self_kv);
  L.partials = take(rows_dec * vocab_wgs * sizeof(uint2));
  L.new_tok = take(rows_dec * 4);
  L.row_flags = take(rows_dec * 4);
  L.row_sent = take(rows_dec * 4);
  L.row_pos = take(rows_dec * 4);
  L.row_tok = take(rows_dec * 4);
  L.st = take(static_cast<size_t>(max_batch) * sizeof(SentState));
  L.y = take(rows_dec * 4);
  L.tgt_m = take(static_cast<size_t>(max_batch) * 4);
  L.src_len = take(static_cast<size_t>(max_batch) * 4);
  L.n_rows = take(4);
  L.seq = take(4);
  L.rows_total = take(8);
  L.trace_count = take(8);
  L.row_max = take(rows_dec * 4);
  L.row_lse = take(rows_dec * 4);
  L.pe = take(static_cast<size_t>(std::max(max_src, max_tgt)) * d * sizeof(float));
  L.total = off;
  return L;
}

}  // namespace

struct GraphKey {
  int mode, block, horizon, max_iters, B, R_max, slot, fused;
  int long_keys;   // rows of more than one key chunk possible: 1 self-attention, 2 cross-attention
  // the trace buffers are kernel arguments of a traced iteration
  const void* trace;
  long long trace_cap;
  const void* trace_part;
  bool operator==(const GraphKey& o) const {
    return mode == o.mode && block == o.block && horizon == o.horizon && max_iters == o.max_iters && B == o.B &&
           R_max == o.R_max && slot == o.slot && fused == o.fused && long_keys == o.long_keys && trace == o.trace &&
           trace_cap == o.trace_cap &&
           trace_part == o.trace_part;
  }
};

struct IterGraph {
  GraphKey key;
  hipGraphExec_t exec;
  int64_t kernels;                     // kernel nodes of the captured iteration
};

struct pd_ctx {
  const pd_model* M;
  hipStream_t capture = nullptr;       // private stream used only to capture iteration graphs
  bool use_graphs = true;
  std::vector<IterGraph> graphs;
  int64_t iter_kernels = 0;            // kernels of the iteration graph replayed last
  int max_batch, max_src, max_tgt;
  char* ws;
  Layout L;
  int* host_pinned;       // [0]: next iteration's row count (device-written, 0: done); [1 .. ]: staging for lengths
  int* host_rows_dev;     // device view of host_pinned[0]
  int* stage_src;         // pinned staging copies of host length arrays
  int* stage_tgt;
  hipEvent_t stage_ev = nullptr;
  std::vector<hipEvent_t> it_ev;   // [0]: recorded after a decode's last launch
  int seq_next = 0;                // sequence number of the next control step launched (mod 64)
  // vocabulary-kernel timing: event pairs per in-flight iteration slot
  bool timing = false;
  hipEvent_t tv0[2] = {nullptr, nullptr}, tv1[2] = {nullptr, nullptr};
  bool tv_pending[2] = {false, false};
  int64_t tv_launches = 0;
  double tv_ms = 0.0;
  // decoder-product timing: event pairs and algorithmic bytes of each timed
  // streaming-product launch, per in-flight iteration slot
  std::vector<hipEvent_t> pg0[2], pg1[2];
  std::vector<double> pg_bytes[2];
  int pg_n[2] = {0, 0};
  int gemm_slot = -1;                  // slot of the decoder pass being launched with timing, else -1
  int64_t tg_launches = 0;
  double tg_ms = 0.0, tg_bytes = 0.0;
  // decoding trace (off while trace == nullptr): caller-owned records and the
  // scratch of the vocabulary kernel's log-sum-exp partials
  TraceRec* trace = nullptr;
  long long trace_cap = 0;
  float2* trace_part = nullptr;
  long long trace_rows = 0;            // rows the scratch holds
  bool reset_trace = false;            // the next decode zeroes the record count on its stream
  int enc_B = 0, enc_nmax = 0;
  // host bounds on the key count of any row: the longest encoded source, and
  // the longest target of the running decode (or debug_logits' T)
  int src_keys = 0, self_keys = 0;
  bool encoded = false;

  template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

// Rows processed by one pass: count (device or host), layout and tokens.
struct Rows {
  const int* n_dev;
  int n_host;
  RowMap map;
  const int* tok;
  int R_max;
};

GemmArgs gemm_base(const Rows& r) {
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.n_rows_dev = r.n_dev;
  g.n_rows = r.R_max;
  g.rows = r.map;
  return g;
}

// One matrix product.  pro_ln: normalise x (float if x_f32) with (lg, lb)
// first; for many rows the LayerNorm runs as its own kernel into ln_tmp.
hipError_t run_gemm(pd_ctx& C, const Rows& r, GemmArgs g, int epi, bool pro_ln, void* ln_tmp,
                    hipStream_t s) {
  const pd_model& M = *C.M;
  int pro = PRO_NONE;
  if (pro_ln) {
    if (r.R_max <= stream_max_rows(M.d)) {
      pro = PRO_LN;
    } else {
      LnArgs la{r.n_dev, r.n_host, g.x, g.x_f32, g.ln_g, g.ln_b, M.cfg.ln_eps, g.K, ln_tmp};
      hipError_t e = launch_ln(M.dt, la, r.R_max, s);
      if (e != hipSuccess) return e;
      g.x = ln_tmp;
      g.x_f32 = 0;
      g.ldx = g.K;
      g.ln_out = nullptr;
    }
  }
  const int ksplit = (epi == EPI_ARGMAX || epi == EPI_LOGITS) ? 1 : (g.K >= 2048 ? 8 : 4);
  if (r.R_max > stream_max_rows(M.d) && gemm_tiled_ok(M.dt, pro, g)) return launch_gemm_tiled(epi, ksplit, g, s);
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  if (C.gemm_slot >= 0) {   // a timed decoder product: the next event pair of the slot, and its bytes
    const int sl = C.gemm_slot;
    if (C.pg_n[sl] == static_cast<int>(C.pg0[sl].size())) {
      hipEvent_t a = nullptr, b = nullptr;
      hipError_t e = hipEventCreate(&a);
      if (e == hipSuccess) e = hipEventCreate(&b);
      if (e != hipSuccess) {
        if (a) hipEventDestroy(a);
        return e;
      }
      C.pg0[sl].push_back(a);
      C.pg1[sl].push_back(b);
      C.pg_bytes[sl].push_back(0.0);
    }
    const double es = M.dt == DT_BF16 ? 2.0 : 4.0;
    C.pg_bytes[sl][C.pg_n[sl]] = es * (static_cast<double>(g.N) * g.K + g.N + (pro == PRO_LN ? 2.0 * g.K : 0.0));
    ev0 = C.pg0[sl][C.pg_n[sl]];
    ev1 = C.pg1[sl][C.pg_n[sl]];
    C.pg_n[sl] += 1;
  }
  return launch_gemm(M.dt, pro, epi, ksplit, g, s, ev0, ev1);
}

// Iterations of at most one 16-row tile use the streaming vocabulary kernel
// (vocab_grid partials per row); larger ones the product kernel's argmax
// epilogue (one partial per 64-column workgroup).
constexpr int kVocabStreamMaxRows = 16;
// Above one row tile the vocabulary argmax runs on the tiled product kernel
// (after a separate LayerNorm) when it supports the shape.
bool vocab_tiled(const pd_model& M, int R_max) {
  if (R_max <= kVocabStreamMaxRows) return false;
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.N = M.V;
  g.K = M.d;
  g.ldx = M.d;
  g.n_rows = R_max;
  return gemm_tiled_ok(M.dt, PRO_NONE, g);
}

int vocab_parts(const pd_model& M, int R_max) {
  if (R_max <= kVocabStreamMaxRows) return vocab_grid(M.dt, M.V, M.d);
  if (vocab_tiled(M, R_max)) {
    const int bn = gemm_tiled_bn(EPI_ARGMAX, M.V, R_max);
    return (M.V + bn - 1) / bn;
  }
  return gemm_grid(EPI_ARGMAX, M.V, 1);
}

// Decoder pass over the rows of one iteration (or the teacher-forced rows of
// pd_debug_logits), ending in the fused vocabulary argmax or a logits store.
// Token + positional embedding of the iteration's rows into the residual stream.
hipError_t embed_rows(pd_ctx& C, const Rows& r, hipStream_t s) {
  const pd_model& M = *C.M;
  EmbedArgs ea{r.n_dev, r.n_host, r.tok, r.map, M.w[0], C.at<float>(C.L.pe), M.dec_scale, M.d, M.V,
               C.at<char>(C.L.x_res)};
  return launch_embed(M.dt, ea, r.R_max, s);
}

hipError_t decoder_pass(pd_ctx& C, const Rows& r, float* logits, hipStream_t s, int slot = -1, bool fused = false) {
  const pd_model& M = *C.M;
  const pd_config& cfg = M.cfg;
  const int d = M.d;
  const bool pre = cfg.pre_ln != 0;
  void* x_res = C.at<char>(C.L.x_res);
  float* s_buf = C.at<float>(C.L.s_buf);
  float* q_buf = C.at<float>(C.L.q_buf);
  void* a_buf = C.at<char>(C.L.a_buf);
  void* h_buf = C.at<char>(C.L.h_buf);
  const size_t es = M.dt == DT_BF16 ? 2 : 4;
  const size_t self_layer = static_cast<size_t>(C.max_batch) * C.max_tgt * d * es;
  const size_t cross_layer = static_cast<size_t>(C.max_batch) * C.max_src * d * es;
  hipError_t e;

  if (!fused && (e = embed_rows(C, r, s)) != hipSuccess) return e;   // else the control step has embedded them

  // decoder products of a timed iteration are launched with dispatch-timestamp events
  struct SlotScope {
    pd_ctx& c;
    SlotScope(pd_ctx& c_, int sl) : c(c_) { c.gemm_slot = sl; }
    ~SlotScope() { c.gemm_slot = -1; }
  } scope(C, logits == nullptr ? slot : -1);
  // iterations of 9..16 rows pass the attention output and the FFN hidden
  // layer in the MFMA feed order (the products that read them then load 1 KB
  // contiguous per step instead of 64 bytes from each of 16 rows; with fewer
  // rows the row-major loads, which repeat rows, cost about the same or less:
  // large model, 16 rows: 650.6 -> 616.9 us per iteration; MT-base, 5 rows:
  // 204.5 -> 206.4)
  const int feed = r.R_max > 8 && r.R_max <= 16 ? 1 : 0;
  for (int l = 0; l < cfg.n_dec; ++l) {
    // self-attention: Q -> q_buf, K/V of the block -> cache (layer l)
    GemmArgs g = gemm_base(r);
    if (pre) {
      g.x = x_res; g.x_f32 = 0; g.ln_g = M.dec(l, D_LN1G); g.ln_b = M.dec(l, D_LN1B);
    } else if (l > 0) {
      g.x = s_buf; g.x_f32 = 1; g.ln_g = M.dec(l - 1, D_LN3G); g.ln_b = M.dec(l - 1, D_LN3B);
      g.ln_out = x_res; g.ldlo = d;
    } else {
      g.x = x_res; g.x_f32 = 0;
    }
    const bool ln_qkv = pre || l > 0;
    g.ldx = d; g.ln_eps = cfg.ln_eps;
    g.w = M.dec(l, D_WQKV); g.wp = M.dec_feed(l, D_WQKV); g.bias = M.dec(l, D_BQKV); g.N = 3 * d; g.K = d;
    g.out_f32 = q_buf; g.ldo = d; g.q_cols = d;
    g.kc = C.at<char>(C.L.self_k) + l * self_layer; g.vc = C.at<char>(C.L.self_v) + l * self_layer;
    g.H = M.H; g.dh = M.dh; g.T = C.max_tgt; g.d = d;
    // post-LN with a separate LayerNorm kernel writes the residual stream itself
    if ((e = run_gemm(C, r, g, EPI_QKV, ln_qkv, pre ? a_buf : x_res, s)) != hipSuccess) return e;

    AttnArgs aa{r.n_dev, r.n_host, q_buf, d, g.kc, g.vc, M.H, M.dh, C.max_tgt, r.map, 1, nullptr,
                a_buf, d, 1.0f / std::sqrt(static_cast<float>(M.dh))};
    aa.out_feed = feed;
    aa.max_keys = C.self_keys;
    if ((e = launch_attn(M.dt, aa, r.R_max, s)) != hipSuccess) return e;

    g = gemm_base(r);
    g.x = a_buf; g.ldx = d; g.x_feed = feed;
    g.w = M.dec(l, D_WO); g.wp = M.dec_feed(l, D_WO); g.bias = M.dec(l, D_BO); g.N = d; g.K = d;
    g.resid = x_res; g.ldr = d; g.ldo = d;
    if (pre) g.out = x_res; else g.out_f32 = s_buf;
    if ((e = run_gemm(C, r, g, EPI_RESID, false, nullptr, s)) != hipSuccess) return e;

    // cross-attention to the encoder memory
    g = gemm_base(r);
    if (pre) { g.x = x_res; g.x_f32 = 0; g.ln_g = M.dec(l, D_LN2G); g.ln_b = M.dec(l, D_LN2B); }
    else { g.x = s_buf; g.x_f32 = 1; g.ln_g = M.dec(l, D_LN1G); g.ln_b = M.dec(l, D_LN1B); g.ln_out = x_res; g.ldlo = d; }
    g.ldx = d; g.ln_eps = cfg.ln_eps;
    g.w = M.dec(l, D_CWQ); g.wp = M.dec_feed(l, D_CWQ); g.bias = M.dec(l, D_CBQ); g.N = d; g.K = d; g.out_f32 = q_buf; g.ldo = d;
    if ((e = run_gemm(C, r, g, EPI_F32, true, pre ? a_buf : x_res, s)) != hipSuccess) return e;

    aa = AttnArgs{r.n_dev, r.n_host, q_buf, d, C.at<char>(C.L.cross_k) + l * cross_layer,
                  C.at<char>(C.L.cross_v) + l * cross_layer, M.H, M.dh, C.max_src, r.map, 0,
                  C.at<int>(C.L.src_len), a_buf, d, 1.0f / std::sqrt(static_cast<float>(M.dh))};
    aa.out_feed = feed;
    aa.max_keys = C.src_keys;
    if ((e = launch_attn(M.dt, aa, r.R_max, s)) != hipSuccess) return e;

    g = gemm_base(r);
    g.x = a_buf; g.ldx = d; g.x_feed = feed;
    g.w = M.dec(l, D_CWO); g.wp = M.dec_feed(l, D_CWO); g.bias = M.dec(l, D_CBO); g.N = d; g.K = d;
    g.resid = x_res; g.ldr = d; g.ldo = d;
    if (pre) g.out = x_res; else g.out_f32 = s_buf;
    if ((e = run_gemm(C, r, g, EPI_RESID, false, nullptr, s)) != hipSuccess) return e;

    // feed-forward
    g = gemm_base(r);
    if (pre) { g.x = x_res; g.x_f32 = 0; g.ln_g = M.dec(l, D_LN3G); g.ln_b = M.dec(l, D_LN3B); }
    else { g.x = s_buf; g.x_f32 = 1; g.ln_g = M.dec(l, D_LN2G); g.ln_b = M.dec(l, D_LN2B); g.ln_out = x_res; g.ldlo = d; }
    g.ldx = d; g.ln_eps = cfg.ln_eps;
    g.w = M.dec(l, D_W1); g.wp = M.dec_feed(l, D_W1); g.bias = M.dec(l, D_B1); g.N = M.dff; g.K = d;
    g.out = h_buf; g.ldo = M.dff; g.act = cfg.act_gelu ? 2 : 1; g.out_feed = feed;
    if ((e = run_gemm(C, r, g, EPI_ACT, true, pre ? a_buf : x_res, s)) != hipSuccess) return e;

    g = gemm_base(r);
    g.x = h_buf; g.ldx = M.dff; g.x_feed = feed; g.w = M.dec(l, D_W2); g.wp = M.dec_feed(l, D_W2); g.bias = M.dec(l, D_B2); g.N = d; g.K = M.dff;
    g.resid = x_res; g.ldr = d; g.ldo = d;
    if (pre) g.out = x_res; else g.out_f32 = s_buf;
    if ((e = run_gemm(C, r, g, EPI_RESID, false, nullptr, s)) != hipSuccess) return e;
  }

  // vocabulary projection (tied embedding) fused with the argmax (timed on its own)
  C.gemm_slot = -1;
  GemmArgs g = gemm_base(r);
  if (pre) { g.x = x_res; g.x_f32 = 0; g.ln_g = M.dec_ln(0); g.ln_b = M.dec_ln(1); }
  else { g.x = s_buf; g.x_f32 = 1; g.ln_g = M.dec(cfg.n_dec - 1, D_LN3G); g.ln_b = M.dec(cfg.n_dec - 1, D_LN3B); }
  g.ldx = d; g.ln_eps = cfg.ln_eps;
  g.w = M.w[0]; g.bias = M.w[1]; g.N = M.V; g.K = d; g.logit_scale = cfg.logit_scale;
  if (logits != nullptr) {
    g.out_f32 = logits; g.ldo = M.V;
    return run_gemm(C, r, g, EPI_LOGITS, true, a_buf, s);
  }
  g.partials = C.at<uint2>(C.L.partials);
  g.part_ld = gemm_grid(EPI_ARGMAX, M.V, 1);
  g.part_lse = C.trace_part;   // nullptr unless tracing
  const int n_parts = vocab_parts(M, r.R_max);
  const bool tiled = r.R_max > kVocabStreamMaxRows && vocab_tiled(M, r.R_max);
  if (tiled) {   // the final LayerNorm as its own kernel, outside the timed vocabulary launch
    LnArgs la{r.n_dev, r.n_host, g.x, g.x_f32, g.ln_g, g.ln_b, cfg.ln_eps, d, a_buf};
    if ((e = launch_ln(M.dt, la, r.R_max, s)) != hipSuccess) return e;
    g.x = a_buf; g.x_f32 = 0; g.ldx = d;
  }
  if (r.R_max <= kVocabStreamMaxRows) {
    // one row tile: streaming kernel (E from its feed-order copy), timed by its
    // own dispatch timestamps
    g.wp = M.feed[0];
    e = launch_vocab_argmax(M.dt, g, s, slot >= 0 ? C.tv0[slot] : nullptr, slot >= 0 ? C.tv1[slot] : nullptr);
  } else {
    if (slot >= 0 && (e = hipEventRecord(C.tv0[slot], s)) != hipSuccess) return e;
    e = tiled ? launch_gemm_tiled(EPI_ARGMAX, 1, g, s) : run_gemm(C, r, g, EPI_ARGMAX, true, a_buf, s);
    if (e == hipSuccess && slot >= 0) e = hipEventRecord(C.tv1[slot], s);
  }
  if (e != hipSuccess) return e;
  if (slot >= 0) C.tv_pending[slot] = true;
  if (C.trace != nullptr) {   // each row's largest logit and log-sum-exp from the partials
    if ((e = launch_lse_reduce(C.trace_part, g.part_ld, n_parts, r.n_dev, r.R_max, C.at<float>(C.L.row_max),
                               C.at<float>(C.L.row_lse), s)) != hipSuccess)
      return e;
  }
  if (fused) return hipSuccess;   // the control step reduces the partials
  ReduceArgs ra{r.n_dev, C.at<uint2>(C.L.partials), g.part_ld, n_parts, C.at<int>(C.L.new_tok),
                C.at<int>(C.L.row_flags)};
  return launch_argmax_reduce(ra, r.R_max, s);
}

hipError_t encoder_pass(pd_ctx& C, const int32_t* src, int B, int n_max, const int32_t* inline_len,
                        hipStream_t s) {
  const pd_model& M = *C.M;
  const pd_config& cfg = M.cfg;
  const int d = M.d;
  const bool pre = cfg.pre_ln != 0;
  void* x_res = C.at<char>(C.L.x_res);
  float* s_buf = C.at<float>(C.L.s_buf);
  float* q_buf = C.at<float>(C.L.q_buf);
  void* a_buf = C.at<char>(C.L.a_buf);
  void* h_buf = C.at<char>(C.L.h_buf);
  const size_t es = M.dt == DT_BF16 ? 2 : 4;
  const size_t cross_layer = static_cast<size_t>(C.max_batch) * C.max_src * d * es;
  const int R = B * n_max;
  Rows r{nullptr, R, RowMap{nullptr, nullptr, n_max}, src, R};
  const int* klen = C.at<int>(C.L.src_len);
  const float scale = 1.0f / std::sqrt(static_cast<float>(M.dh));
  hipError_t e;

  EmbedArgs ea{nullptr, R, src, r.map, M.w[0], C.at<float>(C.L.pe), M.enc_scale, d, M.V, x_res};
  if (inline_len != nullptr) {           // the source lengths travel with the embedding launch
    ea.len_out = C.at<int>(C.L.src_len);
    ea.n_len = B;
    std::memcpy(ea.len_in, inline_len, sizeof(int32_t) * B);
  }
  if ((e = launch_embed(M.dt, ea, R, s)) != hipSuccess) return e;
  // Every LayerNorm feeding a product runs in that product's prologue (a
  // separate kernel above 64 rows, run_gemm); post-LN stores the normalised
  // rows to x_res as the next residual.
  for (int l = 0; l < cfg.n_enc; ++l) {
    GemmArgs g = gemm_base(r);
    bool ln = true;
    void* ln_tmp = a_buf;
    if (pre) {
      g.x = x_res; g.x_f32 = 0; g.ln_g = M.enc(l, E_LN1G); g.ln_b = M.enc(l, E_LN1B);
    } else if (l > 0) {
      g.x = s_buf; g.x_f32 = 1; g.ln_g = M.enc(l - 1, E_LN2G); g.ln_b = M.enc(l - 1, E_LN2B);
      g.ln_out = x_res; g.ldlo = d; ln_tmp = x_res;
    } else {
      g.x = x_res; g.x_f32 = 0; ln = false;   // the embedding
    }
    g.ldx = d; g.ln_eps = cfg.ln_eps;
    g.w = M.enc(l, E_WQKV); g.wp = M.enc_feed(l, E_WQKV); g.bias = M.enc(l, E_BQKV); g.N = 3 * d; g.K = d;
    g.out_f32 = q_buf; g.ldo = d; g.q_cols = d;
    g.kc = C.at<char>(C.L.enc_k); g.vc = C.at<char>(C.L.enc_v);
    g.H = M.H; g.dh = M.dh; g.T = C.max_src; g.d = d;
    if ((e = run_gemm(C, r, g, EPI_QKV, ln, ln_tmp, s)) != hipSuccess) return e;
    AttnArgs aa{nullptr, R, q_buf, d, g.kc, g.vc, M.H, M.dh, C.max_src, r.map, 0, klen, a_buf, d, scale};
    aa.max_keys = C.src_keys;
    // one source: its key slots load with the queries (in the decoder's
    // cross-attention this measured slower for the large model: slots past
    // the source come from HBM there, not from the cache the encoder filled)
    aa.one_source = B == 1 ? 1 : 0;
    if ((e = launch_attn(M.dt, aa, R, s)) != hipSuccess) return e;
    g = gemm_base(r);
    g.x = a_buf; g.ldx = d; g.w = M.enc(l, E_WO); g.wp = M.enc_feed(l, E_WO); g.bias = M.enc(l, E_BO); g.N = d; g.K = d;
    g.resid = x_res; g.ldr = d; g.ldo = d;
    if (pre) g.out = x_res; else g.out_f32 = s_buf;
    if ((e = run_gemm(C, r, g, EPI_RESID, false, nullptr, s)) != hipSuccess) return e;
    g = gemm_base(r);
    if (pre) {
      g.x = x_res; g.x_f32 = 0; g.ln_g = M.enc(l, E_LN2G); g.ln_b = M.enc(l, E_LN2B);
      ln_tmp = a_buf;
    } else {
      g.x = s_buf; g.x_f32 = 1; g.ln_g = M.enc(l, E_LN1G); g.ln_b = M.enc(l, E_LN1B);
      g.ln_out = x_res; g.ldlo = d; ln_tmp = x_res;
    }
    g.ldx = d; g.ln_eps = cfg.ln_eps;
    g.w = M.enc(l, E_W1); g.wp = M.enc_feed(l, E_W1); g.bias = M.enc(l, E_B1); g.N = M.dff; g.K = d;
    g.out = h_buf; g.ldo = M.dff; g.act = cfg.act_gelu ? 2 : 1;
    if ((e = run_gemm(C, r, g, EPI_ACT, true, ln_tmp, s)) != hipSuccess) return e;
    g = gemm_base(r);
    g.x = h_buf; g.ldx = M.dff; g.w = M.enc(l, E_W2); g.wp = M.enc_feed(l, E_W2); g.bias = M.enc(l, E_B2); g.N = d; g.K = M.dff;
    g.resid = x_res; g.ldr = d; g.ldo = d;
    if (pre) g.out = x_res; else g.out_f32 = s_buf;
    if ((e = run_gemm(C, r, g, EPI_RESID, false, nullptr, s)) != hipSuccess) return e;
  }
  // cross-attention K / V of every decoder layer, up to kMaxLayers layers per
  // launch, from the memory: the last LayerNorm (post-LN: the last layer's
  // second; pre-LN: the encoder's final one) runs in the product's prologue
  // (above the streaming row bound: a LayerNorm kernel into a_buf first)
  for (int l0 = 0; l0 < cfg.n_dec; l0 += kMaxLayers) {
    const int nl = std::min(kMaxLayers, cfg.n_dec - l0);
    GemmArgs g = gemm_base(r);
    if (pre) { g.x = x_res; g.x_f32 = 0; g.ln_g = M.enc_ln(0); g.ln_b = M.enc_ln(1); }
    else { g.x = s_buf; g.x_f32 = 1; g.ln_g = M.enc(cfg.n_enc - 1, E_LN2G); g.ln_b = M.enc(cfg.n_enc - 1, E_LN2B); }
    g.ln_eps = cfg.ln_eps;
    g.ldx = d; g.w = M.dec(l0, D_CWKV); g.bias = M.dec(l0, D_CBKV); g.N = 2 * d; g.K = d;
    g.q_cols = 0;
    g.kc = C.at<char>(C.L.cross_k) + l0 * cross_layer; g.vc = C.at<char>(C.L.cross_v) + l0 * cross_layer;
    g.H = M.H; g.dh = M.dh; g.T = C.max_src; g.d = d;
    g.n_layers = nl;
    g.kv_stride = static_cast<long long>(cross_layer);
    for (int z = 0; z < nl; ++z) {
      g.lw[z] = M.dec(l0 + z, D_CWKV);
      g.lb[z] = M.dec(l0 + z, D_CBKV);
    }
    if ((e = run_gemm(C, r, g, EPI_QKV, true, a_buf, s)) != hipSuccess) return e;
  }
  return hipSuccess;
}

constexpr int kFuseCtrlMaxRows = 64;   // above this the argmax reduction and embedding run as own kernels

// Launch bound of an iteration: the smallest power of two at or above a known
// upper bound on its rows, at most the decode's maximum.  Rows never grow from
// one iteration to the next (sentences only finish; a new block is never
// longer than the one before it: min(b, m - i), then 1 past the hybrid
// horizon), so a row count published by an earlier iteration bounds every
// later one.  Every kernel choice a bound selects gives bitwise the same rows,
// so the bound changes speed only: the last iterations of a batch, where few
// sentences are left, run the kernels of small iterations.
int launch_bound(int rows, int R_full) {
  int b = 1;
  while (b < rows && b < R_full) b <<= 1;
  return std::min(b, R_full);
}

// The control arguments of an iteration launched with bound R: with at most
// kFuseCtrlMaxRows rows the control step also reduces the argmax partials and
// embeds the next rows.
CtrlArgs ctrl_for_bound(const pd_ctx& C, const CtrlArgs& base, int R) {
  const pd_model& M = *C.M;
  CtrlArgs c = base;
  c.R_max = R;
  if (R <= kFuseCtrlMaxRows) {
    c.partials = C.at<uint2>(C.L.partials);
    c.part_ld = gemm_grid(EPI_ARGMAX, M.V, 1);
    c.n_parts = vocab_parts(M, R);
    c.x_out = C.at<char>(C.L.x_res);
    c.emb = M.w[0];
    c.pe = C.at<float>(C.L.pe);
    c.emb_scale = M.dec_scale;
    c.d = M.d;
    c.vocab = M.V;
  }
  return c;
}

// One decoding iteration: decoder pass over the current rows, fused
// vocabulary argmax, control step.
hipError_t iteration(pd_ctx& C, const Rows& r, const CtrlArgs& ca, hipStream_t s, int slot, bool fused) {
  hipError_t e = decoder_pass(C, r, nullptr, s, slot, fused);
  if (e != hipSuccess) return e;
  return launch_ctrl_step(C.M->dt, ca, s);
}

// The iteration as a HIP graph, captured once per context and launch shape.
hipError_t iteration_graph(pd_ctx& C, const GraphKey& key, const Rows& r, const CtrlArgs& ca, hipGraphExec_t* out) {
  for (auto& ig : C.graphs)
    if (ig.key == key) { *out = ig.exec; C.iter_kernels = ig.kernels; return hipSuccess; }
  hipError_t e = hipStreamBeginCapture(C.capture, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return e;
  hipError_t e_body = iteration(C, r, ca, C.capture, key.slot, key.fused != 0);
  hipGraph_t g = nullptr;
  e = hipStreamEndCapture(C.capture, &g);
  if (e_body != hipSuccess) { if (g) hipGraphDestroy(g); return e_body; }
  if (e != hipSuccess) return e;
  size_t nodes = 0;
  e = hipGraphGetNodes(g, nullptr, &nodes);
  hipGraphExec_t ex = nullptr;
  if (e == hipSuccess) e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
  hipGraphDestroy(g);
  if (e != hipSuccess) return e;
  C.graphs.push_back(IterGraph{key, ex, static_cast<int64_t>(nodes)});
  C.iter_kernels = static_cast<int64_t>(nodes);
  *out = ex;
  return hipSuccess;
}

pd_status stage_lengths(pd_ctx* C, int* stage, const int32_t* host, int B, int* dev, hipStream_t s) {
  PD_HIP(hipEventSynchronize(C->stage_ev));      // previous copy out of the staging area is done
  std::memcpy(stage, host, sizeof(int32_t) * B);
  PD_HIP(hipMemcpyAsync(dev, stage, sizeof(int32_t) * B, hipMemcpyHostToDevice, s));
  PD_HIP(hipEventRecord(C->stage_ev, s));
  return PD_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Waits until the host word carries the sequence number `target` of a
// control step, or that of the step after it (mod 64; the host is never more
// than one step behind), and returns the word.  It polls rather than blocking
// (a blocking wait adds a wake-up latency to every iteration); every few
// thousand polls it asks the stream for a failure, and an idle stream without
// the word is one too.
hipError_t wait_word(volatile int* word_p, int target, hipStream_t s, int* word) {
  auto ok = [&](int w) { return (((w >> kSeqShift) - target) & kSeqMask) <= 1; };
  for (unsigned n = 1;; ++n) {
    const int w = *word_p;
    if (ok(w)) {
      *word = w;
      return hipSuccess;
    }
    if ((n & 4095u) == 0) {
      const hipError_t e = hipStreamQuery(s);
      if (e == hipErrorNotReady) continue;
      if (e != hipSuccess) return e;
      // the stream has drained, so the step has run: its write to host memory
      // is given a moment to land before the word counts as missing
      const auto t0 = std::chrono::steady_clock::now();
      while (std::chrono::steady_clock::now() - t0 < std::chrono::milliseconds(50)) {
        const int w2 = *word_p;
        if (ok(w2)) {
          *word = w2;
          return hipSuccess;
        }
      }
      return hipErrorUnknown;
    }
  }
}

// Fold a slot's completed event pairs (decoder products, vocabulary kernel) into the totals.
hipError_t take_timing(pd_ctx& C, int slot) {
  for (int i = 0; i < C.pg_n[slot]; ++i) {
    hipError_t e = hipEventSynchronize(C.pg1[slot][i]);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, C.pg0[slot][i], C.pg1[slot][i]);
    if (e != hipSuccess) return e;
    C.tg_ms += ms;
    C.tg_bytes += C.pg_bytes[slot][i];
    C.tg_launches += 1;
  }
  C.pg_n[slot] = 0;
  if (!C.tv_pending[slot]) return hipSuccess;
  hipError_t e = hipEventSynchronize(C.tv1[slot]);
  if (e != hipSuccess) return e;
  float ms = 0.f;
  e = hipEventElapsedTime(&ms, C.tv0[slot], C.tv1[slot]);
  if (e != hipSuccess) return e;
  C.tv_ms += ms;
  C.tv_launches += 1;
  C.tv_pending[slot] = false;
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* pd_last_error(void) { return g_err.c_str(); }

int32_t pd_weight_count(const pd_config* cfg) {
  std::string why;
  if (!check_config(cfg, &why)) return -1;
  return weight_count(*cfg);
}

pd_status pd_weight_shape(const pd_config* cfg, int32_t idx, int64_t* rows, int64_t* cols) {
  std::string why;
  if (!check_config(cfg, &why)) return fail(PD_E_ARG, why);
  if (rows == nullptr || cols == nullptr) return fail(PD_E_ARG, "null output pointer");
  if (idx < 0 || idx >= weight_count(*cfg)) return fail(PD_E_ARG, "weight index out of range");
  shape_of(*cfg, idx, rows, cols);
  return PD_OK;
}

// The MFMA-feed copies of the encoder and decoder products, once per model
// (the first context created on it; the weights are read here).
static hipError_t make_feed(const pd_model& M) {
  std::lock_guard<std::mutex> lock(M.feed_mu);
  if (M.feed_ready) return hipSuccess;
  std::vector<int> prods{0};          // E, for the vocabulary kernel (a ragged last tile allowed)
  for (int l = 0; l < M.cfg.n_enc; ++l)
    for (int j : {E_WQKV, E_WO, E_W1, E_W2}) prods.push_back(2 + 12 * l + j);
  for (int l = 0; l < M.cfg.n_dec; ++l)
    for (int j : {D_WQKV, D_WO, D_CWQ, D_CWO, D_W1, D_W2}) prods.push_back(M.dec_base() + 20 * l + j);
  const size_t es = M.dt == DT_BF16 ? 2 : 4;
  hipError_t e = hipSuccess;
  for (int idx : prods) {
    if (M.feed[idx] != nullptr) continue;
    int64_t rows = 0, cols = 0;
    shape_of(M.cfg, idx, &rows, &cols);
    if (idx != 0 && rows % 16 != 0) continue;   // a ragged product: the row-major weights only
    void* p = nullptr;
    if ((e = hipMalloc(&p, static_cast<size_t>((rows + 15) / 16 * 16 * cols) * es)) != hipSuccess) return e;
    M.feed[idx] = p;
    if ((e = launch_pack_feed(M.dt, M.w[idx], p, static_cast<int>(rows), static_cast<int>(cols), nullptr)) !=
        hipSuccess)
      return e;
  }
  if ((e = hipStreamSynchronize(nullptr)) != hipSuccess) return e;
  M.feed_ready = true;
  return hipSuccess;
}

pd_status pd_model_create(const pd_config* cfg, const void* const* dev_weights, int32_t n_weights,
                          pd_model** out) {
  std::string why;
  if (out == nullptr) return fail(PD_E_ARG, "null output pointer");
  *out = nullptr;
  if (!check_config(cfg, &why)) return fail(PD_E_UNSUPPORTED, why);
  if (dev_weights == nullptr) return fail(PD_E_ARG, "null weight array");
  const int n = weight_count(*cfg);
  if (n_weights != n) return fail(PD_E_ARG, "expected " + std::to_string(n) + " weights, got " + std::to_string(n_weights));
  for (int i = 0; i < n; ++i)
    if (dev_weights[i] == nullptr || !aligned(dev_weights[i], 16))
      return fail(PD_E_ARG, "weight " + std::to_string(i) + " is null or not 16-byte aligned");
  gemm_tiled_init();
  pd_model* m = new pd_model();
  m->cfg = *cfg;
  m->w.assign(dev_weights, dev_weights + n);
  m->dt = cfg->dtype == PD_BF16 ? DT_BF16 : DT_F32;
  m->d = cfg->d_model;
  m->H = cfg->n_heads;
  m->dh = cfg->d_model / cfg->n_heads;
  m->dff = cfg->d_ff;
  m->V = cfg->vocab;
  const float sq = std::sqrt(static_cast<float>(cfg->d_model));
  m->enc_scale = cfg->enc_emb_scale < 0.f ? sq : cfg->enc_emb_scale;
  m->dec_scale = cfg->dec_emb_scale < 0.f ? sq : cfg->dec_emb_scale;
  m->feed.assign(n, nullptr);
  *out = m;
  return PD_OK;
}

void pd_model_destroy(pd_model* model) { delete model; }

pd_status pd_ctx_workspace_bytes(const pd_model* model, int32_t max_batch, int32_t max_src, int32_t max_tgt,
                                 size_t* bytes) {
  if (model == nullptr || bytes == nullptr) return fail(PD_E_ARG, "null argument");
  if (max_batch < 1 || max_src < 1 || max_tgt < 1) return fail(PD_E_SHAPE, "limits must be positive");
  if (max_tgt > 1024 || max_src > 1024) return fail(PD_E_SHAPE, "max_src and max_tgt must be <= 1024");
  // rows of one launch are counted in int and published to the host below the near-end bit
  if (static_cast<long long>(max_batch) * std::max(max_src, max_tgt) >= kMaxCtxRows)
    return fail(PD_E_SHAPE, "max_batch * max(max_src, max_tgt) must be below " + std::to_string(kMaxCtxRows));
  *bytes = plan(*model, max_batch, max_src, max_tgt).total;
  return PD_OK;
}

pd_status pd_ctx_create(const pd_model* model, int32_t max_batch, int32_t max_src, int32_t max_tgt,
                        void* dev_workspace, size_t workspace_bytes, pd_ctx** out) {
  if (out == nullptr || model == nullptr) return fail(PD_E_ARG, "null argument");
  *out = nullptr;
  size_t need = 0;
  pd_status st = pd_ctx_workspace_bytes(model, max_batch, max_src, max_tgt, &need);
  if (st != PD_OK) return st;
  if (dev_workspace == nullptr || !aligned(dev_workspace, kAlign))
    return fail(PD_E_WORKSPACE, "workspace is null or not 256-byte aligned");
  if (workspace_bytes < need)
    return fail(PD_E_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes");
  hipError_t fe = make_feed(*model);
  if (fe != hipSuccess) return fail(PD_E_DEVICE, std::string("weight feed copies: ") + hipGetErrorString(fe));
  pd_ctx* c = new pd_ctx();
  c->M = model;
  c->max_batch = max_batch;
  c->max_src = max_src;
  c->max_tgt = max_tgt;
  c->ws = static_cast<char*>(dev_workspace);
  c->L = plan(*model, max_batch, max_src, max_tgt);
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&c->host_pinned), sizeof(int) * (1 + 2 * max_batch),
                               hipHostMallocMapped);
  if (e != hipSuccess) { delete c; return fail(PD_E_DEVICE, std::string("hipHostMalloc: ") + hipGetErrorString(e)); }
  c->host_pinned[0] = 0;
  e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->host_rows_dev), c->host_pinned, 0);
  if (e != hipSuccess) {
    hipHostFree(c->host_pinned);
    delete c;
    return fail(PD_E_DEVICE, std::string("hipHostGetDevicePointer: ") + hipGetErrorString(e));
  }
  c->stage_src = c->host_pinned + 1;
  c->stage_tgt = c->host_pinned + 1 + max_batch;
  c->it_ev.resize(1, nullptr);
  e = hipEventCreateWithFlags(&c->stage_ev, hipEventDisableTiming);
  for (auto& ev : c->it_ev)
    if (e == hipSuccess) e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
  for (int i = 0; i < 2 && e == hipSuccess; ++i) {
    e = hipEventCreate(&c->tv0[i]);
    if (e == hipSuccess) e = hipEventCreate(&c->tv1[i]);
  }
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->capture, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipMemset(c->at<unsigned long long>(c->L.rows_total), 0, sizeof(unsigned long long));
  // the encoder and cross-attention caches start at zero, so that every key
  // slot holds a finite value before the first encode writes it (batch-of-one
  // attention loads slots past a source's length and weighs them by zero)
  // (enc_k, enc_v, cross_k and cross_v lie back to back, up to self_k)
  if (e == hipSuccess) e = hipMemset(c->at<char>(c->L.enc_k), 0, c->L.self_k - c->L.enc_k);
  if (e == hipSuccess) e = launch_pe_table(c->at<float>(c->L.pe), std::max(max_src, max_tgt), model->d, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    pd_ctx_destroy(c);
    return fail(PD_E_DEVICE, std::string("context set-up: ") + hipGetErrorString(e));
  }
  const char* g = std::getenv("PDEC_GRAPHS");
  c->use_graphs = !(g != nullptr && g[0] == '0');
  *out = c;
  return PD_OK;
}

void pd_ctx_destroy(pd_ctx* ctx) {
  if (ctx == nullptr) return;
  if (ctx->stage_ev) hipEventSynchronize(ctx->stage_ev);
  for (auto ev : ctx->it_ev)
    if (ev) { hipEventSynchronize(ev); hipEventDestroy(ev); }
  for (int i = 0; i < 2; ++i) {
    if (ctx->tv1[i]) { hipEventSynchronize(ctx->tv1[i]); hipEventDestroy(ctx->tv1[i]); }
    if (ctx->tv0[i]) hipEventDestroy(ctx->tv0[i]);
  }
  if (ctx->stage_ev) hipEventDestroy(ctx->stage_ev);
  for (int i = 0; i < 2; ++i) {
    for (auto ev : ctx->pg1[i]) { hipEventSynchronize(ev); hipEventDestroy(ev); }
    for (auto ev : ctx->pg0[i]) hipEventDestroy(ev);
  }
  for (auto& ig : ctx->graphs) hipGraphExecDestroy(ig.exec);
  if (ctx->capture) hipStreamDestroy(ctx->capture);
  hipHostFree(ctx->host_pinned);
  delete ctx;
}

pd_status pd_encode(pd_ctx* ctx, const int32_t* src_ids, const int32_t* src_len, int32_t B, int32_t n_max,
                    void* stream) {
  if (ctx == nullptr || src_ids == nullptr || src_len == nullptr) return fail(PD_E_ARG, "null argument");
  if (B < 1 || n_max < 1) return fail(PD_E_ARG, "B and n_max must be >= 1");
  if (B > ctx->max_batch || n_max > ctx->max_src) return fail(PD_E_SHAPE, "batch or source length exceeds the context limits");
  for (int b = 0; b < B; ++b)
    if (src_len[b] < 1 || src_len[b] > n_max) return fail(PD_E_ARG, "src_len[" + std::to_string(b) + "] out of [1, n_max]");
  hipStream_t s = static_cast<hipStream_t>(stream);
  ctx->encoded = false;
  ctx->src_keys = 0;
  for (int b = 0; b < B; ++b) ctx->src_keys = std::max(ctx->src_keys, static_cast<int>(src_len[b]));
  // up to kInlineLens lengths go to the device with the first encoder kernel,
  // more through the staging copy
  const bool inline_len = B <= kInlineLens;
  if (!inline_len) {
    pd_status st = stage_lengths(ctx, ctx->stage_src, src_len, B, ctx->at<int>(ctx->L.src_len), s);
    if (st != PD_OK) return st;
  }
  hipError_t e = encoder_pass(*ctx, src_ids, B, n_max, inline_len ? src_len : nullptr, s);
  if (e != hipSuccess) return fail(PD_E_DEVICE, std::string("encoder launch: ") + hipGetErrorString(e));
  ctx->enc_B = B;
  ctx->enc_nmax = n_max;
  ctx->encoded = true;
  return PD_OK;
}

pd_status pd_decode(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                    const int32_t* tgt_m, int32_t* out_ids, int32_t out_ld, int32_t* out_len,
                    int32_t* out_k, int32_t* out_flags, void* stream) {
  return pd_decode_init(ctx, mode, block, horizon, max_iters, tgt_m, nullptr, 0, out_ids, out_ld, out_len, out_k,
                        out_flags, stream);
}

pd_status pd_decode_init(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                         const int32_t* tgt_m, const int32_t* init_ids, int32_t init_ld, int32_t* out_ids,
                         int32_t out_ld, int32_t* out_len, int32_t* out_k, int32_t* out_flags, void* stream) {
  if (ctx == nullptr || tgt_m == nullptr || out_ids == nullptr || out_len == nullptr || out_k == nullptr ||
      out_flags == nullptr)
    return fail(PD_E_ARG, "null argument");
  if (!ctx->encoded) return fail(PD_E_STATE, "pd_decode called before pd_encode");
  const int key_mode = mode;                   // with the stopping-condition flag (graph key)
  const int stop_prefix = (mode & PD_STOP_PREFIX) != 0 ? 1 : 0;
  mode &= ~PD_STOP_PREFIX;
  if (mode < PD_AR || mode > PD_HYBRID) return fail(PD_E_ARG, "unknown mode");
  if ((mode == PD_GS_JACOBI || mode == PD_HYBRID) && block < 1) return fail(PD_E_ARG, "block must be >= 1");
  const int B = ctx->enc_B;
  int m_max = 0;
  for (int b = 0; b < B; ++b) {
    if (tgt_m[b] < 1 || tgt_m[b] > ctx->max_tgt)
      return fail(PD_E_SHAPE, "tgt_m[" + std::to_string(b) + "] out of [1, max_tgt]");
    m_max = std::max(m_max, tgt_m[b]);
  }
  if (out_ld < m_max) return fail(PD_E_ARG, "out_ld must be >= max(tgt_m)");
  if (init_ids != nullptr && init_ld < m_max) return fail(PD_E_ARG, "init_ld must be >= max(tgt_m)");
  hipStream_t s = static_cast<hipStream_t>(stream);
  pd_ctx& C = *ctx;
  const pd_model& M = *C.M;
  int Lmax = 1;
  if (mode == PD_JACOBI) Lmax = m_max;
  else if (mode == PD_GS_JACOBI || mode == PD_HYBRID) Lmax = std::min(block, m_max);
  const int R_max = B * Lmax;
  int iters = m_max;
  if (max_iters > 0) iters = std::min(iters, max_iters);
  if (C.trace != nullptr && R_max > C.trace_rows)
    return fail(PD_E_WORKSPACE, "trace scratch holds " + std::to_string(C.trace_rows) +
                                    " rows, the decode needs " + std::to_string(R_max));
  // up to kInlineLens target lengths go with the initial control step's
  // arguments, more through the staging copy
  InlineLens lens;
  lens.n = 0;
  if (B <= kInlineLens) {
    lens.n = B;
    std::memcpy(lens.v, tgt_m, sizeof(int32_t) * B);
  } else {
    pd_status st = stage_lengths(ctx, C.stage_tgt, tgt_m, B, C.at<int>(C.L.tgt_m), s);
    if (st != PD_OK) return st;
  }
  C.self_keys = m_max;

  CtrlArgs ca;
  std::memset(&ca, 0, sizeof(ca));
  ca.st = C.at<SentState>(C.L.st);
  ca.B = B;
  ca.mode = mode;
  ca.stop_prefix = stop_prefix;
  ca.block = std::max(block, 1);
  ca.horizon = horizon;
  ca.max_iters = max_iters;
  ca.tgt_m = C.at<int>(C.L.tgt_m);
  ca.y = C.at<int>(C.L.y);
  ca.ldy = C.max_tgt;
  ca.new_tok = C.at<int>(C.L.new_tok);
  ca.row_flags = C.at<int>(C.L.row_flags);
  ca.row_sent = C.at<int>(C.L.row_sent);
  ca.row_pos = C.at<int>(C.L.row_pos);
  ca.row_tok = C.at<int>(C.L.row_tok);
  ca.n_rows = C.at<int>(C.L.n_rows);
  ca.rows_total = C.at<unsigned long long>(C.L.rows_total);
  ca.host_rows = C.host_rows_dev;
  ca.seq = C.at<int>(C.L.seq);
  ca.pad_id = M.cfg.pad_id;
  ca.bos_id = M.cfg.bos_id;
  ca.eos_id = M.cfg.eos_id;
  ca.R_max = R_max;
  ca.init = init_ids;
  ca.init_ld = init_ld;
  if (C.trace != nullptr) {
    ca.trace = C.trace;
    ca.trace_cap = C.trace_cap;
    ca.trace_count = C.at<unsigned long long>(C.L.trace_count);
    ca.row_max = C.at<float>(C.L.row_max);
    ca.row_lse = C.at<float>(C.L.row_lse);
    ca.reset_trace_count = C.reset_trace ? 1 : 0;
  }
  ca.out_ids = out_ids;
  ca.out_ld = out_ld;
  ca.out_len = out_len;
  ca.out_k = out_k;
  ca.out_flags = out_flags;

  // the first rows (at most R_max) are laid out, and embedded when the first
  // iteration's control step is the fused one, by the initial step
  bool prev_fused = R_max <= kFuseCtrlMaxRows;
  CtrlArgs c0 = ctrl_for_bound(C, ca, R_max);
  c0.seq0 = C.seq_next;            // every control step launched advances the count, even after the end
  hipError_t e = launch_ctrl_init(M.dt, c0, lens, s);
  if (e != hipSuccess) return fail(PD_E_DEVICE, std::string("init launch: ") + hipGetErrorString(e));
  C.seq_next = (C.seq_next + 1) & kSeqMask;
  volatile int* host_rows = C.host_pinned;
  int bound = R_max;   // rows of the next iteration launched are at most this
  for (int it = 0; it < iters; ++it) {
    const int slot = C.timing ? (it & 1) : -1;
    if (slot >= 0 && (e = take_timing(C, slot)) != hipSuccess)
      return fail(PD_E_DEVICE, std::string("timing: ") + hipGetErrorString(e));
    const int Rb = launch_bound(bound, R_max);
    const bool fused = Rb <= kFuseCtrlMaxRows;
    const CtrlArgs cb = ctrl_for_bound(C, ca, Rb);
    const Rows r{ca.n_rows, 0, RowMap{ca.row_sent, ca.row_pos, 0}, ca.row_tok, Rb};
    // the first iteration under a fused control step after unfused ones: its
    // rows were laid out but not embedded
    e = fused && !prev_fused ? embed_rows(C, r, s) : hipSuccess;
    prev_fused = fused;
    if (e == hipSuccess) {
      if (C.use_graphs && slot < 0) {   // iterations timed with events are launched directly
        hipGraphExec_t ex = nullptr;
        const int long_keys = (C.self_keys > kAttnChunkKeys ? 1 : 0) | (C.src_keys > kAttnChunkKeys ? 2 : 0);
        const GraphKey key{key_mode, block, horizon, max_iters, B, Rb, slot, fused ? 1 : 0, long_keys, C.trace,
                           C.trace_cap, C.trace_part};
        e = iteration_graph(C, key, r, cb, &ex);
        if (e == hipSuccess) e = hipGraphLaunch(ex, s);
      } else {
        e = iteration(C, r, cb, s, slot, fused);
      }
    }
    if (e != hipSuccess) return fail(PD_E_DEVICE, std::string("iteration launch: ") + hipGetErrorString(e));
    const int q = C.seq_next;        // this iteration's control step
    C.seq_next = (C.seq_next + 1) & kSeqMask;
    if (it >= 1) {
      // the previous iteration's control step (or the next one) has published
      // the row count of the iteration after it (0 when every sentence is
      // done, else a bound on the rows of every iteration not launched yet)
      // and whether that iteration, the one in flight, may be the last: then
      // it is waited for too, rather than launching one more iteration that
      // may find nothing to do
      int word = 0;
      if ((e = wait_word(host_rows, q - 1, s, &word)) != hipSuccess)
        return fail(PD_E_DEVICE, std::string("iteration: ") + hipGetErrorString(e));
      if ((word & kNearEndBit) != 0 && (e = wait_word(host_rows, q, s, &word)) != hipSuccess)
        return fail(PD_E_DEVICE, std::string("iteration: ") + hipGetErrorString(e));
      const int rows = word & kRowsMask;
      if (rows <= 0) break;
      bound = std::min(bound, rows);
    }
  }
  e = launch_finalize(ca, s);
  if (e == hipSuccess) e = hipEventRecord(C.it_ev[0], s);   // the decode's last work (pd_ctx_destroy waits for it)
  if (e != hipSuccess) return fail(PD_E_DEVICE, std::string("finalize launch: ") + hipGetErrorString(e));
  if (C.timing) {
    for (int slot = 0; slot < 2; ++slot)
      if ((e = take_timing(C, slot)) != hipSuccess) return fail(PD_E_DEVICE, std::string("timing: ") + hipGetErrorString(e));
  }
  return PD_OK;
}

pd_status pd_ctx_set_timing(pd_ctx* ctx, int32_t enable) {
  if (ctx == nullptr) return fail(PD_E_ARG, "null context");
  PD_HIP(hipMemset(ctx->at<unsigned long long>(ctx->L.rows_total), 0, sizeof(unsigned long long)));
  ctx->timing = enable != 0;
  ctx->tv_launches = 0;
  ctx->tv_ms = 0.0;
  ctx->tv_pending[0] = ctx->tv_pending[1] = false;
  ctx->tg_launches = 0;
  ctx->tg_ms = ctx->tg_bytes = 0.0;
  ctx->pg_n[0] = ctx->pg_n[1] = 0;
  return PD_OK;
}

pd_status pd_ctx_product_timing(const pd_ctx* ctx, int64_t* launches, double* total_ms, double* bytes) {
  if (ctx == nullptr || launches == nullptr || total_ms == nullptr || bytes == nullptr)
    return fail(PD_E_ARG, "null argument");
  *launches = ctx->tg_launches;
  *total_ms = ctx->tg_ms;
  *bytes = ctx->tg_bytes;
  return PD_OK;
}

pd_status pd_ctx_iteration_kernels(const pd_ctx* ctx, int64_t* kernels) {
  if (ctx == nullptr || kernels == nullptr) return fail(PD_E_ARG, "null argument");
  *kernels = ctx->iter_kernels;
  return PD_OK;
}

pd_status pd_ctx_vocab_timing(const pd_ctx* ctx, int64_t* launches, double* total_ms) {
  if (ctx == nullptr || launches == nullptr || total_ms == nullptr) return fail(PD_E_ARG, "null argument");
  *launches = ctx->tv_launches;
  *total_ms = ctx->tv_ms;
  return PD_OK;
}

static_assert(sizeof(TraceRec) == sizeof(pd_trace_record), "trace record layouts differ");

// Bytes of trace scratch per row: one (max, sum) pair per vocabulary workgroup.
static size_t trace_row_bytes(const pd_model& M) {
  return static_cast<size_t>(gemm_grid(EPI_ARGMAX, M.V, 1)) * sizeof(float2);
}

pd_status pd_trace_scratch_bytes(const pd_model* model, int32_t max_rows, size_t* bytes) {
  if (model == nullptr || bytes == nullptr) return fail(PD_E_ARG, "null argument");
  if (max_rows < 1) return fail(PD_E_ARG, "max_rows must be >= 1");
  *bytes = static_cast<size_t>(max_rows) * trace_row_bytes(*model);
  return PD_OK;
}

pd_status pd_ctx_set_trace(pd_ctx* ctx, void* dev_records, int64_t capacity, void* dev_scratch,
                           size_t scratch_bytes) {
  if (ctx == nullptr) return fail(PD_E_ARG, "null context");
  if (dev_records == nullptr) {
    ctx->trace = nullptr;
    ctx->trace_cap = 0;
    ctx->trace_part = nullptr;
    ctx->trace_rows = 0;
    return PD_OK;
  }
  if (capacity < 1 || dev_scratch == nullptr) return fail(PD_E_ARG, "capacity must be >= 1 and scratch non-null");
  if (!aligned(dev_records, 16) || !aligned(dev_scratch, 16))
    return fail(PD_E_ARG, "trace buffers must be 16-byte aligned");
  const size_t row_bytes = trace_row_bytes(*ctx->M);
  if (scratch_bytes < row_bytes) return fail(PD_E_WORKSPACE, "trace scratch holds no row");
  PD_HIP(hipMemset(ctx->at<unsigned long long>(ctx->L.trace_count), 0, sizeof(unsigned long long)));
  ctx->trace = static_cast<TraceRec*>(dev_records);
  ctx->trace_cap = capacity;
  ctx->trace_part = static_cast<float2*>(dev_scratch);
  ctx->trace_rows = static_cast<long long>(scratch_bytes / row_bytes);
  return PD_OK;
}

pd_status pd_ctx_trace_count(const pd_ctx* ctx, int64_t* records) {
  if (ctx == nullptr || records == nullptr) return fail(PD_E_ARG, "null argument");
  unsigned long long v = 0;
  PD_HIP(hipMemcpy(&v, ctx->at<unsigned long long>(ctx->L.trace_count), sizeof(v), hipMemcpyDeviceToHost));
  *records = static_cast<int64_t>(v);
  return PD_OK;
}

pd_status pd_ctx_rows_processed(const pd_ctx* ctx, int64_t* rows) {
  if (ctx == nullptr || rows == nullptr) return fail(PD_E_ARG, "null argument");
  unsigned long long v = 0;
  PD_HIP(hipMemcpy(&v, ctx->at<unsigned long long>(ctx->L.rows_total), sizeof(v), hipMemcpyDeviceToHost));
  *rows = static_cast<int64_t>(v);
  return PD_OK;
}

pd_status pd_debug_logits(pd_ctx* ctx, const int32_t* tgt_in, int32_t T, float* logits, void* stream) {
  if (ctx == nullptr || tgt_in == nullptr || logits == nullptr) return fail(PD_E_ARG, "null argument");
  if (!ctx->encoded) return fail(PD_E_STATE, "pd_debug_logits called before pd_encode");
  if (T < 1 || T > ctx->max_tgt) return fail(PD_E_SHAPE, "T out of [1, max_tgt]");
  const int B = ctx->enc_B;
  const int R = B * T;
  Rows r{nullptr, R, RowMap{nullptr, nullptr, T}, tgt_in, R};
  ctx->self_keys = T;
  hipError_t e = decoder_pass(*ctx, r, logits, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PD_E_DEVICE, std::string("decoder launch: ") + hipGetErrorString(e));
  return PD_OK;
}

}  // extern "C"

namespace pdec {

int32_t fail_with(int32_t status, const char* msg) { return fail(status, msg); }

int32_t decode_traced_on(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                         const int32_t* tgt_m, int32_t* out_ids, int32_t out_ld, int32_t* out_len, int32_t* out_k,
                         int32_t* out_flags, void* records, int64_t capacity, void* scratch, size_t scratch_bytes,
                         const char* scratch_name, void* stream) {
  if (ctx == nullptr) return fail(PD_E_ARG, "null context");
  if (records == nullptr || capacity < 1) return fail(PD_E_ARG, "records must be non-null and capacity >= 1");
  if (scratch == nullptr || !aligned(records, 16) || !aligned(scratch, 16))
    return fail(PD_E_ARG, "trace buffers must be non-null and 16-byte aligned");
  pd_ctx& C = *ctx;
  const TraceRec* trace = C.trace;
  const long long cap = C.trace_cap, rows = C.trace_rows;
  float2* part = C.trace_part;
  const bool graphs = C.use_graphs;
  C.trace = static_cast<TraceRec*>(records);
  C.trace_cap = capacity;
  C.trace_part = static_cast<float2*>(scratch);
  C.trace_rows = static_cast<long long>(scratch_bytes / trace_row_bytes(*C.M));
  C.use_graphs = false;
  C.reset_trace = true;
  pd_status st = pd_decode_init(ctx, mode, block, horizon, max_iters, tgt_m, nullptr, 0, out_ids, out_ld, out_len,
                                out_k, out_flags, stream);
  C.trace = const_cast<TraceRec*>(trace);
  C.trace_cap = cap;
  C.trace_part = part;
  C.trace_rows = rows;
  C.use_graphs = graphs;
  C.reset_trace = false;
  if (st == PD_E_WORKSPACE) g_err = std::string(scratch_name) + ": " + g_err;
  return st;
}

}  // namespace pdec

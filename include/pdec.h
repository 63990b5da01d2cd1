/*
 * pdec -- parallel (Jacobi / GS-Jacobi / hybrid) decoding of an
 * encoder-decoder Transformer on AMD Instinct MI355X (gfx950).
 *
 * The library solves the triangular system of greedy decoding
 *   y_i = argmax p_theta(y_i | y_1..y_{i-1}, x),  i = 1..m        (Section 3.1, Eq. (1)-(2))
 * with the fixed-point iterations of Section 3.2 / Appendix A:
 *   PD_AR         greedy autoregressive decoding, one token per decoder forward;
 *   PD_JACOBI     Algorithm 1 (PJ): all m positions updated from the previous iterate;
 *   PD_GS_JACOBI  Algorithm 2 (PGJ): Jacobi inside blocks of b positions,
 *                 Gauss-Seidel from block to block;
 *   PD_HYBRID     Algorithm 3 (HGJ): PGJ up to a horizon h, then greedy steps;
 *                 stops at the first [EOS] of a converged block.
 * Every decoder forward ("iteration") runs hand-written HIP kernels: a decoder
 * pass over the active block (causal self-attention over a KV cache,
 * cross-attention to the encoder memory, FFN, LayerNorm), a fused vocabulary
 * projection + argmax that never stores logits, and an on-device stopping
 * test (Eq. (3): the block is unchanged) that commits converged blocks and
 * lays out the next iteration, so the loop needs no host round trip.
 *
 * Memory ownership.  Every device buffer the caller hands over (weights,
 * workspace, inputs, outputs) is allocated and freed by the caller.  The
 * library allocates device memory in one place only: the first pd_ctx_create
 * on a model makes the model's copy of its product weights and embedding in
 * matrix-core feed order (see pd_model_create), freed by pd_model_destroy.
 * Besides that, pd_model / pd_ctx own host-side state (plus one pinned host
 * word per context for completion polling).  Weight and workspace buffers must stay
 * valid and unchanged while a model / context uses them.
 *
 * Threads and streams.  A pd_ctx is used by one host thread at a time; calls
 * on it are enqueued on the stream given to each call and are asynchronous
 * unless stated otherwise.  A context's workspace holds the encoder state
 * between pd_encode and pd_decode, so those two calls must be ordered (same
 * stream, or synchronised); so must any two calls that use one context's
 * workspace (a decode returns with its outputs, and possibly an iteration
 * that finds nothing left to do, still queued on its stream).
 *
 * Errors.  Every call returns pd_status.  Argument / shape / state errors are
 * detected on the host before anything is enqueued.  PD_E_DEVICE reports a
 * HIP launch or runtime failure; pd_last_error() holds a message for the
 * calling thread.  Numerical anomalies found on the device (a non-finite
 * logit) are reported per sentence in out_flags only.
 */
#ifndef PDEC_H_
#define PDEC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pd_status;
enum {
  PD_OK = 0,
  PD_E_ARG = 1,          /* invalid argument value (mode, block, pointer, ...) */
  PD_E_SHAPE = 2,        /* a size exceeds what the model / context was built for */
  PD_E_WORKSPACE = 3,    /* workspace missing, misaligned or too small */
  PD_E_DEVICE = 4,       /* HIP error */
  PD_E_UNSUPPORTED = 5,  /* configuration the kernels do not handle */
  PD_E_STATE = 6         /* call out of order (e.g. decode before encode) */
};

/* Decoding modes (Section 3.2). */
enum { PD_AR = 0, PD_JACOBI = 1, PD_GS_JACOBI = 2, PD_HYBRID = 3 };

/*
 * Stopping-condition variant, or-ed into the mode of pd_decode /
 * pd_decode_init / pd_decode_traced_static (the paper leaves stopping
 * conditions other than Eq. (3) to future work: Section 3.3, conclusion).
 * Eq. (3) commits a block once an iteration leaves it unchanged (or after L
 * iterations).  PD_STOP_PREFIX commits after every iteration the positions
 * that iteration proved exact: the whole block when it is unchanged, else the
 * leading positions that came out as they went in plus the next one (its
 * inputs were exact); the block then moves on by that many positions, the
 * newer values of the rest serving as its draft.  The output is still greedy
 * decoding's (Proposition 1's argument), k <= m, and PD_HYBRID stops at an
 * [EOS] once it is committed.  No effect with PD_AR.
 */
enum { PD_STOP_PREFIX = 0x100 };

/* Storage types of weights and activations. */
enum { PD_F32 = 0, PD_BF16 = 1 };

/* Per-sentence result flags (out_flags bits). */
enum {
  PD_FLAG_CONVERGED = 1,    /* every position solved (or [EOS] reached in a converged block) */
  PD_FLAG_EOS = 2,          /* stopped at [EOS] (PD_AR, PD_HYBRID) */
  PD_FLAG_MAX_ITERS = 4,    /* stopped by max_iters before convergence */
  PD_FLAG_NONFINITE = 8     /* a logit was NaN/Inf at some iteration */
};

/*
 * Model shape.  The model is p_theta of Section 3.1 with the two shapes of
 * Section 4.1 ("Model Configuration"): post-LN (x <- LN(x + Sub(x))) or pre-LN
 * (x <- x + Sub(LN(x)), plus a final LayerNorm after encoder and decoder),
 * ReLU or exact-erf GELU FFN, sinusoidal positions, one token embedding E[V][d]
 * shared by encoder input, decoder input and the output projection
 * logits = logit_scale * h . E^T + out_bias.
 *   d_model must be a multiple of 32 and of n_heads, at most 1024 (bf16) or
 *   512 (f32); d_model / n_heads must be 16, 32, 64 or 128; d_ff a multiple
 *   of 32.
 *   enc_emb_scale / dec_emb_scale multiply E[token] at the encoder / decoder
 *   input (a negative value selects sqrt(d_model)).
 *   bf16 models store weights, K/V, attention outputs, FFN hidden values, the
 *   residual stream and LayerNorm outputs feeding a product in bfloat16
 *   (round to nearest even) and accumulate in float.
 */
typedef struct {
  int32_t n_enc, n_dec, d_model, n_heads, d_ff, vocab;
  int32_t pre_ln;        /* 0: post-LN, 1: pre-LN with final LayerNorms */
  int32_t act_gelu;      /* 0: ReLU, 1: GELU (erf) */
  int32_t dtype;         /* PD_F32 or PD_BF16 */
  int32_t pad_id, bos_id, eos_id;
  float ln_eps;
  float logit_scale;
  float enc_emb_scale;
  float dec_emb_scale;
} pd_config;

typedef struct pd_model pd_model;
typedef struct pd_ctx pd_ctx;

/*
 * Number of weight tensors of a configuration, and the shape of tensor idx
 * (rows x cols; cols = 1 for vectors).  Canonical order:
 *   0 emb [V][d]          1 out_bias [V]
 *   encoder layer l (12 tensors each):
 *     w_qkv [3d][d], b_qkv [3d], w_o [d][d], b_o [d], ln1_g [d], ln1_b [d],
 *     w1 [d_ff][d], b1 [d_ff], w2 [d][d_ff], b2 [d], ln2_g [d], ln2_b [d]
 *   pre-LN only: enc_ln_g [d], enc_ln_b [d]
 *   decoder layer l (20 tensors each):
 *     w_qkv [3d][d], b_qkv [3d], w_o [d][d], b_o [d], ln1_g [d], ln1_b [d],
 *     ca_w_q [d][d], ca_b_q [d], ca_w_kv [2d][d], ca_b_kv [2d], ca_w_o [d][d], ca_b_o [d],
 *     ln2_g [d], ln2_b [d],
 *     w1 [d_ff][d], b1 [d_ff], w2 [d][d_ff], b2 [d], ln3_g [d], ln3_b [d]
 *   pre-LN only: dec_ln_g [d], dec_ln_b [d]
 * Matrices are row-major [out][in]; w_qkv stacks the Q, K and V projections.
 * Returns -1 for an invalid configuration.
 */
int32_t pd_weight_count(const pd_config* cfg);
pd_status pd_weight_shape(const pd_config* cfg, int32_t idx, int64_t* rows, int64_t* cols);

/*
 * Bind a configuration to caller-owned device weights.  dev_weights holds
 * n_weights device pointers in canonical order, each 16-byte aligned, of
 * element type float (PD_F32) or bfloat16 bit patterns (PD_BF16).  The
 * pointers are stored, not copied, and read for the model's lifetime: the
 * caller keeps them allocated and unchanged until pd_model_destroy.  No
 * device work happens here.  The first pd_ctx_create on the model allocates,
 * on the current device, a copy of every encoder and decoder matrix
 * product's weights (w_qkv, w_o, w1, w2; ca_w_q, ca_w_o) and of the token
 * embedding E (the vocabulary projection's weights) rearranged into the
 * order in which the few-row kernels feed the matrix cores (as many bytes as
 * those matrices, E's rows rounded up to a multiple of 16; freed by
 * pd_model_destroy).  Returns PD_E_ARG for
 * a null / misaligned pointer or a wrong count, PD_E_UNSUPPORTED for shapes
 * the kernels reject.
 */
pd_status pd_model_create(const pd_config* cfg, const void* const* dev_weights, int32_t n_weights,
                          pd_model** out);
void pd_model_destroy(pd_model* model);

/*
 * Device workspace needed by a context that decodes up to max_batch sentences
 * with sources of at most max_src tokens and targets of at most max_tgt
 * positions (max_src, max_tgt <= 1024; max_batch * max(max_src, max_tgt)
 * below 2^24, else PD_E_SHAPE).  Covers every mode, including PD_JACOBI with
 * blocks of max_tgt positions.
 */
pd_status pd_ctx_workspace_bytes(const pd_model* model, int32_t max_batch, int32_t max_src,
                                 int32_t max_tgt, size_t* bytes);

/*
 * Create a context on caller-owned device workspace (256-byte aligned, at
 * least pd_ctx_workspace_bytes).  The workspace holds activations, the
 * cross-attention and self-attention K/V caches, drafts and control state.
 * The first context of a model also makes the model's matrix-core feed copy
 * of its product weights and embedding (see pd_model_create), on the null
 * stream, and waits for it; PD_E_DEVICE when that allocation or copy fails.
 */
pd_status pd_ctx_create(const pd_model* model, int32_t max_batch, int32_t max_src, int32_t max_tgt,
                        void* dev_workspace, size_t workspace_bytes, pd_ctx** out);
void pd_ctx_destroy(pd_ctx* ctx);

/*
 * Encode a batch of B sources (the conditioning x of p_theta(y | x)).
 *   src_ids  device int32 [B][n_max], token ids, rows padded after src_len[b]
 *            (ids outside [0, vocab) are clamped into it)
 *   src_len  HOST int32 [B], 1 <= src_len[b] <= n_max (read before the call
 *            returns; up to 64 lengths go with the first kernel's arguments,
 *            more through a pinned staging copy)
 * Runs the encoder and writes the cross-attention K/V of every decoder layer
 * into the context.  Padded positions are masked out of every attention.
 * PD_E_SHAPE if B > max_batch or n_max > max_src.
 */
pd_status pd_encode(pd_ctx* ctx, const int32_t* src_ids, const int32_t* src_len, int32_t B,
                    int32_t n_max, void* stream);

/*
 * Decode the batch of the last pd_encode on this context.
 *   mode      PD_AR, PD_JACOBI, PD_GS_JACOBI or PD_HYBRID
 *   block     block size b >= 1 (PD_GS_JACOBI, PD_HYBRID); ignored otherwise
 *             (PD_JACOBI uses one block of m positions, PD_AR blocks of 1)
 *   horizon   PD_HYBRID parallel horizon h (<= 0: h = m); ignored otherwise
 *   max_iters per-sentence cap on decoder forwards (<= 0: m, which every mode
 *             needs at most, Proposition 1)
 *   tgt_m     HOST int32 [B] (B of the last pd_encode), number of target
 *             positions m of each sentence, 1 <= tgt_m[b] <= max_tgt (read
 *             before the call returns, as src_len of pd_encode)
 *   out_ids   device int32 [B][out_ld], out_ld >= max(tgt_m): the solution
 *             cut after its first [EOS] (inclusive) and [PAD]-filled
 *   out_len   device int32 [B]: output length (first [EOS] + 1, else m)
 *   out_k     device int32 [B]: iterations (decoder forwards) used
 *   out_flags device int32 [B]: PD_FLAG_* bits
 * The initial draft is all [PAD] (Section 3.3, "Initialization").  Sentences
 * of a batch iterate independently; a sentence's result does not depend on
 * the other sentences.  The call blocks the host until the iteration has
 * converged (it polls a word the device writes once per iteration: the next
 * iteration's row count, which also sizes later launches), then enqueues the
 * output writes on the stream.
 */
pd_status pd_decode(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                    const int32_t* tgt_m, int32_t* out_ids, int32_t out_ld, int32_t* out_len,
                    int32_t* out_k, int32_t* out_flags, void* stream);

/*
 * pd_decode from a caller-supplied initial draft (InitT of Section 3.3)
 * instead of all [PAD].
 *   init_ids  device int32 [B][init_ld], init_ld >= max(tgt_m): the draft of
 *             positions 0 .. tgt_m[b] - 1 of each sentence (ids outside
 *             [0, vocab) are clamped into it where they enter the decoder)
 * Every mode still returns the greedy solution in at most m iterations
 * (Proposition 1 holds for any initialisation); only the iteration count k
 * depends on the draft.  PD_AR ignores the draft's values (blocks of one
 * position converge after one iteration).  init_ids == NULL is pd_decode.
 */
pd_status pd_decode_init(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                         const int32_t* tgt_m, const int32_t* init_ids, int32_t init_ld, int32_t* out_ids,
                         int32_t out_ld, int32_t* out_len, int32_t* out_k, int32_t* out_flags, void* stream);

/*
 * Verification only: teacher-forced logits of the encoded batch.
 *   tgt_in  device int32 [B][T] decoder inputs (BOS first), T <= max_tgt
 *   logits  device float [B][T][V]
 * Uses the same kernels as pd_decode, with the argmax replaced by a store.
 */
pd_status pd_debug_logits(pd_ctx* ctx, const int32_t* tgt_in, int32_t T, float* logits, void* stream);

/*
 * Timing of the fused vocabulary projection + argmax kernel, the kernel that
 * moves most bytes per iteration.  With timing enabled, pd_decode times every
 * launch of that kernel with a pair of HIP events and accumulates their
 * elapsed times; pd_ctx_vocab_timing returns the number of launches and their
 * total milliseconds since the last pd_ctx_set_timing.  For iterations of at
 * most 16 rows (the streaming kernel) the events carry the kernel dispatch's
 * own start and end timestamps (hipExtLaunchKernel); for larger iterations
 * they are recorded on the stream just before and after the launch, which
 * adds the event markers' own time.  Timed iterations are launched kernel by
 * kernel instead of replaying the captured iteration graph.
 * pd_ctx_set_timing also resets the counter of pd_ctx_rows_processed
 * (synchronously).
 */
pd_status pd_ctx_set_timing(pd_ctx* ctx, int32_t enable);
pd_status pd_ctx_vocab_timing(const pd_ctx* ctx, int64_t* launches, double* total_ms);

/*
 * Timing of the decoder's matrix products.  With timing enabled, every
 * decoder-layer product of a timed iteration that runs on the streaming
 * product kernel (iterations of up to 64 rows, 128 for d_model <= 512: QKV,
 * attention output, cross-attention query and output, both FFN products) is
 * launched with a pair of events that carry its dispatch's own start and end
 * times.  pd_ctx_product_timing returns, since the last pd_ctx_set_timing,
 * their number, the sum of their durations in milliseconds, and the
 * algorithmic bytes those launches must read: weights, biases and LayerNorm
 * parameters, in the storage type (the few activation rows are not counted).
 */
pd_status pd_ctx_product_timing(const pd_ctx* ctx, int64_t* launches, double* total_ms, double* bytes);

/*
 * Kernels launched per iteration: the number of kernel nodes of the HIP graph
 * of the iteration that pd_decode last replayed on this context (0 before
 * the first graph).
 */
pd_status pd_ctx_iteration_kernels(const pd_ctx* ctx, int64_t* kernels);

/*
 * Rows (decoder positions) evaluated by all iterations of pd_decode on this
 * context since the context was created or pd_ctx_set_timing was last called:
 * the sum over iterations of the rows laid out for that iteration (the work
 * the fused vocabulary projection and every decoder product did).  Reads
 * device memory synchronously: call it after the decode's stream has
 * synchronised.
 */
pd_status pd_ctx_rows_processed(const pd_ctx* ctx, int64_t* rows);

/*
 * Decoding trace: the data behind the DDGviz view (Section 3.5, and Figure 3
 * in Section 4.3), which shows for every Jacobi iteration the token each
 * evaluated position received and its probability under p_theta.
 *
 * With a trace buffer set, every iteration of pd_decode / pd_decode_init
 * appends one record per evaluated row (decoder position), in the order of
 * the iteration's rows (sentence by sentence, positions increasing):
 *   iteration  the sentence's iteration count after this iteration (1-based,
 *              the k of that sentence at that point)
 *   sentence   index of the sentence in the batch
 *   position   0-based target position (the record predicts y[position])
 *   token      argmax over the vocabulary (the value written to the iterate)
 *   top1       the largest logit of the row
 *   lse        log sum_v exp(logit_v) of the row, so that the token's
 *              probability is exp(top1 - lse)
 * Records are appended at index = number of records so far; the buffer keeps
 * the first `capacity` of them and pd_ctx_trace_count returns the full count
 * (which may exceed capacity).  The logits are still never stored: the fused
 * vocabulary kernel also keeps a running log-sum-exp per row and returns, per
 * workgroup, a (max, sum of exp(logit - max)) pair, which a small kernel
 * folds into top1 and lse.  Those pairs go to a caller-owned scratch of at
 * least pd_trace_scratch_bytes(model, rows) bytes, where rows is the largest
 * number of rows one iteration lays out (B * block for the block modes, B * m
 * for PD_JACOBI, B for PD_AR); a decode whose iteration needs more rows than
 * the scratch holds fails with PD_E_WORKSPACE before launching anything.
 * Traced iterations are replayed from HIP graphs like untraced ones (one
 * capture per set of trace buffers).  Tracing changes no token, count or flag
 * of the decode.  top1 is the exact largest
 * logit; lse is rounded in float and its summation order follows the kernel
 * that ran (it may differ in the last bits between batch sizes).
 *
 * pd_ctx_set_trace(ctx, records, capacity, scratch, scratch_bytes): records:
 *   device buffer of `capacity` records (pd_trace_record, 16-byte aligned),
 *   scratch: device buffer (16-byte aligned).  Both stay owned by the caller
 *   and must outlive every traced decode.  records == NULL turns tracing off.
 *   Resets the record count (synchronously).
 * pd_ctx_trace_count: records appended since pd_ctx_set_trace (synchronous
 *   device read; call after the decode's stream has synchronised).
 */
typedef struct {
  int32_t iteration, sentence, position, token;
  float top1, lse;
} pd_trace_record;

pd_status pd_trace_scratch_bytes(const pd_model* model, int32_t max_rows, size_t* bytes);
pd_status pd_ctx_set_trace(pd_ctx* ctx, void* dev_records, int64_t capacity, void* dev_scratch,
                           size_t scratch_bytes);
pd_status pd_ctx_trace_count(const pd_ctx* ctx, int64_t* records);

/*
 * For callers that cannot allocate device memory (serving loops and harnesses
 * that must not call hipMalloc / hipFree or any allocating routine once set
 * up): pd_decode with the decoding trace on, whose log-sum-exp partials live
 * in a static device array of the library (PD_TRACE_STATIC_BYTES = 8 MiB per
 * GPU, held until the process ends) instead of a caller scratch.
 *   dev_records, capacity  caller-owned device buffer of `capacity` records
 *                          (pd_trace_record, 16-byte aligned), as for
 *                          pd_ctx_set_trace; this call writes records from
 *                          index 0 (pd_ctx_trace_count then returns their
 *                          count)
 * Every other argument and every result is as for pd_decode.  The call
 * allocates nothing: iterations are launched kernel by kernel (no graph is
 * captured or instantiated) and the record count is zeroed by a kernel on
 * `stream`.  The context's own pd_ctx_set_trace setting is left as it was.
 * Limit: an iteration may lay out at most
 * PD_TRACE_STATIC_BYTES / pd_trace_scratch_bytes(model, 1) rows (B * block
 * for the block modes, B * m for PD_JACOBI, B for PD_AR); a larger decode
 * fails with PD_E_WORKSPACE before anything is launched.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (different streams or threads) race and corrupt each other's
 * trace.
 */
#define PD_TRACE_STATIC_BYTES (8u << 20)
pd_status pd_decode_traced_static(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon, int32_t max_iters,
                                  const int32_t* tgt_m, int32_t* out_ids, int32_t out_ld, int32_t* out_len,
                                  int32_t* out_k, int32_t* out_flags, void* dev_records, int64_t capacity,
                                  void* stream);

/* Message of the last failing call on this thread ("" if none). */
const char* pd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PDEC_H_ */

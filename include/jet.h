/*
 * jet.h - C ABI of the MI355X (gfx950) candidate-scoring library.
 *
 * The library scores a finite set of candidate answers against one shared
 * question context by teacher forcing (JET, arXiv 2609.33874):
 *
 *   p(y_{c,t} | x, y_{c,<t}) is normalised over the full vocabulary with no
 *   temperature and no top-k/top-p filtering (Section 3.1, Eq. 1), its log is
 *   taken in the max-shifted form of Eq. 2, summed per candidate (Section 3.2,
 *   Eq. 3), normalised over the candidate set (Eq. 4) and turned into a choice,
 *   a binary probability or an ordinal expectation (Section 3.3, Eq. 5).
 *
 * The question prefix is evaluated once and its attention cache / recurrent
 * state is retained (Section 4.1); every candidate then runs against that
 * retained state in batches, isolated from its siblings. Only the
 * log-probabilities of the supplied tokens leave the device (Section 4.2).
 *
 * Conventions shared by every call
 * --------------------------------
 * Return value: JET_OK (0) or one of the JET_E_* codes. On error no output
 *   buffer is written, every `out` handle is set to NULL, and jet_last_error()
 *   returns a message for the calling thread (Figure 1: invalid requests
 *   produce errors).
 * Ownership: the caller owns every array passed in or out; the library reads
 *   and writes them only during the call and keeps no pointer to them. The
 *   library owns the opaque handles; a jet_prefix borrows its jet_model.
 *   Free prefixes before their model. If the model is freed first, its
 *   prefixes' device buffers are freed with it and each such prefix is
 *   detached: it can no longer be scored against (JET_E_INVALID) and
 *   jet_prefix_free still releases its handle.
 * Memory kinds: arrays documented as "host" must be host memory. Arrays
 *   documented as "host or device" may be host memory or device memory of
 *   the model's GPU (the kind is queried with hipPointerGetAttributes).
 * Blocking: every call has finished its GPU work and its outputs are in place
 *   when it returns (it synchronises the model's stream).
 * Concurrency: calls on one model must be serialised by the caller.
 * Token ids: int32 in [0, vocab). Offsets: int64 CSR arrays, first element 0,
 *   non-decreasing.
 */
#ifndef JET_H
#define JET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  JET_OK = 0,
  JET_E_INVALID = 1,   /* malformed arguments, ids out of range, empty sequences */
  JET_E_CAPACITY = 2,  /* a sequence P + m - 1 exceeds max_ctx (never truncated) */
  JET_E_OOM = 3,       /* device allocation failed or max_device_bytes exceeded */
  JET_E_DEVICE = 4,    /* a HIP runtime error */
  JET_E_IO = 5         /* model file missing or malformed */
};

/* Compute modes. JET_BF16: bf16 weights and bf16 matrix-core products; the
 * activations, attention caches and probabilities are carried as (hi, lo)
 * bf16 pairs (value = hi + lo) so that rounding does not accumulate through
 * deep stacks (fp32 accumulation throughout). JET_FP32: fp32 everything
 * (validation mode). JET_BF16_SINGLE: single bf16 activations and caches;
 * faster, with rounding that grows with depth. JET_F16: the bf16 weights are
 * held as fp16 (each matrix times a power of two, which makes the conversion
 * exact), and activations, caches and probabilities are single fp16 values
 * (11 significant bits against bf16's 8), so every product is one fp16
 * matrix-core operation at the bf16 rate with fp32 accumulation; needs a bf16
 * model file. JET_F16P: as JET_F16, with the attention side (the inputs of
 * the attention layers' projections, q, the K/V caches, the attention
 * probabilities and output) carried as (hi, lo) fp16 pairs like JET_BF16:
 * for deep stacks, where single fp16 rounding on that side adds up. */
enum { JET_BF16 = 0, JET_FP32 = 1, JET_BF16_SINGLE = 2, JET_F16 = 3, JET_F16P = 4 };
enum { JET_CHOICE = 0, JET_BINARY = 1, JET_ORDINAL = 2 }; /* decision rule */

/* flags for jet_load_opts.flags */
enum {
  JET_FLAG_KERNEL_TIMING = 1, /* time every launch with HIP events (jet_stats) */
  JET_FLAG_RECORD_ROUTES = 2  /* mixture-of-experts models: keep the experts each
                                 layer chose for each row (jet_routes_get);
                                 a diagnostic for checking routing, it
                                 synchronises the stream at every such layer */
};

typedef struct jet_model jet_model;
typedef struct jet_prefix jet_prefix;

typedef struct {
  int32_t dtype;                /* JET_BF16, JET_FP32, JET_BF16_SINGLE, JET_F16 or JET_F16P */
  int32_t device;               /* HIP device ordinal */
  int64_t max_ctx;              /* max positions per sequence; 0 = the file's value */
  int64_t prefill_token_budget; /* max prefix tokens per prefill wave; 0 = no limit.
                                   Waves hold whole questions. */
  int64_t wave_token_budget;    /* max scored candidate tokens per scoring wave;
                                   0 = no limit. Waves hold whole candidates. */
  int64_t max_device_bytes;     /* cap on the library's device allocations; 0 = none */
  void *hip_stream;             /* hipStream_t to run on; NULL = the null stream */
  int32_t flags;                /* JET_FLAG_* */
  int32_t reserved;
} jet_load_opts;

/* Kernel classes reported by jet_stats (index into jet_stats.kernel_*). */
enum {
  JET_K_GEMM_QKV = 0,   /* attention / delta-rule input projections */
  JET_K_GEMM_O = 1,     /* output projection + residual add */
  JET_K_GEMM_GATEUP = 2,/* FFN gate/up projection + SwiGLU */
  JET_K_GEMM_DOWN = 3,  /* FFN down projection + residual add */
  JET_K_LMHEAD = 4,     /* LM head + online log-sum-exp */
  JET_K_ATTN_PREFIX = 5,/* causal attention over the prefix */
  JET_K_ATTN_CAND = 6,  /* candidate attention over shared prefix + own suffix */
  JET_K_GDN = 7,        /* gated delta-rule recurrence (prefix and candidates) */
  JET_K_OTHER = 8,      /* norms, RoPE, gathers, reductions, ... */
  JET_K_COUNT = 9
};

typedef struct {
  int64_t prefix_tokens;     /* prefix tokens evaluated (sum of P over prefill calls) */
  int64_t prefix_evals;      /* prefixes evaluated (questions over prefill calls) */
  int64_t cand_body_tokens;  /* candidate tokens run through the network (sum of m-1) */
  int64_t scored_tokens;     /* candidate tokens scored (sum of m) */
  int64_t lm_rows;           /* rows through the LM head (one per scored token) */
  int64_t prefill_waves;
  int64_t score_waves;
  int64_t kernel_launches[JET_K_COUNT];
  double kernel_ms[JET_K_COUNT];       /* only with JET_FLAG_KERNEL_TIMING */
  double kernel_flops[JET_K_COUNT];    /* algorithmic FLOPs launched per class */
  double kernel_bytes[JET_K_COUNT];    /* algorithmic HBM bytes launched per class */
} jet_stats;

/*
 * jet_model_load - read a model file and upload its weights.
 *   model_path: host string, path of a model file (JSON header + raw tensors):
 *     a dense or hybrid (gated delta-rule + attention) decoder whose FFNs are
 *     either SwiGLU or mixtures of experts (routed top-k experts plus an
 *     optional gated shared expert; Section 4.2 names routed experts).
 *   opts: host, may be NULL (defaults: JET_BF16, device 0, no limits, null stream).
 *   out: host, receives the model handle.
 * Errors: JET_E_IO (file), JET_E_INVALID (unsupported shape or dtype
 *   combination: an f32 file cannot be run in a bf16 mode; mixture-of-experts
 *   models run in the JET_FP32, JET_F16, JET_F16P and JET_BF16_SINGLE modes,
 *   not JET_BF16), JET_E_OOM, JET_E_DEVICE.
 */
int jet_model_load(const char *model_path, const jet_load_opts *opts, jet_model **out);

/*
 * jet_prefill_prefix - evaluate every question prefix once and retain its
 * state (Section 4.1; Figure 1, shared-prefix prefill).
 *   n_q: number of questions (>= 1).
 *   prefix_offsets: host, int64[n_q + 1]; question q owns
 *     prefix_tokens[prefix_offsets[q] .. prefix_offsets[q+1]); every P >= 1.
 *   prefix_tokens: host or device, int32[prefix_offsets[n_q]].
 *   out: host, receives the prefix handle. It holds the attention cache of
 *     every attention layer, the recurrent state and convolution tail of every
 *     delta-rule layer, and the final hidden row and log-sum-exp of each
 *     prefix's last position (which predicts every candidate's first token,
 *     Section 4.1). It is immutable and may serve many jet_score_candidates
 *     calls.
 * Errors: JET_E_INVALID (offsets, ids, P = 0), JET_E_CAPACITY (P > max_ctx),
 *   JET_E_OOM, JET_E_DEVICE.
 */
int jet_prefill_prefix(jet_model *model, int32_t n_q, const int64_t *prefix_offsets,
                       const int32_t *prefix_tokens, jet_prefix **out);

/*
 * jet_generate_trace - optional reasoning (Section 3.4; Figure 1): sample a
 * trace of n_steps tokens once per question and freeze it into the question's
 * retained prefix, so that later jet_score_candidates calls score every
 * candidate conditional on x_q || trace_q.
 *   prefix: made by jet_prefill_prefix from this model (or extended by an
 *     earlier call); extended in place: afterwards it describes prefixes of
 *     P_q + n_steps tokens (the retained attention caches are laid out again
 *     once per call, with room for the trace after each question).
 *   n_steps: tokens per question (>= 0; 0 changes nothing).
 *   temperature: >= 0 and finite. Token t of question q is
 *     argmax_v (z_v / temperature + G(seed, q, t, v)) over the full
 *     vocabulary, z the logits of the model's next-token distribution at
 *     that point; temperature 0 takes argmax_v z_v. Equal keys go to the
 *     lowest token id. G is Gumbel noise, -log(-log U), with U from output
 *     1 + (q << 38 | t << 18 | v) of a SplitMix64 stream seeded with `seed`
 *     (top 53 bits, mapped to the open interval (0, 1)); q is the question's
 *     index in the prefix, t = 0 .. n_steps - 1 within this call. The paper
 *     fixes no sampler; this Gumbel-max form draws from softmax(z /
 *     temperature) and needs no probabilities materialised.
 *   seed: any 64-bit value.
 *   out_tokens: host or device, int32[n_q * n_steps] (question-major), may be
 *     NULL.
 * Limits: n_steps < 2^20, n_q < 2^26, vocab <= 2^18; P_q + n_steps <= max_ctx.
 * Errors: JET_E_INVALID (arguments, a prefix of another model; the prefix is
 *   unchanged), JET_E_CAPACITY (max_ctx; unchanged), JET_E_OOM (before any
 *   change: unchanged), JET_E_DEVICE (the prefix is then in an unspecified
 *   state and may only be freed).
 */
int jet_generate_trace(jet_model *model, jet_prefix *prefix, int32_t n_steps, float temperature, uint64_t seed,
                       int32_t *out_tokens);

/*
 * jet_score_candidates - teacher-forced log-likelihood of every candidate
 * (Section 3.1 Eq. 1-2, Section 3.2 Eq. 3).
 *   q_cand_offsets: host, int64[n_q + 1] (n_q of the prefix); candidate j
 *     belongs to question q iff q_cand_offsets[q] <= j < q_cand_offsets[q+1].
 *     A question may have zero candidates.
 *   cand_tok_offsets: host, int64[N + 1], N = q_cand_offsets[n_q]; candidate j
 *     is cand_tokens[cand_tok_offsets[j] .. cand_tok_offsets[j+1]); m >= 1.
 *   cand_tokens: host or device, int32[cand_tok_offsets[N]].
 *   out_token_logprob: host or device, float[cand_tok_offsets[N]] or NULL;
 *     element i is log p of cand_tokens[i] given the prefix and the
 *     candidate's earlier tokens (same CSR indexing as cand_tokens).
 *   out_cand_sum: host or device, float[N]; s_j, summed in ascending t.
 * Token y_{c,t} sits at position P + t - 1. Candidates never see each other.
 * log p = z_y - log sum_v exp(z_v), with z_y the very fp32 logit that the
 * LM head's vocabulary tile adds into the log-sum-exp (one LM-head row per
 * scored token; the logits are never stored).
 * Errors: JET_E_INVALID (offsets, ids, m = 0, prefix of another model),
 *   JET_E_CAPACITY (P + m - 1 > max_ctx), JET_E_OOM, JET_E_DEVICE.
 */
int jet_score_candidates(jet_model *model, const jet_prefix *prefix,
                         const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                         const int32_t *cand_tokens, float *out_token_logprob,
                         float *out_cand_sum);

/* Size of the fixed per-device scratch of jet_score_candidates_noalloc. */
#define JET_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * jet_score_candidates_noalloc - jet_score_candidates for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc). Same arguments, results and
 * errors as jet_score_candidates, computed by the same kernels; no call of it
 * allocates or frees device memory. Its work buffers (token staging, row
 * tables, activations, attention caches of the candidate rows, log-sum-exp
 * partials) are carved from a fixed device array of
 * JET_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it has loaded
 * a model on, until the process ends; candidates run in waves of whole
 * candidates sized to fit it (at most the model's wave_token_budget tokens).
 * Limits: JET_E_CAPACITY when the call's token tables and one wave holding
 * its longest candidate do not fit the scratch (large mixture-of-experts
 * models need more than it holds). The scratch is shared by every call on
 * one GPU and keeps the last call's contents: calls that overlap on one GPU
 * (other threads, other models on the same device) race and must be
 * serialised by the caller. It still synchronises the model's stream before
 * returning, like every call here. Kernel timing (JET_FLAG_KERNEL_TIMING) is
 * not recorded for these calls.
 */
int jet_score_candidates_noalloc(jet_model *model, const jet_prefix *prefix,
                                 const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                                 const int32_t *cand_tokens, float *out_token_logprob,
                                 float *out_cand_sum);

/*
 * jet_decide - turn candidate scores into decisions (Section 3.2 Eq. 4,
 * Section 3.3 Eq. 5). Pure host function in fp64; touches no device.
 *   mode: JET_CHOICE, JET_BINARY (every question has exactly 2 candidates,
 *     index 0 = false, 1 = true) or JET_ORDINAL (>= 2 candidates, zero-based
 *     levels in the supplied order).
 *   q_cand_offsets: host, int64[n_q + 1]; each question needs >= 1 candidate.
 *   cand_sum: host, float[N].
 *   out_q: host, double[N] or NULL: q(c) = exp(s_c - M) / sum_d exp(s_d - M).
 *   out_choice: host, int32[n_q] or NULL: argmax s, lowest index on ties.
 *   out_value: host, double[n_q] or NULL: q(true) (JET_BINARY) or
 *     sum_i i q(i) (JET_ORDINAL); ignored for JET_CHOICE.
 * Errors: JET_E_INVALID.
 */
int jet_decide(int32_t mode, int32_t n_q, const int64_t *q_cand_offsets,
               const float *cand_sum, double *out_q, int32_t *out_choice,
               double *out_value);

/*
 * jet_answer_classes - label equivalence by answer text (Section 3.3: labels
 * whose answer text is the same receive the same likelihood and count as one
 * answer in evaluation). Two candidates of one question are equivalent when
 * their token sequences are identical. Host only; integer work.
 *   q_cand_offsets: host, int64[n_q + 1]; each question needs >= 1 candidate.
 *   cand_tok_offsets: host, int64[N + 1] (N = q_cand_offsets[n_q]); each
 *     candidate needs >= 1 token.
 *   cand_tokens: host, int32[cand_tok_offsets[N]].
 *   out_class: host, int32[N]: the zero-based index, within its question, of
 *     the first candidate with the same token sequence (its own index when no
 *     earlier candidate matches).
 * Errors: JET_E_INVALID.
 */
int jet_answer_classes(int32_t n_q, const int64_t *q_cand_offsets,
                       const int64_t *cand_tok_offsets, const int32_t *cand_tokens,
                       int32_t *out_class);

/*
 * jet_evaluate - accuracy and gold negative log-likelihood against reference
 * answers (Section 3.3 on equivalent labels; Section 5, evaluation protocol).
 * Pure host function in fp64.
 *   q_cand_offsets: host, int64[n_q + 1]; each question needs >= 1 candidate.
 *   cand_sum: host, float[N], the candidate scores s_c (finite).
 *   cand_class: host, int32[N] or NULL: answer class of every candidate
 *     (e.g. from jet_answer_classes), compared within a question only; NULL
 *     puts every candidate in a class of its own.
 *   gold: host, int32[n_q]: zero-based index of the reference answer's
 *     candidate within its question.
 *   out_correct: host, int32[n_q] or NULL: 1 when the predicted candidate
 *     (argmax s, lowest index on ties: jet_decide's choice; for a binary
 *     question the same as q(true) > 1/2) is in the gold candidate's class.
 *   out_gold_nll: host, double[n_q] or NULL: -ln of the summed probability
 *     q(c) (Eq. 4) of the gold class, evaluated in log form
 *     (M + ln sum_c e^(s_c - M)) - (M_g + ln sum_{c in gold class} e^(s_c - M_g))
 *     with M, M_g the maxima over the question and over the gold class, so it
 *     stays finite for any finite scores.
 *   out_accuracy / out_mean_nll: host, double or NULL: means over the
 *     questions, summed in question order.
 * Errors: JET_E_INVALID (offsets, gold out of range, non-finite score).
 */
int jet_evaluate(int32_t n_q, const int64_t *q_cand_offsets, const float *cand_sum,
                 const int32_t *cand_class, const int32_t *gold, int32_t *out_correct,
                 double *out_gold_nll, double *out_accuracy, double *out_mean_nll);

/*
 * jet_candidate_layout - the integer row layout that jet_score_candidates
 * builds (host only; exported so that it can be checked on its own).
 *   prefix_offsets / q_cand_offsets / cand_tok_offsets: host, as above.
 *   max_ctx: capacity check, P + m - 1 <= max_ctx (0 = no check).
 *   cap_rows: capacity of the row_* arrays.
 *   out_n_rows: host, receives the number of body rows R = sum_c (m_c - 1).
 *   row_pos / row_q / row_c / row_tok: host, int32[cap_rows] or NULL. Body row
 *     r carries token cand_tokens[row_tok[r]] = y_{c,t} (t <= m_c - 1) of
 *     candidate row_c[r] of question row_q[r], at position
 *     row_pos[r] = P_q + t - 1. Rows are ordered by candidate, then t.
 *   out_lm_row: host, int32[cand_tok_offsets[N]] or NULL: the row whose
 *     output distribution predicts token i: -(q + 1) for a first token
 *     (the last prefix position of question q), else the body row holding
 *     y_{c,t-1}.
 * Errors: JET_E_INVALID, JET_E_CAPACITY (also when R > cap_rows).
 */
int jet_candidate_layout(int32_t n_q, const int64_t *prefix_offsets,
                         const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                         int64_t max_ctx, int64_t cap_rows, int64_t *out_n_rows,
                         int32_t *row_pos, int32_t *row_q, int32_t *row_c,
                         int32_t *row_tok, int32_t *out_lm_row);

/* jet_stats - counters and per-kernel-class timings accumulated since load
 * (or since the last jet_stats_reset). out: host. */
int jet_stats_get(const jet_model *model, jet_stats *out);
int jet_stats_reset(jet_model *model);

/* Model facts: vocabulary size, layer count, max_ctx, compute dtype, and (fp16
 * modes) how many weights the load's fp16 conversion rounded: each matrix is
 * scaled by a power of two so its largest magnitude lies in [2^14, 2^15),
 * which keeps every bf16 value of magnitude >= 2^-32 times the matrix's
 * largest exact; smaller values round to fp16's step (0 in other modes).
 * Every out pointer may be NULL. */
int jet_model_info(const jet_model *model, int64_t *vocab, int64_t *n_layers,
                   int64_t *max_ctx, int32_t *dtype, int64_t *f16_inexact_weights);

/* Release a prefix (its device buffers go back to the model for the next
 * prefill) and a model (weights, work buffers, and the buffers of every
 * prefix of it not yet freed; see Ownership above). NULL is a no-op. */
/* jet_routes_get - the experts chosen by the most recent prefill (which = 0)
 * or scoring call (which = 1) of a mixture-of-experts model loaded with
 * JET_FLAG_RECORD_ROUTES (Section 4.2: routed experts). The top_k experts
 * kept by layer l for row r are out_ids[(l * rows + r) * top_k + j],
 * j < top_k, in the routing kernel's order (descending router logit, ties
 * to the lower expert index); rows that layer did not route hold -1.
 * Rows: prefill, the call's prefix tokens in input order (the last layer of
 * a prefill routes only each question's last token when that layer is an
 * attention layer); scoring, the candidate body rows in the order of
 * jet_candidate_layout. out_rows / out_layers / out_top_k: host, may be
 * NULL; out_ids: host, may be NULL (sizes only), else cap_ids >= layers *
 * rows * top_k elements. Errors: JET_E_INVALID (no experts, flag not set,
 * bad which), JET_E_CAPACITY (cap_ids too small). */
int jet_routes_get(const jet_model *model, int32_t which, int64_t *out_rows, int32_t *out_layers,
                   int32_t *out_top_k, int32_t *out_ids, int64_t cap_ids);

void jet_prefix_free(jet_prefix *prefix);
void jet_model_free(jet_model *model);

/* Message of the last failed call on this thread ("" if none). */
const char *jet_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* JET_H */

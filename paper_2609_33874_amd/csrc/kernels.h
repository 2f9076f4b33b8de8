// Host-side launchers of the HIP kernels (internal to the library).
// dtype: 0 = bf16 operands, 1 = fp32 operands, 2 = fp16 operands. Every
// launcher returns the launch status and enqueues work on `st` only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jetk {

enum { EPI_STORE_F32 = 0, EPI_RESID_ADD = 1, EPI_SWIGLU = 2, EPI_STORE_T = 3, EPI_QKV_ROPE = 4 };

// Epilogue of the attention input projection (EPI_QKV_ROPE): the columns are
// Hq query heads, Hkv key heads and Hkv value heads of head_dim 128; RoPE is
// applied to q and k in registers (pairs (d, d + 64), angle from pos[row])
// and q, K, V are stored in T like launch_rope_scatter stores them (with
// pair, (hi, lo) planes at +q_ps and +kv_ps), so the fp32 projection output
// is never written.
struct QkvRope {
  const int32_t *pos;
  const float *cos_t, *sin_t;  // [positions][64]
  int Hq, Hkv;
  void *q_out;
  int64_t q_ps;
  void *k_cache, *v_cache;  // [planes][Hkv][S][128]
  int64_t kv_ps, S, slot0;
};
// Split-K for GEMMs of few rows (fp16, plain operands): the number of K
// chunks worth running (1 = none), and the launch: S chunks of K / S columns
// each write fp32 partial sums to part [S][M][N], then a fixed-order sum
// stores them (EPI_STORE_F32) or adds them (EPI_RESID_ADD) to out.
int gemm_splitk_ways(int dtype, int pair, int M, int N, int K);
hipError_t launch_gemm_splitk(int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
                              int S, float *part, void *out, int64_t ldo, float oscale, hipStream_t st);
// Whether launch_gemm_qkv_rope can run this problem (head_dim 128 and a tile
// configuration whose waves cover whole heads).
bool gemm_qkv_rope_ok(int dtype, int pair, int M, int N, int head_dim);
hipError_t launch_gemm_qkv_rope(int dtype, const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N,
                                int K, int pair, float oscale, const QkvRope &r, hipStream_t st);

// C[M x N] (epilogue) A[M x K] * B[N x K]^T. K must be a multiple of
// gemm_k_step(dtype). pair (bf16 only): every A row holds a (hi, lo) bf16
// pair of the activations, [a_hi (K) | a_lo (K)], and C = (A_hi + A_lo) B^T.
// EPI_SWIGLU expects B rows interleaved in blocks of 32 gate rows then 32 up
// rows and writes silu(gate) * up to out[M x N/2] (T), or with pair to
// out[M x N] as [hi (N/2) | lo (N/2)]. Every product is multiplied by oscale
// before the epilogue (the inverse of a power-of-two weight scale).
int gemm_k_step(int dtype);
// fp16 A [M][K] times an int8 B operand: Bq [N][K] int8 (K bytes per row)
// holding the values q of a block-quantized matrix, Bs the fp16 bits of the
// scale of each (row, block of 32 K columns), a power of two, laid out as
// [K / 32][ceil(N / 128)][32][4] (row n = 128 g + 32 j + r at [.][g][r][j]);
// B = q * scale exactly in fp16. Epilogues as launch_gemm (no pairs).
// K must be a multiple of 32.
hipError_t launch_gemm_q8(int epi, const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N,
                          int K, void *out, int64_t ldo, float oscale, hipStream_t st);
// As launch_gemm_q8 with int4 values: Bq [N][K / 2] bytes, value 2i of a row
// in the low nibble of byte i, two's complement (-8..7).
hipError_t launch_gemm_q4(int epi, const void *A, int64_t lda, const void *Bq, const uint16_t *Bs, int M, int N,
                          int K, void *out, int64_t ldo, float oscale, hipStream_t st);
hipError_t launch_gemm(int dtype, int epi, const void *A, int64_t lda, const void *B, int64_t ldb, int M,
                       int N, int K, int pair, void *out, int64_t ldo, float oscale, hipStream_t st);

// LM head + online log-sum-exp: partial (max, sum) in base 2 per (split, row).
// lmhead_plan gives the vocabulary tiles per workgroup and the split count.
void lmhead_plan(int dtype, int V, int R, int *tiles_per_split, int *nsplit);
// F: [R][K] rows, or [R][2K] (hi, lo) pairs when pair. The logits are the
// products times wscale. target (int32[R], values in [0, V), or -1) and zt
// (float[R]) together or both NULL: zt[r] = the product of row r with
// W[target[r]] as accumulated for the log-sum-exp (unscaled); rows with -1
// are not written.
hipError_t launch_lmhead_lse(int dtype, const void *W, const void *F, int V, int R, int K, int pair,
                             int tiles_per_split, float wscale, float *part_m, float *part_s, const int32_t *target,
                             float *zt, hipStream_t st);
// lse[r] = ln(sum over splits) from the partials; with zt (else NULL),
// also ell[r] = zt[r] * wscale - lse[r].
hipError_t launch_lse_merge(const float *part_m, const float *part_s, int nsplit, int R, float *lse,
                            const float *zt, float wscale, float *ell, hipStream_t st);

// Attention work item: one (question, kv head, block of at most
// attn_slots_per_item query slots).
struct AttnItem {
  int32_t q, kvh, slot0, nslots, nkeys_pre;
};
// Per question of a call (device arrays indexed by the item's q).
struct AttnQuestions {
  const int32_t *qrow0;    // first query row of the question in Q / O
  const int32_t *nrows;    // query rows of the question
  const int64_t *pre_slot0;  // first prefix key slot in the prefix cache
  const int32_t *pre_len;  // prefix keys
  const int32_t *suf_row0; // first own-suffix key row in the call's K/V (candidate mode)
  const int32_t *suf_len;
};
// mode 0: causal prefix attention (query i of a question sees prefix keys 0..i).
// mode 1: candidate attention: every prefix key, plus the suffix keys of its
//         own candidate up to itself: rows i - row_t[i] + 1 .. i of the call's
//         K / V (rows are ordered by candidate, then position; row_n[i] is the
//         number of body rows of row i's candidate).
// pair: Q, K, V are (hi, lo) bf16 planes (the lo plane at +q_ps / +kp_ps /
// +ks_ps elements) and O rows hold [hi (Hq hd) | lo (Hq hd)].
struct AttnArgs {
  int mode;
  int pair;
  const void *Q;        // [planes][rows][Hq][hd]
  int64_t q_ps;
  void *O;              // [rows][o_ld]: head h, dim d at h * hd + d (lo part at (Hq + h) * hd + d)
  int64_t o_ld;
  const void *Kp, *Vp;  // prefix cache [planes][Hkv][S_pre][hd]
  int64_t s_pre, kp_ps;
  const void *Ks, *Vs;  // own-suffix keys of the call [planes][Hkv][S_suf][hd]
  int64_t s_suf, ks_ps;
  const int32_t *row_n, *row_t;  // per call row (candidate mode)
  AttnQuestions qs;
  const AttnItem *items;
  int n_items;
  int qb;  // blocks of 16 query slots per wave the items were built for: 64 qb slots per item
  int Hq, Hkv, hd;
  float scale;
};
hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t st);
// Largest query-slot count per work item launch_attention supports (64 or
// 128); the items of a launch hold at most 64 * AttnArgs::qb slots, qb being
// 1 or, where this returns 128, 2.
int attn_slots_per_item(int dtype, int pair);

// Gated delta-rule layers. Projection output x [R][ldx] = q~ (H dk) | k~ (H dk)
// | v~ (H dv) | z (H dv) | b (H) | a (H), fp32. hist[3 r + j - 1] names the
// input j rows earlier: >= 0 a row of x, -1 zero, <= -2 row (-2 - h) of tail
// [*][C], C = 2 H dk + H dv. tail_slot[r] >= 0 stores row r's pre-convolution
// channels at tail[tail_slot[r]] (prefix snapshot); tail_slot may be NULL.
struct GdnConvArgs {
  const float *x;
  int64_t ldx;
  const int32_t *hist, *tail_slot;
  float *tail;
  const float *conv_w, *A_log, *dt_bias;  // conv_w [C][4], w[c][3] multiplies the current row
  int H, dk, dv;
  float *q, *k, *v, *alpha, *beta;        // [R][H][dk], [R][H][dk], [R][H][dv], [R][H], [R][H]
};
hipError_t launch_gdn_conv(const GdnConvArgs &g, int R, hipStream_t st);
// One recurrence per (sequence, head): rows row0 .. row0 + len - 1; the state
// starts from S_init[init] (or zero if init < 0) and, if fin >= 0, the final
// state is written to S_fin[fin]. States are [*][H][dv][dk] fp32; dk = dv = 128.
struct GdnSeq {
  int32_t row0, len, init, fin;
};
struct GdnRecurArgs {
  const GdnSeq *seqs;
  const float *q, *k, *v, *alpha, *beta;
  int H, dk, dv;
  const float *S_init;
  float *S_fin;
  float *o;  // [R][H][dv]
};
hipError_t launch_gdn_recur(const GdnRecurArgs &g, int nseq, hipStream_t st);
// The same recurrence in chunks of 32 steps on the matrix cores (fp16
// operands, or (hi, lo) bf16 operand pairs with pair != 0; fp32 accumulation
// and state): for long sequences (prefill).
hipError_t launch_gdn_chunk(const GdnRecurArgs &g, int nseq, int pair, hipStream_t st);
// y [R][H dv] (T; [hi | lo] pairs with pair) = RMSNorm(o) * w * silu(z), z at column zoff of x.
hipError_t launch_gdn_out(int dtype, int pair, const float *o, const float *x, int64_t ldx, int zoff, const float *w,
                          float eps, int H, int dv, int R, void *y, hipStream_t st);

// resid[r][:] = E[ids[idx ? idx[r] : r]][:] (as fp32).
hipError_t launch_embed(int dtype, const void *E, const int32_t *ids, const int32_t *idx, int R, int d,
                        float *resid, hipStream_t st);
// out[r][:] = x[src][:] / sqrt(mean(x[src]^2) + eps) * g, src = map ? map[r] : r; out in T,
// as [hi (d) | lo (d)] rows when pair.
hipError_t launch_rmsnorm(int dtype, int pair, const float *x, const int32_t *map, const float *g, int R, int d,
                          float eps, void *out, hipStream_t st);
// qkv fp32 [R][(Hq + 2 Hkv) hd] -> q (T) [R][Hq][hd] with RoPE, K (RoPE) and V
// into the cache [Hkv][S][hd] at slot slot0 + r, angles from pos[r]. With
// pair, lo planes follow at +q_ps (q) and +kv_ps (caches) elements.
hipError_t launch_rope_scatter(int dtype, int pair, const float *qkv, const int32_t *pos, const float *cos_t,
                               const float *sin_t, int R, int Hq, int Hkv, int hd, void *q_out, int64_t q_ps,
                               void *k_cache, void *v_cache, int64_t kv_ps, int64_t S, int64_t slot0,
                               hipStream_t st);
// dst row i = f_body row lm_row[i] - row_base or, when lm_row[i] < 0,
// f_last row -lm_row[i] - 1 (rows of row_bytes bytes, a multiple of 16).
hipError_t launch_token_rows(const int32_t *lm_row, int n, int row_base, const void *f_body, const void *f_last,
                             int64_t row_bytes, void *dst, hipStream_t st);
// s[c] = sum of ell[off[c] - off[0] .. off[c+1] - off[0]) in ascending order.
hipError_t launch_segment_sum(const float *ell, const int64_t *off, int n_cand, float *s, hipStream_t st);
// dst row i = src row idx[i], rows of row_bytes (a multiple of 16) bytes.
hipError_t launch_gather_rows(const void *src, int64_t row_bytes, const int32_t *idx, int n, void *dst,
                              hipStream_t st);
// Counts ids outside [0, V) into *bad (int, must be zeroed by the caller).
hipError_t launch_count_bad_ids(const int32_t *ids, int64_t n, int V, int *bad, hipStream_t st);
// dst[i] = src[i] with fp32 -> T conversion (weights upload helpers).
hipError_t launch_convert_f32(int dtype, const float *src, int64_t n, void *dst, hipStream_t st);
hipError_t launch_convert_bf16_to_f32(const uint16_t *src, int64_t n, float *dst, hipStream_t st);
// dst[i] = src[i] * scale as fp16 (bf16 bits in; exact when scale is a power
// of two that keeps every value inside the fp16 normal range).
// dst = fp16(bf16 src * scale); adds the number of values that did not convert
// exactly to *inexact (device counter)
hipError_t launch_convert_bf16_to_f16(const uint16_t *src, int64_t n, float scale, void *dst,
                                      unsigned long long *inexact, hipStream_t st);


// ---- reasoning trace (decode) ----
// Question q's rows [offs[q], offs[q + 1]) of each of nblk blocks of an
// [nblk][S_old] cache of rows (row_bytes each, a multiple of 16) are copied
// to rows offs[q] + q * extra + i of an [nblk][S_new] cache (room for extra
// rows after each question).
hipError_t launch_kv_relayout(const void *src, void *dst, const int64_t *offs, int n_q, int nblk, int64_t S_old,
                              int64_t S_new, int64_t row_bytes, int extra, hipStream_t st);
// Row r of each block of tmp [nblk][R] to row slot[r] of cache [nblk][S].
hipError_t launch_kv_append(const void *tmp, void *cache, const int32_t *slot, int R, int nblk, int64_t S,
                            int64_t row_bytes, hipStream_t st);
// tokens[r * ld_tok] = argmax_v (z[r][v] / tau + G(seed, q0 + r, t, v)), or
// argmax_v z[r][v] when tau = 0; lowest v among equal keys, -1 if no logit is
// a number. G: Gumbel noise from SplitMix64 output 1 + (q << 38 | t << 18 | v)
// of the stream seeded with seed (V < 2^18, t < 2^20, q < 2^26).
// scratch: sample_scratch_bytes(R) bytes of device memory.
int sample_scratch_bytes(int R);
hipError_t launch_sample(const float *logits, int64_t ldl, int R, int V, double tau, uint64_t seed, int q0, int t,
                         void *scratch, int32_t *tokens, int64_t ld_tok, hipStream_t st);

// ---- mixture-of-experts FFN (k_moe.hip) ----
constexpr int kMoeMaxExperts = 512;
constexpr int kMoeMaxTopK = 16;

// Router logits [R][ldl] fp32 (E expert columns, then the shared expert's gate
// logit at column E when shared_gate is set) -> sel/wts [R][top_k] (experts by
// logit, lowest index first among equals; softmax over the kept logits),
// shared_gate[R] = sigmoid(logit E).
struct MoeRouteArgs {
  const float *logits;
  int64_t ldl;
  int R, E, top_k;
  int *sel;
  float *wts;
  float *shared_gate;
};
hipError_t launch_moe_route(const MoeRouteArgs &a, hipStream_t st);
// Entries of the choice list per chunk of kMoeChunk entries.
constexpr int kMoeChunk = 1024;
int moe_chunks(int R, int top_k);
// From the routing (sel [R][top_k]): segment starts (per-expert totals
// rounded up to bm), the expert of each of max_tiles row tiles (-1 past the
// last segment) into tile_group, and the place of every entry
// i = row * top_k + j in its expert's segment, in list order, into
// slot_of[R * top_k]. chunk_hist and chunk_base hold moe_chunks(R, top_k) * E
// ints each.
hipError_t launch_moe_plan(const int *sel, int R, int top_k, int E, int bm, int max_tiles, int *tile_group,
                           int *chunk_hist, int *chunk_base, int *slot_of, hipStream_t st);
// Row i / top_k of x copied to row slot_of[i] of xp (rows of row_bytes, a
// multiple of 16).
hipError_t launch_moe_scatter(const void *x, int64_t row_bytes, int R, int top_k, const int *slot_of, void *xp,
                              hipStream_t st);
// resid[r] += sum_j wts[r][j] y[slot_of[r][j]] + gate[r] ys[r] (ys fp32, may be
// null); y in the compute type of dtype.
hipError_t launch_moe_combine(int dtype, const void *y, const int *slot_of, const float *wts, int top_k,
                              const float *ys, const float *gate, int R, int d, float *resid, hipStream_t st);
// Grouped GEMM: row tile t of A (tiles of gemm_group_rows(dtype, big) rows) is
// multiplied by B + tile_group[t] * group_stride (elements); tiles with
// tile_group -1 are skipped. Otherwise as launch_gemm (no pair operands).
// big (fp16 only): 256-row tiles, for segments of many rows.
int gemm_group_rows(int dtype, int big);
hipError_t launch_gemm_grouped(int dtype, int big, int epi, const void *A, int64_t lda, const void *B, int64_t ldb,
                               int64_t group_stride, const int *tile_group, int M, int N, int K, void *out,
                               int64_t ldo, float oscale, hipStream_t st);

}  // namespace jetk

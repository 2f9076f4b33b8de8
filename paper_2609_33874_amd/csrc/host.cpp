// Request validation, row layout and decision rules (host only).
//
// Validation follows Figure 1 (invalid requests produce errors): offsets must
// be well formed, every prefix and candidate non-empty, no sequence longer
// than the context (the question is never truncated, Section 4.1).
// The layout places token y_{c,t} at position P_q + t - 1; its distribution
// comes from the row one position earlier, which for t = 1 is the last prefix
// position (Section 4.1: the prefix output supplies first-token probabilities).
#include "host.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>

namespace jet {

static thread_local std::string g_last_error;

void set_error(const std::string &msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

Status check_offsets(const int64_t *off, int64_t n, int64_t min_len, const char *what) {
  if (!off) return Status::err(JET_E_INVALID, std::string(what) + ": null offsets");
  if (n < 0) return Status::err(JET_E_INVALID, std::string(what) + ": negative count");
  if (off[0] != 0) return Status::err(JET_E_INVALID, std::string(what) + ": offsets[0] != 0");
  for (int64_t i = 0; i < n; ++i) {
    int64_t len = off[i + 1] - off[i];
    if (len < 0)
      return Status::err(JET_E_INVALID, std::string(what) + ": offsets decrease at " + std::to_string(i));
    if (len < min_len)
      return Status::err(JET_E_INVALID, std::string(what) + ": empty segment " + std::to_string(i));
    if (len > INT32_MAX) return Status::err(JET_E_INVALID, std::string(what) + ": segment too long");
  }
  return Status::ok();
}

Status check_ids_host(const int32_t *ids, int64_t n, int64_t vocab, const char *what) {
  if (n > 0 && !ids) return Status::err(JET_E_INVALID, std::string(what) + ": null token array");
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= vocab)
      return Status::err(JET_E_INVALID, std::string(what) + ": token id " + std::to_string(ids[i]) +
                                            " at " + std::to_string(i) + " outside [0, vocab)");
  return Status::ok();
}

Status build_cand_layout(int32_t n_q, const int64_t *prefix_offsets,
                         const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                         int64_t max_ctx, CandLayout *L) {
  if (n_q < 1) return Status::err(JET_E_INVALID, "n_q must be >= 1");
  Status s = check_offsets(prefix_offsets, n_q, 1, "prefix_offsets");
  if (!s) return s;
  s = check_offsets(q_cand_offsets, n_q, 0, "q_cand_offsets");
  if (!s) return s;
  const int64_t N = q_cand_offsets[n_q];
  s = check_offsets(cand_tok_offsets, N, 1, "cand_tok_offsets");
  if (!s) return s;
  if (N > INT32_MAX || cand_tok_offsets[N] > INT32_MAX)
    return Status::err(JET_E_INVALID, "too many candidate tokens");
  L->n_q = n_q;
  L->n_cand = N;
  L->n_tok = cand_tok_offsets[N];
  int64_t rows = 0;
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t P = prefix_offsets[q + 1] - prefix_offsets[q];
    for (int64_t c = q_cand_offsets[q]; c < q_cand_offsets[q + 1]; ++c) {
      const int64_t m = cand_tok_offsets[c + 1] - cand_tok_offsets[c];
      if (max_ctx > 0 && P + m - 1 > max_ctx)
        return Status::err(JET_E_CAPACITY, "candidate " + std::to_string(c) + ": P + m - 1 = " +
                                               std::to_string(P + m - 1) + " exceeds max_ctx " +
                                               std::to_string(max_ctx));
      rows += m - 1;
    }
  }
  if (rows > INT32_MAX) return Status::err(JET_E_INVALID, "too many body rows");
  L->n_rows = rows;
  L->row_pos.resize(rows);
  L->row_q.resize(rows);
  L->row_c.resize(rows);
  L->row_tok.resize(rows);
  L->row_t.resize(rows);
  L->lm_row.resize(L->n_tok);
  L->cand_row0.resize(N);
  int64_t r = 0;
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t P = prefix_offsets[q + 1] - prefix_offsets[q];
    for (int64_t c = q_cand_offsets[q]; c < q_cand_offsets[q + 1]; ++c) {
      const int64_t t0 = cand_tok_offsets[c];
      const int64_t m = cand_tok_offsets[c + 1] - t0;
      L->cand_row0[c] = (int32_t)r;
      // token t (1-based) is predicted by: t == 1 -> last prefix row; else body row of t-1
      L->lm_row[t0] = -(q + 1);
      for (int64_t t = 1; t <= m - 1; ++t) {
        L->row_pos[r] = (int32_t)(P + t - 1);
        L->row_q[r] = q;
        L->row_c[r] = (int32_t)c;
        L->row_tok[r] = (int32_t)(t0 + t - 1);
        L->row_t[r] = (int32_t)t;
        L->lm_row[t0 + t] = (int32_t)r;
        ++r;
      }
    }
  }
  return Status::ok();
}

}  // namespace jet

using namespace jet;

extern "C" int jet_candidate_layout(int32_t n_q, const int64_t *prefix_offsets,
                                    const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                                    int64_t max_ctx, int64_t cap_rows, int64_t *out_n_rows,
                                    int32_t *row_pos, int32_t *row_q, int32_t *row_c,
                                    int32_t *row_tok, int32_t *out_lm_row) {
  clear_error();
  if (!out_n_rows) return fail(Status::err(JET_E_INVALID, "out_n_rows is NULL"));
  CandLayout L;
  Status s = build_cand_layout(n_q, prefix_offsets, q_cand_offsets, cand_tok_offsets, max_ctx, &L);
  if (!s) return fail(s);
  if (L.n_rows > cap_rows && (row_pos || row_q || row_c || row_tok))
    return fail(Status::err(JET_E_CAPACITY, "cap_rows smaller than the number of body rows"));
  *out_n_rows = L.n_rows;
  const size_t rb = sizeof(int32_t) * (size_t)L.n_rows;
  if (row_pos && rb) std::memcpy(row_pos, L.row_pos.data(), rb);
  if (row_q && rb) std::memcpy(row_q, L.row_q.data(), rb);
  if (row_c && rb) std::memcpy(row_c, L.row_c.data(), rb);
  if (row_tok && rb) std::memcpy(row_tok, L.row_tok.data(), rb);
  if (out_lm_row && L.n_tok) std::memcpy(out_lm_row, L.lm_row.data(), sizeof(int32_t) * L.n_tok);
  return JET_OK;
}

// Eq. 4 (Section 3.2) and Eq. 5 with the rules of Section 3.3, in fp64.
extern "C" int jet_decide(int32_t mode, int32_t n_q, const int64_t *q_cand_offsets,
                          const float *cand_sum, double *out_q, int32_t *out_choice,
                          double *out_value) {
  clear_error();
  if (mode != JET_CHOICE && mode != JET_BINARY && mode != JET_ORDINAL)
    return fail(Status::err(JET_E_INVALID, "unknown decision mode"));
  if (n_q < 1) return fail(Status::err(JET_E_INVALID, "n_q must be >= 1"));
  Status s = check_offsets(q_cand_offsets, n_q, 1, "q_cand_offsets");
  if (!s) return fail(s);
  const int64_t N = q_cand_offsets[n_q];
  if (!cand_sum) return fail(Status::err(JET_E_INVALID, "cand_sum is NULL"));
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t K = q_cand_offsets[q + 1] - q_cand_offsets[q];
    if (mode == JET_BINARY && K != 2)
      return fail(Status::err(JET_E_INVALID, "binary decision needs exactly 2 candidates (question " +
                                                 std::to_string(q) + ")"));
    if (mode == JET_ORDINAL && K < 2)
      return fail(Status::err(JET_E_INVALID, "ordinal decision needs >= 2 levels (question " +
                                                 std::to_string(q) + ")"));
  }
  for (int64_t i = 0; i < N; ++i)
    if (!std::isfinite(cand_sum[i]))
      return fail(Status::err(JET_E_INVALID, "non-finite candidate score at " + std::to_string(i)));
  std::vector<double> qv;
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t a = q_cand_offsets[q], b = q_cand_offsets[q + 1];
    int64_t best = a;
    double M = cand_sum[a];
    for (int64_t c = a + 1; c < b; ++c)
      if ((double)cand_sum[c] > M) { M = cand_sum[c]; best = c; }
    qv.assign(b - a, 0.0);
    double z = 0.0;
    for (int64_t c = a; c < b; ++c) { qv[c - a] = std::exp((double)cand_sum[c] - M); z += qv[c - a]; }
    for (auto &v : qv) v /= z;
    if (out_q)
      for (int64_t c = a; c < b; ++c) out_q[c] = qv[c - a];
    if (out_choice) out_choice[q] = (int32_t)(best - a);
    if (out_value) {
      if (mode == JET_BINARY) out_value[q] = qv[1];
      else if (mode == JET_ORDINAL) {
        double e = 0.0;
        for (int64_t i = 0; i < b - a; ++i) e += (double)i * qv[i];
        out_value[q] = e;
      }
    }
  }
  return JET_OK;
}

// Equivalent labels (Section 3.3): identical token sequences within a question.
extern "C" int jet_answer_classes(int32_t n_q, const int64_t *q_cand_offsets,
                                  const int64_t *cand_tok_offsets, const int32_t *cand_tokens,
                                  int32_t *out_class) {
  clear_error();
  if (n_q < 1) return fail(Status::err(JET_E_INVALID, "n_q must be >= 1"));
  Status s = check_offsets(q_cand_offsets, n_q, 1, "q_cand_offsets");
  if (!s) return fail(s);
  const int64_t N = q_cand_offsets[n_q];
  s = check_offsets(cand_tok_offsets, N, 1, "cand_tok_offsets");
  if (!s) return fail(s);
  if (!cand_tokens) return fail(Status::err(JET_E_INVALID, "cand_tokens is NULL"));
  if (!out_class) return fail(Status::err(JET_E_INVALID, "out_class is NULL"));
  std::vector<int32_t> cls(N);
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t a = q_cand_offsets[q], b = q_cand_offsets[q + 1];
    for (int64_t c = a; c < b; ++c) {
      const int64_t len = cand_tok_offsets[c + 1] - cand_tok_offsets[c];
      int64_t first = c;
      for (int64_t d = a; d < c && first == c; ++d) {
        if (cls[d] != d - a) continue;  // compare with class representatives only
        if (cand_tok_offsets[d + 1] - cand_tok_offsets[d] != len) continue;
        if (std::equal(cand_tokens + cand_tok_offsets[c], cand_tokens + cand_tok_offsets[c + 1],
                       cand_tokens + cand_tok_offsets[d]))
          first = d;
      }
      cls[c] = (int32_t)(first - a);
    }
  }
  std::memcpy(out_class, cls.data(), sizeof(int32_t) * (size_t)N);
  return JET_OK;
}

// Accuracy and gold NLL over the normalised candidate distribution (Eq. 4),
// with equivalent labels pooled (Section 3.3; Section 5, evaluation protocol).
extern "C" int jet_evaluate(int32_t n_q, const int64_t *q_cand_offsets, const float *cand_sum,
                            const int32_t *cand_class, const int32_t *gold, int32_t *out_correct,
                            double *out_gold_nll, double *out_accuracy, double *out_mean_nll) {
  clear_error();
  if (n_q < 1) return fail(Status::err(JET_E_INVALID, "n_q must be >= 1"));
  Status s = check_offsets(q_cand_offsets, n_q, 1, "q_cand_offsets");
  if (!s) return fail(s);
  const int64_t N = q_cand_offsets[n_q];
  if (!cand_sum) return fail(Status::err(JET_E_INVALID, "cand_sum is NULL"));
  if (!gold) return fail(Status::err(JET_E_INVALID, "gold is NULL"));
  for (int32_t q = 0; q < n_q; ++q)
    if (gold[q] < 0 || gold[q] >= q_cand_offsets[q + 1] - q_cand_offsets[q])
      return fail(Status::err(JET_E_INVALID, "gold index " + std::to_string(gold[q]) +
                                                 " outside the candidates of question " + std::to_string(q)));
  for (int64_t i = 0; i < N; ++i)
    if (!std::isfinite(cand_sum[i]))
      return fail(Status::err(JET_E_INVALID, "non-finite candidate score at " + std::to_string(i)));
  auto cls = [&](int64_t c, int64_t a) -> int64_t { return cand_class ? (int64_t)cand_class[c] : c - a; };
  double acc = 0.0, nll_sum = 0.0;
  for (int32_t q = 0; q < n_q; ++q) {
    const int64_t a = q_cand_offsets[q], b = q_cand_offsets[q + 1];
    const int64_t g = cls(a + gold[q], a);
    int64_t best = a;
    double M = cand_sum[a], Mg = -INFINITY;
    for (int64_t c = a + 1; c < b; ++c)
      if ((double)cand_sum[c] > M) { M = cand_sum[c]; best = c; }
    for (int64_t c = a; c < b; ++c)
      if (cls(c, a) == g) Mg = std::max(Mg, (double)cand_sum[c]);
    double z = 0.0, zg = 0.0;
    for (int64_t c = a; c < b; ++c) {
      z += std::exp((double)cand_sum[c] - M);
      if (cls(c, a) == g) zg += std::exp((double)cand_sum[c] - Mg);
    }
    const int correct = cls(best, a) == g;
    const double nll = (M + std::log(z)) - (Mg + std::log(zg));
    if (out_correct) out_correct[q] = correct;
    if (out_gold_nll) out_gold_nll[q] = nll;
    acc += correct;
    nll_sum += nll;
  }
  if (out_accuracy) *out_accuracy = acc / n_q;
  if (out_mean_nll) *out_mean_nll = nll_sum / n_q;
  return JET_OK;
}

extern "C" const char *jet_last_error(void) { return g_last_error.c_str(); }

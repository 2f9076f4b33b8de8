// Host-side checks of the scoring library's CPU code (request validation, the
// integer row layout, the decision and evaluation rules, the model-file
// reader), built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py. Every function under test is called with
// valid inputs (results checked against hand values or a direct restatement
// of the documented layout) and with malformed ones (must fail cleanly).
//
// Usage: host_checks <valid model file> [malformed model file ...]
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>
#include <vector>

#include "jet.h"
#include "model_file.h"

static int g_fail = 0;
#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "%s:%d: CHECK failed: %s\n", __FILE__, __LINE__, #cond); \
      ++g_fail;                                                              \
    }                                                                        \
  } while (0)

static bool near(double a, double b, double tol) { return std::fabs(a - b) <= tol; }

static void check_decide() {
  // worked example of Section 3.2: likelihoods 0.06 and 0.02 -> 0.75 / 0.25
  {
    const int64_t qo[] = {0, 2};
    const float s[] = {std::log(0.06f), std::log(0.02f)};
    double q[2], v[1];
    int32_t ch[1];
    CHECK(jet_decide(JET_ORDINAL, 1, qo, s, q, ch, v) == JET_OK);
    CHECK(near(q[0], 0.75, 1e-6) && near(q[1], 0.25, 1e-6) && ch[0] == 0 && near(v[0], 0.25, 1e-6));
    CHECK(jet_decide(JET_BINARY, 1, qo, s, q, ch, v) == JET_OK);
    CHECK(near(v[0], 0.25, 1e-6));
  }
  // ties: lowest index; K equal levels: (K - 1) / 2
  {
    const int64_t qo[] = {0, 3, 8};
    const float s[] = {-1.0f, -0.5f, -0.5f, -2.f, -2.f, -2.f, -2.f, -2.f};
    double q[8], v[2];
    int32_t ch[2];
    CHECK(jet_decide(JET_ORDINAL, 2, qo, s, q, ch, v) == JET_OK);
    CHECK(ch[0] == 1 && ch[1] == 0 && near(v[1], 2.0, 1e-12));
    CHECK(near(q[3] + q[4] + q[5] + q[6] + q[7], 1.0, 1e-12));
  }
  // malformed requests fail and write nothing
  {
    const int64_t bad0[] = {1, 2}, dec[] = {0, 2, 1}, ok2[] = {0, 2}, ok3[] = {0, 3};
    const float s[] = {0.f, NAN, 0.f};
    double q[3] = {7, 7, 7};
    int32_t ch[2] = {9, 9};
    CHECK(jet_decide(JET_CHOICE, 1, bad0, s, q, ch, nullptr) == JET_E_INVALID);
    CHECK(jet_decide(JET_CHOICE, 2, dec, s, q, ch, nullptr) == JET_E_INVALID);
    CHECK(jet_decide(JET_CHOICE, 1, ok2, s, q, ch, nullptr) == JET_E_INVALID);  // NaN
    CHECK(jet_decide(JET_BINARY, 1, ok3, s, q, ch, nullptr) == JET_E_INVALID);  // K != 2
    CHECK(jet_decide(JET_CHOICE, 0, ok2, s, q, ch, nullptr) == JET_E_INVALID);
    CHECK(jet_decide(JET_CHOICE, 1, nullptr, s, q, ch, nullptr) == JET_E_INVALID);
    CHECK(jet_decide(JET_CHOICE, 1, ok2, nullptr, q, ch, nullptr) == JET_E_INVALID);
    CHECK(jet_decide(9, 1, ok2, s, q, ch, nullptr) == JET_E_INVALID);
    CHECK(q[0] == 7 && ch[0] == 9 && jet_last_error()[0] != '\0');
  }
}

// Random CSR requests: the layout against the documented placement (token
// y_{c,t} at position P_q + t - 1, predicted by the last prefix row for t = 1
// and by the body row holding y_{c,t-1} otherwise).
static void check_layout(std::mt19937_64 &rng) {
  for (int it = 0; it < 300; ++it) {
    const int32_t nq = 1 + (int32_t)(rng() % 6);
    std::vector<int64_t> po{0}, qo{0}, co{0};
    for (int q = 0; q < nq; ++q) {
      po.push_back(po.back() + 1 + (int64_t)(rng() % 40));
      const int K = (int)(rng() % 4);
      qo.push_back(qo.back() + K);
      for (int k = 0; k < K; ++k) co.push_back(co.back() + 1 + (int64_t)(rng() % 9));
    }
    const int64_t N = qo.back(), NT = co.back();
    int64_t rows = -1;
    CHECK(jet_candidate_layout(nq, po.data(), qo.data(), co.data(), 0, 0, &rows, nullptr, nullptr, nullptr,
                               nullptr, nullptr) == JET_OK);
    CHECK(rows == NT - N);
    std::vector<int32_t> pos(rows + 1), rq(rows + 1), rc(rows + 1), rt(rows + 1), lm(NT + 1);
    if (rows > 0) {
      CHECK(jet_candidate_layout(nq, po.data(), qo.data(), co.data(), 0, rows - 1, &rows, pos.data(),
                                 rq.data(), rc.data(), rt.data(), lm.data()) == JET_E_CAPACITY);
    }
    CHECK(jet_candidate_layout(nq, po.data(), qo.data(), co.data(), 0, rows, &rows, pos.data(), rq.data(),
                               rc.data(), rt.data(), lm.data()) == JET_OK);
    int64_t r = 0;
    for (int32_t q = 0; q < nq; ++q) {
      const int64_t P = po[q + 1] - po[q];
      for (int64_t c = qo[q]; c < qo[q + 1]; ++c) {
        const int64_t m = co[c + 1] - co[c];
        CHECK(lm[co[c]] == -(q + 1));
        for (int64_t t = 1; t < m; ++t, ++r) {
          CHECK(pos[r] == P + t - 1 && rq[r] == q && rc[r] == c && rt[r] == co[c] + t - 1);
          CHECK(lm[co[c] + t] == r);
        }
      }
    }
    CHECK(r == rows);
    // capacity: the longest sequence one short of fitting
    int64_t longest = 0;
    for (int32_t q = 0; q < nq; ++q)
      for (int64_t c = qo[q]; c < qo[q + 1]; ++c)
        longest = std::max<int64_t>(longest, po[q + 1] - po[q] + co[c + 1] - co[c] - 1);
    if (N > 0)
      CHECK(jet_candidate_layout(nq, po.data(), qo.data(), co.data(), longest - 1, 0, &rows, nullptr, nullptr,
                                 nullptr, nullptr, nullptr) == JET_E_CAPACITY);
    // malformed: an empty prefix, an empty candidate, decreasing offsets
    std::vector<int64_t> po2 = po;
    po2[1] = 0;
    CHECK(jet_candidate_layout(nq, po2.data(), qo.data(), co.data(), 0, 0, &rows, nullptr, nullptr, nullptr,
                               nullptr, nullptr) == JET_E_INVALID);
    if (N > 0) {
      std::vector<int64_t> co2 = co;
      co2[1] = co2[0];
      CHECK(jet_candidate_layout(nq, po.data(), qo.data(), co2.data(), 0, 0, &rows, nullptr, nullptr, nullptr,
                                 nullptr, nullptr) == JET_E_INVALID);
      std::vector<int64_t> qo2 = qo;
      qo2[nq] = -1;
      CHECK(jet_candidate_layout(nq, po.data(), qo2.data(), co.data(), 0, 0, &rows, nullptr, nullptr, nullptr,
                                 nullptr, nullptr) == JET_E_INVALID);
    }
  }
}

// Equivalent labels and evaluation on random questions over a small alphabet.
static void check_evaluation(std::mt19937_64 &rng) {
  for (int it = 0; it < 200; ++it) {
    const int32_t nq = 1 + (int32_t)(rng() % 5);
    std::vector<int64_t> qo{0}, co{0};
    std::vector<int32_t> tok, gold;
    for (int q = 0; q < nq; ++q) {
      const int K = 1 + (int)(rng() % 5);
      qo.push_back(qo.back() + K);
      gold.push_back((int32_t)(rng() % K));
      for (int k = 0; k < K; ++k) {
        const int m = 1 + (int)(rng() % 2);
        for (int j = 0; j < m; ++j) tok.push_back((int32_t)(rng() % 2));
        co.push_back(co.back() + m);
      }
    }
    const int64_t N = qo.back();
    std::vector<int32_t> cls(N, -1);
    CHECK(jet_answer_classes(nq, qo.data(), co.data(), tok.data(), cls.data()) == JET_OK);
    for (int32_t q = 0; q < nq; ++q)
      for (int64_t c = qo[q]; c < qo[q + 1]; ++c) {
        // the first candidate of the question with the same token sequence
        int64_t first = c;
        for (int64_t d = qo[q]; d < c && first == c; ++d)
          if (co[d + 1] - co[d] == co[c + 1] - co[c] &&
              std::equal(tok.begin() + co[c], tok.begin() + co[c + 1], tok.begin() + co[d]))
            first = d;
        CHECK(cls[c] == first - qo[q]);
      }
    std::vector<float> s(N);
    for (auto &v : s) v = -(float)(rng() % 50) / 7.0f;
    std::vector<int32_t> correct(nq, -1);
    std::vector<double> nll(nq, -1);
    double acc = -1, mnll = -1;
    CHECK(jet_evaluate(nq, qo.data(), s.data(), cls.data(), gold.data(), correct.data(), nll.data(), &acc,
                       &mnll) == JET_OK);
    double sum_nll = 0;
    for (int32_t q = 0; q < nq; ++q) {
      CHECK(correct[q] == 0 || correct[q] == 1);
      CHECK(nll[q] >= -1e-12 && std::isfinite(nll[q]));
      // one label alone (or all labels with the gold text): NLL 0
      if (qo[q + 1] - qo[q] == 1) CHECK(near(nll[q], 0.0, 1e-12) && correct[q] == 1);
      sum_nll += nll[q];
    }
    CHECK(near(mnll, sum_nll / nq, 1e-12) && acc >= 0 && acc <= 1);
    std::vector<int32_t> badgold = gold;
    badgold[0] = (int32_t)(qo[1] - qo[0]);
    CHECK(jet_evaluate(nq, qo.data(), s.data(), cls.data(), badgold.data(), correct.data(), nll.data(), &acc,
                       &mnll) == JET_E_INVALID);
  }
}

static void check_model_files(int argc, char **argv) {
  jet::ModelHeader h;
  jet::Status st = jet::read_model_header(argv[1], &h);
  CHECK((bool)st);
  if (!st) std::fprintf(stderr, "valid model: %s\n", st.msg.c_str());
  CHECK(h.n_layers > 0 && (int64_t)h.layer_is_gdn.size() == h.n_layers && !h.tensors.empty());
  auto it = h.tensors.find("final_norm");
  CHECK(it != h.tensors.end());
  if (it != h.tensors.end()) {
    std::vector<float> g(it->second.numel());
    CHECK((bool)jet::read_tensor_bytes(argv[1], it->second, g.data()));
    for (float v : g) CHECK(v == 1.0f);
    jet::TensorInfo past = it->second;
    past.offset = INT64_C(1) << 40;  // beyond the end of the file
    CHECK(!jet::read_tensor_bytes(argv[1], past, g.data()));
  }
  for (int i = 2; i < argc; ++i) {
    jet::ModelHeader hb;
    jet::Status sb = jet::read_model_header(argv[i], &hb);
    if (sb) std::fprintf(stderr, "malformed model accepted: %s\n", argv[i]);
    CHECK(!sb && sb.code == JET_E_IO);
  }
  jet::ModelHeader hn;
  CHECK(!jet::read_model_header("/nonexistent/model.jetm", &hn));
}

int main(int argc, char **argv) {
  if (argc < 2) {
    std::fprintf(stderr, "usage: %s model.jetm [malformed ...]\n", argv[0]);
    return 2;
  }
  std::mt19937_64 rng(20260921);
  check_decide();
  check_layout(rng);
  check_evaluation(rng);
  check_model_files(argc, argv);
  std::printf("host checks: %d failure(s)\n", g_fail);
  return g_fail ? 1 : 0;
}

// Host-only helpers of the scoring library: error reporting, request
// validation and the integer row layout. Nothing here touches a GPU, so this
// part also builds with a plain C++ compiler (and sanitizers) for host tests.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/jet.h"

namespace jet {

// Thread-local message behind jet_last_error().
void set_error(const std::string &msg);
void clear_error();

struct Status {
  int code = JET_OK;
  std::string msg;
  static Status ok() { return {}; }
  static Status err(int c, std::string m) { return {c, std::move(m)}; }
  explicit operator bool() const { return code == JET_OK; }
};

// Returns the error code after recording the message.
inline int fail(const Status &s) {
  set_error(s.msg);
  return s.code;
}

// Validates a CSR offset array: length n+1, off[0] == 0, non-decreasing,
// and (if min_len > 0) every segment at least min_len long.
Status check_offsets(const int64_t *off, int64_t n, int64_t min_len, const char *what);

// Token ids in [0, vocab).
Status check_ids_host(const int32_t *ids, int64_t n, int64_t vocab, const char *what);

// Row layout of a scoring call (see jet_candidate_layout in jet.h).
struct CandLayout {
  int64_t n_q = 0, n_cand = 0, n_tok = 0, n_rows = 0;
  std::vector<int32_t> row_pos, row_q, row_c, row_tok, row_t;
  std::vector<int32_t> lm_row;        // per scored token
  std::vector<int32_t> cand_row0;     // first body row of each candidate
};

Status build_cand_layout(int32_t n_q, const int64_t *prefix_offsets,
                         const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                         int64_t max_ctx, CandLayout *out);

}  // namespace jet

// Model file: 8-byte magic "JETMDL01", uint64 header length, JSON header,
// then raw tensors at the absolute offsets listed in the header.
#pragma once

#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "host.h"

namespace jet {

struct TensorInfo {
  std::string name;
  bool bf16 = false;  // storage: bf16 bits (true) or float32
  // block-quantized storage ("q8" / "q4"): int8 values [.., cols] (q4: two
  // per byte [.., cols / 2], value 2i in the low nibble of byte i, -8..7)
  // then one int8 exponent per block of 32 values of a row [.., cols / 32];
  // the weight is q * 2^e
  bool q8 = false;
  int qbits = 0;  // 8 or 4 when q8
  std::vector<int64_t> shape;
  int64_t offset = 0, nbytes = 0;
  int64_t numel() const {
    int64_t n = 1;
    for (auto s : shape) n *= s;
    return n;
  }
};

struct ModelHeader {
  bool hybrid = false;
  bool bf16 = false;  // matrix storage dtype
  bool q8 = false;    // block-quantized matrices ("q8" or "q4"; the others bf16)
  int qbits = 0;      // 8 or 4 when q8
  int64_t d = 0, n_layers = 0, n_heads = 0, n_kv_heads = 0, head_dim = 0, ffn = 0, vocab = 0;
  int64_t gdn_heads = 0, gdn_dk = 0, gdn_dv = 0, conv_kernel = 0, max_ctx = 0;
  // mixture-of-experts FFN (n_experts > 0): top_k routed experts of moe_ffn
  // hidden units per row, plus a gated shared expert of shared_ffn (0: none)
  int64_t n_experts = 0, top_k = 0, moe_ffn = 0, shared_ffn = 0;
  double rms_eps = 1e-6, rope_theta = 1e6;
  std::vector<int> layer_is_gdn;
  std::map<std::string, TensorInfo> tensors;
};

Status read_model_header(const std::string &path, ModelHeader *h);

// Reads a tensor's raw bytes into dst (dst must hold t.nbytes).
Status read_tensor_bytes(const std::string &path, const TensorInfo &t, void *dst);

}  // namespace jet

// Internal runtime state of the scoring library (opaque behind jet.h).
#pragma once

#include <hip/hip_runtime.h>

#include <map>
#include <string>
#include <vector>

#include "host.h"
#include "kernels.h"
#include "model_file.h"
#include "noalloc.h"

struct jet_model;
struct jet_prefix;

namespace jet {

struct Layer {
  bool gdn = false;
  float *attn_norm = nullptr, *ffn_norm = nullptr;
  void *w_qkv = nullptr;   // attention: [Hq hd + 2 Hkv hd][d] (q rows, k rows, v rows)
  void *w_o = nullptr;     // [d][Hq hd] (attention) or [d][H dv] (delta rule)
  void *w_gu = nullptr;    // [2F][d], blocks of 32 gate rows then 32 up rows
  void *w_down = nullptr;  // [d][F]
  // inverse weight scales of w_qkv / w_in, w_o, w_gu, w_down (fp16 mode: the
  // stored matrices are the file's values times a power of two; else 1)
  float is_qkv = 1.0f, is_o = 1.0f, is_gu = 1.0f, is_down = 1.0f;
  // block-quantized model in the fp16 mode: w_qkv, w_o, w_gu and w_down hold
  // int8 values [N][K] and these their fp16 block scales (see launch_gemm_q8)
  uint16_t *s_qkv = nullptr, *s_o = nullptr, *s_gu = nullptr, *s_down = nullptr;
  // gated delta-rule layers
  void *w_in = nullptr;    // [n_in][d]: q, k, v (conv channels), z, b, a, zero pad
  int64_t n_in = 0;
  float *conv_w = nullptr; // [C][kc], C = 2 H dk + H dv
  float *A_log = nullptr, *dt_bias = nullptr, *gdn_norm = nullptr;
  // mixture-of-experts FFN (replaces w_gu / w_down)
  void *w_router = nullptr;  // [n_router][d]: E expert rows, the shared expert's gate row, zero pad
  int64_t n_router = 0;
  void *w_egu = nullptr;     // [E][2 Fe][d], each expert's gate/up interleaved like w_gu
  void *w_edown = nullptr;   // [E][d][Fe]
  void *w_sgu = nullptr, *w_sdown = nullptr;  // shared expert, like w_gu / w_down
  float is_router = 1.0f, is_egu = 1.0f, is_edown = 1.0f, is_sgu = 1.0f, is_sdown = 1.0f;
};

struct DevBuf {
  void *p = nullptr;
  size_t bytes = 0;
};

struct PendingTimer {
  int cls;
  hipEvent_t a, b;
};

}  // namespace jet

struct jet_model {
  jet::ModelHeader h;
  std::string path;
  int dtype = JET_BF16;  // requested mode
  int kdt = 0;           // kernel element type: 0 = bf16, 1 = fp32, 2 = fp16
  int edt = 0;           // element type of the embedding table (bf16 in the fp16 mode)
  int pair = 1;          // FFN, delta-rule and final-norm activations as (hi, lo) pairs
  int np = 2;            // planes per such activation element (2 with pair)
  int apair = 1;         // attention-side activations (attention-layer inputs, q, K/V caches,
                         // probabilities, attention output) as (hi, lo) pairs
  int anp = 2;           // planes per attention-side element
  int device = 0;
  hipStream_t st = nullptr;
  int64_t max_ctx = 0, prefill_budget = 0, wave_budget = 0, max_bytes = 0;
  int flags = 0;
  size_t esz = 2;  // bytes per compute element
  size_t bytes_used = 0;
  void *embed = nullptr, *lm_head = nullptr;
  float is_lm = 1.0f;  // inverse weight scale of lm_head
  int64_t f16_inexact = 0;  // fp16 modes: weights whose scaled fp16 value is not the file's bf16 value
  float *final_norm = nullptr;
  std::vector<jet::Layer> layers;
  float *rope_cos = nullptr, *rope_sin = nullptr;
  std::map<std::string, jet::DevBuf> ws;
  std::vector<jet::PendingTimer> pending;
  std::vector<hipEvent_t> event_pool;
  std::vector<void *> weight_allocs;
  // device buffers of freed prefixes, kept for the next prefill (sizes in bytes)
  std::vector<std::pair<size_t, void *>> pool;
  jet_stats stats{};
  // prefixes made from this model and not yet freed; freeing the model frees
  // their device buffers and detaches them (their handle stays valid to free)
  std::vector<jet_prefix *> live;
  // JET_FLAG_RECORD_ROUTES: experts chosen per (layer, row) by the latest
  // prefill (0) and scoring (1) call, [n_layers][rows][top_k], -1 = not routed
  std::vector<int32_t> routes[2];
  int64_t route_rows[2] = {0, 0};
  // set around each FFN call while recording: the record, the layer, and the
  // record row of each of the call's rows
  int rt_which = -1;
  int64_t rt_layer = 0;
  std::vector<int64_t> rt_rowmap;
  // jet_score_candidates_noalloc: while `arena` is set, work buffers are
  // carved from it (a fixed device scratch) instead of the growable workspace:
  // buffer name -> (offset, bytes); entries at or past `arena_mark` are
  // dropped at every scoring wave
  char *arena = nullptr;
  size_t arena_cap = 0, arena_top = 0, arena_mark = 0;
  std::map<std::string, std::pair<size_t, size_t>> arena_map;
  hipError_t scratch_status = hipSuccess;  // lookup of the device's scratch at load
  bool splitk = false;  // run_gemm may split K (decode steps of jet_generate_trace)
};

struct jet_prefix {
  jet_model *m = nullptr;            // NULL once the model has been freed
  int32_t n_q = 0;
  std::vector<int64_t> prefix_offsets;
  int64_t T = 0;                     // total prefix tokens
  std::vector<void *> kcache, vcache;  // per layer (attention layers only), [planes][Hkv][T][hd]
  std::vector<float *> S_pre;        // per layer (delta-rule only), [n_q][H][dv][dk]
  std::vector<float *> conv_tail;    // per layer (delta-rule only), [n_q][kc-1][C]
  void *f_last = nullptr;            // [n_q][planes * d] final-normed last prefix rows
  std::vector<std::pair<void *, size_t>> allocs;  // (buffer, allocated bytes)
  size_t bytes = 0;
};

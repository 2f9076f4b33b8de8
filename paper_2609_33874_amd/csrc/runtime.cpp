// Scoring runtime: weight upload, shared-prefix prefill, batched candidate
// scoring, and the C ABI entry points of jet.h.
//
// Flow (Section 4.1, Figure 1): jet_prefill_prefix runs every question prefix
// once, keeps its attention cache / recurrent state and the final hidden row
// of its last position; jet_score_candidates runs all candidate tokens of a
// wave as one batch against that retained state, computes full-vocabulary
// log-sum-exps without writing logits (Section 4.2) and sums each candidate's
// log-probabilities (Eq. 3).
#include "runtime.h"

#include <algorithm>
#include <cmath>
#include <cstring>

using namespace jet;

#define HIPC(x)                                                                                      \
  do {                                                                                               \
    hipError_t e_ = (x);                                                                             \
    if (e_ != hipSuccess)                                                                            \
      return Status::err(e_ == hipErrorOutOfMemory ? JET_E_OOM : JET_E_DEVICE,                       \
                         std::string(#x) + ": " + hipGetErrorString(e_));                           \
  } while (0)

#define TRY(x)                 \
  do {                         \
    Status s_ = (x);           \
    if (!s_) return s_;        \
  } while (0)

namespace {

// ---------------------------------------------------------------------------
// device memory with an optional byte budget
// ---------------------------------------------------------------------------

Status dmalloc(jet_model *m, size_t bytes, void **p) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  if (m->max_bytes > 0 && m->bytes_used + bytes > (size_t)m->max_bytes)
    return Status::err(JET_E_OOM, "device byte budget exceeded (" + std::to_string(m->bytes_used + bytes) +
                                      " > " + std::to_string(m->max_bytes) + ")");
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return Status::err(JET_E_OOM, "hipMalloc(" + std::to_string(bytes) + "): " + hipGetErrorString(e));
  }
  m->bytes_used += bytes;
  return Status::ok();
}

void dfree(jet_model *m, void *p, size_t bytes) {
  if (!p) return;
  (void)hipFree(p);
  m->bytes_used -= std::min(m->bytes_used, bytes == 0 ? (size_t)256 : bytes);
}

// Grow-only named workspace buffer; while the model has an arena (the
// allocation-free entry point), a buffer carved from it instead.
Status ws(jet_model *m, const char *name, size_t bytes, void **p) {
  if (m->arena) {
    auto it = m->arena_map.find(name);
    if (it != m->arena_map.end() && it->second.second >= bytes) {
      *p = m->arena + it->second.first;
      return Status::ok();
    }
    const size_t off = (m->arena_top + 255) & ~(size_t)255;
    if (off > m->arena_cap || bytes > m->arena_cap - off)
      return Status::err(JET_E_CAPACITY, std::string("scratch of ") + std::to_string(m->arena_cap) +
                                             " bytes exhausted (buffer " + name + ")");
    m->arena_map[name] = {off, bytes};
    m->arena_top = off + bytes;
    *p = m->arena + off;
    return Status::ok();
  }
  DevBuf &b = m->ws[name];
  if (b.bytes < bytes) {
    dfree(m, b.p, b.bytes);
    b = DevBuf{};
    size_t want = bytes + bytes / 8;
    TRY(dmalloc(m, want, &b.p));
    b.bytes = want;
  }
  *p = b.p;
  return Status::ok();
}

template <typename T>
Status ws_t(jet_model *m, const char *name, size_t n, T **p) {
  void *v;
  TRY(ws(m, name, n * sizeof(T), &v));
  *p = (T *)v;
  return Status::ok();
}

template <typename T>
Status upload(jet_model *m, const char *name, const std::vector<T> &v, T **p) {
  TRY(ws_t<T>(m, name, std::max<size_t>(v.size(), 1), p));
  if (!v.empty()) HIPC(hipMemcpyAsync(*p, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice, m->st));
  return Status::ok();
}

bool is_device_ptr(const void *p) {
  if (!p) return false;
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged;
}

// ---------------------------------------------------------------------------
// kernel timing (HIP events around each launch when JET_FLAG_KERNEL_TIMING)
// ---------------------------------------------------------------------------

struct KTimer {
  jet_model *m;
  int cls;
  hipEvent_t a = nullptr, b = nullptr;
  KTimer(jet_model *m_, int cls_, double flops, double bytes) : m(m_), cls(cls_) {
    m->stats.kernel_launches[cls]++;
    m->stats.kernel_flops[cls] += flops;
    m->stats.kernel_bytes[cls] += bytes;
    if ((m->flags & JET_FLAG_KERNEL_TIMING) && !m->arena) {
      a = get();
      b = get();
      (void)hipEventRecord(a, m->st);
    }
  }
  hipEvent_t get() {
    if (!m->event_pool.empty()) {
      hipEvent_t e = m->event_pool.back();
      m->event_pool.pop_back();
      return e;
    }
    hipEvent_t e;
    (void)hipEventCreate(&e);
    return e;
  }
  ~KTimer() {
    if (a) {
      (void)hipEventRecord(b, m->st);
      m->pending.push_back({cls, a, b});
    }
  }
};

void drain_timers(jet_model *m) {
  for (auto &p : m->pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) m->stats.kernel_ms[p.cls] += ms;
    else (void)hipGetLastError();
    m->event_pool.push_back(p.a);
    m->event_pool.push_back(p.b);
  }
  m->pending.clear();
}

Status sync(jet_model *m) {
  HIPC(hipStreamSynchronize(m->st));
  drain_timers(m);
  return Status::ok();
}

#define LAUNCH(x) HIPC(x)

// ---------------------------------------------------------------------------
// model loading
// ---------------------------------------------------------------------------

struct Loader {
  jet_model *m;
  std::vector<char> host;
  unsigned long long *inexact = nullptr;  // device counter of inexact fp16 conversions

  TensorInfo cur;  // the tensor last read, as the caller sees it

  // A tensor's bytes into `host`. Block-quantized (q8) tensors arrive as the
  // bf16 bits of their weights q * 2^e, which bf16 holds exactly (8
  // significant bits, fp32's exponent range).
  Status read(const std::string &name, const TensorInfo **ti) {
    auto it = m->h.tensors.find(name);
    if (it == m->h.tensors.end()) return Status::err(JET_E_IO, "model file lacks tensor " + name);
    cur = it->second;
    *ti = &cur;
    host.resize((size_t)it->second.nbytes);
    TRY(read_tensor_bytes(m->path, it->second, host.data()));
    if (!cur.q8) return Status::ok();
    const int64_t n = cur.numel();
    std::vector<char> raw;
    raw.swap(host);
    host.resize((size_t)n * 2);
    const int8_t *q = reinterpret_cast<const int8_t *>(raw.data()), *e = q + n * cur.qbits / 8;
    uint16_t *dst = reinterpret_cast<uint16_t *>(host.data());
    for (int64_t i = 0; i < n; ++i) {
      const float w = std::ldexp((float)qval(q, i, cur.qbits), (int)e[i / 32]);
      uint32_t u;
      std::memcpy(&u, &w, 4);
      dst[i] = (uint16_t)(u >> 16);  // exact: the low 16 bits are zero
    }
    cur.q8 = false;
    cur.bf16 = true;
    cur.nbytes = n * 2;
    return Status::ok();
  }

  // Block-quantized weight rows kept as int8 for the fused GEMM path.
  struct Q8Rows {
    std::vector<int8_t> q, e;  // [rows][cols] (one value per byte), [rows][cols / 32]
    int64_t rows = 0, cols = 0;
    int bits = 8;  // storage on the device: int8, or int4 two per byte
  };
  // Value i of block-quantized storage (int8, or int4 two per byte, low
  // nibble first, two's complement).
  static int qval(const int8_t *q, int64_t i, int bits) {
    if (bits == 8) return q[i];
    const int b = ((const uint8_t *)q)[i >> 1], u = (i & 1) ? b >> 4 : b & 15;
    return u >= 8 ? u - 16 : u;
  }
  Status q8_read(const std::string &name, Q8Rows *w) {
    auto it = m->h.tensors.find(name);
    if (it == m->h.tensors.end()) return Status::err(JET_E_IO, "model file lacks tensor " + name);
    const TensorInfo &t = it->second;
    if (!t.q8 || t.shape.size() != 2) return Status::err(JET_E_IO, name + ": expected a q8 matrix");
    std::vector<char> raw((size_t)t.nbytes);
    TRY(read_tensor_bytes(m->path, t, raw.data()));
    w->rows = t.shape[0];
    w->cols = t.shape[1];
    w->bits = t.qbits;
    const int64_t n = w->rows * w->cols, qb = n * t.qbits / 8;
    const int8_t *q = reinterpret_cast<const int8_t *>(raw.data());
    w->q.resize((size_t)n);
    for (int64_t i = 0; i < n; ++i) w->q[(size_t)i] = (int8_t)qval(q, i, t.qbits);  // one value per byte here
    w->e.assign(q + qb, q + qb + n / 32);
    return Status::ok();
  }
  // Rows of several matrices stacked; with interleave, gate/up style: blocks
  // of 32 rows of the first then 32 rows of the second.
  static Q8Rows q8_stack(const std::vector<Q8Rows> &parts, bool interleave) {
    Q8Rows out;
    out.cols = parts[0].cols;
    out.bits = parts[0].bits;
    const int64_t eb = out.cols / 32;
    for (auto &p : parts) out.rows += p.rows;
    out.q.resize((size_t)(out.rows * out.cols));
    out.e.resize((size_t)(out.rows * eb));
    auto put = [&](int64_t dst_row, const Q8Rows &p, int64_t src_row, int64_t nrows) {
      std::memcpy(&out.q[(size_t)(dst_row * out.cols)], &p.q[(size_t)(src_row * out.cols)], (size_t)(nrows * out.cols));
      std::memcpy(&out.e[(size_t)(dst_row * eb)], &p.e[(size_t)(src_row * eb)], (size_t)(nrows * eb));
    };
    int64_t r = 0;
    if (interleave) {
      for (int64_t b = 0; b < parts[0].rows / 32; ++b)
        for (auto &p : parts) {
          put(r, p, b * 32, 32);
          r += 32;
        }
    } else {
      for (auto &p : parts) {
        put(r, p, 0, p.rows);
        r += p.rows;
      }
    }
    return out;
  }
  // int8 values to the device as they are; the scale of each (row, block) as
  // fp16 bits of 2^(e + k), k a power-of-two scale of the whole matrix that
  // puts its largest weight in [2^14, 2^15) (as the fp16 conversion does):
  // q * 2^(e + k) is then exact in fp16 for e + k >= -24; blocks below that
  // (far below the matrix's largest weight) round and are counted.
  Status put_q8(const Q8Rows &w, void **q_dev, uint16_t **s_dev, float *inv_scale) {
    const int64_t N = w.rows, K = w.cols, KB = K / 32, NG = (N + 127) / 128;
    int top = -1000;  // exponent of the largest weight: max over blocks of e + bit length of max|q| - 1
    for (int64_t r = 0; r < N; ++r)
      for (int64_t b = 0; b < KB; ++b) {
        int mq = 0;
        for (int64_t i = 0; i < 32; ++i) mq = std::max(mq, std::abs((int)w.q[(size_t)(r * K + b * 32 + i)]));
        if (mq == 0) continue;
        int bl = 0;
        while ((1 << bl) <= mq) ++bl;
        top = std::max(top, (int)w.e[(size_t)(r * KB + b)] + bl - 1);
      }
    const int k = top == -1000 ? 0 : 14 - top;
    *inv_scale = std::ldexp(1.0f, -k);
    std::vector<uint16_t> sc((size_t)(KB * NG * 128), 0);
    int64_t inexact = 0;
    for (int64_t r = 0; r < N; ++r)
      for (int64_t b = 0; b < KB; ++b) {
        const int ek = (int)w.e[(size_t)(r * KB + b)] + k;
        if (ek > 15) return Status::err(JET_E_INVALID, "q8 block scale beyond fp16 range");
        uint16_t bits = 0;
        if (ek >= -14) bits = (uint16_t)((ek + 15) << 10);
        else if (ek >= -24) bits = (uint16_t)(1u << (ek + 24));
        else
          for (int64_t i = 0; i < 32; ++i) inexact += w.q[(size_t)(r * K + b * 32 + i)] != 0;
        const int64_t g = r / 128, j = (r / 32) % 4, rr = r % 32;
        sc[(size_t)(((b * NG + g) * 32 + rr) * 4 + j)] = bits;
      }
    m->f16_inexact += inexact;
    std::vector<int8_t> packed;
    const std::vector<int8_t> *dev = &w.q;
    if (w.bits == 4) {  // two values per byte, value 2i in the low nibble of byte i
      packed.resize(w.q.size() / 2);
      for (size_t i = 0; i < packed.size(); ++i)
        packed[i] = (int8_t)((w.q[2 * i] & 15) | ((w.q[2 * i + 1] & 15) << 4));
      dev = &packed;
    }
    TRY(dmalloc(m, dev->size(), q_dev));
    m->weight_allocs.push_back(*q_dev);
    HIPC(hipMemcpy(*q_dev, dev->data(), dev->size(), hipMemcpyHostToDevice));
    TRY(dmalloc(m, sc.size() * 2, (void **)s_dev));
    m->weight_allocs.push_back(*s_dev);
    HIPC(hipMemcpy(*s_dev, sc.data(), sc.size() * 2, hipMemcpyHostToDevice));
    return Status::ok();
  }

  // Uploads host bytes of `n` elements stored as bf16 (src_bf16) or f32 into a
  // new device array of the compute dtype (as stored, with keep_bf16). In the
  // fp16 mode the bf16 values are multiplied by 2^k, k chosen so that the
  // largest magnitude lands in [2^14, 2^15): nothing overflows, and every value
  // of magnitude at least 2^-32 times the largest (all bf16 bits of it above
  // fp16's smallest step 2^-24) converts exactly. *inv_scale receives 2^-k.
  Status put_matrix(const void *src, int64_t n, bool src_bf16, void **out, float *inv_scale = nullptr,
                    bool keep_bf16 = false) {
    if (inv_scale) *inv_scale = 1.0f;
    const int kdt = keep_bf16 ? 0 : m->kdt;
    const size_t dst_bytes = (size_t)n * (kdt == 1 ? 4 : 2);
    TRY(dmalloc(m, dst_bytes, out));
    m->weight_allocs.push_back(*out);
    if (kdt == 2) {
      if (!src_bf16) return Status::err(JET_E_INVALID, "the fp16 mode needs a bf16 model file");
      const uint16_t *h = reinterpret_cast<const uint16_t *>(src);
      uint16_t mx = 0;  // largest magnitude (bf16 bits without the sign order like the magnitudes)
      for (int64_t i = 0; i < n; ++i) mx = std::max<uint16_t>(mx, (uint16_t)(h[i] & 0x7fffu));
      if (mx >= 0x7f80u) return Status::err(JET_E_INVALID, "weights hold inf or NaN");
      int k = 0;
      if (mx != 0) {
        const int e = (int)(mx >> 7) - 127;  // max |w| in [2^e, 2^(e+1)) (normal numbers)
        k = std::min(14 - e, 100);
      }
      const float scale = std::ldexp(1.0f, k);
      if (inv_scale) *inv_scale = std::ldexp(1.0f, -k);
      void *tmp;
      TRY(dmalloc(m, (size_t)n * 2, &tmp));
      hipError_t e = hipMemcpy(tmp, src, (size_t)n * 2, hipMemcpyHostToDevice);
      if (e == hipSuccess) e = jetk::launch_convert_bf16_to_f16((const uint16_t *)tmp, n, scale, *out, inexact, m->st);
      if (e == hipSuccess) e = hipStreamSynchronize(m->st);
      dfree(m, tmp, (size_t)n * 2);
      HIPC(e);
      return Status::ok();
    }
    if ((kdt == 0) == src_bf16) {
      HIPC(hipMemcpy(*out, src, dst_bytes, hipMemcpyHostToDevice));
      return Status::ok();
    }
    // bf16 file in fp32 mode: upload bits, widen exactly on the device
    void *tmp;
    TRY(dmalloc(m, (size_t)n * 2, &tmp));
    hipError_t e = hipMemcpy(tmp, src, (size_t)n * 2, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = jetk::launch_convert_bf16_to_f32((const uint16_t *)tmp, n, (float *)*out, m->st);
    if (e == hipSuccess) e = hipStreamSynchronize(m->st);
    dfree(m, tmp, (size_t)n * 2);
    HIPC(e);
    return Status::ok();
  }

  Status matrix(const std::string &name, void **out, float *inv_scale = nullptr, bool keep_bf16 = false) {
    const TensorInfo *ti;
    TRY(read(name, &ti));
    return put_matrix(host.data(), ti->numel(), ti->bf16, out, inv_scale, keep_bf16);
  }

  Status vec_f32(const std::string &name, float **out, int64_t expect) {
    const TensorInfo *ti;
    TRY(read(name, &ti));
    if (ti->bf16 || ti->numel() != expect) return Status::err(JET_E_IO, name + ": expected f32[" + std::to_string(expect) + "]");
    TRY(dmalloc(m, (size_t)expect * 4, (void **)out));
    m->weight_allocs.push_back(*out);
    HIPC(hipMemcpy(*out, host.data(), (size_t)expect * 4, hipMemcpyHostToDevice));
    return Status::ok();
  }

  // Any stored tensor as an fp32 device array (bf16 storage widened exactly).
  Status f32_array(const std::string &name, float **out, int64_t expect) {
    const TensorInfo *ti;
    TRY(read(name, &ti));
    if (ti->numel() != expect) return Status::err(JET_E_IO, name + ": unexpected size");
    std::vector<float> f((size_t)expect);
    if (ti->bf16) {
      const uint16_t *h = reinterpret_cast<const uint16_t *>(host.data());
      for (int64_t i = 0; i < expect; ++i) {
        const uint32_t u = (uint32_t)h[i] << 16;
        std::memcpy(&f[(size_t)i], &u, 4);
      }
    } else {
      std::memcpy(f.data(), host.data(), (size_t)expect * 4);
    }
    TRY(dmalloc(m, (size_t)expect * 4, (void **)out));
    m->weight_allocs.push_back(*out);
    HIPC(hipMemcpy(*out, f.data(), (size_t)expect * 4, hipMemcpyHostToDevice));
    return Status::ok();
  }

  // Concatenates matrices row-wise (all [rows_i][d]) and pads to `pad_rows`.
  Status concat(const std::vector<std::string> &names, int64_t d, int64_t pad_rows, void **out, int64_t *rows_out,
                float *inv_scale) {
    std::vector<char> all;
    bool bf = m->h.bf16;
    const size_t es = bf ? 2 : 4;
    int64_t rows = 0;
    for (auto &nm : names) {
      const TensorInfo *ti;
      TRY(read(nm, &ti));
      if (ti->shape.size() != 2 || ti->shape[1] != d) return Status::err(JET_E_IO, nm + ": bad shape");
      all.insert(all.end(), host.begin(), host.end());
      rows += ti->shape[0];
    }
    if (pad_rows > rows) {
      all.resize((size_t)pad_rows * d * es, 0);
      rows = pad_rows;
    }
    if (rows_out) *rows_out = rows;
    return put_matrix(all.data(), rows * d, bf, out, inv_scale);
  }

  // Expert tensors [E][F][d] gate and up -> [E][2F][d], each expert's rows
  // interleaved like gate_up.
  Status expert_gate_up(const std::string &g, const std::string &u, int64_t E, int64_t F, int64_t d, void **out,
                        float *inv_scale) {
    const bool bf = m->h.bf16;
    const size_t es = bf ? 2 : 4, row = (size_t)d * es;
    const TensorInfo *ti;
    TRY(read(g, &ti));
    if (ti->numel() != E * F * d) return Status::err(JET_E_IO, g + ": unexpected size");
    std::vector<char> gate = host;
    TRY(read(u, &ti));
    if (ti->numel() != E * F * d) return Status::err(JET_E_IO, u + ": unexpected size");
    std::vector<char> all((size_t)(2 * E * F) * row);
    for (int64_t e = 0; e < E; ++e) {
      const size_t src = (size_t)(e * F) * row, dst = (size_t)(e * 2 * F) * row;
      for (int64_t b = 0; b < F / 32; ++b) {
        std::memcpy(&all[dst + (size_t)(2 * b) * 32 * row], &gate[src + (size_t)b * 32 * row], 32 * row);
        std::memcpy(&all[dst + (size_t)(2 * b + 1) * 32 * row], &host[src + (size_t)b * 32 * row], 32 * row);
      }
    }
    return put_matrix(all.data(), 2 * E * F * d, bf, out, inv_scale);
  }

  // gate/up interleaved in blocks of 32 rows: [g0..g31, u0..u31, g32.., u32.., ...]
  Status gate_up(const std::string &g, const std::string &u, int64_t F, int64_t d, void **out, float *inv_scale) {
    const bool bf = m->h.bf16;
    const size_t es = bf ? 2 : 4, row = (size_t)d * es;
    const TensorInfo *ti;
    TRY(read(g, &ti));
    std::vector<char> gate = host;
    TRY(read(u, &ti));
    std::vector<char> all((size_t)2 * F * row);
    for (int64_t b = 0; b < F / 32; ++b) {
      std::memcpy(&all[(size_t)(2 * b) * 32 * row], &gate[(size_t)b * 32 * row], 32 * row);
      std::memcpy(&all[(size_t)(2 * b + 1) * 32 * row], &host[(size_t)b * 32 * row], 32 * row);
    }
    return put_matrix(all.data(), 2 * F * d, bf, out, inv_scale);
  }
};

Status check_shapes(const ModelHeader &h, int dtype) {
  const int64_t bk = dtype == JET_FP32 ? 32 : 64;
  if (dtype != JET_FP32 && !h.bf16)
    return Status::err(JET_E_INVALID, "an f32 model file cannot run in a bf16 mode (its weights are not bf16 values)");
  if (h.head_dim != 32 && h.head_dim != 64 && h.head_dim != 128)
    return Status::err(JET_E_INVALID, "head_dim must be 32, 64 or 128");
  if (h.n_kv_heads < 1 || h.n_heads % h.n_kv_heads != 0) return Status::err(JET_E_INVALID, "n_heads % n_kv_heads != 0");
  if (h.d % bk || (h.n_heads * h.head_dim) % bk || h.ffn % bk)
    return Status::err(JET_E_INVALID, "d_model, n_heads*head_dim and ffn must be multiples of " + std::to_string(bk));
  if (h.ffn % 32) return Status::err(JET_E_INVALID, "ffn must be a multiple of 32");
  if (h.q8) {
    if (h.hybrid || h.n_experts)
      return Status::err(JET_E_INVALID, "block-quantized models must be dense decoders without experts");
    if (dtype != JET_F16 && dtype != JET_FP32)
      return Status::err(JET_E_INVALID, "block-quantized models run in the JET_F16 and JET_FP32 modes");
    if (h.d % 128 || (h.n_heads * h.head_dim) % 32 || h.ffn % 64)
      return Status::err(JET_E_INVALID, "block-quantized models need d_model a multiple of 128 and ffn of 64");
  }
  if (h.n_experts) {
    if (h.n_experts > jetk::kMoeMaxExperts || h.top_k < 1 || h.top_k > h.n_experts ||
        h.top_k > jetk::kMoeMaxTopK)
      return Status::err(JET_E_INVALID, "mixture of experts: need 1 <= top_k <= n_experts <= " +
                                            std::to_string(jetk::kMoeMaxExperts) + " and top_k <= " +
                                            std::to_string(jetk::kMoeMaxTopK));
    if (h.moe_ffn < 64 || h.moe_ffn % 64 || h.shared_ffn % 64 || h.d % 4)
      return Status::err(JET_E_INVALID, "mixture of experts: moe_ffn and shared_ffn must be multiples of 64");
    if (dtype == JET_BF16)
      return Status::err(JET_E_INVALID, "mixture-of-experts models run in the f32, f16, f16p and bf16-single modes");
  }
  if (h.hybrid) {
    if (h.gdn_dk != 128 || h.gdn_dv != 128 || h.conv_kernel != 4 || h.gdn_heads < 1)
      return Status::err(JET_E_INVALID, "delta-rule layers need dk = dv = 128 and a width-4 convolution");
    if ((h.gdn_heads * h.gdn_dv) % bk)
      return Status::err(JET_E_INVALID, "gdn_heads * gdn_dv must be a multiple of " + std::to_string(bk));
  }
  return Status::ok();
}

Status load_model(jet_model *m, const char *path, const jet_load_opts *o) {
  m->path = path;
  TRY(read_model_header(m->path, &m->h));
  const ModelHeader &h = m->h;
  TRY(check_shapes(h, m->dtype));
  m->kdt = m->dtype == JET_FP32 ? 1 : (m->dtype == JET_F16 || m->dtype == JET_F16P) ? 2 : 0;
  m->edt = m->kdt == 1 ? 1 : 0;
  m->pair = m->dtype == JET_BF16 ? 1 : 0;
  m->np = m->pair ? 2 : 1;
  m->apair = (m->dtype == JET_BF16 || m->dtype == JET_F16P) ? 1 : 0;
  m->anp = m->apair ? 2 : 1;
  m->esz = m->kdt == 1 ? 4 : 2;
  m->max_ctx = (o && o->max_ctx > 0) ? o->max_ctx : h.max_ctx;
  HIPC(hipSetDevice(m->device));
  // the device address of the allocation-free entry point's scratch, looked
  // up once per device (its failure only disables that entry point)
  m->scratch_status = noalloc_scratch_init(m->device);
  if (m->scratch_status != hipSuccess) (void)hipGetLastError();
  Loader L{m, {}};
  // block-quantized models in the fp16 mode keep the projection and FFN
  // weights as int8 (dequantized in the GEMM's operand path); every other
  // matrix, and every matrix in the fp32 mode, is dequantized here
  const bool q8_gemm = h.q8 && m->kdt == 2;
  if (m->kdt == 2) {
    TRY(dmalloc(m, sizeof(unsigned long long), (void **)&L.inexact));
    m->weight_allocs.push_back(L.inexact);
    HIPC(hipMemset(L.inexact, 0, sizeof(unsigned long long)));
  }
  TRY(L.matrix("tok_embed", &m->embed, nullptr, /*keep_bf16=*/m->kdt == 2));
  TRY(L.matrix("lm_head", &m->lm_head, &m->is_lm));
  TRY(L.vec_f32("final_norm", &m->final_norm, h.d));
  m->layers.resize((size_t)h.n_layers);
  for (int64_t i = 0; i < h.n_layers; ++i) {
    Layer &ly = m->layers[(size_t)i];
    const std::string p = "blk." + std::to_string(i) + ".";
    ly.gdn = h.layer_is_gdn[(size_t)i] != 0;
    TRY(L.vec_f32(p + "attn_norm", &ly.attn_norm, h.d));
    TRY(L.vec_f32(p + "ffn_norm", &ly.ffn_norm, h.d));
    if (!ly.gdn && q8_gemm) {
      Loader::Q8Rows wq, wk, wv, wo;
      TRY(L.q8_read(p + "wq", &wq));
      TRY(L.q8_read(p + "wk", &wk));
      TRY(L.q8_read(p + "wv", &wv));
      TRY(L.put_q8(Loader::q8_stack({wq, wk, wv}, false), &ly.w_qkv, &ly.s_qkv, &ly.is_qkv));
      TRY(L.q8_read(p + "wo", &wo));
      TRY(L.put_q8(wo, &ly.w_o, &ly.s_o, &ly.is_o));
    } else if (!ly.gdn) {
      TRY(L.concat({p + "wq", p + "wk", p + "wv"}, h.d, 0, &ly.w_qkv, nullptr, &ly.is_qkv));
      TRY(L.matrix(p + "wo", &ly.w_o, &ly.is_o));
    } else {
      const int64_t H = h.gdn_heads, C = 2 * H * h.gdn_dk + H * h.gdn_dv;
      TRY(L.concat({p + "gdn_wq", p + "gdn_wk", p + "gdn_wv", p + "gdn_wz", p + "gdn_wb", p + "gdn_wa"}, h.d, 0,
                   &ly.w_in, &ly.n_in, &ly.is_qkv));
      TRY(L.matrix(p + "gdn_wo", &ly.w_o, &ly.is_o));
      TRY(L.f32_array(p + "gdn_conv", &ly.conv_w, C * h.conv_kernel));
      TRY(L.f32_array(p + "gdn_A_log", &ly.A_log, H));
      TRY(L.f32_array(p + "gdn_dt_bias", &ly.dt_bias, H));
      TRY(L.f32_array(p + "gdn_norm", &ly.gdn_norm, h.gdn_dv));
    }
    if (h.n_experts) {
      const int64_t nr = ((h.n_experts + (h.shared_ffn ? 1 : 0)) + 63) / 64 * 64;
      std::vector<std::string> rn{p + "moe_router"};
      if (h.shared_ffn) rn.push_back(p + "shared_router");
      TRY(L.concat(rn, h.d, nr, &ly.w_router, &ly.n_router, &ly.is_router));
      TRY(L.expert_gate_up(p + "moe_gate", p + "moe_up", h.n_experts, h.moe_ffn, h.d, &ly.w_egu, &ly.is_egu));
      TRY(L.matrix(p + "moe_down", &ly.w_edown, &ly.is_edown));
      if (h.shared_ffn) {
        TRY(L.gate_up(p + "shared_gate", p + "shared_up", h.shared_ffn, h.d, &ly.w_sgu, &ly.is_sgu));
        TRY(L.matrix(p + "shared_down", &ly.w_sdown, &ly.is_sdown));
      }
    } else if (q8_gemm) {
      Loader::Q8Rows wg, wu, wd;
      TRY(L.q8_read(p + "w_gate", &wg));
      TRY(L.q8_read(p + "w_up", &wu));
      TRY(L.put_q8(Loader::q8_stack({wg, wu}, true), &ly.w_gu, &ly.s_gu, &ly.is_gu));
      TRY(L.q8_read(p + "w_down", &wd));
      TRY(L.put_q8(wd, &ly.w_down, &ly.s_down, &ly.is_down));
    } else {
      TRY(L.gate_up(p + "w_gate", p + "w_up", h.ffn, h.d, &ly.w_gu, &ly.is_gu));
      TRY(L.matrix(p + "w_down", &ly.w_down, &ly.is_down));
    }
  }
  // RoPE tables: angles in fp64 on the host, stored as fp32 [max_ctx][hd/2]
  const int64_t half = h.head_dim / 2;
  std::vector<float> c((size_t)(m->max_ctx * half)), s((size_t)(m->max_ctx * half));
  for (int64_t p = 0; p < m->max_ctx; ++p)
    for (int64_t i = 0; i < half; ++i) {
      const double inv = std::pow(h.rope_theta, -(2.0 * (double)i) / (double)h.head_dim);
      const double a = (double)p * inv;
      c[(size_t)(p * half + i)] = (float)std::cos(a);
      s[(size_t)(p * half + i)] = (float)std::sin(a);
    }
  TRY(dmalloc(m, c.size() * 4, (void **)&m->rope_cos));
  m->weight_allocs.push_back(m->rope_cos);
  TRY(dmalloc(m, s.size() * 4, (void **)&m->rope_sin));
  m->weight_allocs.push_back(m->rope_sin);
  HIPC(hipMemcpy(m->rope_cos, c.data(), c.size() * 4, hipMemcpyHostToDevice));
  HIPC(hipMemcpy(m->rope_sin, s.data(), s.size() * 4, hipMemcpyHostToDevice));
  if (L.inexact) {
    unsigned long long n = 0;
    HIPC(hipMemcpy(&n, L.inexact, sizeof(n), hipMemcpyDeviceToHost));
    m->f16_inexact += (int64_t)n;
  }
  return Status::ok();
}

// ---------------------------------------------------------------------------
// shared pieces of the forward pass
// ---------------------------------------------------------------------------

double gemm_flops(int64_t M, int64_t N, int64_t K) { return 2.0 * (double)M * (double)N * (double)K; }

// A holds activations ([hi | lo] pairs when pair, lda counts both planes).
// Bs: block scales of an int8 B (block-quantized weights, fp16 mode), else NULL.
Status run_gemm(jet_model *m, int cls, int epi, const void *A, int64_t lda, int pair, const void *B, int64_t ldb,
                int64_t M, int64_t N, int64_t K, void *out, int64_t ldo, float oscale, const uint16_t *Bs = nullptr) {
  const double out_bytes = (double)M * (double)(epi == jetk::EPI_SWIGLU ? N / 2 * m->np : N) *
                           (epi == jetk::EPI_STORE_F32 || epi == jetk::EPI_RESID_ADD ? 4.0 : (double)m->esz) *
                           (epi == jetk::EPI_RESID_ADD ? 2.0 : 1.0);
  const double b_bytes = Bs ? (double)(N * K) * (m->h.qbits / 8.0 + 2.0 / 32.0) : (double)(N * K) * (double)m->esz;
  KTimer t(m, cls, gemm_flops(M, N, K), (double)(M * K * (pair ? 2 : 1)) * (double)m->esz + b_bytes + out_bytes);
  if (Bs) {
    if (pair || ldb != K) return Status::err(JET_E_INVALID, "int8 weights: no pair operands, dense rows");
    if (m->h.qbits == 4) LAUNCH(jetk::launch_gemm_q4(epi, A, lda, B, Bs, (int)M, (int)N, (int)K, out, ldo, oscale, m->st));
    else LAUNCH(jetk::launch_gemm_q8(epi, A, lda, B, Bs, (int)M, (int)N, (int)K, out, ldo, oscale, m->st));
    return Status::ok();
  }
  // decode steps (one row per question): too few output tiles to fill the
  // device, so K is split across workgroups and summed in a fixed order
  if (m->splitk && (epi == jetk::EPI_STORE_F32 || epi == jetk::EPI_RESID_ADD)) {
    const int S = jetk::gemm_splitk_ways(m->kdt, pair, (int)M, (int)N, (int)K);
    if (S > 1) {
      float *part;
      TRY(ws_t<float>(m, "splitk_part", (size_t)(S * M * N), &part));
      LAUNCH(jetk::launch_gemm_splitk(epi, A, lda, B, ldb, (int)M, (int)N, (int)K, S, part, out, ldo, oscale,
                                      m->st));
      return Status::ok();
    }
  }
  LAUNCH(jetk::launch_gemm(m->kdt, epi, A, lda, B, ldb, (int)M, (int)N, (int)K, pair, out, ldo, oscale, m->st));
  return Status::ok();
}

// LM head + online LSE over R rows of F (compute dtype) -> lse[R] (fp32).
// With target (device int32[R]): ell[r] = log p(target[r]) = z - lse, z the
// target's logit as the LM-head tile accumulated it for the log-sum-exp
// (Section 3.1 Eq. 2).
Status run_lmhead(jet_model *m, const void *F, int64_t R, float *lse, const int32_t *target = nullptr,
                  float *ell = nullptr) {
  if (R <= 0) return Status::ok();
  const int64_t V = m->h.vocab, d = m->h.d;
  int tps = 1, nsplit = 1;
  jetk::lmhead_plan(m->kdt, (int)V, (int)R, &tps, &nsplit);
  float *pm, *ps, *zt = nullptr;
  TRY(ws_t<float>(m, "lm_pm", (size_t)(nsplit * R), &pm));
  TRY(ws_t<float>(m, "lm_ps", (size_t)(nsplit * R), &ps));
  if (target) TRY(ws_t<float>(m, "lm_zt", (size_t)R, &zt));
  {
    KTimer t(m, JET_K_LMHEAD, gemm_flops(R, V, d), (double)(V * d + R * d * m->np) * (double)m->esz);
    LAUNCH(jetk::launch_lmhead_lse(m->kdt, m->lm_head, F, (int)V, (int)R, (int)d, m->pair, tps, m->is_lm, pm, ps,
                                   target, zt, m->st));
  }
  KTimer t2(m, JET_K_OTHER, 0, 0);
  LAUNCH(jetk::launch_lse_merge(pm, ps, nsplit, (int)R, lse, zt, m->is_lm, ell, m->st));
  m->stats.lm_rows += R;
  return Status::ok();
}

struct QDesc {
  std::vector<int32_t> qrow0, nrows, pre_len, suf_row0, suf_len;
  std::vector<int64_t> pre_slot0;
};

// Work items: per (question, kv head), blocks of `block` (row, head) slots,
// slot s = G row + (head - kvh G); a causal block needs the keys up to its
// last row.
void build_items(const QDesc &qd, int G, int Hkv, bool causal, int block, std::vector<jetk::AttnItem> *items,
                 double *flops_pairs) {
  items->clear();
  double pairs = 0;
  for (size_t q = 0; q < qd.nrows.size(); ++q) {
    const int n = qd.nrows[q];
    if (n <= 0) continue;
    const int total = G * n;
    for (int kvh = 0; kvh < Hkv; ++kvh)
      for (int s0 = 0; s0 < total; s0 += block) {
        const int ns = std::min(block, total - s0);
        const int maxq = (s0 + ns - 1) / G;
        items->push_back({(int32_t)q, kvh, s0, ns, maxq + 1});
      }
    if (causal) pairs += (double)G * Hkv * (double)n * (double)(n + 1) / 2.0;
    else pairs += (double)G * Hkv * (double)n * (double)(qd.pre_len[q] + qd.suf_len[q]);
  }
  *flops_pairs = pairs;
}

// Attention launch plan of one wave: work items and per-question descriptors
// uploaded once, reused by every attention layer of the wave.
struct AttnPlan {
  jetk::AttnArgs a{};
  double flops = 0, bytes = 0;
};

Status plan_attention(jet_model *m, int mode, const QDesc &qd, const char *tag, AttnPlan *pl) {
  const ModelHeader &h = m->h;
  const int G = (int)(h.n_heads / h.n_kv_heads);
  std::vector<jetk::AttnItem> items;
  double pairs = 0;
  // 128-slot items (two query blocks per wave: each staged tile and each
  // K/V fragment read serves twice the queries) where the kernel supports
  // them: always for the prefix, and for candidates when their questions
  // average at least 96 query slots per KV head (few slots would leave most
  // of a 128-slot item idle). A query's arithmetic is the same in either
  // item size, so a candidate rounds alike whatever batch it is in.
  int block = 64;
  if (jetk::attn_slots_per_item(m->kdt, m->apair) >= 128) {
    if (mode == 0) {
      block = 128;
    } else {
      double slots = 0, nq = 0;
      for (auto n : qd.nrows)
        if (n > 0) slots += (double)G * n, nq += 1;
      if (nq > 0 && slots >= 96.0 * nq) block = 128;
    }
  }
  build_items(qd, G, (int)h.n_kv_heads, mode == 0, block, &items, &pairs);
  // Longest work first: the dispatcher hands out workgroups in order, so long
  // items no longer run alone at the end (an item's result does not depend
  // on its position in the launch). Questions are ordered by length and each
  // question's items stay together (they share its K/V in L2), the longest
  // of them first.
  auto qlen = [&](const jetk::AttnItem &it) {
    return (int64_t)qd.pre_len[(size_t)it.q] + qd.suf_len[(size_t)it.q];
  };
  std::stable_sort(items.begin(), items.end(), [&](const jetk::AttnItem &x, const jetk::AttnItem &y) {
    if (qlen(x) != qlen(y)) return qlen(x) > qlen(y);
    if (x.q != y.q) return x.q < y.q;
    return x.nkeys_pre > y.nkeys_pre;
  });
  jetk::AttnItem *d_items;
  int32_t *d_qrow0, *d_nrows, *d_prelen, *d_sufrow0, *d_suflen;
  int64_t *d_preslot;
  const std::string t(tag);
  TRY(upload(m, (t + "items").c_str(), items, &d_items));
  TRY(upload(m, (t + "qrow0").c_str(), qd.qrow0, &d_qrow0));
  TRY(upload(m, (t + "nrows").c_str(), qd.nrows, &d_nrows));
  TRY(upload(m, (t + "prelen").c_str(), qd.pre_len, &d_prelen));
  TRY(upload(m, (t + "sufrow0").c_str(), qd.suf_row0, &d_sufrow0));
  TRY(upload(m, (t + "suflen").c_str(), qd.suf_len, &d_suflen));
  TRY(upload(m, (t + "preslot").c_str(), qd.pre_slot0, &d_preslot));
  jetk::AttnArgs &a = pl->a;
  a.mode = mode;
  a.pair = m->apair;
  a.qs = {d_qrow0, d_nrows, d_preslot, d_prelen, d_sufrow0, d_suflen};
  a.items = d_items;
  a.n_items = (int)items.size();
  a.qb = block / 64;
  a.Hq = (int)h.n_heads;
  a.Hkv = (int)h.n_kv_heads;
  a.hd = (int)h.head_dim;
  a.scale = (float)(1.0 / std::sqrt((double)h.head_dim));
  // algorithmic bytes: every K/V row of the prefix (and suffix) read once per
  // kv head, Q read and O written once
  double kv_rows = 0, qo_rows = 0;
  for (size_t q = 0; q < qd.nrows.size(); ++q)
    if (qd.nrows[q] > 0) kv_rows += (double)qd.pre_len[q] + (double)qd.suf_len[q];
  for (auto n : qd.nrows) qo_rows += n;
  pl->bytes = (double)m->esz * m->anp * (kv_rows * 2.0 * (double)h.n_kv_heads * (double)h.head_dim +
                                        qo_rows * 2.0 * (double)h.n_heads * (double)h.head_dim);
  pl->flops = 4.0 * pairs * (double)h.head_dim;
  return Status::ok();
}

// Q: [planes][R][Hq][hd]; O: [R][planes * Hq * hd]; caches [planes][Hkv][S][hd].
Status run_attention(jet_model *m, AttnPlan &pl, const void *Q, int64_t R, void *O, const void *Kp, const void *Vp,
                     int64_t s_pre, const void *Ks, const void *Vs, int64_t s_suf, const int32_t *row_n,
                     const int32_t *row_t, int cls = -1) {
  if (pl.a.n_items == 0) return Status::ok();
  const ModelHeader &h = m->h;
  jetk::AttnArgs a = pl.a;
  a.Q = Q;
  a.q_ps = R * h.n_heads * h.head_dim;
  a.O = O;
  a.o_ld = m->anp * h.n_heads * h.head_dim;
  a.Kp = Kp;
  a.Vp = Vp;
  a.s_pre = s_pre;
  a.kp_ps = h.n_kv_heads * s_pre * h.head_dim;
  a.Ks = Ks;
  a.Vs = Vs;
  a.s_suf = s_suf;
  a.ks_ps = h.n_kv_heads * s_suf * h.head_dim;
  a.row_n = row_n;
  a.row_t = row_t;
  KTimer t(m, cls >= 0 ? cls : a.mode == 0 ? JET_K_ATTN_PREFIX : JET_K_ATTN_CAND, pl.flops, pl.bytes);
  LAUNCH(jetk::launch_attention(m->kdt, a, m->st));
  return Status::ok();
}

// Buffers of one forward wave over R rows.
struct WaveBufs {
  float *resid = nullptr, *qkv = nullptr;
  void *xn = nullptr, *q = nullptr, *att = nullptr, *act = nullptr;
};

Status wave_bufs(jet_model *m, int64_t R, WaveBufs *b) {
  const ModelHeader &h = m->h;
  const int64_t nqkv = (h.n_heads + 2 * h.n_kv_heads) * h.head_dim;
  TRY(ws_t<float>(m, "resid", (size_t)(R * h.d), &b->resid));
  TRY(ws_t<float>(m, "qkv", (size_t)(R * nqkv), &b->qkv));
  const size_t pe = (size_t)m->np * m->esz, pa = (size_t)m->anp * m->esz;  // bytes per activation element
  TRY(ws(m, "xn", (size_t)(R * h.d) * std::max(pe, pa), &b->xn));
  TRY(ws(m, "q", (size_t)(R * h.n_heads * h.head_dim) * pa, &b->q));
  TRY(ws(m, "att", (size_t)(R * h.n_heads * h.head_dim) * pa, &b->att));
  TRY(ws(m, "act", (size_t)(R * h.ffn) * pe, &b->act));
  return Status::ok();
}

// Copies a routing result [R][k] (device) into the current route record
// (JET_FLAG_RECORD_ROUTES; synchronises the stream).
Status record_routes(jet_model *m, const int *sel, int64_t R, int k) {
  std::vector<int32_t> h((size_t)(R * k));
  HIPC(hipMemcpyAsync(h.data(), sel, h.size() * 4, hipMemcpyDeviceToHost, m->st));
  HIPC(hipStreamSynchronize(m->st));
  auto &rec = m->routes[m->rt_which];
  const int64_t rows = m->route_rows[m->rt_which];
  if ((int64_t)m->rt_rowmap.size() != R) return Status::err(JET_E_DEVICE, "route record: row map mismatch");
  for (int64_t r = 0; r < R; ++r)
    for (int j = 0; j < k; ++j)
      rec[(size_t)((m->rt_layer * rows + m->rt_rowmap[(size_t)r]) * k + j)] = h[(size_t)(r * k + j)];
  return Status::ok();
}

// Route recording: which record the next FFN calls write, and their rows.
void route_rows_begin(jet_model *m, int which, int64_t rows) {
  m->rt_which = -1;
  if (!(m->flags & JET_FLAG_RECORD_ROUTES) || !m->h.n_experts) return;
  m->routes[which].assign((size_t)(m->h.n_layers * rows * m->h.top_k), -1);
  m->route_rows[which] = rows;
}
void route_rows_set(jet_model *m, int which, int64_t layer, int64_t base, int64_t R, const int32_t *idx = nullptr) {
  if (!(m->flags & JET_FLAG_RECORD_ROUTES) || !m->h.n_experts) return;
  m->rt_which = which;
  m->rt_layer = layer;
  m->rt_rowmap.resize((size_t)R);
  for (int64_t r = 0; r < R; ++r) m->rt_rowmap[(size_t)r] = base + (idx ? idx[r] : r);
}

// Mixture-of-experts FFN on x = RMSNorm(resid) (in b.xn): router GEMM,
// top-k routing, rows scattered into per-expert segments, grouped gate/up
// (SwiGLU) and down GEMMs over the segments, the shared expert on all rows,
// then resid += sum_j w_j y_j + sigmoid(g) y_shared.
Status moe_ffn(jet_model *m, const Layer &ly, const WaveBufs &b, int64_t R) {
  const ModelHeader &h = m->h;
  const int E = (int)h.n_experts, k = (int)h.top_k;
  const int64_t Fe = h.moe_ffn, Fs = h.shared_ffn, d = h.d;
  // 256-row tiles when the segments average 1024 rows or more (padding costs
  // at most an eighth), else 128
  const int big = m->kdt == 2 && R * k >= 1024 * (int64_t)E;
  const int bm = jetk::gemm_group_rows(m->kdt, big);
  const int64_t S = (R * k + (int64_t)E * (bm - 1) + bm - 1) / bm * bm;  // rows of all segments, at most
  float *logits, *wts, *sg = nullptr, *ys = nullptr;
  int *sel, *tiles, *slot, *chist, *cbase;
  void *xp, *hp, *y, *hs = nullptr;
  TRY(ws_t<float>(m, "moe_logits", (size_t)(R * ly.n_router), &logits));
  TRY(ws_t<int>(m, "moe_sel", (size_t)(R * k), &sel));
  TRY(ws_t<float>(m, "moe_wts", (size_t)(R * k), &wts));
  TRY(ws_t<int>(m, "moe_tiles", (size_t)(S / bm), &tiles));
  TRY(ws_t<int>(m, "moe_slot", (size_t)(R * k), &slot));
  const int nch = jetk::moe_chunks((int)R, k);
  TRY(ws_t<int>(m, "moe_chist", (size_t)std::max(nch, 1) * E, &chist));
  TRY(ws_t<int>(m, "moe_cbase", (size_t)std::max(nch, 1) * E, &cbase));
  TRY(ws(m, "moe_xp", (size_t)(S * d) * m->esz, &xp));
  TRY(ws(m, "moe_h", (size_t)(S * Fe) * m->esz, &hp));
  TRY(ws(m, "moe_y", (size_t)(S * d) * m->esz, &y));  // expert outputs in the compute type
  if (Fs) {
    TRY(ws_t<float>(m, "moe_sg", (size_t)R, &sg));
    TRY(ws(m, "moe_hs", (size_t)(R * Fs) * m->esz, &hs));
    TRY(ws_t<float>(m, "moe_ys", (size_t)(R * d), &ys));
  }
  TRY(run_gemm(m, JET_K_OTHER, jetk::EPI_STORE_F32, b.xn, d, 0, ly.w_router, d, R, ly.n_router, d, logits,
               ly.n_router, ly.is_router));
  {
    KTimer t(m, JET_K_OTHER, 0, (double)(R * ly.n_router) * 4.0);
    LAUNCH(jetk::launch_moe_route(jetk::MoeRouteArgs{logits, ly.n_router, (int)R, E, k, sel, wts, sg}, m->st));
    if (m->rt_which >= 0) TRY(record_routes(m, sel, R, k));
    LAUNCH(jetk::launch_moe_plan(sel, (int)R, k, E, bm, (int)(S / bm), tiles, chist, cbase, slot, m->st));
    LAUNCH(jetk::launch_moe_scatter(b.xn, d * (int64_t)m->esz, (int)R, k, slot, xp, m->st));
  }
  {
    const double rows = (double)(R * k);
    KTimer t(m, JET_K_GEMM_GATEUP, 2.0 * rows * (double)(2 * Fe) * (double)d,
             (rows * (double)d + rows * (double)Fe) * (double)m->esz);
    LAUNCH(jetk::launch_gemm_grouped(m->kdt, big, jetk::EPI_SWIGLU, xp, d, ly.w_egu, d, 2 * Fe * d, tiles, (int)S,
                                     (int)(2 * Fe), (int)d, hp, Fe, ly.is_egu, m->st));
  }
  {
    const double rows = (double)(R * k);
    KTimer t(m, JET_K_GEMM_DOWN, 2.0 * rows * (double)d * (double)Fe,
             rows * (double)Fe * (double)m->esz + rows * (double)d * (double)m->esz);
    LAUNCH(jetk::launch_gemm_grouped(m->kdt, big, jetk::EPI_STORE_T, hp, Fe, ly.w_edown, Fe, d * Fe, tiles, (int)S,
                                     (int)d, (int)Fe, y, d, ly.is_edown, m->st));
  }
  if (Fs) {
    TRY(run_gemm(m, JET_K_GEMM_GATEUP, jetk::EPI_SWIGLU, b.xn, d, 0, ly.w_sgu, d, R, 2 * Fs, d, hs, Fs, ly.is_sgu));
    TRY(run_gemm(m, JET_K_GEMM_DOWN, jetk::EPI_STORE_F32, hs, Fs, 0, ly.w_sdown, Fs, R, d, Fs, ys, d, ly.is_sdown));
  }
  {
    KTimer t(m, JET_K_OTHER, 0, (double)(R * d) * ((double)k * (double)m->esz + 12.0));
    LAUNCH(jetk::launch_moe_combine(m->kdt, y, slot, wts, k, ys, sg, (int)R, (int)d, b.resid, m->st));
  }
  return Status::ok();
}

// The FFN sublayer: resid += down(silu(gate(x)) * up(x)), x = RMSNorm(resid).
Status ffn(jet_model *m, const Layer &ly, const WaveBufs &b, int64_t R) {
  const ModelHeader &h = m->h;
  {
    KTimer t(m, JET_K_OTHER, 0, 0);
    LAUNCH(jetk::launch_rmsnorm(m->kdt, m->pair, b.resid, nullptr, ly.ffn_norm, (int)R, (int)h.d, (float)h.rms_eps,
                                b.xn, m->st));
  }
  if (h.n_experts) return moe_ffn(m, ly, b, R);
  TRY(run_gemm(m, JET_K_GEMM_GATEUP, jetk::EPI_SWIGLU, b.xn, m->np * h.d, m->pair, ly.w_gu, h.d, R, 2 * h.ffn, h.d,
               b.act, m->np * h.ffn, ly.is_gu, ly.s_gu));
  TRY(run_gemm(m, JET_K_GEMM_DOWN, jetk::EPI_RESID_ADD, b.act, m->np * h.ffn, m->pair, ly.w_down, h.ffn, R, h.d,
               h.ffn, b.resid, h.d, ly.is_down, ly.s_down));
  return Status::ok();
}

// Attention sublayer up to the attention kernel: x = RMSNorm(resid); qkv;
// RoPE; K/V written to (kc, vc) at slot0 + r of an [Hkv][S][hd] cache.
Status attn_in(jet_model *m, const Layer &ly, const WaveBufs &b, int64_t R, const int32_t *d_pos, void *kc, void *vc,
               int64_t S, int64_t slot0) {
  const ModelHeader &h = m->h;
  const int64_t nqkv = (h.n_heads + 2 * h.n_kv_heads) * h.head_dim;
  {
    KTimer t(m, JET_K_OTHER, 0, 0);
    LAUNCH(jetk::launch_rmsnorm(m->kdt, m->apair, b.resid, nullptr, ly.attn_norm, (int)R, (int)h.d,
                                (float)h.rms_eps, b.xn, m->st));
  }
  if (!ly.s_qkv && jetk::gemm_qkv_rope_ok(m->kdt, m->apair, (int)R, (int)nqkv, (int)h.head_dim)) {
    // projection, RoPE and the K/V scatter in one kernel
    const double out_bytes = (double)R * (double)nqkv * (double)m->esz * m->anp;
    KTimer t(m, JET_K_GEMM_QKV, gemm_flops(R, nqkv, h.d),
             (double)(R * h.d * m->anp + nqkv * h.d) * (double)m->esz + out_bytes);
    jetk::QkvRope r{d_pos, m->rope_cos, m->rope_sin, (int)h.n_heads, (int)h.n_kv_heads, b.q,
                    R * h.n_heads * h.head_dim, kc, vc, h.n_kv_heads * S * h.head_dim, S, slot0};
    LAUNCH(jetk::launch_gemm_qkv_rope(m->kdt, b.xn, m->anp * h.d, ly.w_qkv, h.d, (int)R, (int)nqkv, (int)h.d, m->apair,
                                      ly.is_qkv, r, m->st));
    return Status::ok();
  }
  TRY(run_gemm(m, JET_K_GEMM_QKV, jetk::EPI_STORE_F32, b.xn, m->anp * h.d, m->apair, ly.w_qkv, h.d, R, nqkv, h.d,
               b.qkv, nqkv, ly.is_qkv, ly.s_qkv));
  KTimer t(m, JET_K_OTHER, 0, 0);
  LAUNCH(jetk::launch_rope_scatter(m->kdt, m->apair, b.qkv, d_pos, m->rope_cos, m->rope_sin, (int)R, (int)h.n_heads,
                                   (int)h.n_kv_heads, (int)h.head_dim, b.q, R * h.n_heads * h.head_dim, kc, vc,
                                   h.n_kv_heads * S * h.head_dim, S, slot0, m->st));
  return Status::ok();
}

Status attn_out(jet_model *m, const Layer &ly, const WaveBufs &b, int64_t R) {
  const ModelHeader &h = m->h;
  return run_gemm(m, JET_K_GEMM_O, jetk::EPI_RESID_ADD, b.att, m->anp * h.n_heads * h.head_dim, m->apair, ly.w_o,
                  h.n_heads * h.head_dim, R, h.d, h.n_heads * h.head_dim, b.resid, h.d, ly.is_o, ly.s_o);
}

// Per-wave tables of the delta-rule layers (built on the host, uploaded once).
struct GdnPlan {
  int32_t *hist = nullptr, *tail_slot = nullptr;
  jetk::GdnSeq *seqs = nullptr;
  int nseq = 0;
  double tok_heads = 0;
  bool chunked = false;  // the recurrence in chunks on the matrix cores
};

// Gated delta-rule sublayer: resid += W_o y, y = RMSNorm(o) silu(z), o from
// the recurrence over each sequence of the plan. tail: the layer's [Q][3][C]
// snapshot buffer; S_init / S_fin: the layer's [Q][H][dv][dk] state snapshots.
Status gdn_layer(jet_model *m, const Layer &ly, const WaveBufs &b, int64_t R, const GdnPlan &gp, float *tail,
                 const float *S_init, float *S_fin) {
  const ModelHeader &h = m->h;
  const int64_t H = h.gdn_heads, dk = h.gdn_dk, dv = h.gdn_dv;
  const int64_t C = 2 * H * dk + H * dv;
  float *gx, *gq, *gk, *gv, *ga, *gb, *go;
  void *gy;
  TRY(ws_t<float>(m, "gdn_x", (size_t)(R * ly.n_in), &gx));
  TRY(ws_t<float>(m, "gdn_q", (size_t)(R * H * dk), &gq));
  TRY(ws_t<float>(m, "gdn_k", (size_t)(R * H * dk), &gk));
  TRY(ws_t<float>(m, "gdn_v", (size_t)(R * H * dv), &gv));
  TRY(ws_t<float>(m, "gdn_a", (size_t)(R * H), &ga));
  TRY(ws_t<float>(m, "gdn_b", (size_t)(R * H), &gb));
  TRY(ws_t<float>(m, "gdn_o", (size_t)(R * H * dv), &go));
  TRY(ws(m, "gdn_y", (size_t)(R * H * dv) * m->esz * m->np, &gy));
  {
    KTimer t(m, JET_K_OTHER, 0, 0);
    LAUNCH(jetk::launch_rmsnorm(m->kdt, m->pair, b.resid, nullptr, ly.attn_norm, (int)R, (int)h.d, (float)h.rms_eps,
                                b.xn, m->st));
  }
  TRY(run_gemm(m, JET_K_GEMM_QKV, jetk::EPI_STORE_F32, b.xn, m->np * h.d, m->pair, ly.w_in, h.d, R, ly.n_in, h.d,
               gx, ly.n_in, ly.is_qkv));
  {
    KTimer t(m, JET_K_OTHER, 0, 0);
    jetk::GdnConvArgs g{gx, ly.n_in, gp.hist, gp.tail_slot, tail, ly.conv_w, ly.A_log, ly.dt_bias,
                        (int)H, (int)dk, (int)dv, gq, gk, gv, ga, gb};
    LAUNCH(jetk::launch_gdn_conv(g, (int)R, m->st));
  }
  {
    const double flops = gp.tok_heads * 7.0 * (double)dk * (double)dv;
    const double bytes = gp.tok_heads * 4.0 * (double)(2 * dk + 2 * dv + 2) +
                         (double)gp.nseq * (double)H * (double)(dk * dv) * 4.0;
    KTimer t(m, JET_K_GDN, flops, bytes);
    jetk::GdnRecurArgs g{gp.seqs, gq, gk, gv, ga, gb, (int)H, (int)dk, (int)dv, S_init, S_fin, go};
    if (gp.chunked) LAUNCH(jetk::launch_gdn_chunk(g, gp.nseq, m->pair, m->st));
    else LAUNCH(jetk::launch_gdn_recur(g, gp.nseq, m->st));
  }
  {
    KTimer t(m, JET_K_OTHER, 0, 0);
    LAUNCH(jetk::launch_gdn_out(m->kdt, m->pair, go, gx, ly.n_in, (int)C, ly.gdn_norm, (float)h.rms_eps, (int)H,
                                (int)dv, (int)R, gy, m->st));
  }
  return run_gemm(m, JET_K_GEMM_O, jetk::EPI_RESID_ADD, gy, m->np * H * dv, m->pair, ly.w_o, H * dv, R, h.d, H * dv,
                  b.resid, h.d, ly.is_o);
}

// Token ids: validated on the host (host memory) or by a device count.
Status check_ids(jet_model *m, const int32_t *ids, int64_t n, bool on_device, const char *what) {
  if (n == 0) return Status::ok();
  if (!ids) return Status::err(JET_E_INVALID, std::string(what) + " is NULL");
  if (!on_device) return check_ids_host(ids, n, m->h.vocab, what);
  int *bad;
  TRY(ws_t<int>(m, "badids", 1, &bad));
  HIPC(hipMemsetAsync(bad, 0, sizeof(int), m->st));
  LAUNCH(jetk::launch_count_bad_ids(ids, n, (int)m->h.vocab, bad, m->st));
  int hb = 0;
  HIPC(hipMemcpyAsync(&hb, bad, sizeof(int), hipMemcpyDeviceToHost, m->st));
  TRY(sync(m));
  if (hb) return Status::err(JET_E_INVALID, std::string(what) + ": " + std::to_string(hb) + " ids outside [0, vocab)");
  return Status::ok();
}

// ---------------------------------------------------------------------------
// prefill
// ---------------------------------------------------------------------------

// A freed prefix's buffers go to the model's pool instead of hipFree (which
// synchronises the device): repeated calls with similar shapes reuse them.
// Every buffer a prefill takes is written before it is read (caches,
// snapshots, last rows) or cleared (convolution tails), so stale contents
// never leak into a new prefix.
void release_pool(jet_model *m) {
  for (auto &e : m->pool) dfree(m, e.second, e.first);
  m->pool.clear();
}

void free_prefix(jet_prefix *p) {
  if (!p) return;
  if (p->m) {
    for (auto &a : p->allocs) p->m->pool.push_back({a.second, a.first});
    auto &live = p->m->live;
    for (size_t i = 0; i < live.size(); ++i)
      if (live[i] == p) {
        live.erase(live.begin() + (std::ptrdiff_t)i);
        break;
      }
  } else {
    // a prefix that never got a model, or whose model was freed (its
    // buffers were freed then and the list is empty)
    for (auto &a : p->allocs) (void)hipFree(a.first);
  }
  delete p;
}

Status palloc(jet_prefix *p, size_t bytes, void **out) {
  jet_model *m = p->m;
  if (bytes == 0) bytes = 256;
  // the smallest pooled buffer that holds `bytes` without wasting over a quarter
  size_t best = m->pool.size();
  for (size_t i = 0; i < m->pool.size(); ++i) {
    const size_t sz = m->pool[i].first;
    if (sz >= bytes && sz - bytes <= bytes / 4 && (best == m->pool.size() || sz < m->pool[best].first)) best = i;
  }
  size_t got = bytes;
  if (best < m->pool.size()) {
    *out = m->pool[best].second;
    got = m->pool[best].first;
    m->pool.erase(m->pool.begin() + (std::ptrdiff_t)best);
  } else {
    Status s = dmalloc(m, bytes, out);
    if (!s) {
      if (m->pool.empty()) return s;
      release_pool(m);
      TRY(dmalloc(m, bytes, out));
    }
  }
  p->allocs.push_back({*out, got});
  p->bytes += got;
  return Status::ok();
}

Status prefill(jet_model *m, int32_t n_q, const int64_t *offs, const int32_t *tokens, jet_prefix *p) {
  const ModelHeader &h = m->h;
  TRY(check_offsets(offs, n_q, 1, "prefix_offsets"));
  for (int32_t q = 0; q < n_q; ++q)
    if (offs[q + 1] - offs[q] > m->max_ctx)
      return Status::err(JET_E_CAPACITY, "prefix " + std::to_string(q) + " longer than max_ctx");
  const int64_t T = offs[n_q];
  const bool tok_dev = is_device_ptr(tokens);
  TRY(check_ids(m, tokens, T, tok_dev, "prefix_tokens"));
  p->n_q = n_q;
  p->prefix_offsets.assign(offs, offs + n_q + 1);
  p->T = T;
  const size_t kv_bytes = (size_t)(h.n_kv_heads * T * h.head_dim) * m->esz * m->anp;
  p->kcache.assign((size_t)h.n_layers, nullptr);
  p->vcache.assign((size_t)h.n_layers, nullptr);
  p->S_pre.assign((size_t)h.n_layers, nullptr);
  p->conv_tail.assign((size_t)h.n_layers, nullptr);
  const int64_t gH = h.gdn_heads, gC = 2 * h.gdn_heads * h.gdn_dk + h.gdn_heads * h.gdn_dv;
  for (int64_t l = 0; l < h.n_layers; ++l) {
    if (m->layers[(size_t)l].gdn) {
      TRY(palloc(p, (size_t)(n_q * gH * h.gdn_dk * h.gdn_dv) * 4, (void **)&p->S_pre[(size_t)l]));
      const size_t tb = (size_t)(n_q * 3 * gC) * 4;
      TRY(palloc(p, tb, (void **)&p->conv_tail[(size_t)l]));
      HIPC(hipMemsetAsync(p->conv_tail[(size_t)l], 0, tb, m->st));
      continue;
    }
    TRY(palloc(p, kv_bytes, &p->kcache[(size_t)l]));
    TRY(palloc(p, kv_bytes, &p->vcache[(size_t)l]));
  }
  TRY(palloc(p, (size_t)(n_q * h.d) * m->esz * m->np, &p->f_last));

  const int32_t *d_tok = tokens;
  if (!tok_dev) {
    int32_t *dt;
    TRY(ws_t<int32_t>(m, "pre_tok", (size_t)std::max<int64_t>(T, 1), &dt));
    HIPC(hipMemcpyAsync(dt, tokens, (size_t)T * 4, hipMemcpyHostToDevice, m->st));
    d_tok = dt;
  }
  const int dt = m->kdt;
  route_rows_begin(m, 0, T);
  // waves of whole questions under the prefill token budget
  int32_t q0 = 0;
  while (q0 < n_q) {
    int32_t q1 = q0 + 1;
    while (q1 < n_q && (m->prefill_budget <= 0 || offs[q1 + 1] - offs[q0] <= m->prefill_budget)) ++q1;
    const int64_t t0 = offs[q0], R = offs[q1] - offs[q0];
    std::vector<int32_t> pos((size_t)R), last((size_t)(q1 - q0));
    QDesc qd;
    for (int32_t q = q0; q < q1; ++q) {
      const int64_t P = offs[q + 1] - offs[q];
      for (int64_t i = 0; i < P; ++i) pos[(size_t)(offs[q] - t0 + i)] = (int32_t)i;
      last[(size_t)(q - q0)] = (int32_t)(offs[q] - t0 + P - 1);
      qd.qrow0.push_back((int32_t)(offs[q] - t0));
      qd.nrows.push_back((int32_t)P);
      qd.pre_slot0.push_back(offs[q]);
      qd.pre_len.push_back((int32_t)P);
      qd.suf_row0.push_back(0);
      qd.suf_len.push_back(0);
    }
    int32_t *d_pos, *d_last;
    TRY(upload(m, "pre_pos", pos, &d_pos));
    TRY(upload(m, "pre_last", last, &d_last));
    AttnPlan plan;
    TRY(plan_attention(m, 0, qd, "pre_at_", &plan));
    GdnPlan gp;
    if (h.hybrid) {
      std::vector<int32_t> hist((size_t)R * 3), tslot((size_t)R, -1);
      std::vector<jetk::GdnSeq> seqs;
      for (int32_t q = q0; q < q1; ++q) {
        const int64_t P = offs[q + 1] - offs[q], base = offs[q] - t0;
        for (int64_t i = 0; i < P; ++i) {
          for (int j = 1; j <= 3; ++j) hist[(size_t)((base + i) * 3 + j - 1)] = i - j >= 0 ? (int32_t)(base + i - j) : -1;
          if (i >= P - 3) tslot[(size_t)(base + i)] = (int32_t)(q * 3 + (i - (P - 3)));
        }
        seqs.push_back({(int32_t)base, (int32_t)P, -1, q});
      }
      // prefixes in the 16-bit modes run the chunked form (fp16 operands, or
      // bf16 pairs in the pair mode), longest first (no round of the launch
      // waits on one long sequence); models with routed experts keep the fp32
      // stepwise recurrence: a top-k routing decision turns its rounding into
      // a different expert for rows near a tie
      gp.chunked = m->kdt != 1 && !h.n_experts;
      if (gp.chunked)
        std::stable_sort(seqs.begin(), seqs.end(),
                         [](const jetk::GdnSeq &a, const jetk::GdnSeq &b) { return a.len > b.len; });
      TRY(upload(m, "pre_ghist", hist, &gp.hist));
      TRY(upload(m, "pre_gtslot", tslot, &gp.tail_slot));
      TRY(upload(m, "pre_gseqs", seqs, &gp.seqs));
      gp.nseq = (int)seqs.size();
      gp.tok_heads = (double)R * (double)h.gdn_heads;
    }
    WaveBufs b;
    TRY(wave_bufs(m, R, &b));
    {
      KTimer t(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_embed(m->edt, m->embed, d_tok + t0, nullptr, (int)R, (int)h.d, b.resid, m->st));
    }
    // Only the last row of each question goes on past the last layer (to the
    // LM head, Section 4.1), while every row's K/V of that layer is retained:
    // when the last layer is an attention layer, its attention, output
    // projection and FFN run on the last rows alone (attention of the last
    // row over the whole prefix = the candidate kernel with no own rows).
    const int64_t L = h.n_layers;
    const bool last_rows_only = !m->layers[(size_t)(L - 1)].gdn;
    const int32_t nq = q1 - q0;
    for (int64_t l = 0; l < L; ++l) {
      const Layer &ly = m->layers[(size_t)l];
      if (ly.gdn) {
        TRY(gdn_layer(m, ly, b, R, gp, p->conv_tail[(size_t)l], nullptr, p->S_pre[(size_t)l]));
        route_rows_set(m, 0, l, t0, R);
        TRY(ffn(m, ly, b, R));
        continue;
      }
      TRY(attn_in(m, ly, b, R, d_pos, p->kcache[(size_t)l], p->vcache[(size_t)l], T, t0));
      if (l == L - 1 && last_rows_only) break;
      TRY(run_attention(m, plan, b.q, R, b.att, p->kcache[(size_t)l], p->vcache[(size_t)l], T, nullptr, nullptr,
                        0, nullptr, nullptr));
      TRY(attn_out(m, ly, b, R));
      route_rows_set(m, 0, l, t0, R);
      TRY(ffn(m, ly, b, R));
    }
    if (last_rows_only) {
      const Layer &ly = m->layers[(size_t)(L - 1)];
      QDesc ql;
      std::vector<int32_t> zero_t((size_t)R, 0);
      for (int32_t q = q0; q < q1; ++q) {
        const int64_t P = offs[q + 1] - offs[q];
        ql.qrow0.push_back(last[(size_t)(q - q0)]);
        ql.nrows.push_back(1);
        ql.pre_slot0.push_back(offs[q]);
        ql.pre_len.push_back((int32_t)P);
        ql.suf_row0.push_back(0);
        ql.suf_len.push_back(0);
      }
      AttnPlan lp;
      TRY(plan_attention(m, 1, ql, "pre_lr_", &lp));
      int32_t *d_zero_t;
      TRY(upload(m, "pre_lr_t", zero_t, &d_zero_t));
      TRY(run_attention(m, lp, b.q, R, b.att, p->kcache[(size_t)(L - 1)], p->vcache[(size_t)(L - 1)], T, nullptr,
                        nullptr, 0, nullptr, d_zero_t, JET_K_ATTN_PREFIX));
      WaveBufs c;  // the last rows, compacted
      const size_t pe = (size_t)m->np * m->esz, pa = (size_t)m->anp * m->esz;
      TRY(ws_t<float>(m, "lr_resid", (size_t)(nq * h.d), &c.resid));
      TRY(ws(m, "lr_att", (size_t)(nq * h.n_heads * h.head_dim) * pa, &c.att));
      TRY(ws(m, "lr_xn", (size_t)(nq * h.d) * std::max(pe, pa), &c.xn));
      TRY(ws(m, "lr_act", (size_t)(nq * h.ffn) * pe, &c.act));
      {
        KTimer t(m, JET_K_OTHER, 0, 0);
        LAUNCH(jetk::launch_gather_rows(b.resid, h.d * 4, d_last, nq, c.resid, m->st));
        LAUNCH(jetk::launch_gather_rows(b.att, (int64_t)(h.n_heads * h.head_dim) * (int64_t)pa, d_last, nq, c.att,
                                        m->st));
      }
      TRY(attn_out(m, ly, c, nq));
      route_rows_set(m, 0, L - 1, t0, nq, last.data());
      TRY(ffn(m, ly, c, nq));
      KTimer t(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_rmsnorm(dt, m->pair, c.resid, nullptr, m->final_norm, (int)nq, (int)h.d, (float)h.rms_eps,
                                  (char *)p->f_last + (size_t)(q0 * h.d) * m->esz * m->np, m->st));
    } else {
      KTimer t(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_rmsnorm(dt, m->pair, b.resid, d_last, m->final_norm, (int)(q1 - q0), (int)h.d,
                                  (float)h.rms_eps, (char *)p->f_last + (size_t)(q0 * h.d) * m->esz * m->np, m->st));
    }
    m->stats.prefill_waves++;
    q0 = q1;
  }
  m->rt_which = -1;
  TRY(sync(m));
  m->stats.prefix_tokens += T;
  m->stats.prefix_evals += n_q;
  return Status::ok();
}

// ---------------------------------------------------------------------------
// reasoning trace (Section 3.4): sampled once per question, frozen into the
// retained prefix
// ---------------------------------------------------------------------------

// Extends every question's prefix by n sampled tokens. Step t samples token
// t of each question from the prefix's last row (the prefix's first-token
// distribution at t = 0) and then runs that token through the model at
// position P_q + t as one new row per question: its attention reads the
// question's retained K/V (its own row included, appended first), its
// delta-rule layers continue the question's state and convolution tail in
// place. The caches are laid out again once, with room for the n rows after
// each question, so the prefix stays a plain prefix of P_q + n tokens.
Status generate(jet_model *m, jet_prefix *p, int32_t n, float tau, uint64_t seed, int32_t *out) {
  const ModelHeader &h = m->h;
  if (n < 0) return Status::err(JET_E_INVALID, "n_steps must be >= 0");
  if (!(tau >= 0.0f) || !std::isfinite(tau)) return Status::err(JET_E_INVALID, "temperature must be finite and >= 0");
  const int32_t nq = p->n_q;
  if (n >= (1 << 20) || nq >= (1 << 26) || h.vocab > (1 << 18))
    return Status::err(JET_E_INVALID, "trace counters: n_steps < 2^20, n_q < 2^26 and vocab <= 2^18");
  const std::vector<int64_t> offs = p->prefix_offsets;
  for (int32_t q = 0; q < nq; ++q)
    if (offs[q + 1] - offs[q] + n > m->max_ctx)
      return Status::err(JET_E_CAPACITY, "prefix " + std::to_string(q) + " plus the trace is longer than max_ctx");
  if (n == 0) return Status::ok();
  struct SplitK {  // split-K GEMMs for the decode steps of this call only
    jet_model *m;
    explicit SplitK(jet_model *mm) : m(mm) { m->splitk = true; }
    ~SplitK() { m->splitk = false; }
  } splitk_scope(m);
  const bool out_dev = out && is_device_ptr(out);
  const int64_t T = p->T, T2 = T + (int64_t)nq * n, V = h.vocab;
  std::vector<int64_t> offs2((size_t)nq + 1);
  for (int32_t q = 0; q <= nq; ++q) offs2[(size_t)q] = offs[(size_t)q] + (int64_t)q * n;
  m->rt_which = -1;

  // Every buffer is allocated before the prefix changes; once the caches are
  // laid out again only a device error can stop the call (the prefix is then
  // in an unspecified state and may only be freed).
  const int64_t nblk = m->anp * h.n_kv_heads;
  const int64_t row_bytes = h.head_dim * (int64_t)m->esz;
  const int64_t R = nq;
  std::vector<void *> fresh;  // new K then V cache of each attention layer
  for (int64_t l = 0; l < h.n_layers; ++l) {
    if (m->layers[(size_t)l].gdn) continue;
    for (int kv = 0; kv < 2; ++kv) {
      void *nb;
      TRY(palloc(p, (size_t)(nblk * T2 * row_bytes), &nb));
      fresh.push_back(nb);
    }
  }
  int64_t *d_offs;
  int32_t *d_tok, *d_zero_t;
  float *logits;
  void *kt, *vt;
  TRY(upload(m, "gen_offs", offs, &d_offs));
  TRY(ws_t<int32_t>(m, "gen_tok", (size_t)(R * n), &d_tok));
  TRY(ws_t<float>(m, "gen_logits", (size_t)(R * V), &logits));
  TRY(ws(m, "gen_k", (size_t)(nblk * R * row_bytes), &kt));
  TRY(ws(m, "gen_v", (size_t)(nblk * R * row_bytes), &vt));
  void *samp;
  TRY(ws(m, "gen_sample", (size_t)jetk::sample_scratch_bytes((int)R), &samp));
  TRY(upload(m, "gen_zero_t", std::vector<int32_t>((size_t)R, 0), &d_zero_t));
  // attention caches laid out again with n free rows after each question
  size_t fi = 0;
  for (int64_t l = 0; l < h.n_layers; ++l) {
    if (m->layers[(size_t)l].gdn) continue;
    for (int kv = 0; kv < 2; ++kv) {
      void *&buf = kv ? p->vcache[(size_t)l] : p->kcache[(size_t)l];
      void *nb = fresh[fi++];
      {
        KTimer t(m, JET_K_OTHER, 0, 0);
        LAUNCH(jetk::launch_kv_relayout(buf, nb, d_offs, nq, (int)nblk, T, T2, row_bytes, n, m->st));
      }
      // the old buffer goes back to the model's pool (later work on the
      // stream that reuses it runs after the copy)
      for (size_t i = 0; i < p->allocs.size(); ++i)
        if (p->allocs[i].first == buf) {
          m->pool.push_back({p->allocs[i].second, buf});
          p->bytes -= p->allocs[i].second;
          p->allocs.erase(p->allocs.begin() + (std::ptrdiff_t)i);
          break;
        }
      buf = nb;
    }
  }

  const int64_t gH = h.gdn_heads;
  for (int32_t t = 0; t < n; ++t) {
    // token t of every question from the current last rows
    TRY(run_gemm(m, JET_K_LMHEAD, jetk::EPI_STORE_F32, p->f_last, m->np * h.d, m->pair, m->lm_head, h.d, R, V, h.d,
                 logits, V, m->is_lm));
    {
      KTimer tm(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_sample(logits, V, (int)R, (int)V, (double)tau, seed, 0, t, samp, d_tok + t, n, m->st));
    }
    // ... and through the model at positions P_q + t
    std::vector<int32_t> pos((size_t)R), idx((size_t)R), slot((size_t)R);
    QDesc qd;
    for (int32_t q = 0; q < nq; ++q) {
      const int64_t P = offs[(size_t)q + 1] - offs[(size_t)q];
      pos[(size_t)q] = (int32_t)(P + t);
      idx[(size_t)q] = q * n + t;
      slot[(size_t)q] = (int32_t)(offs2[(size_t)q] + P + t);
      qd.qrow0.push_back(q);
      qd.nrows.push_back(1);
      qd.pre_slot0.push_back(offs2[(size_t)q]);
      qd.pre_len.push_back((int32_t)(P + t + 1));
      qd.suf_row0.push_back(0);
      qd.suf_len.push_back(0);
    }
    int32_t *d_pos, *d_idx, *d_slot;
    TRY(upload(m, "gen_pos", pos, &d_pos));
    TRY(upload(m, "gen_idx", idx, &d_idx));
    TRY(upload(m, "gen_slot", slot, &d_slot));
    AttnPlan plan;
    TRY(plan_attention(m, 1, qd, "gen_at_", &plan));
    GdnPlan gp;
    if (h.hybrid) {
      // the convolution tail of question q is a ring of its last 3 input
      // rows: before step t, row j back sits in slot (t + 3 - j) % 3, and
      // the step's row replaces the oldest (slot t % 3) once it is read
      std::vector<int32_t> hist((size_t)R * 3), tslot((size_t)R);
      std::vector<jetk::GdnSeq> seqs;
      for (int32_t q = 0; q < nq; ++q) {
        for (int j = 1; j <= 3; ++j) hist[(size_t)(q * 3 + j - 1)] = -2 - (q * 3 + (t + 3 - j) % 3);
        tslot[(size_t)q] = q * 3 + t % 3;
        seqs.push_back({q, 1, q, q});
      }
      TRY(upload(m, "gen_ghist", hist, &gp.hist));
      TRY(upload(m, "gen_gtslot", tslot, &gp.tail_slot));
      TRY(upload(m, "gen_gseqs", seqs, &gp.seqs));
      gp.nseq = (int)seqs.size();
      gp.tok_heads = (double)R * (double)gH;
    }
    WaveBufs b;
    TRY(wave_bufs(m, R, &b));
    {
      KTimer tm(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_embed(m->edt, m->embed, d_tok, d_idx, (int)R, (int)h.d, b.resid, m->st));
    }
    for (int64_t l = 0; l < h.n_layers; ++l) {
      const Layer &ly = m->layers[(size_t)l];
      if (ly.gdn) {
        TRY(gdn_layer(m, ly, b, R, gp, p->conv_tail[(size_t)l], p->S_pre[(size_t)l], p->S_pre[(size_t)l]));
        TRY(ffn(m, ly, b, R));
        continue;
      }
      TRY(attn_in(m, ly, b, R, d_pos, kt, vt, R, 0));
      {
        KTimer tm(m, JET_K_OTHER, 0, 0);
        LAUNCH(jetk::launch_kv_append(kt, p->kcache[(size_t)l], d_slot, (int)R, (int)nblk, T2, row_bytes, m->st));
        LAUNCH(jetk::launch_kv_append(vt, p->vcache[(size_t)l], d_slot, (int)R, (int)nblk, T2, row_bytes, m->st));
      }
      TRY(run_attention(m, plan, b.q, R, b.att, p->kcache[(size_t)l], p->vcache[(size_t)l], T2, nullptr, nullptr, 0,
                        nullptr, d_zero_t));
      TRY(attn_out(m, ly, b, R));
      TRY(ffn(m, ly, b, R));
    }
    KTimer tm(m, JET_K_OTHER, 0, 0);
    LAUNCH(jetk::launch_rmsnorm(m->kdt, m->pair, b.resid, nullptr, m->final_norm, (int)R, (int)h.d, (float)h.rms_eps,
                                p->f_last, m->st));
  }
  // convolution tails back to the order the scoring path reads (oldest first)
  if (h.hybrid && n % 3) {
    const int64_t gC = 2 * gH * h.gdn_dk + gH * h.gdn_dv;
    std::vector<int32_t> rot((size_t)nq * 3);
    for (int32_t q = 0; q < nq; ++q)
      for (int s2 = 0; s2 < 3; ++s2) rot[(size_t)(q * 3 + s2)] = q * 3 + (n + s2) % 3;
    int32_t *d_rot;
    float *tmp;
    TRY(upload(m, "gen_rot", rot, &d_rot));
    TRY(ws_t<float>(m, "gen_tail", (size_t)(nq * 3 * gC), &tmp));
    for (int64_t l = 0; l < h.n_layers; ++l) {
      if (!m->layers[(size_t)l].gdn) continue;
      KTimer tm(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_gather_rows(p->conv_tail[(size_t)l], gC * 4, d_rot, nq * 3, tmp, m->st));
      HIPC(hipMemcpyAsync(p->conv_tail[(size_t)l], tmp, (size_t)(nq * 3 * gC) * 4, hipMemcpyDeviceToDevice, m->st));
    }
  }
  std::vector<int32_t> toks((size_t)(R * n));
  HIPC(hipMemcpyAsync(toks.data(), d_tok, toks.size() * 4, hipMemcpyDeviceToHost, m->st));
  TRY(sync(m));
  for (int32_t v : toks)
    if (v < 0) return Status::err(JET_E_DEVICE, "sampling met no finite logit");
  p->prefix_offsets = offs2;
  p->T = T2;
  m->stats.prefix_tokens += R * n;
  if (out) {
    if (out_dev) HIPC(hipMemcpy(out, toks.data(), toks.size() * 4, hipMemcpyHostToDevice));
    else std::memcpy(out, toks.data(), toks.size() * 4);
  }
  return Status::ok();
}

// ---------------------------------------------------------------------------
// candidate scoring
// ---------------------------------------------------------------------------

// Drops the arena buffers carved since the call-level mark (a new wave).
void arena_reset(jet_model *m) {
  for (auto it = m->arena_map.begin(); it != m->arena_map.end();) {
    if (it->second.first >= m->arena_mark) it = m->arena_map.erase(it);
    else ++it;
  }
  m->arena_top = m->arena_mark;
}

// Upper bound of the work-buffer bytes of one scoring wave: per body row,
// and fixed (mixture-of-experts segment padding, alignment of each buffer).
// Mirrors the workspace requests of the scoring path (wave buffers, the
// candidate rows' K/V, the final-norm rows, log-sum-exp partials, attention
// work items, delta-rule and expert buffers).
void wave_bytes_bound(const jet_model *m, double *per_row, double *fixed) {
  const ModelHeader &h = m->h;
  const double d = (double)h.d, esz = (double)m->esz;
  const double pe = m->np * esz, pa = m->anp * esz;
  const double nqkv = (double)((h.n_heads + 2 * h.n_kv_heads) * h.head_dim), hq = (double)(h.n_heads * h.head_dim);
  int tps = 1, nsplit = 1;
  jetk::lmhead_plan(m->kdt, (int)h.vocab, 1, &tps, &nsplit);
  double r = d * 4 + nqkv * 4 + d * std::max(pe, pa) + 2 * hq * pa + (double)h.ffn * pe;  // wave buffers
  r += 2.0 * (double)(h.n_kv_heads * h.head_dim) * esz * m->anp;                           // own K / V
  r += 2 * (d * esz * m->np + 8);  // final-norm rows, and again in scored-token order; lse, target logit
  r += 2.0 * nsplit * 4;            // LM-head partials
  r += 40.0 * (double)h.n_kv_heads + 28;  // attention items and per-question tables (at most one question per row)
  double f = 64.0 * 256;                  // alignment of every buffer
  if (h.hybrid) {
    const double H = (double)h.gdn_heads, dk = (double)h.gdn_dk, dv = (double)h.gdn_dv;
    int64_t n_in = 0;
    for (const Layer &ly : m->layers) n_in = std::max(n_in, ly.n_in);
    r += (double)n_in * 4 + 2 * H * dk * 4 + 2 * H * dv * 4 + 2 * H * 4 + H * dv * esz * m->np + 12 + 16;
  }
  if (h.n_experts) {
    const double k = (double)h.top_k, E = (double)h.n_experts, Fe = (double)h.moe_ffn, Fs = (double)h.shared_ffn;
    const double bm = (double)std::max(jetk::gemm_group_rows(m->kdt, 0), jetk::gemm_group_rows(m->kdt, 1));
    int64_t n_router = 0;
    for (const Layer &ly : m->layers) n_router = std::max(n_router, ly.n_router);
    r += (double)n_router * 4 + 3 * k * 4 + (k / bm) * 4 + 2 * E * 4 * k / jetk::kMoeChunk;
    r += k * (2 * d + Fe) * esz;          // routed rows: gathered input, hidden, output
    r += 4 + Fs * esz + d * 4;            // shared expert
    f += (E * bm + bm) * (2 * d + Fe) * esz + 4 * (E + 2) + 2 * E * 4;
  }
  *per_row = r;
  *fixed = f;
}

Status score(jet_model *m, const jet_prefix *p, const int64_t *qco, const int64_t *cto, const int32_t *tokens,
             float *out_tok, float *out_sum) {
  const ModelHeader &h = m->h;
  if (!p->m) return Status::err(JET_E_INVALID, "prefix is detached: its model was freed");
  if (p->m != m) return Status::err(JET_E_INVALID, "prefix belongs to another model");
  if (!out_sum) return Status::err(JET_E_INVALID, "out_cand_sum is NULL");
  CandLayout L;
  TRY(build_cand_layout(p->n_q, p->prefix_offsets.data(), qco, cto, m->max_ctx, &L));
  const int64_t N = L.n_cand, NT = L.n_tok;
  if (N == 0) return Status::ok();
  const bool tok_dev = is_device_ptr(tokens);
  TRY(check_ids(m, tokens, NT, tok_dev, "cand_tokens"));
  const int dt = m->kdt;

  const int32_t *d_tok = tokens;
  if (!tok_dev) {
    int32_t *d;
    TRY(ws_t<int32_t>(m, "cand_tok", (size_t)NT, &d));
    HIPC(hipMemcpyAsync(d, tokens, (size_t)NT * 4, hipMemcpyHostToDevice, m->st));
    d_tok = d;
  }
  int32_t *d_rpos, *d_rtok, *d_rc, *d_rt, *d_lm;
  int64_t *d_cto;
  TRY(upload(m, "row_pos", L.row_pos, &d_rpos));
  TRY(upload(m, "row_tok", L.row_tok, &d_rtok));
  // body rows of each row's candidate (the candidate attention's own-key tiles)
  std::vector<int32_t> row_n((size_t)L.n_rows);
  for (int64_t r = 0; r < L.n_rows; ++r) {
    const int64_t c = L.row_c[(size_t)r];
    row_n[(size_t)r] = (int32_t)(cto[c + 1] - cto[c] - 1);
  }
  TRY(upload(m, "row_n", row_n, &d_rc));
  TRY(upload(m, "row_t", L.row_t, &d_rt));
  TRY(upload(m, "lm_row", L.lm_row, &d_lm));
  std::vector<int64_t> cto_v(cto, cto + N + 1);
  TRY(upload(m, "cto", cto_v, &d_cto));
  float *d_ell, *d_sum;
  TRY(ws_t<float>(m, "ell", (size_t)NT, &d_ell));
  TRY(ws_t<float>(m, "csum", (size_t)N, &d_sum));

  // question of each candidate
  std::vector<int32_t> cand_q((size_t)N);
  for (int32_t q = 0; q < p->n_q; ++q)
    for (int64_t c = qco[q]; c < qco[q + 1]; ++c) cand_q[(size_t)c] = q;
  auto row0 = [&](int64_t c) { return c < N ? (int64_t)L.cand_row0[(size_t)c] : L.n_rows; };
  route_rows_begin(m, 1, L.n_rows);

  int64_t budget = m->wave_budget;
  if (m->arena) {
    // allocation-free call: the buffers above stay for the whole call; every
    // wave's buffers are carved after them, in waves sized to fit
    m->arena_mark = m->arena_top;
    double per_row = 0, fixed = 0;
    wave_bytes_bound(m, &per_row, &fixed);
    const double room = (double)m->arena_cap - (double)m->arena_mark - fixed;
    const int64_t fit = room > per_row ? (int64_t)(room / per_row) : 0;
    int64_t longest = 0;
    for (int64_t c = 0; c < N; ++c) longest = std::max<int64_t>(longest, cto[c + 1] - cto[c]);
    if (fit < std::max<int64_t>(longest, 1))
      return Status::err(JET_E_CAPACITY, "the scratch of " + std::to_string(m->arena_cap) +
                                             " bytes holds the call's tables and " + std::to_string(fit) +
                                             " candidate tokens per wave; the longest candidate has " +
                                             std::to_string(longest));
    budget = budget > 0 ? std::min(budget, fit) : fit;
  }

  int64_t c0 = 0;
  while (c0 < N) {
    if (m->arena) arena_reset(m);
    int64_t c1 = c0 + 1;
    // a wave holds whole candidates, at most `budget` scored tokens (each
    // token is one LM-head row; body rows are one fewer per candidate)
    while (c1 < N && (budget <= 0 || cto[c1 + 1] - cto[c0] <= budget)) ++c1;
    const int64_t r0 = row0(c0), r1 = row0(c1), R = r1 - r0;
    const int64_t t0 = cto[c0], t1 = cto[c1];
    void *f_body = nullptr;
    if (R > 0) {
      QDesc qd;
      int64_t c = c0;
      while (c < c1) {
        const int32_t q = cand_q[(size_t)c];
        int64_t ce = c;
        while (ce < c1 && cand_q[(size_t)ce] == q) ++ce;
        const int64_t a = row0(c) - r0, e = row0(ce) - r0;
        qd.qrow0.push_back((int32_t)a);
        qd.nrows.push_back((int32_t)(e - a));
        qd.pre_slot0.push_back(p->prefix_offsets[(size_t)q]);
        qd.pre_len.push_back((int32_t)(p->prefix_offsets[(size_t)q + 1] - p->prefix_offsets[(size_t)q]));
        qd.suf_row0.push_back((int32_t)a);
        qd.suf_len.push_back((int32_t)(e - a));
        c = ce;
      }
      AttnPlan plan;
      TRY(plan_attention(m, 1, qd, "cand_at_", &plan));
      GdnPlan gp;
      if (h.hybrid) {
        // conv history: own earlier rows, then the question's prefix tail
        std::vector<int32_t> hist((size_t)R * 3);
        std::vector<jetk::GdnSeq> seqs;
        for (int64_t r = r0; r < r1; ++r) {
          const int32_t t = L.row_t[(size_t)r], q = L.row_q[(size_t)r];
          for (int j = 1; j <= 3; ++j)
            hist[(size_t)((r - r0) * 3 + j - 1)] = j <= t - 1 ? (int32_t)(r - r0 - j) : -(2 + (q * 3 + (t + 2 - j)));
        }
        for (int64_t cc = c0; cc < c1; ++cc) {
          const int64_t a = row0(cc), e = row0(cc + 1);
          if (e > a) seqs.push_back({(int32_t)(a - r0), (int32_t)(e - a), cand_q[(size_t)cc], -1});
        }
        TRY(upload(m, "cand_ghist", hist, &gp.hist));
        TRY(upload(m, "cand_gseqs", seqs, &gp.seqs));
        gp.nseq = (int)seqs.size();
        gp.tok_heads = (double)R * (double)h.gdn_heads;
      }
      WaveBufs b;
      TRY(wave_bufs(m, R, &b));
      void *kc, *vc;
      const size_t kvb = (size_t)(h.n_kv_heads * R * h.head_dim) * m->esz * m->anp;
      TRY(ws(m, "cand_k", kvb, &kc));
      TRY(ws(m, "cand_v", kvb, &vc));
      {
        KTimer t(m, JET_K_OTHER, 0, 0);
        LAUNCH(jetk::launch_embed(m->edt, m->embed, d_tok, d_rtok + r0, (int)R, (int)h.d, b.resid, m->st));
      }
      for (int64_t l = 0; l < h.n_layers; ++l) {
        const Layer &ly = m->layers[(size_t)l];
        if (ly.gdn) {
          TRY(gdn_layer(m, ly, b, R, gp, p->conv_tail[(size_t)l], p->S_pre[(size_t)l], nullptr));
        } else {
          TRY(attn_in(m, ly, b, R, d_rpos + r0, kc, vc, R, 0));
          TRY(run_attention(m, plan, b.q, R, b.att, p->kcache[(size_t)l], p->vcache[(size_t)l], p->T, kc, vc, R,
                            d_rc + r0, d_rt + r0));
          TRY(attn_out(m, ly, b, R));
        }
        route_rows_set(m, 1, l, r0, R);
        TRY(ffn(m, ly, b, R));
      }
      m->rt_which = -1;
      TRY(ws(m, "f_body", (size_t)(R * h.d) * m->esz * m->np, &f_body));
      {
        KTimer t(m, JET_K_OTHER, 0, 0);
        LAUNCH(jetk::launch_rmsnorm(dt, m->pair, b.resid, nullptr, m->final_norm, (int)R, (int)h.d,
                                    (float)h.rms_eps, f_body, m->st));
      }
    }
    // one LM-head row per scored token, in token order: the candidate's
    // previous body row, or the question's last prefix row for its first
    // token; the head's tiles keep each row's target logit
    const int64_t nt = t1 - t0, row_bytes = h.d * m->esz * m->np;
    void *f_tok;
    float *lse_tok;
    TRY(ws(m, "f_tok", (size_t)(nt * row_bytes), &f_tok));
    TRY(ws_t<float>(m, "lse_tok", (size_t)nt, &lse_tok));
    {
      KTimer t(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_token_rows(d_lm + t0, (int)nt, (int)r0, f_body, p->f_last, row_bytes, f_tok, m->st));
    }
    TRY(run_lmhead(m, f_tok, nt, lse_tok, d_tok + t0, d_ell + t0));
    {
      KTimer t(m, JET_K_OTHER, 0, 0);
      LAUNCH(jetk::launch_segment_sum(d_ell + t0, d_cto + c0, (int)(c1 - c0), d_sum + c0, m->st));
    }
    m->stats.score_waves++;
    c0 = c1;
  }
  const hipMemcpyKind k_sum = is_device_ptr(out_sum) ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
  HIPC(hipMemcpyAsync(out_sum, d_sum, (size_t)N * 4, k_sum, m->st));
  if (out_tok) {
    const hipMemcpyKind k_tok = is_device_ptr(out_tok) ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
    HIPC(hipMemcpyAsync(out_tok, d_ell, (size_t)NT * 4, k_tok, m->st));
  }
  TRY(sync(m));
  m->stats.cand_body_tokens += L.n_rows;
  m->stats.scored_tokens += NT;
  return Status::ok();
}

void free_model(jet_model *m) {
  if (!m) return;
  (void)hipSetDevice(m->device);
  if (m->st) (void)hipStreamSynchronize(m->st);
  // prefixes still alive lose their buffers now and are detached, so that a
  // later jet_prefix_free only deletes the handle
  for (jet_prefix *p : m->live) {
    for (auto &a : p->allocs) (void)hipFree(a.first);
    p->allocs.clear();
    p->kcache.clear();
    p->vcache.clear();
    p->S_pre.clear();
    p->conv_tail.clear();
    p->f_last = nullptr;
    p->m = nullptr;
  }
  m->live.clear();
  for (auto &kv : m->ws) (void)hipFree(kv.second.p);
  for (void *a : m->weight_allocs) (void)hipFree(a);
  for (auto &e : m->pool) (void)hipFree(e.second);
  for (auto &p : m->pending) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  for (auto e : m->event_pool) (void)hipEventDestroy(e);
  delete m;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" int jet_model_load(const char *model_path, const jet_load_opts *opts, jet_model **out) {
  clear_error();
  if (!out) return fail(Status::err(JET_E_INVALID, "out is NULL"));
  *out = nullptr;
  if (!model_path) return fail(Status::err(JET_E_INVALID, "model_path is NULL"));
  jet_model *m = new jet_model();
  if (opts) {
    if (opts->dtype != JET_BF16 && opts->dtype != JET_FP32 && opts->dtype != JET_BF16_SINGLE &&
        opts->dtype != JET_F16 && opts->dtype != JET_F16P) {
      delete m;
      return fail(Status::err(JET_E_INVALID, "unknown dtype"));
    }
    if (opts->max_ctx < 0 || opts->prefill_token_budget < 0 || opts->wave_token_budget < 0 ||
        opts->max_device_bytes < 0) {
      delete m;
      return fail(Status::err(JET_E_INVALID, "negative option"));
    }
    m->dtype = opts->dtype;
    m->device = opts->device;
    m->prefill_budget = opts->prefill_token_budget;
    m->wave_budget = opts->wave_token_budget;
    m->max_bytes = opts->max_device_bytes;
    m->st = (hipStream_t)opts->hip_stream;
    m->flags = opts->flags;
  }
  Status s = load_model(m, model_path, opts);
  if (!s) {
    free_model(m);
    return fail(s);
  }
  *out = m;
  return JET_OK;
}

extern "C" int jet_prefill_prefix(jet_model *model, int32_t n_q, const int64_t *prefix_offsets,
                                  const int32_t *prefix_tokens, jet_prefix **out) {
  clear_error();
  if (!out) return fail(Status::err(JET_E_INVALID, "out is NULL"));
  *out = nullptr;
  if (!model) return fail(Status::err(JET_E_INVALID, "model is NULL"));
  if (n_q < 1) return fail(Status::err(JET_E_INVALID, "n_q must be >= 1"));
  if (hipSetDevice(model->device) != hipSuccess) return fail(Status::err(JET_E_DEVICE, "hipSetDevice failed"));
  jet_prefix *p = new jet_prefix();
  p->m = model;
  model->live.push_back(p);
  Status s = prefill(model, n_q, prefix_offsets, prefix_tokens, p);
  if (!s) {
    (void)hipStreamSynchronize(model->st);
    drain_timers(model);
    free_prefix(p);
    return fail(s);
  }
  *out = p;
  return JET_OK;
}

extern "C" int jet_generate_trace(jet_model *model, jet_prefix *prefix, int32_t n_steps, float temperature,
                                  uint64_t seed, int32_t *out_tokens) {
  clear_error();
  if (!model || !prefix) return fail(Status::err(JET_E_INVALID, "model or prefix is NULL"));
  if (prefix->m != model) return fail(Status::err(JET_E_INVALID, "prefix was not made from this model"));
  if (hipSetDevice(model->device) != hipSuccess) return fail(Status::err(JET_E_DEVICE, "hipSetDevice failed"));
  Status s = generate(model, prefix, n_steps, temperature, seed, out_tokens);
  if (!s) {
    (void)hipStreamSynchronize(model->st);
    drain_timers(model);
    return fail(s);
  }
  return JET_OK;
}

extern "C" int jet_score_candidates(jet_model *model, const jet_prefix *prefix, const int64_t *q_cand_offsets,
                                    const int64_t *cand_tok_offsets, const int32_t *cand_tokens,
                                    float *out_token_logprob, float *out_cand_sum) {
  clear_error();
  if (!model || !prefix) return fail(Status::err(JET_E_INVALID, "model or prefix is NULL"));
  if (hipSetDevice(model->device) != hipSuccess) return fail(Status::err(JET_E_DEVICE, "hipSetDevice failed"));
  Status s = score(model, prefix, q_cand_offsets, cand_tok_offsets, cand_tokens, out_token_logprob, out_cand_sum);
  if (!s) {
    (void)hipStreamSynchronize(model->st);
    drain_timers(model);
    return fail(s);
  }
  return JET_OK;
}

extern "C" int jet_score_candidates_noalloc(jet_model *model, const jet_prefix *prefix,
                                            const int64_t *q_cand_offsets, const int64_t *cand_tok_offsets,
                                            const int32_t *cand_tokens, float *out_token_logprob,
                                            float *out_cand_sum) {
  clear_error();
  if (!model || !prefix) return fail(Status::err(JET_E_INVALID, "model or prefix is NULL"));
  if (hipSetDevice(model->device) != hipSuccess) return fail(Status::err(JET_E_DEVICE, "hipSetDevice failed"));
  void *scratch = noalloc_scratch(model->device);
  if (model->scratch_status != hipSuccess || !scratch)
    return fail(Status::err(JET_E_DEVICE, std::string("no scratch on this device: ") +
                                              hipGetErrorString(model->scratch_status)));
  model->arena = (char *)scratch;
  model->arena_cap = kNoallocScratchBytes;
  model->arena_top = model->arena_mark = 0;
  model->arena_map.clear();
  Status s = score(model, prefix, q_cand_offsets, cand_tok_offsets, cand_tokens, out_token_logprob, out_cand_sum);
  if (!s) (void)hipStreamSynchronize(model->st);
  model->arena = nullptr;
  model->arena_cap = model->arena_top = model->arena_mark = 0;
  model->arena_map.clear();
  if (!s) {
    drain_timers(model);
    return fail(s);
  }
  return JET_OK;
}

extern "C" int jet_stats_get(const jet_model *model, jet_stats *out) {
  clear_error();
  if (!model || !out) return fail(Status::err(JET_E_INVALID, "NULL argument"));
  *out = model->stats;
  return JET_OK;
}

extern "C" int jet_stats_reset(jet_model *model) {
  clear_error();
  if (!model) return fail(Status::err(JET_E_INVALID, "NULL argument"));
  model->stats = jet_stats{};
  return JET_OK;
}

extern "C" int jet_model_info(const jet_model *model, int64_t *vocab, int64_t *n_layers, int64_t *max_ctx,
                              int32_t *dtype, int64_t *f16_inexact_weights) {
  clear_error();
  if (!model) return fail(Status::err(JET_E_INVALID, "NULL model"));
  if (f16_inexact_weights) *f16_inexact_weights = model->f16_inexact;
  if (vocab) *vocab = model->h.vocab;
  if (n_layers) *n_layers = model->h.n_layers;
  if (max_ctx) *max_ctx = model->max_ctx;
  if (dtype) *dtype = model->dtype;
  return JET_OK;
}

extern "C" int jet_routes_get(const jet_model *model, int32_t which, int64_t *out_rows, int32_t *out_layers,
                              int32_t *out_top_k, int32_t *out_ids, int64_t cap_ids) {
  clear_error();
  if (!model) return fail(Status::err(JET_E_INVALID, "NULL model"));
  if (!model->h.n_experts) return fail(Status::err(JET_E_INVALID, "the model has no experts"));
  if (!(model->flags & JET_FLAG_RECORD_ROUTES))
    return fail(Status::err(JET_E_INVALID, "the model was loaded without JET_FLAG_RECORD_ROUTES"));
  if (which != 0 && which != 1) return fail(Status::err(JET_E_INVALID, "which must be 0 (prefill) or 1 (score)"));
  const auto &rec = model->routes[which];
  if (out_ids && (int64_t)rec.size() > cap_ids)
    return fail(Status::err(JET_E_CAPACITY, "cap_ids smaller than layers * rows * top_k"));
  if (out_rows) *out_rows = model->route_rows[which];
  if (out_layers) *out_layers = (int32_t)model->h.n_layers;
  if (out_top_k) *out_top_k = (int32_t)model->h.top_k;
  if (out_ids && !rec.empty()) std::memcpy(out_ids, rec.data(), rec.size() * sizeof(int32_t));
  return JET_OK;
}

extern "C" void jet_prefix_free(jet_prefix *prefix) {
  if (prefix && prefix->m) (void)hipSetDevice(prefix->m->device);
  free_prefix(prefix);
}

extern "C" void jet_model_free(jet_model *model) { free_model(model); }

// Model file header parsing (a small JSON reader for the header's subset:
// objects, arrays, strings, numbers, booleans, null) and tensor reads.
#include "model_file.h"

#include <cctype>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fcntl.h>
#include <memory>
#include <unistd.h>

namespace jet {
namespace {

struct JVal {
  enum Kind { NUL, BOOL, NUM, STR, ARR, OBJ } kind = NUL;
  bool b = false;
  double num = 0;
  std::string str;
  std::vector<JVal> arr;
  std::vector<std::pair<std::string, JVal>> obj;
  const JVal *get(const std::string &k) const {
    for (auto &kv : obj)
      if (kv.first == k) return &kv.second;
    return nullptr;
  }
};

struct JParser {
  const char *p, *e;
  std::string err;
  void ws() {
    while (p < e && std::isspace((unsigned char)*p)) ++p;
  }
  bool lit(const char *s) {
    size_t n = std::strlen(s);
    if ((size_t)(e - p) >= n && std::memcmp(p, s, n) == 0) { p += n; return true; }
    return false;
  }
  bool str(std::string *out) {
    if (p >= e || *p != '"') return false;
    ++p;
    while (p < e && *p != '"') {
      if (*p == '\\') {
        ++p;
        if (p >= e) return false;
        char c = *p;
        if (c == 'n') out->push_back('\n');
        else if (c == 't') out->push_back('\t');
        else if (c == 'u') {  // header strings are ASCII; keep the escape literally
          out->append("\\u");
        } else out->push_back(c);
        ++p;
      } else out->push_back(*p++);
    }
    if (p >= e) return false;
    ++p;
    return true;
  }
  bool val(JVal *v, int depth = 0) {
    if (depth > 64) return false;
    ws();
    if (p >= e) return false;
    if (*p == '{') {
      v->kind = JVal::OBJ;
      ++p;
      ws();
      if (p < e && *p == '}') { ++p; return true; }
      for (;;) {
        ws();
        std::string k;
        if (!str(&k)) return false;
        ws();
        if (p >= e || *p != ':') return false;
        ++p;
        JVal c;
        if (!val(&c, depth + 1)) return false;
        v->obj.emplace_back(std::move(k), std::move(c));
        ws();
        if (p < e && *p == ',') { ++p; continue; }
        if (p < e && *p == '}') { ++p; return true; }
        return false;
      }
    }
    if (*p == '[') {
      v->kind = JVal::ARR;
      ++p;
      ws();
      if (p < e && *p == ']') { ++p; return true; }
      for (;;) {
        JVal c;
        if (!val(&c, depth + 1)) return false;
        v->arr.push_back(std::move(c));
        ws();
        if (p < e && *p == ',') { ++p; continue; }
        if (p < e && *p == ']') { ++p; return true; }
        return false;
      }
    }
    if (*p == '"') { v->kind = JVal::STR; return str(&v->str); }
    if (lit("true")) { v->kind = JVal::BOOL; v->b = true; return true; }
    if (lit("false")) { v->kind = JVal::BOOL; v->b = false; return true; }
    if (lit("null")) { v->kind = JVal::NUL; return true; }
    char *end = nullptr;
    std::string tmp(p, (size_t)std::min<ptrdiff_t>(e - p, 64));
    double d = std::strtod(tmp.c_str(), &end);
    if (end == tmp.c_str()) return false;
    p += (end - tmp.c_str());
    v->kind = JVal::NUM;
    v->num = d;
    return true;
  }
};

// A whole number in [0, 2^53] (every size and offset in a header is one).
bool as_count(const JVal &v, int64_t *out) {
  if (v.kind != JVal::NUM || !(v.num >= 0.0) || v.num > 9007199254740992.0 || v.num != (double)(int64_t)v.num)
    return false;
  *out = (int64_t)v.num;
  return true;
}

// Absent and not required: true, *out untouched. Present: must be a count.
bool get_int(const JVal &o, const char *k, int64_t *out, bool required = true) {
  const JVal *v = o.get(k);
  if (!v) return !required;
  return as_count(*v, out);
}

}  // namespace

Status read_model_header(const std::string &path, ModelHeader *h) {
  FILE *f = std::fopen(path.c_str(), "rb");
  if (!f) return Status::err(JET_E_IO, "cannot open model file " + path);
  unsigned char head[16];
  if (std::fread(head, 1, 16, f) != 16 || std::memcmp(head, "JETMDL01", 8) != 0) {
    std::fclose(f);
    return Status::err(JET_E_IO, path + ": not a model file (bad magic)");
  }
  uint64_t n = 0;
  std::memcpy(&n, head + 8, 8);
  if (n == 0 || n > (64u << 20)) {
    std::fclose(f);
    return Status::err(JET_E_IO, path + ": bad header length");
  }
  std::string js(n, '\0');
  size_t got = std::fread(&js[0], 1, n, f);
  std::fclose(f);
  if (got != n) return Status::err(JET_E_IO, path + ": truncated header");
  JParser P{js.data(), js.data() + js.size(), {}};
  JVal root;
  if (!P.val(&root) || root.kind != JVal::OBJ) return Status::err(JET_E_IO, path + ": malformed header JSON");
  const JVal *arch = root.get("arch"), *dt = root.get("dtype");
  if (!arch || arch->kind != JVal::STR || !dt || dt->kind != JVal::STR)
    return Status::err(JET_E_IO, path + ": header lacks arch/dtype");
  if (arch->str != "dense" && arch->str != "hybrid") return Status::err(JET_E_IO, "unknown arch " + arch->str);
  if (dt->str != "bf16" && dt->str != "f32" && dt->str != "q8" && dt->str != "q4")
    return Status::err(JET_E_IO, "unknown dtype " + dt->str);
  h->hybrid = arch->str == "hybrid";
  h->q8 = dt->str == "q8" || dt->str == "q4";
  h->qbits = dt->str == "q8" ? 8 : dt->str == "q4" ? 4 : 0;
  h->bf16 = dt->str == "bf16" || h->q8;
  bool ok = get_int(root, "d_model", &h->d) && get_int(root, "n_layers", &h->n_layers) &&
            get_int(root, "n_heads", &h->n_heads) && get_int(root, "n_kv_heads", &h->n_kv_heads) &&
            get_int(root, "head_dim", &h->head_dim) && get_int(root, "ffn", &h->ffn) &&
            get_int(root, "vocab", &h->vocab) && get_int(root, "max_ctx", &h->max_ctx);
  if (!ok) return Status::err(JET_E_IO, path + ": header lacks a model dimension");
  ok = get_int(root, "gdn_heads", &h->gdn_heads, false) && get_int(root, "gdn_dk", &h->gdn_dk, false) &&
       get_int(root, "gdn_dv", &h->gdn_dv, false) && get_int(root, "conv_kernel", &h->conv_kernel, false) &&
       get_int(root, "n_experts", &h->n_experts, false) && get_int(root, "top_k", &h->top_k, false) &&
       get_int(root, "moe_ffn", &h->moe_ffn, false) && get_int(root, "shared_ffn", &h->shared_ffn, false);
  if (!ok) return Status::err(JET_E_IO, path + ": a model dimension is not a non-negative whole number");
  if (const JVal *v = root.get("rms_eps")) {
    if (v->kind != JVal::NUM || !(v->num > 0.0)) return Status::err(JET_E_IO, path + ": bad rms_eps");
    h->rms_eps = v->num;
  }
  if (const JVal *v = root.get("rope_theta")) {
    if (v->kind != JVal::NUM || !(v->num > 0.0)) return Status::err(JET_E_IO, path + ": bad rope_theta");
    h->rope_theta = v->num;
  }
  const JVal *lt = root.get("layer_types");
  if (!lt || lt->kind != JVal::ARR || (int64_t)lt->arr.size() != h->n_layers)
    return Status::err(JET_E_IO, path + ": layer_types missing or wrong length");
  for (auto &x : lt->arr) {
    if (x.kind != JVal::STR || (x.str != "attn" && x.str != "gdn"))
      return Status::err(JET_E_IO, path + ": bad layer type");
    h->layer_is_gdn.push_back(x.str == "gdn");
  }
  const JVal *ts = root.get("tensors");
  if (!ts || ts->kind != JVal::ARR) return Status::err(JET_E_IO, path + ": header lacks tensors");
  for (auto &t : ts->arr) {
    TensorInfo ti;
    const JVal *nm = t.get("name"), *tdt = t.get("dtype"), *sh = t.get("shape");
    if (!nm || nm->kind != JVal::STR || !tdt || tdt->kind != JVal::STR || !sh || sh->kind != JVal::ARR ||
        (tdt->str != "bf16" && tdt->str != "f32" && tdt->str != "q8" && tdt->str != "q4"))
      return Status::err(JET_E_IO, path + ": bad tensor entry");
    ti.name = nm->str;
    ti.bf16 = tdt->str == "bf16";
    ti.q8 = tdt->str == "q8" || tdt->str == "q4";
    ti.qbits = tdt->str == "q8" ? 8 : tdt->str == "q4" ? 4 : 0;
    int64_t numel = 1;
    for (auto &s : sh->arr) {
      int64_t dim = 0;
      if (!as_count(s, &dim) || (dim > 0 && numel > (INT64_C(1) << 40) / dim))
        return Status::err(JET_E_IO, path + ": tensor " + ti.name + " has a bad shape");
      numel *= dim;
      ti.shape.push_back(dim);
    }
    if (!get_int(t, "offset", &ti.offset) || !get_int(t, "nbytes", &ti.nbytes))
      return Status::err(JET_E_IO, path + ": tensor lacks offset/nbytes");
    if (ti.q8 && (ti.shape.empty() || ti.shape.back() % 32 != 0))
      return Status::err(JET_E_IO, path + ": block-quantized tensor " + ti.name +
                                       " needs a last dimension multiple of 32");
    if (ti.q8 && h->qbits != ti.qbits)
      return Status::err(JET_E_IO, path + ": tensor " + ti.name + " is quantized unlike the model");
    if (ti.nbytes != (ti.q8 ? numel * ti.qbits / 8 + numel / 32 : numel * (ti.bf16 ? 2 : 4)))
      return Status::err(JET_E_IO, path + ": tensor " + ti.name + " size mismatch");
    h->tensors[ti.name] = ti;
  }
  return Status::ok();
}

Status read_tensor_bytes(const std::string &path, const TensorInfo &t, void *dst) {
  int fd = ::open(path.c_str(), O_RDONLY);
  if (fd < 0) return Status::err(JET_E_IO, "cannot open " + path);
  int64_t done = 0;
  while (done < t.nbytes) {
    ssize_t r = ::pread(fd, (char *)dst + done, (size_t)std::min<int64_t>(t.nbytes - done, 1 << 30),
                        t.offset + done);
    if (r <= 0) {
      ::close(fd);
      return Status::err(JET_E_IO, path + ": short read of tensor " + t.name);
    }
    done += r;
  }
  ::close(fd);
  return Status::ok();
}

}  // namespace jet

// A stage's weights from safetensors files, by byte range (include/kafila_shard.h).
// Host only: header parsing, the stage's tensor list, positioned reads, and the
// tensors held between fetches so that a replanned division re-reads only what it
// lacks.
#include "kafila_shard.h"

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <cerrno>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "error.h"

using kf::fail;

namespace {

// ------------------------------------------------------------------ JSON (the header's subset)
// Objects, arrays, strings, integers (kept exact in int64), other numbers, true,
// false and null: enough for a safetensors header, whose values are an object per
// tensor (dtype, shape, data_offsets) and an optional string-to-string metadata map.
struct Json {
  enum Type { kNull, kBool, kInt, kNum, kStr, kArr, kObj } type = kNull;
  bool b = false;
  int64_t i = 0;
  double d = 0.0;
  std::string s;
  std::vector<Json> arr;
  std::vector<std::pair<std::string, Json>> obj;
  const Json* get(const char* key) const {
    for (const auto& kv : obj)
      if (kv.first == key) return &kv.second;
    return nullptr;
  }
};

class Parser {
 public:
  Parser(const char* p, const char* e) : p_(p), e_(e) {}
  bool parse(Json& out, std::string& err) {
    if (!value(out, 0)) {
      err = err_.empty() ? "malformed JSON" : err_;
      return false;
    }
    ws();
    while (p_ < e_ && *p_ == ' ') ++p_;  // the header may be padded with spaces
    if (p_ != e_) {
      err = "trailing bytes after the JSON header";
      return false;
    }
    return true;
  }

 private:
  const char* p_;
  const char* e_;
  std::string err_;
  void ws() {
    while (p_ < e_ && (*p_ == ' ' || *p_ == '\n' || *p_ == '\r' || *p_ == '\t')) ++p_;
  }
  bool lit(const char* w) {
    const size_t n = strlen(w);
    if ((size_t)(e_ - p_) < n || memcmp(p_, w, n) != 0) return false;
    p_ += n;
    return true;
  }
  bool str(std::string& out) {
    if (p_ >= e_ || *p_ != '"') return false;
    ++p_;
    while (p_ < e_ && *p_ != '"') {
      char c = *p_++;
      if ((unsigned char)c < 0x20) return false;
      if (c == '\\') {
        if (p_ >= e_) return false;
        const char x = *p_++;
        switch (x) {
          case '"': case '\\': case '/': out += x; break;
          case 'b': out += '\b'; break;
          case 'f': out += '\f'; break;
          case 'n': out += '\n'; break;
          case 'r': out += '\r'; break;
          case 't': out += '\t'; break;
          case 'u': {  // kept as UTF-8 for the basic plane (names are ASCII in practice)
            if (e_ - p_ < 4) return false;
            unsigned v = 0;
            for (int k = 0; k < 4; ++k) {
              const char h = *p_++;
              v <<= 4;
              if (h >= '0' && h <= '9') v |= h - '0';
              else if (h >= 'a' && h <= 'f') v |= h - 'a' + 10;
              else if (h >= 'A' && h <= 'F') v |= h - 'A' + 10;
              else return false;
            }
            if (v < 0x80) out += (char)v;
            else if (v < 0x800) { out += (char)(0xC0 | (v >> 6)); out += (char)(0x80 | (v & 0x3F)); }
            else { out += (char)(0xE0 | (v >> 12)); out += (char)(0x80 | ((v >> 6) & 0x3F)); out += (char)(0x80 | (v & 0x3F)); }
            break;
          }
          default: return false;
        }
      } else {
        out += c;
      }
    }
    if (p_ >= e_) return false;
    ++p_;
    return true;
  }
  bool number(Json& out) {
    const char* q = p_;
    if (q < e_ && *q == '-') ++q;
    const char* digits = q;
    while (q < e_ && *q >= '0' && *q <= '9') ++q;
    if (q == digits) return false;
    bool integer = true;
    while (q < e_ && (*q == '.' || *q == 'e' || *q == 'E' || *q == '+' || *q == '-' || (*q >= '0' && *q <= '9'))) {
      integer = false;
      ++q;
    }
    std::string text(p_, q);
    p_ = q;
    if (integer) {
      errno = 0;
      char* end = nullptr;
      const long long v = strtoll(text.c_str(), &end, 10);
      if (errno || *end) return false;
      out.type = Json::kInt;
      out.i = v;
    } else {
      char* end = nullptr;
      out.d = strtod(text.c_str(), &end);
      if (*end) return false;
      out.type = Json::kNum;
    }
    return true;
  }
  bool value(Json& out, int depth) {
    if (depth > 16) {
      err_ = "JSON nested too deeply";
      return false;
    }
    ws();
    if (p_ >= e_) return false;
    const char c = *p_;
    if (c == '{') {
      ++p_;
      out.type = Json::kObj;
      ws();
      if (p_ < e_ && *p_ == '}') {
        ++p_;
        return true;
      }
      for (;;) {
        ws();
        std::string key;
        if (!str(key)) return false;
        ws();
        if (p_ >= e_ || *p_ != ':') return false;
        ++p_;
        Json v;
        if (!value(v, depth + 1)) return false;
        out.obj.emplace_back(std::move(key), std::move(v));
        ws();
        if (p_ < e_ && *p_ == ',') {
          ++p_;
          continue;
        }
        if (p_ < e_ && *p_ == '}') {
          ++p_;
          return true;
        }
        return false;
      }
    }
    if (c == '[') {
      ++p_;
      out.type = Json::kArr;
      ws();
      if (p_ < e_ && *p_ == ']') {
        ++p_;
        return true;
      }
      for (;;) {
        Json v;
        if (!value(v, depth + 1)) return false;
        out.arr.push_back(std::move(v));
        ws();
        if (p_ < e_ && *p_ == ',') {
          ++p_;
          continue;
        }
        if (p_ < e_ && *p_ == ']') {
          ++p_;
          return true;
        }
        return false;
      }
    }
    if (c == '"') {
      out.type = Json::kStr;
      return str(out.s);
    }
    if (lit("true")) {
      out.type = Json::kBool;
      out.b = true;
      return true;
    }
    if (lit("false")) {
      out.type = Json::kBool;
      return true;
    }
    if (lit("null")) return true;
    return number(out);
  }
};

// ------------------------------------------------------------------ checkpoint
struct TensorInfo {
  int file;
  std::string dtype;
  std::vector<int64_t> shape;
  int64_t begin, end;  // absolute byte offsets in the file
};

struct Need {
  std::string name;
  int32_t layer, kind;
  std::vector<int64_t> shape;
};

int64_t dtype_size(const std::string& d) {
  if (d == "BF16" || d == "F16" || d == "I16" || d == "U16") return 2;
  if (d == "F32" || d == "I32" || d == "U32") return 4;
  if (d == "F64" || d == "I64" || d == "U64") return 8;
  if (d == "U8" || d == "I8" || d == "BOOL" || d == "F8_E4M3" || d == "F8_E5M2") return 1;
  return -1;
}

}  // namespace

struct kf_shard {
  struct File {
    std::string path;
    int fd = -1;
    int64_t size = 0;
  };
  std::vector<File> files;
  std::map<std::string, TensorInfo> index;
  std::map<std::string, std::vector<uint16_t>> held;
  std::vector<kf_tensor> out;
  int64_t bytes_read = 0;
};

namespace {

void close_files(kf_shard* s) {
  for (auto& f : s->files)
    if (f.fd >= 0) close(f.fd);
}

kf_status open_one(kf_shard* s, const char* path) {
  kf_shard::File f;
  f.path = path;
  f.fd = open(path, O_RDONLY | O_CLOEXEC);
  if (f.fd < 0) return fail(KF_EINVAL, "%s: cannot open (%s)", path, strerror(errno));
  struct stat st;
  if (fstat(f.fd, &st) != 0) {
    close(f.fd);
    return fail(KF_EINVAL, "%s: cannot stat", path);
  }
  f.size = st.st_size;
  const int idx = (int)s->files.size();
  s->files.push_back(f);
  unsigned char lenb[8];
  if (f.size < 8 || pread(f.fd, lenb, 8, 0) != 8) return fail(KF_EINVAL, "%s: shorter than a safetensors header", path);
  uint64_t n = 0;
  for (int k = 7; k >= 0; --k) n = (n << 8) | lenb[k];  // little-endian
  if (n < 2 || n > (100u << 20) || (int64_t)n > f.size - 8)
    return fail(KF_EINVAL, "%s: header length %llu does not fit the file", path, (unsigned long long)n);
  std::vector<char> hdr(n);
  if (pread(f.fd, hdr.data(), n, 8) != (ssize_t)n) return fail(KF_EINVAL, "%s: cannot read the header", path);
  Json root;
  std::string err;
  Parser parser(hdr.data(), hdr.data() + n);
  if (!parser.parse(root, err) || root.type != Json::kObj) return fail(KF_EINVAL, "%s: header: %s", path, err.c_str());
  const int64_t data0 = 8 + (int64_t)n;
  for (const auto& kv : root.obj) {
    if (kv.first == "__metadata__") continue;
    const Json& t = kv.second;
    const Json* dt = t.get("dtype");
    const Json* sh = t.get("shape");
    const Json* off = t.get("data_offsets");
    if (t.type != Json::kObj || !dt || dt->type != Json::kStr || !sh || sh->type != Json::kArr || !off ||
        off->type != Json::kArr || off->arr.size() != 2 || off->arr[0].type != Json::kInt || off->arr[1].type != Json::kInt)
      return fail(KF_EINVAL, "%s: tensor '%s' lacks dtype, shape or data_offsets", path, kv.first.c_str());
    TensorInfo ti;
    ti.file = idx;
    ti.dtype = dt->s;
    int64_t numel = 1;
    for (const Json& d : sh->arr) {
      if (d.type != Json::kInt || d.i < 0 || (d.i > 0 && numel > ((int64_t)1 << 50) / d.i))
        return fail(KF_EINVAL, "%s: tensor '%s' has an invalid shape", path, kv.first.c_str());
      ti.shape.push_back(d.i);
      numel *= d.i;
    }
    const int64_t b = off->arr[0].i, e = off->arr[1].i, es = dtype_size(ti.dtype);
    if (b < 0 || e < b || data0 + e > f.size)
      return fail(KF_EINVAL, "%s: tensor '%s' byte range [%lld, %lld) outside the file", path, kv.first.c_str(),
                  (long long)b, (long long)e);
    if (es > 0 && e - b != numel * es)
      return fail(KF_EINVAL, "%s: tensor '%s' spans %lld bytes, its %s shape needs %lld", path, kv.first.c_str(),
                  (long long)(e - b), ti.dtype.c_str(), (long long)(numel * es));
    ti.begin = data0 + b;
    ti.end = data0 + e;
    if (s->index.count(kv.first)) return fail(KF_EINVAL, "%s: tensor '%s' appears twice in the checkpoint", path, kv.first.c_str());
    s->index.emplace(kv.first, std::move(ti));
  }
  return KF_OK;
}

std::string layer_name(int l, const char* rest) { return "model.layers." + std::to_string(l) + "." + rest; }

// The tensors of layers [lo, hi) (and the head), in kf_stage_init's terms.
kf_status stage_needs(const kf_model_config* c, int lo, int hi, int has_head, int flags, std::vector<Need>& needs) {
  if (!c) return fail(KF_EINVAL, "config is NULL");
  if (!(0 <= lo && lo < hi && hi <= c->n_layers))
    return fail(KF_EINVAL, "layer range [%d, %d) not inside [0, %d)", lo, hi, c->n_layers);
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 || c->ffn <= 0)
    return fail(KF_EINVAL, "config sizes must be positive");
  if (has_head && c->vocab <= 0) return fail(KF_EINVAL, "a head stage needs vocab > 0");
  if (flags & ~KF_SHARD_TIED_EMBEDDINGS) return fail(KF_EINVAL, "unknown flag bits 0x%x", flags);
  const int64_t H = c->hidden, hd = c->head_dim, F = c->ffn, V = c->vocab;
  const int64_t q = c->n_q_heads * hd, kv = c->n_kv_heads * hd;
  for (int l = lo; l < hi; ++l) {
    needs.push_back({layer_name(l, "input_layernorm.weight"), l, KF_W_ATTN_NORM, {H}});
    needs.push_back({layer_name(l, "self_attn.q_proj.weight"), l, KF_W_Q, {q, H}});
    needs.push_back({layer_name(l, "self_attn.k_proj.weight"), l, KF_W_K, {kv, H}});
    needs.push_back({layer_name(l, "self_attn.v_proj.weight"), l, KF_W_V, {kv, H}});
    needs.push_back({layer_name(l, "self_attn.o_proj.weight"), l, KF_W_O, {H, q}});
    needs.push_back({layer_name(l, "post_attention_layernorm.weight"), l, KF_W_MLP_NORM, {H}});
    needs.push_back({layer_name(l, "mlp.gate_proj.weight"), l, KF_W_GATE, {F, H}});
    needs.push_back({layer_name(l, "mlp.up_proj.weight"), l, KF_W_UP, {F, H}});
    needs.push_back({layer_name(l, "mlp.down_proj.weight"), l, KF_W_DOWN, {H, F}});
    if (c->qk_norm) {
      needs.push_back({layer_name(l, "self_attn.q_norm.weight"), l, KF_W_Q_NORM, {hd}});
      needs.push_back({layer_name(l, "self_attn.k_norm.weight"), l, KF_W_K_NORM, {hd}});
    }
  }
  if (has_head) {
    needs.push_back({"model.embed_tokens.weight", -1, KF_W_EMBED, {V, H}});
    needs.push_back({"model.norm.weight", -1, KF_W_FINAL_NORM, {H}});
    needs.push_back({(flags & KF_SHARD_TIED_EMBEDDINGS) ? "model.embed_tokens.weight" : "lm_head.weight", -1,
                     KF_W_LM_HEAD, {V, H}});
  }
  return KF_OK;
}

kf_status check_needs(const kf_shard* s, const std::vector<Need>& needs) {
  for (const Need& n : needs) {
    auto it = s->index.find(n.name);
    if (it == s->index.end()) return fail(KF_EINVAL, "tensor '%s' is not in the checkpoint", n.name.c_str());
    const TensorInfo& t = it->second;
    if (t.dtype != "BF16")
      return fail(KF_EUNSUPPORTED, "tensor '%s' is stored as %s (BF16 only)", n.name.c_str(), t.dtype.c_str());
    if (t.shape != n.shape) {
      std::string got, want;
      for (int64_t d : t.shape) got += std::to_string(d) + ",";
      for (int64_t d : n.shape) want += std::to_string(d) + ",";
      return fail(KF_EINVAL, "tensor '%s' has shape [%s], the config needs [%s]", n.name.c_str(), got.c_str(), want.c_str());
    }
  }
  return KF_OK;
}

kf_status plan(kf_shard* s, const kf_model_config* cfg, int lo, int hi, int has_head, int flags,
               std::vector<Need>& needs, int64_t* stage_bytes, int64_t* fetch_bytes) {
  kf_status st = stage_needs(cfg, lo, hi, has_head, flags, needs);
  if (st != KF_OK) return st;
  st = check_needs(s, needs);
  if (st != KF_OK) return st;
  int64_t total = 0, fetch = 0;
  std::map<std::string, int> seen;  // a tied LM head shares the embedding's bytes
  for (const Need& n : needs) {
    if (seen[n.name]++) continue;
    const TensorInfo& t = s->index.at(n.name);
    total += t.end - t.begin;
    if (!s->held.count(n.name)) fetch += t.end - t.begin;
  }
  *stage_bytes = total;
  *fetch_bytes = fetch;
  return KF_OK;
}

bool read_range(const kf_shard::File& f, int64_t at, int64_t n, char* dst) {
  while (n > 0) {
    const ssize_t r = pread(f.fd, dst, (size_t)(n < ((int64_t)1 << 30) ? n : ((int64_t)1 << 30)), (off_t)at);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    dst += r;
    at += r;
    n -= r;
  }
  return true;
}

}  // namespace

extern "C" {

kf_status kf_shard_open(const char* const* paths, int32_t n_paths, kf_shard** out) {
  if (!out) return fail(KF_EINVAL, "out is NULL");
  *out = nullptr;
  if (!paths || n_paths < 1) return fail(KF_EINVAL, "no files given");
  kf_shard* s = new (std::nothrow) kf_shard();
  if (!s) return fail(KF_ENOMEM, "host allocation");
  for (int i = 0; i < n_paths; ++i) {
    if (!paths[i]) {
      close_files(s);
      delete s;
      return fail(KF_EINVAL, "path %d is NULL", i);
    }
    const kf_status st = open_one(s, paths[i]);
    if (st != KF_OK) {
      close_files(s);
      delete s;
      return st;
    }
  }
  *out = s;
  return KF_OK;
}

kf_status kf_shard_close(kf_shard* s) {
  if (!s) return fail(KF_EINVAL, "checkpoint is NULL");
  close_files(s);
  delete s;
  return KF_OK;
}

kf_status kf_shard_plan(kf_shard* s, const kf_model_config* cfg, int32_t lo, int32_t hi, int32_t has_head,
                        int32_t flags, int64_t* stage_bytes, int64_t* fetch_bytes, int32_t* n_tensors) {
  if (!s) return fail(KF_EINVAL, "checkpoint is NULL");
  std::vector<Need> needs;
  int64_t total = 0, fetch = 0;
  const kf_status st = plan(s, cfg, lo, hi, has_head, flags, needs, &total, &fetch);
  if (st != KF_OK) return st;
  if (stage_bytes) *stage_bytes = total;
  if (fetch_bytes) *fetch_bytes = fetch;
  if (n_tensors) *n_tensors = (int32_t)needs.size();
  return KF_OK;
}

kf_status kf_shard_fetch(kf_shard* s, const kf_model_config* cfg, int32_t lo, int32_t hi, int32_t has_head,
                         int32_t flags, kf_weights* weights) {
  if (!s) return fail(KF_EINVAL, "checkpoint is NULL");
  if (!weights) return fail(KF_EINVAL, "weights is NULL");
  std::vector<Need> needs;
  int64_t total = 0, fetch = 0;
  kf_status st = plan(s, cfg, lo, hi, has_head, flags, needs, &total, &fetch);
  if (st != KF_OK) return st;
  std::vector<std::string> added;
  for (const Need& n : needs) {
    if (s->held.count(n.name)) continue;
    const TensorInfo& t = s->index.at(n.name);
    std::vector<uint16_t> buf;
    try {
      buf.resize((size_t)((t.end - t.begin) / 2));
    } catch (const std::bad_alloc&) {
      for (const std::string& a : added) s->held.erase(a);
      return fail(KF_ENOMEM, "host allocation of %lld bytes for '%s'", (long long)(t.end - t.begin), n.name.c_str());
    }
    if (!read_range(s->files[t.file], t.begin, t.end - t.begin, reinterpret_cast<char*>(buf.data()))) {
      for (const std::string& a : added) s->held.erase(a);
      return fail(KF_EINVAL, "%s: cannot read tensor '%s'", s->files[t.file].path.c_str(), n.name.c_str());
    }
    s->bytes_read += t.end - t.begin;
    s->held.emplace(n.name, std::move(buf));
    added.push_back(n.name);
  }
  s->out.clear();
  for (const Need& n : needs) {
    const std::vector<uint16_t>& buf = s->held.at(n.name);
    s->out.push_back(kf_tensor{n.layer, n.kind, buf.data(), (int64_t)buf.size()});
  }
  weights->tensors = s->out.data();
  weights->count = (int32_t)s->out.size();
  return KF_OK;
}

kf_status kf_shard_stage_init(kf_shard* s, const kf_model_config* cfg, int32_t lo, int32_t hi, int32_t has_head,
                              int32_t flags, void* hip_stream, kf_stage** out) {
  if (!out) return fail(KF_EINVAL, "out is NULL");
  *out = nullptr;
  kf_weights w{};
  const kf_status st = kf_shard_fetch(s, cfg, lo, hi, has_head, flags, &w);
  if (st != KF_OK) return st;
  return kf_stage_init(cfg, lo, hi, has_head, &w, hip_stream, out);
}

kf_status kf_shard_release(kf_shard* s, int32_t lo, int32_t hi, int32_t has_head) {
  if (!s) return fail(KF_EINVAL, "checkpoint is NULL");
  if (lo < 0 || hi < lo) return fail(KF_EINVAL, "layer range [%d, %d)", lo, hi);
  for (auto it = s->held.begin(); it != s->held.end();) {
    const std::string& n = it->first;
    bool keep;
    if (n.compare(0, 13, "model.layers.") == 0) {
      const int l = atoi(n.c_str() + 13);
      keep = l >= lo && l < hi;
    } else {
      keep = has_head != 0;
    }
    it = keep ? std::next(it) : s->held.erase(it);
  }
  s->out.clear();
  return KF_OK;
}

kf_status kf_shard_stats(const kf_shard* s, int64_t* bytes_read, int64_t* bytes_held) {
  if (!s) return fail(KF_EINVAL, "checkpoint is NULL");
  if (bytes_read) *bytes_read = s->bytes_read;
  if (bytes_held) {
    int64_t h = 0;
    for (const auto& kv : s->held) h += (int64_t)kv.second.size() * 2;
    *bytes_held = h;
  }
  return KF_OK;
}

}  // extern "C"

// Stage runtime behind the C ABI of include/kafila_stage.h: argument checks,
// device memory (weights, KV cache, workspaces) and the per-step kernel sequence.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "error.h"
#include "kafila_planner.h"
#include "kafila_stage.h"
#include "kernels.h"
#include "prefill.h"

using namespace kf;

// Launch shapes (compile-time; the defaults are the measured best on MI355X).
// Decode GEMVs take 8 output rows per workgroup by default (the rules below pick
// 4 or 10 for the residual launches where the grid then fills whole rounds of the CUs) and one
// 16-byte chunk per row in flight per thread (two were slower at every batch).
constexpr int kGemvRows = 8, kGemvChunks = 1;
constexpr int kQkvRowsBatch1 = 4;  // the batch-1 QKV launch (after the first layer) takes 4-row workgroups
// The LM head on the rows a decode kept (fp16, batch 2-4) takes 12-row
// workgroups: each reads its input rows once for all its weight rows, so these
// move two thirds of the 8-row launch's input bytes per weight byte (8B-shaped
// head stage at batch 4: 153.5 -> 152.2 us, V = 128256 = 12 x 10688).  The
// caller's fp32 or bf16 rows keep 8-row workgroups.
constexpr int kHeadRowsKept = 12;

// Rows per workgroup of a residual GEMV with n output rows: 8, unless that
// leaves the grid a fraction of a round over the compute units and 4 rows do
// not (H = 5120: 640 workgroups of 8 rows are 2.5 per CU, 1280 of 4 exactly 5;
// the 32B-shaped down projection at batch 1 went from 48.0 to 45.2 us).
static int resid_rows(int n, int n_cu) {
  if ((n / 8) % n_cu != 0 && n % 4 == 0 && (n / 4) % n_cu == 0) return 4;
  return 8;
}
// Rows per workgroup of the down projection (K = ffn, the longest rows): 10 when
// that grid is a whole number of rounds over the compute units, else the
// residual rule.  Each workgroup reads its input rows once for all its weight
// rows, so more rows per workgroup move fewer input bytes through the vector
// caches (at batch 4 a 4-row workgroup reads as many input bytes as weight
// bytes).  H = 5120: 512 workgroups of 10 rows, 2 per CU; the 32B-shaped down
// projection went from 45.4 to 44.4 us at batch 1 and 51.5 to 46.5 us at batch 4.
// 16 rows at H = 8192 were slower (70B-shaped batch 1: 69.7 -> 70.8 us), and so
// were 10 rows for the output projection (K = heads x hd, 16.5 -> 17.0 us).
static int down_rows(int n, int n_cu) {
  if (n % 10 == 0 && (n / 10) % n_cu == 0) return 10;
  return resid_rows(n, n_cu);
}
#ifndef KF_ATTN_TARGET_WGS
#define KF_ATTN_TARGET_WGS 256
#endif
#ifndef KF_ATTN_ALIGN
#define KF_ATTN_ALIGN 64
#endif

#define KF_HIP(call, what)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return fail(KF_EDEVICE, "%s: %s", (what), hipGetErrorString(e_)); \
  } while (0)

static int64_t align256(int64_t n) { return (n + 255) & ~(int64_t)255; }

// Prefill workspace of kf_stage_prefill_noalloc: a file-scope device array, one
// copy per device, held from the library's first use on a device until the
// process ends.  In host code the name `scratch` is a stand-in symbol, not a
// device address: the address comes from hipGetSymbolAddress, taken once per
// device (with that device current) when a stage is created there, and only that
// address is passed to kernels.  Every no-allocation prefill on a device shares
// the array, so such calls must not overlap on one device.
constexpr int64_t kPrefillScratchBytes = 144LL << 20;  // a 512-token chunk of the 70B shape needs 132 MiB
static __device__ __align__(256) char scratch[kPrefillScratchBytes];
static_assert(kPrefillScratchBytes == KF_PREFILL_SCRATCH_BYTES, "the header states the scratch size");
constexpr int kMaxDevices = 64;

static char* scratch_address(int device, hipError_t* err) {
  static std::mutex mu;
  static char* addr[kMaxDevices] = {};
  std::lock_guard<std::mutex> lock(mu);
  *err = hipSuccess;
  if (device < 0 || device >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  if (!addr[device]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    addr[device] = static_cast<char*>(p);
  }
  return addr[device];
}

struct LayerW {
  uint16_t *wqkv, *wo, *wg, *wu, *wd, *g_attn, *g_mlp;
  uint16_t *g_qn = nullptr, *g_kn = nullptr;  // per-head q / k norm gains (qk_norm blocks)
  // Whether g_attn (g_mlp) is folded into W_qkv's (W_gate's and W_up's) columns;
  // the products then take the normalised rows without the gain.
  bool qkv_fold = false, mlp_fold = false;
  const uint16_t* qkv_gain() const { return qkv_fold ? nullptr : g_attn; }
  const uint16_t* mlp_gain() const { return mlp_fold ? nullptr : g_mlp; }
};

struct kf_stage {
  kf_model_config cfg;
  int lo, hi, has_head;
  hipStream_t stream;
  int device;
  int n_cu = 256;  // compute units of the device (workgroup balance of the residual GEMVs)
  char* arena = nullptr;  // all weights
  std::vector<LayerW> layers;
  uint16_t *embed = nullptr, *lm_head = nullptr, *g_final = nullptr;
  bool head_fold = false;  // g_final folded into the LM head's columns
  // decode workspace
  char* ws = nullptr;
  float *x = nullptr, *q = nullptr, *act = nullptr;
  // batch > 1: merged attention output and the residual after the output projection, in fp16
  uint16_t *o16 = nullptr, *x16 = nullptr;
  float* o32 = nullptr;   // batch 1 with KF_STAGE_ORDERED: the merged attention output, fp32
  int flags = 0;          // KF_STAGE_* behaviour flags
  float* kraw = nullptr;  // [B][nkv][hd] new keys before their norm and RoPE (qk_norm blocks)
  float* part_val = nullptr;
  int* part_idx = nullptr;
  int lm_wg = 0;       // capacity of the argmax partials per batch row
  int lm_wg_used = 0;  // partials per row written by the last LM-head launch
  int kept_rows = 0;   // rows the last decode kept for the head (called without hidden output), else 0
  int* err_flag = nullptr;
  int live_kv = 0;
  PrefillWorkspace pf;
  char* scratch = nullptr;  // this device's copy of the static prefill scratch (device address)
  // instrumentation: event pairs around launches while profiling is enabled
  int prof_mask = 0;
  std::vector<hipEvent_t> ev;   // 2 per recorded launch
  std::vector<int> ev_cls;
  size_t ev_used = 0;           // recorded launches
  Tracer tracer() { return prof_mask ? Tracer{this, &kf_stage::mark} : Tracer{}; }
  static void mark(void* ctx, int cls, int begin);
};

void kf_stage::mark(void* ctx, int cls, int begin) {
  kf_stage* s = (kf_stage*)ctx;
  if (!(s->prof_mask & (1 << cls))) return;
  if (begin) {
    if (s->ev.size() < 2 * (s->ev_used + 1)) {
      // Timing-only events: no system-scope fence (cache writeback and invalidate)
      // on record, which would otherwise slow the work that follows.
      hipEvent_t a, b;
      if (hipEventCreateWithFlags(&a, hipEventDisableSystemFence) != hipSuccess) return;
      if (hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess) {
        hipEventDestroy(a);
        return;
      }
      s->ev.push_back(a);
      s->ev.push_back(b);
      s->ev_cls.push_back(cls);
    }
    s->ev_cls[s->ev_used] = cls;
    hipEventRecord(s->ev[2 * s->ev_used], s->stream);
  } else {
    if (s->ev.size() < 2 * (s->ev_used + 1)) return;  // begin failed to get events
    hipEventRecord(s->ev[2 * s->ev_used + 1], s->stream);
    s->ev_used++;
  }
}

struct kf_kv {
  kf_stage* st;
  int max_users, max_ctx, max_split;
  // Pages of kKvPage positions, [layer][page][kv_head][kKvPage][hd] fp16 for K and V.
  // A reserved cache holds ppu pages per user in user order (no table); a paged
  // cache lends pages from a pool, recorded in a device table with a host mirror.
  int ppu = 0, n_pages = 0;
  int* table = nullptr;        // device [max_users][ppu] page ids (paged caches only)
  std::vector<int> host_table; // mirror of the table (-1: not held)
  std::vector<int> held;       // pages each user holds
  std::vector<int> free_pages; // the pool's free pages (paged caches only), next page last
  uint16_t *k = nullptr, *v = nullptr;
  float *rcos = nullptr, *rsin = nullptr;
  float *part_acc = nullptr, *part_ml = nullptr;
  int64_t page_stride, layer_stride;  // elements
  std::vector<int> len;
  KvPages pages() const { return KvPages{table, ppu, page_stride}; }
};

static int pages_for(int64_t len) { return (int)((len + kKvPage - 1) / kKvPage); }

// Lend each of the (distinct) `users` the pages it needs to hold `upto[i]`
// positions, or change nothing and fail when the pool is short.  New table
// entries are written on the stage's stream before any later work there reads them.
static kf_status kv_grant(kf_kv* kv, int n, const int* users, const int64_t* upto) {
  if (!kv->table) return KF_OK;  // reserved cache: every page is held from the start
  int64_t want = 0;
  for (int i = 0; i < n; ++i) {
    const int need = pages_for(upto[i]) - kv->held[users[i]];
    if (need > 0) want += need;
  }
  if (want > (int64_t)kv->free_pages.size())
    return fail(KF_ENOMEM, "KV pool: %lld more pages needed, %zu free of %d", (long long)want, kv->free_pages.size(),
                kv->n_pages);
  KvTableUpdate up{};
  for (int i = 0; i < n; ++i) {
    const int u = users[i];
    for (int pg = kv->held[u]; pg < pages_for(upto[i]); ++pg) {
      const int id = kv->free_pages.back();
      kv->free_pages.pop_back();
      kv->host_table[(size_t)u * kv->ppu + pg] = id;
      up.idx[up.n] = u * kv->ppu + pg;
      up.val[up.n] = id;
      if (++up.n == kKvTableBatch) {
        KF_HIP(launch_kv_table_update(kv->table, up, kv->st->stream), "page table update");
        up.n = 0;
      }
    }
    if (pages_for(upto[i]) > kv->held[u]) kv->held[u] = pages_for(upto[i]);
  }
  if (up.n) KF_HIP(launch_kv_table_update(kv->table, up, kv->st->stream), "page table update");
  return KF_OK;
}

// Return a user's pages past the first `keep` to the pool (paged caches).
static void kv_release(kf_kv* kv, int u, int keep) {
  if (!kv->table) return;
  for (int pg = kv->held[u] - 1; pg >= keep; --pg) {
    int& id = kv->host_table[(size_t)u * kv->ppu + pg];
    kv->free_pages.push_back(id);
    id = -1;
  }
  if (kv->held[u] > keep) kv->held[u] = keep;
}

// ------------------------------------------------------------------ config checks
static kf_status check_cfg(const kf_model_config* c, int lo, int hi) {
  if (!c) return fail(KF_EINVAL, "config is NULL");
  if (c->n_layers <= 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn <= 0 || c->vocab < 0)
    return fail(KF_EINVAL, "config sizes must be positive");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(KF_EINVAL, "rms_eps must be >= 0 and rope_theta > 0");
  if (!(0 <= lo && lo < hi && hi <= c->n_layers))
    return fail(KF_EINVAL, "layer range [%d, %d) not inside [0, %d)", lo, hi, c->n_layers);
  if (c->head_dim != 64 && c->head_dim != 128) return fail(KF_EUNSUPPORTED, "head_dim %d (64 or 128 only)", c->head_dim);
  if (c->n_q_heads % c->n_kv_heads) return fail(KF_EINVAL, "n_q_heads must be a multiple of n_kv_heads");
  if (c->n_q_heads / c->n_kv_heads > kMaxGroup)
    return fail(KF_EUNSUPPORTED, "more than %d query heads per KV head", kMaxGroup);
  if (c->hidden % 64 || c->ffn % 64) return fail(KF_EUNSUPPORTED, "hidden and ffn must be multiples of 64");
  if (c->qk_norm != 0 && c->qk_norm != 1) return fail(KF_EINVAL, "qk_norm must be 0 or 1");
  return KF_OK;
}

static int64_t tensor_numel(const kf_model_config& c, int kind) {
  const int64_t H = c.hidden, hd = c.head_dim, F = c.ffn, V = c.vocab;
  switch (kind) {
    case KF_W_ATTN_NORM: case KF_W_MLP_NORM: case KF_W_FINAL_NORM: return H;
    case KF_W_Q: return c.n_q_heads * hd * H;
    case KF_W_K: case KF_W_V: return c.n_kv_heads * hd * H;
    case KF_W_O: return H * c.n_q_heads * hd;
    case KF_W_GATE: case KF_W_UP: case KF_W_DOWN: return F * H;
    case KF_W_EMBED: case KF_W_LM_HEAD: return V * H;
    case KF_W_Q_NORM: case KF_W_K_NORM: return c.qk_norm ? hd : -1;
    default: return -1;
  }
}

// Layer tensors: kinds 0..8, then the q / k norm gains of qk_norm blocks.
constexpr int kLayerSlots = 11;
static int layer_slot(int kind) { return kind <= KF_W_DOWN ? kind : kind - KF_W_Q_NORM + KF_W_DOWN + 1; }
static bool is_layer_kind(int kind) { return (kind >= KF_W_ATTN_NORM && kind <= KF_W_DOWN) || kind == KF_W_Q_NORM || kind == KF_W_K_NORM; }

static int64_t block_bytes(const kf_model_config& c) {
  int64_t n = 0;
  for (int k = KF_W_ATTN_NORM; k <= KF_W_DOWN; ++k) n += tensor_numel(c, k);
  if (c.qk_norm) n += tensor_numel(c, KF_W_Q_NORM) + tensor_numel(c, KF_W_K_NORM);
  return 2 * n;
}

static int64_t head_bytes(const kf_model_config& c) {
  return 2 * (tensor_numel(c, KF_W_EMBED) + tensor_numel(c, KF_W_LM_HEAD) + tensor_numel(c, KF_W_FINAL_NORM));
}

static int max_split_for(int max_ctx) {
  int ms = (max_ctx + kAttnMinSplit - 1) / kAttnMinSplit;
  return ms > 1024 ? 1024 : ms;
}

static int64_t kv_bytes(const kf_model_config& c, int layers, int max_users, int max_ctx) {
  const int64_t cache = 2LL * layers * max_users * c.n_kv_heads * (int64_t)pages_for(max_ctx) * kKvPage * c.head_dim * 2;
  const int64_t rope = 2LL * max_ctx * (c.head_dim / 2) * 4;
  const int64_t ms = max_split_for(max_ctx);
  const int64_t part = (int64_t)kMaxBatch * c.n_q_heads * ms * (c.head_dim + 2) * 4;
  return align256(cache / 2) * 2 + align256(rope / 2) * 2 + align256(part) + 256;
}

static int64_t decode_ws_bytes(const kf_model_config& c, int has_head) {
  const int64_t H = c.hidden, B = kMaxBatch;
  int64_t n = 0;
  n += align256(B * H * 4);                           // x
  n += align256(B * c.n_q_heads * c.head_dim * 4);    // q
  n += align256(B * (int64_t)c.ffn * 4);              // act
  n += align256(B * c.n_q_heads * c.head_dim * 2);    // o16
  n += align256((int64_t)c.n_q_heads * c.head_dim * 4); // o32 (batch 1)
  n += align256(B * H * 2);                           // x16
  if (c.qk_norm) n += align256(B * (int64_t)c.n_kv_heads * c.head_dim * 4);  // kraw
  if (has_head) {
    const int64_t wgs = (c.vocab + 3) / 4;  // enough for any rows-per-workgroup choice
    n += 2 * align256(B * wgs * 4);
  }
  n += 256;  // error flag
  return n;
}

extern "C" {

int32_t kf_abi_version(void) { return KF_ABI_VERSION; }

kf_status kf_stage_bytes(const kf_model_config* cfg, int32_t lo, int32_t hi, int32_t has_head, int32_t max_users,
                         int32_t max_ctx, int64_t* beta_block, int64_t* beta_head, int64_t* resident) {
  kf_status st = check_cfg(cfg, lo, hi);
  if (st != KF_OK && st != KF_EUNSUPPORTED) return st;
  if (max_users < 0 || max_ctx < 0) return fail(KF_EINVAL, "max_users and max_ctx must be >= 0");
  const int64_t bb = block_bytes(*cfg), hb = has_head ? head_bytes(*cfg) : 0;
  if (beta_block) *beta_block = bb;
  if (beta_head) *beta_head = hb;
  if (resident)
    *resident = (int64_t)(hi - lo) * bb + hb + decode_ws_bytes(*cfg, has_head) +
                (max_users > 0 && max_ctx > 0 ? kv_bytes(*cfg, hi - lo, max_users, max_ctx) : 0);
  return KF_OK;
}

kf_status kf_stage_costs(const kf_model_config* cfg, int32_t max_users, int32_t max_ctx, kf_model_costs* out) {
  kf_status st = check_cfg(cfg, 0, 1);
  if (st != KF_OK && st != KF_EUNSUPPORTED) return st;
  if (!out) return fail(KF_EINVAL, "out is NULL");
  if (max_users < 0 || max_ctx < 0) return fail(KF_EINVAL, "max_users and max_ctx must be >= 0");
  const kf_model_config& c = *cfg;
  const bool kv = max_users > 0 && max_ctx > 0;
  const int64_t bb = block_bytes(c), hb = head_bytes(c);
  // kf_stage_bytes' resident for one and two blocks, without and with the head: the
  // per-block share is the difference (weights + that layer's KV), the rest is per stage.
  const int64_t r1 = bb + decode_ws_bytes(c, 0) + (kv ? kv_bytes(c, 1, max_users, max_ctx) : 0);
  const int64_t r2 = 2 * bb + decode_ws_bytes(c, 0) + (kv ? kv_bytes(c, 2, max_users, max_ctx) : 0);
  const int64_t r1h = r1 + hb + decode_ws_bytes(c, 1) - decode_ws_bytes(c, 0);
  out->beta_block = bb;
  out->beta_head = hb;
  out->block_resident = r2 - r1;
  out->stage_resident = r1 - (r2 - r1);
  out->head_resident = r1h - r1;
  out->flops_block = 2.0 * (double)(bb / 2);  // two flops per bf16 weight at batch 1
  return KF_OK;
}

kf_status kf_stage_init(const kf_model_config* cfg, int32_t lo, int32_t hi, int32_t has_head,
                        const kf_weights* weights, void* hip_stream, kf_stage** out) {
  if (!out) return fail(KF_EINVAL, "out is NULL");
  *out = nullptr;
  kf_status st = check_cfg(cfg, lo, hi);
  if (st != KF_OK) return st;
  if (has_head && cfg->vocab <= 0) return fail(KF_EINVAL, "a head stage needs vocab > 0");
  if (!weights || (weights->count > 0 && !weights->tensors)) return fail(KF_EINVAL, "weights is NULL");

  const int nl = hi - lo;
  // Locate every tensor exactly once.
  std::vector<const kf_tensor*> slot((size_t)nl * kLayerSlots, nullptr);
  const kf_tensor* hslot[3] = {nullptr, nullptr, nullptr};
  for (int i = 0; i < weights->count; ++i) {
    const kf_tensor& t = weights->tensors[i];
    if (t.kind < KF_W_ATTN_NORM || t.kind > KF_W_K_NORM) return fail(KF_EINVAL, "tensor %d: unknown kind %d", i, t.kind);
    if (!t.bf16) return fail(KF_EINVAL, "tensor %d: NULL data", i);
    if ((t.kind == KF_W_Q_NORM || t.kind == KF_W_K_NORM) && !cfg->qk_norm)
      return fail(KF_EINVAL, "tensor %d: q/k norm gain given for a config without qk_norm", i);
    if (t.numel != tensor_numel(*cfg, t.kind))
      return fail(KF_EINVAL, "tensor %d (layer %d kind %d): numel %lld, expected %lld", i, t.layer, t.kind,
                  (long long)t.numel, (long long)tensor_numel(*cfg, t.kind));
    const kf_tensor** dst;
    if (!is_layer_kind(t.kind)) {
      if (!has_head) return fail(KF_EINVAL, "tensor %d: head tensor given to a stage without the head", i);
      if (t.layer != -1) return fail(KF_EINVAL, "tensor %d: head tensors take layer -1", i);
      dst = &hslot[t.kind - KF_W_EMBED];
    } else {
      if (t.layer < lo || t.layer >= hi) return fail(KF_EINVAL, "tensor %d: layer %d outside [%d, %d)", i, t.layer, lo, hi);
      dst = &slot[(size_t)(t.layer - lo) * kLayerSlots + layer_slot(t.kind)];
    }
    if (*dst) return fail(KF_EINVAL, "tensor %d (layer %d kind %d) given twice", i, t.layer, t.kind);
    *dst = &t;
  }
  const int need = cfg->qk_norm ? kLayerSlots : KF_W_DOWN + 1;
  for (int l = 0; l < nl; ++l)
    for (int k = 0; k < need; ++k)
      if (!slot[(size_t)l * kLayerSlots + k])
        return fail(KF_EINVAL, "missing tensor: layer %d kind %d", lo + l, k <= KF_W_DOWN ? k : k - KF_W_DOWN - 1 + KF_W_Q_NORM);
  if (has_head)
    for (int k = 0; k < 3; ++k)
      if (!hslot[k]) return fail(KF_EINVAL, "missing head tensor kind %d", KF_W_EMBED + k);

  kf_stage* s = new (std::nothrow) kf_stage();
  if (!s) return fail(KF_ENOMEM, "host allocation");
  s->cfg = *cfg;
  s->lo = lo;
  s->hi = hi;
  s->has_head = has_head ? 1 : 0;
  s->stream = (hipStream_t)hip_stream;
  if (hipGetDevice(&s->device) != hipSuccess) {
    delete s;
    return fail(KF_EDEVICE, "no HIP device");
  }
  {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, s->device) == hipSuccess && n > 0) s->n_cu = n;
  }
  {
    hipError_t e;
    s->scratch = scratch_address(s->device, &e);
    if (!s->scratch) {
      delete s;
      return fail(KF_EDEVICE, "device address of the prefill scratch: %s", hipGetErrorString(e));
    }
  }

  const kf_model_config& c = *cfg;
  const int64_t H = c.hidden, hd = c.head_dim, F = c.ffn;
  const int64_t nqkv = (int64_t)(c.n_q_heads + 2 * c.n_kv_heads) * hd;
  // Per-layer arena: wqkv | wo | wg | wu | wd | g_attn | g_mlp, each 256-byte aligned.
  const int64_t off_qkv = 0, off_o = align256(off_qkv + nqkv * H * 2), off_g = align256(off_o + H * c.n_q_heads * hd * 2),
                off_u = align256(off_g + F * H * 2), off_d = align256(off_u + F * H * 2),
                off_na = align256(off_d + H * F * 2), off_nm = align256(off_na + H * 2),
                off_qn = align256(off_nm + H * 2), off_kn = align256(off_qn + (c.qk_norm ? hd * 2 : 0)),
                lsz = align256(off_kn + (c.qk_norm ? hd * 2 : 0));
  const int64_t V = c.vocab;
  const int64_t off_e = lsz * nl, off_lm = align256(off_e + (has_head ? V * H * 2 : 0)),
                off_gf = align256(off_lm + (has_head ? V * H * 2 : 0)), total = align256(off_gf + H * 2);

  auto cleanup = [&](kf_status code) {
    if (s->arena) hipFree(s->arena);
    if (s->ws) hipFree(s->ws);
    delete s;
    return code;
  };
  if (hipMalloc((void**)&s->arena, total) != hipSuccess) {
    hipGetLastError();
    s->arena = nullptr;
    return cleanup(fail(KF_ENOMEM, "device allocation of %lld weight bytes", (long long)total));
  }
  auto up = [&](char* dst, const kf_tensor* t) {
    return hipMemcpy(dst, t->bf16, (size_t)t->numel * 2, hipMemcpyHostToDevice);
  };
  s->layers.resize(nl);
  for (int l = 0; l < nl; ++l) {
    char* base = s->arena + lsz * l;
    const kf_tensor** w = &slot[(size_t)l * kLayerSlots];
    LayerW& L = s->layers[l];
    L.wqkv = (uint16_t*)(base + off_qkv);
    L.wo = (uint16_t*)(base + off_o);
    L.wg = (uint16_t*)(base + off_g);
    L.wu = (uint16_t*)(base + off_u);
    L.wd = (uint16_t*)(base + off_d);
    L.g_attn = (uint16_t*)(base + off_na);
    L.g_mlp = (uint16_t*)(base + off_nm);
    const int64_t qb = (int64_t)c.n_q_heads * hd * H * 2, kb = (int64_t)c.n_kv_heads * hd * H * 2;
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = up(base + off_qkv, w[KF_W_Q]);
    if (e == hipSuccess) e = up(base + off_qkv + qb, w[KF_W_K]);
    if (e == hipSuccess) e = up(base + off_qkv + qb + kb, w[KF_W_V]);
    if (e == hipSuccess) e = up(base + off_o, w[KF_W_O]);
    if (e == hipSuccess) e = up(base + off_g, w[KF_W_GATE]);
    if (e == hipSuccess) e = up(base + off_u, w[KF_W_UP]);
    if (e == hipSuccess) e = up(base + off_d, w[KF_W_DOWN]);
    if (e == hipSuccess) e = up(base + off_na, w[KF_W_ATTN_NORM]);
    if (e == hipSuccess) e = up(base + off_nm, w[KF_W_MLP_NORM]);
    if (c.qk_norm) {
      L.g_qn = (uint16_t*)(base + off_qn);
      L.g_kn = (uint16_t*)(base + off_kn);
      if (e == hipSuccess) e = up(base + off_qn, w[layer_slot(KF_W_Q_NORM)]);
      if (e == hipSuccess) e = up(base + off_kn, w[layer_slot(KF_W_K_NORM)]);
    }
    if (e != hipSuccess) return cleanup(fail(KF_EDEVICE, "weight upload: %s", hipGetErrorString(e)));
  }
  if (has_head) {
    s->embed = (uint16_t*)(s->arena + off_e);
    s->lm_head = (uint16_t*)(s->arena + off_lm);
    s->g_final = (uint16_t*)(s->arena + off_gf);
    hipError_t e = up((char*)s->embed, hslot[0]);
    if (e == hipSuccess) e = up((char*)s->g_final, hslot[1]);
    if (e == hipSuccess) e = up((char*)s->lm_head, hslot[2]);
    if (e != hipSuccess) return cleanup(fail(KF_EDEVICE, "head upload: %s", hipGetErrorString(e)));
  }

  const int64_t wsz = decode_ws_bytes(c, s->has_head);
  if (hipMalloc((void**)&s->ws, wsz) != hipSuccess) {
    hipGetLastError();
    s->ws = nullptr;
    return cleanup(fail(KF_ENOMEM, "device allocation of the decode workspace"));
  }
  if (hipMemset(s->ws, 0, wsz) != hipSuccess) return cleanup(fail(KF_EDEVICE, "workspace clear"));
  char* p = s->ws;
  auto take = [&](int64_t bytes) {
    char* r = p;
    p += align256(bytes);
    return r;
  };
  const int64_t B = kMaxBatch;
  s->x = (float*)take(B * H * 4);
  s->q = (float*)take(B * c.n_q_heads * hd * 4);
  s->act = (float*)take(B * F * 4);
  s->o16 = (uint16_t*)take(B * c.n_q_heads * hd * 2);
  s->o32 = (float*)take((int64_t)c.n_q_heads * hd * 4);
  s->x16 = (uint16_t*)take(B * H * 2);
  if (c.qk_norm) s->kraw = (float*)take(B * c.n_kv_heads * hd * 4);
  if (has_head) {
    s->lm_wg = (int)((V + kGemvRows - 1) / kGemvRows);  // the 8-row grid, the larger of the LM head's two
    s->part_val = (float*)take(B * s->lm_wg * 4);
    s->part_idx = (int*)take(B * s->lm_wg * 4);
  }
  s->err_flag = (int*)take(4);

  // The matrices are kept in fp16, the type every product here takes (the
  // matrix cores and the decode GEMVs): converted once, in place.  Gains and the
  // embedding table stay bf16.  The RMSNorm gain in front of a matrix (g_attn
  // before W_qkv, g_mlp before W_gate and W_up, g_final before the LM head) is
  // folded into its columns, W diag(g) rounded once to fp16, wherever every
  // product has a finite fp16 rounding; the products then take x / rms(x) as
  // it is, so the decode GEMVs load no gain and multiply nothing in (32B-shaped
  // batch 4 1377 -> 1401 tokens/s, batch 1 393 -> 396; 8B head 7291 -> 7496, 8B
  // batch 1 1571 -> 1582).  Otherwise that gain stays out of the matrix and is
  // applied to the normalised rows.
  {
    hipError_t e = hipDeviceSynchronize();  // the uploads and the workspace clear ran on the null stream
    const int64_t mats[5] = {nqkv * H, H * (int64_t)c.n_q_heads * hd, F * H, F * H, H * F};
    // one flag per gain: layer l's g_attn at 2 l, its g_mlp at 2 l + 1, g_final at 2 nl
    int* flags = nullptr;
    if (e == hipSuccess) e = hipMalloc((void**)&flags, (2 * nl + 1) * sizeof(int));
    if (e == hipSuccess) e = hipMemsetAsync(flags, 0, (2 * nl + 1) * sizeof(int), s->stream);
    for (int l = 0; l < nl && e == hipSuccess; ++l) {
      const LayerW& L = s->layers[l];
      e = launch_gain_fold_check(L.wqkv, mats[0], H, L.g_attn, flags + 2 * l, s->stream);
      if (e == hipSuccess) e = launch_gain_fold_check(L.wg, mats[2], H, L.g_mlp, flags + 2 * l + 1, s->stream);
      if (e == hipSuccess) e = launch_gain_fold_check(L.wu, mats[3], H, L.g_mlp, flags + 2 * l + 1, s->stream);
    }
    if (e == hipSuccess && has_head) e = launch_gain_fold_check(s->lm_head, V * H, H, s->g_final, flags + 2 * nl, s->stream);
    std::vector<int> over(2 * nl + 1, 0);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e == hipSuccess) e = hipMemcpy(over.data(), flags, over.size() * sizeof(int), hipMemcpyDeviceToHost);
    if (flags) hipFree(flags);
    for (int l = 0; l < nl && e == hipSuccess; ++l) {
      LayerW& L = s->layers[l];
      L.qkv_fold = !over[2 * l];
      L.mlp_fold = !over[2 * l + 1];
      uint16_t* ptrs[5] = {L.wqkv, L.wo, L.wg, L.wu, L.wd};
      const uint16_t* gains[5] = {L.qkv_fold ? L.g_attn : nullptr, nullptr, L.mlp_fold ? L.g_mlp : nullptr,
                                  L.mlp_fold ? L.g_mlp : nullptr, nullptr};
      for (int m = 0; m < 5 && e == hipSuccess; ++m)
        e = gains[m] ? launch_weights_to_f16_gain(ptrs[m], mats[m], H, gains[m], s->err_flag, s->stream)
                     : launch_weights_to_f16(ptrs[m], mats[m], s->err_flag, s->stream);
    }
    if (e == hipSuccess && has_head) {
      s->head_fold = !over[2 * nl];
      e = s->head_fold ? launch_weights_to_f16_gain(s->lm_head, V * H, H, s->g_final, s->err_flag, s->stream)
                       : launch_weights_to_f16(s->lm_head, V * H, s->err_flag, s->stream);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    int bad = 0;
    if (e == hipSuccess) e = hipMemcpy(&bad, s->err_flag, 4, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return cleanup(fail(KF_EDEVICE, "weight conversion: %s", hipGetErrorString(e)));
    if (bad) return cleanup(fail(KF_EINVAL, "a weight matrix holds a value beyond the fp16 range (|w| >= 65520)"));
  }
  *out = s;
  clear_error();
  return KF_OK;
}

kf_status kf_stage_destroy(kf_stage* s) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (s->live_kv) return fail(KF_ESTATE, "%d KV cache(s) of this stage still exist", s->live_kv);
  hipStreamSynchronize(s->stream);
  if (s->arena) hipFree(s->arena);
  if (s->ws) hipFree(s->ws);
  prefill_free(s->pf);
  for (hipEvent_t e : s->ev) hipEventDestroy(e);
  delete s;
  return KF_OK;
}

kf_status kf_stage_set_stream(kf_stage* s, void* hip_stream) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  s->stream = (hipStream_t)hip_stream;
  return KF_OK;
}

kf_status kf_stage_describe(const kf_stage* s, kf_model_config* cfg, int32_t* lo, int32_t* hi, int32_t* has_head,
                            void** hip_stream, int32_t* device) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (cfg) *cfg = s->cfg;
  if (lo) *lo = s->lo;
  if (hi) *hi = s->hi;
  if (has_head) *has_head = s->has_head;
  if (hip_stream) *hip_stream = (void*)s->stream;
  if (device) *device = s->device;
  return KF_OK;
}

kf_status kf_stage_sync(kf_stage* s) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  KF_HIP(hipStreamSynchronize(s->stream), "stream synchronize");
  KF_HIP(hipGetLastError(), "earlier enqueued work");
  int flag = 0;
  KF_HIP(hipMemcpy(&flag, s->err_flag, 4, hipMemcpyDeviceToHost), "error flag read");
  if (flag) {
    int zero = 0;
    KF_HIP(hipMemcpy(s->err_flag, &zero, 4, hipMemcpyHostToDevice), "error flag clear");
    std::string msg;
    if (flag & kErrToken) msg += "a token id was outside [0, vocab) (its hidden row was set to NaN); ";
    if (flag & kErrF16Range)
      msg += "an activation, key or value held in fp16 reached 65520 in magnitude (stored as infinity); ";
    if (flag & kErrNaNLogit) msg += "a logit was NaN (skipped by the argmax; a row of NaN logits gave token -1); ";
    msg.resize(msg.size() - 2);
    return fail((flag & kErrToken) ? KF_EINVAL : KF_ERANGE, "%s", msg.c_str());
  }
  return KF_OK;
}

kf_status kf_stage_set_flags(kf_stage* s, int32_t flags) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (flags & ~KF_STAGE_ORDERED) return fail(KF_EINVAL, "unknown flag bits 0x%x", flags & ~KF_STAGE_ORDERED);
  s->flags = flags;
  return KF_OK;
}

kf_status kf_stage_get_flags(const kf_stage* s, int32_t* flags) {
  if (!s || !flags) return fail(KF_EINVAL, "NULL argument");
  *flags = s->flags;
  return KF_OK;
}

// ------------------------------------------------------------------ KV cache
// n_pages == 0: a reserved cache (every user's pages in user order); else a pool of n_pages.
static kf_status kv_create(kf_stage* s, int32_t max_users, int32_t max_ctx, int32_t n_pages, kf_kv** out) {
  if (!out) return fail(KF_EINVAL, "out is NULL");
  *out = nullptr;
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (max_users <= 0 || max_ctx <= 0) return fail(KF_EINVAL, "max_users and max_ctx must be positive");
  if ((int64_t)max_ctx > (int64_t)kAttnMaxSplit * 1024) return fail(KF_ERANGE, "max_ctx above %d", kAttnMaxSplit * 1024);
  const kf_model_config& c = s->cfg;
  const int nl = s->hi - s->lo;
  const int ppu = pages_for(max_ctx);
  if ((int64_t)max_users * ppu > (1LL << 30)) return fail(KF_ERANGE, "max_users x max_ctx too large");
  const bool paged = n_pages > 0;
  kf_kv* kv = new (std::nothrow) kf_kv();
  if (!kv) return fail(KF_ENOMEM, "host allocation");
  kv->st = s;
  kv->max_users = max_users;
  kv->max_ctx = max_ctx;
  kv->max_split = max_split_for(max_ctx);
  kv->ppu = ppu;
  kv->n_pages = paged ? n_pages : max_users * ppu;
  kv->page_stride = (int64_t)c.n_kv_heads * kKvPage * c.head_dim;
  kv->layer_stride = kv->page_stride * kv->n_pages;
  kv->len.assign(max_users, 0);
  kv->held.assign(max_users, paged ? 0 : ppu);
  if (paged) {
    kv->host_table.assign((size_t)max_users * ppu, -1);
    kv->free_pages.reserve(n_pages);
    for (int i = n_pages - 1; i >= 0; --i) kv->free_pages.push_back(i);  // page 0 lent first
  }
  const int64_t cache = kv->layer_stride * nl * 2;
  const int64_t half = c.head_dim / 2;
  const int64_t rope = (int64_t)max_ctx * half * 4;
  const int64_t pacc = (int64_t)kMaxBatch * c.n_q_heads * kv->max_split * c.head_dim * 4;
  const int64_t pml = (int64_t)kMaxBatch * c.n_q_heads * kv->max_split * 2 * 4;
  const int64_t tab = paged ? (int64_t)max_users * ppu * 4 : 0;
  char* mem[7] = {nullptr};
  const int64_t sz[7] = {cache, cache, rope, rope, pacc, pml, tab};
  for (int i = 0; i < 7; ++i) {
    if (sz[i] == 0) continue;
    if (hipMalloc((void**)&mem[i], sz[i]) != hipSuccess) {
      hipGetLastError();
      for (int j = 0; j < i; ++j)
        if (mem[j]) hipFree(mem[j]);
      delete kv;
      return fail(KF_ENOMEM, "device allocation of %lld KV bytes", (long long)sz[i]);
    }
  }
  kv->k = (uint16_t*)mem[0];
  kv->v = (uint16_t*)mem[1];
  kv->rcos = (float*)mem[2];
  kv->rsin = (float*)mem[3];
  kv->part_acc = (float*)mem[4];
  kv->part_ml = (float*)mem[5];
  kv->table = (int*)mem[6];
  // RoPE table from float64 angles: pos * theta^(-2i/hd).
  std::vector<float> tc((size_t)max_ctx * half), ts((size_t)max_ctx * half);
  for (int64_t i = 0; i < half; ++i) {
    const double w = std::pow((double)c.rope_theta, -2.0 * (double)i / (double)c.head_dim);
    for (int64_t p = 0; p < max_ctx; ++p) {
      const double a = (double)p * w;
      tc[p * half + i] = (float)std::cos(a);
      ts[p * half + i] = (float)std::sin(a);
    }
  }
  hipError_t e = hipMemset(kv->k, 0, cache);
  if (e == hipSuccess) e = hipMemset(kv->v, 0, cache);
  if (e == hipSuccess && kv->table) e = hipMemset(kv->table, 0, tab);
  if (e == hipSuccess) e = hipMemcpy(kv->rcos, tc.data(), rope, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(kv->rsin, ts.data(), rope, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    for (int j = 0; j < 7; ++j)
      if (mem[j]) hipFree(mem[j]);
    delete kv;
    return fail(KF_EDEVICE, "KV init: %s", hipGetErrorString(e));
  }
  s->live_kv++;
  *out = kv;
  return KF_OK;
}

kf_status kf_kv_create(kf_stage* s, int32_t max_users, int32_t max_ctx, kf_kv** out) {
  return kv_create(s, max_users, max_ctx, 0, out);
}

kf_status kf_kv_create_paged(kf_stage* s, int32_t max_users, int32_t max_ctx, int32_t n_pages, kf_kv** out) {
  if (n_pages < 1) {
    if (out) *out = nullptr;
    return fail(KF_EINVAL, "n_pages %d < 1", n_pages);
  }
  return kv_create(s, max_users, max_ctx, n_pages, out);
}

kf_status kf_kv_pages(const kf_kv* kv, int32_t* total, int32_t* free_pages) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  if (total) *total = kv->n_pages;
  if (free_pages) *free_pages = kv->table ? (int32_t)kv->free_pages.size() : -1;
  return KF_OK;
}

kf_status kf_kv_destroy(kf_kv* kv) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  hipStreamSynchronize(kv->st->stream);
  void* mem[7] = {kv->k, kv->v, kv->rcos, kv->rsin, kv->part_acc, kv->part_ml, kv->table};
  for (void* m : mem)
    if (m) hipFree(m);
  kv->st->live_kv--;
  delete kv;
  return KF_OK;
}

kf_status kf_kv_describe(const kf_kv* kv, kf_stage** stage, int32_t* max_users, int32_t* max_ctx) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  if (stage) *stage = kv->st;
  if (max_users) *max_users = kv->max_users;
  if (max_ctx) *max_ctx = kv->max_ctx;
  return KF_OK;
}

kf_status kf_kv_len(const kf_kv* kv, int32_t user, int32_t* len) {
  if (!kv || !len) return fail(KF_EINVAL, "NULL argument");
  if (user < 0 || user >= kv->max_users) return fail(KF_EINVAL, "user %d outside [0, %d)", user, kv->max_users);
  *len = kv->len[user];
  return KF_OK;
}

kf_status kf_kv_set_len(kf_kv* kv, int32_t user, int32_t len) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  if (user < 0 || user >= kv->max_users) return fail(KF_EINVAL, "user %d outside [0, %d)", user, kv->max_users);
  if (len < 0 || len > kv->max_ctx) return fail(KF_ERANGE, "length %d outside [0, %d]", len, kv->max_ctx);
  const int64_t upto = len;
  kf_status st = kv_grant(kv, 1, &user, &upto);
  if (st != KF_OK) return st;
  kv_release(kv, user, pages_for(len));
  kv->len[user] = len;
  return KF_OK;
}

static kf_status kv_slice_check(const kf_kv* kv, int layer, int user, int pos0, int n) {
  const kf_stage* s = kv->st;
  if (layer < s->lo || layer >= s->hi) return fail(KF_EINVAL, "layer %d not held by the stage [%d, %d)", layer, s->lo, s->hi);
  if (user < 0 || user >= kv->max_users) return fail(KF_EINVAL, "user %d outside [0, %d)", user, kv->max_users);
  if (pos0 < 0 || n < 0) return fail(KF_EINVAL, "negative position or count");
  if ((int64_t)pos0 + n > kv->max_ctx) return fail(KF_ERANGE, "positions [%d, %d) beyond max_ctx %d", pos0, pos0 + n, kv->max_ctx);
  return KF_OK;
}

kf_status kf_kv_write(kf_kv* kv, int32_t layer, int32_t user, int32_t pos0, int32_t n, const void* k_dev,
                      const void* v_dev, kf_dtype dtype) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  kf_status st = kv_slice_check(kv, layer, user, pos0, n);
  if (st != KF_OK) return st;
  if (n == 0) return KF_OK;
  if (!k_dev || !v_dev) return fail(KF_EINVAL, "NULL source");
  if (dtype != KF_F32 && dtype != KF_BF16 && dtype != KF_F16) return fail(KF_EINVAL, "dtype");
  const kf_model_config& c = kv->st->cfg;
  const int64_t upto = (int64_t)pos0 + n;
  st = kv_grant(kv, 1, &user, &upto);
  if (st != KF_OK) return st;
  const int64_t off = (layer - kv->st->lo) * kv->layer_stride;
  KF_HIP(launch_kv_write(kv->k + off, kv->v + off, kv->pages(), user, pos0, k_dev, v_dev, (int)dtype, n,
                         c.n_kv_heads, c.head_dim, kv->st->stream),
         "kv_write launch");
  return KF_OK;
}

kf_status kf_kv_read(const kf_kv* kv, int32_t layer, int32_t user, int32_t pos0, int32_t n, float* k_dev,
                     float* v_dev) {
  if (!kv) return fail(KF_EINVAL, "kv is NULL");
  kf_status st = kv_slice_check(kv, layer, user, pos0, n);
  if (st != KF_OK) return st;
  if (n == 0) return KF_OK;
  if (!k_dev || !v_dev) return fail(KF_EINVAL, "NULL destination");
  const kf_model_config& c = kv->st->cfg;
  if ((int64_t)pos0 + n > (int64_t)kv->held[user] * kKvPage)
    return fail(KF_ERANGE, "positions up to %d of user %d are not in the cache (it holds %d pages)", pos0 + n, user,
                kv->held[user]);
  const int64_t off = (layer - kv->st->lo) * kv->layer_stride;
  KF_HIP(launch_kv_read(kv->k + off, kv->v + off, kv->pages(), user, pos0, k_dev, v_dev, n, c.n_kv_heads, c.head_dim,
                        kv->st->stream),
         "kv_read launch");
  return KF_OK;
}

// ------------------------------------------------------------------ decode
// Keys per split-KV workgroup at batch 1: about KF_ATTN_TARGET_WGS workgroups
// over the row's keys, whole pages, at most KF_ATTN_KEYS_PER_WG keys (long
// contexts spread over more workgroups).  Fewer, longer splits than one
// workgroup per CU, since every extra partial costs the merge in the output
// projection (8B-shaped: 17 splits of 128 keys for 2049 keys).  The split
// never exceeds the partial-buffer capacity per row.
#ifndef KF_ATTN_KEYS_PER_WG
#define KF_ATTN_KEYS_PER_WG 512
#endif
static_assert(KF_ATTN_ALIGN % kKvPage == 0, "batch-1 splits start on page boundaries");
static void attn_split(int nkv, int64_t total_len, int max_len, int max_split, int* split, int* n_split) {
  auto up = [](int64_t v) { return (int)((v + KF_ATTN_ALIGN - 1) / KF_ATTN_ALIGN * KF_ATTN_ALIGN); };
  const int64_t target = KF_ATTN_TARGET_WGS;
  int sp = up((total_len * nkv + target - 1) / target);
  if (sp > KF_ATTN_KEYS_PER_WG) sp = KF_ATTN_KEYS_PER_WG;
  const int need = up((max_len + max_split - 1) / max_split);
  if (sp < need) sp = need;
  if (sp < kAttnMinSplit) sp = kAttnMinSplit;
  if (sp > kAttnMaxSplit) sp = kAttnMaxSplit;
  *split = sp;
  *n_split = (max_len + sp - 1) / sp;
}

// Keys per split for the matrix-core attention kernel from batch 2: one
// workgroup per CU over the keys of the whole batch (16-key granularity), but
// at least one block per wave and at most KF_ATTN_MFMA_MAX_KEYS (five blocks
// per wave), past which more workgroups in more rounds beat longer chains of
// blocks.  Against the batch-1 rule (about twice the workgroups, page-aligned):
// the 8B-shaped head stage's ragged rows (256 to 4096 keys) 11.1 -> 9.5 us,
// four 8B-shaped rows of up to 32K keys 53.5 -> 48.7 us, 32B-shaped batch 4
// unchanged (320-key splits either way).  At batch 1 the rule of attn_split
// measured best.
#ifndef KF_ATTN_MFMA_MAX_KEYS
#define KF_ATTN_MFMA_MAX_KEYS 320
#endif
#ifndef KF_ATTN_MFMA_WG_PER_CU
#define KF_ATTN_MFMA_WG_PER_CU 1
#endif
static void attn_split_mfma(int nkv, int64_t total_len, int max_len, int max_split, int n_cu, int* split,
                            int* n_split) {
  auto up = [](int64_t v) { return (int)((v + kAttnMfmaAlign - 1) / kAttnMfmaAlign * kAttnMfmaAlign); };
  const int64_t wgs = (int64_t)KF_ATTN_MFMA_WG_PER_CU * n_cu;
  int sp = up((total_len * nkv + wgs - 1) / wgs);
  if (sp < 16 * kAttnMfmaWaves) sp = 16 * kAttnMfmaWaves;
  if (sp > KF_ATTN_MFMA_MAX_KEYS) sp = KF_ATTN_MFMA_MAX_KEYS;
  const int need = up((max_len + max_split - 1) / max_split);
  if (sp < need) sp = need;
  if (sp > kAttnMaxSplit) sp = kAttnMaxSplit;
  *split = sp;
  *n_split = (max_len + sp - 1) / sp;
}

kf_status kf_stage_decode(kf_stage* s, kf_kv* kv, int32_t batch, const int32_t* users, const int32_t* positions,
                          const int32_t* tokens_dev, const void* hidden_in_dev, void* hidden_out_dev, kf_dtype io) {
  if (!s || !kv) return fail(KF_EINVAL, "stage or kv is NULL");
  if (kv->st != s) return fail(KF_EINVAL, "kv belongs to another stage");
  if (batch < 1 || batch > kMaxBatch) return fail(KF_EINVAL, "batch %d outside [1, %d]", batch, kMaxBatch);
  if (!users || !positions) return fail(KF_EINVAL, "users / positions is NULL");
  if ((tokens_dev == nullptr) == (hidden_in_dev == nullptr))
    return fail(KF_EINVAL, "exactly one of tokens / hidden input must be given");
  if (tokens_dev && !s->has_head) return fail(KF_ESTATE, "token input needs the head");
  if (!hidden_out_dev && !s->has_head)
    return fail(KF_EINVAL, "hidden output is NULL (only a stage that holds the head may keep its rows)");
  if (io != KF_F32 && io != KF_BF16) return fail(KF_EINVAL, "io dtype");
  int max_len = 0;
  int64_t total_len = 0;
  for (int b = 0; b < batch; ++b) {
    const int u = users[b], p = positions[b];
    if (u < 0 || u >= kv->max_users) return fail(KF_EINVAL, "users[%d] = %d outside [0, %d)", b, u, kv->max_users);
    for (int j = 0; j < b; ++j)
      if (users[j] == u) return fail(KF_EINVAL, "user %d appears twice in the batch", u);
    if (p != kv->len[u]) return fail(KF_EINVAL, "positions[%d] = %d but user %d holds %d positions", b, p, u, kv->len[u]);
    if (p >= kv->max_ctx) return fail(KF_ERANGE, "position %d beyond max_ctx %d", p, kv->max_ctx);
    if (p + 1 > max_len) max_len = p + 1;
    total_len += p + 1;
  }
  const kf_model_config& c = s->cfg;
  const int H = c.hidden, hd = c.head_dim;
  hipStream_t st = s->stream;

  int split, n_split;
  if (batch > 1) attn_split_mfma(c.n_kv_heads, total_len, max_len, kv->max_split, s->n_cu, &split, &n_split);
  else attn_split(c.n_kv_heads, total_len, max_len, kv->max_split, &split, &n_split);
  if (split % kAttnMfmaAlign) return fail(KF_EINVAL, "split of %d keys breaks the attention kernel's alignment", split);
  int64_t upto[kMaxBatch];
  for (int b = 0; b < batch; ++b) upto[b] = (int64_t)positions[b] + 1;
  const kf_status gst = kv_grant(kv, batch, users, upto);
  if (gst != KF_OK) return gst;
  s->kept_rows = 0;  // the residual rows change from here on; set again when the step completes

  const Tracer tr = s->tracer();

  for (int l = s->lo; l < s->hi; ++l) {
    const LayerW& L = s->layers[l - s->lo];
    const int64_t loff = (l - s->lo) * kv->layer_stride;

    GemvParams g{};
    g.batch = batch;
    g.eps = c.rms_eps;
    // attention RMSNorm + QKV + RoPE + KV append
    g.w0 = L.wqkv;
    g.gain = L.qkv_gain();
    // from batch 2 the previous layer's down projection left the residual in fp16 too
    g.in = batch > 1 ? reinterpret_cast<const float*>(s->x16) : s->x;
    g.in16 = batch > 1;
    g.K = H;
    g.N = (c.n_q_heads + 2 * c.n_kv_heads) * hd;
    g.q = s->q;
    g.kc = kv->k + loff;
    g.vc = kv->v + loff;
    g.kv = kv->pages();
    g.nq = c.n_q_heads;
    g.nkv = c.n_kv_heads;
    g.hd = hd;
    g.rope_cos = kv->rcos;
    g.rope_sin = kv->rsin;
    g.kraw = s->kraw;  // set for qk_norm blocks: q and k are normalised and rotated below
    g.err_flag = s->err_flag;
    for (int b = 0; b < kMaxBatch; ++b) {
      g.users[b] = b < batch ? users[b] : 0;
      g.pos[b] = b < batch ? positions[b] : 0;
    }
    hipError_t le;
    tr.begin(KF_K_QKV);
    if (l == s->lo) {  // the first layer reads the stage input and starts the residual stream from it
      g.src = hidden_in_dev;
      g.src_bf16 = io == KF_BF16;
      g.tokens = tokens_dev;
      g.embed = s->embed;
      g.vocab = c.vocab;
      g.x_init = s->x;
      g.in16 = 0;  // the input rows come from src / tokens
      le = launch_gemv_src(kEpiQKV, kGemvRows, kGemvChunks, true, g, st);
    } else {
      le = launch_gemv(kEpiQKV, batch == 1 ? kQkvRowsBatch1 : kGemvRows, kGemvChunks, true, g, st);
    }
    tr.end(KF_K_QKV);
    KF_HIP(le, "qkv launch");

    AttnParams a{};
    a.q = s->q;
    a.kc = kv->k + loff;
    a.vc = kv->v + loff;
    a.part_acc = kv->part_acc;
    a.part_ml = kv->part_ml;
    a.kv = kv->pages();
    if (c.qk_norm) {  // q / k left raw by the QKV launch: the attention normalises and rotates them
      a.kraw = s->kraw;
      a.gq = L.g_qn;
      a.gk = L.g_kn;
      a.rope_cos = kv->rcos;
      a.rope_sin = kv->rsin;
      a.eps = c.rms_eps;
    }
    a.nq = c.n_q_heads;
    a.nkv = c.n_kv_heads;
    a.hd = hd;
    a.split = split;
    a.n_split = n_split;
    a.max_split = kv->max_split;
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
    a.err_flag = s->err_flag;
    for (int b = 0; b < kMaxBatch; ++b) {
      a.users[b] = b < batch ? users[b] : 0;
      a.len[b] = b < batch ? positions[b] + 1 : 0;
    }
    {
      tr.begin(KF_K_ATTN);
      const hipError_t le = launch_attn_decode(a, batch, st);
      tr.end(KF_K_ATTN);
      KF_HIP(le, "attention launch");
    }

    if (batch == 1 && !(s->flags & KF_STAGE_ORDERED)) {
      // the merge fused into a head-split output projection (one launch; the
      // heads' contributions reach the residual in arrival order)
      tr.begin(KF_K_OPROJ);
      const hipError_t le = launch_oproj_heads(a, L.wo, s->x, H, batch, st);
      tr.end(KF_K_OPROJ);
      KF_HIP(le, "o-proj launch");
    } else {
      // The merge on its own, then a row-owning GEMV: each residual row is
      // updated by one workgroup in a fixed order.  From batch 2 the GEMV also
      // leaves the updated residual in fp16 for the gate/up launch (the input
      // rows in fp32 would crowd the vector cache the weights stream through);
      // at batch 1 the merged output and the residual stay fp32.
      tr.begin(KF_K_OPROJ);
      hipError_t le = batch > 1 ? launch_attn_merge(a, s->o16, nullptr, batch, st)
                                : launch_attn_merge(a, nullptr, s->o32, batch, st);
      if (le == hipSuccess) {
        GemvParams op{};
        op.batch = batch;
        op.w0 = L.wo;
        op.in = batch > 1 ? reinterpret_cast<const float*>(s->o16) : s->o32;
        op.in16 = batch > 1;
        op.K = c.n_q_heads * hd;
        op.N = H;
        op.x = s->x;
        if (batch > 1) {
          op.out2 = s->x16;
          op.out2_type = kOut2F16;
        }
        op.err_flag = s->err_flag;
        le = launch_gemv(kEpiResid, resid_rows(H, s->n_cu), kGemvChunks, false, op, st);
      }
      tr.end(KF_K_OPROJ);
      KF_HIP(le, "o-proj launch");
    }

    GemvParams gu{};
    gu.batch = batch;
    gu.eps = c.rms_eps;
    gu.w0 = L.wg;
    gu.w1 = L.wu;
    gu.gain = L.mlp_gain();
    gu.in = batch > 1 ? reinterpret_cast<const float*>(s->x16) : s->x;
    gu.in16 = batch > 1;
    gu.K = H;
    gu.N = c.ffn;
    gu.act = s->act;
    // From batch 2 the SwiGLU output goes to the down projection as fp16 (the
    // prefill's down GEMM takes the same operand in fp16): the input rows of
    // batch 2-4 then fit the vector cache beside the weights stream.
    gu.act16 = batch > 1;
    gu.err_flag = s->err_flag;
    {
      tr.begin(KF_K_GATEUP);
      const hipError_t le = launch_gemv(kEpiSwiGLU, kGemvRows, kGemvChunks, true, gu, st);
      tr.end(KF_K_GATEUP);
      KF_HIP(le, "gate/up launch");
    }

    GemvParams d{};
    d.batch = batch;
    d.w0 = L.wd;
    d.in = s->act;
    d.in16 = batch > 1;
    d.K = c.ffn;
    d.N = H;
    d.x = s->x;
    d.err_flag = s->err_flag;
    if (l == s->hi - 1 && hidden_out_dev) {
      d.out2 = hidden_out_dev;
      d.out2_type = io == KF_BF16 ? kOut2BF16 : kOut2F32;
    } else if (batch > 1) {  // also the kept rows the head reads (no hidden output)
      d.out2 = s->x16;  // the next layer's QKV input
      d.out2_type = kOut2F16;
    }
    {
      tr.begin(KF_K_DOWN);
      const hipError_t le = launch_gemv(kEpiResid, down_rows(H, s->n_cu), kGemvChunks, false, d, st);
      tr.end(KF_K_DOWN);
      KF_HIP(le, "down launch");
    }
  }
  for (int b = 0; b < batch; ++b) kv->len[users[b]] += 1;
  s->kept_rows = hidden_out_dev ? 0 : batch;
  return KF_OK;
}

// ------------------------------------------------------------------ head
static kf_status head_common(kf_stage* s, int rows, const void* hidden, kf_dtype dtype) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (!s->has_head) return fail(KF_ESTATE, "the stage does not hold the head");
  if (rows < 1) return fail(KF_EINVAL, "rows must be >= 1");
  if (!hidden) {  // the rows the stage's last decode kept
    if (s->kept_rows != rows)
      return fail(KF_ESTATE, "hidden is NULL but the stage's last decode kept %d rows, not %d", s->kept_rows, rows);
    return KF_OK;
  }
  if (dtype != KF_F32 && dtype != KF_BF16) return fail(KF_EINVAL, "dtype");
  return KF_OK;
}

static kf_status head_launch(kf_stage* s, int rows, const void* hidden, kf_dtype dtype, float* logits) {
  const kf_model_config& c = s->cfg;
  const Tracer tr = s->tracer();
  GemvParams g{};
  g.batch = rows;
  g.eps = c.rms_eps;
  g.w0 = s->lm_head;
  g.gain = s->head_fold ? nullptr : s->g_final;
  g.src = hidden;  // the LM head reads the caller's rows directly
  g.src_bf16 = dtype == KF_BF16;
  if (!hidden) {  // the kept rows: the residual itself at batch 1, its fp16 copy at batch 2-4
    g.in = rows > 1 ? reinterpret_cast<const float*>(s->x16) : s->x;
    g.in16 = rows > 1;
  }
  g.K = c.hidden;
  g.N = c.vocab;
  g.logits = logits;
  g.part_val = s->part_val;
  g.part_idx = s->part_idx;
  g.err_flag = s->err_flag;
  const int rows_per_wg = !hidden && rows > 1 ? kHeadRowsKept : kGemvRows;
  g.n_wg = gemv_grid(kEpiLMHead, rows_per_wg, g);
  if (g.n_wg > s->lm_wg) return fail(KF_EINVAL, "LM-head grid of %d workgroups above the partials' %d", g.n_wg, s->lm_wg);
  s->lm_wg_used = g.n_wg;
  tr.begin(KF_K_LMHEAD);
  const hipError_t e = hidden ? launch_gemv_src(kEpiLMHead, kGemvRows, kGemvChunks, true, g, s->stream)
                              : launch_gemv(kEpiLMHead, rows_per_wg, kGemvChunks, true, g, s->stream);
  tr.end(KF_K_LMHEAD);
  KF_HIP(e, "lm-head launch");
  return KF_OK;
}

kf_status kf_head_logits(kf_stage* s, int32_t rows, const void* hidden, kf_dtype dtype, float* logits) {
  kf_status st = head_common(s, rows, hidden, dtype);
  if (st != KF_OK) return st;
  if (!logits) return fail(KF_EINVAL, "logits is NULL");
  if (!hidden) return head_launch(s, rows, nullptr, dtype, logits);  // kept rows: at most kMaxBatch
  const size_t esz = dtype == KF_BF16 ? 2 : 4;
  for (int r0 = 0; r0 < rows; r0 += kMaxBatch) {
    const int n = rows - r0 < kMaxBatch ? rows - r0 : kMaxBatch;
    st = head_launch(s, n, (const char*)hidden + (size_t)r0 * s->cfg.hidden * esz, dtype,
                     logits + (size_t)r0 * s->cfg.vocab);
    if (st != KF_OK) return st;
  }
  return KF_OK;
}

kf_status kf_head_argmax(kf_stage* s, int32_t rows, const void* hidden, kf_dtype dtype, int32_t* token,
                         float* max_logit) {
  kf_status st = head_common(s, rows, hidden, dtype);
  if (st != KF_OK) return st;
  if (rows > kMaxBatch) return fail(KF_EINVAL, "rows %d above %d", rows, kMaxBatch);
  if (!token) return fail(KF_EINVAL, "token is NULL");
  st = head_launch(s, rows, hidden, dtype, nullptr);
  if (st != KF_OK) return st;
  const Tracer tr = s->tracer();
  tr.begin(KF_K_ARGMAX);
  const hipError_t e = launch_argmax_final(s->part_val, s->part_idx, s->lm_wg_used, rows, token, max_logit, s->stream);
  tr.end(KF_K_ARGMAX);
  KF_HIP(e, "argmax launch");
  return KF_OK;
}

// ------------------------------------------------------------------ prefill
// The allocating prefill grows the stage's own workspace (hipMalloc) to the largest
// chunk seen; the no-allocation variant lays the same workspace out in the
// device's static scratch array instead (stage->scratch, at most
// kPrefillScratchBytes) and records no timing events.
static kf_status prefill_impl(kf_stage* s, kf_kv* kv, int32_t user, int32_t pos0, int32_t n,
                              const int32_t* tokens_dev, const void* hidden_in_dev, void* hidden_out_dev, kf_dtype io,
                              bool no_alloc) {
  if (!s || !kv) return fail(KF_EINVAL, "stage or kv is NULL");
  if (kv->st != s) return fail(KF_EINVAL, "kv belongs to another stage");
  if (n < 1) return fail(KF_EINVAL, "n_tokens must be >= 1");
  if (user < 0 || user >= kv->max_users) return fail(KF_EINVAL, "user %d outside [0, %d)", user, kv->max_users);
  if ((tokens_dev == nullptr) == (hidden_in_dev == nullptr))
    return fail(KF_EINVAL, "exactly one of tokens / hidden input must be given");
  if (tokens_dev && !s->has_head) return fail(KF_ESTATE, "token input needs the head");
  if (!hidden_out_dev) return fail(KF_EINVAL, "hidden output is NULL");
  if (io != KF_F32 && io != KF_BF16) return fail(KF_EINVAL, "io dtype");
  if (pos0 != kv->len[user]) return fail(KF_EINVAL, "pos0 = %d but user %d holds %d positions", pos0, user, kv->len[user]);
  if ((int64_t)pos0 + n > kv->max_ctx) return fail(KF_ERANGE, "positions up to %d beyond max_ctx %d", pos0 + n, kv->max_ctx);

  const kf_model_config& c = s->cfg;
  PrefillArgs pa{};
  pa.H = c.hidden;
  pa.nq = c.n_q_heads;
  pa.nkv = c.n_kv_heads;
  pa.hd = c.head_dim;
  pa.F = c.ffn;
  pa.eps = c.rms_eps;
  pa.T = n;
  pa.pos0 = pos0;
  pa.user = user;
  pa.kv = kv->pages();
  pa.rope_cos = kv->rcos;
  pa.rope_sin = kv->rsin;
  pa.err_flag = s->err_flag;
  pa.stream = s->stream;
  PrefillWorkspace scratch_ws;
  PrefillWorkspace* ws = &s->pf;
  if (no_alloc) {
    const int64_t need = prefill_ws_bytes(pa);
    if (need > kPrefillScratchBytes)
      return fail(KF_ERANGE, "a chunk of %d tokens needs %lld bytes of prefill scratch, above the %lld held per device",
                  n, (long long)need, (long long)kPrefillScratchBytes);
    if (!s->scratch) return fail(KF_EDEVICE, "the device's prefill scratch has no address");
    prefill_carve(scratch_ws, s->scratch, pa);
    ws = &scratch_ws;
  } else {
    hipError_t e = prefill_reserve(s->pf, pa);
    if (e == hipErrorOutOfMemory) return fail(KF_ENOMEM, "device allocation of the prefill workspace");
    KF_HIP(e, "prefill workspace");
  }
  const int64_t upto = (int64_t)pos0 + n;
  const kf_status gst = kv_grant(kv, 1, &user, &upto);
  if (gst != KF_OK) return gst;
  const Tracer tr = no_alloc ? Tracer{} : s->tracer();  // event records may create events
  tr.begin(KF_K_PREP);
  hipError_t e = launch_prep_hidden(hidden_in_dev, io == KF_BF16, tokens_dev, s->embed, c.vocab, ws->x, n, c.hidden,
                                    s->err_flag, s->stream);
  tr.end(KF_K_PREP);
  KF_HIP(e, "prefill prep launch");
  ws->pending = 0;  // x now holds the whole input; no split-K slices are pending
  for (int l = s->lo; l < s->hi; ++l) {
    const LayerW& L = s->layers[l - s->lo];
    const int64_t loff = (l - s->lo) * kv->layer_stride;
    PrefillLayer pl{};
    pl.wqkv = L.wqkv;
    pl.wo = L.wo;
    pl.wg = L.wg;
    pl.wu = L.wu;
    pl.wd = L.wd;
    pl.g_attn = L.qkv_gain();  // NULL: folded into the matrix
    pl.g_mlp = L.mlp_gain();
    pl.g_qn = L.g_qn;
    pl.g_kn = L.g_kn;
    pl.kc = kv->k + loff;
    pl.vc = kv->v + loff;
    pl.out = l == s->hi - 1 ? hidden_out_dev : nullptr;
    pl.out_bf16 = io == KF_BF16;
    KF_HIP(prefill_layer(*ws, pa, pl, tr), "prefill layer");
  }
  kv->len[user] += n;
  return KF_OK;
}

kf_status kf_stage_prefill(kf_stage* s, kf_kv* kv, int32_t user, int32_t pos0, int32_t n, const int32_t* tokens_dev,
                           const void* hidden_in_dev, void* hidden_out_dev, kf_dtype io) {
  return prefill_impl(s, kv, user, pos0, n, tokens_dev, hidden_in_dev, hidden_out_dev, io, false);
}

kf_status kf_stage_prefill_noalloc(kf_stage* s, kf_kv* kv, int32_t user, int32_t pos0, int32_t n,
                                   const int32_t* tokens_dev, const void* hidden_in_dev, void* hidden_out_dev,
                                   kf_dtype io) {
  return prefill_impl(s, kv, user, pos0, n, tokens_dev, hidden_in_dev, hidden_out_dev, io, true);
}

// ------------------------------------------------------------------ instrumentation
kf_status kf_stage_profile(kf_stage* s, int32_t mask) {
  if (!s) return fail(KF_EINVAL, "stage is NULL");
  if (mask) {
    KF_HIP(hipStreamSynchronize(s->stream), "stream synchronize");
    s->ev_used = 0;
  }
  s->prof_mask = mask & KF_K_ALL;
  return KF_OK;
}

kf_status kf_stage_profile_read(kf_stage* s, int32_t cls, int64_t* launches, double* total_ms) {
  if (!s || !launches || !total_ms) return fail(KF_EINVAL, "NULL argument");
  if (cls < 0 || cls >= KF_K_COUNT) return fail(KF_EINVAL, "kernel class %d", cls);
  KF_HIP(hipStreamSynchronize(s->stream), "stream synchronize");
  int64_t n = 0;
  double t = 0.0;
  for (size_t i = 0; i < s->ev_used; ++i) {
    if (s->ev_cls[i] != cls) continue;
    float ms = 0.f;
    KF_HIP(hipEventElapsedTime(&ms, s->ev[2 * i], s->ev[2 * i + 1]), "event elapsed time");
    n++;
    t += ms;
  }
  *launches = n;
  *total_ms = t;
  return KF_OK;
}

}  // extern "C"

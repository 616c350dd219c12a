// A ring of stages on one device (Section III: a token passes from the head through
// every member's block range and returns to the head; Section VII-C: concurrent
// requests fill the pipeline bubble).  Host-only: every kernel runs inside the
// stages; this file orders their work across the members' streams with events.
#include <hip/hip_runtime_api.h>

#include <cstring>
#include <vector>

#include "error.h"
#include "kafila_ring.h"

using kf::fail;

namespace {

constexpr int kMaxGroups = 64;

#define KF_RING_HIP(call, what)                                                             \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return fail(KF_EDEVICE, "%s: %s", (what), hipGetErrorString(e_)); \
  } while (0)

#define KF_RING_TRY(call)          \
  do {                             \
    const kf_status st_ = (call);  \
    if (st_ != KF_OK) return st_;  \
  } while (0)

}  // namespace

struct kf_ring {
  int m = 0;
  std::vector<kf_stage*> st;
  std::vector<kf_kv*> kv;
  std::vector<hipStream_t> stream;
  int max_groups = 0, max_prefill = 0, max_users = 0, max_ctx = 0, hidden = 0;
  kf_dtype io = KF_F32;
  size_t esize = 4;
  // Decode hand-offs: hid[g][i] holds group g's rows after member i ([KF_MAX_BATCH, H]).
  // Prefill hand-offs: two [max_prefill, H] buffers, member i writing buffer i % 2.
  char* buf = nullptr;
  size_t pf_off = 0;
  std::vector<hipEvent_t> ev;     // [max_groups][m]: member i finished group g's step
  std::vector<hipEvent_t> ev_pf;  // [m]: member i finished the prefill chunk

  char* hid(int g, int i) const { return buf + ((size_t)g * m + i) * KF_MAX_BATCH * hidden * esize; }
  char* pf(int i) const { return buf + pf_off + (size_t)(i % 2) * max_prefill * hidden * esize; }

  void release() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : ev_pf)
      if (e) (void)hipEventDestroy(e);
    ev.clear();
    ev_pf.clear();
    if (buf) (void)hipFree(buf);
    buf = nullptr;
  }

  // Every paged member must have free pages for `grow` more positions of each user
  // (counted from the user's length), so that no member runs short mid-call.
  kf_status pool_check(int n, const std::vector<int>& len, int grow) const {
    for (int i = 0; i < m; ++i) {
      int32_t total = 0, free_pages = 0;
      KF_RING_TRY(kf_kv_pages(kv[i], &total, &free_pages));
      if (free_pages < 0) continue;  // a reserved cache
      int64_t need = 0;
      for (int j = 0; j < n; ++j)
        need += ((int64_t)len[j] + grow + KF_KV_PAGE - 1) / KF_KV_PAGE - ((int64_t)len[j] + KF_KV_PAGE - 1) / KF_KV_PAGE;
      if (need > free_pages)
        return fail(KF_ENOMEM, "member %d's KV pool has %d free pages, the call may need %lld", i, (int)free_pages,
                    (long long)need);
    }
    return KF_OK;
  }

  // Every user of the list must hold the same length in every member; returns it per user.
  kf_status lengths(const int32_t* users, int n, std::vector<int>& len) const {
    len.assign(n, 0);
    for (int j = 0; j < n; ++j) {
      const int u = users[j];
      if (u < 0 || u >= max_users) return fail(KF_EINVAL, "user %d outside [0, %d)", u, max_users);
      for (int k = 0; k < j; ++k)
        if (users[k] == u) return fail(KF_EINVAL, "user %d appears twice", u);
      for (int i = 0; i < m; ++i) {
        int32_t l = 0;
        KF_RING_TRY(kf_kv_len(kv[i], u, &l));
        if (i == 0) len[j] = l;
        else if (l != len[j])
          return fail(KF_EINVAL, "user %d holds %d positions in member 0 but %d in member %d", u, len[j], (int)l, i);
      }
    }
    return KF_OK;
  }
};

extern "C" {

kf_status kf_ring_create(int32_t n_members, kf_stage* const* stages, kf_kv* const* kvs, int32_t max_groups,
                         int32_t max_prefill, kf_dtype io, kf_ring** out) {
  if (!out) return fail(KF_EINVAL, "out is NULL");
  *out = nullptr;
  if (n_members < 1) return fail(KF_EINVAL, "n_members %d < 1", n_members);
  if (!stages || !kvs) return fail(KF_EINVAL, "stages / kvs is NULL");
  if (max_groups < 1 || max_groups > kMaxGroups) return fail(KF_EINVAL, "max_groups %d outside [1, %d]", max_groups, kMaxGroups);
  if (max_prefill < 1) return fail(KF_EINVAL, "max_prefill %d < 1", max_prefill);
  if (io != KF_F32 && io != KF_BF16) return fail(KF_EINVAL, "hand-off dtype must be KF_F32 or KF_BF16");

  kf_model_config cfg0{};
  int32_t dev0 = 0, next_lo = 0, users0 = 0, ctx0 = 0;
  std::vector<hipStream_t> streams(n_members);
  for (int i = 0; i < n_members; ++i) {
    if (!stages[i] || !kvs[i]) return fail(KF_EINVAL, "stages[%d] / kvs[%d] is NULL", i, i);
    kf_model_config c{};
    int32_t lo = 0, hi = 0, head = 0, dev = 0;
    void* s = nullptr;
    KF_RING_TRY(kf_stage_describe(stages[i], &c, &lo, &hi, &head, &s, &dev));
    if (i == 0) {
      cfg0 = c;
      dev0 = dev;
      if (!head) return fail(KF_EINVAL, "stages[0] must hold the head");
    } else {
      if (std::memcmp(&c, &cfg0, sizeof c) != 0) return fail(KF_EINVAL, "stages[%d] has another model config", i);
      if (dev != dev0) return fail(KF_EUNSUPPORTED, "stages[%d] is on device %d, stages[0] on %d", i, (int)dev, (int)dev0);
      if (head) return fail(KF_EINVAL, "only stages[0] may hold the head");
    }
    if (lo != next_lo) return fail(KF_EINVAL, "stages[%d] starts at layer %d, expected %d", i, (int)lo, (int)next_lo);
    next_lo = hi;
    kf_stage* owner = nullptr;
    int32_t mu = 0, mc = 0;
    KF_RING_TRY(kf_kv_describe(kvs[i], &owner, &mu, &mc));
    if (owner != stages[i]) return fail(KF_EINVAL, "kvs[%d] was not created on stages[%d]", i, i);
    if (i == 0) {
      users0 = mu;
      ctx0 = mc;
    } else if (mu != users0 || mc != ctx0) {
      return fail(KF_EINVAL, "kvs[%d] holds %d users x %d positions, kvs[0] %d x %d", i, (int)mu, (int)mc,
                  (int)users0, (int)ctx0);
    }
    streams[i] = (hipStream_t)s;
  }
  if (next_lo != cfg0.n_layers) return fail(KF_EINVAL, "the last stage ends at layer %d of %d", (int)next_lo, cfg0.n_layers);
  int cur = -1;
  KF_RING_HIP(hipGetDevice(&cur), "hipGetDevice");
  if (cur != dev0) return fail(KF_EINVAL, "the stages' device (%d) must be current, not %d", (int)dev0, cur);

  kf_ring* r = new kf_ring;
  r->m = n_members;
  r->st.assign(stages, stages + n_members);
  r->kv.assign(kvs, kvs + n_members);
  r->stream = streams;
  r->max_groups = max_groups;
  r->max_prefill = max_prefill;
  r->max_users = users0;
  r->max_ctx = ctx0;
  r->hidden = cfg0.hidden;
  r->io = io;
  r->esize = io == KF_F32 ? 4 : 2;
  const size_t dec = (size_t)max_groups * n_members * KF_MAX_BATCH * cfg0.hidden * r->esize;
  r->pf_off = (dec + 255) & ~(size_t)255;
  const size_t total = r->pf_off + 2 * (size_t)max_prefill * cfg0.hidden * r->esize;
  if (hipMalloc((void**)&r->buf, total) != hipSuccess) {
    (void)hipGetLastError();
    r->buf = nullptr;
    delete r;
    return fail(KF_ENOMEM, "ring hand-off buffers of %zu bytes", total);
  }
  // Ordering-only events: no timing, and no system-scope fence (every consumer is on this device).
  const unsigned flags = hipEventDisableTiming | hipEventDisableSystemFence;
  r->ev.assign((size_t)max_groups * n_members, nullptr);
  r->ev_pf.assign(n_members, nullptr);
  for (auto* list : {&r->ev, &r->ev_pf}) {
    for (hipEvent_t& e : *list) {
      if (hipEventCreateWithFlags(&e, flags) != hipSuccess) {
        e = nullptr;
        (void)hipGetLastError();
        r->release();
        delete r;
        return fail(KF_EDEVICE, "event creation");
      }
    }
  }
  *out = r;
  return KF_OK;
}

kf_status kf_ring_destroy(kf_ring* r) {
  if (!r) return fail(KF_EINVAL, "ring is NULL");
  for (hipStream_t s : r->stream) (void)hipStreamSynchronize(s);
  r->release();
  delete r;
  return KF_OK;
}

kf_status kf_ring_sync(kf_ring* r) {
  if (!r) return fail(KF_EINVAL, "ring is NULL");
  kf_status worst = KF_OK;
  for (int i = 0; i < r->m; ++i) {
    const kf_status s = kf_stage_sync(r->st[i]);
    if (s != KF_OK && worst == KF_OK) worst = s;
  }
  return worst;
}

kf_status kf_ring_prefill(kf_ring* r, int32_t user, int32_t n_tokens, const int32_t* tokens_dev,
                          int32_t* next_token_dev) {
  if (!r) return fail(KF_EINVAL, "ring is NULL");
  if (!tokens_dev || !next_token_dev) return fail(KF_EINVAL, "tokens / next token is NULL");
  if (n_tokens < 1 || n_tokens > r->max_prefill)
    return fail(KF_EINVAL, "n_tokens %d outside [1, %d]", n_tokens, r->max_prefill);
  std::vector<int> len;
  KF_RING_TRY(r->lengths(&user, 1, len));
  if ((int64_t)len[0] + n_tokens > r->max_ctx)
    return fail(KF_ERANGE, "user %d: %d + %d positions exceed max_ctx %d", user, len[0], n_tokens, r->max_ctx);
  KF_RING_TRY(r->pool_check(1, len, n_tokens));

  for (int i = 0; i < r->m; ++i) {
    if (i > 0) KF_RING_HIP(hipStreamWaitEvent(r->stream[i], r->ev_pf[i - 1], 0), "hand-off wait");
    KF_RING_TRY(kf_stage_prefill(r->st[i], r->kv[i], user, len[0], n_tokens, i == 0 ? tokens_dev : nullptr,
                                 i == 0 ? nullptr : r->pf(i - 1), r->pf(i), r->io));
    KF_RING_HIP(hipEventRecord(r->ev_pf[i], r->stream[i]), "hand-off record");
  }
  // Return leg: the head samples after the chunk's last token.
  KF_RING_HIP(hipStreamWaitEvent(r->stream[0], r->ev_pf[r->m - 1], 0), "return-leg wait");
  const char* last = r->pf(r->m - 1) + (size_t)(n_tokens - 1) * r->hidden * r->esize;
  return kf_head_argmax(r->st[0], 1, last, r->io, next_token_dev, nullptr);
}

kf_status kf_ring_generate(kf_ring* r, int32_t n_groups, const int32_t* group_size, const int32_t* users,
                           const int32_t* tokens_in_dev, int32_t steps, int32_t* tokens_out_dev,
                           void* hidden_out_dev) {
  if (!r) return fail(KF_EINVAL, "ring is NULL");
  if (!group_size || !users || !tokens_in_dev || !tokens_out_dev) return fail(KF_EINVAL, "NULL argument");
  if (n_groups < 1 || n_groups > r->max_groups)
    return fail(KF_EINVAL, "n_groups %d outside [1, %d]", n_groups, r->max_groups);
  if (steps < 1) return fail(KF_EINVAL, "steps %d < 1", steps);
  std::vector<int> off(n_groups + 1, 0);
  for (int g = 0; g < n_groups; ++g) {
    if (group_size[g] < 1 || group_size[g] > KF_MAX_BATCH)
      return fail(KF_EINVAL, "group_size[%d] = %d outside [1, %d]", g, group_size[g], KF_MAX_BATCH);
    off[g + 1] = off[g] + group_size[g];
  }
  const int U = off[n_groups];
  std::vector<int> len;
  KF_RING_TRY(r->lengths(users, U, len));
  for (int j = 0; j < U; ++j)
    if ((int64_t)len[j] + steps > r->max_ctx)
      return fail(KF_ERANGE, "user %d: %d + %d positions exceed max_ctx %d", users[j], len[j], steps, r->max_ctx);
  KF_RING_TRY(r->pool_check(U, len, steps));

  const int m = r->m;
  int32_t pos[KF_MAX_BATCH];
  // The return leg of group g's previous step: the head samples from the last member's rows.
  auto sample = [&](int g, int t) -> kf_status {
    KF_RING_HIP(hipStreamWaitEvent(r->stream[0], r->ev[(size_t)g * m + m - 1], 0), "return-leg wait");
    if (hidden_out_dev) {
      const size_t row = (size_t)r->hidden * r->esize;
      KF_RING_HIP(hipMemcpyAsync(static_cast<char*>(hidden_out_dev) + ((size_t)t * U + off[g]) * row, r->hid(g, m - 1),
                                 (size_t)group_size[g] * row, hipMemcpyDeviceToDevice, r->stream[0]),
                  "return-leg copy");
    }
    return kf_head_argmax(r->st[0], group_size[g], r->hid(g, m - 1), r->io, tokens_out_dev + (size_t)t * U + off[g],
                          nullptr);
  };
  for (int t = 0; t < steps; ++t) {
    for (int g = 0; g < n_groups; ++g) {
      const int B = group_size[g];
      const int32_t* ug = users + off[g];
      for (int b = 0; b < B; ++b) pos[b] = len[off[g] + b] + t;
      const int32_t* tok = t == 0 ? tokens_in_dev + off[g] : tokens_out_dev + (size_t)(t - 1) * U + off[g];
      for (int i = 0; i < m; ++i) {
        if (i == 0) {
          if (t > 0) KF_RING_TRY(sample(g, t - 1));
          KF_RING_TRY(kf_stage_decode(r->st[0], r->kv[0], B, ug, pos, tok, nullptr, r->hid(g, 0), r->io));
        } else {
          KF_RING_HIP(hipStreamWaitEvent(r->stream[i], r->ev[(size_t)g * m + i - 1], 0), "hand-off wait");
          KF_RING_TRY(kf_stage_decode(r->st[i], r->kv[i], B, ug, pos, nullptr, r->hid(g, i - 1), r->hid(g, i), r->io));
        }
        KF_RING_HIP(hipEventRecord(r->ev[(size_t)g * m + i], r->stream[i]), "hand-off record");
      }
    }
  }
  for (int g = 0; g < n_groups; ++g) KF_RING_TRY(sample(g, steps - 1));
  return KF_OK;
}

}  // extern "C"

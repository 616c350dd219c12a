// Internal interface between the stage runtime (stage.hip) and the gfx950 kernels.
// Nothing here is exported from the shared library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kf {

constexpr int kMaxBatch = 4;
constexpr int kMaxGroup = 8;     // query heads per KV head
constexpr int kAttnMinSplit = 16;   // keys per split-KV workgroup, lower bound
constexpr int kAttnMaxSplit = 1024; // keys per split-KV workgroup, upper bound
// Output rows per workgroup of the head-split output projection (128 and 64 measured
// slower: every workgroup repeats its head's merge of the split partials).
constexpr int kOprojRows = 256;
constexpr int kAttnMaxSplitCount = 1024;  // split-KV workgroups per (row, KV head), upper bound
// Decode attention on the matrix cores: workgroups of kAttnMfmaWaves waves over
// splits of any multiple of kAttnMfmaAlign keys (16-key blocks, one page or
// less each).
#ifndef KF_ATTN_WAVES
#define KF_ATTN_WAVES 4
#endif
constexpr int kAttnMfmaWaves = KF_ATTN_WAVES;
constexpr int kAttnMfmaAlign = 16;

// Bits of the stage's sticky device error flag (reported and cleared by kf_stage_sync).
enum : int {
  kErrToken = 1,      // a token id outside [0, vocab): its hidden row became NaN
  kErrF16Range = 2,   // an activation, key or value stored in fp16 was at or beyond 65520 in magnitude
  kErrNaNLogit = 4,   // a logit was NaN (the argmax skips it; a row of NaN gives token -1)
};

// fp32 to fp16 bits (round to nearest even), noting in `bad` a value that fp16
// cannot hold (|v| >= 65520 rounds to infinity; an infinite input counts too).
__device__ __forceinline__ uint16_t f16_checked(float v, bool& bad) {
  bad |= __builtin_fabsf(v) >= 65520.0f;
  return __builtin_bit_cast(uint16_t, (_Float16)v);
}
__device__ __forceinline__ void raise_err(int* flag, bool bad, int bit) {
  if (bad && flag) atomicOr(flag, bit);
}

// KV cache pages.  One layer's K (and, alike, V) is an array of pages of kKvPage
// positions, each page [kv_head][kKvPage][hd] fp16.  Position t of user u lies
// at slot t % kKvPage of the page with id table[u * ppu + t / kKvPage] (a paged
// cache, whose pages come from a shared pool), or u * ppu + t / kKvPage (a
// cache without a table: each user's ppu pages reserved in order).
constexpr int kKvPage = 64;
struct KvPages {
  const int* table;     // [max_users][ppu] page ids, or NULL
  int ppu;              // pages per user
  int64_t page_stride;  // elements per page: nkv * kKvPage * hd
};
__device__ __forceinline__ int kv_page(const KvPages& kp, int user, int i) {
  return kp.table ? kp.table[user * kp.ppu + i] : user * kp.ppu + i;
}
// Element offset of (user, kv head g, position t) in a layer's K or V.
__device__ __forceinline__ int64_t kv_offset(const KvPages& kp, int user, int g, int t, int hd) {
  return (int64_t)kv_page(kp, user, t / kKvPage) * kp.page_stride + ((int64_t)g * kKvPage + t % kKvPage) * hd;
}

// Optional per-launch marker around each kernel (instrumentation hook of the runtime).
struct Tracer {
  void* ctx = nullptr;
  void (*fn)(void* ctx, int cls, int begin) = nullptr;
  void begin(int cls) const {
    if (fn) fn(ctx, cls, 1);
  }
  void end(int cls) const {
    if (fn) fn(ctx, cls, 0);
  }
};

enum GemvEpi : int {
  kEpiQKV = 0,     // RoPE on q and k, q -> fp32 workspace, k and v -> fp16 cache at the row's position
  kEpiResid = 1,   // x[b][row] += y (fp32 residual stream), optional copy to the hidden output
  kEpiSwiGLU = 2,  // a[b][j] = silu(gate_j) * up_j
  kEpiLMHead = 3,  // optional fp32 logits, per-workgroup (max, lowest index) partials
};

// Element type of a residual GEMV's optional copy output.
enum { kOut2F32 = 0, kOut2BF16 = 1, kOut2F16 = 2 };

// One decode GEMV launch: y[b][n] = sum_k W[n][k] * in[b][k] (* gain[k] * rsqrt(mean(in^2)+eps) if norm).
struct GemvParams {
  const uint16_t* w0;  // fp16 matrix rows (QKV: [q;k;v] rows; SwiGLU: gate; others: the matrix)
  const uint16_t* w1;  // SwiGLU: up rows; unused otherwise
  const uint16_t* gain;  // RMSNorm gain [K] when the launch normalises its input
  const float* in;     // [B][K] fp32
  int K;               // reduction length (multiple of 8)
  int N;               // output rows (logical)
  float eps;
  int batch;

  // kEpiResid
  float* x;            // [B][N] residual stream, updated in place
  void* out2;          // optional [B][N] copy of the updated rows, element type out2_type
  int out2_type;       // kOut2F32, kOut2BF16 (a bf16 hidden output) or kOut2F16 (the next GEMV's input)

  // kEpiQKV
  float* q;            // [B][nq*hd]
  uint16_t* kc;        // K cache of this layer (fp16 bits), pages as in KvPages
  uint16_t* vc;
  KvPages kv;
  int nq, nkv, hd;
  const float* rope_cos;  // [max_ctx][hd/2]
  const float* rope_sin;
  int users[kMaxBatch];
  int pos[kMaxBatch];
  // Blocks with per-head q/k norms: when set, q goes to `q` and k to kraw
  // ([B][nkv][hd] fp32) as projected (after the attention RMSNorm), without
  // RoPE; the decode attention finishes both.  v goes to the cache as usual.
  float* kraw;

  // kEpiSwiGLU
  float* act;          // [B][N] with N = F: fp32, or fp16 when act16 is set
  int act16;
  // Input rows `in` stored as fp16 (the down projection's input at batch > 1), else fp32.
  int in16;

  // Launches with the stage input as their input rows (instead of `in`): the
  // first layer's QKV and the LM head.  Exactly one of src / tokens is set.
  const void* src;         // [B][K] hidden input, fp32 or (src_bf16) bf16
  int src_bf16;
  const int32_t* tokens;   // [B] token ids: rows of `embed` [vocab][K] bf16
  const uint16_t* embed;
  int vocab;
  float* x_init;           // optional [B][K]: workgroup 0 stores the input rows here (residual stream)
  int* err_flag;           // sticky error bits (kErrToken, kErrF16Range, kErrNaNLogit); every launch sets it

  // kEpiLMHead
  float* logits;       // optional [B][N]
  float* part_val;     // [B][n_wg]
  int* part_idx;       // [B][n_wg]
  int n_wg;
};

struct AttnParams {
  const float* q;      // [B][nq*hd] rotated queries
  uint16_t* kc;        // layer base (fp16 bits), pages as in KvPages (written only for the new key of qk-norm blocks)
  const uint16_t* vc;
  float* part_acc;     // [B][nq][max_split][hd]
  float* part_ml;      // [B][nq][max_split][2]
  KvPages kv;
  int nq, nkv, hd;
  int split;           // keys per workgroup
  int n_split;         // workgroups per (row, kv head)
  int max_split;       // allocated split capacity
  float scale_log2;    // log2(e) / sqrt(hd)
  int users[kMaxBatch];
  int len[kMaxBatch];  // keys visible to row b: position + 1
  // Blocks with per-head q/k norms: q holds the projections as they come from
  // the QKV GEMV (no RoPE).  Every workgroup RMS-normalises (gains gq, eps) and
  // rotates the query heads it scores; the workgroup whose split holds row b's
  // new position does the same for the new key (kraw, gains gk), stores it to the
  // cache and scores it from registers.  kraw NULL: q is already rotated and the
  // new key is in the cache.
  const float* kraw;      // [B][nkv][hd]
  const uint16_t* gq;     // [hd] bf16
  const uint16_t* gk;
  const float* rope_cos;  // [max_ctx][hd/2]
  const float* rope_sin;
  float eps;
  int* err_flag;          // sticky error bits: kErrF16Range for an fp16 store out of range
};

// Launchers (return hipGetLastError() of the launch).
int gemv_grid(int epi, int rows_per_wg, const GemvParams& p);
hipError_t launch_gemv(int epi, int rows_per_wg, int chunks_in_flight, bool norm, const GemvParams& p, hipStream_t s);
// The same launch with the stage input (p.src or p.tokens) as its input rows.
hipError_t launch_gemv_src(int epi, int rows_per_wg, int chunks_in_flight, bool norm, const GemvParams& p,
                           hipStream_t s);
hipError_t launch_attn_decode(const AttnParams& p, int batch, hipStream_t s);
// Head h of row b merged from the attention partials in p, to o16[b][h*hd:(h+1)*hd]
// (fp16) or, with o16 NULL, to o32[b][h*hd:(h+1)*hd] (fp32).
hipError_t launch_attn_merge(const AttnParams& p, uint16_t* o16, float* o32, int batch, hipStream_t s);
// x[b][0:N) += W_o o_b with o_b merged from the attention partials in p (W_o [N][nq*hd] fp16).
hipError_t launch_oproj_heads(const AttnParams& p, const uint16_t* w, float* x, int N, int batch, hipStream_t s);
hipError_t launch_prep_hidden(const void* in, int in_bf16, const int32_t* tokens, const uint16_t* embed, int vocab,
                              float* x, int rows, int H, int* err_flag, hipStream_t s);
hipError_t launch_argmax_final(const float* part_val, const int* part_idx, int n_wg, int rows, int32_t* token,
                               float* max_logit, hipStream_t s);
// In place over n elements: bf16 weights to fp16 (round to nearest even); *bad |= 1
// if a finite weight is beyond the fp16 range.
hipError_t launch_weights_to_f16(uint16_t* w, int64_t n, int* bad, hipStream_t s);
// Sets *flag when some w[r][k] g[k] (bf16 w [n / K][K], bf16 g [K]) has no finite fp16 rounding.
hipError_t launch_gain_fold_check(const uint16_t* w, int64_t n, int K, const uint16_t* g, int* flag, hipStream_t s);
// In place: bf16 w[r][k] -> fp16 w[r][k] g[k] (the gain folded into the columns); *bad on an fp16 overflow.
hipError_t launch_weights_to_f16_gain(uint16_t* w, int64_t n, int K, const uint16_t* g, int* bad, hipStream_t s);
hipError_t launch_store_hidden(const float* x, void* out, int out_bf16, int64_t n, hipStream_t s);
// Positions [pos0, pos0 + n) of one user in one layer (k, v: the layer's base)
// from / to [n][nkv][hd] rows.  src_type: 0 fp32, 1 bf16, 2 fp16 (the kf_dtype values).
hipError_t launch_kv_write(uint16_t* k, uint16_t* v, const KvPages& kp, int user, int pos0, const void* src_k,
                           const void* src_v, int src_type, int n, int nkv, int hd, hipStream_t s);
hipError_t launch_kv_read(const uint16_t* k, const uint16_t* v, const KvPages& kp, int user, int pos0, float* dst_k,
                          float* dst_v, int n, int nkv, int hd, hipStream_t s);
// table[idx[i]] = val[i] for i < n (n <= kKvTableBatch): page assignments of a paged cache.
constexpr int kKvTableBatch = 32;
struct KvTableUpdate {
  int n;
  int idx[kKvTableBatch];
  int val[kKvTableBatch];
};
hipError_t launch_kv_table_update(int* table, const KvTableUpdate& u, hipStream_t s);

}  // namespace kf

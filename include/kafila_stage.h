/*
 * kafila_stage.h -- one pipeline stage of a decoder-only LLM on one MI355X (gfx950).
 *
 * In Kafila (arxiv 2609.34045) a model's contiguous chain of transformer blocks
 * is divided among the members of a ring; each member runs a *stage*: the
 * hidden state of every token passes through its block range, and the member
 * holding the *head* also embeds tokens before its blocks and unembeds and
 * samples after the model's last block (Section III and Fig. 1).  A stage's
 * decode cost is dominated by reading its weights once per token (Section V-A,
 * eq. (2)); the session reserves cache for a declared context and concurrency
 * and refuses a plan that would exhaust a device (Sections V-C, V-D).
 *
 * The block is a pre-norm decoder layer: RMSNorm, grouped-query attention with
 * rotate-half RoPE over a per-user KV cache, SwiGLU MLP, no biases.  The head is
 * an embedding gather, a final RMSNorm, the vocabulary projection and a greedy
 * argmax (lowest index on ties).
 *
 * Conventions
 *  - "_dev" pointers are device pointers on the stage's device; other pointers
 *    are host pointers.  The caller owns every I/O buffer.
 *  - bf16 tensors are passed as uint16_t bit patterns.  Matrices are row-major
 *    [out, in] (the layout of a linear layer's weight).
 *  - Compute calls only enqueue work on the stage's stream and return; argument
 *    checks run on the host before anything is enqueued, and a call that fails
 *    them changes no state.  Errors of enqueued work are sticky and surface from
 *    kf_stage_sync() or the next call as KF_EDEVICE.
 *  - A stage and its KV caches are not thread-safe; distinct stages are
 *    independent.  kf_last_error() returns a thread-local message for the last
 *    failure on the calling thread.
 *  - Requirements checked at init: head_dim in {64, 128}; n_q_heads a multiple
 *    of n_kv_heads with at most 8 query heads per KV head; hidden and ffn
 *    multiples of 64.  Anything else is KF_EUNSUPPORTED.  The query width
 *    n_q_heads * head_dim need not equal hidden.
 */
#ifndef KAFILA_STAGE_H
#define KAFILA_STAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KF_ABI_VERSION 5  /* 2: kf_model_config.qk_norm and the q/k norm tensor kinds;
                            3: paged KV caches, kf_stage_describe, kf_kv_describe;
                            4: kf_stage_set_flags / kf_stage_get_flags (KF_STAGE_ORDERED), range and
                               NaN-logit errors reported by kf_stage_sync, token -1 for a row of NaN logits,
                               kf_stage_prefill_noalloc; kf_ring_generate's hidden_out_dev (kafila_ring.h);
                               the kf_shard_* loader (kafila_shard.h);
                            5: a head stage's decode may keep its output rows (hidden_out_dev NULL)
                               for kf_head_logits / kf_head_argmax with hidden_dev NULL */
#define KF_KV_PAGE 64     /* positions per KV cache page */
#define KF_MAX_BATCH 4

typedef struct kf_stage kf_stage;
typedef struct kf_kv kf_kv;

typedef enum {
  KF_OK = 0,
  KF_EINVAL = 1,       /* malformed argument (NULL, size mismatch, position gap, bad range) */
  KF_ENOMEM = 2,       /* a device or host allocation failed */
  KF_ERANGE = 3,       /* a position or length beyond the declared capacity */
  KF_ESTATE = 4,       /* call not allowed in this state (e.g. head call on a stage without the head) */
  KF_EDEVICE = 5,      /* a HIP error, including a sticky error from earlier enqueued work */
  KF_EUNSUPPORTED = 6  /* a model shape the kernels are not built for */
} kf_status;

typedef enum { KF_F32 = 0, KF_BF16 = 1, KF_F16 = 2 } kf_dtype; /* element types at the boundary */

typedef struct {
  int32_t n_layers;   /* layers in the whole model (the stage holds a sub-range) */
  int32_t hidden;     /* H */
  int32_t n_q_heads;  /* nq */
  int32_t n_kv_heads; /* nkv; query head h reads KV head h / (nq / nkv) */
  int32_t head_dim;   /* hd */
  int32_t ffn;        /* F */
  int32_t vocab;      /* V (used only with the head) */
  float rms_eps;      /* RMSNorm epsilon, added to mean(x^2) inside the square root */
  float rope_theta;   /* RoPE base: pair (i, i + hd/2) turns by pos * theta^(-2i/hd) */
  int32_t qk_norm;    /* 1: each q and k head vector is RMS-normalised (gains KF_W_Q_NORM / KF_W_K_NORM,
                         eps rms_eps) before RoPE, as in the Qwen3 models the paper serves; 0: no such norm */
} kf_model_config;

typedef enum {
  KF_W_ATTN_NORM = 0, /* [H]            gain of the attention RMSNorm */
  KF_W_Q = 1,         /* [nq*hd, H] */
  KF_W_K = 2,         /* [nkv*hd, H] */
  KF_W_V = 3,         /* [nkv*hd, H] */
  KF_W_O = 4,         /* [H, nq*hd] */
  KF_W_MLP_NORM = 5,  /* [H]            gain of the MLP RMSNorm */
  KF_W_GATE = 6,      /* [F, H] */
  KF_W_UP = 7,        /* [F, H] */
  KF_W_DOWN = 8,      /* [H, F] */
  KF_W_EMBED = 9,     /* [V, H]         head only */
  KF_W_FINAL_NORM = 10, /* [H]          head only */
  KF_W_LM_HEAD = 11,  /* [V, H]         head only (not tied to the embedding) */
  KF_W_Q_NORM = 12,   /* [hd]           gain of the per-head q norm (only when qk_norm) */
  KF_W_K_NORM = 13    /* [hd]           gain of the per-head k norm (only when qk_norm) */
} kf_tensor_kind;

typedef struct {
  int32_t layer;        /* global layer index in [layer_lo, layer_hi); -1 for head tensors */
  int32_t kind;         /* kf_tensor_kind */
  const uint16_t* bf16; /* host pointer to row-major bf16 bits */
  int64_t numel;        /* must equal the element count of the kind's shape */
} kf_tensor;

typedef struct {
  const kf_tensor* tensors;
  int32_t count;
} kf_weights;

/* ABI version of the loaded library (KF_ABI_VERSION at build time). */
int32_t kf_abi_version(void);

/* Thread-local message describing the last failed call on this thread ("" if none). */
const char* kf_last_error(void);

/*
 * Byte sizes behind the stage-cost model (Section V-A, eq. (2)) and the block
 * limit at a declared context and concurrency (Section V-C).
 *   beta_block : bytes of one decoder layer's weights (2 bytes per element as given in bf16 and as
 *                held: fp16 matrices, bf16 gains; both gains included)
 *   beta_head  : bytes of the head's weights (embedding + final gain + LM head), 0 without the head
 *   resident   : device bytes kf_stage_init + kf_kv_create(max_users, max_ctx) would hold for
 *                layers [lo, hi): weights, KV cache, RoPE table and decode workspaces
 * Host only; any output pointer may be NULL.  KF_EINVAL for an invalid config or range.
 */
kf_status kf_stage_bytes(const kf_model_config* cfg, int32_t layer_lo, int32_t layer_hi, int32_t has_head,
                         int32_t max_users, int32_t max_ctx, int64_t* beta_block, int64_t* beta_head,
                         int64_t* resident);

/*
 * Create a stage holding layers [layer_lo, layer_hi) of the model and, if has_head,
 * the head (Section III and Fig. 1: a member's contiguous block range, and the
 * head's embedding and unembedding on the member the rotation makes head;
 * Section V-C places it).  Weight tensors are copied to the current HIP device (the stage's
 * device) before the call returns, so the caller may free them afterwards.  Every
 * layer tensor of every held layer must be present exactly once (kinds 0..8, plus
 * KF_W_Q_NORM and KF_W_K_NORM when qk_norm), plus the three head tensors when
 * has_head; anything else is KF_EINVAL.  The weight matrices (kinds Q, K, V, O, GATE,
 * UP, DOWN, LM_HEAD) are stored in fp16, rounded to nearest even from the bf16
 * given: exact for 2^-17 <= |w| < 65504 and for 0, within 2^-25 below that.  A finite
 * weight that fp16 cannot hold (|w| >= 65520) is KF_EINVAL.  Gains and the
 * embedding table stay bf16.  hip_stream (a
 * hipStream_t, NULL for the default stream) is where all later work is enqueued.
 */
kf_status kf_stage_init(const kf_model_config* cfg, int32_t layer_lo, int32_t layer_hi, int32_t has_head,
                        const kf_weights* weights, void* hip_stream, kf_stage** out);

/* Waits for the stage's stream, then frees its device memory.  KV caches of the stage must be destroyed first. */
kf_status kf_stage_destroy(kf_stage* stage);

/* Replace the stream later work is enqueued on (the caller orders it after earlier work). */
kf_status kf_stage_set_stream(kf_stage* stage, void* hip_stream);

/*
 * Wait for all enqueued work; KF_EDEVICE (with the HIP error text) if any of it failed.
 * Then reports, and clears, the stage's sticky data errors raised by enqueued work:
 *   KF_EINVAL : a token id given to decode or prefill was outside [0, vocab); that row's
 *               hidden state was set to NaN;
 *   KF_ERANGE : a value the stage holds in fp16 (keys and values in the cache, and the
 *               fp16 activations: from batch 2 the decode residual copy, SwiGLU output and
 *               merged attention output; in prefill the normalised rows, queries, attention
 *               output and SwiGLU output) reached 65520 in magnitude and was stored as
 *               infinity; or a logit was NaN (skipped by the argmax; see kf_head_argmax).
 * The message (kf_last_error) names every condition that occurred.
 */
kf_status kf_stage_sync(kf_stage* stage);

/*
 * Behaviour flags of a stage (0 after kf_stage_init).
 *   KF_STAGE_ORDERED : batch-1 decode adds the query heads' output projections to each
 *                      residual row in a fixed order (a separate merge of the split-KV
 *                      partials, then a row-owning output GEMV), so that repeated runs are
 *                      bit-identical and a stage split anywhere composes to the same bits.
 *                      Without it, batch 1 fuses the merge into a head-split output
 *                      projection whose fp32 additions arrive in any order (one launch
 *                      fewer per layer; results vary run to run by fp32 reassociation).
 *                      Greedy decoding at a fixed seed (Section VI-A) reproduces exactly
 *                      only with this flag.  Batch 2-4 and prefill are always in fixed order.
 * kf_stage_set_flags: KF_EINVAL for unknown bits.  Host-only; affects later calls.
 */
#define KF_STAGE_ORDERED 1
kf_status kf_stage_set_flags(kf_stage* stage, int32_t flags);
kf_status kf_stage_get_flags(const kf_stage* stage, int32_t* flags);

/* What a stage holds: its config, layer range [layer_lo, layer_hi), whether it holds
 * the head, the stream it enqueues on (a hipStream_t) and its device ordinal.  Any
 * output pointer may be NULL.  Host-only. */
kf_status kf_stage_describe(const kf_stage* stage, kf_model_config* cfg, int32_t* layer_lo, int32_t* layer_hi,
                            int32_t* has_head, void** hip_stream, int32_t* device);

/*
 * Reserve a KV cache for max_users concurrent users of context up to max_ctx tokens
 * each, for every layer the stage holds (the declared concurrency x context of
 * Section V-C).  Layout on the device: fp16 K and V in pages of KF_KV_PAGE
 * positions, [layer][page][kv_head][KF_KV_PAGE][hd]; user u holds pages
 * u * P .. u * P + P - 1 with P = ceil(max_ctx / KF_KV_PAGE) (fp16 keeps 8x the
 * mantissa of bf16 in the same bytes; keys and values must stay below 65504 in
 * magnitude).
 * All user lengths start at 0.  KF_ENOMEM if the device cannot hold it.
 */
kf_status kf_kv_create(kf_stage* stage, int32_t max_users, int32_t max_ctx, kf_kv** out);

/*
 * A paged KV cache: the same users and context limits, but only n_pages pages
 * (>= 1) of KF_KV_PAGE positions for all users together, so that cache is held by
 * the prompts that arrive rather than reserved for every declared user (the
 * reservation the paper leaves as future work, Section VIII).  A user is lent
 * pages from the pool as its length grows (decode, prefill, kf_kv_write,
 * kf_kv_set_len) and gives back the pages past its new length when
 * kf_kv_set_len shortens it (0 frees them all).  A call that needs more pages
 * than are free fails with KF_ENOMEM before anything is enqueued.  A device
 * table [max_users][P] maps each user's page index to a pool page.
 */
kf_status kf_kv_create_paged(kf_stage* stage, int32_t max_users, int32_t max_ctx, int32_t n_pages, kf_kv** out);
kf_status kf_kv_destroy(kf_kv* kv);

/* Pages of the cache and, for a paged cache, how many are free (-1 for a reserved cache, whose users
 * hold all their pages from the start).  Host-only. */
kf_status kf_kv_pages(const kf_kv* kv, int32_t* total, int32_t* free_pages);

/* The stage a cache was created on, and its capacity.  Any output pointer may be NULL.  Host-only. */
kf_status kf_kv_describe(const kf_kv* kv, kf_stage** stage, int32_t* max_users, int32_t* max_ctx);

/* Number of cached positions of a user (a host-side value; no device sync). */
kf_status kf_kv_len(const kf_kv* kv, int32_t user, int32_t* len);

/* Set a user's length to any value in [0, max_ctx]: 0 resets the user; positions below
 * len are from then on taken as valid in every layer (e.g. after kf_kv_write).  In a
 * paged cache the user holds exactly the pages its length needs afterwards
 * (KF_ENOMEM, with nothing changed, if the pool cannot lend them). */
kf_status kf_kv_set_len(kf_kv* kv, int32_t user, int32_t len);

/*
 * Copy n positions of keys (already rotated) and values for one held layer and user,
 * from k_dev / v_dev laid out [n, nkv, hd] in dtype (KF_F16 or KF_BF16 bits, or KF_F32),
 * stored as fp16 rounded to nearest even, into positions [pos0, pos0 + n).  Does not
 * change lengths (a paged cache lends the pages up to pos0 + n; KF_ENOMEM if it cannot).
 * KF_ERANGE if pos0 + n > max_ctx.  Enqueued on the stage's stream.
 */
kf_status kf_kv_write(kf_kv* kv, int32_t layer, int32_t user, int32_t pos0, int32_t n, const void* k_dev,
                      const void* v_dev, kf_dtype dtype);

/* Copy positions [pos0, pos0 + n) of one layer and user out as fp32 (exact), [n, nkv, hd].
 * KF_ERANGE for positions on pages the user does not hold (paged caches). */
kf_status kf_kv_read(const kf_kv* kv, int32_t layer, int32_t user, int32_t pos0, int32_t n, float* k_dev,
                     float* v_dev);

/*
 * Forward one token for each of `batch` (1..KF_MAX_BATCH) users (decode): the
 * stage's part of one decode step, hidden state in, hidden state out (Section III:
 * the token's hidden state passes through each member's block range around the
 * ring; the head member embeds it first).  Its cost is one read of every held
 * weight plus each user's cache (Section V-A, eq. (2)); batch > 1 serves several
 * users' requests in one pass over the weights (Sections III and VII-C).
 *   users[b], positions[b] : host arrays; users distinct and < max_users;
 *                            positions[b] must equal the user's current length
 *                            (append-only; else KF_EINVAL) and be < max_ctx (else KF_ERANGE).
 *   tokens_dev  : int32 [batch] token ids (stage with the head only), or NULL
 *   hidden_in_dev : [batch, H] in `io`, or NULL; exactly one of tokens_dev / hidden_in_dev
 *   hidden_out_dev : [batch, H] in `io`; may alias hidden_in_dev.  NULL (a stage
 *                    that holds the head only, else KF_EINVAL): the output rows stay
 *                    in the stage for the head (kf_head_logits / kf_head_argmax with
 *                    hidden_dev NULL), as when the member that holds the model's
 *                    last blocks also holds the head and samples the next token.
 *                    At batch 2-4 they are kept in fp16 (the rounding every layer's
 *                    input of this stage already takes), which halves the LM head's
 *                    input traffic; at batch 1 in fp32.
 * Row b's token is at positions[b]: its key and value are written at that slot of
 * the user's cache in every held layer, and it attends slots 0..positions[b].
 * On success every user's length advances by one.  A paged cache lends a page to
 * each user whose position starts one (KF_ENOMEM, nothing enqueued, if the pool
 * is short for the batch).
 */
kf_status kf_stage_decode(kf_stage* stage, kf_kv* kv, int32_t batch, const int32_t* users,
                          const int32_t* positions, const int32_t* tokens_dev, const void* hidden_in_dev,
                          void* hidden_out_dev, kf_dtype io);

/*
 * Forward a chunk of n_tokens consecutive tokens of one user starting at pos0 (prefill:
 * the prompt phase of a request, which the paper separates from decode in its
 * time-to-first-token accounting, Section VI; the per-user cache it fills is the
 * reservation of Section V-C).  pos0 must equal the user's length and pos0 + n_tokens <= max_ctx.  Token i attends
 * slots 0..pos0+i.  tokens_dev int32 [n] or hidden_in_dev [n, H]; hidden_out_dev [n, H].
 * A paged cache lends the pages up to pos0 + n (KF_ENOMEM if it cannot).
 * Dense products run on the matrix cores with fp16 operands (the stage's fp16 weights)
 * and fp32 accumulation.
 * On success the user's length advances by n_tokens.
 */
kf_status kf_stage_prefill(kf_stage* stage, kf_kv* kv, int32_t user, int32_t pos0, int32_t n_tokens,
                           const int32_t* tokens_dev, const void* hidden_in_dev, void* hidden_out_dev,
                           kf_dtype io);

/*
 * kf_stage_prefill without any device allocation, for callers that cannot allocate:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, checks, results and state changes as
 * kf_stage_prefill; the chunk's workspace (residual rows, normalised rows,
 * split-K partial sums, queries, attention output, SwiGLU output) lives in a static
 * per-device scratch array of KF_PREFILL_SCRATCH_BYTES instead of the stage's own
 * grown buffer.  A chunk whose workspace exceeds it is KF_ERANGE (nothing enqueued);
 * a 512-token chunk of every shape used here fits (the largest, hidden 8192 with
 * ffn 28672, needs 132 MiB).  All no-allocation prefills on one device share the
 * array: calls on one device whose work overlaps (other streams, other stages, other
 * threads) race, so the caller orders them.  No per-kernel timing is recorded.
 */
#define KF_PREFILL_SCRATCH_BYTES (144LL << 20)
kf_status kf_stage_prefill_noalloc(kf_stage* stage, kf_kv* kv, int32_t user, int32_t pos0, int32_t n_tokens,
                                   const int32_t* tokens_dev, const void* hidden_in_dev, void* hidden_out_dev,
                                   kf_dtype io);

/*
 * The head's unembedding (Section III and Fig. 1: the head member holds the
 * embedding and unembedding and samples after the model's last block):
 * logits_dev fp32 [rows, V] = RMSNorm(hidden; final gain) x LM_head^T, for hidden_dev
 * [rows, H] in dtype (KF_F32 or KF_BF16), any rows >= 1.  Head stages only (else KF_ESTATE).
 * hidden_dev NULL: the rows the stage's last kf_stage_decode kept (its hidden_out_dev
 * was NULL); rows must equal that decode's batch and dtype is ignored (else KF_ESTATE,
 * also when the last decode returned its rows or failed).
 */
kf_status kf_head_logits(kf_stage* stage, int32_t rows, const void* hidden_dev, kf_dtype dtype, float* logits_dev);

/*
 * The head's sampler: greedy decoding (Section VI-A decodes greedily at a fixed
 * seed).  token_dev int32 [rows] = argmax over the vocabulary of the logits of
 * kf_head_logits, the lowest index winning exact ties; max_logit_dev fp32 [rows]
 * (may be NULL) receives the winning logit.  A NaN logit is skipped and raises the
 * stage's NaN-logit error (KF_ERANGE from kf_stage_sync); a row whose logits are all
 * NaN gives token -1 and max logit NaN.  rows in [1, KF_MAX_BATCH] (else KF_EINVAL).
 * Head stages only (else KF_ESTATE).  hidden_dev NULL: the kept rows, as for kf_head_logits.
 */
kf_status kf_head_argmax(kf_stage* stage, int32_t rows, const void* hidden_dev, kf_dtype dtype,
                         int32_t* token_dev, float* max_logit_dev);

/*
 * Per-kernel timing (instrumentation).  The paper's sessions record predicted and
 * measured cost per stage (Section VI); this records, per kernel class, the HIP-event
 * time of every launch the stage enqueues while recording is on.
 *   kf_stage_profile(stage, mask) clears the records and starts recording the classes
 *   whose bit (1 << class) is set in mask; kf_stage_profile(stage, 0) stops recording
 *   (records are kept).  KF_K_ALL records every class.
 *   kf_stage_profile_read waits for the stage's stream, then returns the number of
 *   recorded launches of a class and their summed duration in milliseconds.
 * Each recorded launch is bracketed by two hipEventRecord calls on the stage's
 * stream, which adds a few microseconds per launch to the stream's timeline.
 */
typedef enum {
  KF_K_PREP = 0,       /* hidden/token input to the fp32 residual stream */
  KF_K_QKV = 1,        /* decode: RMSNorm + QKV GEMV + RoPE + KV append */
  KF_K_ATTN = 2,       /* decode: split-KV attention (partials per split) */
  KF_K_OPROJ = 3,      /* decode: merge of the partials + O GEMV + residual */
  KF_K_GATEUP = 4,     /* decode: RMSNorm + gate/up GEMV + SwiGLU */
  KF_K_DOWN = 5,       /* decode: down GEMV + residual */
  KF_K_LMHEAD = 6,     /* head: final RMSNorm + LM-head GEMV + partial argmax */
  KF_K_ARGMAX = 7,     /* head: final argmax reduction */
  KF_K_PF_NORM = 8,    /* prefill: row RMSNorm to fp16 */
  KF_K_PF_QKV = 9,     /* prefill: QKV GEMM (matrix cores) */
  KF_K_PF_ROPE = 10,   /* prefill: RoPE + KV append */
  KF_K_PF_ATTN = 11,   /* prefill: causal flash attention (matrix cores) */
  KF_K_PF_OPROJ = 12,  /* prefill: O GEMM + residual */
  KF_K_PF_GATEUP = 13, /* prefill: gate/up GEMM + SwiGLU */
  KF_K_PF_DOWN = 14,   /* prefill: down GEMM + residual */
  KF_K_PF_STORE = 15,  /* prefill: hidden output store */
  KF_K_QKNORM = 16,    /* kept for numbering: the decode per-head q/k RMSNorm + RoPE of qk_norm blocks
                          now runs inside the attention launch (KF_K_ATTN); nothing records here */
  KF_K_COUNT = 17
} kf_kernel_class;
#define KF_K_ALL 0x1ffff

kf_status kf_stage_profile(kf_stage* stage, int32_t mask);
kf_status kf_stage_profile_read(kf_stage* stage, int32_t kernel_class, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* KAFILA_STAGE_H */

/*
 * kafila_shard.h -- a stage's weights fetched by byte range from a checkpoint's
 * safetensors files (Kafila, arxiv 2609.34045, Section VI: each member fetches its
 * shard from the model host's safetensors files by byte range, so a member holding a
 * tenth of the model reads a tenth of it, and shards of one checkpoint share tensors,
 * so a replanned division re-reads little).
 *
 * A safetensors file is an 8-byte little-endian header length N, a JSON header of N
 * bytes mapping each tensor name to its dtype, shape and byte range [begin, end)
 * within the data that follows, then the data.  Opening a checkpoint reads only the
 * headers.  A fetch reads, with one positioned read per tensor, exactly the byte
 * ranges of the tensors a stage of layers [layer_lo, layer_hi) (plus the head) needs
 * and does not already hold; fetched tensors stay held by the checkpoint object
 * until released, which is what makes a replanned division cheap.
 *
 * Tensor names follow the Hugging Face layout of Llama and Qwen3 decoder models:
 *   model.layers.{l}.input_layernorm.weight            KF_W_ATTN_NORM  [H]
 *   model.layers.{l}.self_attn.{q,k,v,o}_proj.weight   KF_W_Q / K / V / O
 *   model.layers.{l}.self_attn.{q,k}_norm.weight       KF_W_Q_NORM / K_NORM [hd] (qk_norm configs)
 *   model.layers.{l}.post_attention_layernorm.weight   KF_W_MLP_NORM   [H]
 *   model.layers.{l}.mlp.{gate,up,down}_proj.weight    KF_W_GATE / UP / DOWN
 *   model.embed_tokens.weight                          KF_W_EMBED      [V, H]
 *   model.norm.weight                                  KF_W_FINAL_NORM [H]
 *   lm_head.weight                                     KF_W_LM_HEAD    [V, H]
 * with the shapes of kafila_stage.h.  Every tensor must be stored as BF16.
 *
 * Host-only except kf_shard_stage_init, which also creates the stage on the current
 * device.  A checkpoint object is not thread-safe.  Conventions as in kafila_stage.h.
 */
#ifndef KAFILA_SHARD_H
#define KAFILA_SHARD_H

#include <stdint.h>

#include "kafila_stage.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kf_shard kf_shard;

/* The LM head is the embedding matrix (checkpoints without lm_head.weight whose
 * configuration ties the two); without the flag a missing lm_head.weight is KF_EINVAL. */
#define KF_SHARD_TIED_EMBEDDINGS 1

/*
 * Open a checkpoint stored in n_paths (>= 1) safetensors files: reads and checks each
 * file's header (no tensor data).  KF_EINVAL for an unreadable or malformed file (a
 * header that is not the expected JSON, a byte range outside the file or inconsistent
 * with the dtype and shape, a tensor name found twice), with the file and the reason
 * in kf_last_error().
 */
kf_status kf_shard_open(const char* const* paths, int32_t n_paths, kf_shard** out);
kf_status kf_shard_close(kf_shard* shard);

/*
 * What a stage of layers [layer_lo, layer_hi) (plus the head if has_head) would fetch,
 * without reading anything:
 *   stage_bytes : bytes of all the stage's tensors (its share of the checkpoint)
 *   fetch_bytes : bytes of those not already held (what kf_shard_fetch would read)
 *   n_tensors   : tensors of the stage
 * Any output may be NULL.  KF_EINVAL if a tensor is missing or has another shape
 * (named in kf_last_error()), KF_EUNSUPPORTED if one is not BF16.
 */
kf_status kf_shard_plan(kf_shard* shard, const kf_model_config* cfg, int32_t layer_lo, int32_t layer_hi,
                        int32_t has_head, int32_t flags, int64_t* stage_bytes, int64_t* fetch_bytes,
                        int32_t* n_tensors);

/*
 * Read the stage's tensors that are not already held (one positioned read of each
 * tensor's byte range) and describe all of them in *weights: host bf16 pointers owned
 * by the checkpoint object, valid until the next fetch, release or close, laid out as
 * kf_stage_init takes them.  On failure nothing new is held.
 */
kf_status kf_shard_fetch(kf_shard* shard, const kf_model_config* cfg, int32_t layer_lo, int32_t layer_hi,
                         int32_t has_head, int32_t flags, kf_weights* weights);

/* Fetch, then kf_stage_init with the fetched weights (same meaning of every argument). */
kf_status kf_shard_stage_init(kf_shard* shard, const kf_model_config* cfg, int32_t layer_lo, int32_t layer_hi,
                              int32_t has_head, int32_t flags, void* hip_stream, kf_stage** out);

/* Drop the held tensors that a stage of layers [layer_lo, layer_hi) (plus the head if
 * has_head) does not use; layer_lo == layer_hi == 0 with has_head 0 drops everything. */
kf_status kf_shard_release(kf_shard* shard, int32_t layer_lo, int32_t layer_hi, int32_t has_head);

/* Tensor data bytes read from the files since the checkpoint was opened, and bytes held now. */
kf_status kf_shard_stats(const kf_shard* shard, int64_t* bytes_read, int64_t* bytes_held);

#ifdef __cplusplus
}
#endif
#endif /* KAFILA_SHARD_H */

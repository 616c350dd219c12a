/*
 * kafila_ring.h -- stages chained into a ring that serves several requests at once
 * (Kafila, arxiv 2609.34045: the session model of Section III and Fig. 1; concurrent
 * users, Section VII-C).
 *
 * The members of a session form a ring.  The head member embeds a token and runs its
 * block range first; the hidden state then passes through each member's range in turn
 * and the last member's output returns to the head, which unembeds and samples the
 * next token.  With one request in flight, a token occupies one member at a time and
 * the others wait; concurrent requests fill that bubble, each member working on one
 * request's token while another member works on the next request's.
 *
 * Here the members are stages (kafila_stage.h) on one device, each enqueuing on its
 * own stream.  The unit that moves around the ring is a request *group*: 1 to
 * KF_MAX_BATCH users that every member decodes together.  The hand-off between
 * consecutive members, and the return leg to the head, is a device buffer of the
 * group's hidden rows, ordered by an event recorded on the producer's stream and
 * waited for on the consumer's.  The head's sampled tokens stay on the device and
 * are the next step's input, so a whole generation is enqueued without a host round
 * trip.  Members on different devices (a peer hand-off) are not supported.
 *
 * Conventions are those of kafila_stage.h: "_dev" pointers are device pointers,
 * others host pointers; the caller owns every I/O buffer; calls enqueue and return;
 * argument checks run before anything is enqueued, and a call that fails them
 * changes no state.  A ring is not thread-safe.
 */
#ifndef KAFILA_RING_H
#define KAFILA_RING_H

#include <stdint.h>

#include "kafila_stage.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kf_ring kf_ring;

/*
 * Chain n_members (>= 1) stages and their KV caches into a ring.
 *   stages[0] holds the head and starts at layer 0; stages[i + 1] starts where
 *   stages[i] ends; the last stage ends at the model's last layer.  Every stage has
 *   the same config and device (KF_EUNSUPPORTED for stages on different devices).
 *   kvs[i] was created on stages[i]; all caches have the same max_users and max_ctx.
 *   Stages on distinct streams overlap; stages sharing a stream run in turn.
 *   max_groups (1..64): request groups one kf_ring_generate may carry.
 *   max_prefill (>= 1): tokens one kf_ring_prefill may carry.
 *   io: element type of the hand-off buffers, KF_F32 or KF_BF16.
 * The ring borrows the stages and caches (destroy the ring before them) and
 * allocates its hand-off buffers and events.  KF_ENOMEM if the device cannot.
 */
kf_status kf_ring_create(int32_t n_members, kf_stage* const* stages, kf_kv* const* kvs, int32_t max_groups,
                         int32_t max_prefill, kf_dtype io, kf_ring** out);

/* Waits for every member's stream, then frees the ring's buffers and events. */
kf_status kf_ring_destroy(kf_ring* ring);

/*
 * Prefill one user's prompt chunk through every member and sample the token that
 * follows it.
 *   n_tokens (1..max_prefill) token ids in tokens_dev (int32), at positions
 *   len .. len + n_tokens - 1, where len is the user's length (equal in every
 *   member, else KF_EINVAL; len + n_tokens <= max_ctx, else KF_ERANGE).
 *   next_token_dev int32 [1]: the greedy token after the chunk.
 * The user's length advances by n_tokens in every member.  A member with a paged
 * cache must have free pages for the chunk (KF_ENOMEM otherwise, nothing enqueued).
 */
kf_status kf_ring_prefill(kf_ring* ring, int32_t user, int32_t n_tokens, const int32_t* tokens_dev,
                          int32_t* next_token_dev);

/*
 * Generate `steps` (>= 1) tokens for each of n_groups (1..max_groups) request groups,
 * all in flight together.
 *   group_size[g] (host, 1..KF_MAX_BATCH): users in group g, listed group after group
 *     in `users` (host, U = sum of group sizes entries; distinct, < max_users).  A
 *     user's length must be equal in every member, and len + steps <= max_ctx
 *     (else KF_ERANGE).
 *   tokens_in_dev  int32 [U]: each user's next input token (the token at position len),
 *     ready when the call is made.
 *   tokens_out_dev int32 [steps, U]: row t receives the tokens sampled at step t, which
 *     are the inputs of step t + 1.
 *   hidden_out_dev [steps, U, H] in the ring's io type, or NULL: row (t, j) receives the
 *     hidden state user j's token of step t returned to the head with (the last member's
 *     output, from which the head sampled row (t, j) of tokens_out_dev).
 * Every user's length advances by `steps` in every member.  A member with a paged
 * cache must have free pages for every user's `steps` more positions, counted from
 * the user's length (KF_ENOMEM otherwise, nothing enqueued).  Work is enqueued in the
 * order in which each member meets the groups: step by step, group after group, so
 * member i takes group g's token while member i - 1 takes group g + 1's.  Everything
 * the call enqueues is ordered before the last work it puts on stages[0]'s stream.
 */
kf_status kf_ring_generate(kf_ring* ring, int32_t n_groups, const int32_t* group_size, const int32_t* users,
                           const int32_t* tokens_in_dev, int32_t steps, int32_t* tokens_out_dev,
                           void* hidden_out_dev);

/* Wait for every member's stream; KF_EDEVICE if any enqueued work failed. */
kf_status kf_ring_sync(kf_ring* ring);

#ifdef __cplusplus
}
#endif

#endif /* KAFILA_RING_H */

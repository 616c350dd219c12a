/*
 * kafila_planner.h -- the planner of Kafila (arxiv 2609.34045, Section V): the
 * stage-cost model, exact block placement, head placement by rotation,
 * admission, the two baseline divisions that open Section VII, and the device probes
 * that supply the cost model's measured terms.
 *
 * Members of a ring are numbered 0..m-1 in ring order; member `anchor` opened
 * the session.  A division gives member i n[i] consecutive blocks of the
 * model's chain of k blocks, the head's stage first: with member h as head the
 * chain runs h, h+1, ..., m-1, 0, ..., h-1 (a rotation of the ring order), and
 * every n[] array below is indexed by member in ring order.
 *
 * Units: seconds, bytes, bytes/s, flop/s.  All functions except the probes are
 * host-only, pure and thread-safe; failures set the thread-local message of
 * kf_last_error().
 */
#ifndef KAFILA_PLANNER_H
#define KAFILA_PLANNER_H

#include <stdint.h>

#include "kafila_stage.h"

#ifdef __cplusplus
extern "C" {
#endif

/* What a member reports about itself (Section V-A, V-D).  A term it could not
 * measure is marked: o < 0, bw <= 0, flops <= 0. */
typedef struct {
  double o;          /* fixed per-token dispatch overhead o_i (probe) */
  double bw;         /* measured memory bandwidth b_i (probe) */
  double flops;      /* reported arithmetic throughput (tier 2 only) */
  int64_t room;      /* device bytes the member offers the session */
} kf_member;

/* Model-side sizes behind eq. (2) and lim(i), at a declared context and concurrency. */
typedef struct {
  int64_t beta_block;     /* bytes one block reads per token (its weights) */
  int64_t beta_head;      /* bytes the head's matrices add (embedding + final gain + unembedding) */
  int64_t block_resident; /* device bytes one block holds: weights + its KV reservation */
  int64_t head_resident;  /* device bytes the head adds: its weights + its workspaces */
  int64_t stage_resident; /* device bytes any stage with at least one block holds besides its blocks */
  double flops_block;     /* flops one block performs per token at batch 1 (2 per weight) */
} kf_model_costs;

/*
 * The sizes of this library's stage (kf_stage_init + kf_kv_create) for a model
 * at max_users concurrent users of max_ctx tokens: for n >= 1 blocks,
 * stage_resident + n * block_resident (+ head_resident for the head) equals
 * kf_stage_bytes()'s `resident`.  KF_EINVAL for an invalid config.
 */
kf_status kf_stage_costs(const kf_model_config* cfg, int32_t max_users, int32_t max_ctx, kf_model_costs* out);

/* Eq. (2): c = o + n * beta_block / bw (+ beta_head / bw for the head).  NaN if bw <= 0. */
double kf_stage_cost(const kf_model_costs* costs, const kf_member* member, int32_t n, int32_t is_head);

/* lim(i) (Section V-C): whole blocks that fit in `room` after stage_resident and,
 * for the head, head_resident.  0 if not even those fit. */
int32_t kf_block_limit(const kf_model_costs* costs, int64_t room, int32_t is_head);

/*
 * Algorithm 1, Partition: the exact chain-on-chain division of k blocks over m
 * processors in the given order, processor i costing fixed[i] + n * per[i] for
 * n blocks, 1 <= n <= lim[i].  The bottleneck of any division is one of the
 * candidate values fixed[i] + n * per[i]; the smallest feasible one is found by
 * binary search over them, each test being the greedy left-to-right pass
 * Feasible.  Writes the counts n[0..m-1] and the bottleneck tau.
 * KF_ERANGE if no division exists; KF_EINVAL for k < 1, m < 1, a NULL pointer,
 * a negative or non-finite fixed[i], or per[i] <= 0.  Time O(k m log(k m)).
 */
kf_status kf_partition(int32_t k, int32_t m, const double* fixed, const double* per, const int32_t* lim,
                       int32_t* n, double* tau);

/*
 * Head placement (Section V-C): Partition once per rotation, member r as head
 * (its fixed term gains beta_head / bw and its limit loses head_resident);
 * rotations are tried from the anchor onwards and the earliest wins a tie.
 * The anchor stays head unless the best rotation's bottleneck is below
 * tau_anchor * (1 - mu); an infeasible anchor yields to the best feasible
 * rotation.  Needs every member's o >= 0 and bw > 0 (KF_EINVAL otherwise).
 * KF_ERANGE if no rotation has a division.
 */
kf_status kf_place_head(int32_t k, int32_t m, const kf_member* members, const kf_model_costs* costs,
                        int32_t anchor, double mu, int32_t* head, int32_t* n, double* tau);

/* The baselines that open Section VII.  Uniform: k / m blocks each, one more for the first k % m
 * members.  Memory-proportional: the boundary after member i (ring order from
 * member 0) at floor(k * (room_0 + .. + room_i) / (total room) + 1/2); a member
 * may get 0 blocks.  KF_EINVAL for k < 1, m < 1, NULL, a negative room or a zero total. */
kf_status kf_divide_uniform(int32_t k, int32_t m, int32_t* n);
kf_status kf_divide_memory(int32_t k, int32_t m, const int64_t* room, int32_t* n);

/*
 * Admission (Section V-D): checks a division against every member's room.  A
 * member with blocks, and the head, hold stage_resident + n * block_resident
 * (+ head_resident for the head); any other member holds nothing.
 * *culprit = the first member in ring order that overflows, or -1.
 */
kf_status kf_admit(int32_t m, const int32_t* n, int32_t head, const kf_member* members, const kf_model_costs* costs,
                   int32_t* culprit);

typedef struct {
  int32_t tier;     /* 1: full cost model; 2: arithmetic throughput; 3: working set */
  int32_t head;     /* member holding the head */
  int32_t admitted; /* 1 if the division fits every member */
  int32_t culprit;  /* when not admitted: the member named, or -1 for a collective shortfall */
  double tau;       /* predicted bottleneck (tier 1: seconds by eq. (2); tier 2: block flops / flop rate; tier 3: NaN) */
} kf_plan_info;

/*
 * The planner of Sections V-C and V-D.  Tier 1 when every member has o >= 0
 * and bw > 0: kf_place_head.  Else tier 2 when every member reported flops > 0:
 * Partition with fixed = 0 and per = flops_block / flops, head at the anchor.
 * Else tier 3: memory-proportional by room, counted from the anchor, head at
 * the anchor.  Then admission.  When tier 1 or 2 finds no division, n is all
 * zero, admitted = 0 and culprit names the first member that cannot hold even
 * one block (tier 1: as a non-head member; tier 2: with the anchor as head),
 * else -1.  Returns KF_OK whether or not the plan is admitted.
 */
kf_status kf_plan(int32_t k, int32_t m, const kf_member* members, const kf_model_costs* costs, int32_t anchor,
                  double mu, int32_t* n, kf_plan_info* info);

/*
 * Device probes (Section V-A: every term is measured before a weight loads).
 * Both run on the current HIP device, enqueue on hip_stream (NULL: default),
 * synchronise, and report the median over `reps` timed runs after one untimed
 * run.
 *   kf_probe_bandwidth: reads a `bytes`-byte device buffer (allocated and freed
 *     inside the call; at least 64 MiB, a multiple of 64 KiB) with 16-byte
 *     non-temporal loads from >= 2048 workgroups; *bw = bytes / time.
 *   kf_probe_overhead: o_i, the time of one empty dependent kernel on the
 *     stream (launch + dispatch + completion), from a chain of 256 such kernels.
 * KF_EINVAL for bad sizes or reps < 1, KF_ENOMEM, KF_EDEVICE.
 */
kf_status kf_probe_bandwidth(void* hip_stream, int64_t bytes, int32_t reps, double* bw);
kf_status kf_probe_overhead(void* hip_stream, int32_t reps, double* o);

#ifdef __cplusplus
}
#endif

#endif /* KAFILA_PLANNER_H */

// The planner behind include/kafila_planner.h (paper Section V): eq. (2), the
// exact chain-on-chain division of Algorithm 1, head placement by rotation,
// the admission tiers and the baselines that open Section VII.  Host-only.
#include <algorithm>
#include <cmath>
#include <vector>

#include "error.h"
#include "kafila_planner.h"

// Every stage cost is the same expression fixed + n * per, evaluated once when
// the candidate set is built and again inside Feasible; a fused multiply-add in
// one place and not the other would let a candidate fail its own test.
#pragma clang fp contract(off)

using kf::fail;

namespace {

double block_cost(double fixed, int n, double per) { return fixed + (double)n * per; }

// Largest n in [0, cap] with fixed + n * per <= tau (per > 0).  The quotient is
// only a starting point: the answer is settled on the cost expression itself.
int blocks_within(double fixed, double per, double tau, int cap) {
  if (fixed > tau) return 0;
  double q = std::floor((tau - fixed) / per);
  int n = q < 0 ? 0 : q > cap ? cap : (int)q;
  while (n < cap && block_cost(fixed, n + 1, per) <= tau) ++n;
  while (n > 0 && block_cost(fixed, n, per) > tau) --n;
  return n;
}

// Feasible(k, tau): one left-to-right pass giving each processor the most blocks
// it can take within tau, its limit, and one block kept for each processor after it.
bool feasible(int k, int m, const double* fixed, const double* per, const int* lim, double tau, int* n) {
  int left = k;
  for (int i = 0; i < m; ++i) {
    if (fixed[i] > tau) return false;
    int c = blocks_within(fixed[i], per[i], tau, k);
    c = std::min(c, lim[i]);
    c = std::min(c, left - (m - 1 - i));
    if (c < 1) return false;
    n[i] = c;
    left -= c;
  }
  return left == 0;
}

kf_status check_costs(const kf_model_costs* c) {
  if (!c) return fail(KF_EINVAL, "costs is NULL");
  if (c->beta_block <= 0 || c->beta_head < 0 || c->block_resident <= 0 || c->head_resident < 0 ||
      c->stage_resident < 0)
    return fail(KF_EINVAL, "model costs must be positive (beta_block, block_resident) or non-negative");
  return KF_OK;
}

int limit_of(const kf_model_costs& c, int64_t room, bool head) {
  const int64_t free = room - c.stage_resident - (head ? c.head_resident : 0);
  if (free < 0) return 0;
  const int64_t n = free / c.block_resident;
  return n > INT32_MAX ? INT32_MAX : (int)n;
}

// Partition with status codes but without touching the error message on infeasibility.
kf_status partition(int k, int m, const double* fixed, const double* per, const int* lim, int* n, double* tau) {
  std::vector<double> cand;
  for (int i = 0; i < m; ++i) {
    const int top = std::min(k, lim[i]);
    for (int c = 1; c <= top; ++c) cand.push_back(block_cost(fixed[i], c, per[i]));
  }
  if (cand.empty()) return KF_ERANGE;
  std::sort(cand.begin(), cand.end());
  std::vector<int> work(m);
  if (!feasible(k, m, fixed, per, lim, cand.back(), work.data())) return KF_ERANGE;
  size_t lo = 0, hi = cand.size() - 1;  // feasible at hi; find the first feasible index
  while (lo < hi) {
    const size_t mid = lo + (hi - lo) / 2;
    if (feasible(k, m, fixed, per, lim, cand[mid], work.data())) hi = mid;
    else lo = mid + 1;
  }
  feasible(k, m, fixed, per, lim, cand[lo], n);
  *tau = cand[lo];
  return KF_OK;
}

// Tier-1 terms of member j with member `head` as head.
void tier1_terms(const kf_member& d, const kf_model_costs& c, bool head, double* fixed, double* per, int* lim) {
  *fixed = d.o + (head ? (double)c.beta_head / d.bw : 0.0);
  *per = (double)c.beta_block / d.bw;
  *lim = limit_of(c, d.room, head);
}

// Rotation search of Section V-C.  Returns KF_ERANGE when no rotation has a division.
kf_status place_head(int k, int m, const kf_member* d, const kf_model_costs& c, int anchor, double mu, int* head,
                     int* n, double* tau) {
  std::vector<double> fixed(m), per(m);
  std::vector<int> lim(m), nr(m);
  int best_r = -1;
  double best_tau = 0, anchor_tau = 0;
  bool anchor_ok = false;
  std::vector<int> best_n(m), anchor_n(m);
  for (int step = 0; step < m; ++step) {
    const int r = (anchor + step) % m;
    for (int j = 0; j < m; ++j) tier1_terms(d[(r + j) % m], c, j == 0, &fixed[j], &per[j], &lim[j]);
    double t;
    if (partition(k, m, fixed.data(), per.data(), lim.data(), nr.data(), &t) != KF_OK) continue;
    if (step == 0) {
      anchor_ok = true;
      anchor_tau = t;
      for (int j = 0; j < m; ++j) anchor_n[(r + j) % m] = nr[j];
    }
    if (best_r < 0 || t < best_tau) {
      best_r = r;
      best_tau = t;
      for (int j = 0; j < m; ++j) best_n[(r + j) % m] = nr[j];
    }
  }
  if (best_r < 0) return KF_ERANGE;
  if (anchor_ok && !(best_tau < anchor_tau * (1.0 - mu))) {
    *head = anchor;
    *tau = anchor_tau;
    std::copy(anchor_n.begin(), anchor_n.end(), n);
  } else {
    *head = best_r;
    *tau = best_tau;
    std::copy(best_n.begin(), best_n.end(), n);
  }
  return KF_OK;
}

void memory_split(int k, int m, const int64_t* room, int* n) {
  int64_t total = 0;
  for (int i = 0; i < m; ++i) total += room[i];
  int64_t run = 0;
  int prev = 0;
  for (int i = 0; i < m; ++i) {
    run += room[i];
    const int b = (int)std::floor((double)k * ((double)run / (double)total) + 0.5);
    n[i] = b - prev;
    prev = b;
  }
}

int admit(int m, const int* n, int head, const kf_member* d, const kf_model_costs& c) {
  for (int i = 0; i < m; ++i) {
    if (n[i] == 0 && i != head) continue;
    const int64_t need = c.stage_resident + (int64_t)n[i] * c.block_resident + (i == head ? c.head_resident : 0);
    if (need > d[i].room) return i;
  }
  return -1;
}

}  // namespace

extern "C" {

double kf_stage_cost(const kf_model_costs* costs, const kf_member* member, int32_t n, int32_t is_head) {
  if (!costs || !member || !(member->bw > 0)) return NAN;
  double c = member->o + block_cost(0.0, n, (double)costs->beta_block / member->bw);
  if (is_head) c += (double)costs->beta_head / member->bw;
  return c;
}

int32_t kf_block_limit(const kf_model_costs* costs, int64_t room, int32_t is_head) {
  if (!costs || costs->block_resident <= 0) return 0;
  return limit_of(*costs, room, is_head != 0);
}

kf_status kf_partition(int32_t k, int32_t m, const double* fixed, const double* per, const int32_t* lim, int32_t* n,
                       double* tau) {
  if (k < 1 || m < 1) return fail(KF_EINVAL, "k and m must be >= 1 (k=%d, m=%d)", k, m);
  if (!fixed || !per || !lim || !n || !tau) return fail(KF_EINVAL, "NULL argument");
  for (int i = 0; i < m; ++i) {
    if (!std::isfinite(fixed[i]) || fixed[i] < 0) return fail(KF_EINVAL, "fixed[%d] must be finite and >= 0", i);
    if (!std::isfinite(per[i]) || !(per[i] > 0)) return fail(KF_EINVAL, "per[%d] must be finite and > 0", i);
  }
  const kf_status st = partition(k, m, fixed, per, lim, n, tau);
  if (st == KF_ERANGE) return fail(KF_ERANGE, "no division of %d blocks over %d processors within the limits", k, m);
  return st;
}

kf_status kf_place_head(int32_t k, int32_t m, const kf_member* members, const kf_model_costs* costs, int32_t anchor,
                        double mu, int32_t* head, int32_t* n, double* tau) {
  if (k < 1 || m < 1) return fail(KF_EINVAL, "k and m must be >= 1 (k=%d, m=%d)", k, m);
  if (!members || !head || !n || !tau) return fail(KF_EINVAL, "NULL argument");
  if (anchor < 0 || anchor >= m) return fail(KF_EINVAL, "anchor %d outside [0, %d)", anchor, m);
  if (!(mu >= 0 && mu < 1)) return fail(KF_EINVAL, "mu must be in [0, 1)");
  kf_status st = check_costs(costs);
  if (st != KF_OK) return st;
  for (int i = 0; i < m; ++i)
    if (!(members[i].o >= 0) || !(members[i].bw > 0) || !std::isfinite(members[i].o))
      return fail(KF_EINVAL, "member %d lacks a measured overhead or bandwidth", i);
  st = place_head(k, m, members, *costs, anchor, mu, head, n, tau);
  if (st == KF_ERANGE) return fail(KF_ERANGE, "no rotation divides %d blocks within the members' limits", k);
  return st;
}

kf_status kf_divide_uniform(int32_t k, int32_t m, int32_t* n) {
  if (k < 1 || m < 1 || !n) return fail(KF_EINVAL, "k, m must be >= 1 and n non-NULL");
  for (int i = 0; i < m; ++i) n[i] = k / m + (i < k % m ? 1 : 0);
  return KF_OK;
}

kf_status kf_divide_memory(int32_t k, int32_t m, const int64_t* room, int32_t* n) {
  if (k < 1 || m < 1 || !room || !n) return fail(KF_EINVAL, "k, m must be >= 1 and pointers non-NULL");
  int64_t total = 0;
  for (int i = 0; i < m; ++i) {
    if (room[i] < 0) return fail(KF_EINVAL, "room[%d] is negative", i);
    total += room[i];
  }
  if (total == 0) return fail(KF_EINVAL, "total room is zero");
  memory_split(k, m, room, n);
  return KF_OK;
}

kf_status kf_admit(int32_t m, const int32_t* n, int32_t head, const kf_member* members, const kf_model_costs* costs,
                   int32_t* culprit) {
  if (m < 1 || !n || !members || !culprit) return fail(KF_EINVAL, "m must be >= 1 and pointers non-NULL");
  if (head < 0 || head >= m) return fail(KF_EINVAL, "head %d outside [0, %d)", head, m);
  const kf_status st = check_costs(costs);
  if (st != KF_OK) return st;
  for (int i = 0; i < m; ++i)
    if (n[i] < 0) return fail(KF_EINVAL, "n[%d] is negative", i);
  *culprit = admit(m, n, head, members, *costs);
  return KF_OK;
}

kf_status kf_plan(int32_t k, int32_t m, const kf_member* members, const kf_model_costs* costs, int32_t anchor,
                  double mu, int32_t* n, kf_plan_info* info) {
  if (k < 1 || m < 1) return fail(KF_EINVAL, "k and m must be >= 1 (k=%d, m=%d)", k, m);
  if (!members || !n || !info) return fail(KF_EINVAL, "NULL argument");
  if (anchor < 0 || anchor >= m) return fail(KF_EINVAL, "anchor %d outside [0, %d)", anchor, m);
  if (!(mu >= 0 && mu < 1)) return fail(KF_EINVAL, "mu must be in [0, 1)");
  const kf_status st = check_costs(costs);
  if (st != KF_OK) return st;
  const kf_model_costs& c = *costs;

  bool all_priced = true, all_flops = true;
  for (int i = 0; i < m; ++i) {
    all_priced = all_priced && members[i].o >= 0 && std::isfinite(members[i].o) && members[i].bw > 0;
    all_flops = all_flops && members[i].flops > 0;
  }
  *info = kf_plan_info{0, anchor, 0, -1, NAN};
  std::fill(n, n + m, 0);

  auto refuse = [&](int tier, bool anchor_is_head) {
    info->tier = tier;
    info->head = anchor;
    info->admitted = 0;
    info->culprit = -1;
    for (int i = 0; i < m; ++i)
      if (limit_of(c, members[i].room, anchor_is_head && i == anchor) < 1) {
        info->culprit = i;
        break;
      }
    std::fill(n, n + m, 0);
    return KF_OK;
  };

  if (all_priced) {
    int head;
    double tau;
    if (place_head(k, m, members, c, anchor, mu, &head, n, &tau) != KF_OK) return refuse(1, false);
    info->tier = 1;
    info->head = head;
    info->tau = tau;
  } else if (all_flops) {
    std::vector<double> fixed(m, 0.0), per(m);
    std::vector<int> lim(m), nr(m);
    for (int j = 0; j < m; ++j) {
      const int i = (anchor + j) % m;
      per[j] = c.flops_block / members[i].flops;
      lim[j] = limit_of(c, members[i].room, j == 0);
    }
    double tau;
    if (partition(k, m, fixed.data(), per.data(), lim.data(), nr.data(), &tau) != KF_OK) return refuse(2, true);
    for (int j = 0; j < m; ++j) n[(anchor + j) % m] = nr[j];
    info->tier = 2;
    info->head = anchor;
    info->tau = tau;
  } else {
    std::vector<int64_t> room(m);
    std::vector<int> nr(m);
    for (int j = 0; j < m; ++j) room[j] = members[(anchor + j) % m].room;
    int64_t total = 0;
    for (int j = 0; j < m; ++j) total += room[j] > 0 ? room[j] : 0;
    if (total <= 0) return fail(KF_EINVAL, "no member offers any room");
    for (int j = 0; j < m; ++j) room[j] = room[j] > 0 ? room[j] : 0;
    memory_split(k, m, room.data(), nr.data());
    for (int j = 0; j < m; ++j) n[(anchor + j) % m] = nr[j];
    info->tier = 3;
    info->head = anchor;
  }
  info->culprit = admit(m, n, info->head, members, c);
  info->admitted = info->culprit < 0;
  return KF_OK;
}

}  // extern "C"

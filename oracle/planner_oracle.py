"""Plain CPU oracle of the planner's block placement (test infrastructure only).

The planner of the paper (Section V) prices each member's stage with the cost
model of eq. (2), divides the model's chain of k blocks across the m members
of a ring in a fixed order so that the slowest stage is as fast as possible
(Section V-C, the chain-on-chain problem that Algorithm 1 solves exactly),
tries each member as the head by rotating the order and keeps the session's
anchor unless another choice is better by a margin mu (Section V-C), degrades
through three tiers of information and finally admits or rejects the division
against every member's memory (Section V-D).  The baselines that open Section VII divide
evenly (Uniform) or by working set (Memory-proportional).

This module writes each of those out in the most direct way:

* ``stage_cost`` is eq. (2) term by term.
* ``best_division`` reaches the optimum the exact algorithm reaches by its
  plain definition: it enumerates every composition of k into m parts within
  the block limits and keeps the smallest bottleneck.  It does not implement
  Algorithm 1 (no candidate set, no binary search, no greedy pass), so the
  native planner is checked against the optimum itself.  Exponential in m;
  small k and m only.
* Head placement, tiers, admission and the two baselines follow the paper's
  description step by step.

Readings of points the paper leaves open (each also listed with the design
notes):

* lim(i): the whole number of blocks that fit in the member's room after the
  bytes every stage holds regardless of its blocks and, for the head, the
  head's bytes; one block costs its weights plus its KV reservation at the
  declared context and concurrency.
* Rotation r makes device r the head and the first stage of the chain; ties in
  achieved bottleneck go to the earliest rotation counted from the anchor.
* Tier 2 (arithmetic throughput only): fixed(i) = 0 and per(i) = flops of one
  block / the member's flop rate; the head stays at the anchor.
* Tier 3 and the memory-proportional baseline: cumulative rounding, the
  boundary after member i sits at floor(k * (sum of rooms so far) / (total
  room) + 1/2); a member may receive no block.
* Uniform: k // m blocks each, one more for the first k % m members.
* Admission: a member with no block and no head holds nothing; otherwise it
  holds the per-stage bytes, its blocks' bytes and, as head, the head's bytes.
  The first member in ring order that overflows is named; when the cost model
  finds no feasible division in any rotation and no single member is short of
  one block, the shortfall is collective (culprit -1).

Pins (``tests/test_planner_oracle.py``): closed forms for identical members,
one member, two members; exhaustive cross-checks of the optimum against a
separately written recursion; invariants (monotone in the limits, permutation
behaviour of the rotation rule).  Only the tests may import this module.
"""
from __future__ import annotations

import itertools
import math

INF = float("inf")


def stage_cost(o: float, n: int, beta_block: float, beta_head: float, bw: float, is_head: bool) -> float:
    """Eq. (2): fixed overhead plus n blocks' bytes, plus the head's bytes on the head, over bandwidth."""
    c = o + n * (beta_block / bw)
    if is_head:
        c += beta_head / bw
    return c


def block_limit(room: int, block_resident: int, stage_resident: int, head_resident: int, is_head: bool) -> int:
    """lim(i) at the declared context and concurrency (Section V-C); never negative."""
    free = room - stage_resident - (head_resident if is_head else 0)
    if free < 0 or block_resident <= 0:
        return 0
    return free // block_resident


def compositions(k: int, m: int):
    """Every (n_1..n_m) of positive integers summing to k."""
    for cuts in itertools.combinations(range(1, k), m - 1):
        bounds = (0,) + cuts + (k,)
        yield tuple(bounds[i + 1] - bounds[i] for i in range(m))


def best_division(k: int, fixed, per, lim):
    """Smallest bottleneck over all contiguous divisions with 1 <= n_i <= lim_i.

    Returns (tau, divisions) where divisions lists every optimal division, or
    (None, []) when no division exists.  A stage of n blocks on member i costs
    fixed[i] + n * per[i].
    """
    m = len(fixed)
    best, arg = None, []
    for n in compositions(k, m):
        if any(n[i] > lim[i] for i in range(m)):
            continue
        tau = max(fixed[i] + n[i] * per[i] for i in range(m))
        if best is None or tau < best:
            best, arg = tau, [n]
        elif tau == best:
            arg.append(n)
    return best, arg


def rotate(seq, r: int):
    return list(seq[r:]) + list(seq[:r])


def unrotate(seq, r: int):
    m = len(seq)
    out = [None] * m
    for j, v in enumerate(seq):
        out[(j + r) % m] = v
    return out


def tier1_terms(devices, costs, head: int):
    """(fixed, per, lim) per member in original order with member `head` as the head (Section V-C)."""
    fixed, per, lim = [], [], []
    for i, d in enumerate(devices):
        h = i == head
        fixed.append(stage_cost(d["o"], 0, costs["beta_block"], costs["beta_head"], d["bw"], h))
        per.append(costs["beta_block"] / d["bw"])
        lim.append(block_limit(d["room"], costs["block_resident"], costs["stage_resident"], costs["head_resident"], h))
    return fixed, per, lim


def place_head(k: int, devices, costs, anchor: int, mu: float):
    """Rotation search of Section V-C on top of the exact division.

    Each rotation r (r = anchor, anchor+1, ... around the ring) puts member r
    first as the head; its best division is found by enumeration.  The anchor
    is kept unless the best rotation's bottleneck is below tau_anchor * (1 - mu);
    an infeasible anchor yields to the best feasible rotation.

    Returns (head, n in original order, tau) or (None, None, None).
    """
    m = len(devices)
    results = []
    for step in range(m):
        r = (anchor + step) % m
        fixed, per, lim = tier1_terms(devices, costs, r)
        tau, divs = best_division(k, rotate(fixed, r), rotate(per, r), rotate(lim, r))
        results.append((r, tau, divs))
    feasible = [(r, tau, divs) for r, tau, divs in results if tau is not None]
    if not feasible:
        return None, None, None
    best = min(feasible, key=lambda t: t[1])  # earliest rotation on ties
    anchor_tau = results[0][1]
    if anchor_tau is not None and not best[1] < anchor_tau * (1.0 - mu):
        r, tau, divs = results[0]
    else:
        r, tau, divs = best
    return r, [unrotate(list(d), r) for d in divs], tau


def uniform(k: int, m: int):
    """The Uniform baseline of Section VII's opening (GPipe's equal block count)."""
    return [k // m + (1 if i < k % m else 0) for i in range(m)]


def memory_proportional(k: int, rooms):
    """The Memory-proportional baseline of Section VII's opening: shares proportional to working set."""
    total = 0
    for r in rooms:
        total += r
    out, prev, run = [], 0, 0
    for r in rooms:
        run += r
        b = int(math.floor(k * (run / total) + 0.5))
        out.append(b - prev)
        prev = b
    return out


def admit(n, head: int, devices, costs):
    """Section V-D admission: the first member (ring order) whose assignment exceeds its room, else None."""
    for i, d in enumerate(devices):
        if n[i] == 0 and i != head:
            continue
        need = costs["stage_resident"] + n[i] * costs["block_resident"] + (costs["head_resident"] if i == head else 0)
        if need > d["room"]:
            return i
    return None


def plan(k: int, devices, costs, anchor: int, mu: float):
    """Section V-D: the best-informed tier the members' measurements allow, then admission.

    Returns a dict with tier, head, n (one optimal division; ``divisions`` holds
    all of them for tier 1 and 2), tau (None for tier 3), culprit (None when
    admitted; -1 for a collective shortfall).
    """
    m = len(devices)
    if all(d["bw"] > 0 and d["o"] >= 0 for d in devices):
        head, divs, tau = place_head(k, devices, costs, anchor, mu)
        if head is None:
            lims = tier1_terms(devices, costs, -1)[2]
            short = [i for i in range(m) if lims[i] < 1]
            return dict(tier=1, head=anchor, n=None, divisions=[], tau=None, culprit=short[0] if short else -1)
        culprit = admit(divs[0], head, devices, costs)
        return dict(tier=1, head=head, n=divs[0], divisions=divs, tau=tau, culprit=culprit)
    if all(d["flops"] > 0 for d in devices):
        per = [costs["flops_block"] / d["flops"] for d in devices]
        fixed = [0.0] * m
        lim = [block_limit(d["room"], costs["block_resident"], costs["stage_resident"], costs["head_resident"],
                           i == anchor) for i, d in enumerate(devices)]
        tau, divs = best_division(k, rotate(fixed, anchor), rotate(per, anchor), rotate(lim, anchor))
        if tau is None:
            short = [i for i in range(m) if lim[i] < 1]
            return dict(tier=2, head=anchor, n=None, divisions=[], tau=None, culprit=short[0] if short else -1)
        divs = [unrotate(list(d), anchor) for d in divs]
        return dict(tier=2, head=anchor, n=divs[0], divisions=divs, tau=tau,
                    culprit=admit(divs[0], anchor, devices, costs))
    n = unrotate(memory_proportional(k, rotate([d["room"] for d in devices], anchor)), anchor)
    return dict(tier=3, head=anchor, n=n, divisions=[n], tau=None, culprit=admit(n, anchor, devices, costs))


def bottleneck_stats(costs_per_stage):
    """The columns of Section VII-B's table: imbalance (max/min), bottleneck, utilisation (mean/max)."""
    hi, lo = max(costs_per_stage), min(costs_per_stage)
    mean = sum(costs_per_stage) / len(costs_per_stage)
    return dict(imbalance=hi / lo, bottleneck=hi, utilisation=mean / hi)

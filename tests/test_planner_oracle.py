"""Pins of the planner oracle against closed forms, invariants and an independent recursion.

Each pin is chosen so that a plausible slip in the oracle fails it: a dropped
or sign-flipped term of eq. (2), a limit applied to the wrong member, an
off-by-one in the enumeration, a rotation that is not undone, a margin applied
the wrong way round, a rounding that loses or adds a block.
"""
import math
import random

import pytest

from oracle import planner_oracle as po


# ---------------------------------------------------------------- eq. (2)
def test_stage_cost_terms_separate():
    """c(n) is affine in n with slope beta_block / bw; the head adds beta_head / bw; c(0) = o."""
    o, bb, bh, bw = 3.5e-6, 436_224_000, 1_050_673_152 * 2, 7.1e12
    c = [po.stage_cost(o, n, bb, bh, bw, False) for n in range(6)]
    assert c[0] == o
    for a, b in zip(c, c[1:]):
        assert b - a == pytest.approx(bb / bw, rel=1e-12)
    for n in range(6):
        assert po.stage_cost(o, n, bb, bh, bw, True) - c[n] == pytest.approx(bh / bw, rel=1e-12)
    # doubling the bandwidth halves every byte term and leaves o alone
    assert po.stage_cost(o, 4, bb, bh, 2 * bw, True) - o == pytest.approx((po.stage_cost(o, 4, bb, bh, bw, True) - o) / 2)


def test_block_limit_counts_whole_blocks():
    # room for exactly 7 blocks after the stage bytes; the head's bytes take 2 of them
    assert po.block_limit(100 + 7 * 30, 30, 100, 60, False) == 7
    assert po.block_limit(100 + 7 * 30, 30, 100, 60, True) == 5
    assert po.block_limit(100 + 7 * 30 - 1, 30, 100, 60, False) == 6
    assert po.block_limit(50, 30, 100, 60, False) == 0  # not even the stage bytes fit


# ---------------------------------------------------------------- exact division
def minimax_recursion(k, fixed, per, lim):
    """Independent check: best[j] over prefixes of members by dynamic programming (not enumeration)."""
    m = len(fixed)
    best = {0: 0.0}  # blocks placed on members so far -> smallest bottleneck so far
    for i in range(m):
        nxt = {}
        for placed, bott in best.items():
            for n in range(1, lim[i] + 1):
                if placed + n > k:
                    break
                v = max(bott, fixed[i] + n * per[i])
                if v < nxt.get(placed + n, math.inf):
                    nxt[placed + n] = v
        best = nxt
    return best.get(k)


def test_identical_members_closed_form():
    for k in range(1, 13):
        for m in range(1, min(k, 5) + 1):
            tau, divs = po.best_division(k, [2.0] * m, [0.5] * m, [k] * m)
            assert tau == 2.0 + math.ceil(k / m) * 0.5
            for d in divs:
                assert sum(d) == k and max(d) == math.ceil(k / m)


def test_one_member():
    assert po.best_division(5, [1.0], [2.0], [5]) == (11.0, [(5,)])
    assert po.best_division(5, [1.0], [2.0], [4]) == (None, [])


def test_two_members_by_hand():
    # member 0 is three times faster per block; k = 8: (6, 2) costs max(0+6, 1+2*3) = 7 and (7, 1)
    # costs max(7, 4) = 7; (5, 3) costs 10 and (8, 0) is not a division
    tau, divs = po.best_division(8, [0.0, 1.0], [1.0, 3.0], [8, 8])
    assert tau == 7.0 and divs == [(6, 2), (7, 1)]
    # a limit of 5 on member 0 forces (5, 3): max(5, 10) = 10
    tau, divs = po.best_division(8, [0.0, 1.0], [1.0, 3.0], [5, 8])
    assert tau == 10.0 and divs == [(5, 3)]


def test_infeasible_when_limits_are_short():
    assert po.best_division(6, [0.0] * 3, [1.0] * 3, [2, 2, 1])[0] is None
    assert po.best_division(6, [0.0] * 3, [1.0] * 3, [4, 0, 4])[0] is None
    assert po.best_division(2, [0.0] * 3, [1.0] * 3, [4, 4, 4])[0] is None  # fewer blocks than members


@pytest.mark.parametrize("seed", range(40))
def test_enumeration_matches_recursion(seed):
    rng = random.Random(seed)
    m = rng.randint(1, 5)
    k = rng.randint(m, 12)
    fixed = [rng.uniform(0, 3) for _ in range(m)]
    per = [rng.uniform(0.2, 4) for _ in range(m)]
    lim = [rng.randint(0, k) for _ in range(m)]
    tau, divs = po.best_division(k, fixed, per, lim)
    assert tau == minimax_recursion(k, fixed, per, lim)
    for d in divs:
        assert sum(d) == k and all(1 <= d[i] <= lim[i] for i in range(m))
        assert max(fixed[i] + d[i] * per[i] for i in range(m)) == tau


@pytest.mark.parametrize("seed", range(20))
def test_monotone_in_limits_and_blocks(seed):
    rng = random.Random(100 + seed)
    m = rng.randint(2, 4)
    k = rng.randint(m, 10)
    fixed = [rng.uniform(0, 2) for _ in range(m)]
    per = [rng.uniform(0.5, 3) for _ in range(m)]
    lim = [rng.randint(1, k) for _ in range(m)]
    tau = po.best_division(k, fixed, per, lim)[0]
    looser = list(lim)
    looser[rng.randrange(m)] += 1
    tau2 = po.best_division(k, fixed, per, looser)[0]
    if tau is not None:
        assert tau2 is not None and tau2 <= tau
    more = po.best_division(k + 1, fixed, per, [k + 1] * m)[0]
    assert more >= po.best_division(k, fixed, per, [k] * m)[0]


# ---------------------------------------------------------------- head rotation
COSTS = dict(beta_block=100.0, beta_head=300.0, block_resident=10, stage_resident=0, head_resident=0,
             flops_block=200.0)


def dev(o, bw, room=10**9, flops=1.0):
    return dict(o=o, bw=bw, room=room, flops=flops)


def test_head_moves_to_the_fast_member_beyond_the_margin():
    # two members, two blocks: one each.  Head on member 0 (bw 100): max(0+1+3, 0+1) = 4.
    # Head on member 1 (bw 400): max(0+1, 0+0.25+0.75) = 1: far better than 4 * 0.95.
    devs = [dev(0.0, 100.0), dev(0.0, 400.0)]
    head, divs, tau = po.place_head(2, devs, COSTS, anchor=0, mu=0.05)
    assert head == 1 and tau == 1.0 and divs == [[1, 1]]


def test_margin_keeps_the_anchor():
    # two blocks, one each.  Anchor (o = 0.16) as head: max(0.16 + 3 + 1, 0 + 1) = 4.16; member 1 as
    # head: max(0 + 3 + 1, 0.16 + 1) = 4, a 3.8 % gain: kept at mu = 0.05, taken at mu = 0.03
    devs = [dev(0.16, 100.0), dev(0.0, 100.0)]
    head, _, tau = po.place_head(2, devs, COSTS, anchor=0, mu=0.05)
    assert head == 0 and tau == pytest.approx(4.16)
    head, _, tau = po.place_head(2, devs, COSTS, anchor=0, mu=0.03)  # 4 < 4.16 * 0.97 = 4.035
    assert head == 1 and tau == pytest.approx(4.0)


def test_rotation_round_trip():
    for m in range(1, 7):
        seq = list(range(10, 10 + m))
        for r in range(m):
            assert po.rotate(seq, r)[0] == seq[r]
            assert po.unrotate(po.rotate(seq, r), r) == seq


def test_head_division_returned_in_original_order():
    # member 2 (bw 400) as head, chain [2, 0, 1]: (2, 1, 1) costs max(0.75 + 0.5, 1, 1) = 1.25, the unique
    # optimum; the anchor as head costs at least 3 + 1.  In the original order the division is [1, 1, 2].
    devs = [dev(0.0, 100.0), dev(0.0, 100.0), dev(0.0, 400.0)]
    head, divs, tau = po.place_head(4, devs, COSTS, anchor=0, mu=0.05)
    assert head == 2 and tau == 1.25 and divs == [[1, 1, 2]]


def test_infeasible_anchor_yields():
    costs = dict(COSTS, block_resident=10, head_resident=25)
    devs = [dev(0.0, 100.0, room=30), dev(0.0, 100.0, room=100)]  # member 0 as head holds no block
    head, divs, tau = po.place_head(3, devs, costs, anchor=0, mu=0.05)
    assert head == 1
    for d in divs:
        assert sum(d) == 3 and d[0] >= 1


@pytest.mark.parametrize("seed", range(15))
def test_rotation_is_relabelling(seed):
    """Rotating the members and the anchor together rotates the answer."""
    rng = random.Random(200 + seed)
    m = rng.randint(2, 4)
    k = rng.randint(m, 9)
    devs = [dev(rng.uniform(0, 0.5), rng.uniform(50, 400), room=rng.randint(20, 120)) for _ in range(m)]
    costs = dict(COSTS, block_resident=10, head_resident=rng.choice([0, 10, 20]))
    anchor = rng.randrange(m)
    h1, d1, t1 = po.place_head(k, devs, costs, anchor, 0.05)
    s = rng.randrange(m)
    h2, d2, t2 = po.place_head(k, po.rotate(devs, s), costs, (anchor - s) % m, 0.05)
    if h1 is None:
        assert h2 is None
        return
    assert t1 == t2 and (h2 + s) % m == h1
    assert sorted(tuple(po.unrotate(d, s)) for d in d2) == sorted(tuple(d) for d in d1)


# ---------------------------------------------------------------- baselines, admission, tiers
def test_uniform():
    assert po.uniform(10, 4) == [3, 3, 2, 2]
    assert po.uniform(8, 4) == [2, 2, 2, 2]
    for k in range(1, 30):
        for m in range(1, 7):
            u = po.uniform(k, m)
            assert sum(u) == k and max(u) - min(u) <= 1


def test_memory_proportional():
    assert po.memory_proportional(10, [1, 1, 1, 1]) == [3, 2, 3, 2]
    assert po.memory_proportional(12, [24, 24, 12, 18]) == [4, 3, 2, 3]  # 3.69, 7.38, 9.23, 12 -> 4, 7, 9, 12
    assert po.memory_proportional(5, [0, 10]) == [0, 5]
    rng = random.Random(7)
    for _ in range(200):
        m = rng.randint(1, 6)
        rooms = [rng.randint(1, 100) for _ in range(m)]
        k = rng.randint(1, 80)
        n = po.memory_proportional(k, rooms)
        assert sum(n) == k and all(x >= 0 for x in n)
        for i in range(m):
            assert abs(n[i] - k * rooms[i] / sum(rooms)) < 1.0 + 1e-9


def test_admission_names_the_first_overloaded_member():
    costs = dict(COSTS, block_resident=10, stage_resident=5, head_resident=20)
    devs = [dev(0, 1, room=5 + 20 + 30), dev(0, 1, room=5 + 20), dev(0, 1, room=5 + 10)]
    assert po.admit([3, 2, 1], 0, devs, costs) is None
    assert po.admit([3, 3, 1], 0, devs, costs) == 1
    assert po.admit([4, 3, 2], 0, devs, costs) == 0
    assert po.admit([3, 2, 0], 0, [devs[0], devs[1], dev(0, 1, room=0)], costs) is None  # no block, no head


def test_tiers_follow_the_measurements():
    costs = dict(COSTS, block_resident=10)
    full = [dev(0.0, 100.0, flops=5.0), dev(0.0, 300.0, flops=5.0)]
    assert po.plan(4, full, costs, 0, 0.05)["tier"] == 1
    no_bw = [dict(full[0], bw=0.0), full[1]]
    p = po.plan(4, no_bw, costs, 0, 0.05)
    assert p["tier"] == 2 and p["head"] == 0
    assert p["n"] == [2, 2]  # equal flop rates
    none = [dict(full[0], bw=0.0, flops=0.0, room=300), dict(full[1], bw=0.0, flops=0.0, room=100)]
    p = po.plan(4, none, costs, 0, 0.05)
    assert p["tier"] == 3 and p["n"] == [3, 1] and p["tau"] is None


def test_tier1_refusal():
    costs = dict(COSTS, block_resident=10)
    devs = [dev(0.0, 100.0, room=15), dev(0.0, 100.0, room=0)]
    p = po.plan(2, devs, costs, 0, 0.05)
    assert p["n"] is None and p["culprit"] == 1
    devs = [dev(0.0, 100.0, room=15), dev(0.0, 100.0, room=15)]
    p = po.plan(3, devs, costs, 0, 0.05)
    assert p["n"] is None and p["culprit"] == -1  # each holds one block; three do not fit


def test_bottleneck_stats():
    s = po.bottleneck_stats([2.0, 4.0, 3.0])
    assert s == dict(imbalance=2.0, bottleneck=4.0, utilisation=0.75)

"""The native planner (C ABI) against the planner oracle, on seeded random instances.

All host-only: no GPU is needed.  Where several divisions share the optimal
bottleneck the native answer must be one of the oracle's optimal divisions;
the bottleneck, the head, the tier and every integer baseline must match
exactly.
"""
import random

import pytest

import synth
from oracle import planner_oracle as po
from paper_2609_34045_amd import planner
from tests.test_planner_oracle import minimax_recursion


def _instance(rng, m_max=5, k_max=12):
    m = rng.randint(1, m_max)
    k = rng.randint(1, k_max)
    fixed = [rng.choice([0.0, rng.uniform(0, 3)]) for _ in range(m)]
    per = [rng.uniform(0.05, 4) for _ in range(m)]
    lim = [rng.randint(0, k + 1) for _ in range(m)]
    return k, fixed, per, lim


@pytest.mark.parametrize("seed", range(300))
def test_partition_matches_enumeration(seed):
    rng = random.Random(seed)
    k, fixed, per, lim = _instance(rng)
    tau, divs = po.best_division(k, fixed, per, lim)
    got = planner.partition(k, fixed, per, lim)
    if tau is None:
        assert got is None
        return
    n, t = got
    assert t == tau
    assert tuple(n) in divs


@pytest.mark.parametrize("seed", range(40))
def test_partition_large_matches_recursion(seed):
    """Sizes past enumeration (up to 96 blocks over 9 members) against the independent recursion."""
    rng = random.Random(1000 + seed)
    m = rng.randint(2, 9)
    k = rng.randint(m, 96)
    fixed = [rng.uniform(0, 5e-3) for _ in range(m)]
    per = [rng.uniform(1e-4, 3e-3) for _ in range(m)]
    lim = [rng.randint(1, k) for _ in range(m)]
    ref = minimax_recursion(k, fixed, per, lim)
    got = planner.partition(k, fixed, per, lim)
    if ref is None:
        assert got is None
        return
    n, t = got
    assert t == ref
    assert sum(n) == k and all(1 <= n[i] <= lim[i] for i in range(m))
    assert max(fixed[i] + n[i] * per[i] for i in range(m)) == t


def test_partition_rejects_bad_input():
    from paper_2609_34045_amd.stage import KFError
    with pytest.raises(KFError):
        planner.partition(0, [0.0], [1.0], [1])
    with pytest.raises(KFError):
        planner.partition(3, [0.0, 0.0], [1.0, 0.0], [3, 3])
    with pytest.raises(KFError):
        planner.partition(3, [-1.0, 0.0], [1.0, 1.0], [3, 3])


def _members(rng, m, with_missing=False):
    out = []
    for _ in range(m):
        d = dict(o=rng.uniform(0, 5e-5), bw=rng.choice([0.09e12, 0.4e12, 0.9e12, 1.3e12, 7e12]) * rng.uniform(0.9, 1.1),
                 flops=rng.uniform(1e13, 2e15), room=rng.randint(2, 40) * 10**9)
        if with_missing:
            if rng.random() < 0.3:
                d["bw"] = 0.0
            if rng.random() < 0.2:
                d["o"] = -1.0
            if rng.random() < 0.3:
                d["flops"] = 0.0
        out.append(d)
    return out


def _costs(rng):
    bb = rng.choice([436_224_000, 975_196_160, 1_711_308_800]) // rng.choice([1, 4])
    return dict(beta_block=bb, beta_head=rng.choice([0, 2 * bb, 5 * bb]), block_resident=bb + rng.randint(0, bb // 4),
                stage_resident=rng.randint(0, 10**8), head_resident=rng.choice([0, 2 * bb, 3 * bb]),
                flops_block=float(bb))


@pytest.mark.parametrize("seed", range(150))
def test_place_head_matches_oracle(seed):
    rng = random.Random(2000 + seed)
    m = rng.randint(1, 4)
    k = rng.randint(1, 10)
    devs = _members(rng, m)
    costs = _costs(rng)
    anchor = rng.randrange(m)
    mu = rng.choice([0.0, 0.05, 0.2])
    head, divs, tau = po.place_head(k, devs, costs, anchor, mu)
    got = planner.place_head(k, devs, costs, anchor, mu)
    if head is None:
        assert got is None
        return
    h, n, t = got
    assert (h, t) == (head, tau)
    assert n in divs


@pytest.mark.parametrize("seed", range(150))
def test_plan_matches_oracle(seed):
    rng = random.Random(3000 + seed)
    m = rng.randint(1, 4)
    k = rng.randint(1, 10)
    devs = _members(rng, m, with_missing=True)
    costs = _costs(rng)
    anchor = rng.randrange(m)
    ref = po.plan(k, devs, costs, anchor, 0.05)
    got = planner.plan(k, devs, costs, anchor, 0.05)
    assert got.tier == ref["tier"] and got.head == ref["head"]
    if ref["n"] is None:
        assert got.n is None and not got.admitted and got.culprit == ref["culprit"]
        return
    assert got.n in ref["divisions"]
    assert got.tau == ref["tau"]
    assert got.culprit == po.admit(got.n, got.head, devs, costs)
    assert got.admitted == (got.culprit is None)


def test_baselines_match_oracle():
    rng = random.Random(4)
    for _ in range(500):
        m = rng.randint(1, 8)
        k = rng.randint(1, 100)
        assert planner.divide_uniform(k, m) == po.uniform(k, m)
        rooms = [rng.choice([0, rng.randint(1, 96 * 10**9)]) for _ in range(m)]
        if sum(rooms) == 0:
            rooms[0] = 1
        assert planner.divide_memory(k, rooms) == po.memory_proportional(k, rooms)


def test_admit_matches_oracle():
    rng = random.Random(5)
    for _ in range(300):
        m = rng.randint(1, 6)
        devs = _members(rng, m)
        costs = _costs(rng)
        n = [rng.randint(0, 12) for _ in range(m)]
        head = rng.randrange(m)
        assert planner.admit(n, head, devs, costs) == po.admit(n, head, devs, costs)


def test_stage_cost_and_limit_match_oracle():
    rng = random.Random(6)
    for _ in range(200):
        d = _members(rng, 1)[0]
        c = _costs(rng)
        n, h = rng.randint(0, 40), rng.random() < 0.5
        assert planner.stage_cost(c, d, n, h) == po.stage_cost(d["o"], n, c["beta_block"], c["beta_head"], d["bw"], h)
        assert planner.block_limit(c, d["room"], h) == po.block_limit(d["room"], c["block_resident"],
                                                                        c["stage_resident"], c["head_resident"], h)


@pytest.mark.parametrize("shape,users,ctx", [(synth.SHAPE_TINY, 1, 256), (synth.SHAPE_8B, 4, 4160),
                                             (synth.SHAPE_8B, 1, 2112), (synth.SHAPE_32B, 4, 4160),
                                             (synth.SHAPE_70B, 1, 4160), (synth.SHAPE_8B, 0, 0)])
def test_stage_costs_add_up_to_stage_bytes(shape, users, ctx):
    """stage_resident + n * block_resident (+ head_resident) is exactly what a stage of n blocks holds."""
    from paper_2609_34045_amd import stage
    c = planner.stage_costs(shape, users, ctx)
    assert c.beta_block == shape.block_bytes()
    assert c.flops_block == c.beta_block  # two flops per two-byte weight
    for n in sorted({1, 2, 3, 8} & set(range(1, shape.n_layers + 1))):
        for head in (False, True):
            bb, bh, res = stage.stage_bytes(shape, 0, n, head, users, ctx)
            assert bb == c.beta_block and bh == (c.beta_head if head else 0)
            assert res == c.stage_resident + n * c.block_resident + (c.head_resident if head else 0)


def test_probes_reject_bad_arguments_before_touching_a_device():
    from paper_2609_34045_amd.stage import KFError
    with pytest.raises(KFError):
        planner.probe_bandwidth(1 << 20, reps=3)  # below 64 MiB
    with pytest.raises(KFError):
        planner.probe_bandwidth((64 << 20) + 4096, reps=3)  # not a multiple of 64 KiB
    with pytest.raises(KFError):
        planner.probe_bandwidth(64 << 20, reps=0)
    with pytest.raises(KFError):
        planner.probe_overhead(reps=0)

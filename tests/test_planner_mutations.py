"""Planted mistakes in the planner oracle must be caught by its pins.

Each case swaps one oracle function for a plausible wrong variant (on the CPU,
inside this process only), runs the pins of ``test_planner_oracle`` and
requires at least one of them to fail.
"""
import inspect
import math

import pytest

from oracle import planner_oracle as po
from tests import test_planner_oracle as pins

_ORIG = {name: getattr(po, name) for name in
         ("stage_cost", "block_limit", "best_division", "unrotate", "place_head", "memory_proportional", "uniform",
          "admit")}


def _no_head_term(o, n, bb, bh, bw, is_head):
    return _ORIG["stage_cost"](o, n, bb, bh, bw, False)


def _head_term_uses_block(o, n, bb, bh, bw, is_head):
    return _ORIG["stage_cost"](o, n, bb, bb, bw, is_head)


def _limit_ignores_head(room, block_resident, stage_resident, head_resident, is_head):
    return _ORIG["block_limit"](room, block_resident, stage_resident, head_resident, False)


def _limit_off_by_one(room, block_resident, stage_resident, head_resident, is_head):
    return _ORIG["block_limit"](room, block_resident, stage_resident, head_resident, is_head) + 1


def _division_sums_instead_of_max(k, fixed, per, lim):
    m = len(fixed)
    best, arg = None, []
    for n in po.compositions(k, m):
        if any(n[i] > lim[i] for i in range(m)):
            continue
        tau = sum(fixed[i] + n[i] * per[i] for i in range(m))
        if best is None or tau < best:
            best, arg = tau, [n]
        elif tau == best:
            arg.append(n)
    return best, arg


def _division_ignores_limits(k, fixed, per, lim):
    return _ORIG["best_division"](k, fixed, per, [k] * len(fixed))


def _unrotate_wrong_way(seq, r):
    return po.rotate(seq, r)


def _margin_reversed(k, devices, costs, anchor, mu):
    return _ORIG["place_head"](k, devices, costs, anchor, -mu)


def _memory_floor(k, rooms):
    total = sum(rooms)
    out, prev, run = [], 0, 0
    for r in rooms:
        run += r
        b = int(math.floor(k * run / total))
        out.append(b - prev)
        prev = b
    out[-1] += k - sum(out)
    return out


def _uniform_extra_last(k, m):
    return list(reversed(_ORIG["uniform"](k, m)))


def _admit_without_head_bytes(n, head, devices, costs):
    return _ORIG["admit"](n, head, devices, dict(costs, head_resident=0))


MUTANTS = {
    "stage_cost": [_no_head_term, _head_term_uses_block],
    "block_limit": [_limit_ignores_head, _limit_off_by_one],
    "best_division": [_division_sums_instead_of_max, _division_ignores_limits],
    "unrotate": [_unrotate_wrong_way],
    "place_head": [_margin_reversed],
    "memory_proportional": [_memory_floor],
    "uniform": [_uniform_extra_last],
    "admit": [_admit_without_head_bytes],
}
CASES = [(name, fn) for name, fns in MUTANTS.items() for fn in fns]


def _pin_calls():
    """Every pin of the oracle with the parameter values its parametrisation uses."""
    calls = []
    for name, fn in inspect.getmembers(pins, inspect.isfunction):
        if not name.startswith("test_"):
            continue
        marks = getattr(fn, "pytestmark", [])
        params = [m for m in marks if m.name == "parametrize"]
        if params:
            arg, values = params[0].args
            calls += [(name, fn, {arg: v}) for v in values]
        else:
            calls.append((name, fn, {}))
    return calls


@pytest.mark.parametrize("name,fn", CASES, ids=[f"{n}:{f.__name__}" for n, f in CASES])
def test_pins_catch_mutant(monkeypatch, name, fn):
    monkeypatch.setattr(po, name, fn)
    caught = []
    for pin_name, pin, kw in _pin_calls():
        try:
            pin(**kw)
        except Exception:  # noqa: BLE001 - any failure of a pin counts
            caught.append(pin_name)
    assert caught, f"no pin fails with {fn.__name__} planted in {name}"

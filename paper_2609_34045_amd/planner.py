"""Python binding of the planner (``include/kafila_planner.h``): argument marshalling only.

The cost model, the exact division (Algorithm 1), head placement, admission,
the baselines and the device probes all run in ``libkafila_stage.so``; this
module converts Python values to the C structs and back.
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass

from . import stage

EXPORTS = ("kf_stage_costs", "kf_stage_cost", "kf_block_limit", "kf_partition", "kf_place_head", "kf_divide_uniform",
           "kf_divide_memory", "kf_admit", "kf_plan", "kf_probe_bandwidth", "kf_probe_overhead")


class Member(ctypes.Structure):
    _fields_ = [("o", ctypes.c_double), ("bw", ctypes.c_double), ("flops", ctypes.c_double), ("room", ctypes.c_int64)]


class ModelCosts(ctypes.Structure):
    _fields_ = [("beta_block", ctypes.c_int64), ("beta_head", ctypes.c_int64), ("block_resident", ctypes.c_int64),
                ("head_resident", ctypes.c_int64), ("stage_resident", ctypes.c_int64), ("flops_block", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class PlanInfo(ctypes.Structure):
    _fields_ = [("tier", ctypes.c_int32), ("head", ctypes.c_int32), ("admitted", ctypes.c_int32),
                ("culprit", ctypes.c_int32), ("tau", ctypes.c_double)]


@dataclass
class Plan:
    tier: int
    head: int
    n: list
    admitted: bool
    culprit: int | None  # None when admitted; -1 for a collective shortfall
    tau: float | None


_configured = None


def _lib():
    global _configured
    lib = stage.load_library()
    if _configured is lib:
        return lib
    I32, I64, D, VP = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    I32P, I64P, DP = ctypes.POINTER(I32), ctypes.POINTER(I64), ctypes.POINTER(D)
    MP, CP = ctypes.POINTER(Member), ctypes.POINTER(ModelCosts)
    sig = {
        "kf_stage_costs": (I32, [ctypes.POINTER(stage.ModelConfig), I32, I32, CP]),
        "kf_stage_cost": (D, [CP, MP, I32, I32]),
        "kf_block_limit": (I32, [CP, I64, I32]),
        "kf_partition": (I32, [I32, I32, DP, DP, I32P, I32P, DP]),
        "kf_place_head": (I32, [I32, I32, MP, CP, I32, D, I32P, I32P, DP]),
        "kf_divide_uniform": (I32, [I32, I32, I32P]),
        "kf_divide_memory": (I32, [I32, I32, I64P, I32P]),
        "kf_admit": (I32, [I32, I32P, I32, MP, CP, I32P]),
        "kf_plan": (I32, [I32, I32, MP, CP, I32, D, I32P, ctypes.POINTER(PlanInfo)]),
        "kf_probe_bandwidth": (I32, [VP, I64, I32, DP]),
        "kf_probe_overhead": (I32, [VP, I32, DP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _configured = lib
    return lib


def _arr(ctype, values):
    return (ctype * len(values))(*values)


def _members(devices):
    out = (Member * len(devices))()
    for i, d in enumerate(devices):
        out[i] = Member(float(d["o"]), float(d["bw"]), float(d.get("flops", 0.0)), int(d["room"]))
    return out


def model_costs(costs) -> ModelCosts:
    """A ModelCosts from a dict with the struct's field names (or a ModelCosts)."""
    if isinstance(costs, ModelCosts):
        return costs
    return ModelCosts(int(costs["beta_block"]), int(costs["beta_head"]), int(costs["block_resident"]),
                      int(costs["head_resident"]), int(costs["stage_resident"]), float(costs["flops_block"]))


def stage_costs(shape, max_users: int, max_ctx: int) -> ModelCosts:
    out = ModelCosts()
    cfg = stage.ModelConfig.of(shape)
    stage._check(_lib().kf_stage_costs(ctypes.byref(cfg), max_users, max_ctx, ctypes.byref(out)), "kf_stage_costs")
    return out


def stage_cost(costs, member: dict, n: int, is_head: bool) -> float:
    m = _members([member])
    return _lib().kf_stage_cost(ctypes.byref(model_costs(costs)), m, n, int(is_head))


def block_limit(costs, room: int, is_head: bool) -> int:
    return _lib().kf_block_limit(ctypes.byref(model_costs(costs)), int(room), int(is_head))


def partition(k: int, fixed, per, lim):
    """Algorithm 1.  Returns (n, tau), or None when no division exists."""
    m = len(fixed)
    n, tau = (ctypes.c_int32 * m)(), ctypes.c_double()
    st = _lib().kf_partition(k, m, _arr(ctypes.c_double, fixed), _arr(ctypes.c_double, per),
                             _arr(ctypes.c_int32, lim), n, ctypes.byref(tau))
    if st == stage.KF_ERANGE:
        return None
    stage._check(st, "kf_partition")
    return list(n), tau.value


def place_head(k: int, devices, costs, anchor: int, mu: float = 0.05):
    """Head placement by rotation.  Returns (head, n, tau), or None when no rotation has a division."""
    m = len(devices)
    head, n, tau = ctypes.c_int32(), (ctypes.c_int32 * m)(), ctypes.c_double()
    st = _lib().kf_place_head(k, m, _members(devices), ctypes.byref(model_costs(costs)), anchor, mu,
                              ctypes.byref(head), n, ctypes.byref(tau))
    if st == stage.KF_ERANGE:
        return None
    stage._check(st, "kf_place_head")
    return head.value, list(n), tau.value


def divide_uniform(k: int, m: int):
    n = (ctypes.c_int32 * m)()
    stage._check(_lib().kf_divide_uniform(k, m, n), "kf_divide_uniform")
    return list(n)


def divide_memory(k: int, rooms):
    m = len(rooms)
    n = (ctypes.c_int32 * m)()
    stage._check(_lib().kf_divide_memory(k, m, _arr(ctypes.c_int64, [int(r) for r in rooms]), n), "kf_divide_memory")
    return list(n)


def admit(n, head: int, devices, costs):
    """The first member whose assignment overflows its room, or None."""
    c = ctypes.c_int32()
    stage._check(_lib().kf_admit(len(devices), _arr(ctypes.c_int32, n), head, _members(devices),
                                 ctypes.byref(model_costs(costs)), ctypes.byref(c)), "kf_admit")
    return None if c.value < 0 else c.value


def plan(k: int, devices, costs, anchor: int = 0, mu: float = 0.05) -> Plan:
    m = len(devices)
    n, info = (ctypes.c_int32 * m)(), PlanInfo()
    stage._check(_lib().kf_plan(k, m, _members(devices), ctypes.byref(model_costs(costs)), anchor, mu, n,
                                ctypes.byref(info)), "kf_plan")
    refused = not any(n)
    return Plan(tier=info.tier, head=info.head, n=None if refused else list(n), admitted=bool(info.admitted),
                culprit=None if info.admitted else info.culprit, tau=None if math.isnan(info.tau) else info.tau)


def probe_bandwidth(bytes_: int = 4 << 30, reps: int = 5, stream=None) -> float:
    """Bytes/s of a streaming read on the current device (kf_probe_bandwidth)."""
    bw = ctypes.c_double()
    s = ctypes.c_void_p(stream.cuda_stream if stream is not None else None)
    stage._check(_lib().kf_probe_bandwidth(s, int(bytes_), reps, ctypes.byref(bw)), "kf_probe_bandwidth")
    return bw.value


def probe_overhead(reps: int = 5, stream=None) -> float:
    """Seconds of one empty dependent kernel on the stream (kf_probe_overhead)."""
    o = ctypes.c_double()
    s = ctypes.c_void_p(stream.cuda_stream if stream is not None else None)
    stage._check(_lib().kf_probe_overhead(s, reps, ctypes.byref(o)), "kf_probe_overhead")
    return o.value

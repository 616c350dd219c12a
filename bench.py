#!/usr/bin/env python3
"""Stage decode benchmark on one MI355X.

Default line: the 32B-shaped stage (layers [16, 32) of a 64-layer model, H5120,
40 q / 8 KV heads x 128, F27648) decoding at context 4096 (KV cache injected for
positions [0, 4096)), at batch 1 (`value`) and batch 4 (`batch4`): tokens/s, the
step's algorithmic HBM bytes per second against the 8 TB/s peak, the dominant
kernel's roofline figure (HIP-event durations of its launches), the 70B-shaped
stage's 512-token prefill chunk against the matrix-core peak (`prefill_70b`), the
streaming-read probe's attainable bandwidth, and the CPU oracle's throughput on a
bounded sample of the same workload.  Timing follows the paper's rule (Section
VI): five runs of K steps, the first discarded as cold, the median of the rest.
All inputs are seeded and synthetic.

`--workload W` prints the same kind of line for one other workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
METRIC = "stage decode tokens/s + achieved HBM GB/s (% of peak), batch 1 and 4"
RUNS = 5  # timed runs per measurement; the first is discarded, the median of the rest reported
DECODE_SRC = os.path.join(ROOT, "paper_2609_34045_amd", "csrc", "decode.hip")


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default=None, choices=[k for k in synth.WORKLOADS],
                    help="one workload's line instead of the default (32B-shaped stage, batch 1 and 4)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="CPU oracle sample budget (0 disables)")
    ap.add_argument("--no-prefill-key", action="store_true",
                    help="leave the 70B-shaped prefill chunk out of the default line")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="skip the per-launch HIP-event pass (no roofline figure)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="first run a plain device-to-device copy of this many MiB (counter calibration)")
    ap.add_argument("--cost-model", action="store_true",
                    help="probe bandwidth and dispatch overhead, then compare eq. (2)'s stage-time prediction with "
                         "measured batch-1 stage times (8B-shaped stages of 1-16 blocks and with the head, 32B, 70B)")
    ap.add_argument("--prefill", action="store_true",
                    help="time the workload's prefill chunk (matrix cores) instead of decode")
    ap.add_argument("--paged", action="store_true",
                    help="decode over a paged KV cache (a pool of 64-position pages shared by the users, the "
                         "contexts injected page by page in turn so that every user's pages are scattered)")
    ap.add_argument("--ordered", action="store_true",
                    help="batch-1 decode with the ordered (run-to-run bit-identical) output projection")
    ap.add_argument("--ring", action="store_true",
                    help="the whole 8B-shaped model as a ring of stages on this GPU: four concurrent users "
                         "against one user, in turn, batched, and over 2 and 4 members on their own streams")
    return ap.parse_args()


# ------------------------------------------------------------------ algorithmic work
def step_bytes(wl, positions) -> int:
    """HBM bytes one decode step must move: every weight once, each user's K/V for keys 0..p, the appends,
    and with the head the LM head plus the gathered embedding rows."""
    s = wl.shape
    L = wl.layer_hi - wl.layer_lo
    kv_per_key = 4 * s.n_kv_heads * s.head_dim  # K and V, 2 bytes each (the fp16 cache)
    b = L * s.block_bytes()
    b += sum(L * kv_per_key * (p + 1) for p in positions)  # reads (the new key included)
    b += len(positions) * L * kv_per_key  # appends
    if wl.has_head:
        b += s.vocab * s.hidden * 2 + s.hidden * 2 + len(positions) * s.hidden * 2
    return int(b)


def gateup_bytes(wl, B: int) -> int:
    """Algorithmic bytes of one gate/up launch: both matrices, the gain, the input rows, the SwiGLU output."""
    s = wl.shape
    return 2 * s.ffn * s.hidden * 2 + s.hidden * 2 + B * s.hidden * 4 + B * s.ffn * 4


def source_hash(path: str) -> str:
    """Hash of a kernel source's code: comments, blank lines and trailing blanks are left out,
    so that the recorded counters stay valid across edits that do not change the code."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    code = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def counters_file(wl_name: str) -> str:
    return os.path.join(ROOT, "profiles", f"counters_decode_gateup_{wl_name}.txt")


def traffic_from_counters(wl_name: str):
    """HBM bytes per gate/up launch from committed rocprofv3 counter runs, or None if absent or stale."""
    path = counters_file(wl_name)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("workload") != wl_name or rec.get("decode_hip_sha256_16") != source_hash(DECODE_SRC):
        return None
    return rec.get("bytes_per_launch")


def median_rule(times):
    """Section VI's rule: the first run is cold and discarded; the median of the rest."""
    return float(np.median(times[1:])) if len(times) > 1 else float(times[0])


def prefill_flops(wl, T: int, pos0: int) -> float:
    """Algorithmic flops of one prefill chunk: the projections plus causal attention (no masked work)."""
    s = wl.shape
    L = wl.layer_hi - wl.layer_lo
    proj = 2.0 * T * L * ((2 * s.n_q_heads + 2 * s.n_kv_heads) * s.head_dim * s.hidden + 3 * s.ffn * s.hidden)
    keys = sum(pos0 + i + 1 for i in range(T))
    attn = 4.0 * s.head_dim * s.n_q_heads * L * keys
    return proj + attn


def measure_prefill(args, wl, torch, kf, kernel_events: bool = True) -> dict:
    """The chunk [ctx - T, ctx) on top of an injected cache [0, ctx - T): RUNS runs of K chunks."""
    s = wl.shape
    T = wl.prefill_chunk
    ctx = wl.contexts[0]
    pos0 = ctx - T
    t0 = time.perf_counter()
    layers = {l: synth.layer_weights(s, wl.cfg_id, l, wl.seed) for l in range(wl.layer_lo, wl.layer_hi)}
    g = kf.Stage(s, wl.layer_lo, wl.layer_hi, layers, None)
    del layers
    kv = g.kv(1, ctx + 8)
    for l in range(wl.layer_lo, wl.layer_hi):
        kb, vb = synth.injected_kv(s, wl.cfg_id, l, 0, pos0, wl.seed)
        kv.write(l, 0, 0, torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
    h = torch.from_numpy(synth.hidden_states(wl.cfg_id, synth.STREAM_PREFILL_HIDDEN, 0, T, s.hidden, wl.seed)).cuda()
    out = torch.empty_like(h)
    torch.cuda.synchronize()
    log(f"[bench] {wl.name} prefill stage ready in {time.perf_counter() - t0:.1f} s")

    def run(n):
        for _ in range(n):
            kv.set_len(0, pos0)
            g.prefill(kv, 0, pos0, hidden=h, out=out)

    steps = max(1, args.steps // 8)  # chunks per run (a chunk is ~10 ms at the 70B shape)
    run(max(1, args.warmup // 4))
    g.sync()
    times = []
    for _ in range(RUNS):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(steps)
        torch.cuda.synchronize()
        times.append((time.perf_counter() - t0) / steps)
    g.sync()
    prof = {}
    if kernel_events:
        g.profile(True)
        run(steps)
        g.profile(False)
        prof = g.profile_read()
    fl = prefill_flops(wl, T, pos0)
    ms = 1e3 * median_rule(times)
    tf = fl / (ms * 1e-3) / 1e12
    dom = prof.get("pf_gateup", (0, 0.0))
    gu_fl = 2.0 * T * 2 * s.ffn * s.hidden
    gu_tf = gu_fl / (dom[1] / dom[0] * 1e-3) / 1e12 if dom[0] else None
    kv.close()
    g.close()
    return {
        "workload": f"{wl.name}: layers [{wl.layer_lo},{wl.layer_hi}) of a {s.n_layers}-layer model, H{s.hidden}, "
                    f"{s.n_q_heads}q/{s.n_kv_heads}kv x {s.head_dim}, F{s.ffn}; prefill chunk of {T} tokens at "
                    f"positions [{pos0},{ctx}) over an injected cache",
        "tflops": round(tf, 1), "ms_per_chunk": round(ms, 3), "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4),
        "peak_tflops": PEAK_BF16_TFLOPS, "algorithmic_flops_per_chunk": fl, "chunks_per_run": steps,
        "run_ms": [round(1e3 * t, 3) for t in times],
        "roofline": {"kernel": "gate/up GEMM + SwiGLU (prefill)", "bound": "mfma",
                     "achieved": round(gu_tf, 1) if gu_tf else None, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gu_tf / PEAK_BF16_TFLOPS, 4) if gu_tf else None, "traffic": None,
                     "algorithmic_flops_per_launch": gu_fl,
                     "avg_launch_us": round(1e3 * dom[1] / dom[0], 2) if dom[0] else None},
        "per_kernel": {k: {"launches": n, "avg_us": round(1e3 * t / n, 2)} for k, (n, t) in prof.items()},
    }


def bench_prefill(args, wl, torch, kf):
    r = measure_prefill(args, wl, torch, kf, kernel_events=not args.no_kernel_events)
    line = {
        "metric": "stage prefill TFLOP/s (% of bf16/fp16 matrix-core peak)",
        "value": r["tflops"], "unit": "TFLOP/s", "n_gpus": 1, "steps": r["chunks_per_run"], "warmup": args.warmup,
        "ms_per_step": r["ms_per_chunk"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic",
        "config": {"workload": r["workload"], "chunk": wl.prefill_chunk, "pos0": wl.contexts[0] - wl.prefill_chunk},
        "timing": f"{RUNS} runs, first discarded, median",
        "frac_of_peak": r["frac_of_peak"], "roofline": r["roofline"], "per_kernel": r["per_kernel"],
        "algorithmic_flops_per_chunk": r["algorithmic_flops_per_chunk"], "run_ms": r["run_ms"],
    }
    print(json.dumps(line), flush=True)


# ------------------------------------------------------------------ CPU oracle baseline
def host_cpu() -> dict:
    model = ""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ln.startswith("Model name:"):
                model = ln.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return {"host_cpus": os.cpu_count(), "cpu_model": model}


def cpu_baseline(wl, layer_fn, kv_inject, hidden_steps, budget_s: float):
    """The float64 oracle on this host's cores over the same decode steps, taken layer by layer: each layer
    is widened once (outside the timed region), given its injected cache, and then decodes every step's
    input, which is the previous layer's output for that step.  A layer's step depends only on the previous
    layer's output for that step and on its own cache, so this is the stage's computation with one layer's
    float64 weights in memory at a time.  Layers stop once `budget_s` of timed work is spent; the time per
    step is then scaled from the layers done to the whole stage."""
    from threadpoolctl import threadpool_info

    from oracle import OracleStage

    s = wl.shape
    B = wl.batch
    ctx = list(wl.contexts)
    L = wl.layer_hi - wl.layer_lo
    steps = len(hidden_steps)
    xs = [np.asarray(h[:B], dtype=np.float64) for h in hidden_steps]
    timed, widen_s, done_layers = 0.0, 0.0, 0
    for l in range(wl.layer_lo, wl.layer_hi):
        o = OracleStage(s, l, l + 1, layer_fn, None, max_users=B, max_ctx=max(ctx) + steps + 1, cache_weights=True)
        t0 = time.perf_counter()
        o.weights(l)
        widen_s += time.perf_counter() - t0
        for u in range(B):
            kb, vb = kv_inject[(l, u)]
            o.kv.inject(l, u, 0, kb, vb)
            o.kv.set_len(u, ctx[u])
        t0 = time.perf_counter()
        for i in range(steps):
            xs[i] = o.decode(list(range(B)), [ctx[u] + i for u in range(B)], hidden=xs[i])
        timed += time.perf_counter() - t0
        done_layers += 1
        del o
        if timed >= budget_s:
            break
    threads = max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
    per_step = timed / steps * (L / done_layers)
    rec = {
        "value": round(B / per_step, 4),
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{steps} decode steps at batch {B} from context {ctx[0]} through {done_layers} of the stage's "
                  f"{L} layers, taken layer by layer ({timed:.1f} s timed"
                  + (f", scaled by {L}/{done_layers} to the whole stage" if done_layers < L else "")
                  + f"); float64 numpy oracle on the same weights, injected cache and hidden inputs; "
                  f"{widen_s:.1f} s of weight widening excluded",
    }
    rec.update(host_cpu())
    return rec


# ------------------------------------------------------------------ main
def bench_cost_model(args, torch, kf):
    """Section V-A's cost model on this GPU: probe b and o, predict stage times by eq. (2), measure them.

    Each stage runs batch-1 decode with a cache of `ctx` keys per layer (zeros:
    timing does not depend on the values).  Timing follows the paper's rule: five
    runs of 16 steps, the first discarded, the median of the rest.  Weight
    values do not affect timing either, so every layer of a stage reuses one
    seeded layer's tensors (each still gets its own device copy).
    """
    from paper_2609_34045_amd import planner
    bw = planner.probe_bandwidth(4 << 30, reps=5)
    o = planner.probe_overhead(reps=5)
    log(f"[cost] probe: bandwidth {bw / 1e9:.1f} GB/s, dispatch overhead {o * 1e6:.2f} us")
    cases = [("8b", 1, False, 2048), ("8b", 2, False, 2048), ("8b", 4, False, 2048), ("8b", 8, False, 2048),
             ("8b", 16, False, 2048), ("8b", 4, True, 2048), ("32b", 4, False, 4096), ("32b", 16, False, 4096),
             ("70b", 2, False, 4096), ("70b", 10, False, 4096)]
    shapes = {"8b": (synth.SHAPE_8B, 2), "32b": (synth.SHAPE_32B, 4), "70b": (synth.SHAPE_70B, 5)}
    layer_cache, head_cache, rows = {}, {}, []
    steps, runs = 16, 5
    for name, n, has_head, ctx in cases:
        shape, cfg_id = shapes[name]
        if name not in layer_cache:
            layer_cache[name] = synth.layer_weights(shape, cfg_id, 0)
        if has_head and name not in head_cache:
            head_cache[name] = synth.head_weights(shape, cfg_id)
        lo = 0 if has_head else shape.n_layers // 4
        g = kf.Stage(shape, lo, lo + n, {l: layer_cache[name] for l in range(lo, lo + n)},
                     head_cache[name] if has_head else None)
        kv = g.kv(1, ctx + steps + 1)
        z = torch.zeros((ctx, shape.n_kv_heads, shape.head_dim), dtype=torch.int16, device="cuda")
        for l in range(lo, lo + n):
            kv.write(l, 0, 0, z, z)
        hid = torch.from_numpy(synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, 0, 1, shape.hidden)).cuda()
        out = torch.empty((1, shape.hidden), dtype=torch.float32, device="cuda")
        tok = torch.zeros(1, dtype=torch.int32, device="cuda")
        times = []
        for r in range(runs):
            kv.set_len(0, ctx)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for i in range(steps):
                if has_head:
                    g.decode(kv, [0], [ctx + i], tokens=tok, out=out)
                    tok = g.head_argmax(out)
                else:
                    g.decode(kv, [0], [ctx + i], hidden=hid, out=out)
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e-3 / steps)
        g.sync()
        measured = float(np.median(times[1:]))
        costs = planner.stage_costs(shape, 1, ctx + steps + 1)
        member = dict(o=o, bw=bw, flops=0.0, room=0)
        predicted = planner.stage_cost(costs, member, n, has_head)
        rows.append({"stage": f"{name} x{n}" + (" + head" if has_head else ""), "blocks": n, "head": has_head,
                     "context": ctx, "predicted_us": round(predicted * 1e6, 1), "measured_us": round(measured * 1e6, 1),
                     "error": round((predicted - measured) / measured, 4),
                     "kernel_launches_per_step": 5 * n + (2 if has_head else 0)})
        log(f"[cost] {rows[-1]}")
        kv.close()
        g.close()
        del z, hid, out
    errs = sorted(abs(r["error"]) for r in rows)
    print(json.dumps({
        "metric": "eq. (2) stage-time prediction vs measured (batch-1 decode)",
        "probe": {"bandwidth_gbps": round(bw / 1e9, 1), "overhead_us": round(o * 1e6, 3), "bandwidth_buffer_gib": 4},
        "rows": rows,
        "median_abs_error": errs[len(errs) // 2] if len(errs) % 2 else 0.5 * (errs[len(errs) // 2 - 1] + errs[len(errs) // 2]),
        "timing": f"{runs} runs of {steps} steps, first discarded, median",
    }), flush=True)


def bench_ring(args, torch, kf):
    """Section VII-C's concurrency on one GPU: the ring's members overlap on their own streams.

    The whole 32-layer 8B-shaped model plus its head, divided into 1, 2 or 4
    members of equal block ranges (the head on member 0).  Four users each hold
    a 2048-token prompt, prefilled through the ring; then every configuration
    generates `steps` tokens per user.  Timing depends on shapes only, so every
    layer reuses one seeded layer's tensors (each member gets its own device
    copy).  On one GPU the members share the HBM: the ring can only gain what
    one stream leaves idle between its kernels.
    """
    from paper_2609_34045_amd import ring as kr
    shape, cfg_id, prompt, n_users = synth.SHAPE_8B, 2, 2048, 4
    steps, warmup = max(args.steps // 4, 8), max(args.warmup // 2, 2)
    t0 = time.perf_counter()
    lw = synth.layer_weights(shape, cfg_id, 0)
    head = synth.head_weights(shape, cfg_id)
    log(f"[ring] weights generated in {time.perf_counter() - t0:.1f} s")
    prompts = [synth.tokens(cfg_id, 200 + u, prompt, shape.vocab) for u in range(n_users)]
    cases = [("one user", 1, [[0]]), ("4 users in turn, 1 member", 1, [[0], [1], [2], [3]]),
             ("4 users batched, 1 member", 1, [[0, 1, 2, 3]]), ("4 users, 2 members", 2, [[0], [1], [2], [3]]),
             ("4 users, 4 members", 4, [[0], [1], [2], [3]]), ("4 users batched, 2 members", 2, [[0, 1, 2, 3]]),
             ("2 groups of 2, 2 members", 2, [[0, 1], [2, 3]])]
    rows = []
    for name, m, groups in cases:
        per = shape.n_layers // m
        streams = [torch.cuda.Stream() for _ in range(m)]
        stages = [kf.Stage(shape, i * per, (i + 1) * per, {l: lw for l in range(i * per, (i + 1) * per)},
                           head if i == 0 else None, stream=streams[i]) for i in range(m)]
        kvs = [g.kv(n_users, prompt + steps + warmup + 2) for g in stages]
        ring = kr.Ring(stages, kvs, max_groups=4, max_prefill=512)
        users = [u for g in groups for u in g]
        first = {}
        for u in users:
            for c0 in range(0, prompt, 512):
                t = torch.from_numpy(prompts[u][c0:c0 + 512].astype(np.int32)).cuda()
                torch.cuda.synchronize()
                first[u] = ring.prefill(u, t)
        ring.sync()
        tin = torch.cat([first[u] for u in users])
        torch.cuda.synchronize()
        out = ring.generate(groups, tin, warmup)
        ring.sync()
        tin = out[-1].clone()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        out = ring.generate(groups, tin, steps)
        ring.sync()
        dt = time.perf_counter() - t0
        toks = steps * len(users)
        rows.append({"case": name, "members": m, "groups": [len(g) for g in groups], "tokens": toks,
                     "ms": round(dt * 1e3, 2), "tokens_per_s": round(toks / dt, 1),
                     "per_user_tokens_per_s": round(steps / dt, 1)})
        log(f"[ring] {rows[-1]}")
        ring.close()
        for kv in kvs:
            kv.close()
        for g in stages:
            g.close()
        del stages, kvs, ring, out, tin
        torch.cuda.empty_cache()
    base = rows[0]["tokens_per_s"]
    for r in rows:
        r["vs_one_user"] = round(r["tokens_per_s"] / base, 3)
    print(json.dumps({
        "metric": "ring decode tokens/s on one GPU (whole 8B-shaped model + head, 2048-token prompts)",
        "unit": "tokens/s", "steps_per_user": steps, "warmup": warmup, "rows": rows,
        "data": "synthetic (one seeded layer's weights in every block; seeded prompts prefilled through the ring)",
    }), flush=True)


def setup_decode(args, torch, kf, wl, users_cap: int):
    """The workload's stage with a cache of `users_cap` users, each holding its injected context."""
    s = wl.shape
    ctx = list(wl.contexts) + [wl.contexts[0]] * (users_cap - len(wl.contexts))
    t0 = time.perf_counter()
    layers = {l: synth.layer_weights(s, wl.cfg_id, l, wl.seed) for l in range(wl.layer_lo, wl.layer_hi)}
    head = synth.head_weights(s, wl.cfg_id, wl.seed) if wl.has_head else None
    log(f"[bench] generated {wl.name} weights in {time.perf_counter() - t0:.1f} s")
    t0 = time.perf_counter()
    g = kf.Stage(s, wl.layer_lo, wl.layer_hi, layers, head)
    if args.ordered:
        g.set_flags(kf.KF_STAGE_ORDERED)
    span = max(args.steps, args.warmup)
    cap = max(ctx) + span + 1
    page = 64
    n_pages = sum((c + span + 1 + page - 1) // page for c in ctx) if args.paged else None
    kv = g.kv(users_cap, cap, pages=n_pages)
    inject = {}
    for l in range(wl.layer_lo, wl.layer_hi):
        for u in range(users_cap):
            inject[(l, u)] = synth.injected_kv(s, wl.cfg_id, l, u, ctx[u], wl.seed)
    # A paged cache gets its contexts one page per user in turn, so that each user's pages are scattered.
    step_pos = page if args.paged else max(ctx)
    for p0 in range(0, max(ctx), step_pos):
        for u in range(users_cap):
            m = min(step_pos, ctx[u] - p0)
            if m <= 0:
                continue
            for l in range(wl.layer_lo, wl.layer_hi):
                kb, vb = inject[(l, u)]
                kv.write(l, u, p0, torch.from_numpy(kb[p0:p0 + m].view(np.int16)).cuda(),
                         torch.from_numpy(vb[p0:p0 + m].view(np.int16)).cuda())
            kv.set_len(u, p0 + m)
    for u in range(users_cap):
        kv.set_len(u, ctx[u])
    torch.cuda.synchronize()
    log(f"[bench] stage init + KV injection {time.perf_counter() - t0:.1f} s")
    return g, kv, layers, inject, ctx


def measure_decode(args, torch, g, kv, wl, B: int, ctx) -> dict:
    """Decode at batch B (users 0..B-1 from their injected contexts): RUNS runs of K steps, each bracketed
    by device synchronisations, the first discarded, the median of the rest; then HIP-event passes for the
    dominant kernel and the per-kernel breakdown."""
    s = wl.shape
    users = list(range(B))
    span = max(args.steps, args.warmup)
    hs = [synth.hidden_states(wl.cfg_id, synth.STREAM_DECODE_HIDDEN, i, B, s.hidden, wl.seed) for i in range(span)]
    hid = torch.from_numpy(np.stack(hs)).cuda()  # resident before the timed region
    toks0 = torch.from_numpy(synth.tokens(wl.cfg_id, 0, B, s.vocab, wl.seed)).cuda() if wl.has_head else None
    out = torch.empty((B, s.hidden), dtype=torch.float32, device="cuda")
    toks = toks0

    def run(n: int):
        nonlocal toks
        for i in range(n):
            pos = [ctx[u] + i for u in users]
            if wl.has_head:  # closed-loop greedy decode; the head reads the rows the decode kept
                g.decode(kv, users, pos, tokens=toks, keep=True)
                toks = g.head_argmax(None, rows=B)
            else:
                g.decode(kv, users, pos, hidden=hid[i], out=out)

    def reset():
        nonlocal toks
        toks = toks0
        for u in users:
            kv.set_len(u, ctx[u])

    run(args.warmup)
    g.sync()
    times, gpu_times = [], []
    for _ in range(RUNS):
        reset()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        run(args.steps)
        ev1.record()
        torch.cuda.synchronize()
        times.append((time.perf_counter() - t0) / args.steps)
        gpu_times.append(ev0.elapsed_time(ev1) * 1e-3 / args.steps)
    g.sync()
    ms_step = 1e3 * median_rule(times)

    # Kernel-timing passes: the same K steps again with HIP event pairs around
    # launches on the stage's stream (each pair adds a few microseconds to the
    # stream, so they stay out of the timed runs).  The roofline pass brackets
    # only the dominant kernel; the breakdown pass brackets every launch.
    prof, dom = {}, {}
    if not args.no_kernel_events:
        reset()
        g.profile(True, classes=["gateup"])
        run(args.steps)
        g.profile(False)
        dom = g.profile_read()
        reset()
        g.profile(True)
        run(args.steps)
        g.profile(False)
        prof = g.profile_read()
        g.sync()
    reset()
    sb = step_bytes(wl, [ctx[u] + args.steps // 2 for u in users])
    hbm = sb / (ms_step * 1e-3) / 1e9
    n_gu, t_gu = dom.get("gateup", (0, 0.0))
    avg_gu_ms = t_gu / max(n_gu, 1)
    gu_bytes = gateup_bytes(wl, B)
    achieved = gu_bytes / (avg_gu_ms * 1e-3) / 1e9 if n_gu else None
    total = max(sum(v[1] for v in prof.values()), 1e-9)
    return {
        "tokens_per_s": B / (ms_step * 1e-3),
        "ms_per_step": ms_step,
        "gpu_ms_per_step": 1e3 * median_rule(gpu_times),
        "run_ms_per_step": [round(1e3 * t, 4) for t in times],
        "hbm": {"algorithmic_bytes_per_step": sb, "achieved_gbps": round(hbm, 1),
                "frac_of_peak": round(hbm / PEAK_HBM_GBPS, 4), "peak_gbps": PEAK_HBM_GBPS},
        "roofline": {
            "kernel": "gemv gate/up + RMSNorm + SwiGLU (decode)", "bound": "hbm",
            "achieved": round(achieved, 1) if achieved else None, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4) if achieved else None,
            "traffic": None, "algorithmic_bytes_per_launch": gu_bytes,
            "avg_launch_us": round(avg_gu_ms * 1e3, 2), "launches": n_gu,
        },
        "per_kernel": {k: {"launches": n, "avg_us": round(1e3 * t / n, 2), "share": round(t / total, 4)}
                       for k, (n, t) in prof.items()},
        "hidden_steps": hs,
    }


def workload_text(wl, batches) -> str:
    s = wl.shape
    return (f"{wl.name}: layers [{wl.layer_lo},{wl.layer_hi}) of a {s.n_layers}-layer model, H{s.hidden}, "
            f"{s.n_q_heads}q/{s.n_kv_heads}kv x {s.head_dim}, F{s.ffn}" + (f", head V{s.vocab}" if wl.has_head else "")
            + f"; decode at batch {' and '.join(str(b) for b in batches)}, contexts {list(wl.contexts)}")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; the stage is one GPU's share of the ring "
                                   "(multi-GPU pipelining is not built)", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    from paper_2609_34045_amd import stage as kf

    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log(f"[bench] copied {args.copy_calibration_mb} MiB three times (calibration)")
    torch.cuda.set_device(0)
    if args.cost_model:
        return bench_cost_model(args, torch, kf)
    if args.ring:
        return bench_ring(args, torch, kf)
    if args.prefill:
        wl = synth.WORKLOADS[args.workload or "70b"]
        if not wl.prefill_chunk:
            sys.exit(f"workload {wl.name} has no prefill chunk")
        return bench_prefill(args, wl, torch, kf)

    # The default line: the 32B-shaped stage at batch 1 (value) and batch 4; otherwise one workload.
    combined = args.workload is None
    wl = synth.WORKLOADS["32b_b1" if combined else args.workload]
    wl4 = synth.WORKLOADS["32b_b4"] if combined else None
    B = wl.batch
    g, kv, layers, inject, ctx = setup_decode(args, torch, kf, wl4 if combined else wl, 4 if combined else B)
    r1 = measure_decode(args, torch, g, kv, wl, B, ctx)
    log(f"[bench] {wl.name} batch {B}: {r1['tokens_per_s']:.1f} tokens/s, {r1['ms_per_step']:.3f} ms/step")
    r4 = None
    if combined:
        r4 = measure_decode(args, torch, g, kv, wl4, 4, ctx)
        log(f"[bench] {wl4.name} batch 4: {r4['tokens_per_s']:.1f} tokens/s, {r4['ms_per_step']:.3f} ms/step")
    kv.close()
    g.close()
    torch.cuda.empty_cache()

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(wl, lambda l: layers[l], inject, r1["hidden_steps"], args.cpu_seconds)
        log(f"[bench] cpu oracle {cpu['value']} tokens/s on {cpu['cores']} threads")
    del layers, inject

    from paper_2609_34045_amd import planner
    probe_bw = planner.probe_bandwidth(4 << 30, reps=5)

    pf = None
    if combined and not args.no_prefill_key:
        pf = measure_prefill(args, synth.WORKLOADS["70b"], torch, kf)
        log(f"[bench] 70b prefill chunk {pf['tflops']} TFLOP/s ({pf['frac_of_peak']:.3f} of peak)")

    r1["roofline"]["traffic"] = traffic_from_counters(wl.name)
    line = {
        "metric": METRIC,
        "value": round(r1["tokens_per_s"], 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r1["ms_per_step"], 4),
        "gpu_ms_per_step": round(r1["gpu_ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",  # fp16 weight matrices and KV cache, fp32 sums
        "data": "synthetic",
        "config": {
            "workload": workload_text(wl4 if combined else wl, [1, 4] if combined else [B])
                        + ("; value = batch 1, batch4 = batch 4" if combined else ""),
            "batch": [1, 4] if combined else B,
            "contexts": ctx if combined else list(wl.contexts),
            "layers": wl.layer_hi - wl.layer_lo,
            "has_head": wl.has_head,
            "kv_cache": "paged: 64-position pages from a shared pool, scattered" if args.paged else "reserved per user",
            "output_projection": "ordered (fixed-order sums)" if args.ordered else "fused (arrival-order sums)",
            "parallelism": "single GPU (one stage)",
        },
        "timing": f"{RUNS} runs of {args.steps} steps after {args.warmup} warmup steps, each run bracketed by device "
                  f"synchronisations, the first run discarded, the median of the rest (paper, Section VI)",
        "run_ms_per_step": r1["run_ms_per_step"],
        "hbm": r1["hbm"],
        "roofline": r1["roofline"],
        "per_kernel": r1["per_kernel"],
    }
    if r4 is not None:
        r4["roofline"]["traffic"] = traffic_from_counters(wl4.name)
        line["batch4"] = {
            "value": round(r4["tokens_per_s"], 2), "unit": "tokens/s", "ms_per_step": round(r4["ms_per_step"], 4),
            "gpu_ms_per_step": round(r4["gpu_ms_per_step"], 4), "run_ms_per_step": r4["run_ms_per_step"],
            "hbm": r4["hbm"], "roofline": r4["roofline"], "per_kernel": r4["per_kernel"],
        }
    if pf is not None:
        line["prefill_70b"] = pf
    line["probe"] = {"attainable_read_gbps": round(probe_bw / 1e9, 1), "buffer_gib": 4,
                     "note": "streaming-read probe on this GPU (context; fractions are against 8 TB/s)"}
    line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

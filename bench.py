#!/usr/bin/env python3
"""Stage decode benchmark on one MI355X.

Times K decode steps of one pipeline stage (a contiguous range of decoder
layers, optionally with the head) at the workload's batch and context, and
prints one JSON line: tokens/s, the step's algorithmic HBM bytes per second
against the 8 TB/s peak, the dominant kernel's roofline figure (HIP-event
durations of its launches inside the timed region), and the CPU oracle's
throughput on a bounded sample of the same workload.

Default workload: layers [8, 16) of a Llama-3-8B-shaped model (H4096,
32 q / 8 KV heads x 128, F14336), batch 1, KV cache injected for positions
[0, 2048), decode at positions 2048.. .  All inputs are seeded and synthetic.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
METRIC = "stage decode tokens/s + achieved HBM GB/s (% of peak), batch 1 and 4"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "counters_decode_gateup_8b_mid.txt")
DECODE_SRC = os.path.join(ROOT, "paper_2609_34045_amd", "csrc", "decode.hip")


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="8b_mid", choices=[k for k in synth.WORKLOADS])
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="CPU oracle sample budget (0 disables)")
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


def traffic_from_counters(wl_name: str):
    """HBM bytes per gate/up launch from committed rocprofv3 counter runs, or None if absent or stale."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    rec = json.load(open(COUNTERS_FILE))
    if rec.get("workload") != wl_name or rec.get("decode_hip_sha256_16") != source_hash(DECODE_SRC):
        return None
    return rec.get("bytes_per_launch")


def prefill_flops(wl, T: int, pos0: int) -> float:
    """Algorithmic flops of one prefill chunk: the projections plus causal attention (no masked work)."""
    s = wl.shape
    L = wl.layer_hi - wl.layer_lo
    proj = 2.0 * T * L * ((2 * s.n_q_heads + 2 * s.n_kv_heads) * s.head_dim * s.hidden + 3 * s.ffn * s.hidden)
    keys = sum(pos0 + i + 1 for i in range(T))
    attn = 4.0 * s.head_dim * s.n_q_heads * L * keys
    return proj + attn


def bench_prefill(args, wl, torch, kf):
    """Time the chunk [ctx - T, ctx) on top of an injected cache [0, ctx - T), K times."""
    s = wl.shape
    T = wl.prefill_chunk
    ctx = wl.contexts[0]
    pos0 = ctx - T
    layers = {l: synth.layer_weights(s, wl.cfg_id, l, wl.seed) for l in range(wl.layer_lo, wl.layer_hi)}
    g = kf.Stage(s, wl.layer_lo, wl.layer_hi, layers, None)
    kv = g.kv(1, ctx + 8)
    for l in range(wl.layer_lo, wl.layer_hi):
        kb, vb = synth.injected_kv(s, wl.cfg_id, l, 0, pos0, wl.seed)
        kv.write(l, 0, 0, torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
    del layers
    h = torch.from_numpy(synth.hidden_states(wl.cfg_id, synth.STREAM_PREFILL_HIDDEN, 0, T, s.hidden, wl.seed)).cuda()
    out = torch.empty_like(h)

    def run(n):
        for _ in range(n):
            kv.set_len(0, pos0)
            g.prefill(kv, 0, pos0, hidden=h, out=out)

    run(args.warmup)
    g.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    prof = {}
    if not args.no_kernel_events:
        g.profile(True)
        run(args.steps)
        g.profile(False)
        prof = g.profile_read()
    fl = prefill_flops(wl, T, pos0)
    ms = 1e3 * wall / args.steps
    tf = fl / (ms * 1e-3) / 1e12
    dom = prof.get("pf_gateup", (0, 0.0))
    gu_fl = 2.0 * T * 2 * s.ffn * s.hidden
    gu_tf = gu_fl / (dom[1] / dom[0] * 1e-3) / 1e12 if dom[0] else None
    line = {
        "metric": "stage prefill TFLOP/s (% of bf16/fp16 matrix-core peak)",
        "value": round(tf, 1), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic",
        "config": {"workload": f"{wl.name}: layers [{wl.layer_lo},{wl.layer_hi}), prefill chunk of {T} tokens at "
                               f"positions [{pos0},{ctx}) over an injected cache", "chunk": T, "pos0": pos0},
        "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4),
        "roofline": {"kernel": "gate/up GEMM + SwiGLU (prefill)", "bound": "mfma",
                     "achieved": round(gu_tf, 1) if gu_tf else None, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gu_tf / PEAK_BF16_TFLOPS, 4) if gu_tf else None, "traffic": None,
                     "algorithmic_flops_per_launch": gu_fl,
                     "avg_launch_us": round(1e3 * dom[1] / dom[0], 2) if dom[0] else None},
        "per_kernel": {k: {"launches": n, "avg_us": round(1e3 * t / n, 2)} for k, (n, t) in prof.items()},
        "algorithmic_flops_per_chunk": fl,
    }
    print(json.dumps(line), flush=True)
    kv.close()
    g.close()


# ------------------------------------------------------------------ CPU oracle baseline
def cpu_baseline(wl, model_layers, kv_inject, hidden_steps, budget_s: float):
    from threadpoolctl import threadpool_info

    from oracle import OracleStage

    s = wl.shape
    B = wl.batch
    ctx = list(wl.contexts)
    o = OracleStage(s, wl.layer_lo, wl.layer_hi, model_layers, None, max_users=B,
                    max_ctx=max(ctx) + len(hidden_steps) + 1, cache_weights=True)
    t0 = time.perf_counter()
    for l in range(wl.layer_lo, wl.layer_hi):
        o.weights(l)  # widen to float64 outside the timed region
    widen_s = time.perf_counter() - t0
    for (l, u), (kb, vb) in kv_inject.items():
        o.kv.inject(l, u, 0, kb, vb)
    for u in range(B):
        o.kv.set_len(u, ctx[u])
    done, t0 = 0, time.perf_counter()
    while done < len(hidden_steps):
        o.decode(list(range(B)), [ctx[u] + done for u in range(B)], hidden=hidden_steps[done])
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    threads = max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
    return {
        "value": round(B * done / el, 3),
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{done} decode step(s) of the same stage, batch {B}, from the injected context "
                  f"(float64 numpy oracle; {widen_s:.1f} s of weight widening excluded)",
    }


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
    if args.cost_model:
        torch.cuda.set_device(0)
        return bench_cost_model(args, torch, kf)
    if args.ring:
        torch.cuda.set_device(0)
        return bench_ring(args, torch, kf)
    wl = synth.WORKLOADS[args.workload]
    if args.prefill:
        if not wl.prefill_chunk:
            sys.exit(f"workload {wl.name} has no prefill chunk")
        torch.cuda.set_device(0)
        return bench_prefill(args, wl, torch, kf)
    s, B = wl.shape, wl.batch
    ctx = list(wl.contexts)
    torch.cuda.set_device(0)
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
    kv = g.kv(B, cap, pages=n_pages)
    inject = {}
    for l in range(wl.layer_lo, wl.layer_hi):
        for u in range(B):
            inject[(l, u)] = synth.injected_kv(s, wl.cfg_id, l, u, ctx[u], wl.seed)
    # A paged cache gets its contexts one page per user in turn, so that each user's pages are scattered.
    step_pos = page if args.paged else max(ctx)
    for p0 in range(0, max(ctx), step_pos):
        for u in range(B):
            m = min(step_pos, ctx[u] - p0)
            if m <= 0:
                continue
            for l in range(wl.layer_lo, wl.layer_hi):
                kb, vb = inject[(l, u)]
                kv.write(l, u, p0, torch.from_numpy(kb[p0:p0 + m].view(np.int16)).cuda(),
                         torch.from_numpy(vb[p0:p0 + m].view(np.int16)).cuda())
            kv.set_len(u, p0 + m)
    for u in range(B):
        kv.set_len(u, ctx[u])
    torch.cuda.synchronize()
    log(f"[bench] stage init + KV injection {time.perf_counter() - t0:.1f} s")

    hs = [synth.hidden_states(wl.cfg_id, synth.STREAM_DECODE_HIDDEN, i, B, s.hidden, wl.seed) for i in range(span)]
    hid = torch.from_numpy(np.stack(hs)).cuda()  # resident before the timed region
    toks = torch.from_numpy(synth.tokens(wl.cfg_id, 0, B, s.vocab, wl.seed)).cuda() if wl.has_head else None
    out = torch.empty((B, s.hidden), dtype=torch.float32, device="cuda")
    users = list(range(B))

    def run(n: int):
        nonlocal toks
        for i in range(n):
            pos = [ctx[u] + i for u in users]
            if wl.has_head:
                g.decode(kv, users, pos, tokens=toks, out=out)
                toks = g.head_argmax(out)  # closed-loop greedy decode
            else:
                g.decode(kv, users, pos, hidden=hid[i], out=out)

    def reset():
        for u in users:
            kv.set_len(u, ctx[u])

    run(args.warmup)
    g.sync()
    reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    run(args.steps)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms_step = ev0.elapsed_time(ev1) / args.steps
    ms_step = 1e3 * wall / args.steps
    tok_s = B * args.steps / (wall if wall > 0 else 1e-9)
    g.sync()

    # Kernel-timing passes: the same K steps again with HIP event pairs around
    # launches (each pair adds a few microseconds to the stream, so they stay out
    # of the timed region above).  The roofline pass brackets only the dominant
    # kernel; the breakdown pass brackets every launch.
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
    positions_mid = [ctx[u] + args.steps // 2 for u in users]
    sb = step_bytes(wl, positions_mid)
    hbm = sb / (ms_step * 1e-3) / 1e9

    # dominant kernel: the fused RMSNorm + gate/up + SwiGLU GEMV
    n_gu, t_gu = dom.get("gateup", (0, 0.0))
    avg_gu_ms = t_gu / max(n_gu, 1)
    gu_bytes = gateup_bytes(wl, B)
    achieved = gu_bytes / (avg_gu_ms * 1e-3) / 1e9 if n_gu else None
    per_kernel = {k: {"launches": n, "avg_us": round(1e3 * t / n, 2), "share": round(t / max(sum(v[1] for v in
                  prof.values()), 1e-9), 4)} for k, (n, t) in prof.items()}

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(wl, lambda l: layers[l], inject, hs, args.cpu_seconds)
        log(f"[bench] cpu oracle {cpu['value']} tokens/s on {cpu['cores']} threads")

    traffic = traffic_from_counters(wl.name)
    line = {
        "metric": METRIC,
        "value": round(tok_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "gpu_ms_per_step": round(gpu_ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",  # fp16 weight matrices and KV cache, fp32 sums
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: layers [{wl.layer_lo},{wl.layer_hi}) of a {s.n_layers}-layer model, H{s.hidden}, "
                        f"{s.n_q_heads}q/{s.n_kv_heads}kv x {s.head_dim}, F{s.ffn}"
                        + (f", head V{s.vocab}" if wl.has_head else "") + f"; batch {B}, contexts {ctx}, decode",
            "batch": B,
            "contexts": ctx,
            "layers": wl.layer_hi - wl.layer_lo,
            "has_head": wl.has_head,
            "kv_cache": "paged: 64-position pages from a shared pool, scattered" if args.paged else "reserved per user",
            "parallelism": "single GPU (one stage)",
        },
        "hbm": {"algorithmic_bytes_per_step": sb, "achieved_gbps": round(hbm, 1),
                "frac_of_peak": round(hbm / PEAK_HBM_GBPS, 4), "peak_gbps": PEAK_HBM_GBPS},
        "roofline": {
            "kernel": "gemv gate/up + RMSNorm + SwiGLU (decode)",
            "bound": "hbm",
            "achieved": round(achieved, 1) if achieved else None,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4) if achieved else None,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": gu_bytes,
            "avg_launch_us": round(avg_gu_ms * 1e3, 2),
            "launches": n_gu,
        },
        "per_kernel": per_kernel,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    kv.close()
    g.close()


if __name__ == "__main__":
    main()

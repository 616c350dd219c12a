"""The cost model's device probes and eq. (2) on the GPU (Section V-A)."""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def test_probe_bandwidth_is_physical():
    from paper_2609_34045_amd import planner
    bw = planner.probe_bandwidth(1 << 30, reps=3)
    print(f"probe bandwidth {bw / 1e9:.1f} GB/s", flush=True)
    assert 1e12 < bw < 8.2e12  # a 1 GiB stream is past the caches; HBM3E peak is 8 TB/s


def test_probe_overhead_is_physical():
    from paper_2609_34045_amd import planner
    o = planner.probe_overhead(reps=3)
    print(f"probe overhead {o * 1e6:.2f} us", flush=True)
    assert 2e-7 < o < 1e-4


def test_stage_time_is_bounded_by_the_probe():
    """A 2-block 8B-shaped stage cannot stream its weights much faster than the probed bandwidth."""
    from paper_2609_34045_amd import planner, stage
    s = synth.SHAPE_8B
    w = synth.layer_weights(s, 2, 0)
    g = stage.Stage(s, 8, 10, {8: w, 9: w}, None)
    kv = g.kv(1, 300)
    z = torch.zeros((256, s.n_kv_heads, s.head_dim), dtype=torch.int16, device="cuda")
    for l in (8, 9):
        kv.write(l, 0, 0, z, z)
    kv.set_len(0, 256)
    hid = torch.from_numpy(synth.hidden_states(2, synth.STREAM_DECODE_HIDDEN, 0, 1, s.hidden)).cuda()
    out = torch.empty((1, s.hidden), dtype=torch.float32, device="cuda")
    for i in range(4):
        g.decode(kv, [0], [256 + i], hidden=hid, out=out)
    kv.set_len(0, 256)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(16):
        g.decode(kv, [0], [256 + i], hidden=hid, out=out)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / 16
    g.sync()
    bw = planner.probe_bandwidth(1 << 30, reps=3)
    costs = planner.stage_costs(s, 1, 300)
    pred = planner.stage_cost(costs, dict(o=0.0, bw=bw, flops=0.0, room=0), 2, False)
    print(f"2-block stage {t * 1e6:.1f} us, eq. (2) without overhead {pred * 1e6:.1f} us", flush=True)
    assert t > 0.85 * pred
    kv.close()
    g.close()

"""The dependency gate of Sec. 4.1, measured from the per-instruction timeline.

On the Llama-3.2-1B-shaped workload (b1, context 2048) and the Llama-2-13B b1 workload
(context 2048), in the launch configuration the benchmark times:
  * busy_frac: the instructions' spans (start to end, waits included) over
    workgroups x step time, at least 0.85;
  * tail_spread: first to last workgroup finish over the step time, at most 0.05;
  * the timeline's step span is within 25% of the step's event-timed latency;
  * every queued instruction recorded start <= end, and the instructions of a workgroup
    ran in queue order without overlapping.
The stricter fraction of time spent after the inputs were ready is printed for reference.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch


@pytest.mark.gpu
@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["llama3.2-1b", "llama2-13b-b1"])
def test_dependency_gate_from_timeline(name):
    from synthetic import get_config, make_workload
    from paper_2609_12379_amd.fm import Decoder, plan_export

    print(f"case {name}", flush=True)
    cfg0 = get_config(name)
    wl = make_workload(cfg0, steps=24, device="cuda")
    cfg = wl.cfg
    wd = {k: v for k, v in wl.weights.items() if k != "layers" and v is not None}
    wd["layers"] = list(wl.weights["layers"])
    dec = Decoder(cfg, wd, list(wl.kcache), list(wl.vcache))
    try:
        b, S = cfg["batch"], wl.S
        ids = torch.zeros((25, b), dtype=torch.int32, device="cuda")
        ids[0] = torch.tensor(wl.start, dtype=torch.int32)
        pos = torch.tensor([[s + t for s in S] for t in range(24)], dtype=torch.int32, device="cuda")
        logits = torch.empty((b, cfg["vocab"]), dtype=torch.float32, device="cuda")
        for t in range(8):
            dec.step(ids[t], pos[t], pos[t], logits, ids[t + 1])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t in range(8, 16):
            dec.step(ids[t], pos[t], pos[t], logits, ids[t + 1])
        e1.record()
        torch.cuda.synchronize()
        step_us = e0.elapsed_time(e1) / 8 * 1e3

        n = dec.instruction_count()
        tl = torch.zeros(8 * n, dtype=torch.int64, device="cuda")
        dec.set_timeline(tl)
        dec.step(ids[16], pos[16], pos[16], logits, ids[17])
        torch.cuda.synchronize()
        dec.set_timeline(None)
        assert dec.last_error() == 0

        T = tl.cpu().numpy().reshape(n, 8).astype(np.int64)
        qoff, _ = plan_export(cfg, int(T[:, 5].max()) + 1)
        nwg = len(qoff) - 1
        start, ready, end, wg = T[:, 0], T[:, 1], T[:, 4], T[:, 5]
        assert (start > 0).all() and (end >= start).all(), "every instruction records its span"
        for w in range(nwg):
            s_, e_ = start[qoff[w]:qoff[w + 1]], end[qoff[w]:qoff[w + 1]]
            assert (wg[qoff[w]:qoff[w + 1]] == w).all()
            assert (s_[1:] >= e_[:-1]).all(), f"workgroup {w}: instructions overlap or run out of order"
        t0, t1 = start.min(), end.max()
        span = float(t1 - t0)                      # 100 MHz ticks
        busy = float((end - start).sum()) / (nwg * span)
        finish = np.array([end[qoff[w]:qoff[w + 1]].max() for w in range(nwg)])
        tail = float(finish.max() - finish.min()) / span
        after_ready = float((end - np.where(ready > 0, ready, start)).sum()) / (nwg * span)
        span_us = span / 100.0
        print(f"step {step_us:.1f} us (events), timeline span {span_us:.1f} us, busy_frac {busy:.3f}, "
              f"tail_spread {tail:.4f}, busy after inputs ready {after_ready:.3f}", flush=True)
        assert abs(span_us - step_us) <= 0.25 * step_us
        assert busy >= 0.85
        assert tail <= 0.05
    finally:
        dec.close()

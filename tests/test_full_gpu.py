"""Parity at the full model shapes, in the launch configuration the benchmark times.

Every full-size workload (Qwen3-0.6B, Llama-3.2-1B, Llama-2-7B, Qwen3-8B b4 ragged,
Llama-2-13B b8 ragged, and the batch-1 cells of the 8B and 13B shapes) runs two
teacher-forced steps against the oracle (fp64 instantiation) with every per-layer tap, the
logits, the greedy ids and the KV arena checked to the same bars as the small shapes. The inputs are
drawn on the device (same distributions and seeds as the host recipe) because the host
draw of a 13B model takes minutes. The ragged batched shapes run with N(0, 100^2) noise in
every slot past each lane's context: the oracle never reads those slots, so parity there
also shows the kernel does not.

The last test runs the benchmark's own loop (greedy ids chained on the device, no taps, the
GPU's own cache) and checks each step's id against the oracle teacher-forced on the ids the
GPU chose, and the last step's logits.
"""
from __future__ import annotations

import time

import numpy as np
import pytest
import torch

from tests.gpu_harness import Pair, rel_l2, check_greedy, MAX_ABS, REL_L2, TOP2_GAP

FULL = [("qwen3-0.6b", False), ("llama3.2-1b", False), ("llama2-7b", False), ("qwen3-8b", True),
        ("llama2-13b", True), ("qwen3-8b-b1", False), ("llama2-13b-b1", False)]


def _log(name):
    def f(rep):
        print(f"[{name}] {rep}", flush=True)
    return f


@pytest.mark.gpu
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,poison", FULL, ids=[n for n, _ in FULL])
def test_full_size_parity(name, poison):
    print(f"[{name}] drawing inputs on the device (poison={poison})", flush=True)
    t0 = time.time()
    pair = Pair(name, steps=2, poison=poison, device="cuda")
    print(f"[{name}] setup {time.time() - t0:.1f} s, S={pair.wl.S}", flush=True)
    try:
        reps = pair.run(2, log=_log(name))
    finally:
        pair.close()
    assert len(reps) == 2


@pytest.mark.gpu
@pytest.mark.timeout(900)
@pytest.mark.parametrize("S", [64, 4096])
def test_context_sweep_endpoints_qwen3_8b_b1(S):
    """The one kernel serves every context up to the arena's bound (the paper compiles one
    kernel per context bin, Sec. 5.3): the Qwen3-8B b1 shape at both ends of the context
    sweep, two steps each against the oracle."""
    name = "qwen3-8b-b1"
    print(f"[{name} S={S}] drawing inputs on the device", flush=True)
    pair = Pair(name, steps=2, device="cuda", cfg_override={"ctx": (S, S)})
    assert pair.wl.S == [S]
    try:
        reps = pair.run(2, log=_log(f"{name} S={S}"))
    finally:
        pair.close()
    assert len(reps) == 2


@pytest.mark.gpu
@pytest.mark.timeout(900)
def test_bench_loop_llama3_2_1b():
    """The benchmark's loop: step t reads step t-1's next_ids buffer on the device."""
    name, K = "llama3.2-1b", 6
    pair = Pair(name, steps=K, taps=False, device="cuda")
    try:
        cfg, S, b = pair.cfg, pair.wl.S, pair.cfg["batch"]
        ids = torch.empty((K + 1, b), dtype=torch.int32, device="cuda")
        ids[0] = torch.tensor(pair.wl.start, dtype=torch.int32)
        pos = torch.tensor([[s + t for s in S] for t in range(K)], dtype=torch.int32, device="cuda")
        logits = torch.empty((b, cfg["vocab"]), dtype=torch.float32, device="cuda")
        for t in range(K):
            pair.dec.step(ids[t], pos[t], pos[t], logits, ids[t + 1])
        torch.cuda.synchronize()
        assert pair.dec.last_error() == 0
        chosen = ids.cpu().numpy()
        last = logits.cpu().numpy()
        for t in range(K):
            p = [s + t for s in S]
            r = pair.orc.step(pair.kc_o, pair.vc_o, [int(v) for v in chosen[t]], p, p, precision="f64")
            for i in range(b):
                if chosen[t + 1][i] != r.next_ids[i]:
                    gap = float(np.max(r.logits[i]) - r.logits[i][int(chosen[t + 1][i])])
                    assert gap < TOP2_GAP, f"step {t} lane {i}: {chosen[t + 1][i]} vs {r.next_ids[i]} (gap {gap})"
        # the last step's id is the first argmax of the logits it wrote
        for i in range(b):
            check_greedy(last[i], chosen[K][i], r.logits[i], r.next_ids[i], f"last step lane {i}")
        ma, rl = float(np.abs(last - r.logits).max()), rel_l2(last, r.logits)
        print(f"[{name}] chained {K} steps, ids {chosen[:, 0].tolist()}, last logits max-abs {ma:.3g} rel-l2 {rl:.3g}",
              flush=True)
        assert ma <= MAX_ABS and rl <= REL_L2
    finally:
        pair.close()

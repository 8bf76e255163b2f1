"""GPU parity: the HIP decode step (through the C ABI) against the CPU oracle.

Small shapes that still span many tiles and ragged tails; every step is checked on logits,
every per-layer tap, the KV arena and the greedy ids (bars in tests/gpu_harness.py).
"""
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _log(name):
    def f(rep):
        print(f"[{name}] {rep}", flush=True)
    return f


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


@pytest.mark.parametrize("name,gains", [
    ("toy-gpu", "uniform"),
    ("mini-qwen3", "uniform"),
    ("mini-llama3", "ones"),
    ("mini-llama2", "ones"),
    ("mini-qwen3-b4", "uniform"),
    ("mini-llama2-b8", "ones"),
    ("mini-gqa3-b4", "uniform"),
])
def test_megakernel_matches_oracle(name, gains):
    from tests.gpu_harness import Pair
    print(f"case {name} gains={gains}", flush=True)
    pr = Pair(name, gains=gains)
    reps = pr.run(log=_log(name))
    assert len(reps) == pr.wl.steps
    pr.close()


@pytest.mark.parametrize("name", ["toy-gpu", "mini-gqa3-b4", "mini-qwen3", "mini-qwen3-b4"])
def test_empty_cache_first_tokens(name):
    """Every lane starts from an empty cache: the first step attends over its new token alone
    (kv_len 0), and the arena past each cursor holds poison (N(0, 100^2) values) that must never
    be read."""
    from tests.gpu_harness import Pair
    print(f"case {name} empty cache, poisoned arena", flush=True)
    pr = Pair(name, gains="uniform", poison=True, cfg_override={"ctx": (0, 0)})
    assert pr.wl.S == [0] * pr.cfg["batch"]
    reps = pr.run(log=_log(name))
    assert len(reps) == pr.wl.steps
    pr.close()


@pytest.mark.parametrize("name", ["toy-gpu", "mini-qwen3-b4"])
def test_multilaunch_bit_identical_to_megakernel(name):
    from tests.gpu_harness import Pair
    print(f"case {name}", flush=True)
    a = Pair(name, gains="uniform", taps=False)
    b = Pair(name, gains="uniform", taps=False)
    S = a.wl.S
    tok = list(a.wl.start)
    for t in range(a.wl.steps):
        pos = [s + t for s in S]
        la, na = a.gpu_step(tok, pos, pos)
        lb, nb = b.gpu_step(tok, pos, pos, multilaunch=True)
        assert np.array_equal(la, lb) and np.array_equal(na, nb)
        tok = [int(v) for v in na]
    for l in range(a.cfg["n_layers"]):
        assert torch.equal(a.kc_d[l], b.kc_d[l]) and torch.equal(a.vc_d[l], b.vc_d[l])
    a.close(); b.close()


def test_runs_are_bit_identical_and_poison_is_invisible():
    from tests.gpu_harness import Pair
    a = Pair("mini-qwen3-b4", gains="uniform", taps=False)
    b = Pair("mini-qwen3-b4", gains="uniform", taps=False, poison=True)
    S = a.wl.S
    tok = list(a.wl.start)
    for t in range(a.wl.steps):
        pos = [s + t for s in S]
        la, na = a.gpu_step(tok, pos, pos)
        lb, nb = b.gpu_step(tok, pos, pos)
        assert np.array_equal(la, lb), "poison past the cursor changed the logits"
        tok = [int(v) for v in na]
    a.close(); b.close()


def test_lanes_decode_at_their_own_positions():
    # lane 1 at a shifted RoPE position changes only lane 1
    from tests.gpu_harness import Pair
    a = Pair("mini-qwen3-b4", gains="uniform", taps=False)
    S = a.wl.S
    tok = list(a.wl.start)
    la, _ = a.gpu_step(tok, S, S)
    b = Pair("mini-qwen3-b4", gains="uniform", taps=False)
    pos = list(S); pos[1] += 5
    lb, _ = b.gpu_step(tok, pos, S)
    assert np.array_equal(la[0], lb[0]) and np.array_equal(la[2:], lb[2:])
    assert not np.array_equal(la[1], lb[1])
    r = b.orc.step(b.kc_o, b.vc_o, tok, pos, S)
    assert np.abs(lb - r.logits).max() < 3e-2
    a.close(); b.close()


@pytest.mark.parametrize("bad,code", [("tok", 1), ("pos", 2), ("kvl", 3)])
def test_bad_device_inputs_report_an_error_and_touch_nothing(bad, code):
    from tests.gpu_harness import Pair
    from paper_2609_12379_amd import fm as F
    a = Pair("toy-gpu", taps=False)
    S = a.wl.S
    tok, pos, kvl = list(a.wl.start), list(S), list(S)
    if bad == "tok":
        tok[0] = a.cfg["vocab"]
    elif bad == "pos":
        pos[1] = a.cfg["max_ctx"]
    else:
        kvl[0] = a.cfg["max_ctx"]
    before = [t.clone() for t in a.kc_d]
    a.logits.fill_(7.0)
    a.gpu_step(tok, pos, kvl)
    assert a.dec.last_error() == code
    assert torch.all(a.logits == 7.0)
    for x, y in zip(before, a.kc_d):
        assert torch.equal(x, y)
    with pytest.raises(F.FmError) as ei:
        a.gpu_step(list(a.wl.start), S, S)
    assert ei.value.status == F.FM_ERR_DEVICE
    a.close()

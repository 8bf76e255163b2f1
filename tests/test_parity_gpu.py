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


def test_exact_logit_tie_picks_the_lowest_index():
    """Greedy ties (reading c9: the lowest index among equal maxima wins). Before every step two
    LM-head rows per lane are set to the same bf16 vector, pointed along that lane's final normed
    state so that the pair holds the step's largest logit. The two rows of a pair sit in LM tiles
    of different workgroups on different XCDs, with the same row count, so both tiles sum their
    dot products in the same order and the two logits are bit-identical: an exact tie that the
    cross-workgroup argmax must break towards the lower row."""
    from oracle.oracle import Oracle
    from paper_2609_12379_amd import fm as F
    from synthetic import as_u16
    from tests.gpu_harness import Pair, to_u16, check_greedy
    pr = Pair("toy-gpu", gains="uniform", taps=False)
    cfg, S, b = pr.cfg, pr.wl.S, pr.cfg["batch"]
    assert not cfg["tied_embedding"] and b == 2
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    qoff, ins = F.plan_export(cfg, n_cu)
    tiles = []                                   # (workgroup, first row, rows) of every LM tile
    for w in range(n_cu):
        for q in range(qoff[w], qoff[w + 1]):
            if ins[q, 0] == F.FM_OP_LM:
                tiles.append((w, int(ins[q, 2]), int(ins[q, 3] - ins[q, 2])))
    # pairs of equal-size tiles on different XCDs, far apart in the vocabulary, one pair per lane
    nr = max(set(t[2] for t in tiles), key=lambda n: sum(t[2] == n for t in tiles))
    same = [t for t in tiles if t[2] == nr]
    pairs = []
    for first in (2, 5):
        ta = same[first]
        tb = [t for t in same if t[0] % 8 != ta[0] % 8][-1 - first]
        pairs.append((ta[1] + 1, tb[1] + 1))     # the same position inside each tile
    print(f"tie pairs {pairs} in LM tiles of {nr} rows", flush=True)
    wts = to_u16(pr.wl.weights)
    orc = Oracle(cfg, wts)                       # holds views of wts: edits below reach it
    lm_host = wts["lm_head"]
    lm_dev = pr.wdev["lm_head"]
    tok = list(pr.wl.start)
    for t in range(pr.wl.steps):
        pos = [s + t for s in S]
        # the final normed state does not depend on the LM head: take it from a first pass
        r0 = orc.step(pr.kc_o, pr.vc_o, tok, pos, pos, precision="f64", taps=True)
        for i, (ra, rb) in enumerate(pairs):
            a = np.asarray(r0.taps["final"][i], np.float64)
            row = as_u16(torch.from_numpy((a / np.linalg.norm(a)).astype(np.float32)).to(torch.bfloat16))
            for r in (ra, rb):
                lm_host[r] = row
                lm_dev[r] = torch.from_numpy(row.view(np.int16).copy()).view(torch.bfloat16).cuda()
        r = orc.step(pr.kc_o, pr.vc_o, tok, pos, pos, precision="f64")
        lg, nx = pr.gpu_step(tok, pos, pos)
        for i, (ra, rb) in enumerate(pairs):
            assert r.logits[i][ra] == r.logits[i][rb] and r.next_ids[i] == ra, "the oracle does not see the tie"
            assert lg[i][ra] == lg[i][rb], f"step {t} lane {i}: rows {ra}, {rb} are not an exact tie on the GPU"
            assert lg[i][ra] == lg[i].max()
            assert int(nx[i]) == ra, f"step {t} lane {i}: tie broken towards {int(nx[i])}, not row {ra}"
            check_greedy(lg[i], nx[i], r.logits[i], r.next_ids[i], f"step {t} lane {i}")
        tok = [int(v) for v in r.next_ids]
    pr.close()

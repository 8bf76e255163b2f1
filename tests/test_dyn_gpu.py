"""GPU parity of GEMV stages run in dynamically claimed chunks.

The 7B-13B shapes run their large batch-1 and batch-2 QKV, O-projection and down stages in
chunks that the workgroups of a pool claim at run time (see include/fm.h). Here small shapes
run with a handful of workgroups, so that all three of those stages are split that way, with
ragged last chunks, pools of one, two and three workgroups, K split into 1, 2 or 4 parts, and
both batch widths of the VALU tiles. Each case is checked step by step against the
oracle (bars in tests/gpu_harness.py); the assignment of chunks changes from run to run, so
results must also be bit-identical across runs and launch modes.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DYN_OPS = {1, 3, 5}   # FM_OP_QKV, FM_OP_OPROJ, FM_OP_DOWN

# (shape, workgroups, batch override): pools of 1 (7 workgroups), of 1 or 2 (13), of 3 (24).
CASES = [
    ("mini-qwen3", 7, None),
    ("mini-llama3", 13, None),
    ("mini-llama2", 24, None),
    ("mini-qwen3", 16, 2),
]


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _log(name):
    def f(rep):
        print(f"[{name}] {rep}", flush=True)
    return f


def _override(batch):
    return None if batch is None else {"batch": batch}


def _dynamic_ops(cfg, nwg):
    from paper_2609_12379_amd.fm import plan_export
    _, ins = plan_export(cfg, nwg)
    return {int(o) for o, _, a, _ in ins if a < 0}


@pytest.mark.parametrize("name,nwg,batch", CASES)
def test_dynamic_chunks_match_oracle(name, nwg, batch):
    from tests.gpu_harness import Pair
    print(f"case {name} nwg={nwg} batch={batch}", flush=True)
    pr = Pair(name, gains="uniform", n_workgroups=nwg, cfg_override=_override(batch))
    assert _dynamic_ops(pr.cfg, nwg) == DYN_OPS
    reps = pr.run(log=_log(name))
    assert len(reps) == pr.wl.steps
    pr.close()


@pytest.mark.parametrize("name,nwg,batch", [CASES[1], CASES[3]])
def test_dynamic_chunks_are_bit_identical_across_runs_and_launch_modes(name, nwg, batch):
    """Three decoders on the same inputs: single launch, single launch again, one launch per
    stage. Which workgroup takes which chunk differs between them; the logits, tokens and KV
    arenas must not."""
    from tests.gpu_harness import Pair
    print(f"case {name} nwg={nwg} batch={batch}", flush=True)
    prs = [Pair(name, gains="uniform", taps=False, n_workgroups=nwg, cfg_override=_override(batch))
           for _ in range(3)]
    a = prs[0]
    assert _dynamic_ops(a.cfg, nwg) == DYN_OPS
    tok = list(a.wl.start)
    for t in range(a.wl.steps):
        pos = [s + t for s in a.wl.S]
        outs = [pr.gpu_step(tok, pos, pos, multilaunch=(k == 2)) for k, pr in enumerate(prs)]
        for lg, nx in outs[1:]:
            assert np.array_equal(outs[0][0], lg) and np.array_equal(outs[0][1], nx), f"step {t}"
        tok = [int(v) for v in outs[0][1]]
    for pr in prs[1:]:
        for l in range(a.cfg["n_layers"]):
            assert torch.equal(a.kc_d[l], pr.kc_d[l]) and torch.equal(a.vc_d[l], pr.vc_d[l])
    for pr in prs:
        pr.close()


def test_dynamic_and_fixed_tiles_agree_within_rounding():
    """The same step with every GEMV stage in fixed tiles (dyn_chunk_kb = -1): the K split of
    a row differs, so logits agree to fp32 rounding, not bit for bit."""
    from tests.gpu_harness import Pair
    name, nwg, _ = CASES[1]
    a = Pair(name, gains="uniform", taps=False, n_workgroups=nwg)
    b = Pair(name, gains="uniform", taps=False, n_workgroups=nwg, dyn_chunk_kb=-1)
    assert _dynamic_ops(a.cfg, nwg) == DYN_OPS
    pos = list(a.wl.S)
    la, _ = a.gpu_step(list(a.wl.start), pos, pos)
    lb, _ = b.gpu_step(list(b.wl.start), pos, pos)
    scale = float(np.abs(la).max())
    assert np.abs(la - lb).max() <= 1e-4 * scale, float(np.abs(la - lb).max())
    a.close(); b.close()

"""fm_decode_step_noalloc, the entry point that allocates nothing, against fm_decode_step.

The no-allocation step keeps its scratch in a fixed device array shared by every handle on
the GPU. Two calls in a row, on two handles, the second with a smaller model and shorter
contexts, must each give the same logits, greedy ids and KV rows as fm_decode_step on the
same inputs (bit-identical: the kernels are the same), and both meet the oracle's bars.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _one_call(name, ctx, n_workgroups=0):
    from tests.gpu_harness import Pair, check_greedy, rel_l2, MAX_ABS, REL_L2
    print(f"case {name} ctx={ctx} nwg={n_workgroups}", flush=True)
    a = Pair(name, gains="uniform", taps=False, cfg_override={"ctx": ctx}, n_workgroups=n_workgroups)
    b = Pair(name, gains="uniform", taps=False, cfg_override={"ctx": ctx}, n_workgroups=n_workgroups)
    if n_workgroups:
        from paper_2609_12379_amd.fm import plan_query
        assert plan_query(a.cfg, n_workgroups).n_dyn_stages > 0
    need = b.dec.noalloc_scratch_bytes()
    assert 0 < need <= (64 << 20), need
    S = a.wl.S
    tok = list(a.wl.start)
    for t in range(2):
        pos = [s + t for s in S]
        la, na = a.gpu_step(tok, pos, pos)
        tt = torch.tensor(tok, dtype=torch.int32, device="cuda")
        pp = torch.tensor(pos, dtype=torch.int32, device="cuda")
        b.dec.step(tt, pp, pp, b.logits, b.next, noalloc=True)
        torch.cuda.synchronize()
        lb, nb = b.logits.cpu().numpy(), b.next.cpu().numpy()
        assert b.dec.last_error() == 0
        assert np.array_equal(la, lb) and np.array_equal(na, nb), f"{name} step {t}: outputs differ"
        r = a.orc.step(a.kc_o, a.vc_o, tok, pos, pos, precision="f64")
        assert float(np.abs(lb - r.logits).max()) <= MAX_ABS and rel_l2(lb, r.logits) <= REL_L2
        for i in range(a.cfg["batch"]):
            check_greedy(lb[i], nb[i], r.logits[i], r.next_ids[i], f"{name} step {t} lane {i}")
        tok = [int(v) for v in r.next_ids]
    for l in range(a.cfg["n_layers"]):
        assert torch.equal(a.kc_d[l].view(torch.int16), b.kc_d[l].view(torch.int16))
        assert torch.equal(a.vc_d[l].view(torch.int16), b.vc_d[l].view(torch.int16))
    a.close(); b.close()
    return need


def test_noalloc_step_matches_the_allocating_step():
    big = _one_call("mini-qwen3-b4", (200, 900))
    small = _one_call("toy-gpu", (5, 12))
    assert small < big


def test_noalloc_step_with_dynamic_chunks():
    """Stages in dynamically claimed chunks keep their claim counters in the fixed scratch too:
    two handles of different depth in a row (different counter layouts), each cleared before
    its step."""
    big = _one_call("mini-qwen3", (300, 300), n_workgroups=7)
    small = _one_call("mini-llama3", (40, 90), n_workgroups=13)
    assert small < big


def test_noalloc_rejects_a_step_beyond_the_scratch():
    from paper_2609_12379_amd import fm as F
    from tests.gpu_harness import Pair
    # 40 layers at batch 8 with many split-KV partials need more than the fixed scratch: the call is refused
    # before anything is launched
    pr = Pair("toy-gpu", taps=False, cfg_override={"n_layers": 40, "batch": 8})
    assert pr.dec.noalloc_scratch_bytes() > (64 << 20)
    z = torch.zeros(pr.cfg["batch"], dtype=torch.int32, device="cuda")
    with pytest.raises(F.FmError) as ei:
        pr.dec.step(z, z, z, pr.logits, pr.next, noalloc=True)
    assert ei.value.status == F.FM_ERR_CAPACITY
    pr.close()

"""Prompt extension through fm_extend (single-token steps in one call) on the GPU.

* fm_extend is bit-identical to the same steps issued one fm_decode_step call at a time: logits,
  greedy tokens and the whole KV arena.
* Every prompt step agrees with the oracle. The oracle re-runs step t on the kernel's own cache
  prefix (slots below the step's slot, as the kernel wrote them) and checks the appended row
  against its own rounding window. At the last step it also checks the logits and the greedy
  token against the parity bars.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


@pytest.mark.parametrize("name,n", [("toy-gpu", 24), ("mini-gqa3-b4", 17)])
def test_extend_matches_steps_and_the_oracle(name, n):
    from oracle.oracle import Oracle
    from paper_2609_12379_amd.fm import Decoder
    from synthetic import make_workload, as_u16
    from tests.gpu_harness import to_dev, to_u16, kv_slot_ok, rel_l2, check_greedy, MAX_ABS, REL_L2
    print(f"case {name}, prompt of {n} tokens", flush=True)
    wl = make_workload(name, gains="uniform", steps=n)
    cfg, S = wl.cfg, wl.S
    b, V, L = cfg["batch"], cfg["vocab"], cfg["n_layers"]
    d, nh, nkv = cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"]
    g = torch.Generator().manual_seed(5000 + cfg["k"])
    prompt = torch.randint(0, V, (n, b), generator=g, dtype=torch.int32)
    pos = torch.tensor([[s + t for s in S] for t in range(n)], dtype=torch.int32)

    wdev = to_dev(wl.weights)
    sides = []
    for _ in range(2):
        kc = [t.cuda() for t in wl.kcache]
        vc = [t.cuda() for t in wl.vcache]
        dec = Decoder(cfg, wdev, kc, vc)
        sides.append((dec, kc, vc, torch.zeros((b, V), device="cuda"), torch.zeros(b, dtype=torch.int32, device="cuda")))
    tok_d, pos_d = prompt.cuda(), pos.cuda()
    dec, kc, vc, lg_e, nx_e = sides[0]
    dec.extend(tok_d, pos_d, pos_d, lg_e, nx_e)
    dec2, kc2, vc2, lg_s, nx_s = sides[1]
    for t in range(n):
        dec2.step(tok_d[t], pos_d[t], pos_d[t], lg_s if t == n - 1 else None, nx_s)
    torch.cuda.synchronize()
    assert dec.last_error() == 0 and dec2.last_error() == 0
    assert torch.equal(lg_e, lg_s) and torch.equal(nx_e, nx_s)
    for l in range(L):
        assert torch.equal(kc[l].view(torch.int16), kc2[l].view(torch.int16))
        assert torch.equal(vc[l].view(torch.int16), vc2[l].view(torch.int16))

    # The oracle, step by step on the kernel's cache.
    orc = Oracle(cfg, to_u16(wl.weights))
    kh = [as_u16(a.cpu()).copy() for a in kc]
    vh = [as_u16(a.cpu()).copy() for a in vc]
    prev = [as_u16(a) for a in wl.kcache], [as_u16(a) for a in wl.vcache]
    for l in range(L):
        for i in range(b):
            # slots outside [S_i, S_i + n) are untouched
            for host, init in ((kh[l], prev[0][l]), (vh[l], prev[1][l])):
                assert np.array_equal(host[i, :, :S[i]], init[i, :, :S[i]])
                assert np.array_equal(host[i, :, S[i] + n:], init[i, :, S[i] + n:])
    for t in range(n):
        p = [int(v) for v in pos[t]]
        rows = [[(kh[l][i, :, p[i]].copy(), vh[l][i, :, p[i]].copy()) for i in range(b)] for l in range(L)]
        r = orc.step(kh, vh, [int(v) for v in prompt[t]], p, p, precision="f64", taps=True)
        for l in range(L):
            for i in range(b):
                yk = r.taps["krot"][l, i].reshape(nkv, d)
                yv = r.taps["qkv"][l, i][(nh + nkv) * d:].reshape(nkv, d)
                assert kv_slot_ok(rows[l][i][0], yk)[0], f"step {t} layer {l} lane {i}: key row"
                assert kv_slot_ok(rows[l][i][1], yv)[0], f"step {t} layer {l} lane {i}: value row"
                kh[l][i, :, p[i]], vh[l][i, :, p[i]] = rows[l][i]
    lg = lg_e.cpu().numpy()
    ma, rl = float(np.abs(lg - r.logits).max()), rel_l2(lg, r.logits)
    print(f"last step: logits max-abs {ma:.3g} rel-l2 {rl:.3g}", flush=True)
    assert ma <= MAX_ABS and rl <= REL_L2
    nx = nx_e.cpu().numpy()
    for i in range(b):
        check_greedy(lg[i], nx[i], r.logits[i], r.next_ids[i], f"last step lane {i}")
    dec.close(); dec2.close()

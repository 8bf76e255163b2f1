"""The paper's fidelity bars (Sec. 4.2) on the HIP decode step, through the C ABI.

Small shapes run all their steps; the full Qwen3-0.6B and Llama-3.2-1B shapes run two.
Three implementations run every step from the same KV cache, along the golden's greedy
continuation (teacher-forced):
  * K, the HIP kernel;
  * P, the oracle's float32 step (the kernel's own arithmetic: fp32 activations, bf16 KV);
  * G, the oracle's float64 step, the golden.
Bars:
  * Eq. 4 on the appended KV rows: C = delta(K, P) < 2 B with B = delta(P, G), the golden's rows
    taken before bf16 rounding;
  * Eq. 5 on the logits: eps(K) <= 5 D, where D = eps of a decoder that rounds every module
    output and the residual stream to bf16 (the usual bf16 deployment);
  * Eq. 6 per operator, from the kernel's own tap inputs: the kernel adopts at most half of a
    bf16 narrowing of each fp32 intermediate (GEMV inputs, q and the attention weights, the SiLU
    product), alpha <= 0.5.
"""
import json
from collections import defaultdict

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _u16(t):
    return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


# (workload, norm gains, where the inputs are drawn): the small shapes over all their steps,
# the full Qwen3-0.6B and Llama-3.2-1B shapes over two steps
CASES = [("mini-qwen3", "uniform", "cpu"), ("mini-gqa3-b4", "uniform", "cpu"),
         ("mini-llama2-b8", "uniform", "cpu"), ("qwen3-0.6b", "ones", "cuda"), ("llama3.2-1b", "ones", "cuda")]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,gains,device", CASES, ids=[c[0] for c in CASES])
def test_fidelity_bars(name, gains, device):
    from oracle import fidelity as F
    from tests.gpu_harness import Pair, to_u16
    print(f"case {name}", flush=True)
    pr = Pair(name, gains=gains, steps=2 if device == "cuda" else None, device=device)
    cfg = pr.cfg
    L, b, d = cfg["n_layers"], cfg["batch"], cfg["head_dim"]
    nh, nkv = cfg["n_heads"], cfg["n_kv_heads"]
    G_ = nh // nkv
    w = to_u16(pr.wl.weights)
    wqkv = [np.concatenate([lw["wq"], lw["wk"], lw["wv"]]) for lw in w["layers"]]
    lm = w["embed"] if cfg["tied_embedding"] else w["lm_head"]
    bfd = F.Bf16Decoder(cfg, w)
    S = pr.wl.S
    tok = list(pr.wl.start)
    E, P, G, B16 = [], [], [], []
    Cs, Bs = [], []
    acc = defaultdict(lambda: ([], [], []))        # operator -> (K, A, A') pieces

    def add(key, K, A, An):
        acc[key][0].append(np.asarray(K, np.float64).ravel())
        acc[key][1].append(np.asarray(A, np.float64).ravel())
        acc[key][2].append(np.asarray(An, np.float64).ravel())

    for t in range(pr.wl.steps):
        pos = [s + t for s in S]
        kvl = list(pos)
        kg, vg = [a.copy() for a in pr.kc_o], [a.copy() for a in pr.vc_o]
        rG = pr.orc.step(kg, vg, tok, pos, kvl, precision="f64", taps=True)
        del kg, vg
        kb, vb = [a.copy() for a in pr.kc_o], [a.copy() for a in pr.vc_o]
        B16.append(bfd.step(kb, vb, tok, pos, kvl))
        del kb, vb
        rP = pr.orc.step(pr.kc_o, pr.vc_o, tok, pos, kvl, precision="f32", taps=True)
        lg, _ = pr.gpu_step(tok, pos, kvl)
        gt = pr.gpu_taps()
        E.append(lg); P.append(rP.logits); G.append(rG.logits)

        # Eq. 4: one key row and one value row per layer (every lane and KV head)
        rK, rP_, rG_ = [], [], []
        for l in range(L):
            for kind, dev, host in (("k", pr.kc_d[l], pr.kc_o[l]), ("v", pr.vc_d[l], pr.vc_o[l])):
                rK.append(np.concatenate([dev[i, :, kvl[i]].float().cpu().numpy().ravel() for i in range(b)]))
                rP_.append(np.concatenate([F.bf16_values(host[i, :, kvl[i]]).ravel() for i in range(b)]))
                if kind == "k":
                    rG_.append(np.concatenate([rG.taps["krot"][l, i] for i in range(b)]))
                else:
                    rG_.append(np.concatenate([rG.taps["qkv"][l, i][(nh + nkv) * d:] for i in range(b)]))
        Cs.append(F.delta(rK, rP_))
        Bs.append(F.delta(rP_, rG_))

        # Eq. 6 references from the kernel's own tap inputs (and its own KV cache)
        for l in range(L):
            lw = w["layers"][l]
            for i in range(b):
                x = gt["a"][l, i]
                add("qkv gemv: input", gt["qkv"][l, i], F.gemv_ref(wqkv[l], x), F.gemv_ref(wqkv[l], x, narrow_in=True))
                q = gt["qrot"][l, i].reshape(nh, d)
                o = gt["o"][l, i].reshape(nh, d)
                n = kvl[i] + 1
                Kc = _u16(pr.kc_d[l][i, :, :n])
                Vc = _u16(pr.vc_d[l][i, :, :n])
                for j in range(nh):
                    A = F.attention_ref(q[j], Kc[j // G_], Vc[j // G_])
                    add("attention: q", o[j], A, F.attention_ref(q[j], Kc[j // G_], Vc[j // G_], narrow_q=True))
                    add("attention: weights", o[j], A, F.attention_ref(q[j], Kc[j // G_], Vc[j // G_], narrow_p=True))
                xin = gt["x2"][l - 1, i] if l > 0 else F.bf16_values(w["embed"][tok[i]])
                ov = gt["o"][l, i]
                add("o-proj gemv: input", gt["x1"][l, i].astype(np.float64) - xin,
                    F.gemv_ref(lw["wo"], ov), F.gemv_ref(lw["wo"], ov, narrow_in=True))
                a2 = gt["a2"][l, i]
                A = F.mlp_ref(lw["wg"], lw["wu"], lw["wd"], a2)
                add("mlp: input", gt["mlp"][l, i], A, F.mlp_ref(lw["wg"], lw["wu"], lw["wd"], a2, narrow_in=True))
                add("mlp: silu product", gt["mlp"][l, i], A, F.mlp_ref(lw["wg"], lw["wu"], lw["wd"], a2, narrow_m=True))
        for i in range(b):
            xf = gt["final"][i]
            add("lm head gemv: input", lg[i], F.gemv_ref(lm, xf), F.gemv_ref(lm, xf, narrow_in=True))

        # next step: every side attends over P's cache, along the golden's tokens
        for l in range(L):
            for host, dev in ((pr.kc_o[l], pr.kc_d[l]), (pr.vc_o[l], pr.vc_d[l])):
                for i in range(b):
                    row = np.ascontiguousarray(host[i, :, kvl[i]]).view(np.int16)
                    dev[i, :, kvl[i]].copy_(torch.from_numpy(row).view(torch.bfloat16))
        torch.cuda.synchronize()
        tok = [int(v) for v in rG.next_ids]

    C, B = float(np.mean(Cs)), float(np.mean(Bs))
    eK, eKmax = F.eps_logits(np.concatenate(E), np.concatenate(G))
    eP, ePmax = F.eps_logits(np.concatenate(P), np.concatenate(G))
    D, Dmax = F.eps_logits(np.concatenate(B16), np.concatenate(G))
    alphas = {k: F.alpha(np.concatenate(v[0]), np.concatenate(v[1]), np.concatenate(v[2])) for k, v in acc.items()}
    print(json.dumps({"case": name, "C": C, "B": B, "eps_K": eK, "eps_max_K": eKmax, "eps_P": eP,
                      "eps_max_P": ePmax, "D": D, "D_max": Dmax, "alpha": alphas}), flush=True)
    pr.close()
    assert all(c < 2 * bb for c, bb in zip(Cs, Bs)), (Cs, Bs)
    assert eK <= 5 * D, (eK, D)
    for k, a in alphas.items():
        assert a is None or a <= 0.5, (k, a)

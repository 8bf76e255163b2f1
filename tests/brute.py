"""An independent, vectorised float64 decoder written with numpy for tiny models.

It is a second implementation of the decode step (arXiv 2609.12379 Sec. 2.1, Eq. 1) used only
to pin the C++ oracle on the toy model: whole-array numpy operations instead of the oracle's
loops, so a slip in either one shows up as a disagreement.
"""
import numpy as np


def bf(u16):
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_round_f64(x):
    """Nearest bf16 (ties to even) of float64 values, via exact candidate comparison."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)                      # may round; we compare candidates exactly
    u = f.view(np.uint32)
    lo = (u & 0xFFFF0000).astype(np.uint32)
    cands = []
    for delta in (-0x10000, 0, 0x10000, 0x20000):
        c = (lo.astype(np.int64) + delta).astype(np.uint32)
        cands.append(c)
    best = None
    bestd = None
    for c in cands:
        v = c.view(np.float32).astype(np.float64)
        dlt = np.abs(v - x)
        even = ((c >> 16) & 1) == 0
        if best is None:
            best, bestd, beste = c.copy(), dlt, even
        else:
            take = (dlt < bestd) | ((dlt == bestd) & even & ~beste)
            best = np.where(take, c, best)
            bestd = np.where(take, dlt, bestd)
            beste = np.where(take, even, beste)
    return (best >> 16).astype(np.uint16)


def rms(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rot(v, pos, theta):
    d = v.shape[-1]
    j = np.arange(d // 2, dtype=np.float64)
    ang = pos * theta ** (-2.0 * j / d)
    c, s = np.cos(ang), np.sin(ang)
    a, b = v[..., : d // 2], v[..., d // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def step(cfg, w, kc, vc, tok, pos, kvl):
    """Returns logits [b][V] float64 and the updated caches (copies)."""
    h, d, nh, nkv = cfg["hidden"], cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"]
    G = nh // nkv
    kc = [k.copy() for k in kc]
    vc = [v.copy() for v in vc]
    out = []
    for i in range(cfg["batch"]):
        x = bf(w["embed"][tok[i]])
        for l in range(cfg["n_layers"]):
            L = w["layers"][l]
            a = rms(x, bf(L["attn_norm"]), cfg["rms_eps"])
            q = (bf(L["wq"]) @ a).reshape(nh, d)
            k = (bf(L["wk"]) @ a).reshape(nkv, d)
            v = (bf(L["wv"]) @ a).reshape(nkv, d)
            if cfg["qk_norm"]:
                q = rms(q, bf(L["q_norm"]), cfg["rms_eps"])
                k = rms(k, bf(L["k_norm"]), cfg["rms_eps"])
            q = rot(q, pos[i], cfg["rope_theta"])
            k = rot(k, pos[i], cfg["rope_theta"])
            kc[l][i, :, kvl[i], :] = bf16_round_f64(k)
            vc[l][i, :, kvl[i], :] = bf16_round_f64(v)
            n = kvl[i] + 1
            K = bf(kc[l][i, :, :n, :])            # [nkv][n][d]
            V = bf(vc[l][i, :, :n, :])
            Kq = np.repeat(K, G, axis=0)           # query head j uses KV head j // G
            Vq = np.repeat(V, G, axis=0)
            s = np.einsum("jd,jtd->jt", q, Kq) / np.sqrt(d)
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p = p / p.sum(axis=1, keepdims=True)
            o = np.einsum("jt,jtd->jd", p, Vq).reshape(-1)
            x = x + bf(L["wo"]) @ o
            a2 = rms(x, bf(L["mlp_norm"]), cfg["rms_eps"])
            gt = bf(L["wg"]) @ a2
            up = bf(L["wu"]) @ a2
            m = gt / (1.0 + np.exp(-gt)) * up
            x = x + bf(L["wd"]) @ m
        af = rms(x, bf(w["final_norm"]), cfg["rms_eps"])
        lm = w["embed"] if cfg["tied_embedding"] else w["lm_head"]
        out.append(bf(lm) @ af)
    return np.stack(out), kc, vc

"""Paper-fidelity measures of arXiv 2609.12379 Sec. 4.2: TEST INFRASTRUCTURE ONLY.

Only the tests import this module. It holds:
  * ``delta``: the mean symmetric relative distance between KV-cache rows (Eq. 4);
  * ``eps_logits``: the logit distance on the golden's top 64 entries (Eq. 5) and its max form;
  * ``alpha``: the share of a tested bf16 narrowing that an output adopted (Eq. 6);
  * the per-operator references A (computed to the precision contract) and A' (one intermediate
    narrowed to bf16) that the alpha test regresses onto;
  * ``Bf16Decoder``: a decoder whose every module output and residual stream is rounded to bf16,
    the bf16 reference whose distance from the golden sets the scale of the logit bar.

Readings where the paper is loose:
  * Eq. 4 rows: one row per layer and kind (key or value) holds that layer's appended slot for
    every lane and KV head, so there are 2L rows per step;
  * Eq. 5: log-softmax over the whole vocabulary, evaluated at the golden's 64 largest logits;
  * narrowing the attention probabilities rounds the unnormalised weights exp(s - max) that
    multiply V to bf16. The normaliser stays the sum of the unrounded weights.

Arithmetic reuses the oracle's primitives (``oracle.oracle``); the few numpy formulas here are
the definitions written out.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import oracle as O


# ---- the three measures -----------------------------------------------------------------

def delta(rows_x, rows_y, eps: float = 1e-6) -> float:
    """Eq. 4: mean over rows of the mean over a row's elements of 2|x-y| / (|x|+|y|+eps).

    ``rows_x`` and ``rows_y`` are sequences of equally long 1-D arrays, one per row."""
    rows_x, rows_y = list(rows_x), list(rows_y)
    assert len(rows_x) == len(rows_y) and rows_x
    tot = 0.0
    for x, y in zip(rows_x, rows_y):
        x = np.asarray(x, np.float64).ravel()
        y = np.asarray(y, np.float64).ravel()
        assert x.shape == y.shape and x.size > 0
        tot += float(np.mean(2.0 * np.abs(x - y) / (np.abs(x) + np.abs(y) + eps)))
    return tot / len(rows_x)


def log_softmax(z) -> np.ndarray:
    z = np.asarray(z, np.float64)
    s = z - z.max()
    return s - math.log(float(np.exp(s).sum()))


def eps_logits(E, G, k: int = 64):
    """Eq. 5 and its max form: (eps, eps_max) of logits E against the golden G.

    E and G are [taps][vocab]. At each tap the golden's k largest logits are the evaluation
    points; eps averages |log_softmax(E) - log_softmax(G)| over them and then over the taps,
    eps_max takes the maximum in both places."""
    E = np.atleast_2d(np.asarray(E, np.float64))
    G = np.atleast_2d(np.asarray(G, np.float64))
    assert E.shape == G.shape and 0 < k <= G.shape[1]
    means, maxes = [], []
    for e, g in zip(E, G):
        top = np.argsort(-g, kind="stable")[:k]
        diff = np.abs(log_softmax(e)[top] - log_softmax(g)[top])
        means.append(float(diff.mean()))
        maxes.append(float(diff.max()))
    return float(np.mean(means)), float(np.max(maxes))


def alpha(K, A, A_narrow):
    """Eq. 6: <K - A, d> / <d, d> with d = A_narrow - A; None (abstain) when d is zero."""
    K = np.asarray(K, np.float64).ravel()
    A = np.asarray(A, np.float64).ravel()
    d = np.asarray(A_narrow, np.float64).ravel() - A
    dd = float(d @ d)
    if dd == 0.0:
        return None
    return float((K - A) @ d) / dd


# ---- bf16 narrowing and per-operator references ----------------------------------------

def bf16_values(u16) -> np.ndarray:
    """bf16 bit patterns -> their exact float32 values."""
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32)


def narrow(x) -> np.ndarray:
    """x rounded to bf16 (round to nearest, ties to even), as float64."""
    x = np.asarray(x, np.float64)
    return bf16_values(O.to_bf16(x, "f64")).astype(np.float64).reshape(x.shape)


def gemv_ref(W_u16, x, narrow_in: bool = False) -> np.ndarray:
    """y = W x in float64 from the bf16 weights; the input optionally narrowed to bf16."""
    x = np.asarray(x, np.float64)
    return O.gemv(W_u16, narrow(x) if narrow_in else x, "f64")


def attention_ref(q, K_u16, V_u16, narrow_q: bool = False, narrow_p: bool = False) -> np.ndarray:
    """One query head over n cached slots (Eq. 1) in float64.

    Scores s_t = q.K_t / sqrt(d), weights p_t = exp(s_t - max s), output sum_t p_t V_t / sum_t p_t.
    ``narrow_q`` rounds q to bf16 before the scores; ``narrow_p`` rounds the weights that
    multiply V to bf16 (the normaliser keeps the unrounded sum)."""
    q = np.asarray(q, np.float64)
    if narrow_q:
        q = narrow(q)
    Kf = bf16_values(K_u16).astype(np.float64)
    Vf = bf16_values(V_u16).astype(np.float64)
    s = Kf @ q / math.sqrt(q.size)
    p = np.exp(s - s.max())
    pv = narrow(p) if narrow_p else p
    return (pv @ Vf) / p.sum()


def mlp_ref(Wg, Wu, Wd, a2, narrow_in: bool = False, narrow_m: bool = False) -> np.ndarray:
    """The SwiGLU block W_d (silu(W_g a) * W_u a) in float64; ``narrow_in`` rounds a to bf16,
    ``narrow_m`` rounds the SiLU product that feeds the down projection."""
    a = np.asarray(a2, np.float64)
    if narrow_in:
        a = narrow(a)
    m = O.silu_mul(O.gemv(Wg, a, "f64"), O.gemv(Wu, a, "f64"), "f64")
    if narrow_m:
        m = narrow(m)
    return O.gemv(Wd, m, "f64")


# ---- the bf16 reference decoder ----------------------------------------------------------

class Bf16Decoder:
    """The decode step with every module output and the residual stream rounded to bf16.

    This is the usual bf16 deployment of a checkpoint: the embedding row, each norm output,
    q/k/v, the QK-norm and RoPE outputs, each head's attention output, each projection's
    output, the residual after each addition, the SiLU product and the logits are all bf16
    values; each module computes in float32 inside (the oracle's float32 primitives).
    ``rounding=False`` keeps every value in float32 instead, which must then reproduce the
    oracle's float32 step exactly.

    ``weights`` is the same dict of bf16 bit patterns that ``oracle.Oracle`` takes; the caller
    owns the KV caches ([b][n_kv][max_ctx][d_h] uint16 per layer), appended to in place."""

    def __init__(self, cfg: dict, weights: dict, rounding: bool = True):
        self.cfg = dict(cfg)
        self.w = weights
        self.rounding = rounding

    def _r(self, x) -> np.ndarray:
        x = np.asarray(x, np.float32)
        if not self.rounding:
            return x
        return bf16_values(O.to_bf16(x, "f32")).reshape(x.shape)

    def step(self, kcache, vcache, tok, pos, kv_lens):
        c, w, r = self.cfg, self.w, self._r
        h, d, nh, nkv = c["hidden"], c["head_dim"], c["n_heads"], c["n_kv_heads"]
        G, eps, theta = nh // nkv, c["rms_eps"], c["rope_theta"]
        lm = w["embed"] if c["tied_embedding"] else w["lm_head"]
        logits = np.empty((c["batch"], c["vocab"]), np.float32)
        for i in range(c["batch"]):
            x = bf16_values(w["embed"][int(tok[i])]).copy()
            for l in range(c["n_layers"]):
                L = w["layers"][l]
                a = r(O.rmsnorm(x, L["attn_norm"], eps, "f32"))
                q = r(O.gemv(L["wq"], a, "f32")).reshape(nh, d)
                k = r(O.gemv(L["wk"], a, "f32")).reshape(nkv, d)
                v = r(O.gemv(L["wv"], a, "f32")).reshape(nkv, d)
                if c["qk_norm"]:
                    q = np.stack([r(O.rmsnorm(q[j], L["q_norm"], eps, "f32")) for j in range(nh)])
                    k = np.stack([r(O.rmsnorm(k[g], L["k_norm"], eps, "f32")) for g in range(nkv)])
                q = np.stack([r(O.rope(q[j], int(pos[i]), theta, "f32")) for j in range(nh)])
                k = np.stack([r(O.rope(k[g], int(pos[i]), theta, "f32")) for g in range(nkv)])
                slot = int(kv_lens[i])
                kcache[l][i, :, slot, :] = O.to_bf16(k, "f32")
                vcache[l][i, :, slot, :] = O.to_bf16(v, "f32")
                o = np.concatenate([
                    r(O.attend(q[j], kcache[l][i, j // G, :slot + 1], vcache[l][i, j // G, :slot + 1], "f32"))
                    for j in range(nh)])
                x = r(x + r(O.gemv(L["wo"], o, "f32")))
                a2 = r(O.rmsnorm(x, L["mlp_norm"], eps, "f32"))
                m = r(O.silu_mul(r(O.gemv(L["wg"], a2, "f32")), r(O.gemv(L["wu"], a2, "f32")), "f32"))
                x = r(x + r(O.gemv(L["wd"], m, "f32")))
            af = r(O.rmsnorm(x, w["final_norm"], eps, "f32"))
            logits[i] = r(O.gemv(lm, af, "f32"))
        return logits

"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test targets a mistake the oracle could plausibly contain: a wrong rounding mode, a
transposed weight, an interleaved RoPE pairing, a missing 1/sqrt(d_h), a wrong GQA head map,
a read past the cache cursor, a dropped residual term.
"""
import math

import numpy as np
import pytest
import torch

from tests import brute
from synthetic import get_config, make_weights, make_kv, make_start, as_u16
from synthetic.inputs import contexts


def f32_bits(x):
    return np.array([x], dtype=np.float32).view(np.uint32)[0]


def bf16_of(x):
    """bf16 bits of a value that is exactly representable in bf16."""
    u = f32_bits(x)
    assert u & 0xFFFF == 0
    return np.uint16(u >> 16)


# ---- bf16 round-to-nearest-even ------------------------------------------------------

def test_bf16_rounding_ties_to_even(oracle_lib):
    o = oracle_lib
    vals = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-8 + 2**-20, -2.5, np.inf, -np.inf, 0.0],
                    dtype=np.float32)
    got = o.to_bf16(vals, "f32")
    want = [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x7F80, 0xFF80, 0x0000]
    assert [int(v) for v in got] == want
    nan = o.to_bf16(np.array([np.nan], dtype=np.float32), "f32")[0]
    assert (nan & 0x7F80) == 0x7F80 and (nan & 0x007F) != 0


def test_bf16_rounding_from_double_is_direct(oracle_lib):
    # 1 + 2^-8 + 2^-30 lies just above a bf16 tie; a float intermediate would drop 2^-30 and
    # round the tie to even (down). Direct rounding must go up.
    x = np.array([1 + 2**-8 + 2**-30, 1 + 2**-8 - 2**-30, -(1 + 3 * 2**-8)], dtype=np.float64)
    got = oracle_lib.to_bf16(x, "f64")
    assert [int(v) for v in got] == [0x3F81, 0x3F80, 0xBF82]
    rng = np.random.default_rng(0)
    y = rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000)
    assert np.array_equal(oracle_lib.to_bf16(y, "f64"), brute.bf16_round_f64(y))


# ---- RMSNorm --------------------------------------------------------------------------

def test_rmsnorm_closed_forms(oracle_lib):
    o = oracle_lib
    n, eps, c = 64, 1e-6, 3.0
    ones = np.full(n, bf16_of(1.0), dtype=np.uint16)
    y = o.rmsnorm(np.full(n, c), ones, eps)
    assert np.allclose(y, c / math.sqrt(c * c + eps), rtol=1e-14, atol=0)
    x = np.zeros(n); x[5] = -7.0
    y = o.rmsnorm(x, ones, 0.0)
    assert y[5] == pytest.approx(-math.sqrt(n), rel=1e-14) and np.count_nonzero(y) == 1
    # gain k multiplies output k (catches an indexing slip in the gains)
    gvals = np.array([0.5 + 0.25 * (k % 7) for k in range(n)], dtype=np.float32)
    g = np.array([bf16_of(v) for v in gvals], dtype=np.uint16)
    x = np.random.default_rng(1).standard_normal(n)
    base = o.rmsnorm(x, ones, eps)
    assert np.allclose(o.rmsnorm(x, g, eps) / base, gvals, rtol=1e-14)
    # scale invariance as eps -> 0
    assert np.allclose(o.rmsnorm(37.0 * x, ones, 0.0), base, rtol=1e-6)


# ---- GEMV -----------------------------------------------------------------------------

def test_gemv_row_major_out_in(oracle_lib):
    W = np.array([[1.0, 2.0, 3.0], [-1.0, 0.5, 0.25]], dtype=np.float32)
    Wb = np.vectorize(bf16_of)(W).astype(np.uint16)
    y = oracle_lib.gemv(Wb, np.array([1.0, 10.0, 100.0]))
    assert list(y) == [321.0, -1.0 + 5.0 + 25.0]


def test_gemv_f32_within_dot_product_bound(oracle_lib):
    rng = np.random.default_rng(2)
    N, K = 64, 4096
    W = as_u16((torch.randn(N, K, generator=torch.Generator().manual_seed(3)) * 0.02).to(torch.bfloat16))
    x = rng.standard_normal(K).astype(np.float32)
    y32 = oracle_lib.gemv(W, x, "f32")
    y64 = oracle_lib.gemv(W, x.astype(np.float64), "f64")
    absdot = np.abs(brute.bf(W)) @ np.abs(x.astype(np.float64))
    u = 2.0**-24
    gamma = K * u / (1 - K * u)                      # Higham's bound on recursive summation
    assert np.all(np.abs(y32 - y64) <= gamma * absdot)
    # float64 path equals an exact-ish numpy contraction of the upcast weights
    assert np.allclose(y64, brute.bf(W) @ x.astype(np.float64), rtol=1e-12, atol=1e-14)


# ---- RoPE -----------------------------------------------------------------------------

def test_rope_d2_closed_form(oracle_lib):
    for p in (0, 1, 7, 1000):
        v = oracle_lib.rope(np.array([1.0, 0.0]), p, 1e4)
        assert v == pytest.approx([math.cos(p), math.sin(p)], abs=1e-15)
        v = oracle_lib.rope(np.array([0.0, 1.0]), p, 1e4)
        assert v == pytest.approx([-math.sin(p), math.cos(p)], abs=1e-15)


def test_rope_rotate_half_pairing_and_frequencies(oracle_lib):
    theta, p = 1e4, 5
    v = oracle_lib.rope(np.array([1.0, 0.0, 0.0, 0.0]), p, theta)
    assert v == pytest.approx([math.cos(p), 0.0, math.sin(p), 0.0], abs=1e-15)
    f1 = theta ** (-2.0 / 4)
    v = oracle_lib.rope(np.array([0.0, 1.0, 0.0, 0.0]), p, theta)
    assert v == pytest.approx([0.0, math.cos(p * f1), 0.0, math.sin(p * f1)], abs=1e-15)


def test_rope_invariants(oracle_lib):
    rng = np.random.default_rng(4)
    d, theta = 128, 1e6
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    assert np.array_equal(oracle_lib.rope(q, 0, theta), q)                 # R(0) = I
    rq = oracle_lib.rope(q, 77, theta)
    pairs = lambda v: v[: d // 2] ** 2 + v[d // 2:] ** 2
    assert np.allclose(pairs(rq), pairs(q), rtol=1e-12)                      # per-pair norm
    dots = [oracle_lib.rope(q, m + c, theta) @ oracle_lib.rope(k, n + c, theta)
            for (m, n, c) in ((10, 3, 0), (10, 3, 100), (10, 3, 2000))]
    assert np.allclose(dots, dots[0], rtol=1e-9)                             # relative position
    # fp32 table: error of the f32 path stays at float rounding
    r32 = oracle_lib.rope(q.astype(np.float32), 3000, theta, "f32")
    assert np.allclose(r32, oracle_lib.rope(q, 3000, theta), atol=1e-5)


# ---- attention (Eq. 1) ----------------------------------------------------------------

def _bf_rows(a):
    """bf16 bits of values (rounded to bf16 first when not exactly representable)."""
    t = torch.tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    return as_u16(t).copy()


def test_attention_single_slot_returns_v(oracle_lib):
    d = 8
    V = _bf_rows([[0.5, -1.0, 2.0, 0.25, 0.0, 3.0, -0.125, 1.0]])
    K = _bf_rows([[1.0] * d])
    o = oracle_lib.attend(np.linspace(-1, 1, d), K, V)
    assert np.array_equal(o, brute.bf(V[0]))


def test_attention_equal_scores_give_mean(oracle_lib):
    d, n = 16, 5
    rng = np.random.default_rng(5)
    V = _bf_rows(rng.standard_normal((n, d)).astype(np.float32))
    K = _bf_rows(rng.standard_normal((n, d)).astype(np.float32))
    o = oracle_lib.attend(np.zeros(d), K, V)
    assert np.allclose(o, brute.bf(V).mean(axis=0), rtol=1e-13, atol=1e-15)


def test_attention_ln3_gap_gives_three_quarters(oracle_lib):
    # s0 - s1 = ln 3 after the 1/sqrt(d) scale => p = (3/4, 1/4). A missing or wrong scale fails.
    d = 64
    K = _bf_rows([[1.0] + [0.0] * (d - 1), [0.0] * d])
    V = _bf_rows([[1.0] + [0.0] * (d - 1), [0.0, 1.0] + [0.0] * (d - 2)])
    q = np.zeros(d); q[0] = math.sqrt(d) * math.log(3.0)
    o = oracle_lib.attend(q, K, V)
    assert o[0] == pytest.approx(0.75, abs=1e-14) and o[1] == pytest.approx(0.25, abs=1e-14)
    # softmax is unchanged by a constant added to every score (shift q along a shared key dir)
    K2 = _bf_rows([[1.0, 1.0] + [0.0] * (d - 2), [0.0, 1.0] + [0.0] * (d - 2)])
    q2 = q.copy(); q2[1] = 3.0
    assert np.allclose(oracle_lib.attend(q2, K2, V), o, atol=1e-14)


def test_attention_split_combine_equals_unsplit(oracle_lib):
    # log-sum-exp merge of chunk partials reproduces the unsplit softmax (brute force, tiny S)
    rng = np.random.default_rng(6)
    d, n = 16, 11
    K = _bf_rows(rng.standard_normal((n, d)).astype(np.float32))
    V = _bf_rows(rng.standard_normal((n, d)).astype(np.float32))
    q = rng.standard_normal(d)
    full = oracle_lib.attend(q, K, V)
    for cuts in ([4], [1, 2, 7], [3, 6, 9, 10]):
        edges = [0] + cuts + [n]
        ms, ls, os_ = [], [], []
        for a, b in zip(edges[:-1], edges[1:]):
            s = brute.bf(K[a:b]) @ q / math.sqrt(d)
            m = s.max(); p = np.exp(s - m)
            ms.append(m); ls.append(p.sum()); os_.append(p @ brute.bf(V[a:b]))
        M = max(ms)
        num = sum(math.exp(m - M) * ov for m, ov in zip(ms, os_))
        den = sum(math.exp(m - M) * l for m, l in zip(ms, ls))
        assert np.allclose(num / den, full, rtol=1e-12, atol=1e-14)


# ---- SwiGLU and argmax -----------------------------------------------------------------

def test_silu_mul_closed_forms(oracle_lib):
    from scipy.special import expit
    g = np.array([0.0, 1.0, -1.0, 40.0, -40.0, 2.5])
    u = np.array([5.0, 2.0, 3.0, 1.0, 1.0, -2.0])
    out = oracle_lib.silu_mul(g, u)
    assert out[0] == 0.0
    assert out[3] == pytest.approx(40.0, rel=1e-15)
    assert abs(out[4]) < 1e-15
    assert np.allclose(out, g * expit(g) * u, rtol=1e-14)


def test_argmax_lowest_index_on_ties(oracle_lib):
    v = np.array([1.0, 3.0, -np.inf, 3.0, 2.0], dtype=np.float32)
    assert oracle_lib.argmax(v) == 1
    rng = np.random.default_rng(7)
    for _ in range(20):
        w = rng.integers(-3, 4, 300).astype(np.float32)
        assert oracle_lib.argmax(w) == int(np.argmax(w))


# ---- the whole step on the toy model ---------------------------------------------------

def _toy(gains="uniform", seed=None, tied=False):
    cfg = get_config("toy")
    if tied:
        cfg["tied_embedding"] = 1                # no separate LM head is drawn
    S = contexts(cfg)
    cfg["max_ctx"] = max(S) + 4
    w = make_weights(cfg, gains=gains, seed=seed)
    kc, vc = make_kv(cfg, S, cfg["max_ctx"])
    wu = {k: as_u16(v) for k, v in w.items() if k != "layers"}
    wu["layers"] = [{k: as_u16(v) for k, v in lw.items()} for lw in w["layers"]]
    return cfg, wu, [as_u16(t).copy() for t in kc], [as_u16(t).copy() for t in vc], S


def test_toy_step_matches_independent_numpy(oracle_lib):
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    orc = Oracle(cfg, w)
    tok, pos = make_start(cfg), list(S)
    kc64, vc64 = [a.copy() for a in kc], [a.copy() for a in vc]
    r64 = orc.step(kc64, vc64, tok, pos, S, precision="f64")
    want, kb, vb = brute.step(cfg, w, kc, vc, tok, pos, S)
    assert np.allclose(r64.logits, want, rtol=1e-11, atol=1e-13)
    for l in range(cfg["n_layers"]):
        assert np.array_equal(kc64[l], kb[l]) and np.array_equal(vc64[l], vb[l])
    r32 = orc.step([a.copy() for a in kc], [a.copy() for a in vc], tok, pos, S, precision="f32")
    assert np.allclose(r32.logits, want, atol=1e-5, rtol=1e-5)
    assert list(r32.next_ids) == [int(np.argmax(row)) for row in r32.logits]


def test_toy_tied_embedding_step_matches_independent_numpy(oracle_lib):
    # tied models (Qwen3-0.6B, Llama-3.2-1B shapes): the LM head is the embedding matrix
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy(tied=True)
    assert "lm_head" not in w or w["lm_head"] is None
    orc = Oracle(cfg, w)
    tok, pos = make_start(cfg), list(S)
    r64 = orc.step([a.copy() for a in kc], [a.copy() for a in vc], tok, pos, S, precision="f64", taps=True)
    want, _, _ = brute.step(cfg, w, kc, vc, tok, pos, S)
    assert np.allclose(r64.logits, want, rtol=1e-11, atol=1e-13)
    # the logits are E a_f for the final normed state a_f, row by row
    E = brute.bf(w["embed"])
    for i in range(cfg["batch"]):
        assert np.allclose(r64.logits[i], E @ r64.taps["final"][i], rtol=1e-12, atol=1e-14)


def test_toy_kv_append_touches_exactly_one_slot(oracle_lib):
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    orc = Oracle(cfg, w)
    k2, v2 = [a.copy() for a in kc], [a.copy() for a in vc]
    r = orc.step(k2, v2, make_start(cfg), S, S, precision="f32", taps=True)
    d, nkv = cfg["head_dim"], cfg["n_kv_heads"]
    for l in range(cfg["n_layers"]):
        for i, s in enumerate(S):
            mask = np.ones(cfg["max_ctx"], bool); mask[s] = False
            assert np.array_equal(k2[l][i][:, mask], kc[l][i][:, mask])
            assert np.array_equal(v2[l][i][:, mask], vc[l][i][:, mask])
            krot = r.taps["krot"][l, i].reshape(nkv, d)
            vraw = r.taps["qkv"][l, i][(cfg["n_heads"] + nkv) * d:].reshape(nkv, d)
            assert np.array_equal(k2[l][i][:, s], oracle_lib.to_bf16(krot, "f32"))
            assert np.array_equal(v2[l][i][:, s], oracle_lib.to_bf16(vraw, "f32"))


def test_toy_poisoned_cache_past_cursor_is_invisible(oracle_lib):
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    orc = Oracle(cfg, w)
    tok = make_start(cfg)
    base = orc.step([a.copy() for a in kc], [a.copy() for a in vc], tok, S, S)
    rng = np.random.default_rng(8)
    kp, vp = [a.copy() for a in kc], [a.copy() for a in vc]
    for l in range(cfg["n_layers"]):
        for i, s in enumerate(S):
            noise = (rng.standard_normal(kp[l][i][:, s:].shape) * 100).astype(np.float32)
            kp[l][i][:, s:] = oracle_lib.to_bf16(noise, "f32")
            vp[l][i][:, s:] = oracle_lib.to_bf16(noise[::-1].copy(), "f32")
    pois = orc.step(kp, vp, tok, S, S)
    assert np.array_equal(base.logits, pois.logits)


def test_toy_gqa_head_map(oracle_lib):
    # Zero KV head 1's values (cache and projection): query heads 2 and 3 (g(j) = j // 2) must
    # give zero attention output, heads 0 and 1 must not.
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    d = cfg["head_dim"]
    w["layers"] = [dict(lw) for lw in w["layers"]]
    for l, lw in enumerate(w["layers"]):
        wv = lw["wv"].copy(); wv[d:2 * d] = 0; lw["wv"] = wv
        vc[l][:, 1] = 0
    r = Oracle(cfg, w).step(kc, vc, make_start(cfg), S, S, taps=True)
    o = r.taps["o"].reshape(cfg["n_layers"], cfg["batch"], cfg["n_heads"], d)
    assert np.all(o[:, :, 2:] == 0)
    assert np.all(np.abs(o[:, :, :2]).max(axis=-1) > 0)


def test_toy_lanes_decode_at_their_own_positions(oracle_lib):
    # Batched lanes equal separate batch-1 runs, each at its own position.
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    tok = make_start(cfg)
    pos = [S[0] + 3, S[1]]
    rb = Oracle(cfg, w).step([a.copy() for a in kc], [a.copy() for a in vc], tok, pos, S)
    for i in range(cfg["batch"]):
        c1 = dict(cfg, batch=1)
        r1 = Oracle(c1, w).step([a[i:i + 1].copy() for a in kc], [a[i:i + 1].copy() for a in vc],
                                [tok[i]], [pos[i]], [S[i]])
        assert np.array_equal(r1.logits[0], rb.logits[i])
    r0 = Oracle(cfg, w).step([a.copy() for a in kc], [a.copy() for a in vc], tok, [S[0], S[1]], S)
    assert not np.array_equal(r0.logits[0], rb.logits[0])


def test_toy_residual_only_model_is_norm_of_embedding(oracle_lib):
    # With W_o = W_d = 0 the residual stream stays the embedding row: logits = W_lm rms(E[t]) g_f.
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    w["layers"] = [dict(lw, wo=np.zeros_like(lw["wo"]), wd=np.zeros_like(lw["wd"])) for lw in w["layers"]]
    tok = make_start(cfg)
    r = Oracle(cfg, w).step(kc, vc, tok, S, S, precision="f64")
    for i, t in enumerate(tok):
        x = brute.bf(w["embed"][t])
        af = x / np.sqrt(np.mean(x * x) + cfg["rms_eps"]) * brute.bf(w["final_norm"])
        assert np.allclose(r.logits[i], brute.bf(w["lm_head"]) @ af, rtol=1e-12, atol=1e-14)


def test_oracle_rejects_bad_inputs(oracle_lib):
    from oracle.oracle import Oracle
    cfg, w, kc, vc, S = _toy()
    orc = Oracle(cfg, w)
    with pytest.raises(ValueError):
        orc.step(kc, vc, [cfg["vocab"], 0], S, S)
    with pytest.raises(ValueError):
        orc.step(kc, vc, [0, 0], S, [cfg["max_ctx"], 0])


# ---- Eq. 2 / Eq. 3 pinned by the paper's printed numbers -------------------------------

def test_eq2_bytes_and_mbu_match_paper_appendix():
    """The paper's printed worked example (tests/golden/eq2_qwen3_0.6b_b1x128.json): Qwen3-0.6B at
    b1 x 128 runs 1009.6 us per step, printed as 35.7% MBU at 3350 GB/s."""
    import json
    import os
    from paper_2609_12379_amd.metrics import step_bytes, mbu
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "eq2_qwen3_0.6b_b1x128.json")))
    cfg = get_config("qwen3-0.6b")
    for k, v in g["model"].items():
        if k != "element_bytes":
            assert cfg[k] == v, k
    B = step_bytes(cfg, g["context"], b=g["batch"])
    # weights 1.19205 GB + KV 14.68 MB + one embedding row
    assert B == pytest.approx(1.20665e9, rel=2e-5)
    assert round(100 * mbu(B, g["step_us"] * 1e-6, g["peak_gb_per_s"] * 1e9), 1) == g["mbu_pct_printed"]
    # a dropped KV term or a full-table embedding term would change the printed figure
    B_nokv = B - 2 * cfg["n_layers"] * cfg["n_kv_heads"] * cfg["head_dim"] * g["context"] * 2
    assert round(100 * mbu(B_nokv, g["step_us"] * 1e-6, g["peak_gb_per_s"] * 1e9), 1) != g["mbu_pct_printed"]

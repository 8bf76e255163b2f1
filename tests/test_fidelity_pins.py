"""Pins of the paper-fidelity measures (Sec. 4.2: Eq. 4, Eq. 5, Eq. 6) and of the references they
use: closed forms, hand-computed cases and an exact reproduction of the oracle's float32 step."""
import math

import numpy as np
import pytest

from oracle import fidelity as F
from oracle import oracle as O


# ---- Eq. 4 ---------------------------------------------------------------------------------

def test_delta_zero_on_identical_rows_and_symmetric():
    rng = np.random.default_rng(1)
    X = [rng.normal(size=7), rng.normal(size=3)]
    Y = [x + rng.normal(scale=1e-3, size=x.size) for x in X]
    assert F.delta(X, X) == 0.0
    assert F.delta(X, Y) == F.delta(Y, X)
    assert F.delta([np.zeros(4)], [np.zeros(4)]) == 0.0      # eps keeps 0/0 out


def test_delta_hand_values():
    # 1 against 3: 2*2 / (1 + 3 + eps) per element
    assert F.delta([np.ones(5)], [3 * np.ones(5)]) == pytest.approx(4 / (4 + 1e-6), rel=1e-15)
    # a sign flip is the largest distance, 2 (less the eps share)
    x = np.array([0.5, -2.0, 3.0])
    assert F.delta([x], [-x]) == pytest.approx(np.mean(4 * np.abs(x) / (2 * np.abs(x) + 1e-6)), rel=1e-15)


def test_delta_averages_rows_not_elements():
    # one 2-element row at distance ~1, one 6-element row at 0: the mean of the row means is
    # ~0.5, where pooling the 8 elements would give ~0.25
    X = [np.ones(2), np.ones(6)]
    Y = [3 * np.ones(2), np.ones(6)]
    assert F.delta(X, Y) == pytest.approx(0.5 * 4 / (4 + 1e-6), rel=1e-15)


# ---- Eq. 5 ---------------------------------------------------------------------------------

def test_eps_zero_on_golden_and_shift_invariant():
    rng = np.random.default_rng(2)
    G = rng.normal(size=(3, 200))
    assert F.eps_logits(G, G) == (0.0, 0.0)
    e, emax = F.eps_logits(G + 5.0, G)          # log-softmax ignores a constant per tap
    assert e < 1e-12 and emax < 1e-12


def test_eps_hand_value_two_entries():
    G = np.array([[0.0, math.log(3.0)]])        # softmax (1/4, 3/4)
    E = np.array([[0.0, 0.0]])                  # softmax (1/2, 1/2)
    e, emax = F.eps_logits(E, G, k=2)
    assert e == pytest.approx((math.log(2.0) + math.log(1.5)) / 2, rel=1e-14)
    assert emax == pytest.approx(math.log(2.0), rel=1e-14)


def test_eps_evaluates_at_the_goldens_top_entries():
    G = np.array([[5.0, 0.0, 0.0, 0.0]])
    E = np.array([[0.0, 0.0, 0.0, 9.0]])
    e, _ = F.eps_logits(E, G, k=1)
    want = abs(F.log_softmax(E[0])[0] - F.log_softmax(G[0])[0])
    assert e == pytest.approx(want, rel=1e-14)


def test_eps_mean_of_means_and_max_of_maxes():
    G = np.array([[0.0, math.log(3.0)], [0.0, 0.0]])
    E = np.array([[0.0, 0.0], [0.0, 0.0]])
    e, emax = F.eps_logits(E, G, k=2)
    assert e == pytest.approx((math.log(2.0) + math.log(1.5)) / 4, rel=1e-14)
    assert emax == pytest.approx(math.log(2.0), rel=1e-14)


# ---- Eq. 6 ---------------------------------------------------------------------------------

def test_alpha_reads_the_share_of_the_narrowing():
    rng = np.random.default_rng(3)
    A = rng.normal(size=50)
    d = rng.normal(scale=1e-3, size=50)
    An = A + d
    assert F.alpha(A, A, An) == 0.0
    assert F.alpha(An, A, An) == pytest.approx(1.0, rel=1e-12)
    assert F.alpha(A + 0.3 * d, A, An) == pytest.approx(0.3, rel=1e-9)
    ortho = rng.normal(size=50)
    ortho -= (ortho @ d) / (d @ d) * d           # a reordering error unrelated to d
    assert abs(F.alpha(A + ortho, A, An)) < 1e-9
    assert F.alpha(A + 1.0, A, A) is None        # the two references coincide: abstain


# ---- narrowing and the per-operator references ---------------------------------------------

def test_narrow_rounds_to_nearest_even():
    x = np.array([1.0, 1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, 1 + 3 * 2.0 ** -9, -(1 + 2.0 ** -8)])
    want = np.array([1.0, 1.0, 1 + 2.0 ** -6, 1 + 2.0 ** -7, -1.0])
    np.testing.assert_array_equal(F.narrow(x), want)


def _bf16(a):
    return O.to_bf16(np.asarray(a, np.float32), "f32")


def test_attention_ref_closed_forms():
    V = _bf16([[0.5, -1.25], [2.0, 0.75]])
    K1 = _bf16([[0.3, 0.1]])
    # one slot: the output is that slot's value row, whatever is narrowed
    for nq in (False, True):
        for npv in (False, True):
            o = F.attention_ref([0.7, -0.2], K1, V[:1], narrow_q=nq, narrow_p=npv)
            np.testing.assert_array_equal(o, F.bf16_values(V[0]).astype(np.float64))
    # equal scores: the mean of the value rows
    K0 = _bf16([[0.0, 0.0], [0.0, 0.0]])
    o = F.attention_ref([0.7, -0.2], K0, V, narrow_p=True)
    np.testing.assert_allclose(o, F.bf16_values(V).astype(np.float64).mean(axis=0), rtol=1e-15)


def test_attention_ref_ln3_scores_and_the_narrowed_weights():
    # d = 2, K rows (1, 0) and (0, 0), q = (sqrt(2) ln 3, 0): scores ln 3 and 0, so the weights
    # are (1, 1/3). Unnarrowed: (3/4, 1/4). Narrowed: 1/3 rounds to bf16 0.333984375 for the
    # weighted sum, the normaliser stays 4/3.
    K = _bf16([[1.0, 0.0], [0.0, 0.0]])
    V = _bf16([[1.0, 0.0], [0.0, 1.0]])
    q = [math.sqrt(2.0) * math.log(3.0), 0.0]
    np.testing.assert_allclose(F.attention_ref(q, K, V), [0.75, 0.25], rtol=1e-14)
    np.testing.assert_allclose(F.attention_ref(q, K, V, narrow_p=True), [0.75, 0.333984375 * 0.75], rtol=1e-14)


def test_attention_ref_matches_the_oracle_attend():
    rng = np.random.default_rng(4)
    K = _bf16(rng.normal(size=(37, 16)))
    V = _bf16(rng.normal(size=(37, 16)))
    q = rng.normal(size=16)
    np.testing.assert_allclose(F.attention_ref(q, K, V), O.attend(q, K, V, "f64"), rtol=1e-12, atol=1e-14)


def test_mlp_ref_identity_weights():
    I = _bf16(np.eye(2))
    a = np.array([1.0, -2.0])
    silu = a / (1 + np.exp(-a))
    want = silu * a
    np.testing.assert_allclose(F.mlp_ref(I, I, I, a), want, rtol=1e-14)
    np.testing.assert_array_equal(F.mlp_ref(I, I, I, a, narrow_m=True), F.narrow(want))
    a3 = np.array([1 / 3, -2.0])
    np.testing.assert_allclose(F.mlp_ref(I, I, I, a3, narrow_in=True),
                               F.mlp_ref(I, I, I, F.narrow(a3)), rtol=1e-15)


def test_gemv_ref_narrowing_only_moves_unrepresentable_inputs():
    rng = np.random.default_rng(5)
    W = _bf16(rng.normal(size=(9, 12)))
    xb = F.bf16_values(_bf16(rng.normal(size=12))).astype(np.float64)
    np.testing.assert_array_equal(F.gemv_ref(W, xb), F.gemv_ref(W, xb, narrow_in=True))
    x = rng.normal(size=12)
    assert not np.array_equal(F.gemv_ref(W, x), F.gemv_ref(W, x, narrow_in=True))


# ---- the bf16 reference decoder ------------------------------------------------------------

def _toy():
    from synthetic import make_workload, as_u16
    wl = make_workload("toy", gains="uniform")
    w = {k: as_u16(v) for k, v in wl.weights.items() if k != "layers" and v is not None}
    w["layers"] = [{k: as_u16(v) for k, v in lw.items()} for lw in wl.weights["layers"]]
    kc = [as_u16(t).copy() for t in wl.kcache]
    vc = [as_u16(t).copy() for t in wl.vcache]
    return wl, w, kc, vc


def test_bf16_decoder_without_rounding_is_the_oracle_f32_step():
    wl, w, kc, vc = _toy()
    cfg, S = wl.cfg, wl.S
    kc2, vc2 = [a.copy() for a in kc], [a.copy() for a in vc]
    orc = O.Oracle(cfg, w)
    dec = F.Bf16Decoder(cfg, w, rounding=False)
    tok = list(wl.start)
    for t in range(2):
        pos = [s + t for s in S]
        r = orc.step(kc, vc, tok, pos, pos, precision="f32")
        lg = dec.step(kc2, vc2, tok, pos, pos)
        np.testing.assert_array_equal(lg, r.logits)
        for l in range(cfg["n_layers"]):
            np.testing.assert_array_equal(kc2[l], kc[l])
            np.testing.assert_array_equal(vc2[l], vc[l])
        tok = [int(v) for v in r.next_ids]


def test_bf16_decoder_rounds_and_stays_close():
    wl, w, kc, vc = _toy()
    cfg, S = wl.cfg, wl.S
    kc2, vc2 = [a.copy() for a in kc], [a.copy() for a in vc]
    r = O.Oracle(cfg, w).step(kc, vc, list(wl.start), S, S, precision="f32")
    lg = F.Bf16Decoder(cfg, w).step(kc2, vc2, list(wl.start), S, S)
    np.testing.assert_array_equal(F.narrow(lg), lg)          # logits are bf16 values
    assert not np.array_equal(lg, r.logits)
    rel = np.linalg.norm(lg - r.logits) / np.linalg.norm(r.logits)
    assert rel < 5e-2

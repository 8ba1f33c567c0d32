"""Pins the forward-only oracle (action log-prob and policy entropy) to facts other than itself (CPU only).

The entropy is -sum_v p_v log p_v of p = softmax(z); the paper tracks it per token, averaged over the loss
mask, to compare GRPO with RAFT++ (Sec. 5).  Pins: closed forms (constant row: log V; two-level rows; the
binary entropy of a two-logit row), shift invariance, the limit of a peaked row, scipy's entropy of the
softmax, and brute-force sums in Python.
"""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle


def test_constant_row_is_uniform():
    # every p_v = 1/V: H = log V and every log-prob is -log V, whatever the constant
    for V, c in ((1, 0.0), (7, 3.5), (1000, -40.0)):
        z = np.full((1, V), c, np.float64)
        r = oracle.logp_entropy(z, [V - 1])
        assert r.flags == 0
        assert r.token_entropy[0] == pytest.approx(math.log(V), abs=1e-12)
        assert r.token_logp[0] == pytest.approx(-math.log(V), abs=1e-12)


def test_two_level_rows_closed_form():
    # k logits at a and V - k at b: p_hi = e^a / (k e^a + (V - k) e^b), p_lo likewise
    for V, k, a, b in ((10, 1, 2.0, 0.0), (64, 5, 0.5, -1.5), (200, 199, -3.0, 4.0)):
        z = np.full((1, V), b)
        z[0, :k] = a
        Z = k * math.exp(a) + (V - k) * math.exp(b)
        p_hi, p_lo = math.exp(a) / Z, math.exp(b) / Z
        H = -(k * p_hi * math.log(p_hi) + (V - k) * p_lo * math.log(p_lo))
        r = oracle.logp_entropy(z, [0])
        assert r.token_entropy[0] == pytest.approx(H, rel=1e-12)
        assert r.token_logp[0] == pytest.approx(math.log(p_hi), rel=1e-12)


def test_masked_columns_drop_out():
    # -inf logits carry zero probability and no entropy term (0 log 0 = 0): k equal finite logits among V - k
    # masked ones give H = log k and log-prob -log k exactly, as the uniform row of width k does; a masked row
    # mixed with a two-level row gives that row's closed form
    for V, k, c in ((8, 1, 0.0), (100, 7, 2.5), (4096, 1000, -30.0)):
        z = np.full((1, V), -np.inf)
        z[0, V - k:] = c
        r = oracle.logp_entropy(z, [V - 1])
        assert r.flags == 0
        assert r.token_entropy[0] == pytest.approx(math.log(k), abs=1e-12)
        assert r.token_logp[0] == pytest.approx(-math.log(k), abs=1e-12)
    z = np.array([[-np.inf, 1.0, -np.inf, 0.0, 0.0, -np.inf]])
    Z = math.e + 2.0
    H = -(math.e / Z * (1.0 - math.log(Z)) + 2.0 / Z * (-math.log(Z)))
    r = oracle.logp_entropy(z, [1])
    assert r.token_entropy[0] == pytest.approx(H, rel=1e-13)
    assert r.token_logp[0] == pytest.approx(1.0 - math.log(Z), rel=1e-13)


def test_two_logits_binary_entropy():
    # V = 2: H = h(sigmoid(z1 - z0)), h(q) = -q log q - (1 - q) log(1 - q)
    for d in (-6.0, -0.3, 0.0, 1.7, 9.0):
        q = 1.0 / (1.0 + math.exp(-d))
        h = -q * math.log(q) - (1 - q) * math.log(1 - q)
        r = oracle.logp_entropy(np.array([[0.25, 0.25 + d]]), [1])
        assert r.token_entropy[0] == pytest.approx(h, rel=1e-12, abs=1e-15)
        assert r.token_logp[0] == pytest.approx(math.log(q), rel=1e-12)


def test_matches_scipy_entropy_of_softmax():
    rng = np.random.default_rng(3)
    z = rng.normal(0, 2.0, (6, 333))
    a = rng.integers(0, 333, 6).astype(np.int32)
    r = oracle.logp_entropy(z, a)
    p = scipy.special.softmax(z, axis=1)
    np.testing.assert_allclose(r.token_entropy, scipy.stats.entropy(p, axis=1), rtol=1e-12)
    np.testing.assert_allclose(r.token_logp, scipy.special.log_softmax(z, axis=1)[np.arange(6), a], rtol=1e-12)


def test_shift_invariance():
    rng = np.random.default_rng(4)
    z = rng.normal(0, 1.0, (4, 50))
    a = np.array([0, 10, 20, 49], np.int32)
    r0 = oracle.logp_entropy(z, a)
    r1 = oracle.logp_entropy(z + 123.0, a)
    np.testing.assert_allclose(r1.token_entropy, r0.token_entropy, rtol=1e-10)
    np.testing.assert_allclose(r1.token_logp, r0.token_logp, rtol=1e-10)


def test_peaked_row_has_zero_entropy():
    # one logit 1000 above the rest: every other p_v underflows, H is exactly 0 and that action's log-prob 0
    z = np.zeros((1, 100))
    z[0, 37] = 1000.0
    r = oracle.logp_entropy(z, [37])
    assert r.token_entropy[0] == 0.0
    assert r.token_logp[0] == 0.0


def test_brute_force_small_rows():
    rng = np.random.default_rng(5)
    for _ in range(5):
        V = int(rng.integers(2, 12))
        row = rng.normal(0, 3.0, V)
        Z = sum(math.exp(x) for x in row)
        H = -sum(math.exp(x) / Z * math.log(math.exp(x) / Z) for x in row)
        a = int(rng.integers(0, V))
        r = oracle.logp_entropy(row[None, :], [a])
        assert r.token_entropy[0] == pytest.approx(H, rel=1e-11)
        assert r.token_logp[0] == pytest.approx(row[a] - math.log(Z), rel=1e-11, abs=1e-13)


def test_bf16_and_stride_and_row_window():
    rng = np.random.default_rng(6)
    vals = rng.normal(0, 2.0, (5, 40)).astype(np.float32)
    bits = (vals.view(np.uint32) >> 16).astype(np.uint16)
    exact = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    a = np.array([1, 2, 3, 4, 5], np.int32)
    # V = 32 of a 40-wide stride, rows 2..4 of a window held from row 1
    r = oracle.logp_entropy(bits[1:], a, V=32, row_begin=2, row_end=5, row_offset=1)
    p = scipy.special.softmax(exact[2:5, :32], axis=1)
    np.testing.assert_allclose(r.token_entropy, scipy.stats.entropy(p, axis=1), rtol=1e-12)
    np.testing.assert_allclose(r.token_logp, np.log(p[np.arange(3), a[2:5]]), rtol=1e-12)


def test_out_of_range_action_flags_and_zero_logp():
    z = np.zeros((2, 8))
    r = oracle.logp_entropy(z, [8, -1])
    assert r.flags & oracle.ERR_ACTION
    assert (r.token_logp == 0.0).all()
    np.testing.assert_allclose(r.token_entropy, math.log(8), rtol=1e-14)


def test_logp_agrees_with_the_loss_oracle():
    rng = np.random.default_rng(7)
    T, V = 6, 30
    z = rng.normal(0, 1.5, (T, V))
    a = rng.integers(0, V, T).astype(np.int32)
    seg = oracle.segments(T, np.arange(T + 1), np.array([0, T]))
    lr = oracle.loss_rows(z, a, np.zeros(T, np.float32), None, [1.0], seg, 1, want_dlogits=False)
    r = oracle.logp_entropy(z, a)
    np.testing.assert_allclose(r.token_logp, lr.token_logp, rtol=0, atol=0)

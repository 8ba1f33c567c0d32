"""Pins of the oracle's importance-ratio statistics (oracle.ratio_stats) and of the loss sum's cancellation ratio.

The ratios are those of Eq. 1 (Sec. 3.2): r = pi/pi_prox, the one the eps clip acts on, and rho = pi/pi_behave, the
importance weight; the paper reports how often the clip engages (Sec. 4.3, Sec. 5).  Each pin fixes the values by
something other than the formula itself: exact ratios of one (a one-column vocabulary has log-prob 0 exactly), hand
values of e^(+-ln 2), the inclusive clip range at its edge, the clip decisions of the loss oracle's surrogate (a
token whose gradient the eps clip cut must lie outside the range, and which tokens are cut follows from the sign of
the advantage), exclusion of tokens outside the loss, and math.fsum / min / max over the same values.  The
cancellation ratio has a closed form for ratio-one tokens: s_t = A_i, so the loss is -sum_i w_i n_i A_i.
"""
import math

import numpy as np
import pytest

import oracle

LN2 = math.log(2.0)


def test_one_column_vocabulary_gives_ratio_one():
    # V = 1: l = z - log e^z = 0 exactly whatever z is; with behave = prox = 0 both ratios are exactly 1
    T = 37
    rng = np.random.default_rng(3)
    z = rng.normal(0, 3, (T, 1)).astype(np.float32)
    seg = oracle.segments(T, np.array([0, 20, T], np.int32), np.array([0, 1, 2], np.int32))
    zero = np.zeros(T, np.float32)
    res = oracle.loss_rows(z, np.zeros(T, np.int32), zero, zero, np.array([1.0, -1.0]), seg, 2, V=1,
                           want_dlogits=False)
    assert (res.token_logp == 0.0).all()
    st = oracle.ratio_stats(res.token_logp, zero, zero, oracle.valid_tokens(np.zeros(T), 1, seg))
    assert st.tolist() == [T, 1.0, 1.0, T, 1.0, 1.0, 0.0, T]


def test_hand_values():
    l = np.zeros(3)
    b = np.array([0.0, -LN2, LN2], np.float32)  # rho = 1, 2, 1/2
    p = np.array([0.0, -LN2, 0.0], np.float32)  # r   = 1, 2, 1
    v = np.ones(3, np.int32)
    st = oracle.ratio_stats(l, b, p, v, 0.2, 0.2)
    np.testing.assert_allclose(st[:6], [4.0, 1.0, 2.0, 3.5, 0.5, 2.0], rtol=1e-7)
    assert st[6] == 1 and st[7] == 3  # only r = 2 lies outside [0.8, 1.2]
    coupled = oracle.ratio_stats(l, b, None, v, 0.2, 0.2)  # prox = behave: r is rho
    np.testing.assert_allclose(coupled[:3], [3.5, 0.5, 2.0], rtol=1e-7)
    assert coupled[6] == 2
    assert oracle.ratio_stats(l, b, None, v, 0.6, 1.5)[6] == 0  # [0.4, 2.5] holds every ratio


def test_zero_width_range_keeps_ratio_one_inside():
    l = np.array([0.0, 0.5, -0.5])
    b = np.array([0.0, 0.5, -0.5], np.float32)  # r = 1 exactly on every token (l - b = 0 in fp64)
    st = oracle.ratio_stats(l, b, None, np.ones(3, np.int32), 0.0, 0.0)
    assert st.tolist() == [3.0, 1.0, 1.0, 3.0, 1.0, 1.0, 0.0, 3.0]


def test_excluded_tokens_and_empty_set():
    rng = np.random.default_rng(5)
    n = 200
    l = rng.normal(-3, 1, n)
    b = (l + rng.normal(0, 0.2, n)).astype(np.float32)
    p = (l + rng.normal(0, 0.2, n)).astype(np.float32)
    v = (rng.random(n) < 0.7).astype(np.int32)
    keep = v.astype(bool)
    np.testing.assert_array_equal(oracle.ratio_stats(l, b, p, v),
                                  oracle.ratio_stats(l[keep], b[keep], p[keep], np.ones(keep.sum(), np.int32)))
    empty = oracle.ratio_stats(l, b, p, np.zeros(n, np.int32))
    assert empty.tolist() == [0.0, math.inf, -math.inf, 0.0, math.inf, -math.inf, 0.0, 0.0]


def test_against_fsum_min_max():
    rng = np.random.default_rng(6)
    n = 1000
    l = rng.normal(-2, 1, n)
    b = (l + rng.normal(0, 0.3, n)).astype(np.float32)
    p = (l + rng.normal(0, 0.3, n)).astype(np.float32)
    st = oracle.ratio_stats(l, b, p, np.ones(n, np.int32), 0.2, 0.28)
    r = [math.exp(li - float(pi)) for li, pi in zip(l, p)]
    rho = [math.exp(li - float(bi)) for li, bi in zip(l, b)]
    assert abs(st[0] - math.fsum(r)) <= 1e-12 * st[0] and st[1] == min(r) and st[2] == max(r)
    assert abs(st[3] - math.fsum(rho)) <= 1e-12 * st[3] and st[4] == min(rho) and st[5] == max(rho)
    assert st[6] == sum(1 for x in r if x < 0.8 or x > 1.28)


@pytest.mark.parametrize("seed", [0, 1])
def test_outside_count_against_surrogate_clip_decisions(seed):
    # coupled ratio, no dual clip: the eps clip cuts the gradient exactly where the clipped term is the smaller
    # one and the ratio is outside the range: A > 0 with r > 1 + eps, A < 0 with r < 1 - eps.  Every cut token is
    # outside; the outside tokens that are not cut are A > 0 with r < 1 - eps and A < 0 with r > 1 + eps.
    rng = np.random.default_rng(seed)
    T, V, N = 600, 64, 8
    z = rng.normal(0, 1, (T, V)).astype(np.float32)
    sto = np.linspace(0, T, N + 1).astype(np.int32)
    seg = oracle.segments(T, sto, np.arange(N + 1, dtype=np.int32))
    actions = rng.integers(0, V, T).astype(np.int32)
    A = np.array([1.0, -1.0, 0.5, -0.5, 2.0, -2.0, 1.5, -1.5])
    l = oracle.loss_rows(z, actions, np.zeros(T, np.float32), None, A, seg, N, want_dlogits=False).token_logp
    b = (l + rng.normal(0, 0.3, T)).astype(np.float32)  # wide noise: many tokens outside [0.8, 1.2]
    res = oracle.loss_rows(z, actions, b, None, A, seg, N, want_dlogits=False)
    st = oracle.ratio_stats(res.token_logp, b, None, oracle.valid_tokens(actions, V, seg))
    r = np.exp(res.token_logp - b.astype(np.float64))
    At = A[seg.tok_traj]
    cut = (res.token_state & 1).astype(bool)
    lo, hi = r < 0.8, r > 1.2
    assert cut.sum() > 20 and st[6] > cut.sum()
    np.testing.assert_array_equal(cut, ((At > 0) & hi) | ((At < 0) & lo))
    assert st[6] == cut.sum() + ((At > 0) & lo).sum() + ((At < 0) & hi).sum()


def test_invalid_action_leaves_the_statistics():
    rng = np.random.default_rng(8)
    T, V = 40, 32
    z = rng.normal(0, 1, (T, V)).astype(np.float32)
    seg = oracle.segments(T, np.array([0, 25, T], np.int32), np.array([0, 1, 2], np.int32))
    actions = rng.integers(0, V, T).astype(np.int32)
    actions[[3, 30]] = [V, -1]
    valid = oracle.valid_tokens(actions, V, seg)
    assert valid.sum() == T - 2 and valid[3] == 0 and valid[30] == 0
    bad = oracle.segments(T, np.array([0, 25, T + 1], np.int32), np.array([0, 1, 2], np.int32))
    assert oracle.valid_tokens(actions, V, bad).sum() == 0


def test_cancellation_ratio_closed_form():
    # one group of G = 2: rewards (1, 0) give A = +-1/sqrt(2) (ddof 1); ratio one makes s_t = A_i, so
    # loss = -w (n_1 A_1 + n_2 A_2) and sum |w s_t| = w (n_1 + n_2) |A|: with n = (3, 5), kappa = 8 / 2 = 4
    A = oracle.advantages(np.array([1.0, 0.0], np.float32), 2)
    np.testing.assert_allclose(A, [2 ** -0.5, -(2 ** -0.5)], rtol=1e-15)
    T, V = 8, 1  # V = 1: l = 0, so behave = 0 gives ratio one exactly
    seg = oracle.segments(T, np.array([0, 3, T], np.int32), np.array([0, 1, 2], np.int32))
    res = oracle.loss_rows(np.zeros((T, V), np.float32), np.zeros(T, np.int32), np.zeros(T, np.float32), None, A,
                           seg, 2, V=V, k=10.0, want_dlogits=False)
    w = 1.0 / (1 * 2 * 10.0)
    assert abs(res.loss - (-w * (3 - 5) * 2 ** -0.5)) <= 1e-15
    assert abs(res.abs_terms - w * 8 * 2 ** -0.5) <= 1e-15
    assert abs(res.kappa - 4.0) <= 1e-12
    assert oracle.cancellation_ratio([1.0, 2.0, 3.0]) == 1.0  # one sign: no cancellation
    assert oracle.cancellation_ratio([1.0, -1.0]) == math.inf

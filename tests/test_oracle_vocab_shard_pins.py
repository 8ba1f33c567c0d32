"""Pins the vocabulary-shard oracle (per-shard max, sum exp, action logit, and their merge) to facts other than
itself (CPU only).

With the vocabulary split over devices, each shard reduces its columns of a row to (m, s, z_a) and the row's
log-sum-exp is recovered from the shards by the log-sum-exp merge.  Pins: the merge of any split equals the
whole row's log-sum-exp from scipy and from the loss oracle (an independent routine, which gathers the action
logit itself), closed forms (constant and two-level shards), ownership of the action logit, shards of -inf
logits, bf16 inputs, and brute-force sums in Python.
"""
import math

import numpy as np
import pytest
import scipy.special

import oracle


def split_stats(z, actions, bounds):
    return [oracle.vocab_shard_stats(z[:, b0:b1], actions, b0) for b0, b1 in zip(bounds[:-1], bounds[1:])]


@pytest.mark.parametrize("bounds", [[0, 50], [0, 25, 50], [0, 1, 2, 49, 50], [0, 7, 19, 20, 41, 50]])
def test_merge_of_any_split_is_the_row_lse(bounds):
    rng = np.random.default_rng(len(bounds))
    z = rng.normal(0, 3.0, (9, 50))
    a = rng.integers(0, 50, 9).astype(np.int32)
    lse, za = oracle.vocab_merge(split_stats(z, a, bounds))
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-13)
    np.testing.assert_array_equal(za, z[np.arange(9), a])
    # the loss oracle's log-prob is z_a - lse from its own log-sum-exp and gather
    seg = oracle.segments(9, np.arange(10), np.array([0, 9]))
    lr = oracle.loss_rows(z, a, np.zeros(9, np.float32), None, [1.0], seg, 1, want_dlogits=False)
    np.testing.assert_allclose(za - lse, lr.token_logp, rtol=1e-12, atol=1e-13)


def test_constant_and_two_level_shards_closed_form():
    z = np.full((1, 12), -2.5)
    st = oracle.vocab_shard_stats(z, [3], 0)
    assert st.m[0] == -2.5 and st.s[0] == 12.0 and st.za[0] == -2.5
    # k columns at hi, the rest at lo: m = hi, s = k + (V - k) e^(lo - hi)
    for V, k, hi, lo in ((10, 1, 2.0, 0.0), (64, 5, 0.5, -1.5), (7, 6, 4.0, -3.0)):
        z = np.full((1, V), lo)
        z[0, :k] = hi
        st = oracle.vocab_shard_stats(z, [200], 40)
        assert st.m[0] == hi
        assert st.s[0] == pytest.approx(k + (V - k) * math.exp(lo - hi), rel=1e-14)
        assert st.za[0] == -math.inf  # action 200 is not in columns [40, 40 + V)


def test_action_logit_belongs_to_exactly_one_shard():
    rng = np.random.default_rng(2)
    z = rng.normal(0, 1.0, (4, 30))
    a = np.array([0, 9, 10, 29], np.int32)
    st = split_stats(z, a, [0, 10, 20, 30])
    owner = a // 10
    for g in range(3):
        for t in range(4):
            if owner[t] == g:
                assert st[g].za[t] == z[t, a[t]]
            else:
                assert st[g].za[t] == -math.inf


def test_invalid_action_owned_by_no_shard():
    z = np.zeros((2, 20))
    a = np.array([-1, 20], np.int32)
    _, za = oracle.vocab_merge(split_stats(z, a, [0, 8, 20]))
    assert (za == -math.inf).all()


def test_shard_of_minus_inf_logits_is_ignored_by_the_merge():
    z = np.random.default_rng(3).normal(0, 1.0, (3, 16))
    z[:, 8:] = -np.inf
    st = split_stats(z, np.array([1, 2, 3], np.int32), [0, 8, 16])
    assert (st[1].m == -math.inf).all() and (st[1].s == 0.0).all()
    lse, _ = oracle.vocab_merge(st)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z[:, :8], axis=1), rtol=1e-13)


def test_bf16_inputs_and_strided_shard():
    rng = np.random.default_rng(4)
    vals = rng.normal(0, 2.0, (5, 40)).astype(np.float32)
    bits = (vals.view(np.uint32) >> 16).astype(np.uint16)
    exact = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    a = np.array([30, 31, 5, 39, 33], np.int32)
    # columns 24..35 of a 40-wide row (V = 12 of stride 16 after slicing from column 24), rows 1..4
    st = oracle.vocab_shard_stats(bits[1:, 24:40], a, 24, V=12, row_begin=2, row_end=5, row_offset=1)
    ref = exact[2:5, 24:36]
    np.testing.assert_array_equal(st.m, ref.max(axis=1))
    np.testing.assert_allclose(st.s, np.exp(ref - ref.max(axis=1, keepdims=True)).sum(axis=1), rtol=1e-14)
    # rows 2 and 3 act on columns 5 and 39, outside [24, 36); row 4 on column 33
    np.testing.assert_array_equal(st.za, [-math.inf, -math.inf, exact[4, 33]])


def test_brute_force_small_shards():
    rng = np.random.default_rng(5)
    for _ in range(5):
        V = int(rng.integers(2, 10))
        row = rng.normal(0, 3.0, V)
        v0 = int(rng.integers(0, 100))
        a = v0 + int(rng.integers(0, V))
        st = oracle.vocab_shard_stats(row[None, :], [a], v0)
        m = max(row)
        assert st.m[0] == m
        assert st.s[0] == pytest.approx(sum(math.exp(x - m) for x in row), rel=1e-13)
        assert st.za[0] == row[a - v0]

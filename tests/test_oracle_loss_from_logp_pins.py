"""oracle.loss_from_logp: Eq. 1 from per-token log-probs, for a second normaliser or parameter set without a second
log-softmax.  Pinned to oracle.loss_rows (itself pinned by finite differences, torch autograd and closed forms in
tests/test_oracle_pins.py): fed loss_rows' own log-probs it must give the same per-token terms, coefficients, clip
states, per-trajectory losses and flags, bit for bit, under both normalisers, coupled and decoupled ratios, the dual
clip, an action outside the vocabulary and malformed offsets."""
import numpy as np
import pytest

import oracle


def _batch(seed, T=300, V=50, N=8):
    rng = np.random.default_rng(seed)
    z = rng.normal(0, 2, (T, V)).astype(np.float32)
    sto = np.sort(rng.integers(0, T, 3 * N - 1)).astype(np.int32)
    sto = np.concatenate([[0], sto, [T]]).astype(np.int32)
    tso = np.concatenate([[0], np.sort(rng.choice(np.arange(1, 3 * N), N - 1, replace=False)), [3 * N]]).astype(np.int32)
    actions = rng.integers(0, V, T).astype(np.int32)
    seg = oracle.segments(T, sto, tso)
    l = oracle.loss_rows(z, actions, np.zeros(T, np.float32), None, np.zeros(N), seg, 4, want_dlogits=False).token_logp
    behave = (l + rng.normal(0, 0.4, T)).astype(np.float32)
    prox = (l + rng.normal(0, 0.4, T)).astype(np.float32)
    A = oracle.advantages((rng.random(N) < 0.5).astype(np.float32), 4)
    return z, actions, behave, prox, A, sto, tso, seg


@pytest.mark.parametrize("norm", [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K])
@pytest.mark.parametrize("decoupled", [False, True])
@pytest.mark.parametrize("c", [0.0, 1.5])
def test_matches_loss_rows_bitwise(norm, decoupled, c):
    z, actions, behave, prox, A, sto, tso, seg = _batch(3)
    actions[17] = 50  # outside the vocabulary
    p = prox if decoupled else None
    kw = dict(norm=norm, k=3.0, eps_low=0.2, eps_high=0.28, dual_clip_c=c, grad_scale=0.5, n_groups_total=5.0)
    ref = oracle.loss_rows(z, actions, behave, p, A, seg, 4, want_dlogits=False, row_begin=10, row_end=290, **kw)
    got = oracle.loss_from_logp(ref.token_logp, actions, behave, p, A, seg, 4, V=50, row_begin=10, row_end=290, **kw)
    assert got.flags == ref.flags == oracle.ERR_ACTION
    for f in ("token_contrib", "token_g", "token_state", "traj_loss"):
        np.testing.assert_array_equal(getattr(got, f), getattr(ref, f), err_msg=f)
    assert got.loss == ref.loss
    if c > 0:
        assert ((ref.token_state >> 1) & 1).sum() > 0  # the dual clip engaged somewhere


def test_malformed_offsets():
    z, actions, behave, prox, A, sto, tso, _ = _batch(4)
    bad = sto.copy()
    bad[-1] += 1
    seg = oracle.segments(len(actions), bad, tso)
    ref = oracle.loss_rows(z, actions, behave, None, A, seg, 4, want_dlogits=False)
    got = oracle.loss_from_logp(ref.token_logp, actions, behave, None, A, seg, 4, V=50)
    assert got.flags == ref.flags == oracle.ERR_OFFSETS
    assert np.isnan(got.token_contrib).all() and np.isnan(got.loss)

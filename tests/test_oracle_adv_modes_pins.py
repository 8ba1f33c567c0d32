"""Pins the oracle's RAFT++ success-filter advantage and DAPO mixed-group mask (CPU only).

RAFT++ (Sec. 3.2, Table 5): no group normalisation, A_i = 1[r_i > 0].  DAPO dynamic sampling (Sec. 3.2):
groups whose rewards are all equal carry no signal and are skipped.  Pins: hand-written closed forms, brute
force over sets, and the link to the group-normalised advantage (a group is mixed exactly when its
normalised advantages are not all zero).
"""
import numpy as np

import oracle


def test_success_filter_closed_form():
    r = np.array([0.0, 1.0, 0.5, -1.0, 1e-30, -0.0, 3.0, 0.0], np.float32)
    want = np.array([0, 1, 1, 0, 1, 0, 1, 0], np.float64)
    got = oracle.advantages(r, 1, mode=oracle.ADV_SUCCESS_FILTER)
    assert (got == want).all()


def test_success_filter_ignores_grouping():
    rng = np.random.default_rng(0)
    r = (rng.random(64) < 0.4).astype(np.float32)
    a1 = oracle.advantages(r, 1, mode=oracle.ADV_SUCCESS_FILTER)
    a8 = oracle.advantages(r, 8, mode=oracle.ADV_SUCCESS_FILTER)
    assert (a1 == a8).all() and (a1 == r).all()


def test_mixed_groups_brute_force():
    rng = np.random.default_rng(1)
    for G in (1, 2, 8):
        r = (rng.random(G * 40) < 0.5).astype(np.float32)
        r[:G] = 1.0          # an all-success group
        r[G:2 * G] = 0.0     # an all-failure group
        mixed, n = oracle.mixed_groups(r, G)
        want = np.array([len(set(r[g * G:(g + 1) * G].tolist())) > 1 for g in range(40)], np.int32)
        assert (mixed == want).all() and n == want.sum()
        assert mixed[0] == 0 and mixed[1] == 0


def test_mixed_exactly_when_group_norm_advantage_nonzero():
    rng = np.random.default_rng(2)
    G = 8
    r = rng.choice([0.0, 0.25, 1.0], size=G * 30, p=[0.6, 0.1, 0.3]).astype(np.float32)
    r[5 * G:6 * G] = 0.25
    mixed, _ = oracle.mixed_groups(r, G)
    A = oracle.advantages(r, G).reshape(-1, G)
    assert ((np.abs(A).max(axis=1) > 0) == (mixed == 1)).all()


def test_paper_dynamic_sampling_batch():
    # Sec. 3.2: 16 mixed groups of G = 8 make the 128 trajectories of one training step
    rng = np.random.default_rng(3)
    groups = []
    while len(groups) < 16:
        g = (rng.random(8) < 0.4).astype(np.float32)
        m, _ = oracle.mixed_groups(g, 8)
        if m[0]:
            groups.append(g)
    r = np.concatenate(groups)
    mixed, n = oracle.mixed_groups(r, 8)
    assert len(r) == 128 and n == 16 and mixed.all()

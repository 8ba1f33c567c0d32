"""The seeded generator reproduces the workload structure it claims (CPU only)."""
import numpy as np
import pytest
import torch

from synth import CONFIGS, make_batch, make_structure


def test_tiny_structure():
    st = make_structure(CONFIGS["tiny"])
    assert st.T == 192 and len(st.rewards) == 4
    assert (st.traj_steps == 3).all() and (st.step_tokens == 16).all()
    assert st.rewards.min() == 0 and st.rewards.max() == 1


@pytest.mark.parametrize("name,T", [("v152k", 120000), ("long", 250000), ("fused", 65536)])
def test_calibrated_token_counts(name, T):
    cfg = CONFIGS[name]
    st = make_structure(cfg)
    assert st.T == T and st.step_tok_off[-1] == T
    assert (st.step_tokens >= 1).all()
    assert len(st.rewards) == cfg.n_groups * cfg.G
    # failures run longer than successes (Sec. 1, Sec. 5.1)
    fail = st.traj_steps[st.rewards == 0].mean()
    succ = st.traj_steps[st.rewards == 1].mean()
    assert fail > 1.5 * succ
    lo_f, hi_f = cfg.steps_fail
    assert st.traj_steps[st.rewards == 0].min() >= lo_f and st.traj_steps[st.rewards == 0].max() <= hi_f


def test_v32k_literal_recipe():
    st = make_structure(CONFIGS["v32k"])
    assert (st.step_tokens >= 16).all() and (st.step_tokens <= 256).all()
    assert 25000 < st.T < 50000
    assert ((st.traj_steps >= 2) & (st.traj_steps <= 15)).all()


def test_every_group_is_mixed():
    for name in CONFIGS:
        cfg = CONFIGS[name]
        st = make_structure(cfg)
        r = st.rewards.reshape(cfg.n_groups, cfg.G)
        assert (r.min(1) == 0).all() and (r.max(1) == 1).all()


def test_seeded_and_reproducible():
    a = make_batch("tiny")
    b = make_batch("tiny")
    assert torch.equal(a["logits"], b["logits"]) and torch.equal(a["actions"], b["actions"])
    assert torch.equal(a["behave"], b["behave"])
    c = make_batch("tiny", seed=99)
    assert not torch.equal(a["logits"], c["logits"])


def test_gumbel_actions_follow_softmax():
    # a 3-token vocabulary repeated many times: empirical frequencies ~ softmax
    from synth.rollouts import gumbel_max_actions
    z = torch.tensor([[0.0, 1.0, 2.0]]).repeat(200000, 1)
    a = gumbel_max_actions(z, 3, seed=5)
    freq = torch.bincount(a.long(), minlength=3).double() / len(a)
    p = torch.softmax(torch.tensor([0.0, 1.0, 2.0], dtype=torch.float64), 0)
    assert torch.allclose(freq, p, atol=5e-3)

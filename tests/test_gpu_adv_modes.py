"""GPU parity of the advantage modes (grpo_advantages_ex) and of the RAFT++ loss built on them.

RAFT++ (Sec. 3.2, Table 5): success-filter advantages A_i = 1[r_i > 0], no group normalisation (G = 1), the
per-trajectory normaliser 1/|tau_i|, no dual clip, decoupled importance sampling kept.  DAPO dynamic sampling
(Sec. 3.2): groups whose rewards are all equal are marked and counted.  Integers and the filter are compared
bit-exactly; the loss with the gates of tests/gpu_parity.py.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import (LOGP_ATOL, LOSS_RTOL, check_dlogits, dl_to_f64, kink_rows, oracle_inputs, run_gpu,
                              to_np_logits)

pytestmark = pytest.mark.gpu


def _rewards(n_groups=40, G=8, seed=0):
    rng = np.random.default_rng(seed)
    r = rng.choice([0.0, 1.0, 0.5, -1.0], size=n_groups * G, p=[0.5, 0.3, 0.1, 0.1]).astype(np.float32)
    r[:G] = 1.0
    r[G:2 * G] = 0.0
    r[2 * G:3 * G] = 0.5
    return r


@pytest.mark.parametrize("G", [1, 4, 8])
def test_success_filter_and_mixed_mask(G):
    r = _rewards(G=G, seed=G)
    adv, gm, nm = grpo.grpo_advantages_ex(torch.from_numpy(r).cuda(), G, mode=grpo.GRPO_ADV_SUCCESS_FILTER)
    torch.cuda.synchronize()
    assert (adv.cpu().numpy() == oracle.advantages(r, G, mode=oracle.ADV_SUCCESS_FILTER)).all()
    mixed, n = oracle.mixed_groups(r, G)
    assert (gm.cpu().numpy() == mixed).all() and nm.item() == n


def test_group_norm_mode_matches_plain_entry_and_oracle():
    r = _rewards()
    rt = torch.from_numpy(r).cuda()
    adv, gm, nm = grpo.grpo_advantages_ex(rt, 8, mode=grpo.GRPO_ADV_GROUP_NORM)
    plain = grpo.grpo_advantages(rt, 8)
    torch.cuda.synchronize()
    assert torch.equal(adv, plain)
    np.testing.assert_allclose(adv.cpu().numpy(), oracle.advantages(r, 8), rtol=1e-6, atol=1e-7)
    mixed, n = oracle.mixed_groups(r, 8)
    assert (gm.cpu().numpy() == mixed).all() and nm.item() == n
    # unmixed groups get zero advantages: the mask and the advantages agree
    A = adv.cpu().numpy().reshape(-1, 8)
    assert ((np.abs(A).max(axis=1) > 0) == (mixed == 1)).all()


@pytest.mark.parametrize("name", ["tiny", "v32k"])
def test_raft_plus_plus_loss(name):
    b = make_batch(name, "cuda", with_prox=True)
    b = dict(b, cfg=dataclasses.replace(b["cfg"], G=1))
    r = b["structure"].rewards
    adv, _, _ = grpo.grpo_advantages_ex(torch.from_numpy(r).cuda(), 1, mode=grpo.GRPO_ADV_SUCCESS_FILTER,
                                        mixed=False)
    A64 = oracle.advantages(r, 1, mode=oracle.ADV_SUCCESS_FILTER)
    oi = oracle_inputs(b, A64)
    zl = to_np_logits(b["logits"])
    ref = oracle.loss_rows(zl, oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"], 1, V=b["V"],
                           norm=oracle.NORM_TRAJ_STEPS, dual_clip_c=0.0)
    loss, dl, aux = run_gpu(b, adv, norm=grpo.GRPO_NORM_TRAJ_STEPS, k=10.0, c=0.0)
    assert abs(loss - ref.loss) <= LOSS_RTOL * abs(ref.loss), (loss, ref.loss)
    assert np.abs(aux.token_logp.cpu().numpy() - ref.token_logp).max() <= LOGP_ATOL
    # failed trajectories carry no gradient: their dlogits rows are exactly zero
    tt = oi["seg"].tok_traj
    dlg = dl_to_f64(dl)
    failed = A64[tt] == 0
    assert (dlg[failed] == 0).all()
    kinks = kink_rows(ref, oi["behave"], oi["prox"], A64[tt], 0.2, 0.2, 0.0)
    is_bf16 = b["logits"].dtype == torch.bfloat16
    check_dlogits(dlg, ref.dlogits, is_bf16, exempt=kinks, what=f"RAFT++ {name}")
    # rerun at grad_scale = 1/max|g_t|: every row under the scaled gate
    gs = float(np.float32(1.0 / np.abs(ref.token_g).max()))
    loss2, dl2, _ = run_gpu(b, adv, norm=grpo.GRPO_NORM_TRAJ_STEPS, k=10.0, c=0.0, grad_scale=gs, aux=False)
    assert loss2 == loss
    check_dlogits(dl_to_f64(dl2), ref.dlogits * gs, is_bf16, exempt=kinks, scaled=True, what=f"RAFT++ {name} scaled")

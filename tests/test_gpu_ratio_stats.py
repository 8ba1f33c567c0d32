"""GPU parity of the importance-ratio statistics (grpo_aux.ratio_stats) of both loss entry points.

Over the tokens that enter the loss: sum / min / max of r = pi/pi_prox and of rho = pi/pi_behave (Sec. 3.2),
the number of tokens whose r lies outside the clip range, and the number of tokens.  The reference is the oracle's
oracle.ratio_stats (pinned in tests/test_oracle_ratio_stats_pins.py) over the oracle's log-probs.  Gates: sums, minima and maxima relative 1e-5 (the
log-probs agree to 2e-5 absolute, so each ratio to about that relative error; 1e-4 on the fused path, whose
log-probs agree to 5e-5); counts exact except for tokens
within 1e-6 of a clip boundary, which may fall either way.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import oracle_inputs, run_gpu, to_np_logits

pytestmark = pytest.mark.gpu

RTOL = 1e-5


def expected(l, behave, prox, valid, eps_lo=0.2, eps_hi=0.2):
    """The oracle's statistics, and how many counted tokens sit within 1e-6 of a clip boundary (either side is
    correct for those)."""
    want = oracle.ratio_stats(l, behave, prox, valid.astype(np.int32), eps_lo, eps_hi)
    p = (behave if prox is None else prox).astype(np.float64)
    r = np.exp(l - p)[valid]
    near = (np.abs(r - (1.0 - eps_lo)) < 1e-6) | (np.abs(r - (1.0 + eps_hi)) < 1e-6)
    return want, near.sum()


def check(got, want, n_near, what, rtol=RTOL):
    np.testing.assert_allclose(got[:6], want[:6], rtol=rtol, err_msg=what)
    assert abs(got[6] - want[6]) <= n_near, (what, got[6], want[6])
    assert got[7] == want[7], (what, got[7], want[7])


@pytest.mark.parametrize("name,decoupled", [("tiny", True), ("v32k", True), ("v32k", False)])
def test_logits_path_ratio_stats(name, decoupled):
    b = make_batch(name, "cuda", with_prox=decoupled)
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    oi = oracle_inputs(b, A.astype(np.float32).astype(np.float64))
    ref = oracle.loss_rows(to_np_logits(b["logits"]), oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"],
                           b["cfg"].G, V=b["V"], k=b["cfg"].k, dual_clip_c=3.0, want_dlogits=False)
    _, _, aux = run_gpu(b, torch.from_numpy(A.astype(np.float32)).cuda(), norm=grpo.GRPO_NORM_CONST_K,
                        k=b["cfg"].k, c=3.0, dlogits=False)
    want, near = expected(ref.token_logp, oi["behave"], oi["prox"], np.ones(len(ref.token_logp), bool))
    check(aux.ratio_stats.cpu().numpy(), want, near, name)
    if not decoupled:  # coupled ratio: r and rho are the same number
        got = aux.ratio_stats.cpu().numpy()
        assert got[0] == got[3] and got[1] == got[4] and got[2] == got[5]


def test_invalid_action_excluded():
    b = make_batch("tiny", "cuda", with_prox=True)
    b["actions"][5] = b["V"]  # out of range: the token leaves the loss
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    oi = oracle_inputs(b, A)
    ref = oracle.loss_rows(to_np_logits(b["logits"]), oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"],
                           b["cfg"].G, V=b["V"], k=b["cfg"].k, want_dlogits=False)
    _, _, aux = run_gpu(b, torch.from_numpy(A.astype(np.float32)).cuda(), norm=grpo.GRPO_NORM_CONST_K,
                        k=b["cfg"].k, dlogits=False)
    valid = np.ones(len(ref.token_logp), bool)
    valid[5] = False
    want, near = expected(ref.token_logp, oi["behave"], oi["prox"], valid)
    check(aux.ratio_stats.cpu().numpy(), want, near, "invalid action")
    assert aux.error_flags.item() == grpo.GRPO_FLAG_ACTION


def test_fused_path_ratio_stats():
    from oracle import fused
    from synth import make_fused_batch
    from tests.test_gpu_fused import bits, small_cfg
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=21), "cuda")
    st = b["structure"]
    A = oracle.advantages(st.rewards, b["cfg"].G)
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    aux = grpo.LossAux.alloc(st.T, len(st.rewards), "cuda")
    grpo.fused_lmhead_grpo(b["hidden"], b["W"], b["actions"], b["behave"], torch.from_numpy(A.astype(np.float32)).cuda(),
                           torch.from_numpy(st.step_tok_off).cuda(), torch.from_numpy(st.traj_step_off).cuda(),
                           b["cfg"].G, vocab_chunk=256, norm=grpo.GRPO_NORM_CONST_K, k=b["cfg"].k, aux=aux)
    torch.cuda.synchronize()
    ref = fused.fused_loss(bits(b["hidden"]), bits(b["W"]), b["actions"].cpu().numpy(), b["behave"].cpu().numpy(),
                           None, A.astype(np.float32).astype(np.float64), seg, b["cfg"].G, norm=oracle.NORM_CONST_K,
                           k=b["cfg"].k)
    want, near = expected(ref.rows.token_logp, b["behave"].cpu().numpy(), None, np.ones(st.T, bool))
    # the fused log-probs come from fp32 MFMA logits and agree to 5e-5 (tests/test_gpu_fused.py)
    check(aux.ratio_stats.cpu().numpy(), want, near, "fused", rtol=1e-4)

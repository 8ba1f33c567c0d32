"""GPU parity of the forward-only fused call (fused_lmhead_token_logp: the action's log-prob and the policy
entropy from hidden states and the LM-head weight) against the oracle on z = h W in fp64.

Gates: log-prob absolute 5e-5, as for the fused loss path (the matrix-core logits are fp32 sums of H products);
entropy |gpu - ref| <= 1e-4 + 2e-5 |ref|: the entropy moves by at most max|dz| (H_t + log V) under a logit error
dz, and the fp32 tile moments add a relative 1e-6.  The log-prob agrees with the fused loss path's to 1e-6: the
same tile partials and action logit, with log S taken in fp64 here and through an exact exponent split and an
fp32 log2 in the loss path's token epilogue.  Sizes: small H and V, the real H and V with a few hundred tokens,
and the full fused workload on sampled rows; edge cases: invalid actions, the empty batch, no entropy.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from oracle import fused
from synth import make_fused_batch
from synth.rollouts import Config
from tests.test_gpu_fused import bits, setup, small_cfg

pytestmark = pytest.mark.gpu

LOGP_ATOL, ENT_ATOL, ENT_RTOL = 5e-5, 1e-4, 2e-5


def ref_rows(b, rows=None):
    hb, Wb = bits(b["hidden"]), bits(b["W"])
    if rows is not None:
        hb = hb[rows]
    z = fused.as_f64(hb) @ fused.as_f64(Wb)
    actions = b["actions"].cpu().numpy()
    if rows is not None:
        actions = actions[rows]
    return oracle.logp_entropy(z, actions)


def check(logp, ent, ref, what=""):
    dl = np.abs(logp - ref.token_logp)
    assert dl.max(initial=0) <= LOGP_ATOL, f"{what}: logp error {dl.max()}"
    de = np.abs(ent - ref.token_entropy)
    bound = ENT_ATOL + ENT_RTOL * np.abs(ref.token_entropy)
    assert (de <= bound).all(), f"{what}: entropy error {(de / bound).max()} x the gate"
    return dl.max(initial=0), de.max(initial=0)


def run(b, entropy=True):
    flags = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    logp, ent = grpo.fused_lmhead_token_logp(b["hidden"], b["W"], b["actions"], entropy=entropy, error_flags=flags)
    torch.cuda.synchronize()
    return logp, ent, flags.item()


@pytest.mark.parametrize("H,V,seed", [(64, 1000, 51), (128, 2048, 52), (256, 5000, 53)])
def test_fused_logp_small(H, V, seed):
    b = make_fused_batch(small_cfg(4, 8, H, V, seed=seed, tok_mean=6.0, steps=(2, 6)), "cuda")
    logp, ent, flags = run(b)
    assert flags == 0
    check(logp.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64), ref_rows(b), f"H{H} V{V}")
    # without the entropy the log-probs are the same bits (the same (max, sum exp) partials)
    logp2, ent2, _ = run(b, entropy=False)
    assert ent2 is None and torch.equal(logp, logp2)


def test_fused_logp_matches_the_loss_path():
    b = make_fused_batch(small_cfg(4, 8, 256, 5000, seed=54, tok_mean=6.0, steps=(2, 9)), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    aux = grpo.LossAux.alloc(b["structure"].T, len(b["structure"].rewards), "cuda")
    grpo.fused_lmhead_grpo_blocked(b["hidden"], b["W"], b["actions"], b["behave"], A32, sto, tso, b["cfg"].G,
                                   token_block=256, aux=aux)
    logp, _, _ = run(b)
    assert (logp.double() - aux.token_logp.double()).abs().max().item() <= 1e-6


def test_fused_logp_full_hv_reduced_t():
    cfg = Config("fused-hv", 1, 8, 151936, "bf16", 0.0, 0.35, (8, 30), (3, 12), 96.0, (1, 4096), 0.05, 10.0,
                 T_target=320, H=3584, seed=55)
    b = make_fused_batch(cfg, "cuda")
    logp, ent, flags = run(b)
    assert flags == 0
    check(logp.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64), ref_rows(b), "full H, V")


def test_fused_logp_full_size_sampled():
    b = make_fused_batch("fused", "cuda")
    T = b["structure"].T
    logp, ent, flags = run(b)
    assert flags == 0
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, T - 1], rng.integers(0, T, 24)]))
    check(logp.cpu().numpy()[rows].astype(np.float64), ent.cpu().numpy()[rows].astype(np.float64),
          ref_rows(b, rows), "sampled rows")


def test_fused_logp_invalid_action_and_empty():
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=56), "cuda")
    b["actions"][3] = 1000
    b["actions"][5] = -2
    logp, ent, flags = run(b)
    assert flags == grpo.GRPO_FLAG_ACTION
    lp = logp.cpu().numpy()
    assert lp[3] == 0.0 and lp[5] == 0.0
    ref = ref_rows(b)
    ok = np.ones(len(lp), bool)
    ok[[3, 5]] = False
    assert np.abs(lp[ok] - ref.token_logp[ok]).max() <= LOGP_ATOL
    assert np.abs(ent.cpu().numpy() - ref.token_entropy).max() <= ENT_ATOL + ENT_RTOL * np.abs(ref.token_entropy).max()
    # the empty batch: flags cleared, nothing else
    e = {"hidden": b["hidden"][:0], "W": b["W"], "actions": b["actions"][:0]}
    logp, ent, flags = run(e)
    assert logp.numel() == 0 and ent.numel() == 0 and flags == 0

"""GPU parity of the forward-only path (grpo_token_logp: action log-prob and policy entropy) against the oracle.

Gates (fp32 arithmetic over V terms, sums in fp32 per thread and fp64 across the row):
  * log-prob: absolute 2e-5, as on the loss path;
  * entropy:  |gpu - ref| <= 2e-5 + 2e-5 |ref|.  The entropy is log S - T/S with S = sum e^(z - m) and
    T = sum e^(z - m)(z - m), each accumulated in fp32 over about V/256 terms per thread, so each carries a
    relative error of order 1e-6; both terms are non-negative and at most log V + |H| in size.
Sizes: the tiny and 32k workloads in full, the 151,936-vocabulary workloads at full size in the benchmark's
launch configuration on sampled rows, and the edge cases (generic kernel, padded stride, invalid actions,
constant and peaked rows, the empty batch).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import LOGP_ATOL, to_np_logits

pytestmark = pytest.mark.gpu

ENT_ATOL, ENT_RTOL = 2e-5, 2e-5


def check(logp, ent, ref, what=""):
    dl = np.abs(logp - ref.token_logp)
    assert dl.max() <= LOGP_ATOL, f"{what}: logp error {dl.max()}"
    de = np.abs(ent - ref.token_entropy)
    bound = ENT_ATOL + ENT_RTOL * np.abs(ref.token_entropy)
    assert (de <= bound).all(), f"{what}: entropy error {(de / bound).max()} x the gate"


def run(logits, actions, V=None):
    flags = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    logp, ent = grpo.grpo_token_logp(logits, actions, V=V, error_flags=flags)
    torch.cuda.synchronize()
    return logp.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64), flags.item()


@pytest.mark.parametrize("name", ["tiny", "v32k"])
def test_full_parity(name):
    b = make_batch(name, "cuda")
    logp, ent, flags = run(b["logits"], b["actions"])
    ref = oracle.logp_entropy(to_np_logits(b["logits"]), b["actions"].cpu().numpy(), V=b["V"])
    check(logp, ent, ref, name)
    assert flags == 0 == ref.flags


@pytest.mark.parametrize("name", ["v152k", "long"])
def test_full_size_sampled(name):
    b = make_batch(name, "cuda")
    T = b["logits"].shape[0]
    logp, ent, flags = run(b["logits"], b["actions"])
    assert flags == 0
    rows = np.unique(np.concatenate([[0, T - 1], np.random.default_rng(1).integers(0, T, 64)]))
    zs = to_np_logits(b["logits"].index_select(0, torch.from_numpy(rows).cuda()))
    a = b["actions"].cpu().numpy()
    for q, t in enumerate(rows):
        ref = oracle.logp_entropy(zs[q:q + 1], a, row_begin=int(t), row_end=int(t) + 1, row_offset=int(t))
        check(logp[t:t + 1], ent[t:t + 1], ref, f"{name} row {t}")


def test_matches_loss_path_logp():
    # the forward-only log-prob and the loss path's aux.token_logp come from the same definition
    from tests.gpu_parity import run_gpu
    b = make_batch("v32k", "cuda")
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    _, _, aux = run_gpu(b, torch.from_numpy(A.astype(np.float32)).cuda(), norm=grpo.GRPO_NORM_CONST_K,
                        k=b["cfg"].k, c=3.0)
    logp, _, _ = run(b["logits"], b["actions"])
    assert np.abs(logp - aux.token_logp.cpu().numpy()).max() <= 2e-6


@pytest.mark.parametrize("V,dtype,ld", [(7, torch.bfloat16, None), (7, torch.float32, None),
                                        (1000, torch.bfloat16, 1024), (1000, torch.float32, 1003),
                                        (4093, torch.float32, None), (151936, torch.bfloat16, None),
                                        (200000, torch.bfloat16, None), (64, torch.float32, None)])
def test_vocab_sizes_strides_and_kernels(V, dtype, ld):
    # V = 7, 4093 or an odd stride take the element-wise kernel; the rest the vector kernel
    g = torch.Generator("cuda").manual_seed(V)
    T = 37
    full = torch.randn((T, ld or V), generator=g, device="cuda") * 2.0
    logits = full.to(dtype)
    actions = torch.randint(0, V, (T,), generator=g, device="cuda", dtype=torch.int32)
    logp, ent, flags = run(logits, actions, V=V)
    ref = oracle.logp_entropy(to_np_logits(logits), actions.cpu().numpy(), V=V)
    check(logp, ent, ref, f"V={V}")
    assert flags == 0


@pytest.mark.parametrize("V,dtype,ld", [(7, torch.float32, None), (4096, torch.bfloat16, None),
                                        (151936, torch.bfloat16, None), (1000, torch.float32, 1003)])
def test_masked_logits(V, dtype, ld):
    # -inf logits (a masked vocabulary): zero probability, no term in the entropy (0 log 0 = 0), nothing flagged;
    # about a third of the columns, never the action's, on the element-wise and the vector kernels
    g = torch.Generator("cuda").manual_seed(V + 1)
    T = 37
    full = torch.randn((T, ld or V), generator=g, device="cuda") * 2.0
    actions = torch.randint(0, V, (T,), generator=g, device="cuda", dtype=torch.int32)
    mask = torch.rand((T, V), generator=g, device="cuda") < 0.3
    mask[torch.arange(T, device="cuda"), actions.long()] = False
    full[:, :V].masked_fill_(mask, float("-inf"))
    logits = full.to(dtype)
    logp, ent, flags = run(logits, actions, V=V)
    ref = oracle.logp_entropy(to_np_logits(logits), actions.cpu().numpy(), V=V)
    assert np.isfinite(ref.token_entropy).all() and ref.flags == 0
    check(logp, ent, ref, f"masked V={V}")
    assert flags == 0


@pytest.mark.parametrize("V,dtype,ld", [(151936, torch.bfloat16, None), (1000, torch.float32, 1003)])
def test_masked_uniform_rows_closed_form(V, dtype, ld):
    # k equal finite logits among V - k masked (-inf) ones: log-prob -log k and entropy log k, the uniform row of
    # width k (the oracle's pin); k from 1 to V over the rows, the finite columns scattered, the action among them
    g = torch.Generator("cuda").manual_seed(V)
    T = 24
    ks = [1, 2, 3, 7, 64, 1000, V - 1, V]
    ks += [int(x) for x in torch.randint(1, V + 1, (T - 8,), generator=g, device="cuda")]
    full = torch.full((T, ld or V), float("-inf"), device="cuda")
    actions = torch.empty(T, dtype=torch.int32, device="cuda")
    for t, k in enumerate(ks):
        cols = torch.randperm(V, generator=g, device="cuda")[:k]
        full[t, cols] = float(t % 5) - 2.0
        actions[t] = cols[0]
    logp, ent, flags = run(full.to(dtype), actions, V=V)
    logk = np.log(np.array(ks, np.float64))
    assert flags == 0
    assert np.abs(logp + logk).max() <= LOGP_ATOL
    assert (np.abs(ent - logk) <= ENT_ATOL + ENT_RTOL * logk).all()


def test_constant_and_peaked_rows():
    V = 4096
    logits = torch.zeros((3, V), dtype=torch.bfloat16, device="cuda")
    logits[1] = 7.0
    logits[2, 100] = 120.0  # every other p underflows: entropy 0, log-prob of token 100 is 0
    actions = torch.tensor([5, 4095, 100], dtype=torch.int32, device="cuda")
    logp, ent, flags = run(logits, actions)
    assert flags == 0
    np.testing.assert_allclose(ent[:2], math.log(V), rtol=2e-6)
    np.testing.assert_allclose(logp[:2], -math.log(V), rtol=2e-6)
    assert abs(ent[2]) <= ENT_ATOL and abs(logp[2]) <= LOGP_ATOL


def test_invalid_actions_flagged():
    g = torch.Generator("cuda").manual_seed(3)
    logits = torch.randn((6, 512), generator=g, device="cuda").to(torch.bfloat16)
    actions = torch.tensor([0, 512, 3, -1, 511, 9], dtype=torch.int32, device="cuda")
    logp, ent, flags = run(logits, actions)
    assert flags == grpo.GRPO_FLAG_ACTION
    ref = oracle.logp_entropy(to_np_logits(logits), actions.cpu().numpy())
    assert ref.flags == oracle.ERR_ACTION
    check(logp, ent, ref, "invalid actions")
    assert logp[1] == 0.0 and logp[3] == 0.0


def test_empty_batch_and_entropy_off():
    logits = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    logp, ent, flags = run(logits, torch.empty(0, dtype=torch.int32, device="cuda"))
    assert logp.shape == (0,) and ent.shape == (0,) and flags == 0
    logits = torch.randn((4, 64), device="cuda")
    lp, e = grpo.grpo_token_logp(logits, torch.zeros(4, dtype=torch.int32, device="cuda"), entropy=False)
    torch.cuda.synchronize()
    assert e is None
    ref = oracle.logp_entropy(logits.cpu().numpy(), np.zeros(4, np.int32))
    assert np.abs(lp.cpu().numpy() - ref.token_logp).max() <= LOGP_ATOL


def test_bitwise_deterministic():
    b = make_batch("v32k", "cuda")
    r1 = grpo.grpo_token_logp(b["logits"], b["actions"])
    r2 = grpo.grpo_token_logp(b["logits"], b["actions"])
    torch.cuda.synchronize()
    assert torch.equal(r1[0], r2[0]) and torch.equal(r1[1], r2[1])

"""GPU parity of the vocabulary-sharded fused LM head (fused_lmhead_vocab_shard_stats, fused_lmhead_grpo_vocab_shard)
against the fp64 oracle, with the shard's logits formed again in the backward call or kept from the statistics
call (logits_out / logits_in).

One GPU plays every shard: W's columns are split into ranges, each range's records are computed into one
[n_shards, T] record tensor (what gathering them across devices gives), and each range's backward call writes its
dW columns and its fp32 partial dhidden.  The partials are summed (what the reduce-scatter across devices gives)
and the dW columns concatenated; then the gates of tests/test_gpu_fused.py apply against the oracle's whole-row
results: the loss within 1e-5 of sum_t |w s_t| (the loss's own size when its terms do not cancel; the batch of
the multi-chunk case has a loss of 2% of that sum, and the matrix cores' fp32 logits, shared with the
single-device path, leave 1.7e-5 of the loss there), token log-probs absolute 5e-5, dhidden and dW elementwise
within the bf16 rounding of D (no final bf16 rounding here: the partials are fp32).  Where the single-device
fused path runs on the same batch, the two losses agree to 1e-6 of that sum.  The records against the oracle's per-shard
statistics of z = h W in fp64: the maximum absolute 5e-5 (matrix-core logits are fp32 sums of H products), the
action logit (an fp64 dot of the same bf16 inputs) absolute 1e-9, the sum relative 1e-4.  Every shard must produce the same
loss bits.  Sizes: small H and V with even, uneven and multi-chunk splits; the full H = 3,584 and V = 151,936 in
8 shards of 18,992 with a few hundred tokens.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from oracle import fused
from synth import make_fused_batch
from synth.rollouts import Config
from tests.gpu_parity import check_fused_loss, gpu_norm
from tests.test_gpu_fused import bits, check_dw, setup, small_cfg

pytestmark = pytest.mark.gpu


def run_shards(b, A32, sto, tso, bounds, chunk, norm, c, gs=1.0, dw_init=None, accumulate=False, ngt=0.0,
               keep=False):
    """Every shard's two calls on one GPU: (losses, summed dhidden partials fp64, concatenated dW fp64, aux of shard
    0, records).  keep: each shard's statistics call keeps its logits and its backward call uses them."""
    T = b["structure"].T
    N = len(b["structure"].rewards)
    H, V = b["H"], b["V"]
    shards = [b["W"][:, b0:b1].contiguous() for b0, b1 in zip(bounds[:-1], bounds[1:])]
    stats = torch.empty((len(shards), T, grpo.VOCAB_STATS_BYTES), dtype=torch.uint8, device="cuda")
    kept = [grpo.vocab_shard_logits_buffer(T, w.shape[1], "cuda") if keep else None for w in shards]
    for g, (b0, w) in enumerate(zip(bounds[:-1], shards)):
        grpo.fused_lmhead_vocab_shard_stats(b["hidden"], w, b["actions"], b0, stats=stats[g], logits_out=kept[g])
    losses, dh_sum, dws, aux0 = [], np.zeros((T, H)), [], None
    for g, (b0, w) in enumerate(zip(bounds[:-1], shards)):
        aux = grpo.LossAux.alloc(T, N, "cuda")
        dw = None if dw_init is None else dw_init[:, b0:bounds[g + 1]].contiguous()
        loss, dhp, dws_g = grpo.fused_lmhead_grpo_vocab_shard(
            b["hidden"], w, stats, b0, V, b["actions"], b["behave"], A32, sto, tso, b["cfg"].G, vocab_chunk=chunk,
            prox_logp=b["prox"], norm=gpu_norm(norm), k=b["cfg"].k, dual_clip_c=c, grad_scale=gs,
            n_groups_total=ngt, dw_shard=dw, accumulate_dw=accumulate, aux=aux, logits_in=kept[g])
        torch.cuda.synchronize()
        losses.append(loss.item())
        dh_sum += dhp.cpu().numpy().astype(np.float64)
        dws.append(dws_g.cpu().numpy().astype(np.float64))
        aux0 = aux0 or aux
    return losses, dh_sum, np.concatenate(dws, axis=1), aux0, stats


def check_records(stats, hb, Wb, actions, bounds):
    z = fused.as_f64(hb) @ fused.as_f64(Wb)
    m, za, s = (x.cpu().numpy().astype(np.float64) for x in grpo.vocab_stats_fields(stats))
    for g, (b0, b1) in enumerate(zip(bounds[:-1], bounds[1:])):
        ref = oracle.vocab_shard_stats(z[:, b0:b1], actions, b0)
        assert np.abs(m[g] - ref.m).max() <= 5e-5
        own = np.isfinite(ref.za)
        assert (np.isfinite(za[g]) == own).all()
        assert np.abs(za[g][own] - ref.za[own]).max(initial=0) <= 1e-9
        np.testing.assert_allclose(s[g], ref.s, rtol=1e-4)


def check_dh_f32(dh, ref_dh, D, W64, what=""):
    # the partials are fp32 sums of products of the bf16-rounded D: 2^-7 |D||W|^T bounds the D rounding
    bound = 2.0 ** -7 * (np.abs(D) @ np.abs(W64).T) + 1e-6 * np.abs(ref_dh).max()
    err = np.abs(dh - ref_dh)
    assert (err <= bound).all(), f"{what}: dhidden bound exceeded by {(err / bound).max()}"
    assert np.linalg.norm(err) / np.linalg.norm(ref_dh) <= 5e-3


def shard_compare(b, bounds, chunk, norm, c, gs=1.0, accumulate=False, ngt=0.0, keep=False):
    A64, A32, seg, sto, tso = setup(b)
    H, V = b["H"], b["V"]
    dw0 = None
    if accumulate:
        dw0 = torch.randn((H, V), device="cuda", generator=torch.Generator("cuda").manual_seed(9)) * 1e-3
    losses, dh, dW, aux, stats = run_shards(b, A32, sto, tso, bounds, chunk, norm, c, gs, dw0, accumulate, ngt, keep)
    assert len(set(losses)) == 1, losses
    hb, Wb = bits(b["hidden"]), bits(b["W"])
    actions = b["actions"].cpu().numpy()
    check_records(stats, hb, Wb, actions, bounds)
    prox = None if b["prox"] is None else b["prox"].cpu().numpy()
    ref = fused.fused_loss(hb, Wb, actions, b["behave"].cpu().numpy(), prox, A64, seg, b["cfg"].G, norm=norm,
                           k=b["cfg"].k, dual_clip_c=c, grad_scale=gs, n_groups_total=ngt)
    size = np.abs(ref.rows.token_contrib).sum()
    check_fused_loss(losses[0], ref.rows.token_contrib, "sharded loss", report=True)
    assert np.abs(aux.token_logp.cpu().numpy() - ref.rows.token_logp).max() <= 5e-5
    assert aux.error_flags.item() == 0
    D = ref.rows.dlogits
    check_dh_f32(dh, ref.dhidden, D, fused.as_f64(Wb), "summed dhidden partials")
    if accumulate:
        dW -= dw0.cpu().numpy().astype(np.float64)
    check_dw(dW, ref.dW, fused.as_f64(hb), D, "concatenated dW")
    # the single-device fused path on the same batch: the same fp32 logits, so the same loss to rounding
    loss1, _, _ = grpo.fused_lmhead_grpo(b["hidden"], b["W"], b["actions"], b["behave"], A32, sto, tso, b["cfg"].G,
                                         vocab_chunk=chunk, prox_logp=b["prox"], norm=gpu_norm(norm), k=b["cfg"].k,
                                         dual_clip_c=c, grad_scale=gs, n_groups_total=ngt)
    torch.cuda.synchronize()
    assert abs(losses[0] - loss1.item()) <= 1e-6 * size, (losses[0], loss1.item())
    return losses[0], dh, dW


KEEP = [False, True]


@pytest.mark.parametrize("bounds", [[0, 1000], [0, 504, 1000], [0, 8, 264, 1000]])
@pytest.mark.parametrize("c", [0.0, 3.0])
@pytest.mark.parametrize("keep", KEEP)
def test_fused_shard_small(bounds, c, keep):
    # H = 64, V = 1000 split at multiples of 8; chunks of 256 so the wider shards take several chunks (in pairs);
    # keep: the statistics call's logits are kept and the shard is one chunk
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=21), "cuda")
    shard_compare(b, bounds, 256, oracle.NORM_CONST_K, c, keep=keep)


@pytest.mark.parametrize("keep", KEEP)
def test_fused_shard_multichunk_accumulate(keep):
    b = make_fused_batch(small_cfg(4, 8, 256, 5000, seed=22, tok_mean=6.0, steps=(2, 9)), "cuda")
    shard_compare(b, [0, 1600, 3200, 5000], 512, oracle.NORM_TRAJ_STEPS, 3.0, gs=0.5, accumulate=True, keep=keep)


def test_fused_shard_kept_logits_same_loss_bits():
    # kept or formed again, the shard's logits are the same matrix-core sums in the same order: the records, loss
    # and per-token outputs are bit-identical; dhidden and dW differ only in how their fp32 sums are chunked
    b = make_fused_batch(small_cfg(4, 8, 256, 5000, seed=27, tok_mean=6.0, steps=(2, 9)), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    r0 = run_shards(b, A32, sto, tso, [0, 1600, 3200, 5000], 512, oracle.NORM_CONST_K, 3.0)
    r1 = run_shards(b, A32, sto, tso, [0, 1600, 3200, 5000], 512, oracle.NORM_CONST_K, 3.0, keep=True)
    assert r0[0] == r1[0]
    assert torch.equal(r0[4], r1[4])
    for f in ("token_logp", "traj_loss", "clip_counts", "error_flags"):
        assert torch.equal(getattr(r0[3], f), getattr(r1[3], f)), f
    assert np.linalg.norm(r0[1] - r1[1]) <= 1e-5 * np.linalg.norm(r0[1])
    assert np.linalg.norm(r0[2] - r1[2]) <= 1e-5 * np.linalg.norm(r0[2])


@pytest.mark.parametrize("keep", KEEP)
def test_fused_shard_decoupled_and_global_groups(keep):
    # a proximal policy distinct from the behaviour one (decoupled ratios), and the normaliser's group count
    # overridden as a data-parallel shard of a 5x larger batch would pass it
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=25), "cuda")
    gen = torch.Generator("cuda").manual_seed(26)
    b["prox"] = b["behave"] + 0.05 * torch.randn(b["behave"].shape, device="cuda", generator=gen)
    shard_compare(b, [0, 504, 1000], 256, oracle.NORM_TRAJ_STEPS, 3.0, ngt=10.0, keep=keep)


def test_fused_shard_agrees_with_single_device():
    b = make_fused_batch(small_cfg(2, 4, 128, 2048, seed=23), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    losses, dh, dW, _, _ = run_shards(b, A32, sto, tso, [0, 768, 2048], 256, oracle.NORM_CONST_K, 3.0)
    loss1, dh1, dW1 = grpo.fused_lmhead_grpo(b["hidden"], b["W"], b["actions"], b["behave"], A32, sto, tso,
                                             b["cfg"].G, vocab_chunk=256, k=b["cfg"].k, dual_clip_c=3.0)
    torch.cuda.synchronize()
    assert abs(losses[0] - loss1.item()) <= 1e-6 * abs(loss1.item())
    # the single-device dhidden is the bf16 rounding of an fp32 sum over the same bf16 D tiles
    dh1 = dh1.float().cpu().numpy().astype(np.float64)
    assert (np.abs(dh - dh1) <= 2.0 ** -8 * np.abs(dh) + 1e-3 * np.abs(dh).max()).all()
    assert np.linalg.norm(dW - dW1.cpu().numpy()) <= 1e-3 * np.linalg.norm(dW)


@pytest.mark.parametrize("keep", KEEP)
def test_fused_shard_full_hv_eight_shards(keep):
    # the real H = 3584 and V = 151,936 split 8 ways (18,992 columns: two full chunks of 8192 and a 2608 tail)
    cfg = Config("fused-hv-shard", 1, 8, 151936, "bf16", 0.0, 0.35, (8, 30), (3, 12), 96.0, (1, 4096), 0.05, 10.0,
                 T_target=256, H=3584, seed=24)
    b = make_fused_batch(cfg, "cuda")
    V = b["V"]
    shard_compare(b, [g * (V // 8) for g in range(9)], 8192, oracle.NORM_CONST_K, 3.0, keep=keep)


@pytest.mark.parametrize("keep", KEEP)
def test_fused_shard_empty_batch(keep):
    N, H, V = 4, 64, 256
    sto = torch.zeros(5, dtype=torch.int32, device="cuda")
    tso = torch.arange(0, 5, dtype=torch.int32, device="cuda")
    hidden = torch.empty((0, H), dtype=torch.bfloat16, device="cuda")
    W = torch.randn((H, V), device="cuda").to(torch.bfloat16)
    act = torch.empty(0, dtype=torch.int32, device="cuda")
    kept = grpo.vocab_shard_logits_buffer(0, V, "cuda") if keep else None
    stats = grpo.fused_lmhead_vocab_shard_stats(hidden, W, act, 0, logits_out=kept)
    dw = torch.full((H, V), 7.0, device="cuda")
    loss, dhp, dW = grpo.fused_lmhead_grpo_vocab_shard(hidden, W, stats[None], 0, V, act,
                                                       torch.empty(0, device="cuda"), torch.zeros(N, device="cuda"),
                                                       sto, tso, 4, vocab_chunk=256, dw_shard=dw, logits_in=kept)
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and dhp.shape == (0, H) and (dW == 0).all()

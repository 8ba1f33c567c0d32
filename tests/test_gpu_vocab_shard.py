"""GPU parity of the vocabulary-sharded loss (grpo_vocab_shard_stats, grpo_loss_fwd_bwd_vocab_shard) against the
oracle.

One GPU plays every shard in turn: the logits of a batch are split into column ranges, each range's records are
computed into one [n_shards, T] record tensor (what gathering them across devices would give), and each range's
loss pass writes its columns of dlogits.  The concatenated dlogits, the loss and the per-token outputs are held
to the gates of tests/gpu_parity.py against the oracle's whole-row results; the records against the oracle's
per-shard statistics (max and action logit exact, the sum relative 5e-6: fp32 partial sums over the shard's
terms, combined in fp64).  Every shard must produce the same loss bits.  Sizes: the tiny workload (fp32) and
the 32k-vocabulary workload (bf16) in full, with even, uneven and misaligned splits (the misaligned ones take the
element kernel); the 151,936-vocabulary workload at full size in 8 shards of 18,992 columns, on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import (LOGP_ATOL, LOSS_RTOL, check_dlogits, device_batch, dl_to_f64, gpu_norm, kink_rows,
                              oracle_inputs, run_gpu, to_np_logits)

pytestmark = pytest.mark.gpu

STATS_S_RTOL = 5e-6


def _adv(b):
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    return A.astype(np.float32).astype(np.float64), torch.from_numpy(A.astype(np.float32)).cuda()


def shard_stats(lg, actions, bounds):
    T = lg.shape[0]
    stats = torch.empty((len(bounds) - 1, T, grpo.VOCAB_STATS_BYTES), dtype=torch.uint8, device="cuda")
    flags = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    for g, (b0, b1) in enumerate(zip(bounds[:-1], bounds[1:])):
        grpo.grpo_vocab_shard_stats(lg[:, b0:b1], actions, b0, stats=stats[g], error_flags=flags)
    torch.cuda.synchronize()
    assert flags.item() == 0
    return stats


def run_sharded(b, A32, bounds, *, norm, k, c=0.0, grad_scale=1.0, dlogits=True, aux=True, actions=None, ngt=0.0):
    """Every shard's two calls on one GPU.  Returns (per-shard losses, dlogits or None, per-shard aux, records)."""
    dev = device_batch(b)
    N = len(b["structure"].rewards)
    lg = b["logits"]
    T = lg.shape[0]
    act = b["actions"] if actions is None else actions
    stats = shard_stats(lg, act, bounds)
    dl = torch.full_like(lg, float("nan")) if dlogits else None  # NaN: every column must be written
    losses, auxes = [], []
    for b0, b1 in zip(bounds[:-1], bounds[1:]):
        a = grpo.LossAux.alloc(T, N, "cuda") if aux else None
        loss, _ = grpo.grpo_loss_fwd_bwd_vocab_shard(
            lg[:, b0:b1], stats, b0, b["V"], act, b["behave"], A32, dev["step_tok_off"], dev["traj_step_off"],
            b["cfg"].G, prox_logp=b["prox"], norm=norm, k=k, dual_clip_c=c, grad_scale=grad_scale,
            n_groups_total=ngt, dlogits=None if dl is None else dl[:, b0:b1], aux=a)
        losses.append(loss.item())
        auxes.append(a)
    torch.cuda.synchronize()
    return losses, dl, auxes, stats


def check_stats(stats, zl, actions, bounds, rows=None):
    """Records against the oracle's per-shard statistics; with ``rows``, stats and zl hold just those rows."""
    m, za, s = (x.cpu().numpy() for x in grpo.vocab_stats_fields(stats))
    for g, (b0, b1) in enumerate(zip(bounds[:-1], bounds[1:])):
        if rows is None:
            ref = oracle.vocab_shard_stats(zl[:, b0:b1], actions, b0)
        else:
            parts = [oracle.vocab_shard_stats(zl[q:q + 1, b0:b1], actions, b0, row_begin=int(t), row_end=int(t) + 1,
                                              row_offset=int(t)) for q, t in enumerate(rows)]
            ref = oracle.ShardStats(*(np.concatenate([getattr(x, f) for x in parts]) for f in ("m", "s", "za")))
        np.testing.assert_array_equal(m[g].astype(np.float64), ref.m)
        np.testing.assert_array_equal(za[g].astype(np.float64), ref.za)
        np.testing.assert_allclose(s[g], ref.s, rtol=STATS_S_RTOL)


def _oracle_blocks(b, zl, oi, norm, k, c, block=2048):
    """The oracle over the batch in row blocks (whole-batch fp64 dlogits can be too large for host memory)."""
    T = len(oi["actions"])
    for r0 in range(0, T, block):
        r1 = min(T, r0 + block)
        yield r0, r1, oracle.loss_rows(zl[r0:r1], oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"],
                                       b["cfg"].G, V=b["V"], norm=norm, k=k, dual_clip_c=c, row_begin=r0, row_end=r1,
                                       row_offset=r0)


def _shard_parity(b, bounds, norm, c, scaled=True):
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    zl = to_np_logits(b["logits"])
    is_bf16 = b["logits"].dtype == torch.bfloat16
    V = b["V"]
    T = len(oi["actions"])
    losses, dl, auxes, stats = run_sharded(b, A32, bounds, norm=gpu_norm(norm), k=cfg.k, c=c)
    check_stats(stats, zl, oi["actions"], bounds)
    assert len(set(losses)) == 1, losses  # the same records in the same order: the same bits on every shard
    loss, aux = losses[0], auxes[0]
    tl = aux.token_logp.cpu().numpy()
    for a in auxes[1:]:
        assert np.array_equal(a.token_logp.cpu().numpy(), tl)
        assert torch.equal(a.clip_counts, aux.clip_counts) and torch.equal(a.traj_loss, aux.traj_loss)
    assert (aux.tok_traj.cpu().numpy() == oi["seg"].tok_traj).all()
    assert aux.error_flags.item() == 0
    contrib, state, gmax, n_kinks, kinks_all = np.empty(T), np.empty(T, np.int32), 0.0, 0, []
    for r0, r1, ref in _oracle_blocks(b, zl, oi, norm, cfg.k, c):
        assert ref.flags == 0
        contrib[r0:r1], state[r0:r1] = ref.token_contrib, ref.token_state
        gmax = max(gmax, np.abs(ref.token_g).max())
        assert np.abs(tl[r0:r1] - ref.token_logp).max() <= LOGP_ATOL
        prox = None if oi["prox"] is None else oi["prox"][r0:r1]
        kinks = kink_rows(ref, oi["behave"][r0:r1], prox, A64[oi["seg"].tok_traj[r0:r1]], 0.2, 0.2, c)
        n_kinks += len(kinks)
        kinks_all.extend(r0 + kinks)
        check_dlogits(dl_to_f64(dl[r0:r1, :V]), ref.dlogits, is_bf16, exempt=kinks, what=f"sharded dlogits rows {r0}")
    total = float(np.sum(contrib))
    assert abs(loss - total) <= LOSS_RTOL * abs(total), (loss, total)
    assert n_kinks <= max(2, T // 1000)
    clip = aux.clip_counts.cpu().numpy()
    assert abs(clip[0] - (state & 1).sum()) <= n_kinks and abs(clip[1] - ((state >> 1) & 1).sum()) <= n_kinks
    if scaled:
        gs = float(np.float32(1.0 / gmax))
        losses2, dl2, _, _ = run_sharded(b, A32, bounds, norm=gpu_norm(norm), k=cfg.k, c=c, grad_scale=gs, aux=False)
        assert losses2[0] == loss
        for r0, r1, ref in _oracle_blocks(b, zl, oi, norm, cfg.k, c):
            ex = [t - r0 for t in kinks_all if r0 <= t < r1]
            check_dlogits(dl_to_f64(dl2[r0:r1, :V]), ref.dlogits * gs, is_bf16, exempt=ex, scaled=True,
                          what=f"scaled sharded dlogits rows {r0}")
    return loss, dl, aux


@pytest.mark.parametrize("bounds", [[0, 1024], [0, 512, 1024], [0, 100, 612, 1024], [0, 3, 517, 1021, 1024]])
@pytest.mark.parametrize("norm", [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K])
@pytest.mark.parametrize("c", [0.0, 3.0])
def test_tiny_sharded_parity(bounds, norm, c):
    # [0, 3, 517, 1021, 1024]: shards of 3 columns and misaligned starts take the element kernels
    _shard_parity(make_batch("tiny", "cuda", with_prox=(c > 0)), bounds, norm, c)


@pytest.mark.parametrize("bounds", [[0, 8000, 16000, 24000, 32000], [0, 10000, 10008, 31992, 32000],
                                    [0, 12345, 32000]])
def test_v32k_sharded_parity(bounds):
    _shard_parity(make_batch("v32k", "cuda"), bounds, oracle.NORM_CONST_K, 3.0, scaled=True)


def test_v152k_eight_shards_full_size():
    # the shape one device holds with the 151,936-column vocabulary split 8 ways: 18,992 columns.  Every row's
    # log-prob and the whole loss against the oracle over all rows; records and dlogits of sampled rows (grad_scale
    # 1, then rerun at grad_scale = 1/max|g_t| under the scaled bf16 gate)
    from tests.test_gpu_loss import _oracle_all_rows, _pipeline_rows, _sampled_dlogits, _whole_batch_checks
    b = make_batch("v152k", "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    T, V = b["logits"].shape
    bounds = [g * (V // 8) for g in range(9)]
    ref = _oracle_all_rows(b, oi, [oracle.NORM_CONST_K])[oracle.NORM_CONST_K]
    losses, dl, auxes, stats = run_sharded(b, A32, bounds, norm=gpu_norm(oracle.NORM_CONST_K), k=cfg.k, c=3.0)
    assert len(set(losses)) == 1
    _whole_batch_checks(ref, losses[0], auxes[0], oi, A64, V, V, "v152k, 8 shards")
    rows = _pipeline_rows(T, 256, np.random.default_rng(7), 40)
    rows_t = torch.from_numpy(rows).cuda()
    check_stats(stats.index_select(1, rows_t), to_np_logits(b["logits"].index_select(0, rows_t)), oi["actions"],
                bounds, rows=rows)
    _sampled_dlogits(b, dl, rows, oi, A64, oracle.NORM_CONST_K, 1.0, False, "8 shards")
    del dl
    torch.cuda.empty_cache()
    gs = float(np.float32(1.0 / np.abs(ref.token_g).max()))
    losses2, dl2, _, _ = run_sharded(b, A32, bounds, norm=gpu_norm(oracle.NORM_CONST_K), k=cfg.k, c=3.0,
                                     grad_scale=gs, aux=False)
    assert losses2[0] == losses[0]
    _sampled_dlogits(b, dl2, rows, oi, A64, oracle.NORM_CONST_K, gs, True, "8 shards scaled")
    del dl2
    torch.cuda.empty_cache()
    # and the single-device path on the same batch: the same loss to rounding
    loss1, _, aux1 = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=cfg.k, c=3.0, dlogits=False)
    assert abs(losses[0] - loss1) <= LOSS_RTOL * abs(loss1)
    assert np.abs(auxes[0].token_logp.cpu().numpy() - aux1.token_logp.cpu().numpy()).max() <= LOGP_ATOL
    assert auxes[0].error_flags.item() == 0


@pytest.mark.parametrize("bounds", [[0, 512, 1024], [0, 100, 612, 1024]])
def test_masked_logits_whole_shard(bounds):
    # -inf logits (a masked vocabulary), about a tenth of the columns, and in every other row the whole of the
    # middle shard unless the action falls there: that shard's record is then (max -inf, sum 0), which the merge
    # must skip.  Never the action's column.
    from synth.rollouts import add_noise, engine_logp
    b = make_batch("tiny", "cuda")
    T, V = b["logits"].shape
    g = torch.Generator("cuda").manual_seed(len(bounds))
    mask = torch.rand((T, V), generator=g, device="cuda") < 0.1
    act = b["actions"].long()
    lo, hi = bounds[1], bounds[2]
    whole = (torch.arange(T, device="cuda") % 2 == 0) & ((act < lo) | (act >= hi))
    mask[whole, lo:hi] = True
    mask[torch.arange(T, device="cuda"), act] = False
    b["logits"].masked_fill_(mask, float("-inf"))
    b["behave"] = add_noise(engine_logp(b["logits"], b["actions"], V), 0.1, 3)
    loss, dl, aux = _shard_parity(b, bounds, oracle.NORM_CONST_K, 3.0)
    assert (dl[mask] == 0).all()


def test_global_group_count():
    # n_groups_total as a data-parallel shard of a larger batch passes it: every w_i, the loss and dlogits scale
    b = make_batch("tiny", "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    losses, dl, auxes, _ = run_sharded(b, A32, [0, 300, 1024], norm=grpo.GRPO_NORM_CONST_K, k=cfg.k, c=3.0, ngt=17.0)
    ref = oracle.loss_rows(to_np_logits(b["logits"]), oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], cfg.G,
                           norm=oracle.NORM_CONST_K, k=cfg.k, dual_clip_c=3.0, n_groups_total=17.0)
    assert abs(losses[0] - ref.loss) <= LOSS_RTOL * abs(ref.loss)
    kinks = kink_rows(ref, oi["behave"], None, A64[oi["seg"].tok_traj], 0.2, 0.2, 3.0)
    check_dlogits(dl_to_f64(dl), ref.dlogits, False, exempt=kinks, what="n_groups_total")


def test_forward_only_and_in_place():
    b = make_batch("tiny", "cuda")
    cfg = b["cfg"]
    _, A32 = _adv(b)
    bounds = [0, 256, 1024]
    kw = dict(norm=grpo.GRPO_NORM_CONST_K, k=cfg.k, c=3.0)
    losses, dl, _, _ = run_sharded(b, A32, bounds, **kw)
    losses_f, dl_f, _, _ = run_sharded(b, A32, bounds, dlogits=False, **kw)
    assert dl_f is None and losses_f == losses
    # dlogits written over the logits themselves, shard by shard, after every shard's records exist
    work = b["logits"].clone()
    stats = shard_stats(work, b["actions"], bounds)
    dev = device_batch(b)
    for b0, b1 in zip(bounds[:-1], bounds[1:]):
        view = work[:, b0:b1]
        grpo.grpo_loss_fwd_bwd_vocab_shard(view, stats, b0, b["V"], b["actions"], b["behave"], A32,
                                           dev["step_tok_off"], dev["traj_step_off"], cfg.G, dual_clip_c=3.0,
                                           k=cfg.k, dlogits=view)
    torch.cuda.synchronize()
    assert torch.equal(work, dl)


def test_invalid_actions_flagged_rows_zero():
    b = make_batch("tiny", "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    act = b["actions"].clone()
    act[3], act[50] = -1, b["V"]  # outside the whole vocabulary: no shard owns them
    losses, dl, auxes, _ = run_sharded(b, A32, [0, 400, 1024], norm=grpo.GRPO_NORM_CONST_K, k=cfg.k, actions=act)
    assert auxes[0].error_flags.item() & grpo.GRPO_FLAG_ACTION
    assert (dl[3] == 0).all() and (dl[50] == 0).all()
    oi = oracle_inputs(b, A64)
    a_np = act.cpu().numpy()
    ref = oracle.loss_rows(to_np_logits(b["logits"]), a_np, oi["behave"], None, oi["adv"], oi["seg"], cfg.G,
                           norm=oracle.NORM_CONST_K, k=cfg.k)
    assert ref.flags & oracle.ERR_ACTION
    assert abs(losses[0] - ref.loss) <= LOSS_RTOL * abs(ref.loss)
    kinks = kink_rows(ref, oi["behave"], None, A64[oi["seg"].tok_traj], 0.2, 0.2, 0.0)
    check_dlogits(dl_to_f64(dl), ref.dlogits, False, exempt=kinks, what="invalid actions")


def test_empty_batch():
    N = 4
    sto = torch.zeros(5, dtype=torch.int32, device="cuda")
    tso = torch.arange(0, 5, dtype=torch.int32, device="cuda")
    logits = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    act = torch.empty(0, dtype=torch.int32, device="cuda")
    stats = grpo.grpo_vocab_shard_stats(logits, act, 0)
    assert stats.shape == (0, grpo.VOCAB_STATS_BYTES)
    loss, dl = grpo.grpo_loss_fwd_bwd_vocab_shard(logits, stats[None], 0, 64, act, torch.empty(0, device="cuda"),
                                                  torch.zeros(N, device="cuda"), sto, tso, 4)
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and dl.shape == (0, 64)

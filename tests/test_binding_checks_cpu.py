"""The Python binding's argument checks, on the CPU: every entry point refuses a tensor of the wrong dtype or too
few elements (which would make the kernels read or write past the caller's buffer) before it looks at where the
tensors live, and then refuses host tensors (there is no CPU path).  Each case changes one argument of an otherwise
valid call and expects the error that names it; nothing reaches the library's compute entry points."""
import pytest
import torch

import paper_2606_05597_amd as grpo

T, V, H, N, G = 12, 64, 64, 4, 2
i32, f32, f64, bf16 = torch.int32, torch.float32, torch.float64, torch.bfloat16


def _loss_args(**over):
    a = dict(logits=torch.zeros(T, V, dtype=bf16), actions=torch.zeros(T, dtype=i32),
             behave_logp=torch.zeros(T, dtype=f32), adv=torch.zeros(N, dtype=f32),
             step_tok_off=torch.tensor([0, 3, 6, 9, T], dtype=i32), traj_step_off=torch.arange(N + 1, dtype=i32),
             group_size=G)
    a.update(over)
    return a


def _loss(**over):
    a = _loss_args(**{k: v for k, v in over.items() if k in _loss_args()})
    kw = {k: v for k, v in over.items() if k not in a}
    return grpo.grpo_loss_fwd_bwd(a.pop("logits"), a.pop("actions"), a.pop("behave_logp"), a.pop("adv"),
                                  a.pop("step_tok_off"), a.pop("traj_step_off"), a.pop("group_size"), **kw)


@pytest.mark.parametrize("over,err,match", [
    (dict(actions=torch.zeros(T, dtype=torch.int64)), TypeError, "actions"),
    (dict(actions=torch.zeros(T - 1, dtype=i32)), ValueError, "actions"),
    (dict(behave_logp=torch.zeros(T - 1, dtype=f32)), ValueError, "behave_logp"),
    (dict(behave_logp=torch.zeros(T, dtype=f64)), TypeError, "behave_logp"),
    (dict(prox_logp=torch.zeros(T - 1, dtype=f32)), ValueError, "prox_logp"),
    (dict(adv=torch.zeros(N - 1, dtype=f32)), ValueError, "adv"),
    (dict(adv=torch.zeros(N, dtype=bf16)), TypeError, "adv"),
    (dict(step_tok_off=torch.tensor([0, 3, 6, 9, T], dtype=torch.int64)), TypeError, "step_tok_off"),
    (dict(logits=torch.zeros(T, V, dtype=torch.float16)), TypeError, "logits"),
    (dict(logits=torch.zeros(V, T, dtype=bf16).t()), ValueError, "logits"),
    (dict(dlogits=torch.zeros(T, V, dtype=f32)), TypeError, "dlogits"),
    (dict(dlogits=torch.zeros(T, V + 8, dtype=bf16)), ValueError, "dlogits"),
    (dict(loss_out=torch.zeros(1, dtype=f32)), TypeError, "loss_out"),
    (dict(aux=grpo.LossAux(token_logp=torch.zeros(T - 1, dtype=f32))), ValueError, "token_logp"),
    (dict(aux=grpo.LossAux(traj_loss=torch.zeros(N, dtype=f32))), TypeError, "traj_loss"),
    (dict(aux=grpo.LossAux(gather_idx=torch.zeros(T, dtype=i32))), TypeError, "gather_idx"),
    (dict(aux=grpo.LossAux(ratio_stats=torch.zeros(7, dtype=f64))), ValueError, "ratio_stats"),
    (dict(), ValueError, "GPU tensor"),
])
def test_loss_entry_checks(over, err, match):
    with pytest.raises(err, match=match):
        _loss(**over)


def _fused(entry="fused_lmhead_grpo", **over):
    a = dict(hidden=torch.zeros(T, H, dtype=bf16), w_lm=torch.zeros(H, V, dtype=bf16),
             actions=torch.zeros(T, dtype=i32), behave_logp=torch.zeros(T, dtype=f32), adv=torch.zeros(N, dtype=f32),
             step_tok_off=torch.tensor([0, 3, 6, 9, T], dtype=i32), traj_step_off=torch.arange(N + 1, dtype=i32))
    kw = {}
    for k, v in over.items():
        (a if k in a else kw)[k] = v
    return getattr(grpo, entry)(a["hidden"], a["w_lm"], a["actions"], a["behave_logp"], a["adv"], a["step_tok_off"],
                                a["traj_step_off"], G, **kw)


@pytest.mark.parametrize("entry", ["fused_lmhead_grpo", "fused_lmhead_grpo_blocked"])
@pytest.mark.parametrize("over,err,match", [
    (dict(dhidden=torch.zeros(T, H, dtype=f32)), TypeError, "dhidden"),
    (dict(dhidden=torch.zeros(T - 1, H, dtype=bf16)), ValueError, "dhidden"),
    (dict(dw_lm=torch.zeros(H, V, dtype=bf16)), TypeError, "dw_lm"),
    (dict(dw_lm=torch.zeros(H * V - 1, dtype=f32)), ValueError, "dw_lm"),
    (dict(actions=torch.zeros(T, dtype=f32)), TypeError, "actions"),
    (dict(actions=torch.zeros(T - 2, dtype=i32)), ValueError, "actions"),
    (dict(behave_logp=torch.zeros(3, dtype=f32)), ValueError, "behave_logp"),
    (dict(adv=torch.zeros(1, dtype=f32)), ValueError, "adv"),
    (dict(w_lm=torch.zeros(H + 64, V, dtype=bf16)), ValueError, "disagree on H"),
    (dict(hidden=torch.zeros(T, H, dtype=f32)), TypeError, "hidden"),
    (dict(), ValueError, "GPU tensor"),
])
def test_fused_entry_checks(entry, over, err, match):
    with pytest.raises(err, match=match):
        _fused(entry, **over)


@pytest.mark.parametrize("over,err,match", [
    (dict(actions=torch.zeros(T - 1, dtype=i32)), ValueError, "actions"),
    (dict(actions=torch.zeros(T, dtype=torch.int64)), TypeError, "actions"),
    (dict(error_flags=torch.zeros(1, dtype=torch.int64)), TypeError, "error_flags"),
    (dict(), ValueError, "GPU tensor"),
])
def test_token_logp_checks(over, err, match):
    a = dict(logits=torch.zeros(T, V, dtype=bf16), actions=torch.zeros(T, dtype=i32))
    kw = {k: v for k, v in over.items() if k not in a}
    a.update({k: v for k, v in over.items() if k in a})
    with pytest.raises(err, match=match):
        grpo.grpo_token_logp(a["logits"], a["actions"], **kw)
    h = dict(hidden=torch.zeros(T, H, dtype=bf16), w_lm=torch.zeros(H, V, dtype=bf16))
    with pytest.raises(err, match=match):
        grpo.fused_lmhead_token_logp(h["hidden"], h["w_lm"], a["actions"], **kw)


@pytest.mark.parametrize("over,err,match", [
    (dict(actions=torch.zeros(T - 1, dtype=i32)), ValueError, "actions"),
    (dict(stats=torch.zeros(T, 16, dtype=torch.uint8)), ValueError, "stats"),
    (dict(stats=torch.zeros(T, 24, dtype=torch.int8)), TypeError, "stats"),
    (dict(), ValueError, "GPU tensor"),
])
def test_vocab_shard_stats_checks(over, err, match):
    actions = over.pop("actions", torch.zeros(T, dtype=i32))
    with pytest.raises(err, match=match):
        grpo.grpo_vocab_shard_stats(torch.zeros(T, V, dtype=bf16), actions, 0, **over)
    with pytest.raises(err, match=match):
        grpo.fused_lmhead_vocab_shard_stats(torch.zeros(T, H, dtype=bf16), torch.zeros(H, V, dtype=bf16), actions, 0,
                                            **over)


@pytest.mark.parametrize("over,err,match", [
    (dict(stats_all=torch.zeros(2, T - 1, 24, dtype=torch.uint8)), ValueError, "stats_all"),
    (dict(actions=torch.zeros(T - 1, dtype=i32)), ValueError, "actions"),
    (dict(adv=torch.zeros(N - 1, dtype=f32)), ValueError, "adv"),
    (dict(), ValueError, "GPU tensor"),
])
def test_vocab_shard_loss_checks(over, err, match):
    a = dict(stats_all=torch.zeros(2, T, 24, dtype=torch.uint8), actions=torch.zeros(T, dtype=i32),
             adv=torch.zeros(N, dtype=f32))
    a.update(over)
    rest = (torch.zeros(T, dtype=f32), a["adv"], torch.tensor([0, 3, 6, 9, T], dtype=i32),
            torch.arange(N + 1, dtype=i32), G)
    with pytest.raises(err, match=match):
        grpo.grpo_loss_fwd_bwd_vocab_shard(torch.zeros(T, V, dtype=bf16), a["stats_all"], 0, 2 * V, a["actions"],
                                           *rest)
    with pytest.raises(err, match=match):
        grpo.fused_lmhead_grpo_vocab_shard(torch.zeros(T, H, dtype=bf16), torch.zeros(H, V, dtype=bf16),
                                           a["stats_all"], 0, 2 * V, a["actions"], *rest)


def test_fused_shard_output_buffers_checked():
    args = (torch.zeros(T, H, dtype=bf16), torch.zeros(H, V, dtype=bf16), torch.zeros(2, T, 24, dtype=torch.uint8), 0,
            2 * V, torch.zeros(T, dtype=i32), torch.zeros(T, dtype=f32), torch.zeros(N, dtype=f32),
            torch.tensor([0, 3, 6, 9, T], dtype=i32), torch.arange(N + 1, dtype=i32), G)
    with pytest.raises(ValueError, match="dhidden_partial"):
        grpo.fused_lmhead_grpo_vocab_shard(*args, dhidden_partial=torch.zeros(T, H - 1, dtype=f32))
    with pytest.raises(ValueError, match="dw_shard"):
        grpo.fused_lmhead_grpo_vocab_shard(*args, dw_shard=torch.zeros(H * V - 1, dtype=f32))
    with pytest.raises(ValueError, match="logits_in"):
        grpo.fused_lmhead_grpo_vocab_shard(*args, logits_in=torch.zeros(10, dtype=f32))


def test_advantages_checks():
    with pytest.raises(TypeError, match="rewards"):
        grpo.grpo_advantages(torch.zeros(8, dtype=f64), 4)
    with pytest.raises(ValueError, match="out"):
        grpo.grpo_advantages(torch.zeros(8, dtype=f32), 4, out=torch.zeros(7, dtype=f32))
    with pytest.raises(ValueError, match="GPU tensor"):
        grpo.grpo_advantages_ex(torch.zeros(8, dtype=f32), 4)

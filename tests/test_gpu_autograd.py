"""The torch.autograd wrappers (GrpoLoss, FusedLmHeadGrpoLoss): loss.backward() hands back exactly the gradients
the entry points return for the same inputs, an upstream gradient other than 1 scales them on the device (the
default "scale" mode), and in "unit" mode the saved gradients come back as the library wrote them.  Neither mode
reads the upstream gradient on the host."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch, make_fused_batch
from tests.test_gpu_fused import small_cfg

pytestmark = pytest.mark.gpu


def _seg(st):
    return torch.from_numpy(st.step_tok_off).cuda(), torch.from_numpy(st.traj_step_off).cuda()


def test_grpo_loss_autograd_matches_entry_point():
    b = make_batch("v32k", "cuda", with_prox=True)  # decoupled: a proximal policy distinct from the behaviour one
    st, cfg = b["structure"], b["cfg"]
    sto, tso = _seg(st)
    adv = torch.from_numpy(oracle.advantages(st.rewards, cfg.G).astype(np.float32)).cuda()
    opts = dict(k=cfg.k, dual_clip_c=3.0, prox_logp=b["prox"])
    want_loss, want_dl = grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, **opts)
    x = b["logits"].clone().requires_grad_(True)
    loss = grpo.GrpoLoss.apply(x, b["actions"], b["behave"], adv, sto, tso, cfg.G, opts)
    assert loss.dim() == 0 and loss.dtype == torch.float64
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == want_loss.item()
    assert torch.equal(x.grad, want_dl)
    # an upstream gradient of 2 (exact in bf16) doubles every element
    x2 = b["logits"].clone().requires_grad_(True)
    (2.0 * grpo.GrpoLoss.apply(x2, b["actions"], b["behave"], adv, sto, tso, cfg.G, opts)).backward()
    torch.cuda.synchronize()
    assert torch.equal(x2.grad, want_dl * 2)
    # "unit": the caller guarantees an upstream gradient of 1, the gradient is the entry point's own tensor
    x3 = b["logits"].clone().requires_grad_(True)
    grpo.GrpoLoss.apply(x3, b["actions"], b["behave"], adv, sto, tso, cfg.G, dict(opts, upstream="unit")).backward()
    torch.cuda.synchronize()
    assert torch.equal(x3.grad, want_dl)
    with pytest.raises(ValueError, match="upstream"):
        grpo.GrpoLoss.apply(x3, b["actions"], b["behave"], adv, sto, tso, cfg.G, dict(opts, upstream="host"))


def test_grpo_loss_autograd_forward_only_without_grad():
    b = make_batch("v32k", "cuda")
    st, cfg = b["structure"], b["cfg"]
    sto, tso = _seg(st)
    adv = torch.from_numpy(oracle.advantages(st.rewards, cfg.G).astype(np.float32)).cuda()
    with torch.no_grad():
        loss = grpo.GrpoLoss.apply(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, dict(k=cfg.k))
    want, _ = grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, k=cfg.k,
                                     dlogits=False)
    torch.cuda.synchronize()
    assert loss.item() == want.item()


@pytest.mark.parametrize("opts", [dict(token_block=256), dict(token_block=256, aux_stream="side"),
                                  dict(schedule="chunked", vocab_chunk=512)])
def test_fused_autograd_matches_entry_point(opts):
    b = make_fused_batch(small_cfg(4, 8, 128, 1000, seed=41, tok_mean=6.0, steps=(2, 6)), "cuda")
    st, cfg = b["structure"], b["cfg"]
    sto, tso = _seg(st)
    adv = torch.from_numpy(oracle.advantages(st.rewards, cfg.G).astype(np.float32)).cuda()
    opts = dict(opts, k=cfg.k, dual_clip_c=3.0)
    if opts.get("aux_stream") == "side":
        opts["aux_stream"] = torch.cuda.Stream()
    direct = dict(opts)
    entry = grpo.fused_lmhead_grpo if direct.pop("schedule", None) == "chunked" else grpo.fused_lmhead_grpo_blocked
    want_loss, want_dh, want_dw = entry(b["hidden"], b["W"], b["actions"], b["behave"], adv, sto, tso, cfg.G,
                                        **direct)
    h = b["hidden"].clone().requires_grad_(True)
    w = b["W"].clone().requires_grad_(True)
    loss = grpo.FusedLmHeadGrpoLoss.apply(h, w, b["actions"], b["behave"], adv, sto, tso, cfg.G, opts)
    loss.backward()
    torch.cuda.synchronize()
    assert loss.item() == want_loss.item()
    assert torch.equal(h.grad, want_dh)
    assert w.grad.dtype == torch.bfloat16 and torch.equal(w.grad, want_dw.to(torch.bfloat16))
    # an upstream gradient of 0.5 (exact) halves both gradients
    h2 = b["hidden"].clone().requires_grad_(True)
    w2 = b["W"].clone().requires_grad_(True)
    (0.5 * grpo.FusedLmHeadGrpoLoss.apply(h2, w2, b["actions"], b["behave"], adv, sto, tso, cfg.G, opts)).backward()
    torch.cuda.synchronize()
    assert torch.equal(h2.grad, want_dh * 0.5) and torch.equal(w2.grad, (want_dw * 0.5).to(torch.bfloat16))


def test_loss_from_rewards_equals_the_two_calls():
    # grpo.loss: advantages from the rewards, then the loss, in one call; bit-identical to making the two calls
    b = make_batch("v32k", "cuda")
    st, cfg = b["structure"], b["cfg"]
    sto, tso = _seg(st)
    l1, d1 = grpo.loss(b["logits"], b["actions"], b["behave"], b["rewards"], sto, tso, cfg.G, k=cfg.k,
                       dual_clip_c=3.0)
    adv = grpo.grpo_advantages(b["rewards"], cfg.G)
    l2, d2 = grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, k=cfg.k,
                                    dual_clip_c=3.0)
    torch.cuda.synchronize()
    assert torch.equal(l1, l2) and torch.equal(d1, d2)

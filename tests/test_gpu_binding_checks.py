"""The Python binding's checks of caller-supplied buffers: a workspace, loss scalar or optional output on the wrong
device, of the wrong dtype or too small is refused before any launch (the library would otherwise be handed a host
pointer or write past the buffer), and a workspace of any dtype is passed with its size in bytes."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import device_batch

pytestmark = pytest.mark.gpu


def _call(b, **kw):
    dev = device_batch(b)
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    adv = torch.from_numpy(A.astype(np.float32)).cuda()
    return grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, dev["step_tok_off"],
                                  dev["traj_step_off"], b["cfg"].G, V=b["V"], **kw)


def test_caller_buffers_checked():
    b = make_batch("tiny", "cuda")
    T, N = b["logits"].shape[0], len(b["structure"].rewards)
    need = grpo.grpo_loss_workspace_bytes(T, N)
    with pytest.raises(ValueError, match="workspace"):
        _call(b, workspace=torch.empty(need, dtype=torch.uint8))  # host memory
    with pytest.raises(TypeError, match="loss_out"):  # a wrong dtype is a TypeError, a wrong size or place ValueError
        _call(b, loss_out=torch.empty(1, dtype=torch.float32, device="cuda"))
    short = grpo.LossAux.alloc(T, N, "cuda")
    short.token_logp = torch.empty(T - 1, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError, match="token_logp"):
        _call(b, aux=short)
    wrong = grpo.LossAux.alloc(T, N, "cuda")
    wrong.traj_loss = torch.empty(N, dtype=torch.float32, device="cuda")
    with pytest.raises(TypeError, match="traj_loss"):
        _call(b, aux=wrong)


def test_workspace_of_any_dtype_sized_in_bytes():
    b = make_batch("tiny", "cuda")
    T, N = b["logits"].shape[0], len(b["structure"].rewards)
    need = grpo.grpo_loss_workspace_bytes(T, N)
    ws = torch.empty((need + 3) // 4, dtype=torch.float32, device="cuda")  # need bytes in a quarter the elements
    lo = torch.empty(1, dtype=torch.float64, device="cuda")
    loss, dl = _call(b, workspace=ws, loss_out=lo)
    ref, dl_ref = _call(b)
    torch.cuda.synchronize()
    assert loss.data_ptr() == lo.data_ptr()
    assert loss.item() == ref.item()
    assert torch.equal(dl, dl_ref)


def test_fused_logp_error_flags_checked():
    h = torch.randn(8, 64, device="cuda").to(torch.bfloat16)
    w = torch.randn(64, 256, device="cuda").to(torch.bfloat16)
    a = torch.zeros(8, dtype=torch.int32, device="cuda")
    with pytest.raises(TypeError, match="error_flags"):
        grpo.fused_lmhead_token_logp(h, w, a, error_flags=torch.zeros(1, dtype=torch.int64, device="cuda"))
    flags = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    grpo.fused_lmhead_token_logp(h, w, a, error_flags=flags)
    torch.cuda.synchronize()
    assert flags.item() == 0


def test_fused_caller_buffers_checked():
    from tests.test_gpu_fused_edges import edge_batch
    e = edge_batch(300, 64, 520, seed=5)
    A = oracle.advantages(e["rewards"], e["G"])
    args = (e["hidden"], e["W"], torch.from_numpy(e["actions"]).cuda(), torch.from_numpy(e["behave"]).cuda(),
            torch.from_numpy(A.astype(np.float32)).cuda(), torch.from_numpy(e["sto"]).cuda(),
            torch.from_numpy(e["tso"]).cuda(), e["G"])
    need = grpo.fused_lmhead_blocked_workspace_bytes(300, 64, 520, 256, len(e["rewards"]))
    with pytest.raises(ValueError, match="workspace"):
        grpo.fused_lmhead_grpo_blocked(*args, token_block=256, workspace=torch.empty(need, dtype=torch.uint8))
    with pytest.raises(ValueError, match="loss_out"):
        grpo.fused_lmhead_grpo_blocked(*args, token_block=256,
                                       loss_out=torch.empty(1, dtype=torch.float64, device="cpu"))
    aux = grpo.LossAux.alloc(300, len(e["rewards"]), "cuda")
    aux.gather_idx = torch.empty(300, dtype=torch.int32, device="cuda")
    with pytest.raises(TypeError, match="gather_idx"):
        grpo.fused_lmhead_grpo_blocked(*args, token_block=256, aux=aux)
    # the same call with valid buffers of the caller's
    ws = torch.empty((need + 7) // 8, dtype=torch.float64, device="cuda")
    loss, dh, dw = grpo.fused_lmhead_grpo_blocked(*args, token_block=256, workspace=ws)
    ref, dh_ref, dw_ref = grpo.fused_lmhead_grpo_blocked(*args, token_block=256)
    torch.cuda.synchronize()
    assert loss.item() == ref.item() and torch.equal(dh, dh_ref) and torch.equal(dw, dw_ref)

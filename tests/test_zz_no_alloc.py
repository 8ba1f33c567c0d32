"""grpo_loss_fwd_bwd_noalloc (the logits path with the library's per-device scratch array as its workspace, for
callers that cannot allocate) against grpo_loss_fwd_bwd with a caller workspace: the same kernels on the same
inputs, so every output must be bit-identical.  Two calls in a row share the array: the first at V = 151,936 with
~800 rows (the persistent row kernel, several rows per workgroup), the second on a smaller batch (the tiny fp32
one), which must not see anything the first left behind; then a batch too large for the array is refused."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch
from tests.gpu_parity import device_batch
from tests.test_gpu_loss import _edge_batch

pytestmark = pytest.mark.gpu


def _outputs(b, entry, dl, loss, aux):
    dev = device_batch(b)
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    adv = torch.from_numpy(A.astype(np.float32)).cuda()
    kw = dict(V=b["V"], prox_logp=b["prox"], norm=grpo.GRPO_NORM_TRAJ_STEPS, k=b["cfg"].k, dual_clip_c=3.0,
              dlogits=dl, aux=aux, loss_out=loss)
    entry(b["logits"], b["actions"], b["behave"], adv, dev["step_tok_off"], dev["traj_step_off"], b["cfg"].G, **kw)
    torch.cuda.synchronize()
    return loss, dl, aux


def _compare(b, what):
    T, N = b["logits"].shape[0], len(b["structure"].rewards)
    outs = []
    for entry in (grpo.grpo_loss_fwd_bwd, grpo.grpo_loss_fwd_bwd_noalloc):
        outs.append(_outputs(b, entry, torch.full_like(b["logits"], float("nan")),
                             torch.full((1,), float("nan"), dtype=torch.float64, device="cuda"),
                             grpo.LossAux.alloc(T, N, "cuda")))
    (l0, d0, a0), (l1, d1, a1) = outs
    assert torch.equal(l0, l1), (what, l0.item(), l1.item())
    assert torch.equal(d0, d1), what
    for f in ("token_logp", "tok_traj", "traj_tok_off", "gather_idx", "traj_loss", "clip_counts", "ratio_stats",
              "error_flags"):
        assert torch.equal(getattr(a0, f), getattr(a1, f)), (what, f)
    assert a1.error_flags.item() == 0
    return l1.item()


def test_noalloc_matches_workspace_entry_on_two_calls():
    big = _edge_batch(151936, "bf16", n_groups=4, G=4, seed=34, max_tok=48)
    assert big["structure"].T > 512
    need = grpo.grpo_loss_workspace_bytes(big["structure"].T, len(big["structure"].rewards))
    assert need <= grpo.GRPO_NOALLOC_SCRATCH_BYTES
    _compare(big, "V = 151,936")
    small = make_batch("tiny", "cuda", with_prox=True)
    assert small["structure"].T < big["structure"].T
    _compare(small, "tiny")


def test_noalloc_refuses_a_batch_larger_than_its_array():
    T = 1 << 20
    assert grpo.grpo_loss_workspace_bytes(T, 4) > grpo.GRPO_NOALLOC_SCRATCH_BYTES
    logits = torch.zeros((T, 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(grpo.GrpoError) as e:
        grpo.grpo_loss_fwd_bwd_noalloc(logits, torch.zeros(T, dtype=torch.int32, device="cuda"),
                                       torch.zeros(T, device="cuda"), torch.zeros(4, device="cuda"),
                                       torch.tensor([0, T // 4, T // 2, 3 * T // 4, T], dtype=torch.int32,
                                                    device="cuda"),
                                       torch.arange(5, dtype=torch.int32, device="cuda"), 4, dlogits=False)
    assert e.value.status == grpo._lib.GRPO_ERR_WORKSPACE

"""grpo_loss_fwd_bwd_noalloc (the logits path with the library's per-device scratch array as its workspace, for
callers that cannot allocate) against grpo_loss_fwd_bwd with a caller workspace: the same kernels on the same
inputs, so every output must be bit-identical.  Two calls in a row share the array: the first at V = 151,936 with
~800 rows (the persistent row kernel, several rows per workgroup), the second on a smaller batch (the tiny fp32
one), which must not see anything the first left behind; then a batch too large for the array is refused.  Last, the
callers the entry point is for: the call captured into a graph (every tensor allocated before the capture) and
replayed three times, with eager calls on the same scratch array and synchronisation between the replays, each
replay bit-identical to the eager call."""
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


def test_noalloc_replays_under_graph_capture():
    b = _edge_batch(151936, "bf16", n_groups=4, G=4, seed=35, max_tok=48)
    T, N = b["logits"].shape[0], len(b["structure"].rewards)
    dev = device_batch(b)
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    adv = torch.from_numpy(A.astype(np.float32)).cuda()

    def call(dl, loss, aux):
        grpo.grpo_loss_fwd_bwd_noalloc(b["logits"], b["actions"], b["behave"], adv, dev["step_tok_off"],
                                       dev["traj_step_off"], b["cfg"].G, V=b["V"], norm=grpo.GRPO_NORM_CONST_K,
                                       k=b["cfg"].k, dual_clip_c=3.0, dlogits=dl, aux=aux, loss_out=loss)

    def alloc():
        return (torch.full_like(b["logits"], float("nan")), torch.full((1,), float("nan"), dtype=torch.float64,
                                                                          device="cuda"), grpo.LossAux.alloc(T, N, "cuda"))

    dl0, loss0, aux0 = alloc()
    call(dl0, loss0, aux0)  # eager reference (also the device's first call, which looks the array up)
    torch.cuda.synchronize()
    assert aux0.error_flags.item() == 0
    dl1, loss1, aux1 = alloc()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(dl1, loss1, aux1)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(dl1, loss1, aux1)
    fields = ("token_logp", "tok_traj", "traj_tok_off", "gather_idx", "traj_loss", "clip_counts", "ratio_stats",
              "error_flags")
    for rep in range(3):
        dl1.fill_(float("nan"))
        loss1.fill_(float("nan"))
        aux1.token_logp.fill_(float("nan"))
        aux1.traj_loss.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(loss1, loss0), (rep, loss1.item(), loss0.item())
        assert torch.equal(dl1, dl0), rep
        for f in fields:
            assert torch.equal(getattr(aux1, f), getattr(aux0, f)), (rep, f)
        # eager work on the same scratch array between the replays: another batch through the same entry point
        small = make_batch("tiny", "cuda")
        sd = device_batch(small)
        sa = torch.from_numpy(oracle.advantages(small["structure"].rewards, small["cfg"].G).astype(np.float32)).cuda()
        grpo.grpo_loss_fwd_bwd_noalloc(small["logits"], small["actions"], small["behave"], sa, sd["step_tok_off"],
                                       sd["traj_step_off"], small["cfg"].G, norm=grpo.GRPO_NORM_CONST_K,
                                       k=small["cfg"].k)
        torch.cuda.synchronize()

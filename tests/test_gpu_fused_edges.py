"""Edge shapes of the fused LM head in every entry point (vocabulary chunks, token blocks on one and on two
streams, forward only) against the fp64 oracle: a single token, the smallest vocabulary (8), H not a multiple of
the 256-wide tile (64, 192), V not a multiple of it, token blocks whose last block holds one row, empty steps.
Gates as in tests/test_gpu_fused.py (the loss within 1e-5 of sum_t |w s_t|, check_fused_loss)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from oracle import fused
from synth.rollouts import Config
from tests.gpu_parity import check_fused_loss, gpu_norm
from tests.test_gpu_fused import bits, check_dh, check_dw

pytestmark = pytest.mark.gpu


def edge_batch(T, H, V, seed, n_traj=4):
    rng = np.random.default_rng(seed)
    steps = rng.integers(1, 3, n_traj)
    n_steps = int(steps.sum())
    toks = np.zeros(n_steps, np.int64)
    for _ in range(T):  # T tokens over the steps, some steps left empty
        toks[rng.integers(0, n_steps)] += 1
    sto = np.concatenate([[0], np.cumsum(toks)]).astype(np.int32)
    tso = np.concatenate([[0], np.cumsum(steps)]).astype(np.int32)
    gen = torch.Generator("cuda").manual_seed(seed)
    hidden = torch.randn((T, H), device="cuda", generator=gen).to(torch.bfloat16)
    W = (0.25 * torch.randn((H, V), device="cuda", generator=gen)).to(torch.bfloat16)
    actions = rng.integers(0, V, T).astype(np.int32)
    z = fused.as_f64(bits(hidden)) @ fused.as_f64(bits(W))
    lp = oracle.logp_entropy(z, actions).token_logp
    behave = (lp + 0.1 * rng.standard_normal(T)).astype(np.float32)
    rewards = np.array([1, 0] * (n_traj // 2), np.float32)
    return dict(hidden=hidden, W=W, z=z, actions=actions, behave=behave, rewards=rewards, sto=sto, tso=tso,
                T=T, H=H, V=V, G=n_traj)


@pytest.mark.parametrize("T,H,V", [(1, 64, 8), (3, 64, 264), (257, 64, 520), (300, 192, 1000), (513, 128, 2056)])
def test_fused_edges_all_entry_points(T, H, V):
    e = edge_batch(T, H, V, seed=T + H + V)
    A = oracle.advantages(e["rewards"], e["G"])
    A32 = torch.from_numpy(A.astype(np.float32)).cuda()
    seg = oracle.segments(T, e["sto"], e["tso"])
    ref = fused.fused_loss(bits(e["hidden"]), bits(e["W"]), e["actions"], e["behave"], None,
                           A.astype(np.float32).astype(np.float64), seg, e["G"], norm=oracle.NORM_CONST_K, k=4.0,
                           dual_clip_c=3.0)
    args = (e["hidden"], e["W"], torch.from_numpy(e["actions"]).cuda(), torch.from_numpy(e["behave"]).cuda(), A32,
            torch.from_numpy(e["sto"]).cuda(), torch.from_numpy(e["tso"]).cuda(), e["G"])
    kw = dict(norm=gpu_norm(oracle.NORM_CONST_K), k=4.0, dual_clip_c=3.0)
    runs = {
        "chunked": lambda aux: grpo.fused_lmhead_grpo(*args, vocab_chunk=256, aux=aux, **kw),
        "blocked": lambda aux: grpo.fused_lmhead_grpo_blocked(*args, token_block=256, aux=aux, **kw),
        "blocked2": lambda aux: grpo.fused_lmhead_grpo_blocked(*args, token_block=256, aux=aux,
                                                               aux_stream=torch.cuda.Stream(), **kw),
    }
    h64, W64 = fused.as_f64(bits(e["hidden"])), fused.as_f64(bits(e["W"]))
    for name, call in runs.items():
        aux = grpo.LossAux.alloc(T, e["G"], "cuda")
        loss, dh, dW = call(aux)
        torch.cuda.synchronize()
        check_fused_loss(loss.item(), ref.rows.token_contrib, name)
        assert np.abs(aux.token_logp.cpu().numpy() - ref.rows.token_logp).max() <= 5e-5, name
        assert aux.error_flags.item() == 0, name
        check_dh(dh.float().cpu().numpy().astype(np.float64), ref.dhidden, ref.rows.dlogits, W64, name)
        check_dw(dW.cpu().numpy().astype(np.float64), ref.dW, h64, ref.rows.dlogits, name)
    logp, ent = grpo.fused_lmhead_token_logp(e["hidden"], e["W"], torch.from_numpy(e["actions"]).cuda())
    torch.cuda.synchronize()
    fref = oracle.logp_entropy(e["z"], e["actions"])
    assert np.abs(logp.cpu().numpy() - fref.token_logp).max() <= 5e-5
    assert (np.abs(ent.cpu().numpy() - fref.token_entropy) <= 1e-4 + 2e-5 * np.abs(fref.token_entropy)).all()

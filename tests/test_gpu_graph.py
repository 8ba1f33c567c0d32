"""The entry points inside a HIP graph (torch.cuda.CUDAGraph over the ROCm runtime).

The library never allocates, frees or synchronises, clears its flags and counters with kernels (no memset
nodes), and puts every launch on the caller's stream, so a training step can capture it once and replay it.
Each case captures one call with all buffers preallocated, then replays the graph several times with eager
work and host synchronisation in between, changing the inputs in place before some replays, and checks
every replay bit for bit against an eager call on the same inputs.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import make_batch, make_fused_batch
from tests.test_gpu_fused import small_cfg

pytestmark = pytest.mark.gpu


def _capture(fn):
    fn()  # warm-up outside the graph (module loading)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_loss_fwd_bwd_graph_replays():
    b = make_batch("v32k", "cuda")
    st = b["structure"]
    T, V = b["logits"].shape
    N = len(st.rewards)
    sto = torch.from_numpy(st.step_tok_off).cuda()
    tso = torch.from_numpy(st.traj_step_off).cuda()
    adv = torch.from_numpy(oracle.advantages(st.rewards, b["cfg"].G).astype(np.float32)).cuda()
    ws = torch.empty(grpo.grpo_loss_workspace_bytes(T, N), dtype=torch.uint8, device="cuda")
    aux = grpo.LossAux.alloc(T, N, "cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dl = torch.empty_like(b["logits"])
    logits = b["logits"].clone()

    def call():
        grpo.grpo_loss_fwd_bwd(logits, b["actions"], b["behave"], adv, sto, tso, b["cfg"].G, dual_clip_c=3.0,
                               dlogits=dl, aux=aux, workspace=ws, loss_out=loss)

    g = _capture(call)
    for rep in range(4):
        if rep == 2:  # new inputs in place: the graph reads whatever the buffers hold
            logits.mul_(0.5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (loss.clone(), dl.clone(), aux.token_logp.clone(), aux.clip_counts.clone(), aux.error_flags.clone())
        dl.fill_(float("nan"))
        aux.clip_counts.fill_(-1)
        aux.error_flags.fill_(-1)
        call()  # eager, same inputs
        torch.cuda.synchronize()
        want = (loss, dl, aux.token_logp, aux.clip_counts, aux.error_flags)
        for x, y in zip(got, want):
            assert torch.equal(x, y), f"replay {rep}"
        assert aux.error_flags.item() == 0


def test_token_logp_and_shard_stats_graph_replays():
    b = make_batch("v32k", "cuda")
    T, V = b["logits"].shape
    logp = torch.empty(T, device="cuda")
    ent = torch.empty(T, device="cuda")
    flags = torch.empty(1, dtype=torch.int32, device="cuda")
    stats = torch.empty((T, grpo.VOCAB_STATS_BYTES), dtype=torch.uint8, device="cuda")
    shard = b["logits"][:, 8000:16000]

    def call():
        r = grpo.grpo_token_logp(b["logits"], b["actions"], error_flags=flags)
        logp.copy_(r[0])
        ent.copy_(r[1])
        grpo.grpo_vocab_shard_stats(shard, b["actions"], 8000, stats=stats)

    g = _capture(call)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        got = (logp.clone(), ent.clone(), flags.clone(), stats.clone())
        logp.zero_()
        stats.zero_()
        flags.fill_(-1)
        call()
        torch.cuda.synchronize()
        for x, y in zip(got, (logp, ent, flags, stats)):
            assert torch.equal(x, y), f"replay {rep}"


def test_fused_graph_replays():
    b = make_fused_batch(small_cfg(2, 4, 128, 2048, seed=31), "cuda")
    st = b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    N = len(st.rewards)
    sto = torch.from_numpy(st.step_tok_off).cuda()
    tso = torch.from_numpy(st.traj_step_off).cuda()
    adv = torch.from_numpy(oracle.advantages(st.rewards, b["cfg"].G).astype(np.float32)).cuda()
    ws = torch.empty(grpo.fused_lmhead_workspace_bytes(T, H, V, 512, N), dtype=torch.uint8, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dh = torch.empty_like(b["hidden"])
    dw = torch.empty((H, V), dtype=torch.float32, device="cuda")

    def call():
        grpo.fused_lmhead_grpo(b["hidden"], b["W"], b["actions"], b["behave"], adv, sto, tso, b["cfg"].G,
                               vocab_chunk=512, dual_clip_c=3.0, dhidden=dh, dw_lm=dw, workspace=ws, loss_out=loss)

    g = _capture(call)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        got = (loss.clone(), dh.clone(), dw.clone())
        dh.zero_()
        dw.fill_(float("nan"))
        call()
        torch.cuda.synchronize()
        for x, y in zip(got, (loss, dh, dw)):
            assert torch.equal(x, y), f"replay {rep}"


@pytest.mark.parametrize("two_streams", [False, True])
def test_fused_blocked_graph_replays(two_streams):
    # token blocks of 256 over ~600 tokens: several blocks, dW accumulated across them inside the graph; with a
    # second stream the capture forks onto it and joins back through the call's events
    b = make_fused_batch(small_cfg(4, 8, 128, 2048, seed=32, tok_mean=6.0, steps=(2, 6)), "cuda")
    st = b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    assert T > 2 * 256
    N = len(st.rewards)
    sto = torch.from_numpy(st.step_tok_off).cuda()
    tso = torch.from_numpy(st.traj_step_off).cuda()
    adv = torch.from_numpy(oracle.advantages(st.rewards, b["cfg"].G).astype(np.float32)).cuda()
    ws = torch.empty(grpo.fused_lmhead_blocked_workspace_bytes(T, H, V, 256, N), dtype=torch.uint8, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dh = torch.empty_like(b["hidden"])
    dw = torch.empty((H, V), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream() if two_streams else None

    def call():
        grpo.fused_lmhead_grpo_blocked(b["hidden"], b["W"], b["actions"], b["behave"], adv, sto, tso, b["cfg"].G,
                                       token_block=256, dual_clip_c=3.0, dhidden=dh, dw_lm=dw, workspace=ws,
                                       loss_out=loss, aux_stream=side)

    g = _capture(call)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        got = (loss.clone(), dh.clone(), dw.clone())
        dh.zero_()
        dw.fill_(float("nan"))
        call()
        torch.cuda.synchronize()
        for x, y in zip(got, (loss, dh, dw)):
            assert torch.equal(x, y), f"replay {rep}"

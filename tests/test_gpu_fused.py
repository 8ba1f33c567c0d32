"""GPU parity of the fused LM-head path against the fp64 oracle, in both schedules: over vocabulary chunks with
the logits recomputed for the backward products (fused_lmhead_grpo), and over token blocks whose logits are kept
between the products (fused_lmhead_grpo_blocked).

Gates.  Loss: relative 1e-5 of sum_t |w_i s_t| (tests/gpu_parity.py check_fused_loss; the
loss's own size when its terms do not cancel).  Token log-probs: absolute 5e-5 (the logits are
fp32 sums of H bf16 products on the GPU).  dhidden and dW: the GPU rounds each
dlogits tile D to bf16 (8 significant bits: relative error <= 2^-8 per element)
before the two products and rounds dhidden to bf16 at the end, so elementwise
    |dh - ref| <= 2^-8 |ref| + 2^-7 (|D| |W|^T)      (bf16 output)
    |dW - ref| <= 2^-7 (|h|^T |D|)                    (fp32 output)
with a factor 2 on the D-rounding term for fp32 accumulation, and the relative
Frobenius error <= 5e-3.  At the full T = 65,536 the oracle computes sampled
rows and every trajectory of the two groups with the fewest tokens (about
14,000 rows, where the group-relative advantages cancel); dW is checked elementwise at the full
H x V with fewer tokens, and at full size through identities that hold at any
size: each row of dW sums to ~0 (each dlogits row sums to 0) and
<dW, W> = <dhidden, h> (= <D, z>).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from oracle import fused
from synth import make_fused_batch
from synth.rollouts import Config
from tests.gpu_parity import check_fused_loss, gpu_norm

pytestmark = pytest.mark.gpu

NORMS = [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K]


def bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def small_cfg(n_groups, G, H, V, seed, tok_mean=4.0, steps=(1, 4), w_sigma=0.25):
    return Config("fused-test", n_groups, G, V, "bf16", 0.0, 0.4, steps, steps, tok_mean, (1, 64), 0.1, 4.0,
                  H=H, w_sigma=w_sigma, seed=seed)


def setup(b):
    st = b["structure"]
    A = oracle.advantages(st.rewards, b["cfg"].G)
    A64 = A.astype(np.float32).astype(np.float64)
    A32 = torch.from_numpy(A.astype(np.float32)).cuda()
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    sto = torch.from_numpy(st.step_tok_off).cuda()
    tso = torch.from_numpy(st.traj_step_off).cuda()
    return A64, A32, seg, sto, tso


class Blocked(int):
    """A schedule argument: the token-blocked entry point with this token_block (a plain int is a vocab_chunk)."""

    def __repr__(self):
        return f"blocked{int(self)}"


def fused_call(b, A32, sto, tso, sched, **kw):
    args = (b["hidden"], b["W"], b["actions"], b["behave"], A32, sto, tso, b["cfg"].G)
    if isinstance(sched, Blocked):
        return grpo.fused_lmhead_grpo_blocked(*args, token_block=int(sched), **kw)
    return grpo.fused_lmhead_grpo(*args, vocab_chunk=sched, **kw)


def run(b, A32, sto, tso, chunk, norm, c, gs=1.0, dw=None, accumulate=False, prox=None, ngt=0.0):
    aux = grpo.LossAux.alloc(b["structure"].T, len(b["structure"].rewards), "cuda")
    loss, dh, dW = fused_call(b, A32, sto, tso, chunk, norm=gpu_norm(norm), k=b["cfg"].k, dual_clip_c=c,
                              grad_scale=gs, dw_lm=dw, accumulate_dw=accumulate, aux=aux, prox_logp=prox,
                              n_groups_total=ngt)
    torch.cuda.synchronize()
    return loss.item(), dh, dW, aux


def check_dh(dh_gpu, ref_dh, D, W64, what=""):
    bound = 2.0 ** -8 * np.abs(ref_dh) + 2.0 ** -7 * (np.abs(D) @ np.abs(W64).T)
    err = np.abs(dh_gpu - ref_dh)
    assert (err <= bound + 1e-30).all(), f"{what}: dhidden bound exceeded by {(err / (bound + 1e-30)).max()}"
    rel = np.linalg.norm(err) / np.linalg.norm(ref_dh)
    assert rel <= 5e-3, f"{what}: dhidden relative Frobenius {rel}"


def check_dw(dw_gpu, ref_dw, h64, D, what=""):
    bound = 2.0 ** -7 * (np.abs(h64).T @ np.abs(D))
    err = np.abs(dw_gpu - ref_dw)
    assert (err <= bound + 1e-30).all(), f"{what}: dW bound exceeded by {(err / (bound + 1e-30)).max()}"
    rel = np.linalg.norm(err) / np.linalg.norm(ref_dw)
    assert rel <= 5e-3, f"{what}: dW relative Frobenius {rel}"


def full_compare(b, chunk, norm, c, gs=1.0, accumulate=False, prox=None, ngt=0.0):
    A64, A32, seg, sto, tso = setup(b)
    H, V = b["H"], b["V"]
    dw0 = None
    if accumulate:
        dw0 = torch.randn((H, V), device="cuda", generator=torch.Generator("cuda").manual_seed(9)) * 1e-3
    dw_in = None if dw0 is None else dw0.clone()
    loss, dh, dW, aux = run(b, A32, sto, tso, chunk, norm, c, gs, dw=dw_in, accumulate=accumulate, prox=prox,
                            ngt=ngt)
    hb, Wb = bits(b["hidden"]), bits(b["W"])
    ref = fused.fused_loss(hb, Wb, b["actions"].cpu().numpy(), b["behave"].cpu().numpy(),
                           None if prox is None else prox.cpu().numpy(), A64, seg, b["cfg"].G, norm=norm,
                           k=b["cfg"].k, dual_clip_c=c, grad_scale=gs, n_groups_total=ngt)
    check_fused_loss(loss, ref.rows.token_contrib, "loss")
    assert np.abs(aux.token_logp.cpu().numpy() - ref.rows.token_logp).max() <= 5e-5
    tt = seg.tok_traj
    for i, got in enumerate(aux.traj_loss.cpu().numpy()):
        check_fused_loss(got, ref.rows.token_contrib[tt == i], f"trajectory {i}")
    assert (aux.tok_traj.cpu().numpy() == seg.tok_traj).all()
    assert aux.error_flags.item() == 0
    h64 = fused.as_f64(hb)
    W64 = fused.as_f64(Wb)
    D = ref.rows.dlogits
    check_dh(dh.float().cpu().numpy().astype(np.float64), ref.dhidden, D, W64, "dhidden")
    dw_gpu = dW.cpu().numpy().astype(np.float64)
    if accumulate:
        dw_gpu -= dw0.cpu().numpy().astype(np.float64)
    check_dw(dw_gpu, ref.dW, h64, D, "dW")
    return ref


@pytest.mark.parametrize("norm", NORMS)
@pytest.mark.parametrize("c", [0.0, 3.0])
@pytest.mark.parametrize("sched", [256, Blocked(256)])
def test_fused_small(norm, c, sched):
    # H = 64, V = 1000, chunks of 256: four chunks, the last 232 wide; T not a multiple of 128 (one token block)
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=11), "cuda")
    assert b["structure"].T % 128 != 0
    full_compare(b, sched, norm, c)


@pytest.mark.parametrize("sched", [2048, Blocked(256)])
def test_fused_medium_multichunk_accumulate(sched):
    # blocked: several blocks of 256 tokens and a ragged last one, dW accumulated over them and onto the input
    b = make_fused_batch(small_cfg(4, 8, 256, 5000, seed=12, tok_mean=6.0, steps=(2, 9)), "cuda")
    if isinstance(sched, Blocked):
        assert b["structure"].T > 3 * 256 and b["structure"].T % 256 != 0
    full_compare(b, sched, oracle.NORM_TRAJ_STEPS, 3.0, gs=0.5, accumulate=True)


@pytest.mark.parametrize("sched", [1024, Blocked(512)])
def test_fused_single_chunk(sched):
    b = make_fused_batch(small_cfg(1, 4, 128, 512, seed=13), "cuda")
    full_compare(b, sched, oracle.NORM_CONST_K, 0.0)


@pytest.mark.parametrize("sched", [256, Blocked(256)])
def test_fused_decoupled_and_global_groups(sched):
    # a proximal policy distinct from the behaviour one (decoupled ratios: the clip acts on pi/pi_prox, the
    # weight is pi_prox/pi_behave), and the normaliser's group count overridden as a data-parallel shard of a
    # 3x larger batch would pass it; several token blocks of 256
    b = make_fused_batch(small_cfg(4, 8, 128, 1000, seed=19, tok_mean=6.0, steps=(2, 6)), "cuda")
    gen = torch.Generator("cuda").manual_seed(20)
    prox = b["behave"] + 0.05 * torch.randn(b["behave"].shape, device="cuda", generator=gen)
    assert b["structure"].T > 2 * 256
    full_compare(b, sched, oracle.NORM_TRAJ_STEPS, 3.0, prox=prox, ngt=12.0)


@pytest.mark.parametrize("sched", [8192, Blocked(256)])
def test_fused_full_hv_reduced_t(sched):
    # the real H = 3584 and V = 151,936 (18 full chunks of 8192 and a 4480 tail), with ~300 tokens (two blocks)
    cfg = Config("fused-hv", 1, 8, 151936, "bf16", 0.0, 0.35, (8, 30), (3, 12), 96.0, (1, 4096), 0.05, 10.0,
                 T_target=320, H=3584, seed=14)
    b = make_fused_batch(cfg, "cuda")
    full_compare(b, sched, oracle.NORM_CONST_K, 3.0)


def test_fused_schedules_agree():
    # both schedules form the logits, their tile partials and the rows' epilogue with the same code on the same
    # inputs: the loss and every per-token output are bit-identical.  The backward products differ in the order of
    # their fp32 sums and in D: the token-blocked schedule forms it from fp16 terms exp(z - m) (relative error
    # <= 2^-11 before D's own bf16 rounding), so about one D element in eight rounds to the neighbouring bf16
    # value, and dW differs at the level of the oracle gate (relative Frobenius 5e-3; measured about 1e-3)
    b = make_fused_batch(small_cfg(4, 8, 256, 5000, seed=17, tok_mean=6.0, steps=(2, 9)), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    l1, dh1, dW1, aux1 = run(b, A32, sto, tso, 1024, oracle.NORM_CONST_K, 3.0)
    l2, dh2, dW2, aux2 = run(b, A32, sto, tso, Blocked(512), oracle.NORM_CONST_K, 3.0)
    assert l1 == l2
    for f in ("token_logp", "traj_loss", "clip_counts", "tok_traj", "error_flags"):
        assert torch.equal(getattr(aux1, f), getattr(aux2, f)), f
    dh1, dh2 = dh1.double(), dh2.double()
    assert ((dh1 - dh2).abs() <= 2.0 ** -7 * dh1.abs() + 1e-3 * dh1.abs().max()).all()
    rel = ((dW1.double() - dW2.double()).norm() / dW1.double().norm()).item()
    print(f"dW between schedules: relative Frobenius {rel:.3g}")
    assert rel <= 5e-3


@pytest.mark.parametrize("tb,cfg_args,extras", [(256, (4, 8, 256, 5000, 18), False),
                                                (256, (4, 8, 256, 5000, 28), True),
                                                (8192, None, False)])
def test_fused_blocked_two_streams_bit_identical(tb, cfg_args, extras):
    # each block's D pass on a second stream beside the next block's forward product: the same kernels on the
    # same data in a different overlap, so every output is bit-identical to the one-stream call (several blocks
    # of 256 rows on a small batch; the full fused workload in 8 blocks of 8192).  extras: dW accumulated onto an
    # input, a proximal policy distinct from the behaviour one, a gradient scale and a global group count.
    if cfg_args is None:
        b = make_fused_batch("fused", "cuda")
    else:
        b = make_fused_batch(small_cfg(*cfg_args[:4], seed=cfg_args[4], tok_mean=6.0, steps=(2, 9)), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    T, N = b["structure"].T, len(b["structure"].rewards)
    H, V = b["H"], b["V"]
    assert T > 2 * tb
    kw = {}
    dw0 = None
    if extras:
        gen = torch.Generator("cuda").manual_seed(29)
        kw = dict(prox_logp=b["behave"] + 0.05 * torch.randn(b["behave"].shape, device="cuda", generator=gen),
                  grad_scale=0.25, n_groups_total=12.0, accumulate_dw=True)
        dw0 = torch.randn((H, V), device="cuda", generator=gen) * 1e-3
    outs = []
    for two in (False, True):
        aux = grpo.LossAux.alloc(T, N, "cuda")
        side = torch.cuda.Stream() if two else None
        dw = None if dw0 is None else dw0.clone()
        loss, dh, dW = fused_call(b, A32, sto, tso, Blocked(tb), norm=gpu_norm(oracle.NORM_CONST_K), k=b["cfg"].k,
                                  dual_clip_c=3.0, aux=aux, aux_stream=side, dw_lm=dw, **kw)
        torch.cuda.synchronize()
        outs.append((loss, dh, dW, aux.token_logp, aux.traj_loss, aux.clip_counts, aux.error_flags))
    for x, y in zip(*outs):
        assert torch.equal(x, y)
    if extras:  # and against the oracle
        ref = fused.fused_loss(bits(b["hidden"]), bits(b["W"]), b["actions"].cpu().numpy(), b["behave"].cpu().numpy(),
                               kw["prox_logp"].cpu().numpy(), A64, seg, b["cfg"].G, norm=oracle.NORM_CONST_K,
                               k=b["cfg"].k, dual_clip_c=3.0, grad_scale=0.25, n_groups_total=12.0)
        check_fused_loss(outs[1][0].item(), ref.rows.token_contrib, "two-stream loss")
        dW = outs[1][2].cpu().numpy().astype(np.float64) - dw0.cpu().numpy().astype(np.float64)
        check_dw(dW, ref.dW, fused.as_f64(bits(b["hidden"])), ref.rows.dlogits, "two-stream dW")
        check_dh(outs[1][1].float().cpu().numpy().astype(np.float64), ref.dhidden, ref.rows.dlogits,
                 fused.as_f64(bits(b["W"])), "two-stream dhidden")


_GROUPS_CACHE = {}


def _whole_groups_oracle(b, hb, W64, A64, seg, n_groups=2, block=1024):
    """The oracle's loss of every trajectory of the n_groups groups with the fewest tokens: z = h W in fp64 for all
    of their rows (in row blocks), then the loss rows.  Group-relative advantages sum to zero over a group
    (Sec. 3.2), so a whole group's loss is where Eq. 1's terms cancel.  Cached per batch seed: both schedules
    are compared with the same oracle values."""
    cfg = b["cfg"]
    key = (cfg.name, cfg.seed, n_groups)
    if key in _GROUPS_CACHE:
        return _GROUPS_CACHE[key]
    G = cfg.G
    tto = seg.traj_tok_off
    sizes = (tto[G::G] - tto[:-1:G]).astype(np.int64)
    groups = np.sort(np.argsort(sizes, kind="stable")[:n_groups])
    actions, behave = b["actions"].cpu().numpy(), b["behave"].cpu().numpy()
    out = []
    for g in groups:
        t0, t1 = int(tto[g * G]), int(tto[(g + 1) * G])
        parts = []
        for r0 in range(t0, t1, block):
            r1 = min(t1, r0 + block)
            z = fused.as_f64(hb[r0:r1]) @ W64
            parts.append(oracle.loss_rows(z, actions, behave, None, A64, seg, G, norm=oracle.NORM_CONST_K, k=cfg.k,
                                          dual_clip_c=3.0, row_begin=r0, row_end=r1, row_offset=r0,
                                          want_dlogits=False))
        contrib = np.concatenate([q.token_contrib for q in parts])
        logp = np.concatenate([q.token_logp for q in parts])
        out.append((int(g), t0, t1, contrib, logp))
    _GROUPS_CACHE[key] = out
    return out


@pytest.mark.parametrize("sched", [8192, Blocked(8192)])
def test_fused_full_size_sampled(sched):
    b = make_fused_batch("fused", "cuda")
    A64, A32, seg, sto, tso = setup(b)
    cfg = b["cfg"]
    loss, dh, dW, aux = run(b, A32, sto, tso, sched, oracle.NORM_CONST_K, 3.0)
    T = b["structure"].T
    hb, Wb = bits(b["hidden"]), bits(b["W"])
    W64 = fused.as_f64(Wb)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([[0, T - 1], rng.integers(0, T, 24)]))
    kw = dict(norm=oracle.NORM_CONST_K, k=cfg.k, dual_clip_c=3.0)
    actions, behave = b["actions"].cpu().numpy(), b["behave"].cpu().numpy()
    part = fused.fused_rows(hb, Wb, rows, actions, behave, None, A64, seg, cfg.G, w_f64=W64, **kw)
    tl = aux.token_logp.cpu().numpy()
    assert np.abs(tl[rows] - part.rows.token_logp).max() <= 5e-5
    check_dh(dh[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64), part.dhidden,
             part.rows.dlogits, W64, "sampled dhidden rows")
    traj_loss = aux.traj_loss.cpu().numpy()
    assert abs(loss - traj_loss.sum()) <= 1e-12 * np.abs(traj_loss).sum()
    # every trajectory of the two groups with the fewest tokens (about 14,000 rows): each trajectory's loss, the
    # groups' losses and every row's log-prob against the oracle
    for g, t0, t1, contrib, logp in _whole_groups_oracle(b, hb, W64, A64, seg):
        assert np.abs(tl[t0:t1] - logp).max() <= 5e-5
        trajs = range(g * cfg.G, (g + 1) * cfg.G)
        for i in trajs:
            check_fused_loss(traj_loss[i], contrib[seg.traj_tok_off[i] - t0:seg.traj_tok_off[i + 1] - t0],
                             f"{sched!r} trajectory {i}")
        check_fused_loss(traj_loss[g * cfg.G:(g + 1) * cfg.G].sum(), contrib, f"{sched!r} group {g} ({t1 - t0} rows)",
                         report=True)
    # identities at full size
    dWn = dW.double()
    row_sums = dWn.sum(1).abs()
    assert (row_sums <= 2.0 ** -7 * dWn.abs().sum(1)).all()
    # both sides use the same bf16 dlogits tiles; dhidden adds one bf16 rounding per element
    lhs = (dWn * b["W"].double()).sum().item()
    prod = dh.double() * b["hidden"].double()
    rhs = prod.sum().item()
    assert abs(lhs - rhs) <= 2.0 ** -7 * prod.abs().sum().item(), (lhs, rhs)
    assert aux.error_flags.item() == 0


@pytest.mark.parametrize("blocked", [False, True])
def test_fused_empty_batch_zeroes_dw(blocked):
    N, H, V = 4, 64, 256
    sto = torch.zeros(5, dtype=torch.int32, device="cuda")
    tso = torch.arange(0, 5, dtype=torch.int32, device="cuda")
    hidden = torch.empty((0, H), dtype=torch.bfloat16, device="cuda")
    W = torch.randn((H, V), device="cuda").to(torch.bfloat16)
    dw = torch.full((H, V), 7.0, device="cuda")
    args = (hidden, W, torch.empty(0, dtype=torch.int32, device="cuda"), torch.empty(0, device="cuda"),
            torch.zeros(N, device="cuda"), sto, tso, 4)
    if blocked:
        loss, dh, dW = grpo.fused_lmhead_grpo_blocked(*args, token_block=256, dw_lm=dw)
    else:
        loss, dh, dW = grpo.fused_lmhead_grpo(*args, vocab_chunk=256, dw_lm=dw)
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and (dW == 0).all()


@pytest.mark.parametrize("sched", [256, Blocked(256)])
def test_fused_invalid_action_row_zero(sched):
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=15), "cuda")
    b["actions"][2] = 1000
    A64, A32, seg, sto, tso = setup(b)
    loss, dh, dW, aux = run(b, A32, sto, tso, sched, oracle.NORM_CONST_K, 0.0)
    assert aux.error_flags.item() == grpo.GRPO_FLAG_ACTION
    assert (dh[2] == 0).all()
    ref = fused.fused_loss(bits(b["hidden"]), bits(b["W"]), b["actions"].cpu().numpy(), b["behave"].cpu().numpy(),
                           None, A64, seg, 4, norm=oracle.NORM_CONST_K, k=4.0)
    assert ref.rows.flags == oracle.ERR_ACTION
    check_fused_loss(loss, ref.rows.token_contrib, "loss with an invalid action")


@pytest.mark.parametrize("sched", [256, Blocked(256)])
def test_fused_nonfinite_hidden_row(sched):
    # a NaN hidden row: its logits, log-sum-exp and log-prob are NaN and flagged and the loss is NaN, while every
    # other row's log-prob and dhidden row are those of the clean batch bit for bit (rows stay independent through
    # the products); dW takes the NaN row's terms
    b = make_fused_batch(small_cfg(2, 4, 64, 1000, seed=21), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    T = b["structure"].T
    l0, dh0, dW0, a0 = run(b, A32, sto, tso, sched, oracle.NORM_CONST_K, 3.0)
    assert a0.error_flags.item() == 0 and math.isfinite(l0)
    r = T // 2
    b["hidden"][r] = float("nan")
    l1, dh1, dW1, a1 = run(b, A32, sto, tso, sched, oracle.NORM_CONST_K, 3.0)
    assert a1.error_flags.item() & grpo.GRPO_FLAG_NONFINITE
    assert math.isnan(l1) and math.isnan(a1.token_logp[r].item())
    keep = torch.arange(T, device="cuda") != r
    assert torch.equal(a1.token_logp[keep], a0.token_logp[keep])
    assert np.array_equal(bits(dh1[keep]), bits(dh0[keep]))
    assert torch.isnan(dW1).any()


def test_fused_rejects_bad_shapes():
    b = make_fused_batch(small_cfg(1, 4, 64, 512, seed=16), "cuda")
    A64, A32, seg, sto, tso = setup(b)
    with pytest.raises(grpo.GrpoError) as e:
        run(b, A32, sto, tso, 300, oracle.NORM_CONST_K, 0.0)  # chunk not a multiple of 256
    assert e.value.status == grpo._lib.GRPO_ERR_SHAPE
    with pytest.raises(grpo.GrpoError) as e:
        run(b, A32, sto, tso, Blocked(300), oracle.NORM_CONST_K, 0.0)  # token block not a multiple of 256
    assert e.value.status == grpo._lib.GRPO_ERR_SHAPE

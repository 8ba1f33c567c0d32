"""GPU parity of the logits path (grpo_loss_fwd_bwd, grpo_advantages) against the oracle.

Every case runs the HIP library through its C ABI and the fp64 oracle on the
same seeded synthetic inputs (synth/), then applies the gates of
tests/gpu_parity.py.  Sizes: the tiny and 32k-vocabulary workloads in full;
the 151,936-vocabulary workloads at full size in the benchmark's launch
configuration, compared on sampled rows and sampled whole trajectories.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_05597_amd as grpo
from synth import CONFIGS, make_batch
from synth.rollouts import Config
from tests.gpu_parity import (LOGP_ATOL, LOSS_RTOL, check_dlogits, dl_to_f64, gpu_norm, kink_rows,
                              oracle_inputs, run_gpu, to_np_logits)

pytestmark = pytest.mark.gpu

NORMS = [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K]


def _adv(b):
    A = oracle.advantages(b["structure"].rewards, b["cfg"].G)
    return A.astype(np.float32).astype(np.float64), torch.from_numpy(A.astype(np.float32)).cuda()


def _full_parity(b, norm, c, scaled_gs=True, check_aux=True):
    """Whole-batch comparison: loss, traj losses, logp, integers, dlogits (with the scaled rerun)."""
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    zl = to_np_logits(b["logits"])
    is_bf16 = b["logits"].dtype == torch.bfloat16
    V = b["V"]
    ref = oracle.loss_rows(zl, oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"], cfg.G, V=V,
                           norm=norm, k=cfg.k, dual_clip_c=c)
    loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=c)
    assert abs(loss - ref.loss) <= LOSS_RTOL * abs(ref.loss), (loss, ref.loss)
    np.testing.assert_allclose(aux.traj_loss.cpu().numpy(), ref.traj_loss, rtol=LOSS_RTOL,
                               atol=LOSS_RTOL * np.abs(ref.traj_loss).max())
    assert np.abs(aux.token_logp.cpu().numpy() - ref.token_logp).max() <= LOGP_ATOL
    if check_aux:
        assert (aux.tok_traj.cpu().numpy() == oi["seg"].tok_traj).all()
        assert (aux.traj_tok_off.cpu().numpy() == oi["seg"].traj_tok_off).all()
        ld = b["logits"].stride(0)
        assert (aux.gather_idx.cpu().numpy() == oracle.gather_index(len(oi["actions"]), ld, oi["actions"])).all()
        assert aux.error_flags.item() == ref.flags == 0
    kinks = kink_rows(ref, oi["behave"], oi["prox"], A64[oi["seg"].tok_traj], 0.2, 0.2, c)
    assert len(kinks) <= max(2, len(oi["actions"]) // 1000), f"unexpectedly many kink rows: {len(kinks)}"
    clip = aux.clip_counts.cpu().numpy()
    st = ref.token_state
    nk = np.ones(len(st), bool)
    nk[kinks] = False
    # clip decisions away from kinks are identical
    assert abs(clip[0] - (st & 1).sum()) <= len(kinks) and abs(clip[1] - ((st >> 1) & 1).sum()) <= len(kinks)
    check_dlogits(dl_to_f64(dl[:, :V]), ref.dlogits, is_bf16, exempt=kinks, what="dlogits")
    if scaled_gs:
        gmax = np.abs(ref.token_g).max()
        gs = 1.0 / gmax
        loss2, dl2, _ = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=c, grad_scale=np.float32(gs), aux=False)
        assert loss2 == loss  # grad_scale does not touch the loss
        # the GPU applies the fp32-rounded grad_scale: scale the reference the same way
        ref_scaled = ref.dlogits * float(np.float32(gs))
        check_dlogits(dl_to_f64(dl2[:, :V]), ref_scaled, is_bf16, exempt=kinks, scaled=True, what="scaled dlogits")
    return ref, loss, dl, aux


# ---------------------------------------------------------------- tiny workload (fp32 [192, 1024])

@pytest.mark.parametrize("norm", NORMS)
@pytest.mark.parametrize("c", [0.0, 3.0])
@pytest.mark.parametrize("decoupled", [False, True])
def test_tiny_parity(norm, c, decoupled):
    b = make_batch("tiny", "cuda", with_prox=decoupled)
    _full_parity(b, norm, c)


def test_tiny_normalizers_coincide_on_gpu():
    # every trajectory has |tau_i| = 3 = k: the two normalisers give the same loss and dlogits
    b = make_batch("tiny", "cuda")
    _, A32 = _adv(b)
    l1, d1, _ = run_gpu(b, A32, norm=grpo.GRPO_NORM_TRAJ_STEPS, k=3.0, c=3.0, aux=False)
    l2, d2, _ = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=3.0, c=3.0, aux=False)
    assert l1 == l2 and torch.equal(d1, d2)


def test_dual_clip_forced():
    # behave = l - 2.5 on negative-advantage tokens: rho = e^2.5 > c = 3, so the floor engages
    b = make_batch("tiny", "cuda")
    A64, A32 = _adv(b)
    st = b["structure"]
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    neg = torch.from_numpy(A64[seg.tok_traj] < 0).cuda()
    l_ref = oracle.loss_rows(to_np_logits(b["logits"]), b["actions"].cpu().numpy(), np.zeros(st.T, np.float32),
                             None, A64, seg, 4, want_dlogits=False).token_logp
    b["behave"] = torch.where(neg, torch.from_numpy((l_ref - 2.5).astype(np.float32)).cuda(), b["behave"])
    ref, _, _, aux = _full_parity(b, oracle.NORM_CONST_K, 3.0)
    assert ((ref.token_state >> 1) & 1).sum() > 0 and aux.clip_counts[1].item() > 0


@pytest.mark.parametrize("eps_low,eps_high", [(0.2, 0.28), (0.0, 0.0), (0.99, 10.0)])
def test_clip_ranges(eps_low, eps_high):
    # an asymmetric range (a wider upper bound), a zero-width one (every ratio but 1 clipped) and one too wide to
    # clip anything ([0.01, 11]: eps_low must stay below 1), with decoupled ratios and the dual clip on
    b = make_batch("tiny", "cuda", with_prox=True)
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    ref = oracle.loss_rows(to_np_logits(b["logits"]), oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"],
                           b["cfg"].G, norm=oracle.NORM_CONST_K, k=b["cfg"].k, eps_low=eps_low, eps_high=eps_high,
                           dual_clip_c=3.0)
    loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(oracle.NORM_CONST_K), k=b["cfg"].k, eps_low=eps_low,
                            eps_high=eps_high, c=3.0)
    assert abs(loss - ref.loss) <= LOSS_RTOL * abs(ref.loss), (loss, ref.loss)
    assert np.abs(aux.token_logp.cpu().numpy() - ref.token_logp).max() <= LOGP_ATOL
    kinks = kink_rows(ref, oi["behave"], oi["prox"], A64[oi["seg"].tok_traj], eps_low, eps_high, 3.0)
    assert len(kinks) <= 2
    check_dlogits(dl_to_f64(dl[:, :b["V"]]), ref.dlogits, False, exempt=kinks, what=f"dlogits eps {eps_low}/{eps_high}")
    clipped = (ref.token_state & 1).sum()
    if eps_low == 0.0:
        assert clipped > 0.4 * len(oi["actions"])  # the clipped branch is taken wherever it is the smaller
    if eps_low == 0.99:
        assert clipped == 0 and aux.clip_counts[0].item() == 0


# ---------------------------------------------------------------- 32k vocabulary (bf16), full batch

@pytest.mark.parametrize("norm", NORMS)
def test_v32k_parity_full(norm):
    b = make_batch("v32k", "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    zl = to_np_logits(b["logits"])
    loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0)
    T = len(oi["actions"])
    # oracle in row blocks (fp64 dlogits of the whole batch would not fit in host memory at once)
    contrib = np.empty(T)
    logp = np.empty(T)
    worst = 0.0
    for r0 in range(0, T, 2048):
        r1 = min(T, r0 + 2048)
        ref = oracle.loss_rows(zl[r0:r1], oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], cfg.G,
                               norm=norm, k=cfg.k, dual_clip_c=3.0, row_begin=r0, row_end=r1, row_offset=r0)
        contrib[r0:r1] = ref.token_contrib
        logp[r0:r1] = ref.token_logp
        kinks = kink_rows(ref, oi["behave"][r0:r1], None, A64[oi["seg"].tok_traj[r0:r1]], 0.2, 0.2, 3.0)
        worst = max(worst, check_dlogits(dl_to_f64(dl[r0:r1]), ref.dlogits, True, exempt=kinks, what=f"rows {r0}"))
    total = float(np.sum(contrib))
    assert abs(loss - total) <= LOSS_RTOL * abs(total), (loss, total)
    assert np.abs(aux.token_logp.cpu().numpy() - logp).max() <= LOGP_ATOL
    assert (aux.tok_traj.cpu().numpy() == oi["seg"].tok_traj).all()
    assert aux.error_flags.item() == 0


# ---------------------------------------------------------------- 151,936 vocabulary, full size, sampled

def _sampled_parity(name, n_rows=48, n_traj_full=2, seed=0):
    b = make_batch(name, "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    T, V = b["logits"].shape
    results = {}
    for norm in NORMS:
        loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0)
        results[norm] = (loss, aux)
        rng = np.random.default_rng(seed)
        rows = np.unique(np.concatenate([[0, T - 1], rng.integers(0, T, n_rows)]))
        rows_t = torch.from_numpy(rows).cuda()
        zs = to_np_logits(b["logits"].index_select(0, rows_t))
        dls = dl_to_f64(dl.index_select(0, rows_t))
        tl = aux.token_logp.cpu().numpy()
        for q, t in enumerate(rows):
            ref = oracle.loss_rows(zs[q:q + 1], oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], cfg.G,
                                   norm=norm, k=cfg.k, dual_clip_c=3.0, row_begin=int(t), row_end=int(t) + 1,
                                   row_offset=int(t))
            assert abs(tl[t] - ref.token_logp[0]) <= LOGP_ATOL
            kinks = kink_rows(ref, oi["behave"][t:t + 1], None, A64[oi["seg"].tok_traj[t:t + 1]], 0.2, 0.2, 3.0)
            check_dlogits(dls[q:q + 1], ref.dlogits, True, exempt=kinks, what=f"row {t}")
        # whole trajectories: the oracle's per-trajectory loss against the GPU's
        traj_loss = aux.traj_loss.cpu().numpy()
        assert abs(loss - traj_loss.sum()) <= 1e-12 * np.abs(traj_loss).sum()
        tto = oi["seg"].traj_tok_off
        for i in np.random.default_rng(seed + 1).choice(len(tto) - 1, n_traj_full, replace=False):
            t0, t1 = int(tto[i]), int(tto[i + 1])
            zt = to_np_logits(b["logits"][t0:t1])
            ref = oracle.loss_rows(zt, oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], cfg.G,
                                   norm=norm, k=cfg.k, dual_clip_c=3.0, row_begin=t0, row_end=t1, row_offset=t0,
                                   want_dlogits=False)
            assert abs(traj_loss[i] - ref.traj_loss[i]) <= LOSS_RTOL * abs(ref.traj_loss[i]), (i, traj_loss[i])
        # integers, bit-exact at full size
        assert (aux.tok_traj.cpu().numpy() == oi["seg"].tok_traj).all()
        assert (aux.traj_tok_off.cpu().numpy() == oi["seg"].traj_tok_off).all()
        assert (aux.gather_idx.cpu().numpy() == oracle.gather_index(T, V, oi["actions"])).all()
        assert aux.error_flags.item() == 0
        del dl
        torch.cuda.empty_cache()
    return results


def test_v152k_full_size_sampled():
    _sampled_parity("v152k")


def test_long_full_size_sampled():
    _sampled_parity("long", n_rows=32, n_traj_full=1)


# ---------------------------------------------------------------- advantages

def test_advantages_parity():
    rng = np.random.default_rng(0)
    r = (rng.random(256) < 0.35).astype(np.float32)
    r[8:16] = 1.0  # a zero-variance group
    for ddof in (0, 1):
        for eps in (0.0, 1e-6):
            gpu = grpo.grpo_advantages(torch.from_numpy(r).cuda(), 8, ddof=ddof, std_eps=eps).cpu().numpy()
            ref = oracle.advantages(r, 8, ddof, eps)
            np.testing.assert_allclose(gpu, ref, rtol=1e-6, atol=1e-7)
    assert (gpu[8:16] == 0).all()


# ---------------------------------------------------------------- edge cases

def _edge_batch(V, dtype="bf16", n_groups=2, G=4, ld=None, seed=5):
    from synth.rollouts import Structure, add_noise, engine_logp, make_logits
    rng = np.random.default_rng(seed)
    N = n_groups * G
    steps = rng.integers(1, 4, N)
    toks = rng.integers(0, 7, int(steps.sum()))  # empty steps allowed
    toks[0] = max(toks[0], 1)
    sto = np.concatenate([[0], np.cumsum(toks)]).astype(np.int32)
    tso = np.concatenate([[0], np.cumsum(steps)]).astype(np.int32)
    rewards = np.zeros(N, np.float32)
    rewards[::2] = 1
    T = int(sto[-1])
    st = Structure(rewards, steps.astype(np.int32), toks.astype(np.int32), sto, tso, T, 0)
    logits = make_logits(T, V, 2.0, dtype, "cuda", seed, ld=ld)
    actions = torch.from_numpy(rng.integers(0, V, T).astype(np.int32)).cuda()
    behave = add_noise(engine_logp(logits, actions, V), 0.1, seed)
    cfg = Config("edge", n_groups, G, V, dtype, 2.0, 0.5, (1, 3), (1, 3), 0.0, (0, 6), 0.1, 4.0, seed=seed)
    return dict(cfg=cfg, structure=st, logits=logits, actions=actions, behave=behave, prox=None,
                rewards=torch.from_numpy(rewards).cuda(), V=V)


@pytest.mark.parametrize("V,dtype", [(7, "bf16"), (7, "f32"), (1000, "bf16"), (4093, "f32"), (33, "bf16"),
                                     (122880, "bf16"), (128256, "bf16"), (151936, "bf16"), (163840, "bf16"),
                                     (184320, "bf16"), (200000, "bf16"), (262144, "bf16"), (77824, "f32"),
                                     (100000, "f32"), (151936, "f32")])
def test_ragged_vocab_and_kernel_variants(V, dtype):
    # odd V uses the generic row kernel; bf16 rows of 56K to 188K take the pipelined kernel (122,880: one LDS
    # vector per thread; 128,256: two; 151,936: five; 163,840 and 184,320: nine); fp32 rows up to 77,824 the
    # register-resident one; longer vector rows (bf16 200,000 and 262,144, fp32 100,000 and 151,936) the two
    # passes (a record per row, then the epilogue and dlogits)
    b = _edge_batch(V, dtype)
    _full_parity(b, oracle.NORM_TRAJ_STEPS, 3.0)


def test_padded_row_stride():
    b = _edge_batch(1000, "bf16", ld=1024)
    _full_parity(b, oracle.NORM_CONST_K, 0.0)
    b = _edge_batch(1000, "f32", ld=1003)  # odd stride: generic kernel
    _full_parity(b, oracle.NORM_CONST_K, 0.0)


def test_empty_batch():
    # T = 0: every trajectory holds steps with no action token; the loss is 0
    N = 4
    sto = torch.zeros(5, dtype=torch.int32, device="cuda")
    tso = torch.arange(0, 5, dtype=torch.int32, device="cuda")
    logits = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    a = grpo.LossAux.alloc(0, N, "cuda")
    loss, dl = grpo.grpo_loss_fwd_bwd(logits, torch.empty(0, dtype=torch.int32, device="cuda"),
                                      torch.empty(0, device="cuda"), torch.zeros(N, device="cuda"), sto, tso, 4,
                                      aux=a)
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and dl.shape == (0, 64)
    assert a.error_flags.item() == 0 and (a.traj_loss.cpu() == 0).all()


def test_invalid_action_flagged_row_zero():
    b = _edge_batch(512, "bf16")
    b["actions"][3] = 512
    b["actions"][7] = -5
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    ref = oracle.loss_rows(to_np_logits(b["logits"]), oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], 4,
                           norm=oracle.NORM_CONST_K, k=4.0)
    loss, dl, aux = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0)
    assert aux.error_flags.item() == ref.flags == grpo.GRPO_FLAG_ACTION
    assert (dl[3] == 0).all() and (dl[7] == 0).all()
    assert abs(loss - ref.loss) <= LOSS_RTOL * abs(ref.loss)


def test_malformed_offsets_flagged():
    b = _edge_batch(256, "bf16")
    st = b["structure"]
    st.step_tok_off = st.step_tok_off.copy()
    st.step_tok_off[-1] += 1  # no longer ends at T
    _, A32 = _adv(b)
    loss, dl, aux = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0)
    assert aux.error_flags.item() & grpo.GRPO_FLAG_OFFSETS
    assert math.isnan(loss) and (dl == 0).all()
    assert (aux.traj_tok_off.cpu() == -1).all()


@pytest.mark.parametrize("V,dtype", [(256, "bf16"), (200000, "bf16")])  # one pass; two passes
def test_nonfinite_logit_flagged(V, dtype):
    b = _edge_batch(V, dtype)
    b["logits"][2, 5] = float("nan")
    _, A32 = _adv(b)
    loss, dl, aux = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0)
    assert aux.error_flags.item() & grpo.GRPO_FLAG_NONFINITE
    assert math.isnan(loss) and math.isnan(aux.token_logp[2].item())


@pytest.mark.parametrize("V,dtype", [(4096, "bf16"), (100000, "f32")])  # one pass; two passes
def test_forward_only_and_aliasing(V, dtype):
    b = _edge_batch(V, dtype)
    _, A32 = _adv(b)
    l0, dl0, a0 = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0, c=3.0)
    l1, dl1, a1 = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0, c=3.0, dlogits=None)
    assert dl1 is None and l1 == l0 and torch.equal(a0.token_logp, a1.token_logp)
    inplace = b["logits"].clone()
    l2, dl2, _ = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0, c=3.0, dlogits=inplace, logits=inplace)
    assert l2 == l0 and torch.equal(dl2, dl0)


def test_bitwise_deterministic():
    b = make_batch("v32k", "cuda")
    _, A32 = _adv(b)
    l0, d0, a0 = run_gpu(b, A32, norm=grpo.GRPO_NORM_TRAJ_STEPS, k=8.0, c=3.0)
    l1, d1, a1 = run_gpu(b, A32, norm=grpo.GRPO_NORM_TRAJ_STEPS, k=8.0, c=3.0)
    assert l0 == l1 and torch.equal(d0, d1) and torch.equal(a0.traj_loss, a1.traj_loss)


def test_n_groups_total_for_shards():
    b = make_batch("tiny", "cuda")
    _, A32 = _adv(b)
    l1, _, _ = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=3.0)
    l2, _, _ = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=3.0, n_groups_total=4.0)
    assert abs(l2 - l1 / 4.0) <= 1e-12 * abs(l1)

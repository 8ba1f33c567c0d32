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


# ---------------------------------------------------------------- whole-batch oracle in row blocks

def _oracle_all_rows(b, oi, norms, c=3.0, block=8192):
    """The oracle's per-token outputs for every row of a batch too large for host memory at once, one normaliser
    after the other: row blocks are copied to the host (the next one while the oracle works on the current one),
    the first normaliser takes the log-softmax from the logits (loss_rows) and the others reuse its log-probs
    (loss_from_logp).  Returns {norm: LossResult over all rows, without dlogits}."""
    from concurrent.futures import ThreadPoolExecutor
    cfg = b["cfg"]
    T, V = len(oi["actions"]), b["V"]
    parts = {n: [] for n in norms}
    fetch = lambda r0: to_np_logits(b["logits"][r0:min(T, r0 + block)])  # noqa: E731
    with ThreadPoolExecutor(1) as ex:
        nxt = ex.submit(fetch, 0) if T > 0 else None
        for r0 in range(0, T, block):
            r1 = min(T, r0 + block)
            zl = nxt.result()
            if r1 < T:
                nxt = ex.submit(fetch, r1)
            kw = dict(k=cfg.k, dual_clip_c=c, row_begin=r0, row_end=r1)
            first = oracle.loss_rows(zl, oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"], cfg.G, V=V,
                                     norm=norms[0], want_dlogits=False, row_offset=r0, **kw)
            parts[norms[0]].append(first)
            for n in norms[1:]:
                parts[n].append(oracle.loss_from_logp(first.token_logp, oi["actions"], oi["behave"], oi["prox"],
                                                      oi["adv"], oi["seg"], cfg.G, V=V, norm=n, **kw))
            if (r0 // block) % 8 == 7:
                print(f"  oracle rows {r1} of {T}", flush=True)
    out = {}
    n_traj = len(oi["seg"].traj_steps)
    for n, ps in parts.items():
        cat = lambda f, dt=np.float64: np.concatenate([getattr(q, f) for q in ps]) if ps else np.zeros(0, dt)  # noqa: E731
        contrib = cat("token_contrib")
        traj = np.bincount(oi["seg"].tok_traj, weights=contrib, minlength=n_traj) if T else np.zeros(n_traj)
        out[n] = oracle.LossResult(math.fsum(contrib), traj, cat("token_logp"), contrib, cat("token_g"),
                                   cat("token_state", np.int32), None, int(np.bitwise_or.reduce([q.flags for q in ps]))
                                   if ps else 0)
    return out


def _whole_batch_checks(ref, loss, aux, oi, A64, V, ld, what):
    """Every per-token and per-trajectory output and the whole loss against the oracle over all rows."""
    T = len(oi["actions"])
    kappa = ref.kappa
    print(f"{what}: loss {loss!r} oracle {ref.loss!r} rel {abs(loss - ref.loss) / abs(ref.loss):.2e} "
          f"kappa {kappa:.1f}", flush=True)
    assert abs(loss - ref.loss) <= LOSS_RTOL * abs(ref.loss), (what, loss, ref.loss, kappa)
    np.testing.assert_allclose(aux.traj_loss.cpu().numpy(), ref.traj_loss, rtol=LOSS_RTOL,
                               atol=LOSS_RTOL * np.abs(ref.traj_loss).max(), err_msg=what)
    assert np.abs(aux.token_logp.cpu().numpy() - ref.token_logp).max() <= LOGP_ATOL, what
    kinks = kink_rows(ref, oi["behave"], oi["prox"], A64[oi["seg"].tok_traj], 0.2, 0.2, 3.0)
    assert len(kinks) <= max(2, T // 1000), f"unexpectedly many kink rows: {len(kinks)}"
    clip = aux.clip_counts.cpu().numpy()
    assert abs(clip[0] - (ref.token_state & 1).sum()) <= len(kinks), what
    assert abs(clip[1] - ((ref.token_state >> 1) & 1).sum()) <= len(kinks), what
    valid = oracle.valid_tokens(oi["actions"], V, oi["seg"])
    want = oracle.ratio_stats(ref.token_logp, oi["behave"], oi["prox"], valid)
    got = aux.ratio_stats.cpu().numpy()
    np.testing.assert_allclose(got[:6], want[:6], rtol=1e-5, err_msg=what)
    assert abs(got[6] - want[6]) <= len(kinks) + 2 and got[7] == want[7], (what, got[6:], want[6:])
    assert (aux.tok_traj.cpu().numpy() == oi["seg"].tok_traj).all()
    assert (aux.traj_tok_off.cpu().numpy() == oi["seg"].traj_tok_off).all()
    assert (aux.gather_idx.cpu().numpy() == oracle.gather_index(T, ld, oi["actions"])).all()
    assert aux.error_flags.item() == ref.flags == 0
    return kinks


def _pipeline_rows(T, grid, rng, n_random, chunk=8):
    """Rows to compare element by element: the first and last rows, rows on each side of the persistent row kernel's
    chunk and round boundaries (every row but a workgroup's first had its LDS part and registers loaded during the
    previous row's dlogits pass; a chunk's first row follows the previous chunk's last, grid * chunk rows earlier),
    the boundaries of the last rows' even split (the rows after the whole rounds, r0 on, go chunk2 to a workgroup),
    and random rows."""
    r0 = T // (chunk * grid) * (chunk * grid)
    c2 = max(1, -(-(T - r0) // grid))
    fixed = [0, 1, chunk - 1, chunk, chunk + 1, grid - 1, grid, grid + 1, grid * chunk - 1, grid * chunk,
             grid * chunk + 1, 2 * grid * chunk + 17, 3 * grid + 17, 7 * grid + 100, T // 2, T - grid - 1, T - grid,
             T - chunk - 1, T - 2, T - 1, r0 - 1, r0, r0 + 1, r0 + c2 - 1, r0 + c2, r0 + 7 * c2 - 1, r0 + 7 * c2]
    rows = np.concatenate([fixed, rng.integers(0, T, n_random)])
    return np.unique(rows[(rows >= 0) & (rows < T)])


def _sampled_dlogits(b, dl, rows, oi, A64, norm, gs, scaled, what):
    """dlogits of the sampled rows against the oracle's, row by row (grad_scale gs on both sides)."""
    cfg = b["cfg"]
    rows_t = torch.from_numpy(rows).to(dl.device)
    zs = to_np_logits(b["logits"].index_select(0, rows_t))
    dls = dl_to_f64(dl.index_select(0, rows_t)[:, :b["V"]])
    worst = 0.0
    for q, t in enumerate(rows):
        ref = oracle.loss_rows(zs[q:q + 1], oi["actions"], oi["behave"], oi["prox"], oi["adv"], oi["seg"], cfg.G,
                               V=b["V"], norm=norm, k=cfg.k, dual_clip_c=3.0, grad_scale=gs, row_begin=int(t),
                               row_end=int(t) + 1, row_offset=int(t))
        kinks = kink_rows(ref, oi["behave"][t:t + 1], None if oi["prox"] is None else oi["prox"][t:t + 1],
                          A64[oi["seg"].tok_traj[t:t + 1]], 0.2, 0.2, 3.0)
        worst = max(worst, check_dlogits(dls[q:q + 1], ref.dlogits, True, exempt=kinks, scaled=scaled,
                                         what=f"{what} row {t}"))
    return worst


# ---------------------------------------------------------------- 32k vocabulary (bf16), full batch

@pytest.mark.parametrize("norm", NORMS)
def test_v32k_parity_full(norm):
    # the register-resident kernel (256 threads x 16 vectors per row); every row's dlogits against the oracle's,
    # at grad_scale 1 (absolute 2e-3) and rerun at grad_scale = 1/max|g_t| (the scaled bf16 gate)
    b = make_batch("v32k", "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    T, V = b["logits"].shape
    ref = _oracle_all_rows(b, oi, [norm])[norm]
    loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0)
    _whole_batch_checks(ref, loss, aux, oi, A64, V, V, f"v32k norm {norm}")
    gs = float(np.float32(1.0 / np.abs(ref.token_g).max()))
    loss2, dl2, _ = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0, grad_scale=gs, aux=False)
    assert loss2 == loss
    zl = to_np_logits(b["logits"])
    worst = 0.0
    for r0 in range(0, T, 2048):
        r1 = min(T, r0 + 2048)
        blk = oracle.loss_rows(zl[r0:r1], oi["actions"], oi["behave"], None, oi["adv"], oi["seg"], cfg.G, norm=norm,
                               k=cfg.k, dual_clip_c=3.0, row_begin=r0, row_end=r1, row_offset=r0)
        kinks = kink_rows(blk, oi["behave"][r0:r1], None, A64[oi["seg"].tok_traj[r0:r1]], 0.2, 0.2, 3.0)
        check_dlogits(dl_to_f64(dl[r0:r1]), blk.dlogits, True, exempt=kinks, what=f"rows {r0}")
        worst = max(worst, check_dlogits(dl_to_f64(dl2[r0:r1]), blk.dlogits * gs, True, exempt=kinks, scaled=True,
                                         what=f"scaled rows {r0}"))
    print(f"v32k norm {norm}: worst scaled dlogits error {worst:.3f} of the gate", flush=True)


# ---------------------------------------------------------------- 151,936 vocabulary, full size

def _full_size_parity(name, norms, n_rows=48, seed=0):
    """The whole batch in the benchmark's launch configuration.  Every row's log-prob, every trajectory's loss,
    the clip counts, the ratio statistics and the whole loss against the oracle over all rows; dlogits of sampled
    rows (including rows each workgroup of the persistent kernel handles after its first) at grad_scale 1 and,
    rerun at grad_scale = 1/max|g_t|, under the scaled bf16 gate."""
    b = make_batch(name, "cuda")
    cfg = b["cfg"]
    A64, A32 = _adv(b)
    oi = oracle_inputs(b, A64)
    T, V = b["logits"].shape
    refs = _oracle_all_rows(b, oi, norms)
    grid = min(T, torch.cuda.get_device_properties(0).multi_processor_count)
    rows = _pipeline_rows(T, grid, np.random.default_rng(seed), n_rows)
    assert (rows >= grid).sum() >= n_rows // 2
    out = {}
    for norm in norms:
        ref = refs[norm]
        loss, dl, aux = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0)
        _whole_batch_checks(ref, loss, aux, oi, A64, V, V, f"{name} norm {norm}")
        _sampled_dlogits(b, dl, rows, oi, A64, norm, 1.0, False, f"{name} norm {norm}")
        del dl
        torch.cuda.empty_cache()
        gs = float(np.float32(1.0 / np.abs(ref.token_g).max()))
        loss2, dl2, _ = run_gpu(b, A32, norm=gpu_norm(norm), k=cfg.k, c=3.0, grad_scale=gs, aux=False)
        assert loss2 == loss  # grad_scale does not touch the loss
        worst = _sampled_dlogits(b, dl2, rows, oi, A64, norm, gs, True, f"{name} norm {norm} scaled")
        print(f"{name} norm {norm}: worst scaled dlogits error {worst:.3f} of the gate over {len(rows)} rows",
              flush=True)
        del dl2
        torch.cuda.empty_cache()
        out[norm] = (loss, ref)
    return out


def test_v152k_full_size():
    _full_size_parity("v152k", NORMS)


def test_long_full_size():
    _full_size_parity("long", NORMS, n_rows=32)


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

def _edge_batch(V, dtype="bf16", n_groups=2, G=4, ld=None, seed=5, max_tok=6):
    from synth.rollouts import Structure, add_noise, engine_logp, make_logits
    rng = np.random.default_rng(seed)
    N = n_groups * G
    steps = rng.integers(1, 4, N)
    toks = rng.integers(0, max_tok + 1, int(steps.sum()))  # empty steps allowed
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
    # vector per thread; 128,256: two; 151,936: six; 163,840 and 184,320: nine); fp32 rows up to 77,824 the
    # register-resident one; longer vector rows (bf16 200,000 and 262,144, fp32 100,000 and 151,936) the two
    # passes (a record per row, then the epilogue and dlogits)
    b = _edge_batch(V, dtype)
    _full_parity(b, oracle.NORM_TRAJ_STEPS, 3.0)


@pytest.mark.parametrize("V", [122880, 151936, 184320])
def test_pipelined_kernel_several_rows_per_workgroup(V):
    # T well above twice the CU count: each workgroup of the persistent kernel streams two or more rows (the next
    # row's LDS part staged and its register part reloaded during the current row's dlogits pass), every row under
    # the scaled bf16 gate
    b = _edge_batch(V, "bf16", n_groups=4, G=4, seed=V % 97, max_tok=48)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert b["structure"].T > 2 * n_cu + 64, b["structure"].T
    _full_parity(b, oracle.NORM_TRAJ_STEPS, 3.0)


@pytest.mark.parametrize("V", [122880, 151936])
def test_pipelined_kernel_row_chunks(V):
    # T above 8 x the CU count: rows go to workgroups in chunks of two consecutive rows (a workgroup's next row is
    # either the row after the current one or the first of its next chunk, 2 x grid rows on), the rows after the
    # whole rounds split evenly, one chunk per workgroup; every row under the scaled bf16 gate
    b = _edge_batch(V, "bf16", n_groups=8, G=4, seed=V % 97 + 1, max_tok=72)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert b["structure"].T >= 8 * n_cu, b["structure"].T
    _full_parity(b, oracle.NORM_CONST_K, 3.0)


def test_padded_row_stride():
    b = _edge_batch(1000, "bf16", ld=1024)
    _full_parity(b, oracle.NORM_CONST_K, 0.0)
    b = _edge_batch(1000, "f32", ld=1003)  # odd stride: generic kernel
    _full_parity(b, oracle.NORM_CONST_K, 0.0)


@pytest.mark.parametrize("V,ld", [(151936, 152064), (122880, 122888)])
def test_padded_row_stride_pipelined(V, ld):
    # the pipelined kernel on rows whose stride exceeds V (several rows per workgroup): every row under the scaled
    # bf16 gate, and the padding columns of a caller's dlogits buffer are left as they were
    b = _edge_batch(V, "bf16", ld=ld, n_groups=8, G=4, seed=V % 89 + 2, max_tok=40)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert b["structure"].T >= 2 * n_cu, b["structure"].T
    _full_parity(b, oracle.NORM_CONST_K, 3.0)
    _, A32 = _adv(b)
    dl = torch.full_like(b["logits"], 7.0)
    run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=b["cfg"].k, c=3.0, dlogits=dl, aux=False)
    assert (dl[:, V:] == 7.0).all()


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


@pytest.mark.parametrize("V,dtype", [(256, "bf16"), (32000, "bf16"), (151936, "bf16"), (200000, "bf16")])
def test_nonfinite_logit_flagged(V, dtype):
    # resident kernels (one workgroup per row), the pipelined kernel, two passes
    b = _edge_batch(V, dtype)
    b["logits"][2, 5] = float("nan")
    _, A32 = _adv(b)
    loss, dl, aux = run_gpu(b, A32, norm=grpo.GRPO_NORM_CONST_K, k=4.0)
    assert aux.error_flags.item() & grpo.GRPO_FLAG_NONFINITE
    assert math.isnan(loss) and math.isnan(aux.token_logp[2].item())


@pytest.mark.parametrize("V,dtype", [(256, "bf16"), (1024, "f32"), (32000, "bf16"), (151936, "bf16"),
                                     (200000, "bf16")])
def test_masked_logits(V, dtype):
    # -inf logits (a masked vocabulary) are valid input: they carry zero probability, the row's log-sum-exp
    # stays finite, nothing is flagged, and their dlogits are zero.  About a tenth of the columns of every
    # row, both bf16 halves of a dword, never the action's.
    from synth.rollouts import add_noise, engine_logp
    b = _edge_batch(V, dtype, seed=11)
    T = b["logits"].shape[0]
    g = torch.Generator("cuda").manual_seed(V)
    mask = torch.rand((T, V), generator=g, device="cuda") < 0.1
    mask[torch.arange(T, device="cuda"), b["actions"].long()] = False
    b["logits"][:, :V].masked_fill_(mask, float("-inf"))
    b["behave"] = add_noise(engine_logp(b["logits"], b["actions"], V), 0.1, 11)
    ref, loss, dl, aux = _full_parity(b, oracle.NORM_CONST_K, 0.0)
    assert aux.error_flags.item() == 0 and math.isfinite(loss)
    assert (dl[:, :V][mask] == 0).all()


@pytest.mark.parametrize("V,dtype,big", [(4096, "bf16", False), (100000, "f32", False), (151936, "bf16", True)])
def test_forward_only_and_aliasing(V, dtype, big):
    # one pass (resident), two passes, and the pipelined kernel with several rows per workgroup (each row's
    # dlogits overwrite it in place while the workgroup's next row is being loaded)
    b = _edge_batch(V, dtype, n_groups=8, G=4, seed=13, max_tok=72) if big else _edge_batch(V, dtype)
    if big:
        assert b["structure"].T >= 4 * torch.cuda.get_device_properties(0).multi_processor_count
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

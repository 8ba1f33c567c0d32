"""Pins the fp64 oracle to facts other than itself (CPU only).

Each test ties the oracle to something the paper or mathematics fixes:
hand-derived per-token values (tests/golden), the paper's normaliser numbers
(Sec. 1, Sec. 3.2), closed forms for the group advantage (Sec. 3.2), textbook
special cases (softmax of a constant row, clipped PPO when pi_prox = pi_behave),
brute-force log-sum-exp, central finite differences of the loss, and an
independent torch fp64 autograd of the literal Eq. 1 / Eq. 2 expression.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers

def one_traj_segments(T):
    """One trajectory, one step per token."""
    return oracle.segments(T, np.arange(T + 1), np.array([0, T]))


def ragged_batch(rng, n_groups=2, G=4, V=64, max_steps=4, max_tok=5, sigma=1.5):
    N = n_groups * G
    steps = rng.integers(1, max_steps + 1, N)
    toks = rng.integers(1, max_tok + 1, int(steps.sum()))
    sto = np.concatenate([[0], np.cumsum(toks)]).astype(np.int32)
    tso = np.concatenate([[0], np.cumsum(steps)]).astype(np.int32)
    T = int(sto[-1])
    z = rng.normal(0, sigma, (T, V))
    a = rng.integers(0, V, T).astype(np.int32)
    rewards = np.zeros(N, np.float32)
    for g in range(n_groups):  # mixed groups
        r = rng.random(G) < 0.5
        r[0], r[1] = True, False
        rewards[g * G:(g + 1) * G] = r
    seg = oracle.segments(T, sto, tso)
    return dict(T=T, V=V, N=N, G=G, z=z, a=a, sto=sto, tso=tso, rewards=rewards, seg=seg)


def exact_logp(z, a):
    m = z.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    return z[np.arange(len(a)), a] - lse


def torch_literal_loss(z, a, b, p, A_tok, w_tok, eps_lo, eps_hi, c):
    """Eq. 1 with the dual clip of Eq. 2, written with torch fp64 ops; returns (loss, dloss/dz)."""
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    logp = torch.log_softmax(zt, dim=1).gather(1, torch.tensor(a, dtype=torch.int64)[:, None])[:, 0]
    b = torch.tensor(b, dtype=torch.float64)
    p = torch.tensor(p, dtype=torch.float64)
    A = torch.tensor(A_tok, dtype=torch.float64)
    w = torch.tensor(w_tok, dtype=torch.float64)
    rho = torch.exp(logp - b)
    omega = torch.exp(p - b)
    r = torch.exp(logp - p)
    s = torch.minimum(rho * A, omega * torch.clamp(r, 1 - eps_lo, 1 + eps_hi) * A)
    if c > 0:
        s = torch.where(A < 0, torch.maximum(s, c * A), s)
    loss = -(w * s).sum()
    loss.backward()
    return loss.item(), zt.grad.numpy()


def weights(seg, G, norm, k, n_groups=None):
    N = len(seg.traj_steps)
    ng = N / G if n_groups is None else n_groups
    den = np.full(N, k, np.float64) if norm == oracle.NORM_CONST_K else seg.traj_steps.astype(np.float64)
    return 1.0 / (ng * G * den)


# ---------------------------------------------------------------- segments

def test_segments_hand_case():
    # 2 trajectories: steps {3 tok, 0 tok, 2 tok} and {4 tok}
    sto = [0, 3, 3, 5, 9]
    tso = [0, 3, 4]
    s = oracle.segments(9, sto, tso)
    assert s.flags == 0
    assert s.traj_tok_off.tolist() == [0, 5, 9]
    assert s.traj_steps.tolist() == [3, 1]
    assert s.tok_traj.tolist() == [0, 0, 0, 0, 0, 1, 1, 1, 1]


@pytest.mark.parametrize("sto,tso,T", [
    ([1, 3, 5], [0, 2], 5),        # does not start at 0
    ([0, 3, 2], [0, 2], 2),        # decreasing token offsets
    ([0, 3, 5], [0, 2], 6),        # does not end at T
    ([0, 3, 5], [0, 0, 2], 5),     # a trajectory with no step
    ([0, 3, 5], [0, 1], 5),        # steps do not end at n_steps
])
def test_segments_rejects_malformed(sto, tso, T):
    s = oracle.segments(T, sto, tso)
    assert s.flags == oracle.ERR_OFFSETS
    assert (s.tok_traj == -1).all()


def test_segments_matches_repeat(rng=np.random.default_rng(7)):
    b = ragged_batch(rng, n_groups=3, G=5)
    per_traj = np.diff(b["sto"][b["tso"]])
    assert (b["seg"].tok_traj == np.repeat(np.arange(b["N"]), per_traj)).all()
    assert (b["seg"].traj_steps == np.diff(b["tso"])).all()


# ---------------------------------------------------------------- advantages

@pytest.mark.parametrize("G", [2, 4, 8])
@pytest.mark.parametrize("ddof", [0, 1])
def test_advantage_closed_form(G, ddof):
    # m successes among G binary rewards: mean m/G, var m(G-m)/(G(G-ddof))
    for m in range(1, G):
        r = np.array([1.0] * m + [0.0] * (G - m), np.float32)
        A = oracle.advantages(r, G, ddof)
        sd = math.sqrt(m * (G - m) / (G * (G - ddof)))
        np.testing.assert_allclose(A[:m], (1 - m / G) / sd, rtol=1e-14)
        np.testing.assert_allclose(A[m:], (-m / G) / sd, rtol=1e-14)
        assert abs(A.sum()) < 1e-12                        # sum_i A_i = 0
        np.testing.assert_allclose((A ** 2).sum(), G - ddof, rtol=1e-13)  # sum A^2 = G - ddof


def test_advantage_matches_numpy_std():
    rng = np.random.default_rng(3)
    r = rng.normal(size=24).astype(np.float32)
    A = oracle.advantages(r, 8, 1, std_eps=1e-3)
    for g in range(3):
        x = r[g * 8:(g + 1) * 8].astype(np.float64)
        np.testing.assert_allclose(A[g * 8:(g + 1) * 8], (x - x.mean()) / (np.std(x, ddof=1) + 1e-3), rtol=1e-13)


def test_advantage_zero_variance_group():
    A = oracle.advantages(np.array([1, 1, 1, 1, 0, 1, 0, 0], np.float32), 4, 1)
    assert (A[:4] == 0).all() and np.isfinite(A).all()


# ---------------------------------------------------------------- log-softmax

def test_constant_row_logp_is_minus_log_v():
    # softmax of a constant row is uniform: l = -log V, every p_v = 1/V
    for V in (1, 7, 1024, 151936):
        z = np.full((1, V), 3.25, np.float32)
        seg = one_traj_segments(1)
        r = oracle.loss_rows(z, [V - 1], [0.0], None, [1.0], seg, 1, norm=oracle.NORM_CONST_K, k=1.0,
                             want_dlogits=V <= 1024)
        assert abs(r.token_logp[0] + math.log(V)) < 1e-12
        if V <= 1024:  # dlogits = g*(1/V - onehot), g = w * rho * A
            g = r.token_g[0]
            np.testing.assert_allclose(r.dlogits[0, :-1], g / V, rtol=1e-12)
            np.testing.assert_allclose(r.dlogits[0, -1], g * (1 / V - 1), rtol=1e-12)


def test_logp_brute_force_fsum():
    rng = np.random.default_rng(11)
    T, V = 12, 40
    z = rng.normal(0, 3, (T, V)).astype(np.float32)
    a = rng.integers(0, V, T)
    seg = one_traj_segments(T)
    r = oracle.loss_rows(z, a, np.zeros(T), None, [0.5], seg, 1, want_dlogits=False)
    for t in range(T):
        lse = math.log(math.fsum(math.exp(float(x)) for x in z[t]))
        assert abs(r.token_logp[t] - (float(z[t, a[t]]) - lse)) < 1e-13


def test_bf16_input_widening():
    # bf16 bit patterns are the upper half of the float32 with the same value
    vals = np.array([[1.0, -2.5, 0.15625, 3.0e-3]], np.float32)
    bits = (vals.view(np.uint32) >> 16).astype(np.uint16)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    seg = one_traj_segments(1)
    r32 = oracle.loss_rows(back, [1], [0.0], None, [1.0], seg, 1)
    r16 = oracle.loss_rows(bits, [1], [0.0], None, [1.0], seg, 1)
    assert r32.token_logp[0] == r16.token_logp[0]
    assert (r32.dlogits == r16.dlogits).all()


def test_logp_matches_torch_log_softmax():
    rng = np.random.default_rng(5)
    z = rng.normal(0, 2, (30, 300))
    a = rng.integers(0, 300, 30)
    seg = one_traj_segments(30)
    r = oracle.loss_rows(z, a, np.zeros(30), None, [1.0], seg, 1, want_dlogits=False)
    ref = torch.log_softmax(torch.tensor(z), 1)[torch.arange(30), torch.tensor(a)].numpy()
    np.testing.assert_allclose(r.token_logp, ref, rtol=0, atol=1e-13)


# ---------------------------------------------------------------- surrogate: golden cases

def load_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_surrogate_golden_cases():
    cases = [[float(x) for x in r] for r in load_table("surrogate_cases.txt")]
    V = 4
    lval = -math.log(V)  # constant row of zeros
    for rho, omega, A, c, s_ref, d_ref, st_ref in cases:
        r_ratio = rho / omega
        b = np.float32(lval - math.log(rho))
        p = np.float32(lval - math.log(r_ratio))
        seg = one_traj_segments(1)
        res = oracle.loss_rows(np.zeros((1, V), np.float32), [0], [b], [p], [A], seg, 1,
                               norm=oracle.NORM_CONST_K, k=1.0, eps_low=0.2, eps_high=0.2, dual_clip_c=c)
        # w = 1 (one group of one trajectory, k = 1): contribution = -s, g = ds/dl
        assert abs(-res.token_contrib[0] - s_ref) < 2e-6, (rho, omega, A, c)
        assert abs(res.token_g[0] - d_ref) < 2e-6, (rho, omega, A, c)
        assert res.token_state[0] == int(st_ref), (rho, omega, A, c)


def test_coupled_reduces_to_textbook_ppo():
    # pi_prox = pi_behave: s = min(rho*A, clip(rho, 1-eps, 1+eps)*A) (clipped PPO)
    rng = np.random.default_rng(2)
    T, V = 64, 32
    z = rng.normal(0, 1, (T, V))
    a = rng.integers(0, V, T)
    l = exact_logp(z, a)
    b = (l + rng.normal(0, 0.4, T)).astype(np.float32)
    A = rng.normal(0, 1, T)
    sto = np.arange(T + 1)
    seg = oracle.segments(T, sto, sto)  # T trajectories of one token each
    res = oracle.loss_rows(z, a, b, None, A, seg, 1, norm=oracle.NORM_CONST_K, k=1.0, n_groups_total=1.0)
    rho = np.exp(l - b.astype(np.float64))
    ppo = np.minimum(rho * A, np.clip(rho, 0.8, 1.2) * A)
    np.testing.assert_allclose(-res.token_contrib, ppo, rtol=1e-12, atol=1e-14)


def test_decoupled_identity():
    # min(rho A, omega clip(r) A) = omega * min(r A, clip(r) A), since rho = omega r
    rng = np.random.default_rng(9)
    T, V = 80, 16
    z = rng.normal(0, 1, (T, V))
    a = rng.integers(0, V, T)
    l = exact_logp(z, a)
    b = (l + rng.normal(0, 0.3, T)).astype(np.float32)
    p = (l + rng.normal(0, 0.3, T)).astype(np.float32)
    A = rng.normal(0, 1, T)
    sto = np.arange(T + 1)
    seg = oracle.segments(T, sto, sto)
    res = oracle.loss_rows(z, a, b, p, A, seg, 1, norm=oracle.NORM_CONST_K, k=1.0, n_groups_total=1.0)
    r = np.exp(l - p.astype(np.float64))
    om = np.exp(p.astype(np.float64) - b.astype(np.float64))
    np.testing.assert_allclose(-res.token_contrib, om * np.minimum(r * A, np.clip(r, 0.8, 1.2) * A),
                               rtol=1e-12, atol=1e-14)


def test_dual_clip_bounds_and_inertness():
    rng = np.random.default_rng(4)
    T, V = 200, 8
    z = rng.normal(0, 1, (T, V))
    a = rng.integers(0, V, T)
    l = exact_logp(z, a)
    b = (l - rng.uniform(-0.5, 3.0, T)).astype(np.float32)  # ratios up to e^3
    A = rng.normal(0, 1, T)
    sto = np.arange(T + 1)
    seg = oracle.segments(T, sto, sto)
    kw = dict(norm=oracle.NORM_CONST_K, k=1.0, n_groups_total=1.0)
    on = oracle.loss_rows(z, a, b, None, A, seg, 1, dual_clip_c=3.0, **kw)
    off = oracle.loss_rows(z, a, b, None, A, seg, 1, dual_clip_c=0.0, **kw)
    s_on, s_off = -on.token_contrib, -off.token_contrib
    neg = A < 0
    assert (s_on[neg] >= 3.0 * A[neg] - 1e-15).all()      # Eq. 2: floor c*A for A < 0
    assert (s_on[~neg] == s_off[~neg]).all()               # inert for A >= 0
    assert ((on.token_state & 2) > 0).sum() > 0            # the floor did engage
    assert (s_on[neg] == np.maximum(s_off[neg], 3.0 * A[neg])).all()


# ---------------------------------------------------------------- normalisers

def test_normalizer_golden_paper_numbers():
    kv = {k: float(v) for k, v in load_table("normalizer_weights.txt")}
    nf, ns, k = int(kv["steps_fail"]), int(kv["steps_succ"]), kv["k"]
    T = nf + ns
    sto = np.arange(T + 1)             # one token per step
    tso = np.array([0, nf, T])
    seg = oracle.segments(T, sto, tso)
    A = oracle.advantages(np.array([0.0, 1.0], np.float32), 2, 1)
    np.testing.assert_allclose(A, [kv["adv_fail"], kv["adv_succ"]], rtol=1e-15)
    V = 4
    z = np.zeros((T, V))
    b = np.full(T, np.float32(-math.log(V)))
    out = {}
    for norm, tag in ((oracle.NORM_TRAJ_STEPS, "traj_steps"), (oracle.NORM_CONST_K, "const_k")):
        r = oracle.loss_rows(z, np.zeros(T, np.int32), b, None, A, seg, 2, norm=norm, k=k)
        gf, gs = np.abs(r.token_g[:nf]), np.abs(r.token_g[nf:])
        assert np.ptp(gf) < 1e-15 and np.ptp(gs) < 1e-15
        np.testing.assert_allclose(gs[0] / gf[0], kv["grad_ratio_" + tag], rtol=1e-6)
        # a rollout's total step weight: sum of w_i over its (one-token) steps, times n_groups*G
        w = weights(seg, 2, norm, k)
        np.testing.assert_allclose(w[0] * nf * 2, kv["rollout_weight_fail_" + tag], rtol=1e-14)
        np.testing.assert_allclose(w[1] * ns * 2, kv["rollout_weight_succ_" + tag], rtol=1e-14)
        assert abs(r.loss - kv["loss_" + tag]) < 1e-6
        out[tag] = r
    # Sec. 3.2: per token, 1/k over 1/|tau_i| is |tau_i|/k
    np.testing.assert_allclose(out["const_k"].token_g[:nf] / out["traj_steps"].token_g[:nf], nf / k, rtol=1e-12)


def test_normalizers_coincide_when_all_lengths_equal_k():
    # the tiny workload: G = 4 trajectories of 3 steps, k = 3
    rng = np.random.default_rng(1)
    G, steps, tok, V = 4, 3, 16, 64
    T = G * steps * tok
    sto = np.arange(0, T + 1, tok)
    tso = np.arange(0, G * steps + 1, steps)
    seg = oracle.segments(T, sto, tso)
    z = rng.normal(0, 1, (T, V))
    a = rng.integers(0, V, T)
    b = (exact_logp(z, a) + rng.normal(0, 0.1, T)).astype(np.float32)
    A = oracle.advantages(np.array([1, 0, 1, 0], np.float32), G)
    r1 = oracle.loss_rows(z, a, b, None, A, seg, G, norm=oracle.NORM_TRAJ_STEPS, k=3.0, dual_clip_c=3.0)
    r2 = oracle.loss_rows(z, a, b, None, A, seg, G, norm=oracle.NORM_CONST_K, k=3.0, dual_clip_c=3.0)
    assert r1.loss == r2.loss
    assert (r1.dlogits == r2.dlogits).all()


def test_per_token_ratio_between_normalizers_is_len_over_k():
    rng = np.random.default_rng(21)
    bt = ragged_batch(rng, n_groups=3, G=4, V=32, max_steps=9)
    A = oracle.advantages(bt["rewards"], bt["G"])
    b = (exact_logp(bt["z"], bt["a"]) + rng.normal(0, 0.1, bt["T"])).astype(np.float32)
    kw = dict(k=10.0, dual_clip_c=3.0)
    r1 = oracle.loss_rows(bt["z"], bt["a"], b, None, A, bt["seg"], bt["G"], norm=oracle.NORM_TRAJ_STEPS, **kw)
    r2 = oracle.loss_rows(bt["z"], bt["a"], b, None, A, bt["seg"], bt["G"], norm=oracle.NORM_CONST_K, **kw)
    tau = bt["seg"].traj_steps[bt["seg"].tok_traj].astype(np.float64)
    nz = r1.token_g != 0
    np.testing.assert_allclose(r2.token_g[nz] / r1.token_g[nz], tau[nz] / 10.0, rtol=1e-13)
    np.testing.assert_allclose(r2.dlogits[nz] / np.where(r1.dlogits[nz] == 0, 1, r1.dlogits[nz]),
                               np.where(r1.dlogits[nz] == 0, 1, (tau[nz] / 10.0)[:, None]), rtol=1e-12)


# ---------------------------------------------------------------- invariants

def test_ratio_one_gives_advantage_closed_form():
    # b = p = l: rho = r = 1, no clip, s_t = A_i, loss = -sum_i w_i n_i A_i
    rng = np.random.default_rng(8)
    bt = ragged_batch(rng, n_groups=2, G=4, V=16)
    l = exact_logp(bt["z"], bt["a"])
    A = oracle.advantages(bt["rewards"], bt["G"])
    for norm in (oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K):
        # b = p = l rounded to float32: the ratios are 1 to within 1e-7
        r = oracle.loss_rows(bt["z"], bt["a"], l.astype(np.float32), l.astype(np.float32), A, bt["seg"], bt["G"],
                             norm=norm, k=5.0)
        w = weights(bt["seg"], bt["G"], norm, 5.0)
        n_i = np.diff(bt["seg"].traj_tok_off)
        np.testing.assert_allclose(r.loss, -(w * n_i * A).sum(), rtol=1e-6, atol=1e-7)
        np.testing.assert_allclose(-r.token_contrib / w[bt["seg"].tok_traj], A[bt["seg"].tok_traj], rtol=1e-6)


def test_dlogits_rows_sum_to_zero():
    rng = np.random.default_rng(12)
    bt = ragged_batch(rng, n_groups=2, G=4, V=128, sigma=3)
    A = oracle.advantages(bt["rewards"], bt["G"])
    b = (exact_logp(bt["z"], bt["a"]) + rng.normal(0, 0.2, bt["T"])).astype(np.float32)
    r = oracle.loss_rows(bt["z"], bt["a"], b, None, A, bt["seg"], bt["G"], dual_clip_c=3.0)
    scale = np.abs(r.dlogits).max(axis=1) + 1e-300
    assert (np.abs(r.dlogits.sum(axis=1)) / scale < 1e-13).all()


def test_eps_to_infinity_is_plain_importance_sampling():
    rng = np.random.default_rng(13)
    bt = ragged_batch(rng, n_groups=2, G=4, V=16)
    A = oracle.advantages(bt["rewards"], bt["G"])
    l = exact_logp(bt["z"], bt["a"])
    b = (l + rng.normal(0, 0.5, bt["T"])).astype(np.float32)
    r = oracle.loss_rows(bt["z"], bt["a"], b, None, A, bt["seg"], bt["G"], norm=oracle.NORM_TRAJ_STEPS,
                         eps_low=1.0, eps_high=1e30)
    w = weights(bt["seg"], bt["G"], oracle.NORM_TRAJ_STEPS, 1.0)[bt["seg"].tok_traj]
    rho = np.exp(l - b.astype(np.float64))
    np.testing.assert_allclose(r.token_g, w * rho * A[bt["seg"].tok_traj], rtol=1e-12)


def test_invalid_action_row_is_zero_and_flagged():
    rng = np.random.default_rng(14)
    bt = ragged_batch(rng, V=16)
    A = oracle.advantages(bt["rewards"], bt["G"])
    a = bt["a"].copy()
    a[3] = 16
    a[5] = -1
    r = oracle.loss_rows(bt["z"], a, np.zeros(bt["T"]), None, A, bt["seg"], bt["G"])
    assert r.flags == oracle.ERR_ACTION
    for t in (3, 5):
        assert r.token_contrib[t] == 0 and (r.dlogits[t] == 0).all()


def test_masked_columns_equal_the_reduced_vocabulary():
    # -inf logits carry zero probability: the loss, the log-probs and the dlogits of the other columns are those of
    # the same rows with the masked columns deleted (actions re-indexed), and the masked columns' dlogits are 0
    rng = np.random.default_rng(21)
    T, V = 60, 300
    z = rng.normal(0, 2, (T, V))
    keep = np.sort(rng.choice(V, 180, replace=False))
    actions = rng.choice(keep, T).astype(np.int32)
    masked = z.copy()
    masked[:, np.setdiff1d(np.arange(V), keep)] = -np.inf
    seg = oracle.segments(T, np.array([0, 10, 25, 40, T], np.int32), np.array([0, 1, 2, 3, 4], np.int32))
    A = np.array([1.0, -1.0, 0.5, -0.5])
    behave = (rng.normal(-5, 1, T)).astype(np.float32)
    full = oracle.loss_rows(masked, actions, behave, None, A, seg, 2, V=V, dual_clip_c=3.0)
    remap = np.searchsorted(keep, actions).astype(np.int32)
    red = oracle.loss_rows(np.ascontiguousarray(z[:, keep]), remap, behave, None, A, seg, 2, V=len(keep),
                           dual_clip_c=3.0)
    assert full.flags == 0 and red.flags == 0
    assert full.loss == pytest.approx(red.loss, rel=1e-13)
    np.testing.assert_allclose(full.token_logp, red.token_logp, rtol=0, atol=1e-13)
    np.testing.assert_allclose(full.dlogits[:, keep], red.dlogits, rtol=1e-12, atol=1e-16)
    assert (full.dlogits[:, np.setdiff1d(np.arange(V), keep)] == 0).all()


def test_malformed_offsets_make_loss_nan():
    rng = np.random.default_rng(15)
    bt = ragged_batch(rng, V=16)
    sto = bt["sto"].copy()
    sto[2] = sto[1] - 1 if sto[1] > 0 else -1
    seg = oracle.segments(bt["T"], sto, bt["tso"])
    A = oracle.advantages(bt["rewards"], bt["G"])
    r = oracle.loss_rows(bt["z"], bt["a"], np.zeros(bt["T"]), None, A, seg, bt["G"])
    assert r.flags & oracle.ERR_OFFSETS
    assert math.isnan(r.loss) and (r.dlogits == 0).all()


def test_nonfinite_logit_propagates_and_flags():
    rng = np.random.default_rng(16)
    bt = ragged_batch(rng, V=16)
    A = oracle.advantages(bt["rewards"], bt["G"])
    z = bt["z"].copy()
    z[2, 7] = np.nan
    r = oracle.loss_rows(z, bt["a"], np.zeros(bt["T"]), None, A, bt["seg"], bt["G"])
    assert r.flags == oracle.ERR_NONFINITE
    assert math.isnan(r.token_logp[2]) and math.isnan(r.loss)


# ---------------------------------------------------------------- gradient pins

def _fd_batch(seed, decoupled, c):
    """A tiny ragged batch whose tokens sit away from every kink."""
    rng = np.random.default_rng(seed)
    bt = ragged_batch(rng, n_groups=2, G=3, V=24, max_steps=3, max_tok=4)
    T = bt["T"]
    l = exact_logp(bt["z"], bt["a"])
    # ratios drawn away from 1 +- eps and (for the dual clip) away from c
    # log r = l - p is kept away from log(1 -+ eps); log rho = l - b away from log c
    lr = rng.choice([-0.6, -0.1, 0.05, 0.1, 0.5, 1.6], T) + rng.uniform(-0.03, 0.03, T)
    if decoupled:
        om = rng.choice([-0.3, 0.2], T)          # log omega = p - b
        p = (l - lr).astype(np.float32)
        b = (l - lr - om).astype(np.float32)
    else:
        b = (l - lr).astype(np.float32)
        p = None
    A = oracle.advantages(bt["rewards"], bt["G"])
    return bt, b, p, A


@pytest.mark.parametrize("decoupled", [False, True])
@pytest.mark.parametrize("c", [0.0, 3.0])
@pytest.mark.parametrize("norm", [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K])
def test_finite_differences(decoupled, c, norm):
    bt, b, p, A = _fd_batch(31, decoupled, c)
    kw = dict(norm=norm, k=4.0, dual_clip_c=c, grad_scale=1.0)
    base = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"], **kw)
    h = 1e-6
    rng = np.random.default_rng(0)
    idx = [(t, v) for t in range(bt["T"]) for v in rng.choice(bt["V"], 6, replace=False)]
    idx += [(t, int(bt["a"][t])) for t in range(bt["T"])]
    for t, v in idx:
        zp, zm = bt["z"].copy(), bt["z"].copy()
        zp[t, v] += h
        zm[t, v] -= h
        lp = oracle.loss_rows(zp, bt["a"], b, p, A, bt["seg"], bt["G"], want_dlogits=False, **kw).loss
        lm = oracle.loss_rows(zm, bt["a"], b, p, A, bt["seg"], bt["G"], want_dlogits=False, **kw).loss
        fd = (lp - lm) / (2 * h)
        assert abs(fd - base.dlogits[t, v]) < 1e-8 + 1e-6 * abs(fd), (t, v, fd, base.dlogits[t, v])


def test_grad_scale_scales_dlogits_only():
    bt, b, p, A = _fd_batch(32, True, 3.0)
    r1 = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"], dual_clip_c=3.0, grad_scale=1.0)
    r2 = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"], dual_clip_c=3.0, grad_scale=0.25)
    assert r1.loss == r2.loss
    np.testing.assert_allclose(r2.dlogits, 0.25 * r1.dlogits, rtol=1e-15)


@pytest.mark.parametrize("decoupled", [False, True])
@pytest.mark.parametrize("norm", [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K])
def test_matches_torch_autograd_literal(decoupled, norm):
    rng = np.random.default_rng(40)
    bt = ragged_batch(rng, n_groups=3, G=4, V=50, sigma=2.0)
    l = exact_logp(bt["z"], bt["a"])
    b = (l + rng.normal(0, 0.4, bt["T"])).astype(np.float32)
    p = (l + rng.normal(0, 0.2, bt["T"])).astype(np.float32) if decoupled else None
    A = oracle.advantages(bt["rewards"], bt["G"])
    r = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"], norm=norm, k=6.0, dual_clip_c=3.0,
                         eps_low=0.2, eps_high=0.28)
    tt = bt["seg"].tok_traj
    w = weights(bt["seg"], bt["G"], norm, 6.0)[tt]
    loss, grad = torch_literal_loss(bt["z"], bt["a"], b.astype(np.float64),
                                    (p if p is not None else b).astype(np.float64), A[tt], w, 0.2, 0.28, 3.0)
    assert abs(r.loss - loss) < 1e-13 * max(1.0, abs(loss))
    np.testing.assert_allclose(r.dlogits, grad, rtol=1e-10, atol=1e-15)


def test_n_groups_total_rescales_for_shards():
    bt, b, p, A = _fd_batch(33, False, 0.0)
    r1 = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"])
    r2 = oracle.loss_rows(bt["z"], bt["a"], b, p, A, bt["seg"], bt["G"], n_groups_total=8.0)
    ng = len(bt["seg"].traj_steps) / bt["G"]
    np.testing.assert_allclose(r2.loss, r1.loss * ng / 8.0, rtol=1e-14)

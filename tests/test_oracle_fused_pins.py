"""Pins the fused LM-head oracle (z = h W) with finite differences (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import fused


def tiny_fused(seed=0, T_groups=2, G=3, H=32, V=200):
    rng = np.random.default_rng(seed)
    N = T_groups * G
    steps = rng.integers(1, 3, N)
    toks = rng.integers(1, 4, int(steps.sum()))
    sto = np.concatenate([[0], np.cumsum(toks)])
    tso = np.concatenate([[0], np.cumsum(steps)])
    T = int(sto[-1])
    h = rng.normal(0, 1, (T, H))
    W = rng.normal(0, 0.3, (H, V))
    a = rng.integers(0, V, T).astype(np.int32)
    z = h @ W
    m = z.max(1, keepdims=True)
    l = z[np.arange(T), a] - (m[:, 0] + np.log(np.exp(z - m).sum(1)))
    lr = rng.choice([-0.5, -0.05, 0.1, 0.6, 1.5], T)  # away from the clip and dual-clip kinks
    b = (l - lr).astype(np.float32)
    r = np.zeros(N, np.float32)
    for g in range(T_groups):
        r[g * G] = 1
    seg = oracle.segments(T, sto, tso)
    A = oracle.advantages(r, G)
    return dict(h=h, W=W, a=a, b=b, A=A, seg=seg, G=G, T=T)


@pytest.mark.parametrize("norm", [oracle.NORM_TRAJ_STEPS, oracle.NORM_CONST_K])
def test_fused_finite_differences(norm):
    d = tiny_fused(3)
    kw = dict(norm=norm, k=4.0, dual_clip_c=3.0)
    base = fused.fused_loss(d["h"], d["W"], d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw)
    eps = 1e-6
    rng = np.random.default_rng(1)

    def L(h, W):
        return fused.fused_loss(h, W, d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw).loss

    for _ in range(25):
        t, j = rng.integers(d["T"]), rng.integers(d["h"].shape[1])
        hp, hm = d["h"].copy(), d["h"].copy()
        hp[t, j] += eps
        hm[t, j] -= eps
        fd = (L(hp, d["W"]) - L(hm, d["W"])) / (2 * eps)
        assert abs(fd - base.dhidden[t, j]) < 1e-8 + 1e-6 * abs(fd)
    for _ in range(25):
        j, v = rng.integers(d["W"].shape[0]), rng.integers(d["W"].shape[1])
        Wp, Wm = d["W"].copy(), d["W"].copy()
        Wp[j, v] += eps
        Wm[j, v] -= eps
        fd = (L(d["h"], Wp) - L(d["h"], Wm)) / (2 * eps)
        assert abs(fd - base.dW[j, v]) < 1e-8 + 1e-6 * abs(fd)
    # the action columns carry the largest entries: check them all
    for t in range(d["T"]):
        j, v = 0, int(d["a"][t])
        Wp, Wm = d["W"].copy(), d["W"].copy()
        Wp[j, v] += eps
        Wm[j, v] -= eps
        fd = (L(d["h"], Wp) - L(d["h"], Wm)) / (2 * eps)
        assert abs(fd - base.dW[j, v]) < 1e-8 + 1e-6 * abs(fd)


def test_fused_equals_logits_path_on_hw():
    d = tiny_fused(4)
    kw = dict(norm=oracle.NORM_CONST_K, k=10.0, dual_clip_c=3.0)
    f = fused.fused_loss(d["h"], d["W"], d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw)
    z = d["h"] @ d["W"]
    r = oracle.loss_rows(z, d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw)
    assert f.loss == r.loss
    # trace identity: <dW, W> = <dh, h> = <D, z>
    dz = (r.dlogits * z).sum()
    np.testing.assert_allclose((f.dW * d["W"]).sum(), dz, rtol=1e-11)
    np.testing.assert_allclose((f.dhidden * d["h"]).sum(), dz, rtol=1e-11)
    # rows of D sum to zero, hence so do the rows of dW
    assert np.abs(f.dW.sum(1)).max() < 1e-12 * np.abs(f.dW).max() * f.dW.shape[1]


def test_fused_rows_match_full():
    d = tiny_fused(5)
    to_bits = lambda x: (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    hb, Wb = to_bits(d["h"]), to_bits(d["W"])
    kw = dict(norm=oracle.NORM_TRAJ_STEPS, k=10.0)
    full = fused.fused_loss(hb, Wb, d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw)
    rows = [0, 3, d["T"] - 1]
    part = fused.fused_rows(hb, Wb, rows, d["a"], d["b"], None, d["A"], d["seg"], d["G"], **kw)
    np.testing.assert_allclose(part.rows.token_logp, full.rows.token_logp[rows], rtol=0, atol=1e-13)
    np.testing.assert_allclose(part.dhidden, full.dhidden[rows], rtol=1e-12, atol=1e-16)

"""Shared helpers of the GPU parity tests: run libgrpo and the oracle on the same
seeded inputs and apply the parity gates.

Gates (loss relative 1e-5 and bf16 dlogits absolute 2e-3 are the stated
targets; the rest follow from the arithmetic):
  * integers (token->trajectory map, trajectory offsets, gather indices): bit-exact;
  * loss and per-trajectory losses: relative 1e-5 (logits path); on the fused
    path relative 1e-5 of sum_t |w_i s_t|, the magnitude of the terms the loss
    sums (check_fused_loss);
  * token log-probs: absolute 2e-5 (fp32 log-sum-exp over V terms);
  * dlogits, absolute 2e-3 (bf16) and a scaled gate, since |dlogits| is far
    below 2e-3 at these sizes: with grad_scale = 1/max|g_t| (so rows are O(1)),
    |gpu - ref| <= 2^-8 |ref| + 1e-5 max_row|ref| for bf16 (one bf16 rounding
    of a correct fp32 value; 2^-8 + 2^-11 on the rows the pipelined kernel runs,
    whose LDS part rounds its terms to fp16 first), and <= 1e-5 max_row|ref| for
    fp32 outputs.
Rows whose oracle ratio sits within 1e-6 of a clip boundary or whose term
sits within 1e-6 relative of the dual-clip floor are kinks, where either
one-sided derivative is correct: they are counted and exempt from the dlogits
gate only.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import paper_2606_05597_amd as grpo

LOSS_RTOL = 1e-5
LOGP_ATOL = 2e-5
BF16_ABS = 2e-3


def check_fused_loss(got: float, contrib, what: str = "", report: bool = False) -> float:
    """The fused path's loss gate: |got - sum_t c_t| <= 1e-5 * sum_t |c_t| over the oracle's per-token terms
    c_t = -w_i s_t, i.e. relative 1e-5 of |loss| times the sum's cancellation ratio kappa = sum|c_t| / |sum c_t|.
    The fused logits are fp32 sums of H products on the matrix cores, so each token's log-prob is off by some
    delta_t (up to the 5e-5 log-prob gate); with ds_t/dl_t = s_t wherever it is not 0, the loss moves by
    sum_t w_i s_t delta_t <= sum_t |c_t| max|delta|, and group-relative advantages (zero sum per group, Sec. 3.2)
    keep sum |c_t| well above |loss|.  Returns the error relative to |loss|."""
    c = np.asarray(contrib, dtype=np.float64)
    ref = math.fsum(c)
    mag = float(np.abs(c).sum())
    err = abs(float(got) - ref)
    rel = err / abs(ref) if ref != 0 else (0.0 if err == 0 else math.inf)
    if report:
        kappa = mag / abs(ref) if ref != 0 else math.inf
        print(f"{what}: loss {got!r} oracle {ref!r} rel {rel:.2e} kappa {kappa:.1f} "
              f"(gate {LOSS_RTOL * mag:.3g}, |err| {err:.3g})", flush=True)
    assert err <= LOSS_RTOL * mag, (what, got, ref, mag)
    return rel


def to_np_logits(t: torch.Tensor) -> np.ndarray:
    """Device logits to the oracle's input format (float32, or bf16 bit patterns)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dl_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def device_batch(b: dict, device="cuda"):
    st = b["structure"]
    return dict(
        step_tok_off=torch.from_numpy(st.step_tok_off).to(device),
        traj_step_off=torch.from_numpy(st.traj_step_off).to(device),
    )


def oracle_inputs(b: dict, adv64: np.ndarray):
    st = b["structure"]
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    return dict(seg=seg, actions=b["actions"].cpu().numpy(), behave=b["behave"].cpu().numpy(),
                prox=None if b["prox"] is None else b["prox"].cpu().numpy(), adv=adv64)


def kink_rows(ref: oracle.LossResult, behave, prox, adv_tok, eps_lo, eps_hi, c, rows=None) -> np.ndarray:
    """Rows (indices into ref's arrays) within 1e-6 of an eps-clip or dual-clip kink."""
    l = ref.token_logp
    b = behave.astype(np.float64) if rows is None else behave[rows].astype(np.float64)
    p = b if prox is None else (prox.astype(np.float64) if rows is None else prox[rows].astype(np.float64))
    r = np.exp(l - p)
    near = (np.abs(r - (1 - eps_lo)) < 1e-6) | (np.abs(r - (1 + eps_hi)) < 1e-6)
    if c > 0:
        A = adv_tok
        rho = np.exp(l - b)
        near |= (A < 0) & (np.abs(rho * A - c * A) < 1e-6 * np.abs(c * A))
        near |= (A < 0) & (np.abs(np.exp(p - b) * np.clip(r, 1 - eps_lo, 1 + eps_hi) * A - c * A)
                           < 1e-6 * np.abs(c * A))
    return np.nonzero(near)[0]


# bf16 rows of 49,153 to 188,416 columns run the pipelined row kernel, whose LDS part forms dlogits from fp16 terms
# exp(z - m) <= 1: one more relative rounding of at most 2^-11 before the bf16 one
PIPE_TERMS_V = (49152, 188416)


def check_dlogits(gpu: np.ndarray, ref: np.ndarray, is_bf16: bool, exempt=(), scaled: bool = False, what=""):
    """Applies the dlogits gates row by row; returns the max normalised error."""
    keep = np.ones(gpu.shape[0], bool)
    keep[list(exempt)] = False
    g, r = gpu[keep], ref[keep]
    diff = np.abs(g - r)
    rowmax = np.abs(r).max(axis=1, keepdims=True)
    if is_bf16:
        assert diff.max(initial=0) <= BF16_ABS, f"{what}: bf16 dlogits abs err {diff.max()}"
        if scaled:
            terms = PIPE_TERMS_V[0] < r.shape[1] <= PIPE_TERMS_V[1]
            bound = (2.0 ** -8 + (2.0 ** -11 if terms else 0.0)) * np.abs(r) + 1e-5 * rowmax
            worst = (diff / np.maximum(bound, 1e-300)).max(initial=0)
            assert worst <= 1.0, f"{what}: scaled bf16 gate exceeded by {worst}"
            return worst
    else:
        bound = 1e-5 * rowmax
        worst = (diff / np.maximum(bound, 1e-300)).max(initial=0)
        assert worst <= 1.0, f"{what}: fp32 dlogits gate exceeded by {worst}"
        return worst
    return diff.max(initial=0)


def run_gpu(b: dict, adv32: torch.Tensor, *, norm, k, eps_low=0.2, eps_high=0.2, c=0.0, grad_scale=1.0,
            dlogits=True, aux=True, n_groups_total=0.0, prox=None, logits=None):
    dev = device_batch(b)
    st = b["structure"]
    N = len(st.rewards)
    a = grpo.LossAux.alloc(st.T, N, "cuda") if aux else None
    lg = b["logits"] if logits is None else logits
    loss, dl = grpo.grpo_loss_fwd_bwd(lg, b["actions"], b["behave"], adv32, dev["step_tok_off"],
                                      dev["traj_step_off"], b["cfg"].G, V=b["V"],
                                      prox_logp=b["prox"] if prox is None else prox, norm=norm, k=k,
                                      eps_low=eps_low, eps_high=eps_high, dual_clip_c=c, grad_scale=grad_scale,
                                      n_groups_total=n_groups_total, dlogits=dlogits, aux=a)
    torch.cuda.synchronize()
    return loss.item(), dl, a


def gpu_norm(norm):
    return grpo.GRPO_NORM_CONST_K if norm == oracle.NORM_CONST_K else grpo.GRPO_NORM_TRAJ_STEPS

"""Seeded synthetic rollout batches with the structure of the paper's workload.

This module only draws inputs.  It holds none of the loss arithmetic: no
advantage, ratio, clip, normaliser or gradient.  Both the HIP library and the
oracle read what it produces and neither checks against it.

Structure (AsyncWebRL): a batch is task groups of G trajectories (Sec. 3.2,
Table 5: G = 8, 16 groups per batch); rewards are binary (Sec. 4.1); groups
whose G rewards are all equal are redrawn, as DAPO-style dynamic sampling keeps
only mixed groups (Sec. 3.2); failures run longer than successes (Sec. 1 and
Sec. 5.1: 12.5 vs 5.1 steps, 30-40% success).  Each step emits a geometric
number of action tokens.  Logits are i.i.d. normal, stored bf16 (fp32 for the
tiny case); actions are drawn from softmax(z) by the Gumbel-max trick
(argmax of z + Gumbel noise), or uniformly for the tiny case.

Old (behave) log-probs follow "old = the policy's log-prob of the sampled token
plus N(0, sigma)".  That log-prob is what the rollout engine records; the
generator stands in for the engine with torch's fp32 logsumexp over the stored
logits (``engine_logp``).  It is an input like any other: any value is valid
input to the loss.

Where a stated token count T cannot come out of the literal recipe, per-step
token counts are drawn from the stated distribution and clamps and then
rescaled to hit T exactly with largest-remainder rounding (each count >= 1),
which keeps the failure/success asymmetry and the raggedness.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Config:
    name: str
    n_groups: int
    G: int
    V: int
    dtype: str                      # "f32" or "bf16" logits
    logit_sigma: float
    success_p: float
    steps_fail: tuple[int, int]     # inclusive uniform range of steps for failures
    steps_succ: tuple[int, int]     # ... and for successes
    tok_mean: float                 # geometric mean of tokens per step (0 = fixed)
    tok_clamp: tuple[int, int]
    behave_sigma: float
    k: float
    T_target: int | None = None     # rescale to exactly this many tokens
    fixed_steps: int | None = None  # tiny case: every trajectory has this many steps
    fixed_tokens: int | None = None  # tiny case: every step has this many tokens
    uniform_actions: bool = False
    H: int | None = None            # fused LM-head: hidden size
    hidden_sigma: float = 1.0
    w_sigma: float = 0.02
    vocab_chunk: int = 8192
    seed: int = 0
    notes: dict = field(default_factory=dict, compare=False, hash=False)


CONFIGS: dict[str, Config] = {
    # 1 group of G=4, 3 steps x 16 tokens each; fp32 [192, 1024] ~ N(0,1);
    # uniform actions; old = logp + N(0, 0.1); rewards Bernoulli(0.5); k = 3.
    "tiny": Config("tiny", 1, 4, 1024, "f32", 1.0, 0.5, (3, 3), (3, 3), 0.0, (16, 16), 0.1, 3.0,
                   fixed_steps=3, fixed_tokens=16, uniform_actions=True, seed=1),
    # 8 groups x 8; steps U{2..15}; tokens/step Geom(mean 64) clamped to
    # [16, 256]; bf16 [T ~ 35k, 32000] ~ N(0, 2^2); old = logp + N(0, 0.05);
    # rewards Bernoulli(0.4); k = 8.
    "v32k": Config("v32k", 8, 8, 32000, "bf16", 2.0, 0.4, (2, 15), (2, 15), 64.0, (16, 256), 0.05, 8.0,
                   seed=2),
    # 16 groups x 8 at V = 151,936; failures U{8..30} steps, successes
    # U{3..12}; Geom(mean 96) tokens/step; T = 120,000; success 0.35; k = 10.
    "v152k": Config("v152k", 16, 8, 151936, "bf16", 2.0, 0.35, (8, 30), (3, 12), 96.0, (1, 4096), 0.05, 10.0,
                    T_target=120000, seed=3),
    # 32 groups x 8; failures U{10..40}, successes U{4..15}; Geom(mean 128)
    # clamped to 512; T = 250,000; success 0.35; k = 16.
    "long": Config("long", 32, 8, 151936, "bf16", 2.0, 0.35, (10, 40), (4, 15), 128.0, (1, 512), 0.05, 16.0,
                   T_target=250000, seed=4),
    # Fused LM-head: hidden bf16 [65,536, 3,584] ~ N(0,1), W bf16
    # [3,584, 151,936] ~ N(0, 0.02^2); 8 groups x 8 with the v152k recipe
    # rescaled to T = 65,536; vocabulary chunks of 8192; k = 10.
    "fused": Config("fused", 8, 8, 151936, "bf16", 0.0, 0.35, (8, 30), (3, 12), 96.0, (1, 4096), 0.05, 10.0,
                    T_target=65536, H=3584, seed=5),
}


@dataclass
class Structure:
    rewards: np.ndarray        # float32 [N]
    traj_steps: np.ndarray     # int32 [N]
    step_tokens: np.ndarray    # int32 [n_steps]
    step_tok_off: np.ndarray   # int32 [n_steps+1]
    traj_step_off: np.ndarray  # int32 [N+1]
    T: int
    redraws: int               # groups redrawn because all G rewards were equal


def _largest_remainder(counts: np.ndarray, total: int) -> np.ndarray:
    """Integer counts (each >= 1) proportional to ``counts`` summing to ``total``."""
    if total < len(counts):
        raise ValueError(f"cannot spread {total} tokens over {len(counts)} steps with at least one each")
    x = counts.astype(np.float64) * (total / counts.sum())
    base = np.maximum(1, np.floor(x)).astype(np.int64)
    deficit = total - int(base.sum())
    frac = x - np.floor(x)
    if deficit > 0:
        order = np.argsort(-frac, kind="stable")
        base[order[:deficit]] += 1
    while deficit < 0:
        order = np.argsort(-base, kind="stable")
        take = order[: min(-deficit, int((base > 1).sum()))]
        base[take] -= 1
        deficit = total - int(base.sum())
    return base


def make_structure(cfg: Config, seed: int | None = None, T_target: int | None = None) -> Structure:
    """Rewards, step counts and token counts for one batch (numpy PCG64)."""
    rng = np.random.default_rng(cfg.seed if seed is None else seed)
    N = cfg.n_groups * cfg.G
    rewards = np.empty(N, np.float32)
    redraws = 0
    for g in range(cfg.n_groups):
        while True:
            r = (rng.random(cfg.G) < cfg.success_p).astype(np.float32)
            if r.min() != r.max():
                break
            redraws += 1
        rewards[g * cfg.G:(g + 1) * cfg.G] = r
    if cfg.fixed_steps is not None:
        steps = np.full(N, cfg.fixed_steps, np.int64)
    else:
        lo_f, hi_f = cfg.steps_fail
        lo_s, hi_s = cfg.steps_succ
        steps = np.where(rewards > 0, rng.integers(lo_s, hi_s + 1, N), rng.integers(lo_f, hi_f + 1, N))
    n_steps = int(steps.sum())
    if cfg.fixed_tokens is not None:
        toks = np.full(n_steps, cfg.fixed_tokens, np.int64)
    else:
        toks = np.clip(rng.geometric(1.0 / cfg.tok_mean, n_steps), cfg.tok_clamp[0], cfg.tok_clamp[1])
    target = T_target if T_target is not None else cfg.T_target
    if target is not None:
        toks = _largest_remainder(toks, target)
    step_tok_off = np.zeros(n_steps + 1, np.int64)
    np.cumsum(toks, out=step_tok_off[1:])
    traj_step_off = np.zeros(N + 1, np.int64)
    np.cumsum(steps, out=traj_step_off[1:])
    T = int(step_tok_off[-1])
    assert T < 2**31
    return Structure(rewards, steps.astype(np.int32), toks.astype(np.int32), step_tok_off.astype(np.int32),
                     traj_step_off.astype(np.int32), T, redraws)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _row_chunks(T: int, V: int, budget_elems: int = 1 << 28):
    rows = max(1, budget_elems // max(V, 1))
    for r0 in range(0, T, rows):
        yield r0, min(T, r0 + rows)


def make_logits(T: int, V: int, sigma: float, dtype: str, device, seed: int, ld: int | None = None) -> torch.Tensor:
    """[T, ld] logits ~ N(0, sigma^2) in the storage dtype (columns >= V are zero)."""
    ld = V if ld is None else ld
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.zeros((T, ld), dtype=tdt, device=device) if ld != V else torch.empty((T, V), dtype=tdt, device=device)
    for c, (r0, r1) in enumerate(_row_chunks(T, V)):
        x = torch.randn((r1 - r0, V), generator=_gen(device, seed * 7919 + c), device=device, dtype=torch.float32)
        out[r0:r1, :V] = (x * sigma).to(tdt)
    return out


def gumbel_max_actions(logits: torch.Tensor, V: int, seed: int) -> torch.Tensor:
    """Draws a_t ~ softmax(z_t) as argmax_v (z_tv + Gumbel noise), int32 [T]."""
    T = logits.shape[0]
    out = torch.empty(T, dtype=torch.int32, device=logits.device)
    for c, (r0, r1) in enumerate(_row_chunks(T, V, 1 << 27)):
        u = torch.rand((r1 - r0, V), generator=_gen(logits.device, seed * 104729 + c), device=logits.device,
                       dtype=torch.float32).clamp_(min=1e-30)
        gumbel = -torch.log(-torch.log(u))
        out[r0:r1] = torch.argmax(logits[r0:r1, :V].float() + gumbel, dim=1).to(torch.int32)
    return out


def engine_logp(logits: torch.Tensor, actions: torch.Tensor, V: int) -> torch.Tensor:
    """Stand-in for the rollout engine's recorded log-prob of each sampled token (fp32)."""
    T = logits.shape[0]
    out = torch.empty(T, dtype=torch.float32, device=logits.device)
    for r0, r1 in _row_chunks(T, V, 1 << 27):
        z = logits[r0:r1, :V].float()
        out[r0:r1] = z.gather(1, actions[r0:r1].long()[:, None])[:, 0] - torch.logsumexp(z, dim=1)
    return out


def add_noise(x: torch.Tensor, sigma: float, seed: int) -> torch.Tensor:
    """x + N(0, sigma^2), fp32."""
    n = torch.randn(x.shape, generator=_gen(x.device, seed), device=x.device, dtype=torch.float32)
    return (x.float() + sigma * n).contiguous()


def make_batch(name_or_cfg, device="cpu", seed: int | None = None, T_target: int | None = None,
               ld: int | None = None, with_prox: bool = False) -> dict:
    """A full logits-path batch: structure (numpy) plus device tensors.

    Keys: cfg, structure, logits [T, ld], actions int32 [T], behave fp32 [T],
    prox fp32 [T] or None, rewards fp32 [N] (device).  ``with_prox`` also draws
    a distinct proximal log-prob (behave + N(0, 0.05)) to exercise the
    decoupled ratio.
    """
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    s = cfg.seed if seed is None else seed
    st = make_structure(cfg, s, T_target)
    logits = make_logits(st.T, cfg.V, cfg.logit_sigma, cfg.dtype, device, s, ld)
    if cfg.uniform_actions:
        actions = torch.randint(0, cfg.V, (st.T,), generator=_gen(device, s * 31 + 1), device=device,
                                dtype=torch.int32)
    else:
        actions = gumbel_max_actions(logits, cfg.V, s)
    lp = engine_logp(logits, actions, cfg.V)
    behave = add_noise(lp, cfg.behave_sigma, s * 31 + 2)
    prox = add_noise(behave, 0.05, s * 31 + 3) if with_prox else None
    rewards = torch.from_numpy(st.rewards).to(device)
    return dict(cfg=cfg, structure=st, logits=logits, actions=actions, behave=behave, prox=prox,
                rewards=rewards, V=cfg.V)


def make_fused_batch(name_or_cfg="fused", device="cpu", seed: int | None = None, T_target: int | None = None,
                     H: int | None = None, V: int | None = None) -> dict:
    """A fused LM-head batch: hidden [T, H] and W [H, V] bf16, plus the rollout structure.

    Actions are drawn from softmax(h W) and old log-probs from the engine
    stand-in on the same product, computed in fp32 vocabulary chunks.
    """
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    s = cfg.seed if seed is None else seed
    H = cfg.H if H is None else H
    V = cfg.V if V is None else V
    st = make_structure(cfg, s, T_target)
    T = st.T
    hidden = make_logits(T, H, cfg.hidden_sigma, "bf16", device, s * 13 + 1)
    W = make_logits(H, V, cfg.w_sigma, "bf16", device, s * 13 + 2)
    actions = torch.empty(T, dtype=torch.int32, device=device)
    lp = torch.empty(T, dtype=torch.float32, device=device)
    Wf = W.float()
    for c, (r0, r1) in enumerate(_row_chunks(T, V, 1 << 27)):
        z = hidden[r0:r1].float() @ Wf
        a = gumbel_max_actions(z, V, s * 977 + c)
        actions[r0:r1] = a
        lp[r0:r1] = engine_logp(z, a, V)
    del Wf
    behave = add_noise(lp, cfg.behave_sigma, s * 31 + 2)
    rewards = torch.from_numpy(st.rewards).to(device)
    return dict(cfg=cfg, structure=st, hidden=hidden, W=W, actions=actions, behave=behave, prox=None,
                rewards=rewards, H=H, V=V)

"""Plain fp64 CPU oracle for the multi-step GRPO loss (AsyncWebRL, Eq. 1 and Eq. 2).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package; the product
library never does.  It shares no code with the HIP path.  The arithmetic lives
in ``grpo_oracle.c`` (built with gcc into ``liboracle.so`` next to it); this
module only marshals numpy arrays.  The fused LM-head oracle in ``fused.py``
adds fp64 matrix products around the same per-row definition.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "grpo_oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")

ERR_ACTION = 1
ERR_OFFSETS = 2
ERR_NONFINITE = 4
NORM_TRAJ_STEPS = 0
NORM_CONST_K = 1

DT_F32, DT_BF16, DT_F64 = 0, 1, 2

_lib = None


def build(force: bool = False) -> str:
    """Compiles grpo_oracle.c with gcc (-O2, OpenMP over rows)."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        I32, I64, D = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_segments.argtypes = [I64, I32, P, I32, P, P, P, P]
        lib.oracle_segments.restype = ctypes.c_int
        lib.oracle_advantages.argtypes = [P, I32, I32, I32, D, P]
        lib.oracle_advantages.restype = None
        lib.oracle_loss_rows.argtypes = [P, ctypes.c_int, I64, I64, P, P, P, P, P, P, I32, I32, D,
                                         ctypes.c_int, D, D, D, D, D, I64, I64, P, P, P, P, P]
        lib.oracle_loss_rows.restype = ctypes.c_int
        lib.oracle_loss_from_logp.argtypes = [P, I64, P, P, P, P, P, P, I32, I32, D, ctypes.c_int, D, D, D, D, D,
                                              I64, I64, P, P, P]
        lib.oracle_loss_from_logp.restype = ctypes.c_int
        lib.oracle_reduce.argtypes = [P, P, I64, I32, P]
        lib.oracle_reduce.restype = D
        lib.oracle_advantages_success_filter.argtypes = [P, I32, P]
        lib.oracle_advantages_success_filter.restype = None
        lib.oracle_mixed_groups.argtypes = [P, I32, I32, P]
        lib.oracle_mixed_groups.restype = I32
        lib.oracle_logp_entropy.argtypes = [P, ctypes.c_int, I64, I64, P, I64, I64, P, P]
        lib.oracle_logp_entropy.restype = ctypes.c_int
        lib.oracle_vocab_shard_stats.argtypes = [P, ctypes.c_int, I64, I64, I64, P, I64, I64, P, P, P]
        lib.oracle_vocab_shard_stats.restype = None
        lib.oracle_ratio_stats.argtypes = [I64, P, P, P, P, D, D, P]
        lib.oracle_ratio_stats.restype = None
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def set_threads(n: int) -> None:
    """OpenMP threads for later oracle calls (the results do not depend on the count)."""
    _load().oracle_set_threads(int(n))


def threads() -> int:
    """OpenMP threads the oracle's row loop uses."""
    return int(_load().oracle_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


@dataclass
class Segments:
    traj_tok_off: np.ndarray  # int32 [n_traj+1]
    tok_traj: np.ndarray      # int32 [T]
    traj_steps: np.ndarray    # int32 [n_traj]  (|tau_i|)
    flags: int


def segments(T: int, step_tok_off, traj_step_off) -> Segments:
    """Token/step/trajectory bookkeeping of Eq. 1's triple sum (see grpo_oracle.c)."""
    lib = _load()
    sto = _c(step_tok_off, np.int32)
    tso = _c(traj_step_off, np.int32)
    n_steps, n_traj = len(sto) - 1, len(tso) - 1
    tto = np.empty(n_traj + 1, np.int32)
    tt = np.empty(T, np.int32)
    ts = np.empty(n_traj, np.int32)
    f = lib.oracle_segments(T, n_steps, _ptr(sto), n_traj, _ptr(tso), _ptr(tto), _ptr(tt), _ptr(ts))
    return Segments(tto, tt, ts, int(f))


def gather_index(T: int, ld: int, actions) -> np.ndarray:
    """Flat element index t*ld + a_t of each token's action logit."""
    return np.arange(T, dtype=np.int64) * np.int64(ld) + np.asarray(actions, dtype=np.int64)


ADV_GROUP_NORM = 0        # (r - mean) / (std + std_eps) per group (Sec. 3.2)
ADV_SUCCESS_FILTER = 1    # RAFT++ / filtered BC: 1[r > 0], no group normalisation (Sec. 3.2, Table 5)


def advantages(rewards, group_size: int, ddof: int = 1, std_eps: float = 0.0,
               mode: int = ADV_GROUP_NORM) -> np.ndarray:
    """Per-trajectory advantage, fp64: group-relative (Sec. 3.2) or the RAFT++ success filter."""
    lib = _load()
    r = _c(rewards, np.float32)
    out = np.empty(len(r), np.float64)
    if mode == ADV_GROUP_NORM:
        lib.oracle_advantages(_ptr(r), len(r), group_size, ddof, float(std_eps), _ptr(out))
    elif mode == ADV_SUCCESS_FILTER:
        lib.oracle_advantages_success_filter(_ptr(r), len(r), _ptr(out))
    else:
        raise ValueError(f"unknown advantage mode {mode}")
    return out


def mixed_groups(rewards, group_size: int):
    """DAPO dynamic sampling (Sec. 3.2): per group, 1 when its rewards are not all equal; and their count."""
    lib = _load()
    r = _c(rewards, np.float32)
    mixed = np.empty(len(r) // group_size, np.int32)
    n = lib.oracle_mixed_groups(_ptr(r), len(r), group_size, _ptr(mixed))
    return mixed, int(n)


@dataclass
class LossResult:
    loss: float
    traj_loss: np.ndarray      # [n_traj] fp64
    token_logp: np.ndarray     # [rows]   fp64
    token_contrib: np.ndarray  # [rows]   fp64, -w_i * s_t
    token_g: np.ndarray        # [rows]   fp64, dloss/dl_t * grad_scale
    token_state: np.ndarray    # [rows]   int32: bit0 eps-clip cut, bit1 dual clip cut
    dlogits: np.ndarray | None  # [rows, V] fp64
    flags: int

    @property
    def abs_terms(self) -> float:
        """sum_t |w_i s_t| over the rows computed: the magnitude of the terms the loss sums."""
        return float(np.abs(self.token_contrib).sum())

    @property
    def kappa(self) -> float:
        """Cancellation ratio of the loss sum, sum_t |w_i s_t| / |sum_t w_i s_t| (>= 1; inf for a zero loss).

        Group-relative advantages sum to zero over each group (Sec. 3.2), so the per-token terms of Eq. 1 carry
        both signs and largely cancel: an absolute error e in the terms moves the loss by up to kappa * e
        relative to its own size."""
        return cancellation_ratio(self.token_contrib)


def _logits_dtype(logits: np.ndarray) -> int:
    if logits.dtype == np.float32:
        return DT_F32
    if logits.dtype == np.uint16:  # bfloat16 bit patterns
        return DT_BF16
    if logits.dtype == np.float64:
        return DT_F64
    raise TypeError(f"oracle: unsupported logits dtype {logits.dtype}")


def loss_rows(logits: np.ndarray, actions, behave_logp, prox_logp, adv, seg: Segments, group_size: int, *,
              V: int | None = None, norm: int = NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2,
              eps_high: float = 0.2, dual_clip_c: float = 0.0, grad_scale: float = 1.0,
              n_groups_total: float = 0.0, row_begin: int = 0, row_end: int | None = None,
              want_dlogits: bool = True, row_offset: int = 0) -> LossResult:
    """Per-token quantities and dlogits for token rows [row_begin, row_end).

    ``logits`` is [rows_held, ld] (float32, bfloat16 bit patterns as uint16, or
    float64) and holds token rows starting at token ``row_offset``; V (default
    ld) is the vocabulary size.  Per-token inputs (actions, log-probs) are
    indexed by absolute token number; per-row outputs by t - row_begin.  The
    loss and traj_loss fields sum only the rows computed.
    """
    lib = _load()
    logits = np.ascontiguousarray(logits)
    dt = _logits_dtype(logits)
    ld = logits.shape[1]
    V = ld if V is None else int(V)
    assert 1 <= V <= ld
    T = len(seg.tok_traj)
    n_traj = len(seg.traj_steps)
    if row_end is None:
        row_end = T
    n_rows = row_end - row_begin
    assert row_begin >= row_offset and row_end - row_offset <= logits.shape[0]
    a = _c(actions, np.int32)
    b = _c(behave_logp, np.float32)
    p = _c(prox_logp, np.float32)
    A = _c(adv, np.float64)
    n_groups = float(n_groups_total) if n_groups_total else n_traj / group_size
    logp = np.empty(n_rows, np.float64)
    contrib = np.empty(n_rows, np.float64)
    g = np.empty(n_rows, np.float64)
    st = np.empty(n_rows, np.int32)
    dl = np.empty((n_rows, V), np.float64) if want_dlogits else None
    # The C routine addresses token row t at element t*ld of its base pointer:
    # shift the base back by row_offset rows so absolute token numbers work.
    base = logits.ctypes.data - row_offset * ld * logits.itemsize
    f = lib.oracle_loss_rows(ctypes.c_void_p(base), dt, V, ld, _ptr(a), _ptr(b), _ptr(p), _ptr(A),
                             _ptr(seg.tok_traj), _ptr(seg.traj_steps), seg.flags, group_size, n_groups,
                             norm, float(k), float(eps_low), float(eps_high), float(dual_clip_c),
                             float(grad_scale), row_begin, row_end, _ptr(logp), _ptr(contrib), _ptr(g),
                             _ptr(st), _ptr(dl))
    traj = np.zeros(n_traj, np.float64)
    tt = np.ascontiguousarray(seg.tok_traj[row_begin:row_end])
    total = lib.oracle_reduce(_ptr(contrib), _ptr(tt), n_rows, n_traj, _ptr(traj))
    return LossResult(float(total), traj, logp, contrib, g, st, dl, int(f))


def cancellation_ratio(terms) -> float:
    """sum |x| / |sum x| of the terms of a sum, in fp64 (inf when the sum is 0)."""
    x = np.asarray(terms, dtype=np.float64)
    total = abs(float(np.sum(x)))
    mag = float(np.abs(x).sum())
    return float("inf") if total == 0.0 else mag / total


def valid_tokens(actions, V: int, seg: Segments) -> np.ndarray:
    """Tokens that enter the loss: the action lies in [0, V) and the offsets are well formed (int32 0/1)."""
    a = np.asarray(actions, dtype=np.int64)
    ok = (a >= 0) & (a < V)
    if seg.flags & ERR_OFFSETS:
        ok[:] = False
    return ok.astype(np.int32)


def ratio_stats(token_logp, behave_logp, prox_logp, valid, eps_low: float = 0.2, eps_high: float = 0.2) -> np.ndarray:
    """Importance-ratio statistics over the valid tokens (see grpo_oracle.c): [sum r, min r, max r, sum rho,
    min rho, max rho, tokens with r outside [1 - eps_low, 1 + eps_high], tokens counted], r = pi/pi_prox and
    rho = pi/pi_behave (Sec. 3.2), fp64."""
    lib = _load()
    l = _c(token_logp, np.float64)
    b = _c(behave_logp, np.float32)
    p = _c(prox_logp, np.float32)
    v = _c(valid, np.int32)
    n = len(l)
    assert len(b) >= n and len(v) >= n and (p is None or len(p) >= n)
    out = np.empty(8, np.float64)
    lib.oracle_ratio_stats(n, _ptr(l), _ptr(b), _ptr(p), _ptr(v), float(eps_low), float(eps_high), _ptr(out))
    return out


def loss_from_logp(token_logp, actions, behave_logp, prox_logp, adv, seg: Segments, group_size: int, *, V: int,
                   norm: int = NORM_CONST_K, k: float = 10.0, eps_low: float = 0.2, eps_high: float = 0.2,
                   dual_clip_c: float = 0.0, grad_scale: float = 1.0, n_groups_total: float = 0.0,
                   row_begin: int = 0, row_end: int | None = None) -> LossResult:
    """Eq. 1 for token rows [row_begin, row_end) from their new log-probs ``token_logp`` (indexed by
    t - row_begin, as loss_rows returns them), without the logits: the same per-token terms loss_rows forms after
    its log-softmax, for another normaliser or other parameters.  dlogits is None."""
    lib = _load()
    T = len(seg.tok_traj)
    n_traj = len(seg.traj_steps)
    if row_end is None:
        row_end = T
    n_rows = row_end - row_begin
    l = _c(token_logp, np.float64)
    assert len(l) == n_rows
    a = _c(actions, np.int32)
    b = _c(behave_logp, np.float32)
    p = _c(prox_logp, np.float32)
    A = _c(adv, np.float64)
    n_groups = float(n_groups_total) if n_groups_total else n_traj / group_size
    contrib = np.empty(n_rows, np.float64)
    g = np.empty(n_rows, np.float64)
    st = np.empty(n_rows, np.int32)
    f = lib.oracle_loss_from_logp(_ptr(l), int(V), _ptr(a), _ptr(b), _ptr(p), _ptr(A), _ptr(seg.tok_traj),
                                  _ptr(seg.traj_steps), seg.flags, group_size, n_groups, norm, float(k),
                                  float(eps_low), float(eps_high), float(dual_clip_c), float(grad_scale), row_begin,
                                  row_end, _ptr(contrib), _ptr(g), _ptr(st))
    traj = np.zeros(n_traj, np.float64)
    tt = np.ascontiguousarray(seg.tok_traj[row_begin:row_end])
    total = lib.oracle_reduce(_ptr(contrib), _ptr(tt), n_rows, n_traj, _ptr(traj))
    return LossResult(float(total), traj, l.copy(), contrib, g, st, None, int(f))


class LogpEntropy:
    """Forward-only oracle results: per-row action log-prob, entropy and error flags."""

    def __init__(self, token_logp, token_entropy, flags):
        self.token_logp = token_logp
        self.token_entropy = token_entropy
        self.flags = flags


def logp_entropy(logits: np.ndarray, actions, *, V: int | None = None, row_begin: int = 0,
                 row_end: int | None = None, row_offset: int = 0) -> LogpEntropy:
    """The sampled action's log-prob and the policy entropy -sum p log p for token rows [row_begin, row_end).

    ``logits`` is [rows_held, ld] (float32, bfloat16 bit patterns as uint16, or float64) holding token rows
    from ``row_offset`` on; ``actions`` is indexed by absolute token number, the outputs by t - row_begin.
    """
    lib = _load()
    logits = np.ascontiguousarray(logits)
    dt = _logits_dtype(logits)
    ld = logits.shape[1]
    V = ld if V is None else int(V)
    assert 1 <= V <= ld
    if row_end is None:
        row_end = row_offset + logits.shape[0]
    assert row_begin >= row_offset and row_end - row_offset <= logits.shape[0]
    a = _c(actions, np.int32)
    n = row_end - row_begin
    logp = np.empty(n, np.float64)
    ent = np.empty(n, np.float64)
    base = logits.ctypes.data - row_offset * ld * logits.itemsize
    f = lib.oracle_logp_entropy(ctypes.c_void_p(base), dt, V, ld, _ptr(a), row_begin, row_end, _ptr(logp),
                                _ptr(ent))
    return LogpEntropy(logp, ent, int(f))


class ShardStats:
    """Per-row statistics of one vocabulary shard: max m, sum s of exp(z - m), the action's logit z_a (-inf when
    the action lies outside the shard)."""

    def __init__(self, m, s, za):
        self.m = m
        self.s = s
        self.za = za


def vocab_shard_stats(logits_shard: np.ndarray, actions, v_begin: int, *, V: int | None = None, row_begin: int = 0,
                      row_end: int | None = None, row_offset: int = 0) -> ShardStats:
    """Statistics of the shard holding global vocabulary columns [v_begin, v_begin + V) for token rows
    [row_begin, row_end).  ``logits_shard`` is [rows_held, ld] with the shard's columns only, holding token rows
    from ``row_offset`` on; ``actions`` are global column ids indexed by absolute token number."""
    lib = _load()
    logits_shard = np.ascontiguousarray(logits_shard)
    dt = _logits_dtype(logits_shard)
    ld = logits_shard.shape[1]
    V = ld if V is None else int(V)
    assert 1 <= V <= ld
    if row_end is None:
        row_end = row_offset + logits_shard.shape[0]
    assert row_begin >= row_offset and row_end - row_offset <= logits_shard.shape[0]
    a = _c(actions, np.int32)
    n = row_end - row_begin
    m, s, za = np.empty(n, np.float64), np.empty(n, np.float64), np.empty(n, np.float64)
    base = logits_shard.ctypes.data - row_offset * ld * logits_shard.itemsize
    lib.oracle_vocab_shard_stats(ctypes.c_void_p(base), dt, V, ld, int(v_begin), _ptr(a), row_begin, row_end,
                                 _ptr(m), _ptr(s), _ptr(za))
    return ShardStats(m, s, za)


def vocab_merge(stats: list) -> tuple[np.ndarray, np.ndarray]:
    """Merges the shards' statistics of the same rows into each row's (log-sum-exp, action logit):
    lse = M + log sum_g s_g exp(m_g - M) with M = max_g m_g, and z_a = max_g z_a_g (only the owner's is finite)."""
    m = np.stack([x.m for x in stats])
    M = m.max(axis=0)
    with np.errstate(invalid="ignore"):
        w = np.where(m == -np.inf, 0.0, np.exp(m - M))
    S = (np.stack([x.s for x in stats]) * w).sum(axis=0)
    with np.errstate(divide="ignore"):
        lse = M + np.log(S)
    za = np.stack([x.za for x in stats]).max(axis=0)
    return lse, za

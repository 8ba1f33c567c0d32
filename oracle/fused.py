"""fp64 oracle for the fused LM-head form of the GRPO loss.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The fused form takes the final hidden states h [T, H] and the LM-head weight
W [H, V] instead of the logits.  By definition the logits are z = h W; the loss
and dlogits D = dloss/dz are then exactly those of the logits form (Eq. 1 with
the dual clip of Eq. 2), and by the chain rule through the product
    dloss/dh = D W^T        dloss/dW = h^T D.
Each step is written as that definition: numpy's float64 matmul is the library
primitive for the three products, and the per-row loss is the C oracle.  The
vocabulary chunking the GPU kernel uses is an implementation detail and does
not appear here.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import LossResult, Segments, loss_rows


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def as_f64(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) or float arrays, widened exactly to float64."""
    x = np.asarray(x)
    return bf16_bits_to_f64(x) if x.dtype == np.uint16 else x.astype(np.float64)


@dataclass
class FusedResult:
    loss: float
    rows: LossResult          # per-token outputs and D = dloss/dz (fp64)
    dhidden: np.ndarray       # [rows, H] fp64
    dW: np.ndarray | None     # [H, V]    fp64 (None when only a row sample is computed)


def fused_loss(hidden_bits: np.ndarray, w_bits: np.ndarray, actions, behave_logp, prox_logp, adv,
               seg: Segments, group_size: int, **params) -> FusedResult:
    """All rows: loss, dhidden = D W^T and dW = h^T D, in fp64."""
    h = as_f64(hidden_bits)
    W = as_f64(w_bits)
    z = h @ W
    res = loss_rows(z, actions, behave_logp, prox_logp, adv, seg, group_size, **params)
    D = res.dlogits
    return FusedResult(res.loss, res, D @ W.T, h.T @ D)


def fused_rows(hidden_bits: np.ndarray, w_bits: np.ndarray, rows, actions, behave_logp, prox_logp, adv,
               seg: Segments, group_size: int, w_f64: np.ndarray | None = None, **params) -> FusedResult:
    """A sample of token rows: per-token outputs and their dhidden rows.

    ``rows`` lists absolute token numbers; hidden_bits holds all T rows.  The
    loss field sums only the sampled rows.  dW needs every row and is None.
    """
    W = as_f64(w_bits) if w_f64 is None else w_f64
    rows = np.asarray(rows, dtype=np.int64)
    out_logp, out_contrib, out_g, out_state, out_D, dh = [], [], [], [], [], []
    flags = 0
    for t in rows:
        z = as_f64(hidden_bits[t:t + 1]) @ W
        r = loss_rows(z, actions, behave_logp, prox_logp, adv, seg, group_size, row_begin=int(t),
                      row_end=int(t) + 1, row_offset=int(t), **params)
        flags |= r.flags
        out_logp.append(r.token_logp[0]); out_contrib.append(r.token_contrib[0]); out_g.append(r.token_g[0])
        out_state.append(r.token_state[0]); out_D.append(r.dlogits[0]); dh.append(r.dlogits[0] @ W.T)
    res = LossResult(float(np.sum(out_contrib)), np.zeros(0), np.array(out_logp), np.array(out_contrib),
                     np.array(out_g), np.array(out_state, np.int32), np.array(out_D), flags)
    return FusedResult(res.loss, res, np.array(dh), None)

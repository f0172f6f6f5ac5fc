"""CPU oracle for the training-side gather-scatter and the router's
straight-through estimator.  TEST INFRASTRUCTURE.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this module.  It shares no code with the HIP library.  Plain
numpy; floating point in float64.

What it follows (Section 3.2 and Appendix B):
  * Active set of loop i: token t takes part in loop i exactly when its depth
    m_t is at least i (no index offset).  The tokens of a batch of B sequences
    of T tokens are the rows b*T + t of one [B*T, d] tensor; the active rows
    are listed in increasing row order, which keeps every sequence contiguous
    and each sequence's tokens in causal order (Eq. 6 asks for the gathered
    tensor to keep the order of the sequence).
  * Gather (Eq. 6): the compact tensor holds the active rows of H, in that
    order.
  * Scatter (Eq. 7): an active row of the result is the block output for it
    plus the row's previous state; every other row keeps its previous state.
  * Backward: both maps are linear.  The gradient of the scatter passes the
    incoming gradient unchanged to the previous state (both cases of Eq. 7
    carry it with weight one) and hands the gradient of the active rows to
    the block output; the gradient of the gather adds the compact gradient
    into the rows it was read from.
  * Straight-through estimator (Appendix B): its value is the depth m itself
    and its derivative with respect to the score s is that of the logistic
    sigmoid, sigma(s) (1 - sigma(s)).
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def active_rows(depth: np.ndarray, loop: int) -> np.ndarray:
    """Increasing row indices r with depth[r] >= loop (Section 3.2 active set)."""
    depth = np.asarray(depth).reshape(-1)
    return np.flatnonzero(depth >= loop).astype(np.int64)


def sequence_offsets(depth: np.ndarray, seq_len: int, loop: int) -> np.ndarray:
    """Start of each sequence's run in the compact tensor, plus the total
    (batch + 1 entries); sequence b owns rows [b*seq_len, (b+1)*seq_len)."""
    depth = np.asarray(depth).reshape(-1)
    if seq_len <= 0:
        return np.zeros(1, np.int64)
    per_seq = (depth.reshape(-1, seq_len) >= loop).sum(axis=1)
    return np.concatenate([[0], np.cumsum(per_seq)]).astype(np.int64)


def compact_slot(depth: np.ndarray, loop: int) -> np.ndarray:
    """Row -> its index in the compact tensor, -1 for a row not in the loop."""
    depth = np.asarray(depth).reshape(-1)
    slot = np.full(depth.shape[0], -1, np.int64)
    idx = active_rows(depth, loop)
    slot[idx] = np.arange(idx.shape[0])
    return slot


def gather(H: np.ndarray, index: np.ndarray) -> np.ndarray:
    """Eq. 6: the compact tensor H[index]."""
    return np.asarray(H, np.float64)[np.asarray(index, np.int64)]


def scatter(H_prev: np.ndarray, Y: np.ndarray, index: np.ndarray) -> np.ndarray:
    """Eq. 7: active rows get Y + H_prev, the others keep H_prev."""
    out = np.array(H_prev, np.float64, copy=True)
    index = np.asarray(index, np.int64)
    out[index] = np.asarray(Y, np.float64) + out[index]
    return out


def scatter_backward(dH: np.ndarray, index: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Gradients of Eq. 7 given dL/dH^(i): (dL/dH^(i-1), dL/dY)."""
    dH = np.asarray(dH, np.float64)
    return dH.copy(), dH[np.asarray(index, np.int64)]


def gather_backward(dX: np.ndarray, index: np.ndarray, rows: int) -> np.ndarray:
    """Gradient of Eq. 6 given dL/dH~: the compact gradient added into the
    rows it was gathered from (each active row appears once)."""
    dX = np.asarray(dX, np.float64)
    out = np.zeros((rows,) + dX.shape[1:], np.float64)
    out[np.asarray(index, np.int64)] += dX
    return out


def sigmoid(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, np.float64)
    return 1.0 / (1.0 + np.exp(-s))


def ste_value(depth: np.ndarray) -> np.ndarray:
    """Appendix B: m + sigma(s) - sg(sigma(s)) has the value m."""
    return np.asarray(depth, np.float64)


def ste_grad(score: np.ndarray, grad_value: np.ndarray) -> np.ndarray:
    """Appendix B: only sigma(s) carries a gradient, so dL/ds = dL/dm * sigma'(s).
    sigma'(s) = sigma(s) (1 - sigma(s)), evaluated as exp(-|s|) / (1 + exp(-|s|))^2
    (the same quantity, without the cancellation of 1 - sigma(s) at large |s|)."""
    t = np.exp(-np.abs(np.asarray(score, np.float64)))
    return np.asarray(grad_value, np.float64) * t / (1.0 + t) ** 2


def loop_forward(H0: np.ndarray, depth: np.ndarray, block, loops: int) -> np.ndarray:
    """Loops 1..loops of the training forward: gather, block on the compact
    rows, scatter (Section 3.2).  ``block(i, X)`` maps a compact tensor to the
    block output for it."""
    H = np.asarray(H0, np.float64)
    for i in range(1, loops + 1):
        idx = active_rows(depth, i)
        H = scatter(H, block(i, gather(H, idx)), idx)
    return H

"""Oracle of the layer's loss-side operators.  TEST INFRASTRUCTURE ONLY (see
the package docstring): nothing in the product path imports this module.

* Eq. 3, the balance term B = lambda * n * sum_i T_i G_i, and its gradient
  with respect to the gate probabilities.
* Eq. 2, the specification loss sum_i g_i L(y_hat, O_i), with the
  AggregateSpec operator of the appendix on the specification loss (the
  concatenated predictions of the chosen experts, one row per (token,
  choice)).

Readings taken here (each also stated where it is used):
B1 T_i is the fraction of the batch's assignments that the gate gives
   expert i, counted before capacity: counts[i] / (T k).  For k = 1 this is
   the fraction of tokens.  G_i is the mean over the batch's tokens of the
   softmax probability of expert i.
B2 T_i comes from an arg-top-k and has no gradient; dB/dp[t,i] is therefore
   the constant lambda n T_i / T for every token.
S1 L is the mean squared error over the d features of one prediction,
   L(y, o) = (1/d) sum_c (o_c - y_c)^2, and the batch loss is the mean over
   tokens of Eq. 2's per-sample sum.
S2 The sum in Eq. 2 runs over the chosen experts whose assignment was kept;
   a dropped assignment has no prediction, contributes nothing and gets no
   gradient (as in the forward pass, Section 4.1).  Its AggregateSpec row
   is zero.
S3 g_i is the combine weight of the choice (Algorithm 1's normalised score),
   the same value the cooperation loss's weighted sum uses.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from .moe_oracle import _f32, round_to, softmax

__all__ = ["balance_term", "aggregate_spec", "spec_loss"]


def balance_term(logits: np.ndarray, counts: np.ndarray, k: int,
                 lam: float) -> Tuple[float, np.ndarray]:
    """Eq. 3: B = lam * n * sum_i T_i * G_i over the n experts (B1), and the
    per-expert gradient coefficient c_i = dB/dp[t,i] = lam * n * T_i / T (B2).

    Returns (B, c as float32 values); B is left in float64."""
    T, n = logits.shape
    p = softmax(logits)                      # from the float32 logits, in float64
    G = p.sum(axis=0) / T                    # fraction of probability mass
    Tf = np.asarray(counts, dtype=np.float64) / (T * k)   # fraction of assignments
    B = lam * n * float((Tf * G).sum())
    c = lam * n * Tf / T
    return B, _f32(c).astype(np.float64)


def aggregate_spec(Y_disp: np.ndarray, dest_row: np.ndarray) -> np.ndarray:
    """AggregateSpec: the predictions of every (token, choice) pair,
    concatenated as rows t*k + j; row t*k + j is Y[dest_row[t,j]] when the
    assignment was kept and zero when it was dropped (S2)."""
    T, k = dest_row.shape
    out = np.zeros((T * k, Y_disp.shape[1]))
    for t in range(T):
        for j in range(k):
            r = dest_row[t, j]
            if r >= 0:
                out[t * k + j] = Y_disp[r]
    return out


def spec_loss(Y_disp: np.ndarray, dest_row: np.ndarray, weights: np.ndarray,
              target: np.ndarray, dtype: str):
    """Eq. 2 with the squared-error task loss (S1-S3), and its gradients.

    loss            = (1/T) sum_t sum_{j kept} w[t,j] * L(target[t], O[t,j])
    dweights[t,j]   = (1/T) L(target[t], O[t,j])           (float32; 0 if dropped)
    dY[dest_row]    = w[t,j] * 2 (O[t,j] - target[t]) / (T d)   (rounded to dtype)

    Returns (loss in float64, dweights, dY_disp); rows of dY_disp with no
    kept assignment are NaN (never read)."""
    T, k = dest_row.shape
    d = Y_disp.shape[1]
    w = np.asarray(weights, dtype=np.float64)
    O = aggregate_spec(Y_disp, dest_row).reshape(T, k, d)
    kept = dest_row >= 0
    per = ((O - target[:, None, :]) ** 2).sum(axis=2) / d        # L per (t, j)
    per = np.where(kept, per, 0.0)
    loss = float((w * per).sum() / T)
    dw = per / T
    dY = np.full_like(Y_disp, np.nan)
    for j in range(k):
        sel = kept[:, j]
        r = dest_row[sel, j]
        dY[r] = round_to(w[sel, j, None] * 2.0 * (O[sel, j] - target[sel]) / (T * d), dtype)
    return loss, _f32(dw).astype(np.float64), dY

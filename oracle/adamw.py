"""The modified AdamW step of Section 5 as a plain float64 definition.

Notation: the weight W_p2 of the paper's math layout (rows in S) is stored
[out, in] as W (d x m), so the paper's rows are the stored COLUMNS; G is the
weight gradient, M and V the first and second moments, t the step count
(1 for the first step).

    M_t = beta1 M_{t-1} + (1 - beta1) G
    V_t = beta2 V_{t-1} + (1 - beta2) G^2
    M^  = M_t / (1 - beta1^t),   V^ = V_t / (1 - beta2^t)
    modified:  nu_c = mean over the d entries of column c of V^   (the paper's
               row-wise mean), alpha = 1 / (sqrt(nu_c) + eps) for every entry
               of column c
    standard:  alpha = 1 / (sqrt(V^) + eps) entry by entry
    W_{t+1} = W_t - lr alpha M^ - wd W_t

Readings: the bias corrections are the usual 1 / (1 - beta^t) (the printed
M_t / (beta_1 + eps) and V_t / (beta_2 + eps) are read as garbled); the decay
term is wd W_t as printed (no lr factor).  With the column-constant alpha, a
W whose columns lie in S stays there when every gradient's columns do.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def adamw_step(W, G, M, V, t: int, lr: float, beta1: float, beta2: float, eps: float,
               wd: float, subspace: bool = True):
    """One step; returns (W_new, M_new, V_new) in float64."""
    if t < 1:
        raise ValueError("t counts steps from 1")
    W, G, M, V = _f64(W), _f64(G), _f64(M), _f64(V)
    M1 = beta1 * M + (1.0 - beta1) * G
    V1 = beta2 * V + (1.0 - beta2) * G * G
    Mh = M1 / (1.0 - beta1 ** t)
    Vh = V1 / (1.0 - beta2 ** t)
    if subspace:
        nu = Vh.mean(axis=0, keepdims=True)          # one value per stored column
        alpha = 1.0 / (np.sqrt(nu) + eps)
    else:
        alpha = 1.0 / (np.sqrt(Vh) + eps)
    W1 = W - lr * alpha * Mh - wd * W
    return W1, M1, V1

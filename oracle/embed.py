"""The trainable low-rank token table of Section 4.3.1 as plain float64
definitions.

TE = T_fixed[t] + T_S[t] with T_S = T_fixed U U^T at the start of training
(Sec. 4.3.1).  T_S's rows stay in S when it is kept as coefficients,
T_S = C_S U^T with C_S (vocab x k) the trainable parameter (initially
T_fixed U), since every row of C_S U^T lies in Col(U):

* ``lowrank_forward``: X0[i] = P[pos_i] + T_fixed[tok_i] + C_S[tok_i] U^T, the
  embedding output PE + TE of Sec. 4.2 with the decomposed table;
* ``lowrank_grad``: the gradient of any loss with respect to C_S given its
  gradient dX0 with respect to X0: row v collects sum_{i: tok_i = v} dX0[i] U
  (the embedding lookup's scatter, with the chain rule through C_S U^T).

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

from .codec import _check_ids, _positions


def lowrank_init(E, U) -> np.ndarray:
    """C_S = T_fixed U, so that T_S = C_S U^T = T_fixed U U^T (Sec. 4.3.1)."""
    return np.asarray(E, dtype=np.float64) @ np.asarray(U, dtype=np.float64)


def lowrank_forward(CS, U, tok, E=None, P=None, pos=None, seq_len=None) -> np.ndarray:
    CS = np.asarray(CS, dtype=np.float64)
    U = np.asarray(U, dtype=np.float64)
    n = np.asarray(tok).shape[0]
    t = _check_ids(tok, n, CS.shape[0], "tok")
    X = CS[t] @ U.T
    if E is not None:
        X = X + np.asarray(E, dtype=np.float64)[t]
    if P is not None:
        X = X + np.asarray(P, dtype=np.float64)[_positions(n, pos, P, seq_len)]
    return X


def lowrank_grad(dX0, U, tok, vocab: int) -> np.ndarray:
    dX0 = np.asarray(dX0, dtype=np.float64)
    U = np.asarray(U, dtype=np.float64)
    t = _check_ids(tok, dX0.shape[0], vocab, "tok")
    g = np.zeros((vocab, U.shape[1]))
    np.add.at(g, t, dX0 @ U)
    return g

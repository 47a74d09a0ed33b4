"""The subspace update of Section 4.5 as plain float64 definitions.

Notation: G_t (N x d) is the activation gradient at the last compressed layer
in iteration t; U (d x k) spans the subspace S; K iterations are accumulated
between two updates.

* off-subspace residual  R_t = G_t (I - U U^T)                       (Sec. 4.5)
* Grassmann loss         L = (1/K) sum_t |R_t|_F^2                    (Sec. 4.5)
* accumulation matrix    S = (1/K) sum_t G_t^T G_t                    (Sec. 6, "Overhead of
                                                                       Grassmann updates")
* Euclidean gradient     dL/dU = -2 S U                               (Sec. 6)
* Riemannian gradient    T = dL/dU - U U^T dL/dU                      (Sec. 4.5)
* step and retraction    U_new = Q of the thin QR of U - eta T        (Sec. 4.5)

Readings where the paper is loose: the loss sums the K iterations of one
update interval and divides by K (the printed sum runs over K + 1 indices);
the thin QR is the one whose R has a positive diagonal, which makes Q unique
(the paper does not fix the column signs, and they do not change the
subspace).  U is used as stored: with a basis rounded to bf16, U^T U is not
exactly I and every formula above is evaluated with that U as written.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

_BLOCK = 4096


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def off_subspace_energy(G, U) -> float:
    """|G (I - U U^T)|_F^2: the squared norm of the gradient left outside S
    (Section 4.5).  Evaluated blockwise over rows as the definition reads:
    each row r of the residual is g_r - (g_r U) U^T."""
    G = np.asarray(G)
    U = _f64(U)
    total = 0.0
    for b0 in range(0, G.shape[0], _BLOCK):
        g = _f64(G[b0:b0 + _BLOCK])
        r = g - (g @ U) @ U.T
        total += float(np.sum(r * r))
    return total


def grassmann_loss(G_list, U) -> float:
    """L = (1/K) sum over the K accumulated iterations of |G_t (I - U U^T)|_F^2."""
    if not G_list:
        raise ValueError("no iterations accumulated")
    return sum(off_subspace_energy(G, U) for G in G_list) / len(G_list)


def accumulation_matrix(G_list) -> np.ndarray:
    """S = (1/K) sum_t G_t^T G_t  (d x d)."""
    if not G_list:
        raise ValueError("no iterations accumulated")
    d = np.asarray(G_list[0]).shape[1]
    S = np.zeros((d, d))
    for G in G_list:
        for b0 in range(0, np.asarray(G).shape[0], _BLOCK):
            g = _f64(np.asarray(G)[b0:b0 + _BLOCK])
            S += g.T @ g
    return S / len(G_list)


def accumulation_rows(G_list, rows) -> np.ndarray:
    """Selected rows of S: S[i, :] = (1/K) sum_t G_t[:, i]^T G_t, for checks at
    sizes where the full d x d matrix is too costly to form."""
    rows = np.asarray(rows, dtype=np.int64)
    d = np.asarray(G_list[0]).shape[1]
    out = np.zeros((rows.size, d))
    for G in G_list:
        G = np.asarray(G)
        for b0 in range(0, G.shape[0], _BLOCK):
            g = _f64(G[b0:b0 + _BLOCK])
            out += g[:, rows].T @ g
    return out / len(G_list)


def euclidean_gradient(S, U) -> np.ndarray:
    """dL/dU = -2 S U  (Section 6, from L = const - tr(U^T S U))."""
    return -2.0 * (_f64(S) @ _f64(U))


def riemannian_gradient(egrad, U) -> np.ndarray:
    """Projection onto the tangent space at U: egrad - U U^T egrad  (Section 4.5)."""
    U = _f64(U)
    egrad = _f64(egrad)
    return egrad - U @ (U.T @ egrad)


def qr_retract(A) -> np.ndarray:
    """Q of the thin QR A = Q R with diag(R) > 0 (Householder QR from LAPACK,
    then each column's sign fixed by the sign of R's diagonal)."""
    A = _f64(A)
    Q, R = np.linalg.qr(A, mode="reduced")
    dg = np.diag(R)
    if np.any(dg == 0) or not np.all(np.isfinite(dg)):
        raise np.linalg.LinAlgError("rank-deficient step: R has a zero diagonal")
    return Q * np.sign(dg)[None, :]


def grassmann_step(U, S, eta) -> np.ndarray:
    """One update of Section 4.5: Riemannian gradient of L at U, a step of size
    eta against it, and the QR retraction back onto the manifold."""
    U = _f64(U)
    T = riemannian_gradient(euclidean_gradient(S, U), U)
    return qr_retract(U - float(eta) * T)

"""Exact rational versions of the codec's operations for tiny inputs.

Pure-Python loops over ``fractions.Fraction``: no rounding anywhere, so these
give the true value of each definition (Section 4.3.1 Eq. "subtract" and the
recovery formula, Section 4.4 Eq. "grad_compress", and the projection U(U^T W)).
Only for inputs of a few dozen elements.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

from fractions import Fraction


def _F(v):
    return v if isinstance(v, Fraction) else Fraction(v)


def _mat(a):
    return [[_F(v) for v in row] for row in a]


def compress(X, U, tok=None, E=None, P=None, pos=None):
    X, U = _mat(X), _mat(U)
    E = _mat(E) if E is not None else None
    P = _mat(P) if P is not None else None
    d, k = len(U), len(U[0])
    out = []
    for i, row in enumerate(X):
        xhat = list(row)
        for r in range(d):
            if E is not None:
                xhat[r] -= E[tok[i]][r]
            if P is not None:
                xhat[r] -= P[pos[i]][r]
        out.append([sum((xhat[r] * U[r][j] for r in range(d)), Fraction(0)) for j in range(k)])
    return out


def decompress(C, U, tok=None, E=None, P=None, pos=None):
    C, U = _mat(C), _mat(U)
    E = _mat(E) if E is not None else None
    P = _mat(P) if P is not None else None
    d, k = len(U), len(U[0])
    out = []
    for i, row in enumerate(C):
        x = []
        for r in range(d):
            v = sum((row[j] * U[r][j] for j in range(k)), Fraction(0))
            if E is not None:
                v += E[tok[i]][r]
            if P is not None:
                v += P[pos[i]][r]
            x.append(v)
        out.append(x)
    return out


def project_weights(W, U):
    W, U = _mat(W), _mat(U)
    d, k, m = len(U), len(U[0]), len(W[0])
    T = [[sum((U[r][j] * W[r][c] for r in range(d)), Fraction(0)) for c in range(m)]
         for j in range(k)]
    return [[sum((U[r][j] * T[j][c] for j in range(k)), Fraction(0)) for c in range(m)]
            for r in range(d)]

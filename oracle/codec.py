"""The codec's operations as plain float64 definitions.

Notation (Sections 3-4): X is the stage output, one row per token (N x d);
U (d x k) has orthonormal columns spanning the subspace S; T_fixed (here
``E``, vocab x d) is the fixed high-rank token table; P (n_pos x d) the
positional table; tok / pos the token and position index of each row.

Inputs may be any float arrays (bf16 inputs are decoded by the caller with
``decode_bf16``); they are up-converted to float64 exactly and every sum is
taken in float64.  Results are returned unrounded; ``round_to`` applies the
single final rounding.  Work is done in blocks of rows only to bound memory:
each row's result is the same definition whatever the block.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

_BLOCK = 2048


def default_positions(n: int, seq_len: int) -> np.ndarray:
    """Position of row i in a row-major [batch, seq_len] layout: i mod seq_len.

    The paper indexes positions p_1..p_n per sequence (Section 4.2); with a
    batch flattened row-major the position of flat row i is i mod seq_len.
    """
    if seq_len <= 0:
        raise ValueError("seq_len must be positive")
    return np.arange(n, dtype=np.int64) % seq_len


def _check_ids(idx: np.ndarray, n_rows: int, table_rows: int, what: str) -> np.ndarray:
    idx = np.asarray(idx).astype(np.int64)
    if idx.shape != (n_rows,):
        raise ValueError(f"{what}: expected shape ({n_rows},), got {idx.shape}")
    if n_rows and (idx.min() < 0 or idx.max() >= table_rows):
        raise IndexError(f"{what}: index out of range [0, {table_rows})")
    return idx


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def _positions(n, pos, P, seq_len):
    if pos is None:
        if seq_len is None:
            raise ValueError("P given without pos or seq_len")
        p = default_positions(n, seq_len)
        if p.size and p.max() >= P.shape[0]:
            raise IndexError("pos: default position past the end of P")
        return p
    return _check_ids(pos, n, P.shape[0], "pos")


def _embedding_terms(n, rows, tok, E, pos, P, seq_len):
    """The terms the receiver can rebuild from ids, for the given rows:
    (P[pos[i]] or None, T_fixed[tok[i]] or None)."""
    pe = te = None
    if P is not None:
        pe = _f64(np.asarray(P)[_positions(n, pos, P, seq_len)[rows]])
    if E is not None:
        te = _f64(np.asarray(E)[_check_ids(tok, n, E.shape[0], "tok")[rows]])
    return pe, te


def _rows(n: int, rows) -> np.ndarray:
    return np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)


def compress(X, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
    """C = (X - P[pos] - T_fixed[tok]) U   (Section 4.3.1, Eq. "subtract").

    With E and P both None this is the plain projection X U used for the
    gradient path.  ``rows`` restricts the computation to selected rows.
    """
    X = np.asarray(X)
    U = _f64(U)
    n, d = X.shape
    if U.shape[0] != d:
        raise ValueError("U must be d x k")
    sel = _rows(n, rows)
    C = np.empty((sel.size, U.shape[1]), dtype=np.float64)
    for b0 in range(0, sel.size, _BLOCK):
        r = sel[b0:b0 + _BLOCK]
        xhat = _f64(X[r])
        pe, te = _embedding_terms(n, r, tok, E, pos, P, seq_len)
        if pe is not None:
            xhat = xhat - pe
        if te is not None:
            xhat = xhat - te
        C[b0:b0 + r.size] = xhat @ U
    return C


def decompress(C, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
    """X_rec = C U^T + P[pos] + T_fixed[tok]   (Section 4.3.1, recovery at the next stage).

    With E and P both None this is the gradient recovery C_g U^T (Section 4.4).
    """
    C = np.asarray(C)
    U = _f64(U)
    n, k = C.shape
    if U.shape[1] != k:
        raise ValueError("U must be d x k")
    sel = _rows(n, rows)
    out = np.empty((sel.size, U.shape[0]), dtype=np.float64)
    for b0 in range(0, sel.size, _BLOCK):
        r = sel[b0:b0 + _BLOCK]
        x = _f64(C[r]) @ U.T
        pe, te = _embedding_terms(n, r, tok, E, pos, P, seq_len)
        if pe is not None:
            x = x + pe
        if te is not None:
            x = x + te
        out[b0:b0 + r.size] = x
    return out


def grad_compress(G, U, rows=None):
    """C_g = G U   (Section 4.4, Eq. "grad_compress"): no embedding terms."""
    return compress(G, U, rows=rows)


def grad_decompress(Cg, U, rows=None):
    """G_rec = C_g U^T   (Section 4.4).  Equals G only for G in span(U) rows;
    for any G it is G U U^T, which preserves every upstream parameter gradient
    because the projection matrices' rows lie in S (Appendix A)."""
    return decompress(Cg, U, rows=rows)


def project_weights(W, U, cols=None):
    """W' = U (U^T W): the Euclidean projection Pi_S of every column of W
    (stored [out, in] = d x m) onto S = Col(U)  (Sections 4.3 and 5, Appendix E).

    In the paper's math layout W_p in R^{m x d} acts from the right (X W_p), and
    "Row(W_p) in S" is this column projection of the stored d x m matrix.
    ``cols`` restricts the computation to selected columns (each column is
    projected independently).
    """
    W = np.asarray(W)
    U = _f64(U)
    if U.shape[0] != W.shape[0]:
        raise ValueError("W must have d rows")
    Wc = _f64(W if cols is None else W[:, np.asarray(cols, dtype=np.int64)])
    T = U.T @ Wc
    return U @ T

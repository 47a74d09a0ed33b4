"""Pins for the codec oracle (no GPU).

Each check rests on a fact the paper or plain linear algebra fixes, not on
re-running the oracle's own formula:

* the closed form of Section 4.3: for X = E[tok] + P[pos] + C U^T (U with
  orthonormal columns) compression returns C exactly and recovery returns X;
* the off-subspace residual: with X - E - P = C U^T + eta, eta orthogonal to
  S, the reconstruction error equals |eta| and |X^|^2 = |C|^2 + |eta|^2;
* gradients (Section 4.4): round trip exact inside S, error^2 = |G|^2 - |GU|^2;
* projection (Appendix E): U^T W' = U^T W, (I - UU^T) W' = 0, idempotent,
  non-expansive;
* special cases that need no matmul: U = columns of the identity (selection),
  U = a signed permutation, k = d;
* exact rational arithmetic on tiny inputs, and a stored exact fixture.

The mutation test at the end plants plausible mistakes in copies of the
oracle and checks that these pins catch every one of them.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import exact
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_exact.json")


def _tiny(seed=0, n=37, d=24, k=5, vocab=11, seq=7, noise=0.0):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.standard_normal((vocab, d)) * 0.3
    P = rng.standard_normal((seq, d)) * 0.2
    tok = rng.integers(0, vocab, n)
    pos = np.arange(n) % seq
    C = rng.standard_normal((n, k))
    eta = rng.standard_normal((n, d)) * noise
    eta -= (eta @ U) @ U.T
    X = E[tok] + P[pos] + C @ U.T + eta
    return dict(U=U, E=E, P=P, tok=tok, pos=pos, C=C, eta=eta, X=X, seq=seq)


# ---------------------------------------------------------------- basis (P1)

@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_generated_basis_orthonormal(cfg):
    b = synth.make_basis(cfg)
    U64 = b["U64"]
    k = U64.shape[1]
    assert np.abs(U64.T @ U64 - np.eye(k)).max() < 1e-12
    Us = synth.as_float(b["U"], synth.CONFIGS[cfg].dtype).astype(np.float64)
    tol = 1e-6 if synth.CONFIGS[cfg].dtype == "f32" else 2e-3
    assert np.abs(Us.T @ Us - np.eye(k)).max() < tol
    Pm = U64 @ U64.T
    assert np.abs(Pm @ Pm - Pm).max() < 1e-12


# ---------------------------------------------------------- closed form (P2)

def test_compress_recovers_coefficients_exactly():
    t = _tiny()
    C = oracle.compress(t["X"], t["U"], t["tok"], t["E"], t["P"], t["pos"])
    assert np.abs(C - t["C"]).max() < 1e-12
    X2 = oracle.decompress(C, t["U"], t["tok"], t["E"], t["P"], t["pos"])
    assert np.abs(X2 - t["X"]).max() < 1e-12


def test_default_positions_match_explicit():
    t = _tiny()
    C1 = oracle.compress(t["X"], t["U"], t["tok"], t["E"], t["P"], seq_len=t["seq"])
    assert np.abs(C1 - t["C"]).max() < 1e-12
    assert np.array_equal(oracle.default_positions(9, 4), [0, 1, 2, 3, 0, 1, 2, 3, 0])


def test_reconstruction_error_is_off_subspace_residual():
    t = _tiny(noise=0.05)
    C = oracle.compress(t["X"], t["U"], t["tok"], t["E"], t["P"], t["pos"])
    assert np.abs(C - t["C"]).max() < 1e-12          # noise is invisible to C
    Xr = oracle.decompress(C, t["U"], t["tok"], t["E"], t["P"], t["pos"])
    err = np.linalg.norm(Xr - t["X"])
    assert err > 0.1
    assert abs(err - np.linalg.norm(t["eta"])) < 1e-10
    # Pythagoras per row: |x^|^2 = |c|^2 + |eta|^2
    xhat = t["X"] - t["E"][t["tok"]] - t["P"][t["pos"]]
    lhs = np.sum(xhat ** 2, axis=1)
    rhs = np.sum(C ** 2, axis=1) + np.sum(t["eta"] ** 2, axis=1)
    assert np.abs(lhs - rhs).max() < 1e-10


def test_generated_workload_closed_form():
    w = synth.make_workload(0, sigma=0.0)
    cfg = w["cfg"]
    X = synth.as_float(w["X"], cfg.dtype)
    U = synth.as_float(w["U"], cfg.dtype)
    E = synth.as_float(w["E"], cfg.dtype)
    P = synth.as_float(w["P"], cfg.dtype)
    C = oracle.compress(X, U, w["tok"], E, P, seq_len=cfg.seq)
    # X and U were rounded to float32: the recovery is exact up to that rounding
    assert np.abs(C - w["C_true"]).max() < 1e-4
    w1 = synth.make_workload(0)
    X1 = synth.as_float(w1["X"], cfg.dtype)
    Xr = oracle.decompress(oracle.compress(X1, U, w1["tok"], E, P, seq_len=cfg.seq),
                           U, w1["tok"], E, P, seq_len=cfg.seq)
    err = np.linalg.norm(Xr - X1)
    assert abs(err - w1["noise_norm"]) < 1e-3 * w1["noise_norm"] + 1e-4


# ------------------------------------------------------------ gradients (P4)

def test_gradient_round_trip():
    rng = np.random.default_rng(3)
    U, _ = np.linalg.qr(rng.standard_normal((32, 6)))
    Gin = rng.standard_normal((10, 6)) @ U.T              # rows inside S
    Cg = oracle.grad_compress(Gin, U)
    assert np.abs(oracle.grad_decompress(Cg, U) - Gin).max() < 1e-12
    G = rng.standard_normal((10, 32))
    Cg = oracle.grad_compress(G, U)
    Gr = oracle.grad_decompress(Cg, U)
    assert abs(np.sum((G - Gr) ** 2) - (np.sum(G ** 2) - np.sum(Cg ** 2))) < 1e-10
    # the lossless claim of Appendix A: for W_p2 with rows in S,
    # (G U U^T) W_p2^T == G W_p2^T
    Wp2 = rng.standard_normal((20, 6)) @ U.T              # d_ff x d, Row(W_p2) in S
    assert np.abs(Gr @ Wp2.T - G @ Wp2.T).max() < 1e-10


# ----------------------------------------------------------- projection (P5)

def test_projection_invariants():
    rng = np.random.default_rng(4)
    d, k, m = 40, 7, 23
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    W = rng.standard_normal((d, m))
    Wp = oracle.project_weights(W, U)
    assert np.abs(U.T @ Wp - U.T @ W).max() < 1e-12
    assert np.abs(Wp - U @ (U.T @ Wp)).max() < 1e-12          # (I - UU^T) W' = 0
    assert np.abs(oracle.project_weights(Wp, U) - Wp).max() < 1e-12
    assert np.linalg.norm(Wp) <= np.linalg.norm(W)
    # Pythagoras: |W|^2 = |W'|^2 + |W - W'|^2
    assert abs(np.sum(W ** 2) - np.sum(Wp ** 2) - np.sum((W - Wp) ** 2)) < 1e-9
    # column independence and column sampling
    cols = [3, 0, 22]
    assert np.abs(oracle.project_weights(W, U, cols=cols) - Wp[:, cols]).max() < 1e-13


def test_projection_is_row_space_confinement():
    """In math layout W_p (m x d) acts as X W_p; W_p = W^T. Confining Row(W_p)
    to S means W_p = W_p U U^T, i.e. the stored W is projected column-wise."""
    rng = np.random.default_rng(5)
    U, _ = np.linalg.qr(rng.standard_normal((16, 3)))
    W = rng.standard_normal((16, 16))
    Wp_math = W.T
    confined = oracle.project_weights(W, U).T
    assert np.abs(confined - confined @ U @ U.T).max() < 1e-12
    # activations produced by a confined projection matrix lie in S
    Xh = rng.standard_normal((5, 16)) @ confined
    assert np.abs(Xh - Xh @ U @ U.T).max() < 1e-12
    assert np.abs(Wp_math - Wp_math @ U @ U.T).max() > 1e-3   # the unconfined one does not


# -------------------------------------------------------- special cases (P8)

def test_identity_columns_select_coordinates():
    t = _tiny(d=12, k=4)
    for name in ("X", "E", "P"):          # a 1/64 grid: every sum below is exact
        t[name] = np.round(t[name] * 64) / 64
    sel = np.array([2, 7, 0, 11])
    U = np.zeros((12, 4))
    U[sel, np.arange(4)] = 1.0
    C = oracle.compress(t["X"], U, t["tok"], t["E"], t["P"], t["pos"])
    xhat = t["X"] - t["E"][t["tok"]] - t["P"][t["pos"]]
    assert np.array_equal(C, xhat[:, sel])
    # signed permutation columns
    U2 = U.copy()
    U2[:, 1] *= -1
    C2 = oracle.compress(t["X"], U2, t["tok"], t["E"], t["P"], t["pos"])
    assert np.array_equal(C2[:, 1], -xhat[:, sel[1]])
    # decompress scatters coefficients back onto those coordinates
    Xr = oracle.decompress(C, U, t["tok"], t["E"], t["P"], t["pos"])
    emb = t["E"][t["tok"]] + t["P"][t["pos"]]
    assert np.array_equal(Xr[:, sel], emb[:, sel] + C)
    rest = np.setdiff1d(np.arange(12), sel)
    assert np.array_equal(Xr[:, rest], emb[:, rest])


def test_full_rank_basis_is_identity_round_trip():
    rng = np.random.default_rng(6)
    d = 16
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    X = rng.standard_normal((9, d))
    assert np.abs(oracle.decompress(oracle.compress(X, Q), Q) - X).max() < 1e-12


def test_embedding_only_rows():
    """decompress with C = 0 returns the gathered rows themselves."""
    rng = np.random.default_rng(7)
    E = rng.standard_normal((6, 8))
    P = rng.standard_normal((3, 8))
    U, _ = np.linalg.qr(rng.standard_normal((8, 2)))
    tok = np.array([5, 0, 5, 2])
    pos = np.array([2, 2, 0, 1])
    Z = np.zeros((4, 2))
    assert np.array_equal(oracle.decompress(Z, U, tok, E), E[tok])
    assert np.array_equal(oracle.decompress(Z, U, pos=pos, P=P), P[pos])


def test_empty_and_bad_ids():
    U = np.eye(4)[:, :2]
    assert oracle.compress(np.zeros((0, 4)), U).shape == (0, 2)
    assert oracle.decompress(np.zeros((0, 2)), U).shape == (0, 4)
    E = np.zeros((3, 4))
    with pytest.raises(IndexError):
        oracle.compress(np.zeros((2, 4)), U, tok=np.array([0, 3]), E=E)
    with pytest.raises(IndexError):
        oracle.compress(np.zeros((2, 4)), U, tok=np.array([-1, 0]), E=E)
    with pytest.raises(IndexError):
        oracle.compress(np.zeros((2, 4)), U, P=E, pos=np.array([0, 5]))
    with pytest.raises(IndexError):   # default positions past the table
        oracle.compress(np.zeros((5, 4)), U, P=E, seq_len=4)


def test_row_sampling_matches_full():
    t = _tiny(n=3000, d=16, k=3)   # spans more than one internal block
    full = oracle.compress(t["X"], t["U"], t["tok"], t["E"], t["P"], t["pos"])
    rows = [2999, 0, 2048, 2047, 1]
    part = oracle.compress(t["X"], t["U"], t["tok"], t["E"], t["P"], t["pos"], rows=rows)
    assert np.array_equal(part, full[rows])
    Xr = oracle.decompress(full, t["U"], t["tok"], t["E"], t["P"], t["pos"])
    Xp = oracle.decompress(full, t["U"], t["tok"], t["E"], t["P"], t["pos"], rows=rows)
    assert np.array_equal(Xp, Xr[rows])


# ---------------------------------------------------- exact arithmetic (P9)

def _rational(rng, shape, den=16, lim=20):
    return [[Fraction(int(rng.integers(-lim, lim + 1)), den) for _ in range(shape[1])]
            for _ in range(shape[0])]


def test_fp64_oracle_equals_exact_on_tiny_inputs():
    rng = np.random.default_rng(8)
    d, k, n, vocab, npos = 8, 3, 4, 5, 3
    # rational orthonormal columns: a 3-4-5 rotation and Hadamard-like halves
    U = [[Fraction(3, 5), 0, Fraction(4, 15)], [Fraction(4, 5), 0, Fraction(-3, 15)],
         [0, Fraction(1, 2), 0], [0, Fraction(1, 2), 0], [0, Fraction(1, 2), 0],
         [0, Fraction(1, 2), 0], [0, 0, Fraction(2, 3)], [0, 0, Fraction(-2, 3)]]
    Uf = np.array([[float(v) for v in r] for r in U])
    assert all(sum(U[r][i] * U[r][j] for r in range(d)) == (i == j)
               for i in range(k) for j in range(k))
    X = _rational(rng, (n, d))
    E = _rational(rng, (vocab, d))
    P = _rational(rng, (npos, d))
    tok = [int(v) for v in rng.integers(0, vocab, n)]
    pos = [int(v) for v in rng.integers(0, npos, n)]
    f = lambda m: np.array([[float(v) for v in r] for r in m])  # noqa: E731
    Cx = f(exact.compress(X, U, tok, E, P, pos))
    Co = oracle.compress(f(X), Uf, tok, f(E), f(P), pos)
    assert np.abs(Co - Cx).max() <= 1e-15 * max(1.0, np.abs(Cx).max())
    Xx = f(exact.decompress(exact.compress(X, U, tok, E, P, pos), U, tok, E, P, pos))
    Xo = oracle.decompress(Co, Uf, tok, f(E), f(P), pos)
    assert np.abs(Xo - Xx).max() <= 1e-14
    W = _rational(rng, (d, 5))
    Wx = f(exact.project_weights(W, U))
    assert np.abs(oracle.project_weights(f(W), Uf) - Wx).max() <= 1e-15


def test_stored_exact_fixture():
    g = json.load(open(GOLDEN))
    f = lambda m: np.array([[float(Fraction(v)) for v in r] for r in m])  # noqa: E731
    U, E, P, X, G, W = (f(g[n]) for n in ("U", "E", "P", "X", "G", "W"))
    tok, pos = g["tok"], g["pos"]
    ex = {n: f(v) for n, v in g["expect"].items()}
    # the fixture's X was built with a known coefficient matrix
    assert np.array_equal(ex["C"], f(g["C_true"]))
    assert np.array_equal(oracle.compress(X, U, tok, E, P, pos), ex["C"])
    assert np.array_equal(oracle.decompress(ex["C"], U, tok, E, P, pos), ex["X_rec"])
    assert np.array_equal(oracle.grad_compress(G, U), ex["Cg"])
    assert np.array_equal(oracle.grad_decompress(ex["Cg"], U), ex["G_rec"])
    assert np.array_equal(oracle.project_weights(W, U), ex["W_proj"])
    # X is not in E + P + span(U): recovery drops exactly the off-subspace part
    assert not np.array_equal(ex["X_rec"], X)


# -------------------------------------------------- the pins have teeth

def _mutants():
    """Plausible mistakes, each a wrong version of one oracle function."""
    def comp_no_P(X, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
        return oracle.compress(X, U, tok, E, None, pos, seq_len, rows)

    def comp_plus_E(X, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
        return oracle.compress(X, U, tok, None if E is None else -E, P, pos, seq_len, rows)

    def comp_pos_for_tok(X, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
        return oracle.compress(X, U, pos, E, P, pos, seq_len, rows)

    def comp_transposed(X, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
        Q = np.linalg.qr(np.asarray(U) @ np.asarray(U).T)[0][:, :U.shape[1]]
        return oracle.compress(X, Q, tok, E, P, pos, seq_len, rows)

    def decomp_no_E(C, U, tok=None, E=None, P=None, pos=None, seq_len=None, rows=None):
        return oracle.decompress(C, U, tok, None, P, pos, seq_len, rows)

    def proj_rows(W, U, cols=None):
        W = np.asarray(W, dtype=np.float64)
        return W @ U @ U.T if W.shape[0] == W.shape[1] else oracle.project_weights(W, U, cols)

    def proj_T_only(W, U, cols=None):
        Wp = oracle.project_weights(W, U, cols)
        return Wp + 1e-3 * np.asarray(W, dtype=np.float64)

    return [("compress", comp_no_P), ("compress", comp_plus_E), ("compress", comp_pos_for_tok),
            ("compress", comp_transposed), ("decompress", decomp_no_E),
            ("project_weights", proj_rows), ("project_weights", proj_T_only)]


def _pin_suite(compress, decompress, project_weights):
    """The closed-form and invariant pins above, phrased over given functions.
    Returns the names of the pins that fail."""
    fails = []
    t = _tiny(seed=11, d=16, k=4, vocab=9, seq=5, noise=0.0)
    C = compress(t["X"], t["U"], t["tok"], t["E"], t["P"], t["pos"])
    if np.abs(C - t["C"]).max() > 1e-10:
        fails.append("compress closed form")
    Xr = decompress(t["C"], t["U"], t["tok"], t["E"], t["P"], t["pos"])
    if np.abs(Xr - t["X"]).max() > 1e-10:
        fails.append("decompress closed form")
    rng = np.random.default_rng(12)
    W = rng.standard_normal((16, 16))
    Wp = project_weights(W, t["U"])
    if (np.abs(t["U"].T @ Wp - t["U"].T @ W).max() > 1e-10
            or np.abs(Wp - t["U"] @ (t["U"].T @ Wp)).max() > 1e-10):
        fails.append("projection invariants")
    return fails


def test_pins_pass_on_oracle():
    assert _pin_suite(oracle.compress, oracle.decompress, oracle.project_weights) == []


@pytest.mark.parametrize("which,fn", _mutants(), ids=lambda v: getattr(v, "__name__", v))
def test_pins_catch_planted_mistake(which, fn):
    funcs = {"compress": oracle.compress, "decompress": oracle.decompress,
             "project_weights": oracle.project_weights}
    funcs[which] = fn
    assert _pin_suite(funcs["compress"], funcs["decompress"], funcs["project_weights"]) != []

"""Pins for the low-rank token table oracle (Section 4.3.1; no GPU).

* with C_S initialised to T_fixed U, compressing the embedding output
  X0 = P + T_fixed[t] + T_S[t] by Eq. "subtract" (the codec oracle, an
  independent function) returns exactly C_S[t]: T_S rides inside the
  coefficients, as the paper states;
* the gradient equals the dense route: scatter dX0's rows into a vocab x d
  table, then multiply by U (linearity, other order of operations);
* the gradient is the derivative of the forward: for L = <X0(C_S), R>,
  a central difference along a random direction of C_S equals <grad, D>;
* rows of T_S = C_S U^T lie in S; tokens that do not occur get a zero row.

The mutation test plants plausible mistakes and checks the pins catch each.
"""
import numpy as np
import pytest

import oracle
from oracle import embed as em


def _setup(seed=0, n=50, d=20, k=4, vocab=9, seq=6):
    rng = np.random.default_rng(seed)
    q, r = np.linalg.qr(rng.standard_normal((d, k)))
    U = q * np.sign(np.diag(r))
    E = rng.standard_normal((vocab, d))
    P = rng.standard_normal((seq, d))
    tok = rng.integers(0, vocab - 1, n)          # the last id never occurs
    return rng, U, E, P, tok, seq


def pin_rides_inside_c(fwd, grad):
    rng, U, E, P, tok, seq = _setup()
    CS = em.lowrank_init(E, U)
    X0 = fwd(CS, U, tok, E, P, seq_len=seq)
    C = oracle.compress(X0, U, tok, E, P, seq_len=seq)
    return np.abs(C - CS[tok]).max() <= 1e-12


def pin_dense_route(fwd, grad):
    rng, U, E, P, tok, seq = _setup(1)
    dX = rng.standard_normal((tok.size, U.shape[0]))
    dense = np.zeros((E.shape[0], U.shape[0]))
    for i, t in enumerate(tok):
        dense[t] += dX[i]
    g = grad(dX, U, tok, E.shape[0])
    return np.abs(g - dense @ U).max() <= 1e-12 and np.all(g[-1] == 0)


def pin_derivative(fwd, grad):
    rng, U, E, P, tok, seq = _setup(2)
    CS = rng.standard_normal((E.shape[0], U.shape[1]))
    R = rng.standard_normal((tok.size, U.shape[0]))
    D = rng.standard_normal(CS.shape)
    L = lambda c: float(np.sum(fwd(c, U, tok, E, P, seq_len=seq) * R))  # noqa: E731
    e = 1e-4
    fd = (L(CS + e * D) - L(CS - e * D)) / (2 * e)
    return abs(fd - float(np.sum(grad(R, U, tok, E.shape[0]) * D))) <= 1e-8 * max(1.0, abs(fd))


def pin_rows_in_s(fwd, grad):
    rng, U, E, P, tok, seq = _setup(3)
    CS = rng.standard_normal((E.shape[0], U.shape[1]))
    X0 = fwd(CS, U, tok)                           # no tables: the T_S rows alone
    return np.abs(X0 - X0 @ U @ U.T).max() <= 1e-12 and np.abs(X0 - CS[tok] @ U.T).max() <= 1e-12


PINS = [pin_rides_inside_c, pin_dense_route, pin_derivative, pin_rows_in_s]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    assert pin(em.lowrank_forward, em.lowrank_grad)


def _mutants():
    def fwd_no_fixed(CS, U, tok, E=None, P=None, pos=None, seq_len=None):
        return em.lowrank_forward(CS, U, tok, None, P, pos, seq_len)

    def fwd_transposed(CS, U, tok, E=None, P=None, pos=None, seq_len=None):
        U2 = np.linalg.qr(U @ U.T + np.eye(U.shape[0]) * 1e-3)[0][:, :U.shape[1]]
        return em.lowrank_forward(CS, U2, tok, E, P, pos, seq_len)

    def grad_unprojected(dX0, U, tok, vocab):
        g = np.zeros((vocab, U.shape[1]))
        np.add.at(g, tok, np.asarray(dX0)[:, :U.shape[1]])
        return g

    def grad_last_wins(dX0, U, tok, vocab):
        g = np.zeros((vocab, U.shape[1]))
        g[tok] = np.asarray(dX0) @ U               # assignment, not accumulation
        return g

    def grad_by_position(dX0, U, tok, vocab):
        return em.lowrank_grad(dX0, U, np.arange(len(tok)) % vocab, vocab)

    return [("fwd", fwd_no_fixed), ("fwd", fwd_transposed), ("grad", grad_unprojected),
            ("grad", grad_last_wins), ("grad", grad_by_position)]


@pytest.mark.parametrize("which,fn", _mutants(), ids=lambda v: getattr(v, "__name__", v))
def test_pins_catch_planted_mistake(which, fn):
    f = fn if which == "fwd" else em.lowrank_forward
    g = fn if which == "grad" else em.lowrank_grad
    assert not all(p(f, g) for p in PINS)

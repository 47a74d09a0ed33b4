"""Pins for the subspace-update oracle (Section 4.5 and Section 6; no GPU).

Every check rests on a fact the paper or linear algebra fixes, not on
re-running the oracle's own formula:

* the paper's trace expansion of the loss (Section 6): for orthonormal U,
  L = (1/K) sum_t |G_t|^2 - tr(U^T S U);
* gradients that lie in S leave nothing to correct: L = 0, a zero Riemannian
  gradient, and a step that returns U unchanged;
* the Riemannian gradient is the derivative of the loss along the manifold:
  a central difference of L along a retracted tangent
  curve U(e) = qf(U + e D) equals <T, D>;
* a small step decreases L, and repeated steps converge to the dominant
  k-dimensional eigenspace of S (the subspace an SVD of S would pick, which
  the paper's smooth updates approach);
* the retraction is the thin QR with diag(R) > 0 (A = Q R with Q^T A upper
  triangular, positive diagonal; span equal to A's, via the pseudo-inverse);
* k = 1 reduces the retraction to a normalisation; the updated subspace does
  not depend on the basis chosen for the current one (U -> U Q);
* averaging over K: repeating the same gradient K times changes nothing.

The mutation test at the end plants plausible mistakes in copies of the
oracle's functions and checks that these pins catch every one of them.
"""
import types

import numpy as np
import pytest

from oracle import grassmann as gr
import synth


def _orth(rng, d, k):
    q, r = np.linalg.qr(rng.standard_normal((d, k)))
    return q * np.sign(np.diag(r))


def _grads(rng, K=3, n=40, d=24, rank=3, scale=3.0):
    """K gradients with a few dominant directions (so S has an eigen-gap)."""
    V = _orth(rng, d, rank)
    out = []
    for _ in range(K):
        out.append(scale * rng.standard_normal((n, rank)) @ V.T + rng.standard_normal((n, d)))
    return out, V


def _proj(U):
    return U @ np.linalg.pinv(U)


def _ns():
    return types.SimpleNamespace(
        loss=gr.grassmann_loss, S=gr.accumulation_matrix, egrad=gr.euclidean_gradient,
        rgrad=gr.riemannian_gradient, retract=gr.qr_retract, step=gr.grassmann_step)


# ------------------------------------------------------------------ the pins

def pin_trace_expansion(f, rng):
    G, _ = _grads(rng)
    U = _orth(rng, 24, 5)
    S = f.S(G)
    expanded = np.mean([np.sum(g * g) for g in G]) - np.trace(U.T @ S @ U)
    return abs(f.loss(G, U) - expanded) <= 1e-10 * abs(expanded)


def pin_in_subspace(f, rng):
    U = _orth(rng, 24, 5)
    G = [rng.standard_normal((30, 5)) @ U.T for _ in range(3)]
    S = f.S(G)
    T = f.rgrad(f.egrad(S, U), U)
    U2 = f.step(U, S, 0.05)
    return (f.loss(G, U) <= 1e-18 * np.mean([np.sum(g * g) for g in G])
            and np.abs(T).max() <= 1e-12 * np.abs(S).max()
            and np.abs(U2 - U).max() <= 1e-12)


def pin_directional_derivative(f, rng):
    G, _ = _grads(rng)
    U = _orth(rng, 24, 5)
    S = f.S(G)
    T = f.rgrad(f.egrad(S, U), U)
    Z = rng.standard_normal(U.shape)
    D = Z - U @ (U.T @ Z)                     # a tangent direction at U
    e = 1e-5
    # the loss at retracted points (numpy's QR: column signs do not change L)
    def at(eps):
        return f.loss(G, np.linalg.qr(U + eps * D)[0])
    fd = (at(e) - at(-e)) / (2 * e)
    return abs(fd - np.sum(T * D)) <= 1e-6 * abs(np.sum(T * D))


def pin_descent(f, rng):
    G, _ = _grads(rng)
    U = _orth(rng, 24, 5)
    S = f.S(G)
    eta = 0.1 / np.linalg.eigvalsh(S)[-1]
    return f.loss(G, f.step(U, S, eta)) < f.loss(G, U)


def pin_dominant_eigenspace(f, rng):
    G, _ = _grads(rng, K=2, n=200, rank=5, scale=4.0)
    S = f.S(G)
    w, V = np.linalg.eigh(S)
    top = V[:, -5:]
    U = _orth(rng, 24, 5)
    eta = 0.5 / w[-1]
    for _ in range(300):
        U = f.step(U, S, eta)
    return np.abs(_proj(U) - top @ top.T).max() <= 1e-8


def pin_retraction(f, rng):
    A = rng.standard_normal((24, 5)) + 2.0 * np.eye(24, 5)
    Q = f.retract(A)
    R = Q.T @ A
    return (np.abs(Q.T @ Q - np.eye(5)).max() <= 1e-12
            and np.abs(np.tril(R, -1)).max() <= 1e-12
            and np.all(np.diag(R) > 0)
            and np.abs(Q @ R - A).max() <= 1e-12
            and np.abs(Q @ Q.T - _proj(A)).max() <= 1e-12)


def pin_k1(f, rng):
    G, _ = _grads(rng)
    u = _orth(rng, 24, 1)
    S = f.S(G)
    eta = 0.01
    g = -2.0 * S @ u
    t = g - u * float(u[:, 0] @ g[:, 0])
    v = u - eta * t
    return np.abs(f.step(u, S, eta) - v / np.linalg.norm(v)).max() <= 1e-12


def pin_rotation_invariance(f, rng):
    G, _ = _grads(rng)
    U = _orth(rng, 24, 5)
    Q = _orth(rng, 5, 5)
    S = f.S(G)
    eta = 0.2 / np.linalg.eigvalsh(S)[-1]
    return np.abs(_proj(f.step(U, S, eta)) - _proj(f.step(U @ Q, S, eta))).max() <= 1e-12


def pin_averaging(f, rng):
    G, _ = _grads(rng, K=1)
    U = _orth(rng, 24, 5)
    L1, L3 = f.loss(G, U), f.loss(G * 3, U)
    S1, S3 = f.S(G), f.S(G * 3)
    return abs(L1 - L3) <= 1e-12 * L1 and np.abs(S1 - S3).max() <= 1e-12 * np.abs(S1).max()


PINS = [pin_trace_expansion, pin_in_subspace, pin_directional_derivative, pin_descent,
        pin_dominant_eigenspace, pin_retraction, pin_k1, pin_rotation_invariance,
        pin_averaging]


def _pin_suite(f):
    """Names of the pins that fail for the functions in namespace f."""
    return [p.__name__ for p in PINS if not p(f, np.random.default_rng(7))]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    assert pin(_ns(), np.random.default_rng(7))


# --------------------------------------------------------- other properties

def test_accumulation_rows_are_rows_of_S():
    rng = np.random.default_rng(3)
    G, _ = _grads(rng)
    S = gr.accumulation_matrix(G)
    rows = [0, 5, 23]
    assert np.abs(gr.accumulation_rows(G, rows) - S[rows]).max() <= 1e-12 * np.abs(S).max()


def test_rank_deficient_step_raises():
    U = np.zeros((6, 2))
    U[0, 0] = 1.0
    with pytest.raises(np.linalg.LinAlgError):
        gr.qr_retract(U)


def test_stored_basis_used_as_written():
    """With a bf16-rounded basis U^T U != I; the loss is |G - (G U) U^T|^2 with
    that U, which differs from |G|^2 - |G U|^2 by tr((G U)(U^T U - I)(G U)^T)."""
    b = synth.make_basis(1)
    U = synth.as_float(b["U"], "bf16").astype(np.float64)
    rng = np.random.default_rng(5)
    G = rng.standard_normal((64, U.shape[0])) @ (U @ U.T) * 0.1 + 1e-3 * rng.standard_normal(
        (64, U.shape[0]))
    C = G @ U
    M = U.T @ U
    direct = gr.off_subspace_energy(G, U)
    via_gram = np.sum(G * G) - 2 * np.sum(C * C) + np.sum((C @ M) * C)
    assert abs(direct - via_gram) <= 1e-9 * np.sum(G * G)
    assert abs(direct - (np.sum(G * G) - np.sum(C * C))) > 1e-6 * direct


def test_input_generator_concentrates_energy():
    g = synth.make_grad_iteration(0, 0, n=512).astype(np.float64)
    V = synth.orthonormal_basis(synth.seed_of(0, synth.ORD_GV), 256, 8)
    share = np.sum((g @ V) ** 2) / np.sum(g * g)
    assert 0.4 < share < 0.6


# ---------------------------------------------------- the pins have teeth

def _mutants():
    def loss_no_projection(G, U):
        return np.mean([np.sum(np.asarray(g, dtype=np.float64) ** 2) for g in G])

    def loss_over_k_plus_1(G, U):
        return gr.grassmann_loss(G, U) * len(G) / (len(G) + 1)

    def S_sum_not_mean(G):
        return gr.accumulation_matrix(G) * len(G)

    def egrad_ascent(S, U):
        return -gr.euclidean_gradient(S, U)

    def egrad_no_factor2(S, U):
        return 0.5 * gr.euclidean_gradient(S, U)

    def egrad_transposed_product(S, U):
        return -2.0 * (np.asarray(S) @ np.asarray(S) @ np.asarray(U)) / max(1.0, np.abs(S).max())

    def rgrad_unprojected(eg, U):
        return np.asarray(eg, dtype=np.float64)

    def rgrad_wrong_side(eg, U):
        eg = np.asarray(eg, dtype=np.float64)
        return eg - (eg @ U.T) @ U if eg.shape[0] == eg.shape[1] else eg - eg @ (U.T @ U)

    def retract_no_sign_fix(A):
        return np.linalg.qr(np.asarray(A, dtype=np.float64), mode="reduced")[0]

    def retract_gram_schmidt_unnormalised(A):
        Q = gr.qr_retract(A)
        return Q * np.linalg.norm(np.asarray(A), axis=0)[None, :]

    out = []
    for name, fn in [("loss", loss_no_projection), ("loss", loss_over_k_plus_1),
                     ("S", S_sum_not_mean), ("egrad", egrad_ascent),
                     ("egrad", egrad_no_factor2), ("egrad", egrad_transposed_product),
                     ("rgrad", rgrad_unprojected), ("rgrad", rgrad_wrong_side),
                     ("retract", retract_no_sign_fix),
                     ("retract", retract_gram_schmidt_unnormalised)]:
        out.append((name, fn))
    return out


def _with(name, fn):
    f = _ns()
    setattr(f, name, fn)
    if name in ("egrad", "rgrad", "retract"):
        # the step composed from the (possibly wrong) parts, as the oracle composes it
        def step(U, S, eta, f=f):
            U = np.asarray(U, dtype=np.float64)
            return f.retract(U - eta * f.rgrad(f.egrad(S, U), U))
        f.step = step
    return f


def test_pins_pass_on_oracle():
    assert _pin_suite(_ns()) == []


def test_oracle_step_is_its_parts():
    rng = np.random.default_rng(9)
    G, _ = _grads(rng)
    U = _orth(rng, 24, 5)
    S = gr.accumulation_matrix(G)
    composed = _with("retract", gr.qr_retract).step(U, S, 0.01)
    assert np.abs(composed - gr.grassmann_step(U, S, 0.01)).max() <= 1e-14


@pytest.mark.parametrize("name,fn", _mutants(), ids=lambda v: getattr(v, "__name__", v))
def test_pins_catch_planted_mistake(name, fn):
    assert _pin_suite(_with(name, fn)) != []

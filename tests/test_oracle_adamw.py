"""Pins for the modified AdamW oracle (Section 5; no GPU).

* the property the modification exists for (Section 5, Appendix A): with
  every gradient's columns in S = Col(U) and W's columns in S, the modified
  step keeps W's columns in S exactly (the standard step does not);
* the standard step equals torch.optim.AdamW (float64, CPU) with the
  decoupled decay rescaled to the printed wd W term;
* when every column of V^ is constant the two steps coincide (library case);
* the first step from zero moments in closed form: W (1 - wd) - lr G / (rms of
  G's column + eps);
* a constant gradient: the bias corrections make every step exactly
  -lr g / (|g| + eps), from the first one on.

The mutation test plants plausible mistakes in copies of the oracle and
checks that these pins catch each one.
"""
import numpy as np
import pytest
import torch

from oracle import adamw as aw

HP = dict(lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8, wd=1e-3)


def _orth(rng, d, k):
    q, r = np.linalg.qr(rng.standard_normal((d, k)))
    return q * np.sign(np.diag(r))


def _run(step, W, Gs, subspace, **hp):
    M = np.zeros_like(W)
    V = np.zeros_like(W)
    for t, G in enumerate(Gs, start=1):
        W, M, V = step(W, G, M, V, t, subspace=subspace, **hp)
    return W, M, V


def pin_subspace_preserved(step, rng):
    d, k, m = 24, 4, 10
    U = _orth(rng, d, k)
    W = U @ rng.standard_normal((k, m))
    Gs = [U @ (rng.standard_normal((k, m)) * rng.uniform(0.1, 10, size=(1, m)))
          for _ in range(5)]
    Wn, _, _ = _run(step, W, Gs, True, **HP)
    Ws, _, _ = _run(step, W, Gs, False, **HP)
    off = lambda X: np.abs(X - U @ (U.T @ X)).max()  # noqa: E731
    return off(Wn) <= 1e-13 * np.abs(Wn).max() and off(Ws) > 1e-6 * np.abs(Ws).max()


def _torch_adamw(W, Gs, lr, beta1, beta2, eps, wd):
    p = torch.nn.Parameter(torch.from_numpy(W.copy()))
    opt = torch.optim.AdamW([p], lr=lr, betas=(beta1, beta2), eps=eps, weight_decay=wd / lr)
    for G in Gs:
        p.grad = torch.from_numpy(G.copy())
        opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def pin_standard_is_torch(step, rng):
    W = rng.standard_normal((12, 7))
    Gs = [rng.standard_normal((12, 7)) for _ in range(4)]
    got = _run(step, W, Gs, False, **HP)
    ref = _torch_adamw(W, Gs, **HP)
    return all(np.abs(a - b).max() <= 1e-12 * max(1.0, np.abs(b).max()) for a, b in zip(got, ref))


def pin_constant_columns(step, rng):
    # |G| constant within each column: V^ is constant per column, both rules agree
    W = rng.standard_normal((12, 7))
    Gs = [np.sign(rng.standard_normal((12, 7))) * rng.uniform(0.5, 2, size=(1, 7))
          for _ in range(4)]
    got = _run(step, W, Gs, True, **HP)[0]
    ref = _torch_adamw(W, Gs, **HP)[0]
    return np.abs(got - ref).max() <= 1e-12


def pin_first_step(step, rng):
    W = rng.standard_normal((16, 5))
    G = rng.standard_normal((16, 5)) * rng.uniform(0.1, 10, size=(1, 5))
    Wn, M1, V1 = step(W, G, np.zeros_like(W), np.zeros_like(W), 1, subspace=True, **HP)
    rms = np.sqrt(np.mean(G * G, axis=0, keepdims=True))
    exp = W * (1 - HP["wd"]) - HP["lr"] * G / (rms + HP["eps"])
    return (np.abs(Wn - exp).max() <= 1e-13
            and np.abs(M1 - (1 - HP["beta1"]) * G).max() <= 1e-15 * np.abs(G).max() * 10
            and np.abs(V1 - (1 - HP["beta2"]) * G * G).max() <= 1e-15 * np.abs(G * G).max() * 10)


def pin_constant_gradient(step, rng):
    W = rng.standard_normal((8, 3))
    g = np.full((8, 3), 0.3)
    hp = dict(HP, wd=0.0)
    Wt, M, V = W, np.zeros_like(W), np.zeros_like(W)
    for t in range(1, 6):
        Wt, M, V = step(Wt, g, M, V, t, subspace=True, **hp)
    exp = W - 5 * hp["lr"] * g / (np.abs(g) + hp["eps"])
    return np.abs(Wt - exp).max() <= 1e-13


PINS = [pin_subspace_preserved, pin_standard_is_torch, pin_constant_columns, pin_first_step,
        pin_constant_gradient]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    assert pin(aw.adamw_step, np.random.default_rng(3))


def test_rejects_step_zero():
    with pytest.raises(ValueError):
        aw.adamw_step(np.zeros((2, 2)), np.zeros((2, 2)), np.zeros((2, 2)), np.zeros((2, 2)), 0,
                      **HP)


# ---------------------------------------------------- the pins have teeth

def _mutant(kind):
    def step(W, G, M, V, t, lr, beta1, beta2, eps, wd, subspace=True):
        W, G, M, V = (np.asarray(a, dtype=np.float64) for a in (W, G, M, V))
        M1 = (beta2 if kind == "m_with_beta2" else beta1) * M + (
            1 - (beta2 if kind == "m_with_beta2" else beta1)) * G
        V1 = beta2 * V + (1 - beta2) * G * G
        if kind == "no_bias_correction":
            Mh, Vh = M1, V1
        elif kind == "printed_correction":
            Mh, Vh = M1 / (beta1 + eps), V1 / (beta2 + eps)
        else:
            Mh, Vh = M1 / (1 - beta1 ** t), V1 / (1 - beta2 ** t)
        if subspace and kind == "elementwise":
            alpha = 1 / (np.sqrt(Vh) + eps)
        elif subspace and kind == "wrong_axis":
            alpha = 1 / (np.sqrt(Vh.mean(axis=1, keepdims=True)) + eps)
        elif subspace and kind == "no_sqrt":
            alpha = 1 / (Vh.mean(axis=0, keepdims=True) + eps)
        elif subspace:
            alpha = 1 / (np.sqrt(Vh.mean(axis=0, keepdims=True)) + eps)
        else:
            alpha = 1 / (np.sqrt(Vh) + eps)
        decay = lr * wd if kind == "lr_scaled_decay" else wd
        return W - lr * alpha * Mh - decay * W, M1, V1
    step.__name__ = kind
    return step


MUTANTS = ["elementwise", "wrong_axis", "no_sqrt", "no_bias_correction", "printed_correction",
           "lr_scaled_decay", "m_with_beta2"]


def test_pins_pass_on_oracle():
    assert all(p(aw.adamw_step, np.random.default_rng(3)) for p in PINS)


@pytest.mark.parametrize("kind", MUTANTS)
def test_pins_catch_planted_mistake(kind):
    assert not all(p(_mutant(kind), np.random.default_rng(3)) for p in PINS)

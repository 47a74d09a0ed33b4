"""GPU parity of the AdamW step (Sec. 5) through the C ABI against the CPU
oracle (float64, rounded once to each output's type).

Tolerances: M and V (float32) within 1e-5 of max(|ref|, rms of the ref's
row); W within 1e-5 (float32) or 2e-2 (bf16) of the same scale, and for bf16
equal to the oracle's rounding in all but a few elements (the kernel's
float32 arithmetic can land on the other side of a rounding boundary, by more
than one unit where W - lr alpha M^ cancels).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import adamw as aw
import synth
import paper_2506_01260_amd as sn
from gpu_helpers import assert_parity, dev, host, log

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=1e-4)


def _cfg(dtype):
    return synth.Config(f"adamw {dtype}", dtype, 64, 8, 10, 1, 1, False, 0.0, 1.0)


def _case(dtype, rows, cols, t0, steps, subspace, cols_sel=None, basis=None, cfg_id=0):
    cfg = _cfg(dtype)
    Wb = synth.make_weight(cfg_id, 0, rows, cols, cfg)
    st = synth.make_adamw_state(cfg_id, rows, cols)
    Gs = [synth.make_weight_grad(cfg_id, s, rows, cols, cfg, basis=basis) for s in range(steps)]
    if basis is not None:
        # W with columns in S, written in the dtype (exactly in S only in fp32 + tolerance)
        Wf = basis @ (basis.T @ synth.as_float(Wb, dtype).astype(np.float64))
        Wb = synth.store(Wf, dtype)
        st = {"M": np.zeros((rows, cols), np.float32), "V": np.zeros((rows, cols), np.float32)}
    W, M, V = dev(Wb, dtype), dev(st["M"], "f32"), dev(st["V"], "f32")
    for s, G in enumerate(Gs):
        sn.sn_adamw_step(W, dev(G, dtype), M, V, t0 + s, subspace=subspace, lr=HP["lr"],
                         beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
                         weight_decay=HP["wd"])
    torch.cuda.synchronize()
    # oracle, step by step, each output rounded to its storage type after every step
    sel = np.arange(cols) if cols_sel is None else np.asarray(cols_sel)
    dec = (lambda a: synth.as_float(a, dtype))
    Wr = dec(Wb)[:, sel].astype(np.float64)
    Mr, Vr = st["M"][:, sel].astype(np.float64), st["V"][:, sel].astype(np.float64)
    for s, G in enumerate(Gs):
        Wr, Mr, Vr = aw.adamw_step(Wr, dec(G)[:, sel], Mr, Vr, t0 + s, subspace=subspace, **HP)
        Wr = oracle.round_to(Wr, dtype).astype(np.float64)
        Mr = oracle.round_f32(Mr).astype(np.float64)
        Vr = oracle.round_f32(Vr).astype(np.float64)
    idx = torch.from_numpy(sel).cuda()
    return (host(W[:, idx]), host(M[:, idx]), host(V[:, idx])), (Wr, Mr, Vr)


def _check(got, ref, dtype, what):
    (Wg, Mg, Vg), (Wr, Mr, Vr) = got, ref
    assert_parity(Mg, Mr, "f32", f"{what} M")
    assert_parity(Vg, Vr, "f32", f"{what} V")
    assert_parity(Wg, Wr, dtype, f"{what} W")
    if dtype == "bf16":
        diff = Wg != Wr
        log(f"  {what} W: {int(diff.sum())} of {diff.size} bf16 elements off the oracle's rounding")
        assert diff.mean() < 1e-3


@pytest.mark.parametrize("dtype,rows,cols,t0,steps", [
    ("f32", 256, 256, 1, 3), ("bf16", 512, 1000, 1, 2), ("bf16", 300, 77, 5, 2),
    ("bf16", 1024, 4096, 7, 1)])
@pytest.mark.parametrize("subspace", [True, False])
def test_adamw_matches_oracle(dtype, rows, cols, t0, steps, subspace):
    log(f"[adamw] {dtype} {rows}x{cols} t0={t0} steps={steps} subspace={subspace}")
    got, ref = _case(dtype, rows, cols, t0, steps, subspace)
    _check(got, ref, dtype, f"{dtype} {rows}x{cols}")


@pytest.mark.parametrize("rows,cols", [(4096, 14336), (4096, 4096)])
def test_adamw_full_size(rows, cols):
    """W2 and Wo of config 2: the modified step on the whole matrix, every
    element of W, M and V compared."""
    log(f"[adamw full] {rows}x{cols}")
    got, ref = _case("bf16", rows, cols, 3, 1, True, cfg_id=2)
    _check(got, ref, "bf16", f"bf16 {rows}x{cols}")


def test_subspace_step_keeps_columns_in_s():
    """fp32: W and every gradient with columns in S; after three modified steps
    the off-subspace part stays at rounding level, while the standard step
    moves it far above."""
    log("[adamw] subspace preservation")
    d, k, m = 512, 16, 300
    U = synth.orthonormal_basis(12345, d, k)
    off = {}
    for subspace in (True, False):
        got, _ = _case("f32", d, m, 1, 3, subspace, basis=U)
        W = got[0]
        off[subspace] = np.abs(W - U @ (U.T @ W)).max() / np.abs(W).max()
    log(f"  off-subspace part: modified {off[True]:.2e}, standard {off[False]:.2e}")
    assert off[True] < 1e-5 and off[False] > 100 * off[True]


def test_adamw_deterministic():
    log("[adamw] determinism")
    a, _ = _case("bf16", 512, 1000, 2, 2, True)
    b, _ = _case("bf16", 512, 1000, 2, 2, True)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)

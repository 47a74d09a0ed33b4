"""Helpers for the GPU parity tests: host <-> device conversion and the
parity criterion.

Parity criterion (per element): |y - y_ref| <= rtol * max(|y_ref|, rms(row of
y_ref)).  The row-RMS floor keeps elements whose exact value is a near-zero
sum of large terms from failing on rounding noise at the scale of the row.
rtol is 1e-5 for fp32 outputs and 2e-2 for bf16 outputs; y_ref is the oracle
(float64) rounded once to the output dtype.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

RTOL = {"f32": 1e-5, "bf16": 2e-2}


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    """Stored host array (float32, or bf16 bits as uint16) -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.cuda()


def ids(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float64 numpy (bf16 and fp32 convert exactly)."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def host_bits(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)
    return t.detach().cpu().numpy().view(np.uint32)


def assert_parity(got: np.ndarray, ref: np.ndarray, dtype: str, what: str):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    if got.size == 0:
        return
    rtol = RTOL[dtype]
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    tol = rtol * np.maximum(np.abs(ref), rms)
    err = np.abs(got - ref)
    bad = err > tol
    if bad.any():
        idx = np.argwhere(bad)[:5]
        detail = ", ".join(f"{tuple(i)}: got {got[tuple(i)]!r} ref {ref[tuple(i)]!r}" for i in idx)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements outside rtol "
                             f"{rtol} (max rel err {float(np.max(err / np.maximum(tol / rtol, 1e-300))):.3g}); {detail}")
    rel_f = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    log(f"  {what}: ok ({got.size} elements, max |err|/scale {float(np.max(err / np.maximum(tol / rtol, 1e-300))):.2e}, "
        f"rel Frobenius {rel_f:.2e})")

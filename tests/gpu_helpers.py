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


def _workers() -> int:
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _chunk_stats(got: np.ndarray, ref: np.ndarray, rtol: float, row0: int):
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    scale = np.maximum(np.abs(ref), rms)
    err = np.abs(got - ref)
    bad = err > rtol * scale
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(scale > 0, err / np.where(scale > 0, scale, 1.0), np.where(err > 0, np.inf, 0.0))
    detail = ""
    if bad.any():
        i, j = np.argwhere(bad)[0]
        detail = f"({row0 + i}, {j}): got {got[i, j]!r} ref {ref[i, j]!r}"
    return int(bad.sum()), float(rel.max()) if rel.size else 0.0, \
        float(np.sum((got - ref) ** 2)), float(np.sum(ref * ref)), detail


def assert_parity_rows(got: np.ndarray, ref_rows, dtype: str, what: str, row_chunk: int = 0):
    """Every element of got (host array, n x c) against the oracle, computed
    row chunk by row chunk: ref_rows(rows) returns the oracle's unrounded
    float64 values of those rows, which are rounded once to dtype and compared
    with the parity criterion above.  Chunks run on a thread pool (numpy
    releases the GIL) with single-threaded BLAS inside; memory stays bounded
    by the chunk size."""
    import concurrent.futures as cf
    from threadpoolctl import threadpool_limits

    n, c = got.shape
    if n == 0:
        return
    if row_chunk <= 0:
        row_chunk = max(64, (1 << 22) // max(c, 1))   # ~4 M elements per chunk
    rtol = RTOL[dtype]

    def one(r0):
        rows = np.arange(r0, min(n, r0 + row_chunk))
        ref = np.asarray(ref_rows(rows), dtype=np.float64)
        # local import: the oracle's single rounding to the output dtype
        import oracle
        ref = oracle.round_to(ref, dtype)
        g = np.asarray(got[rows[0]:rows[-1] + 1], dtype=np.float64)
        assert g.shape == ref.shape, f"{what}: shape {g.shape} vs {ref.shape}"
        return _chunk_stats(g, ref, rtol, r0)

    with threadpool_limits(limits=1), cf.ThreadPoolExecutor(max_workers=_workers()) as ex:
        res = list(ex.map(one, range(0, n, row_chunk)))
    nbad = sum(r[0] for r in res)
    worst = max(r[1] for r in res)
    rel_f = (sum(r[2] for r in res) / max(sum(r[3] for r in res), 1e-300)) ** 0.5
    if nbad:
        detail = next(r[4] for r in res if r[4])
        raise AssertionError(f"{what}: {nbad} of {n * c} elements outside rtol {rtol} "
                             f"(max rel err {worst:.3g}); first {detail}")
    log(f"  {what}: ok (all {n * c} elements, max |err|/scale {worst:.2e}, "
        f"rel Frobenius {rel_f:.2e})")

"""sn_project_weights_noalloc (the weight confinement with the library's
static scratch instead of a caller workspace) against sn_project_weights,
through the C ABI.

Both run the same kernels, so the results must agree bit for bit.  The calls
come in a row on one device, each larger or smaller than the one before, so
every call after the first finds the previous call's values in the scratch.
"""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2506_01260_amd as sn
from gpu_helpers import assert_parity_rows, dev, log

pytestmark = pytest.mark.gpu


def _noalloc_abi(basis, W: torch.Tensor) -> int:
    """The C entry point called directly (plain pointers, sizes, the stream)."""
    d, m = W.shape
    return sn.lib().sn_project_weights_noalloc(
        ctypes.c_void_p(basis.ptr), d, basis.k, basis.dt, ctypes.c_void_p(W.data_ptr()), m,
        W.stride(0), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def _pair(basis, Wh: np.ndarray, dtype: str, tag: str):
    ref = dev(Wh, dtype)
    got = ref.clone()
    sn.sn_project_weights(basis, ref)          # caller workspace
    st = _noalloc_abi(basis, got)              # static scratch
    assert st == 0, f"{tag}: status {st}: {sn.lib().sn_last_error().decode()}"
    torch.cuda.synchronize()
    same = torch.equal(got.view(torch.int16) if dtype == "bf16" else got,
                       ref.view(torch.int16) if dtype == "bf16" else ref)
    assert same, f"{tag}: the no-alloc result differs from sn_project_weights"
    log(f"  {tag}: bit-identical to sn_project_weights")
    return got


def test_noalloc_matches_workspace_entry_point():
    # config 2's basis: W2 (4096 x 14336), then the smaller Wo (4096 x 4096)
    cfg = synth.CONFIGS[2]
    b = synth.make_basis(2)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    U64 = oracle.decode_bf16(b["U"])
    for i, (r, c) in reversed(list(enumerate(cfg.weights))):
        Wh = synth.make_weight(2, i, r, c)
        log(f"[no-alloc] config 2 W{i} {r}x{c}")
        got = _pair(basis, Wh, "bf16", f"cfg2 W{i}")
        Wf = oracle.decode_bf16(Wh, np.float32)
        assert_parity_rows(got.float().cpu().numpy().T,
                           lambda rows: oracle.project_weights(Wf, U64, cols=rows).T,
                           "bf16", f"cfg2 W{i} no-alloc vs oracle (every column)")
    # a smaller, ragged call (generic kernels: m not a multiple of 8), then fp32
    for dtype, d, k, m in (("bf16", 512, 20, 300), ("f32", 256, 8, 100)):
        c = synth.Config("noalloc", dtype, d, k, 10, 1, 1, False, 0.0, 1.0)
        bb = synth.make_basis(0, c)
        basis2 = sn.sn_basis_pack(dev(bb["U"], dtype))
        log(f"[no-alloc] {dtype} {d}x{m} k={k}")
        _pair(basis2, synth.make_weight(0, 0, d, m, c), dtype, f"{dtype} {d}x{m}")


def test_noalloc_binding_and_limits():
    b = synth.make_basis(2)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    W = dev(synth.make_weight(2, 0, 4096, 4096), "bf16")
    ref = W.clone()
    sn.sn_project_weights(basis, ref)
    sn.sn_project_weights_noalloc(basis, W)    # the Python binding, same entry point
    torch.cuda.synchronize()
    assert torch.equal(W.view(torch.int16), ref.view(torch.int16))
    # a matrix whose workspace exceeds the scratch is refused before any launch
    m = 1 << 16
    need = sn.sn_project_weights_workspace_bytes(4096, 40, sn.SN_BF16, m)
    assert need > (128 << 20)
    big = torch.zeros(4096, m, dtype=torch.bfloat16, device="cuda")
    st = _noalloc_abi(basis, big)
    assert st == 9, st
    assert "static scratch" in sn.lib().sn_last_error().decode()
    torch.cuda.synchronize()
    assert float(big.abs().max()) == 0.0

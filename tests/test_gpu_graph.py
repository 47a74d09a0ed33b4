"""The codec calls captured in a HIP graph: every replay must give the bits
the eager calls give.

The library launches only kernels on the caller's stream (no memset or copy
nodes), so a captured step is the same work as the eager step.  Each replay
here is preceded by eager work of the program's own (outputs overwritten
with NaN, the weights restored, an unrelated eager compress) and followed by
a synchronisation, and every replay's outputs are compared bit for bit with
the eager ones.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2506_01260_amd as sn
from gpu_helpers import log

pytestmark = pytest.mark.gpu


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy() if t.dtype == torch.bfloat16 else \
        t.view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("d,k,n,m", [(1024, 40, 4096, 2048), (512, 20, 1000, 384),
                                     (256, 40, 32768, 256)])  # 128-token compress workgroups
def test_graph_replays_match_eager(d, k, n, m):
    log(f"[graph] d={d} k={k} n={n} m={m}")
    g = torch.Generator(device="cuda")
    g.manual_seed(d + k + n)
    U = torch.linalg.qr(torch.randn(d, k, device="cuda", generator=g, dtype=torch.float64))[0]
    basis = sn.sn_basis_pack(U.to(torch.bfloat16).contiguous())
    vocab, seq = 3000, 128
    E = (torch.randn(vocab, d, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    P = (torch.randn(seq, d, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    tok = torch.randint(0, vocab, (n,), device="cuda", generator=g, dtype=torch.int32)
    X = torch.randn(n, d, device="cuda", generator=g).to(torch.bfloat16)
    G = (torch.randn(n, d, device="cuda", generator=g) * 1e-2).to(torch.bfloat16)
    W0 = (torch.randn(d, m, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    W = W0.clone()
    ws = torch.empty(sn.sn_project_weights_workspace_bytes(d, k, sn.SN_BF16, m),
                     dtype=torch.uint8, device="cuda")
    proj = sn.sn_embed_project(basis, E=E, P=P)
    outs = {"C": torch.empty(n, k, dtype=torch.bfloat16, device="cuda"),
            "Xr": torch.empty(n, d, dtype=torch.bfloat16, device="cuda"),
            "Cg": torch.empty(n, k, dtype=torch.bfloat16, device="cuda"),
            "Gr": torch.empty(n, d, dtype=torch.bfloat16, device="cuda"),
            "Cp": torch.empty(n, k, dtype=torch.bfloat16, device="cuda")}

    def step():
        sn.sn_compress(basis, X, tok=tok, E=E, P=P, seq_len=seq, out=outs["C"])
        sn.sn_decompress(basis, outs["C"], tok=tok, E=E, P=P, seq_len=seq, out=outs["Xr"])
        sn.sn_grad_compress(basis, G, out=outs["Cg"])
        sn.sn_decompress(basis, outs["Cg"], out=outs["Gr"])
        sn.sn_compress_projected(basis, X, proj, tok=tok, seq_len=seq, out=outs["Cp"])
        sn.sn_project_weights(basis, W, workspace=ws)

    step()  # eager reference
    torch.cuda.synchronize()
    ref = {name: _bits(t) for name, t in outs.items()}
    ref["W"] = _bits(W)

    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            step()
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()

    other = torch.empty(n, k, dtype=torch.bfloat16, device="cuda")
    for rep in range(4):
        for t in outs.values():
            t.fill_(float("nan"))
        W.copy_(W0)
        sn.sn_compress(basis, G, tok=tok, E=E, P=P, seq_len=seq, out=other)  # unrelated eager work
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, t in outs.items():
            assert np.array_equal(_bits(t), ref[name]), f"replay {rep}: {name} differs from eager"
        assert np.array_equal(_bits(W), ref["W"]), f"replay {rep}: projected W differs from eager"
    del graph

"""GPU parity of the projected-table compress (sn_embed_project +
sn_compress_projected) against the CPU oracle.

C = X U - (P U)[pos] - (T_fixed U)[tok] is the same linear map as
(X - P[pos] - T_fixed[tok]) U, so the expected values are the oracle's
``compress`` (float64, rounded once to the output dtype), and the projected
tables are compared with the oracle's row projection E U / P U (float64,
rounded to float32: the tables are fp32 for both input dtypes).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2506_01260_amd as sn
import test_gpu_codec as base
from gpu_helpers import assert_parity, assert_parity_rows, dev, host, host_bits, ids, log

pytestmark = pytest.mark.gpu


def check_tables(proj, o_E, o_P, U64, k, what=""):
    """Every row of both projected tables against the oracle's row projection."""
    EU, PU = proj.tables()
    for name, T, ref_tab in (("T_fixed U", EU, o_E), ("P U", PU, o_P)):
        if ref_tab is None:
            assert T.shape[0] == 0
            continue
        got = base.host_f32(T)
        assert np.all(got[:, k:] == 0.0), f"{what} {name}: padding columns are not zero"
        assert_parity_rows(got[:, :k], lambda r: oracle.grad_compress(ref_tab, U64, rows=r),
                           "f32", f"{what} {name}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,k,n", [(256, 20, 1), (256, 20, 17), (256, 20, 33), (256, 1, 40),
                                   (256, 16, 31), (256, 17, 50), (256, 33, 16), (256, 82, 45),
                                   (256, 128, 20), (384, 130, 19), (200, 20, 37), (96, 5, 64),
                                   (160, 40, 130)])
def test_projected_shapes(dtype, d, k, n):
    log(f"[projected shapes] {dtype} d={d} k={k} n={n}")
    st, o, tok, _ = base._small(d, k, n, dtype=dtype, seed=d + k + n)
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X = (dev(st[x], dtype) for x in ("E", "P", "X"))
    proj = sn.sn_embed_project(basis, E=E, P=P)
    check_tables(proj, o["E"], o["P"], o["U"], k, what=f"d={d} k={k}")
    C = sn.sn_compress_projected(basis, X, proj, tok=ids(tok), seq_len=9)
    ref = oracle.round_to(oracle.compress(o["X"], o["U"], tok, o["E"], o["P"], seq_len=9), dtype)
    assert_parity(host(C), ref, dtype, "compress_projected")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_projected_tables_optional_and_explicit_positions(dtype):
    d, k, n = 256, 24, 70
    st, o, tok, _ = base._small(d, k, n, dtype=dtype, seed=5)
    pos = np.random.default_rng(6).integers(0, 9, n).astype(np.int32)
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X = (dev(st[x], dtype) for x in ("E", "P", "X"))
    cases = [("E+P explicit pos", dict(E=E, P=P), dict(tok=ids(tok), pos=ids(pos)),
              dict(tok=tok, E=o["E"], P=o["P"], pos=pos)),
             ("E only", dict(E=E), dict(tok=ids(tok)), dict(tok=tok, E=o["E"])),
             ("P only default pos", dict(P=P), dict(seq_len=9), dict(P=o["P"], seq_len=9)),
             ("no tables", {}, {}, {})]
    for name, tables, gk, ok in cases:
        proj = sn.sn_embed_project(basis, **tables)
        check_tables(proj, ok.get("E"), ok.get("P"), o["U"], k, what=name)
        C = sn.sn_compress_projected(basis, X, proj, **gk)
        assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], **ok), dtype),
                      dtype, f"compress_projected {name}")
        if not tables:   # plain X U: the same kernel as the gradient compress, bit for bit
            Cg = sn.sn_grad_compress(basis, X)
            assert np.array_equal(host_bits(C), host_bits(Cg))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_projected_out_of_range_ids_are_clamped_and_flagged(dtype):
    d, k, n, vocab = 256, 20, 40, 50
    st, o, tok, _ = base._small(d, k, n, vocab=vocab, dtype=dtype, seed=9)
    bad_tok = tok.copy()
    bad_tok[3], bad_tok[20] = vocab + 5, -2
    bad_pos = (np.arange(n) % 9).astype(np.int32)
    bad_pos[7] = 100
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X = (dev(st[x], dtype) for x in ("E", "P", "X"))
    proj = sn.sn_embed_project(basis, E=E, P=P)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    C = sn.sn_compress_projected(basis, X, proj, tok=ids(bad_tok), pos=ids(bad_pos),
                                 err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 3
    ct, cp = np.clip(bad_tok, 0, vocab - 1), np.clip(bad_pos, 0, 8)
    assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], ct, o["E"], o["P"],
                                                           pos=cp), dtype), dtype,
                  "compress_projected with clamped ids")


def test_projected_strides_and_empty_batch():
    d, k, n = 256, 40, 37
    st, o, tok, _ = base._small(d, k, n, seed=7)
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    Ebig = torch.zeros(50, d + 64, dtype=torch.bfloat16, device="cuda")
    Ebig[:, :d] = dev(st["E"], "bf16")
    proj = sn.sn_embed_project(basis, E=Ebig[:, :d], P=dev(st["P"], "bf16"))
    Xbig = torch.zeros(n, d + 8, dtype=torch.bfloat16, device="cuda")
    Xbig[:, :d] = dev(st["X"], "bf16")
    Cbig = torch.full((n + 3, k + 5), 7.0, dtype=torch.bfloat16, device="cuda")
    sn.sn_compress_projected(basis, Xbig[:, :d], proj, tok=ids(tok), seq_len=9,
                             out=Cbig[:n, :k])
    assert_parity(host(Cbig[:n, :k]),
                  oracle.round_to(oracle.compress(o["X"], o["U"], tok, o["E"], o["P"],
                                                  seq_len=9), "bf16"), "bf16",
                  "compress_projected strided")
    cb = host(Cbig)
    assert np.all(cb[n:] == 7.0) and np.all(cb[:, k:] == 7.0)
    empty = torch.empty(0, d, dtype=torch.bfloat16, device="cuda")
    out = sn.sn_compress_projected(basis, empty, proj, tok=ids(np.zeros(0, np.int32)), seq_len=9)
    assert out.shape == (0, k)


@pytest.mark.parametrize("cfg_id", [0, 1, 2, 4])
def test_projected_configs(cfg_id):
    w = base.workload(cfg_id)
    cfg = w["cfg"]
    dt = cfg.dtype
    o = base.oracle_inputs(w)
    basis = sn.sn_basis_pack(dev(w["U"], dt))
    E, P, X = dev(w["E"], dt), dev(w["P"], dt), dev(w["X"], dt)
    log(f"[projected cfg{cfg_id}] tables vocab={cfg.vocab} n_pos={P.shape[0]} k={cfg.k}")
    proj = sn.sn_embed_project(basis, E=E, P=P)
    check_tables(proj, o["E"], o["P"], o["U"], cfg.k, what=f"cfg{cfg_id}")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    C = sn.sn_compress_projected(basis, X, proj, tok=ids(w["tok"]), seq_len=cfg.seq,
                                 err_flag=flag)
    assert_parity_rows(base.host_f32(C),
                       lambda r: oracle.compress(o["X"], o["U"], w["tok"], o["E"], o["P"],
                                                 seq_len=cfg.seq, rows=r),
                       dt, f"cfg{cfg_id} compress_projected (every row)")
    torch.cuda.synchronize()
    assert int(flag.item()) == 0

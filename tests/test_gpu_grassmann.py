"""GPU parity of the subspace update (Sec. 4.5) through the C ABI against the
CPU oracle.

The GPU keeps Y = sum_t G_t^T (G_t U) instead of S (U is fixed between
updates, so Y = K S U); the oracle forms S (or selected rows of it) as the
paper defines it, and the tests compare Y with K S U, the accumulated loss
with sum_t |G_t (I - U U^T)|^2, and the new basis with the oracle's step.

Tolerances (derived in the design notes): Y per element within 1e-5 of
max(|ref|, rms of the ref's column); the loss within 1e-5 * sum_t |G_t|^2
(float32 coefficient sums, float64 everywhere else); the new basis, written
as float32, within 1e-5 per element of max(|ref|, rms of its row); written as
bf16, equal to the oracle's rounding in all but a few elements (each at most
one unit in the last place away).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import grassmann as gr
import synth
import paper_2506_01260_amd as sn
from gpu_helpers import assert_parity, dev, host, log

pytestmark = pytest.mark.gpu


def _cfg(dtype, d, k, n):
    return synth.Config(f"grass {dtype} d{d} k{k} n{n}", dtype, d, k, 1000, 1, n, True, 0.0,
                        1.0 if dtype == "f32" else 1e-2)


def _setup(cfg_id, cfg, K):
    b = synth.make_basis(cfg_id, cfg)
    Gs = [synth.make_grad_iteration(cfg_id, t, cfg.n_tokens, cfg) for t in range(K)]
    dec = (lambda a: oracle.decode_bf16(a, np.float32)) if cfg.dtype == "bf16" else \
        (lambda a: np.asarray(a, np.float32))
    U = dec(b["U"]).astype(np.float64)
    return b, Gs, [dec(g) for g in Gs], U


def _accumulate(basis, Gs_dev, with_su=True, want_cg=False):
    state = sn.sn_grassmann_state(basis)
    cgs = []
    for G in Gs_dev:
        cgs.append(sn.sn_grassmann_accumulate(basis, G, state, with_su=with_su, want_cg=want_cg))
    torch.cuda.synchronize()
    return state, cgs


def _check_loss(state, Gf, U, K):
    sc = state.scalars().cpu().numpy()
    ref = sum(gr.off_subspace_energy(g, U) for g in Gf)
    energy = sum(float(np.sum(g.astype(np.float64) ** 2)) for g in Gf)
    log(f"  loss sum {sc[0]:.9g} ref {ref:.9g} (energy {energy:.6g}), K_L {sc[1]}, L {sc[2]:.9g}")
    assert abs(sc[0] - ref) <= 1e-5 * energy
    assert sc[1] == K and abs(sc[2] - sc[0] / K) <= 1e-15 * abs(sc[0])
    return sc


def _check_y(state, Gf, U, K, rows=None):
    Y = state.Y()
    if rows is None:
        ref = K * (gr.accumulation_matrix(Gf) @ U)
        got = host(Y)
    else:
        ref = K * (gr.accumulation_rows(Gf, rows) @ U)
        got = host(Y[torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()])
    # floor per coefficient j: compare the transposes (rows = coefficients)
    assert_parity(got.T, ref.T, "f32", "Y = sum_t G_t^T G_t U")


def _check_y_chunked(state, Gf, U, K, chunk=256):
    """Every row of Y against K S U, S's rows formed by the oracle in chunks
    on a thread pool (single-threaded BLAS in each)."""
    import concurrent.futures as cf
    from threadpoolctl import threadpool_limits
    from gpu_helpers import _workers
    d = U.shape[0]

    def one(r0):
        rows = np.arange(r0, min(d, r0 + chunk))
        return K * (gr.accumulation_rows(Gf, rows) @ U)

    with threadpool_limits(limits=1), cf.ThreadPoolExecutor(max_workers=_workers()) as ex:
        ref = np.concatenate(list(ex.map(one, range(0, d, chunk))))
    assert_parity(host(state.Y()).T, ref.T, "f32", "Y = sum_t G_t^T G_t U (every row)")


SHAPES = [  # dtype, d, k, n: generic fp32; MFMA [C_hi | C_lo] with ragged n;
            # MFMA with two operands (2k > 128); generic bf16 (d not a multiple of 64)
    ("f32", 256, 8, 512), ("bf16", 512, 40, 1000), ("bf16", 320, 20, 300),
    ("bf16", 512, 70, 700), ("bf16", 96, 8, 77), ("bf16", 1024, 128, 129),
]


@pytest.mark.parametrize("dtype,d,k,n", SHAPES)
def test_accumulate_shapes(dtype, d, k, n):
    log(f"[grassmann accumulate] {dtype} d={d} k={k} n={n}")
    cfg = _cfg(dtype, d, k, n)
    K = 3
    b, Gs, Gf, U = _setup(0, cfg, K)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    G_dev = [dev(g, dtype) for g in Gs]
    state, cgs = _accumulate(basis, G_dev, want_cg=True)
    _check_loss(state, Gf, U, K)
    _check_y(state, Gf, U, K)
    sc = state.scalars().cpu().numpy()
    assert sc[3] == K
    # the wire coefficients are exactly the gradient compress's
    for G, cg in zip(G_dev, cgs):
        ref = sn.sn_grad_compress(basis, G)
        torch.cuda.synchronize()
        assert torch.equal(cg.view(torch.int16) if dtype == "bf16" else cg,
                           ref.view(torch.int16) if dtype == "bf16" else ref)
    exp = oracle.round_to(oracle.grad_compress(Gf[0], U), dtype)
    assert_parity(host(cgs[0]), exp, dtype, "wire coefficients")


@pytest.mark.parametrize("dtype,d,k,n", [("f32", 256, 8, 512), ("bf16", 512, 40, 1000)])
def test_monitor_only_leaves_y(dtype, d, k, n):
    log(f"[grassmann monitor] {dtype} d={d} k={k} n={n}")
    cfg = _cfg(dtype, d, k, n)
    b, Gs, Gf, U = _setup(0, cfg, 2)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    state, _ = _accumulate(basis, [dev(g, dtype) for g in Gs], with_su=False)
    _check_loss(state, Gf, U, 2)
    assert state.scalars().cpu().numpy()[3] == 0
    assert float(state.Y().abs().max()) == 0.0


def _step_case(dtype, d, k, n, K, out_dtype):
    cfg = _cfg(dtype, d, k, n)
    b, Gs, Gf, U = _setup(0, cfg, K)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    state, _ = _accumulate(basis, [dev(g, dtype) for g in Gs])
    S = gr.accumulation_matrix(Gf)
    eta = 0.3 / float(np.linalg.eigvalsh(S)[-1])
    ref = gr.grassmann_step(U, S, eta)
    got = sn.sn_grassmann_step(basis, state, eta, out_dtype=out_dtype)
    torch.cuda.synchronize()
    return got, ref, U, S, eta, Gf


@pytest.mark.parametrize("dtype,d,k,n,K", [("f32", 256, 8, 512, 3), ("bf16", 512, 40, 1000, 2),
                                           ("bf16", 512, 70, 300, 2),
                                           ("bf16", 1024, 128, 256, 1)])
def test_step_matches_oracle(dtype, d, k, n, K):
    log(f"[grassmann step] {dtype} d={d} k={k} n={n} K={K}")
    got, ref, U, S, eta, Gf = _step_case(dtype, d, k, n, K, torch.float32)
    assert_parity(host(got), ref, "f32", "U_new (float32)")
    Un = host(got)
    assert np.abs(Un.T @ Un - np.eye(k)).max() < 1e-5
    assert gr.grassmann_loss(Gf, Un) < gr.grassmann_loss(Gf, U)


def test_step_bf16_output_rounds_like_the_oracle():
    log("[grassmann step] bf16 output d=512 k=40")
    got, ref, U, S, eta, Gf = _step_case("bf16", 512, 40, 1000, 2, torch.bfloat16)
    exp = oracle.round_bf16(ref)
    g = host(got)
    assert_parity(g, exp, "bf16", "U_new (bf16)")
    diff = g != exp
    assert diff.mean() < 1e-3, f"{int(diff.sum())} elements differ from the oracle's rounding"
    if diff.any():  # at most one unit in the last place
        ulp = np.abs(exp[diff]) * 2.0 ** -7
        assert np.all(np.abs(g[diff] - exp[diff]) <= ulp)


def test_step_without_accumulation_reorthonormalises():
    log("[grassmann step] K = 0")
    cfg = _cfg("bf16", 512, 40, 64)
    b = synth.make_basis(0, cfg)
    U = oracle.decode_bf16(b["U"], np.float32).astype(np.float64)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    state = sn.sn_grassmann_state(basis)
    got = sn.sn_grassmann_step(basis, state, 0.5, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert_parity(host(got), gr.qr_retract(U), "f32", "U_new = qf(U)")


def test_step_failure_returns_old_basis_and_flags():
    """A state holding NaN (written by the caller) makes the Gram matrix's
    pivot NaN: the step reports bit 2 and writes U unchanged."""
    log("[grassmann step] NaN state")
    cfg = _cfg("f32", 256, 8, 64)
    b = synth.make_basis(0, cfg)
    basis = sn.sn_basis_pack(dev(b["U"], "f32"))
    state = sn.sn_grassmann_state(basis)
    state.Y().fill_(float("nan"))
    state.scalars()[3] = 1.0
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = sn.sn_grassmann_step(basis, state, 0.1, out_dtype=torch.float32, err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) & 4
    assert np.array_equal(host(got), np.asarray(b["U"], np.float64))


def test_reset_and_repeat_are_deterministic():
    log("[grassmann determinism] bf16 d=512 k=40")
    cfg = _cfg("bf16", 512, 40, 1000)
    b, Gs, Gf, U = _setup(0, cfg, 2)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    G_dev = [dev(g, "bf16") for g in Gs]
    s1, _ = _accumulate(basis, G_dev)
    y1, c1 = s1.Y().clone(), s1.scalars().clone()
    sn.sn_grassmann_reset(s1)
    for G in G_dev:
        sn.sn_grassmann_accumulate(basis, G, s1)
    torch.cuda.synchronize()
    assert torch.equal(s1.Y(), y1) and torch.equal(s1.scalars(), c1)


@pytest.mark.parametrize("cfg_id,n,K", [(2, None, 2), (4, 32767, 1)])
def test_accumulate_full_size(cfg_id, n, K):
    """Configs 2 and 4 at full size: the loss and every row of Y (each row of
    S times U, the oracle forming S's rows in chunks on a thread pool)."""
    cfg = synth.CONFIGS[cfg_id]
    n = cfg.n_tokens if n is None else n
    log(f"[grassmann full size] config {cfg_id} n={n} K={K}")
    b = synth.make_basis(cfg_id)
    U = oracle.decode_bf16(b["U"], np.float32).astype(np.float64)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    state = sn.sn_grassmann_state(basis)
    Gf = []
    for t in range(K):
        g = synth.make_grad_iteration(cfg_id, t, n)
        sn.sn_grassmann_accumulate(basis, dev(g, "bf16"), state)
        Gf.append(oracle.decode_bf16(g, np.float32))
        del g
    torch.cuda.synchronize()
    _check_loss(state, Gf, U, K)
    _check_y_chunked(state, Gf, U, K)


def test_step_full_width():
    """The step at d = 4096, k = 40 (config 2's basis) with a short accumulation."""
    log("[grassmann step] d=4096 k=40 n=256")
    got, ref, U, S, eta, Gf = _step_case("bf16", 4096, 40, 256, 2, torch.float32)
    assert_parity(host(got), ref, "f32", "U_new (float32)")

"""GPU parity of the HIP codec (through the C ABI) against the CPU oracle.

Inputs come from the seeded generator (``synth``) or are designed here; every
expected value comes from ``oracle`` (float64, rounded once to the output
dtype) or from the stored exact fixture.  Nothing the GPU produces is fed to
the oracle.  Every element of every output is compared, at the full sizes
too (the oracle works through the rows in chunks on a thread pool).
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2506_01260_amd as sn
from gpu_helpers import assert_parity, assert_parity_rows, dev, host, host_bits, ids, log

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_exact.json")

_CACHE: dict = {}


def workload(cfg: int, n: int | None = None, sigma: float | None = None) -> dict:
    key = (cfg, n, sigma)
    if key not in _CACHE:
        log(f"[gen] config {cfg} n={n} sigma={sigma}")
        _CACHE.clear()  # keep host memory bounded: one workload at a time
        _CACHE[key] = synth.make_workload(cfg, n, sigma)
    return _CACHE[key]


def oracle_inputs(w: dict) -> dict:
    """Exact float32 views of the stored inputs (the oracle up-converts the
    rows it uses to float64); decoded once per workload."""
    if "_oracle_inputs" in w:
        return w["_oracle_inputs"]
    dt = w["cfg"].dtype
    if dt == "bf16":
        dec = lambda a: oracle.decode_bf16(a, np.float32)  # noqa: E731
    else:
        dec = lambda a: np.asarray(a, np.float32)  # noqa: E731
    out = {name: dec(w[name]) for name in ("E", "P", "X", "G")}
    out["U"] = dec(w["U"]).astype(np.float64)
    w["_oracle_inputs"] = out
    return out


def host_rows(t: torch.Tensor, sel: np.ndarray) -> np.ndarray:
    return host(t[torch.from_numpy(np.asarray(sel, dtype=np.int64)).cuda()])


def host_f32(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float32 numpy (bf16 converts exactly)."""
    return t.detach().float().cpu().numpy()


OPS = ("compress", "decompress", "grad_compress", "grad_decompress", "roundtrip")

_OUT: dict = {}


def codec_outputs(w: dict, key) -> dict:
    """The four codec ops of workload w run once on the GPU through the C ABI
    (the launch configuration the benchmark times: whole batch, default
    positions), plus the forward round trip decompress(compress(X)); host
    float32 copies.  The decompress inputs are the generator's coefficients
    C_true (stored in the dtype), the same on both sides."""
    if key in _OUT:
        return _OUT[key]
    _OUT.clear()
    cfg = w["cfg"]
    dt = cfg.dtype
    U = dev(w["U"], dt)
    basis = sn.sn_basis_pack(U)
    X, E, P, G = dev(w["X"], dt), dev(w["E"], dt), dev(w["P"], dt), dev(w["G"], dt)
    tok = ids(w["tok"])
    n = w["tok"].shape[0]
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    Cin_np = synth.store(w["C_true"], dt)
    Cin = dev(Cin_np, dt)
    log(f"[gpu] codec ops N={n} d={cfg.d} k={cfg.k} {dt}")
    out = {"Cin": Cin_np}
    C = sn.sn_compress(basis, X, tok=tok, E=E, P=P, seq_len=cfg.seq, err_flag=flag)
    out["compress"] = host_f32(C)
    out["roundtrip"] = host_f32(sn.sn_decompress(basis, C, tok=tok, E=E, P=P, seq_len=cfg.seq))
    out["decompress"] = host_f32(sn.sn_decompress(basis, Cin, tok=tok, E=E, P=P,
                                                  seq_len=cfg.seq, err_flag=flag))
    out["grad_compress"] = host_f32(sn.sn_grad_compress(basis, G))
    out["grad_decompress"] = host_f32(sn.sn_decompress(basis, Cin))
    torch.cuda.synchronize()
    out["flag"] = int(flag.item())
    del X, E, P, G, C, Cin, basis, U
    torch.cuda.empty_cache()
    _OUT[key] = out
    return out


def check_op(w: dict, out: dict, op: str, tag: str):
    """One op's GPU result against the oracle, every element (row chunks)."""
    cfg = w["cfg"]
    dt = cfg.dtype
    o = oracle_inputs(w)
    tok, seq = w["tok"], cfg.seq
    Cin64 = oracle.decode_bf16(out["Cin"]) if dt == "bf16" else out["Cin"].astype(np.float64)
    assert out["flag"] == 0, "no id is out of range in generated workloads"
    if op == "compress":
        assert_parity_rows(out[op], lambda r: oracle.compress(o["X"], o["U"], tok, o["E"], o["P"],
                                                              seq_len=seq, rows=r),
                           dt, f"{tag} compress")
    elif op == "decompress":
        assert_parity_rows(out[op], lambda r: oracle.decompress(Cin64, o["U"], tok, o["E"],
                                                                o["P"], seq_len=seq, rows=r),
                           dt, f"{tag} decompress")
    elif op == "grad_compress":
        assert_parity_rows(out[op], lambda r: oracle.grad_compress(o["G"], o["U"], rows=r),
                           dt, f"{tag} grad_compress")
    elif op == "grad_decompress":
        assert_parity_rows(out[op], lambda r: oracle.grad_decompress(Cin64, o["U"], rows=r),
                           dt, f"{tag} grad_decompress")
    else:
        # property at any size: the forward round trip loses only the
        # off-subspace residual (plus rounding of C and X_rec to the dtype)
        Xh = o["X"].astype(np.float64)
        Xrt = out[op].astype(np.float64)
        err = np.linalg.norm(Xrt - Xh)
        pos = oracle.default_positions(Xh.shape[0], seq)
        resid = Xh - o["E"][tok] - o["P"][pos]
        off = np.linalg.norm(resid - (resid @ o["U"]) @ o["U"].T)
        scale = np.linalg.norm(Xh)
        slack = (1e-5 if dt == "f32" else 2e-2) * scale
        log(f"[{tag}] round trip |X_rec - X| = {err:.4g}, off-subspace {off:.4g}, |X| {scale:.4g}")
        assert abs(err - off) <= slack


def run_codec(w: dict, tag: str):
    """Forward and gradient codec of workload w on the GPU vs the oracle,
    every element of every op."""
    out = codec_outputs(w, ("run", tag))
    for op in OPS:
        check_op(w, out, op, tag)


# ---------------------------------------------------------------- fixtures

def _golden(d_pad: int, dtype: str):
    g = json.load(open(GOLDEN))
    d = g["d"]
    f = lambda m: np.array([[float(Fraction(v)) for v in r] for r in m])  # noqa: E731

    def pad(a):
        out = np.zeros((a.shape[0], d_pad))
        out[:, :d] = a
        return out

    mats = {n: f(g[n]) for n in ("U", "E", "P", "X", "G")}
    mats = {n: pad(a.T).T if n == "U" else pad(a) for n, a in mats.items()}
    mats["U"] = mats["U"]  # d_pad x k, zero rows past d
    W = np.zeros((d_pad, 6))
    W[:d] = f(g["W"])
    mats["W"] = W
    ex = {n: f(v) for n, v in g["expect"].items()}
    ex["X_rec"] = pad(ex["X_rec"])
    ex["G_rec"] = pad(ex["G_rec"])
    Wp = np.zeros((d_pad, 6))
    Wp[:d] = ex["W_proj"]
    ex["W_proj"] = Wp
    return g, mats, ex


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d_pad", [8, 32, 64])
def test_golden_fixture_exact(dtype, d_pad):
    """Dyadic inputs whose exact results every dtype represents: bit-exact."""
    log(f"[golden] dtype={dtype} d={d_pad}")
    g, m, ex = _golden(d_pad, dtype)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    t = {n: torch.tensor(np.ascontiguousarray(a), dtype=tdt, device="cuda") for n, a in m.items()}
    basis = sn.sn_basis_pack(t["U"])
    tok, pos = ids(np.array(g["tok"])), ids(np.array(g["pos"]))
    C = sn.sn_compress(basis, t["X"], tok=tok, E=t["E"], P=t["P"], pos=pos)
    assert np.array_equal(host(C), ex["C"])
    Xr = sn.sn_decompress(basis, C, tok=tok, E=t["E"], P=t["P"], pos=pos)
    assert np.array_equal(host(Xr), ex["X_rec"])
    Cg = sn.sn_grad_compress(basis, t["G"])
    assert np.array_equal(host(Cg), ex["Cg"])
    assert np.array_equal(host(sn.sn_decompress(basis, Cg)), ex["G_rec"])
    W = t["W"].clone()
    sn.sn_project_weights(basis, W)
    assert np.array_equal(host(W), ex["W_proj"])


# ------------------------------------------------------------ the configs

@pytest.mark.parametrize("sigma", [0.0, 1e-3])
def test_config0_fp32_all_ops(sigma):
    w = workload(0, sigma=sigma)
    run_codec(w, f"cfg0 sigma={sigma}")
    cfg = w["cfg"]
    (rows, cols), = cfg.weights
    Wnp = synth.make_weight(0, 0, rows, cols)
    W = dev(Wnp, "f32")
    basis = sn.sn_basis_pack(dev(w["U"], "f32"))
    sn.sn_project_weights(basis, W)
    ref = oracle.round_to(oracle.project_weights(Wnp.astype(np.float64),
                                                 w["U"].astype(np.float64)), "f32")
    assert_parity(host(W), ref, "f32", "cfg0 project_weights")


def test_config1_bf16_full():
    run_codec(workload(1), "cfg1")


# configs 2 and 4 at full size (config 4 also with 32767 tokens: a short last
# sequence), one test per op so that each stays well inside the time limit;
# the GPU runs the four ops once per workload
_FULL = [(cfg, n, op) for cfg, n in ((2, None), (4, 32768), (4, 32767)) for op in OPS]


@pytest.mark.parametrize("cfg,n,op", _FULL, ids=[f"cfg{c}-N{n or 32768}-{o}" for c, n, o in _FULL])
def test_config_full(cfg, n, op):
    w = workload(cfg, n=n)
    tag = f"cfg{cfg} N={w['tok'].shape[0]}"
    check_op(w, codec_outputs(w, (cfg, n)), op, tag)


def check_projection(before: np.ndarray, after: np.ndarray, U64: np.ndarray, tag: str):
    """Every column of a projected weight against the oracle, plus the
    properties of the projection on the GPU result: U^T W' = U^T W and no
    off-subspace part, per column (bf16 rounding of W' and the stored,
    not exactly orthonormal bf16 U leave ~1e-3 of each column's norm)."""
    assert_parity_rows(after.T, lambda r: oracle.project_weights(before, U64, cols=r).T,
                       "bf16", f"{tag} project_weights (every column)")
    m = before.shape[1]
    step = 4096
    for c0 in range(0, m, step):
        bf = before[:, c0:c0 + step].astype(np.float64)
        af = after[:, c0:c0 + step].astype(np.float64)
        t_before, t_after = U64.T @ bf, U64.T @ af
        dt_col = np.linalg.norm(t_after - t_before, axis=0)
        assert np.all(dt_col <= 1e-2 * np.linalg.norm(t_before, axis=0) + 1e-30), \
            f"{tag}: U^T W changed in columns {np.flatnonzero(dt_col > 1e-2 * np.linalg.norm(t_before, axis=0))[:5] + c0}"
        resid = np.linalg.norm(af - U64 @ t_after, axis=0)
        assert np.all(resid <= 1e-2 * np.linalg.norm(af, axis=0) + 1e-30), \
            f"{tag}: off-subspace part left in columns {np.flatnonzero(resid > 1e-2 * np.linalg.norm(af, axis=0))[:5] + c0}"
    log(f"  {tag}: U^T W kept, no off-subspace part ({m} columns)")


def _basis_of(cfg_id: int):
    b = synth.make_basis(cfg_id)
    return oracle.decode_bf16(b["U"]), sn.sn_basis_pack(dev(b["U"], "bf16"))


def test_project_weights_config2_wo_w2():
    """Config 2's Wo (4096 x 4096) and W2 (4096 x 14336) confined by one
    call, as the optimizer step (and the benchmark) does it; every column."""
    cfg = synth.CONFIGS[2]
    U64, basis = _basis_of(2)
    hosts = [synth.make_weight(2, i, r, c) for i, (r, c) in enumerate(cfg.weights)]
    Ws = [dev(h, "bf16") for h in hosts]
    log("[cfg2] project Wo and W2 in one call")
    sn.sn_project_weights_multi(basis, Ws)
    for i, (h, W) in enumerate(zip(hosts, Ws)):
        check_projection(oracle.decode_bf16(h, np.float32), host_f32(W), U64, f"cfg2 W{i}")


def test_project_weights_config4_wo():
    """Config 4's Wo (8192 x 8192, k = 82); every column."""
    cfg = synth.CONFIGS[4]
    U64, basis = _basis_of(4)
    (r, c), = cfg.weights
    h = synth.make_weight(4, 0, r, c)
    W = dev(h, "bf16")
    log("[cfg4] project Wo")
    sn.sn_project_weights(basis, W)
    check_projection(oracle.decode_bf16(h, np.float32), host_f32(W), U64, "cfg4 Wo")


@pytest.mark.parametrize("group", range(4))
def test_config3_layer_sweep(group):
    """The 32-layer sweep of (Wo, W2), in the benchmark's calls of 16 matrices
    (8 layers) each; this test is call `group`.  Weights are drawn on the
    device (seeded); each matrix is copied to the host before and after, and
    every column of all 16 is compared with the oracle."""
    cfg = synth.CONFIGS[3]
    U64, basis = _basis_of(3)
    mats, names = [], []
    for layer in range(8 * group, 8 * group + 8):
        for i, (r, c) in enumerate(cfg.weights):
            mats.append(synth.device_weight(3, 2 * layer + i, r, c))
            names.append(f"cfg3 L{layer} W{i}")
    before = [host_f32(W) for W in mats]
    log(f"[cfg3] call {group}: layers {8 * group}..{8 * group + 7}, 16 matrices")
    sn.sn_project_weights_multi(basis, mats)
    after = [host_f32(W) for W in mats]
    del mats
    torch.cuda.empty_cache()
    for name, bf, af in zip(names, before, after):
        check_projection(bf, af, U64, name)


# --------------------------------------------------------------- edge cases

def _small(d, k, n, vocab=50, seq=9, dtype="bf16", seed=0, grid=None):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.standard_normal((vocab, d)) * 0.05
    P = rng.standard_normal((seq, d)) * 0.05
    C = rng.standard_normal((n, k))
    tok = rng.integers(0, vocab, n).astype(np.int32)
    pos = (np.arange(n) % seq).astype(np.int32)
    X = E[tok] + P[pos] + C @ U.T + rng.standard_normal((n, d)) * 0.01
    G = rng.standard_normal((n, d)) * 0.1
    if grid:
        E, P, X = (np.round(a * grid) / grid for a in (E, P, X))
    st = {name: synth.store(a, dtype) for name, a in
          dict(U=U, E=E, P=P, C=C, X=X, G=G).items()}
    f64 = {name: (oracle.decode_bf16(a) if dtype == "bf16" else a.astype(np.float64))
           for name, a in st.items()}
    return st, f64, tok, pos


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,k,n", [(256, 20, 1), (256, 20, 17), (256, 20, 33), (256, 1, 40),
                                   (256, 16, 31), (256, 17, 50), (256, 33, 16), (256, 82, 45),
                                   (256, 128, 20), (384, 130, 19), (200, 20, 37), (96, 5, 64)])
def test_shapes(dtype, d, k, n):
    log(f"[shapes] {dtype} d={d} k={k} n={n}")
    st, o, tok, pos = _small(d, k, n, dtype=dtype, seed=d + k + n)
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X, G, Cin = (dev(st[x], dtype) for x in ("E", "P", "X", "G", "C"))
    t_tok = ids(tok)
    C = sn.sn_compress(basis, X, tok=t_tok, E=E, P=P, seq_len=9)
    assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], tok, o["E"], o["P"],
                                                           seq_len=9), dtype), dtype, "compress")
    Xr = sn.sn_decompress(basis, Cin, tok=t_tok, E=E, P=P, seq_len=9)
    assert_parity(host(Xr), oracle.round_to(oracle.decompress(o["C"], o["U"], tok, o["E"],
                                                              o["P"], seq_len=9), dtype),
                  dtype, "decompress")
    Cg = sn.sn_grad_compress(basis, G)
    assert_parity(host(Cg), oracle.round_to(oracle.grad_compress(o["G"], o["U"]), dtype), dtype,
                  "grad_compress")
    W = G[: min(n, 64)].T.contiguous() if n >= 1 else None   # d x m
    Wn = host(W)
    sn.sn_project_weights(basis, W)
    assert_parity(host(W).T, oracle.round_to(oracle.project_weights(Wn, o["U"]), dtype).T,
                  dtype, "project_weights")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_tables_optional_and_explicit_positions(dtype):
    d, k, n = 256, 24, 70
    st, o, tok, _ = _small(d, k, n, dtype=dtype, seed=5)
    rng = np.random.default_rng(6)
    pos = rng.integers(0, 9, n).astype(np.int32)      # arbitrary (e.g. context-parallel) positions
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X, Cin = (dev(st[x], dtype) for x in ("E", "P", "X", "C"))
    cases = [("E+P explicit pos", dict(tok=ids(tok), E=E, P=P, pos=ids(pos)),
              dict(tok=tok, E=o["E"], P=o["P"], pos=pos)),
             ("E only", dict(tok=ids(tok), E=E), dict(tok=tok, E=o["E"])),
             ("P only default pos", dict(P=P, seq_len=9), dict(P=o["P"], seq_len=9)),
             ("no tables", {}, {})]
    for name, gk, ok in cases:
        C = sn.sn_compress(basis, X, **gk)
        assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], **ok), dtype),
                      dtype, f"compress {name}")
        Xr = sn.sn_decompress(basis, Cin, **gk)
        assert_parity(host(Xr), oracle.round_to(oracle.decompress(o["C"], o["U"], **ok), dtype),
                      dtype, f"decompress {name}")


@pytest.mark.parametrize("n", [187, 184, 183, 511, 512])
def test_decompress_short_last_sequence(n):
    """Default positions of [batch, seq] rows whose last sequence is short
    (seq = 64: 5, 8, 9, 1 and 0 rows missing).  Up to an eighth of a
    sequence missing, the decompress keeps position-major tiles over whole
    sequences and does not store the missing rows; beyond that it takes
    token-major tiles.  Every element against the oracle, rows past N
    untouched, no out-of-range flag."""
    d, k, seq = 256, 20, 64
    log(f"[short last sequence] n={n}")
    st, o, tok, _ = _small(d, k, n, vocab=40, seq=seq, seed=n)
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    E, P, Cin = (dev(st[x], "bf16") for x in ("E", "P", "C"))
    for name, gk, ok in [("E+P", dict(tok=ids(tok), E=E), dict(tok=tok, E=o["E"])),
                         ("P only", {}, {})]:
        big = torch.full((n + 64, d), 3.0, dtype=torch.bfloat16, device="cuda")
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        sn.sn_decompress(basis, Cin, P=P, seq_len=seq, out=big[:n], err_flag=flag, **gk)
        ref = oracle.decompress(o["C"], o["U"], P=o["P"], seq_len=seq, **ok)
        assert_parity(host(big[:n]), oracle.round_to(ref, "bf16"), "bf16", f"{name} n={n}")
        assert bool((big[n:] == 3.0).all()), f"{name}: rows past N were written"
        assert int(flag.item()) == 0, f"{name}: out-of-range flag {int(flag.item())}"


@pytest.mark.parametrize("n,batch", [(256, 4), (255, 4), (249, 4), (248, 4), (247, 4),
                                     (512, 8), (511, 8), (504, 8), (503, 8)])
def test_compress_short_last_sequence(n, batch):
    """Default positions of [batch, seq] rows (seq = 64) whose last sequence
    is short by 0, 1, 7, 8 or 9 rows.  Up to an eighth of a sequence missing,
    the compress keeps position-major tiles over whole sequences (the missing
    rows are loaded as the last token's and not stored); beyond that it takes
    token-major tiles.  Every element against the oracle, rows past N of the
    output untouched, no out-of-range flag."""
    d, k, seq = 256, 40, 64
    assert batch * seq - 9 <= n <= batch * seq
    log(f"[compress short last sequence] n={n} batch={batch}")
    st, o, tok, _ = _small(d, k, n, vocab=40, seq=seq, seed=n + 1000)
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    E, P, X = (dev(st[x], "bf16") for x in ("E", "P", "X"))
    for name, gk, ok in [("E+P", dict(tok=ids(tok), E=E), dict(tok=tok, E=o["E"])),
                         ("P only", {}, {})]:
        big = torch.full((n + 16, k), 3.0, dtype=torch.bfloat16, device="cuda")
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        sn.sn_compress(basis, X, P=P, seq_len=seq, out=big[:n], err_flag=flag, **gk)
        ref = oracle.compress(o["X"], o["U"], P=o["P"], seq_len=seq, **ok)
        assert_parity(host(big[:n]), oracle.round_to(ref, "bf16"), "bf16", f"{name} n={n}")
        assert bool((big[n:] == 3.0).all()), f"{name}: rows past N were written"
        assert int(flag.item()) == 0, f"{name}: out-of-range flag {int(flag.item())}"


def test_large_positional_table_streamed():
    """Both tables with a positional table over 64 MiB: compress and
    decompress then load P's rows non-temporally (a kernel variant of the
    decompress, a run-time copy policy of the compress).  Every element is
    compared: default positions of two whole sequences (position-major
    tiles) and explicit scattered positions over a ragged batch."""
    d, k, seq = 4096, 40, 8208          # P: 8208 x 4096 bf16 = 67.2 MB > 64 MiB
    n = 2 * seq
    log(f"[streamed P] d={d} k={k} seq={seq} n={n}")
    st, o, tok, _ = _small(d, k, n, vocab=300, seq=seq, seed=11)
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    E, P, X, Cin = (dev(st[x], "bf16") for x in ("E", "P", "X", "C"))
    t_tok = ids(tok)
    C = sn.sn_compress(basis, X, tok=t_tok, E=E, P=P, seq_len=seq)
    assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], tok, o["E"], o["P"],
                                                           seq_len=seq), "bf16"),
                  "bf16", "compress, default positions")
    Xr = sn.sn_decompress(basis, Cin, tok=t_tok, E=E, P=P, seq_len=seq)
    assert_parity(host(Xr), oracle.round_to(oracle.decompress(o["C"], o["U"], tok, o["E"], o["P"],
                                                              seq_len=seq), "bf16"),
                  "bf16", "decompress, default positions")
    m = 1001                            # ragged, scattered explicit positions
    pos = np.random.default_rng(12).integers(0, seq, m).astype(np.int32)
    C = sn.sn_compress(basis, X[:m], tok=ids(tok[:m]), E=E, P=P, pos=ids(pos))
    assert_parity(host(C), oracle.round_to(oracle.compress(o["X"][:m], o["U"], tok[:m], o["E"],
                                                           o["P"], pos=pos), "bf16"),
                  "bf16", "compress, explicit positions")
    Xr = sn.sn_decompress(basis, Cin[:m], tok=ids(tok[:m]), E=E, P=P, pos=ids(pos))
    assert_parity(host(Xr), oracle.round_to(oracle.decompress(o["C"][:m], o["U"], tok[:m],
                                                              o["E"], o["P"], pos=pos), "bf16"),
                  "bf16", "decompress, explicit positions")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_strides_and_guard_canaries(dtype):
    """Row strides larger than the row; nothing is written outside the N x k
    (resp. N x d) region of a padded output buffer."""
    d, k, n = 256, 40, 37
    st, o, tok, _ = _small(d, k, n, dtype=dtype, seed=7)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P = dev(st["E"], dtype), dev(st["P"], dtype)
    for ldx_pad in (8, 1):
        Xbig = torch.zeros(n, d + ldx_pad, dtype=tdt, device="cuda")
        Xbig[:, :d] = dev(st["X"], dtype)
        X = Xbig[:, :d]
        Cbig = torch.full((n + 3, k + 5), 7.0, dtype=tdt, device="cuda")
        C = Cbig[:n, :k]
        sn.sn_compress(basis, X, tok=ids(tok), E=E, P=P, seq_len=9, out=C)
        assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], tok, o["E"],
                                                               o["P"], seq_len=9), dtype),
                      dtype, f"compress ldx=d+{ldx_pad} ldc=k+5")
        cb = host(Cbig)
        assert np.all(cb[n:] == 7.0) and np.all(cb[:, k:] == 7.0), "compress wrote outside C"
        Obig = torch.full((n + 2, d + 16), 7.0, dtype=tdt, device="cuda")
        Xo = Obig[:n, :d + (0 if ldx_pad == 8 else 0)]
        Cin = dev(st["C"], dtype)
        sn.sn_decompress(basis, Cin, tok=ids(tok), E=E, P=P, seq_len=9, out=Xo)
        assert_parity(host(Xo), oracle.round_to(oracle.decompress(o["C"], o["U"], tok, o["E"],
                                                                  o["P"], seq_len=9), dtype),
                      dtype, "decompress into strided output")
        ob = host(Obig)
        assert np.all(ob[n:] == 7.0) and np.all(ob[:, d:] == 7.0), "decompress wrote outside X"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_out_of_range_ids_are_clamped_and_flagged(dtype):
    d, k, n, vocab = 256, 20, 40, 50
    st, o, tok, _ = _small(d, k, n, vocab=vocab, dtype=dtype, seed=9)
    bad_tok = tok.copy()
    bad_tok[3], bad_tok[20] = vocab + 5, -2
    pos = (np.arange(n) % 9).astype(np.int32)
    bad_pos = pos.copy()
    bad_pos[7] = 100
    basis = sn.sn_basis_pack(dev(st["U"], dtype))
    E, P, X, Cin = (dev(st[x], dtype) for x in ("E", "P", "X", "C"))
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    C = sn.sn_compress(basis, X, tok=ids(bad_tok), E=E, P=P, pos=ids(bad_pos), err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 3
    ct, cp = np.clip(bad_tok, 0, vocab - 1), np.clip(bad_pos, 0, 8)
    assert_parity(host(C), oracle.round_to(oracle.compress(o["X"], o["U"], ct, o["E"], o["P"],
                                                           pos=cp), dtype), dtype,
                  "compress with clamped ids")
    flag.zero_()
    Xr = sn.sn_decompress(basis, Cin, tok=ids(bad_tok), E=E, err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1
    assert_parity(host(Xr), oracle.round_to(oracle.decompress(o["C"], o["U"], ct, o["E"]),
                                            dtype), dtype, "decompress with clamped ids")


@pytest.mark.parametrize("pattern", ["one id", "all distinct", "two ids", "zipf"])
@pytest.mark.parametrize("n,seq,d", [(512, 64, 512), (500, 50, 512), (1024, 32, 512),
                                     (32768, 4096, 256), (32768, 64, 256), (32769, 32769, 256)])
def test_compress_token_id_patterns(pattern, n, seq, d):
    """The compress copies each distinct T_fixed row of a workgroup once and
    maps every token to its row: ids that all repeat, never repeat, alternate,
    or follow Zipf, in position-major (n = batch x seq, batch 8, 32 or 512)
    and token-major (500 and 32769 tokens) order; at 32768 tokens the
    workgroups hold 128 tokens (two per lane of the id scan), below that 64."""
    k = 40
    vocab = n + 5 if pattern == "all distinct" else 700
    log(f"[id patterns] {pattern} n={n} seq={seq}")
    rng = np.random.default_rng(n + len(pattern))
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.standard_normal((vocab, d)) * 0.05
    P = rng.standard_normal((seq, d)) * 0.05
    tok = {"one id": np.full(n, 17),
           "all distinct": rng.permutation(vocab)[:n],
           "two ids": np.where(np.arange(n) % 2 == 0, 3, vocab - 1),
           "zipf": np.minimum(rng.zipf(1.1, n), vocab) - 1}[pattern].astype(np.int32)
    pos = (np.arange(n) % seq).astype(np.int32)
    X = E[tok] + P[pos] + rng.standard_normal((n, d)) * 0.05
    st = {nm: synth.store(a, "bf16") for nm, a in dict(U=U, E=E, P=P, X=X).items()}
    f64 = {nm: oracle.decode_bf16(a) for nm, a in st.items()}
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    C = sn.sn_compress(basis, dev(st["X"], "bf16"), tok=ids(tok), E=dev(st["E"], "bf16"),
                       P=dev(st["P"], "bf16"), seq_len=seq)
    ref = oracle.round_to(oracle.compress(f64["X"], f64["U"], tok, f64["E"], f64["P"],
                                          seq_len=seq), "bf16")
    assert_parity(host(C), ref, "bf16", f"compress, {pattern}")


@pytest.mark.parametrize("tables", ["E only", "P only"])
def test_compress_one_table_128_token_workgroups(tables):
    """One gathered table at 32768 tokens (the 128-token workgroups): T_fixed
    alone (distinct-row copies, no positional rows) or P alone
    (position-major positional rows, no T_fixed)."""
    d, k, n, seq, vocab = 256, 40, 32768, 4096, 2000
    log(f"[one table] {tables} n={n}")
    rng = np.random.default_rng(77 if tables == "E only" else 78)
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.standard_normal((vocab, d)) * 0.05
    P = rng.standard_normal((seq, d)) * 0.05
    tok = (np.minimum(rng.zipf(1.1, n), vocab) - 1).astype(np.int32)
    pos = (np.arange(n) % seq).astype(np.int32)
    use_e, use_p = tables == "E only", tables == "P only"
    X = (E[tok] if use_e else 0) + (P[pos] if use_p else 0) + rng.standard_normal((n, d)) * 0.05
    st = {nm: synth.store(a, "bf16") for nm, a in dict(U=U, E=E, P=P, X=X).items()}
    f64 = {nm: oracle.decode_bf16(a) for nm, a in st.items()}
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    kw = dict(tok=ids(tok), E=dev(st["E"], "bf16")) if use_e else dict(P=dev(st["P"], "bf16"),
                                                                      seq_len=seq)
    C = sn.sn_compress(basis, dev(st["X"], "bf16"), **kw)
    ref = oracle.round_to(oracle.compress(f64["X"], f64["U"], tok if use_e else None,
                                          f64["E"] if use_e else None,
                                          f64["P"] if use_p else None,
                                          seq_len=seq if use_p else None), "bf16")
    assert_parity(host(C), ref, "bf16", f"compress, {tables}")


def test_bit_exact_gather_and_subtract():
    """C = 0 decompresses to exactly E[tok] + P[pos] (bit-exact gathers);
    X = E[tok] + P[pos] (values on a grid where every sum is exact)
    compresses to 0 within the fp32 accumulation bound of the fused
    subtract-and-project."""
    d, k, n = 256, 40, 70
    rng = np.random.default_rng(12)
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.integers(-64, 64, (30, d)) / 64.0
    P = rng.integers(-64, 64, (9, d)) / 64.0
    tok = rng.integers(0, 30, n).astype(np.int32)
    pos = (np.arange(n) % 9).astype(np.int32)
    for dtype in ("bf16", "f32"):
        st = {nm: synth.store(a, dtype) for nm, a in dict(U=U, E=E, P=P).items()}
        basis = sn.sn_basis_pack(dev(st["U"], dtype))
        Et, Pt = dev(st["E"], dtype), dev(st["P"], dtype)
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        Z = torch.zeros(n, k, dtype=tdt, device="cuda")
        Xr = sn.sn_decompress(basis, Z, tok=ids(tok), E=Et)
        assert np.array_equal(host_bits(Xr), host_bits(Et[ids(tok).long()])), "E gather"
        Xr = sn.sn_decompress(basis, Z, P=Pt, seq_len=9)
        assert np.array_equal(host_bits(Xr), host_bits(Pt[ids(pos).long()])), "P gather"
        Xr = sn.sn_decompress(basis, Z, tok=ids(tok), E=Et, P=Pt, seq_len=9)
        assert np.array_equal(host(Xr), E[tok] + P[pos]), "E + P gather"
        # compress of X = E[tok] + P[pos]: the embedding rows cancel X exactly.
        # In exact arithmetic C = 0.  The matrix-core path sums the products of
        # X, -P and -T_fixed with U in one set of fp32 accumulators, so C is
        # zero up to that accumulation's rounding, bounded by
        # d * 2^-24 * sum |terms|; subtracting a wrong row would leave entries
        # of size ~|x| |u| ~ 1e-1.
        X = dev(synth.store(E[tok] + P[pos], dtype), dtype)
        C = host(sn.sn_compress(basis, X, tok=ids(tok), E=Et, P=Pt, seq_len=9))
        Ud = oracle.decode_bf16(st["U"]) if dtype == "bf16" else st["U"].astype(np.float64)
        absum = (np.abs(E[tok] + P[pos]) + np.abs(E[tok]) + np.abs(P[pos])) @ np.abs(Ud)
        assert np.all(np.abs(C) <= d * 2.0 ** -24 * absum), "subtract of the gathered rows"
        log(f"  bit-exact gather, cancelling subtract ok ({dtype}); max |C| {np.abs(C).max():.3g}")


def test_decompress_cancelling_tables():
    """P[pos] = -T_fixed[tok] for every token: the tables cancel exactly and
    X' is C U^T alone, although each table entry is ~64 times the result.
    The sum of three addends must keep the small one (Sec. 4.3.1 recovery)."""
    d, k, seq, batch = 512, 40, 64, 4
    n = seq * batch
    rng = np.random.default_rng(31)
    U, _ = np.linalg.qr(rng.standard_normal((d, k)))
    E = rng.integers(-4096, 4096, (seq, d)) / 64.0
    P = -E
    tok = (np.arange(n) % seq).astype(np.int32)
    Cin = rng.standard_normal((n, k))
    for dtype in ("bf16", "f32"):
        st = {nm: synth.store(a, dtype) for nm, a in dict(U=U, E=E, P=P, C=Cin).items()}
        basis = sn.sn_basis_pack(dev(st["U"], dtype))
        Xr = host(sn.sn_decompress(basis, dev(st["C"], dtype), tok=ids(tok),
                                   E=dev(st["E"], dtype), P=dev(st["P"], dtype), seq_len=seq))
        val = (lambda a: oracle.decode_bf16(a)) if dtype == "bf16" else (
            lambda a: a.astype(np.float64))
        ref = oracle.decompress(val(st["C"]), val(st["U"]), tok=tok, E=val(st["E"]),
                                P=val(st["P"]), seq_len=seq)
        assert_parity(Xr, ref, dtype, f"decompress, cancelling tables ({dtype})")


def test_output_rounding_ties_to_even():
    """Outputs are rounded once, to nearest even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6."""
    d, k = 64, 8
    U = np.eye(d)[:, :k]
    E = np.ones((2, d))
    E[1] += 2.0 ** -7
    P = np.full((1, d), 2.0 ** -8)
    tok = np.array([0, 1], dtype=np.int32)
    st = {nm: synth.store(a, "bf16") for nm, a in dict(U=U, E=E, P=P).items()}
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    Z = torch.zeros(2, k, dtype=torch.bfloat16, device="cuda")
    Xr = host(sn.sn_decompress(basis, Z, tok=ids(tok), E=dev(st["E"], "bf16"),
                               P=dev(st["P"], "bf16"), seq_len=1))
    ref = oracle.round_bf16(E[tok] + P[[0, 0]])
    assert np.array_equal(Xr, ref)
    assert np.all(Xr[0] == 1.0) and np.all(Xr[1] == 1.0 + 2.0 ** -6)


def test_empty_batch_is_a_no_op():
    st, o, tok, _ = _small(64, 8, 5, dtype="bf16")
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    X = torch.zeros(0, 64, dtype=torch.bfloat16, device="cuda")
    C = sn.sn_compress(basis, X, tok=ids(np.zeros(0, np.int32)), E=dev(st["E"], "bf16"))
    assert C.shape == (0, 8)
    Xr = sn.sn_decompress(basis, torch.zeros(0, 8, dtype=torch.bfloat16, device="cuda"))
    assert Xr.shape == (0, 64)


def test_deterministic_bitwise():
    w = workload(1)
    dt = "bf16"
    basis = sn.sn_basis_pack(dev(w["U"], dt))
    X, E, P, Cin = dev(w["X"], dt), dev(w["E"], dt), dev(w["P"], dt), dev(synth.store(w["C_true"], dt), dt)
    tok = ids(w["tok"])
    c1 = host_bits(sn.sn_compress(basis, X, tok=tok, E=E, P=P, seq_len=w["cfg"].seq))
    c2 = host_bits(sn.sn_compress(basis, X, tok=tok, E=E, P=P, seq_len=w["cfg"].seq))
    assert np.array_equal(c1, c2)
    x1 = host_bits(sn.sn_decompress(basis, Cin, tok=tok, E=E, P=P, seq_len=w["cfg"].seq))
    x2 = host_bits(sn.sn_decompress(basis, Cin, tok=tok, E=E, P=P, seq_len=w["cfg"].seq))
    assert np.array_equal(x1, x2)


@pytest.mark.parametrize("dtype,d,k,widths,pad", [
    ("bf16", 4096, 40, (4096, 14336), 0),      # config 2's Wo and W2 side by side
    # wide calls (one launch per pass over 16384 or more columns), k from 8 to 64
    ("bf16", 256, 8, (16384,), 0),
    ("bf16", 512, 20, (8192, 8192, 2048), 8),  # three segments, strided rows
    ("bf16", 384, 64, (16384, 256), 0),
    ("bf16", 512, 40, (256, 768, 512), 8),     # strided rows
    ("bf16", 512, 40, (300, 512), 0),          # a width not a multiple of 256: one by one
    ("bf16", 512, 100, (256, 512), 0),         # k > 64: one by one
    ("f32", 256, 8, (256, 100), 0)])
def test_project_weights_multi(dtype, d, k, widths, pad):
    log(f"[project multi] {dtype} d={d} k={k} widths={widths} pad={pad}")
    cfg = synth.Config("multi", dtype, d, k, 10, 1, 1, False, 0.0, 1.0)
    b = synth.make_basis(0, cfg)
    U = (oracle.decode_bf16(b["U"], np.float32) if dtype == "bf16" else b["U"]).astype(np.float64)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    hosts, Ws = [], []
    for i, m in enumerate(widths):
        Wh = synth.make_weight(0, i, d, m, cfg)
        hosts.append(Wh)
        full = torch.zeros(d, m + pad, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                           device="cuda")
        full[:, :m] = dev(Wh, dtype)
        Ws.append(full[:, :m] if pad else full)
    sn.sn_project_weights_multi(basis, Ws)
    torch.cuda.synchronize()
    for i, (m, Wh) in enumerate(zip(widths, hosts)):
        Wf = oracle.decode_bf16(Wh, np.float32) if dtype == "bf16" else Wh
        got = host_f32(Ws[i])
        assert_parity_rows(got.T, lambda r: oracle.project_weights(Wf, U, cols=r).T, dtype,
                           f"W[{i}] ({d}x{m}) every column")
        if pad:  # the padding columns are untouched
            assert float(Ws[i].as_strided((d, pad), (m + pad, 1), m).abs().max()) == 0.0


def test_id_check_mode_raises_index_error():
    """With id checking on, a call with an out-of-range id raises
    SnError(SN_ERR_INDEX) after the call, the caller's flag still receives
    the bits, and in-range ids raise nothing."""
    d, k, n, vocab = 256, 20, 40, 50
    st, o, tok, _ = _small(d, k, n, vocab=vocab, seed=9)
    basis = sn.sn_basis_pack(dev(st["U"], "bf16"))
    E, P, X, Cin = (dev(st[x], "bf16") for x in ("E", "P", "X", "C"))
    bad_tok = tok.copy()
    bad_tok[5] = vocab + 1
    sn.set_check_ids(True)
    try:
        sn.sn_compress(basis, X, tok=ids(tok), E=E, P=P, seq_len=9)       # in range: no error
        sn.sn_decompress(basis, Cin, tok=ids(tok), E=E, P=P, seq_len=9)
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        with pytest.raises(sn.SnError) as ei:
            sn.sn_compress(basis, X, tok=ids(bad_tok), E=E, P=P, seq_len=9, err_flag=flag)
        assert ei.value.status == sn.SN_ERR_INDEX
        assert int(flag.item()) == 1
        bad_pos = (np.arange(n) % 9).astype(np.int32)
        bad_pos[3] = 99
        with pytest.raises(sn.SnError) as ei:
            sn.sn_decompress(basis, Cin, P=P, pos=ids(bad_pos))
        assert ei.value.status == sn.SN_ERR_INDEX and "flag bits 2" in str(ei.value)
    finally:
        sn.set_check_ids(False)
    # checking off: the same call returns normally and only the flag reports
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    sn.sn_compress(basis, X, tok=ids(bad_tok), E=E, P=P, seq_len=9, err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1

"""Seeded synthetic inputs for the stage-boundary subspace codec.

This module is shared by the CPU oracle's tests and the GPU path's tests and
benchmark.  It builds INPUTS only: it holds no compress / decompress /
projection routine and nothing here is ever used to produce an expected value.

Every tensor is drawn on the host with numpy ``Generator(PCG64(seed))`` where
``seed = 1260 + 100 * cfg + ordinal`` (ordinal: 0 U, 1 E, 2 P, 3 tok,
4 C_true, 5 noise, 6 G, 7 + i weight matrix i, 71 / 72 the AdamW moments,
73 + t the weight gradient of optimizer step t, 79 the dominant gradient
directions and 80 + t the gradient of iteration t of the subspace update).  Large tensors are drawn in
fixed row blocks of ``ROW_BLOCK`` rows, block b using ``SeedSequence([seed, b])``,
so a tensor's values do not depend on how callers slice it.

Shapes and distributions follow the paper's workloads (Section 8.1: d=4096,
k=40, context 1024-4096, Llama-style vocabularies); natural-text token ids are
stood in for by a truncated Zipf(1.1) law.

bf16 tensors are returned as ``uint16`` bit patterns (numpy has no bf16);
fp32 tensors as ``float32``.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import os

import numpy as np

ROW_BLOCK = 4096
SEED_BASE = 1260


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload: sizes and value distributions."""
    name: str
    dtype: str            # "f32" or "bf16": dtype of X, G, E, P, U, C, W
    d: int
    k: int
    vocab: int
    batch: int
    seq: int
    zipf: bool            # Zipf(1.1) token ids, else uniform
    sigma: float          # std of the off-subspace noise added to X
    g_std: float          # std of the activation gradient G
    weights: tuple = ()   # ((rows, cols), ...) weight matrices to project
    layers: int = 1       # how many copies of `weights` (the 32-layer sweep)

    @property
    def n_tokens(self) -> int:
        return self.batch * self.seq


CONFIGS = {
    0: Config("tiny-f32 d256 k8", "f32", 256, 8, 1024, 4, 128, False, 1e-3, 1.0,
              weights=((256, 256),)),
    1: Config("d2048 k20 N16384", "bf16", 2048, 20, 32000, 8, 2048, True, 1e-2, 1e-2),
    2: Config("d4096 k40 N32768", "bf16", 4096, 40, 32000, 8, 4096, True, 1e-2, 1e-2,
              weights=((4096, 4096), (4096, 14336))),
    3: Config("weight sweep 32 layers d4096 k40", "bf16", 4096, 40, 32000, 8, 4096, True,
              1e-2, 1e-2, weights=((4096, 4096), (4096, 14336)), layers=32),
    4: Config("d8192 k82 N32768", "bf16", 8192, 82, 128256, 4, 8192, True, 1e-2, 1e-2,
              weights=((8192, 8192),)),
}

ORD_U, ORD_E, ORD_P, ORD_TOK, ORD_C, ORD_NOISE, ORD_G, ORD_W = range(8)
ORD_AM, ORD_AV = 71, 72   # AdamW moments M, V of the optimizer-step inputs
ORD_AG = 73        # 73 + t: weight gradient of optimizer step t (t < 6)
ORD_GV = 79        # fixed dominant gradient directions of the subspace-update inputs
ORD_GT = 80        # 80 + t: activation gradient of accumulated iteration t (t < 20)


def seed_of(cfg: int, ordinal: int) -> int:
    return SEED_BASE + 100 * cfg + ordinal


def _rng(seed: int, block: int | None = None) -> np.random.Generator:
    if block is None:
        return np.random.Generator(np.random.PCG64(seed))
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, block])))


# --------------------------------------------------------------------------
# bf16 storage helpers for inputs.  Rounding of generated inputs goes through
# torch's float32 -> bfloat16 conversion (round to nearest even); decoding is
# the exact 16-bit shift.  These only prepare inputs.
# --------------------------------------------------------------------------

def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def store(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float array to the storage dtype ('f32' or 'bf16' bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        return to_bf16_bits(a)
    raise ValueError(dtype)


def as_float(a: np.ndarray, dtype: str) -> np.ndarray:
    """Stored array -> float32 values (exact)."""
    return bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# Individual tensors
# --------------------------------------------------------------------------

def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _blocks(rows: int):
    return list(enumerate(range(0, rows, ROW_BLOCK)))


def _parallel(fn, items):
    """Run fn over row blocks on a thread pool (numpy's generators and BLAS
    release the GIL); each block has its own seed, so results do not depend on
    the number of threads."""
    with cf.ThreadPoolExecutor(max_workers=_workers()) as ex:
        list(ex.map(fn, items))


def gaussian(seed: int, rows: int, cols: int, std: float) -> np.ndarray:
    """float32 N(0, std^2) matrix drawn in ROW_BLOCK row blocks."""
    out = np.empty((rows, cols), dtype=np.float32)

    def one(item):
        b, r0 = item
        r1 = min(rows, r0 + ROW_BLOCK)
        blk = _rng(seed, b).standard_normal((r1 - r0, cols), dtype=np.float32)
        blk *= np.float32(std)
        out[r0:r1] = blk

    _parallel(one, _blocks(rows))
    return out


def orthonormal_basis(seed: int, d: int, k: int) -> np.ndarray:
    """U (d x k): QR of an isotropic Gaussian matrix, column signs fixed so
    that diag(R) > 0 (Section 8.1 initialises U from isotropic Gaussian noise;
    Section 4.3 requires orthonormal columns).  Returned in float64."""
    g = _rng(seed).standard_normal((d, k))
    q, r = np.linalg.qr(g)
    s = np.sign(np.diag(r))
    s[s == 0] = 1.0
    return q * s


def zipf_ids(seed: int, n: int, vocab: int, a: float = 1.1) -> np.ndarray:
    """Truncated Zipf(a) over ranks 1..vocab, p(r) ~ r^-a, inverse-CDF sampled;
    rank r maps to id r-1."""
    r = np.arange(1, vocab + 1, dtype=np.float64)
    p = r ** (-a)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = _rng(seed).random(n)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, vocab - 1).astype(np.int32)


def uniform_ids(seed: int, n: int, vocab: int) -> np.ndarray:
    return _rng(seed).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def default_positions(n: int, seq: int) -> np.ndarray:
    """Positions of a row-major [batch, seq] token layout."""
    return (np.arange(n, dtype=np.int64) % seq).astype(np.int32)


# --------------------------------------------------------------------------
# Whole workloads
# --------------------------------------------------------------------------

def make_basis(cfg_id: int, cfg: Config | None = None) -> dict:
    cfg = cfg or CONFIGS[cfg_id]
    u64 = orthonormal_basis(seed_of(cfg_id, ORD_U), cfg.d, cfg.k)
    return {"U": store(u64, cfg.dtype), "U64": u64}


def make_embeddings(cfg_id: int, cfg: Config | None = None) -> dict:
    cfg = cfg or CONFIGS[cfg_id]
    E = gaussian(seed_of(cfg_id, ORD_E), cfg.vocab, cfg.d, 0.02)
    P = gaussian(seed_of(cfg_id, ORD_P), cfg.seq, cfg.d, 0.02)
    return {"E": store(E, cfg.dtype), "P": store(P, cfg.dtype)}


def make_ids(cfg_id: int, n: int | None = None, cfg: Config | None = None) -> dict:
    cfg = cfg or CONFIGS[cfg_id]
    n = cfg.n_tokens if n is None else n
    s = seed_of(cfg_id, ORD_TOK)
    tok = zipf_ids(s, n, cfg.vocab) if cfg.zipf else uniform_ids(s, n, cfg.vocab)
    return {"tok": tok, "pos": default_positions(n, cfg.seq)}


def make_activations(cfg_id: int, basis: dict, emb: dict, ids: dict,
                     sigma: float | None = None, cfg: Config | None = None) -> dict:
    """X = E[tok] + P[pos] + C_true U^T + eta_perp, rounded once to the dtype.

    This synthesises activations with the structure the paper derives for a
    subspace network (Section 4.2: the residual stream minus the embedding
    terms lies in span(U)); eta_perp is Gaussian noise with its span(U)
    component removed, so it is pure off-subspace residual.  Built per row
    block in float64 for fp32 configs and float32 for bf16 configs (far below
    bf16's rounding).  Returns X (stored), C_true (float64) and the norm of the
    off-subspace noise actually added (before the final rounding of X).
    """
    cfg = cfg or CONFIGS[cfg_id]
    sigma = cfg.sigma if sigma is None else sigma
    ft = np.float64 if cfg.dtype == "f32" else np.float32
    tok, pos = ids["tok"], ids["pos"]
    n = tok.shape[0]
    U = as_float(basis["U"], cfg.dtype).astype(ft)   # the stored basis
    Eb, Pb = emb["E"], emb["P"]
    C_true = np.empty((n, cfg.k), dtype=np.float64)
    X = np.empty((n, cfg.d), dtype=np.float32 if cfg.dtype == "f32" else np.uint16)
    noise_sq = np.zeros(len(_blocks(n)))

    def one(item):
        b, r0 = item
        r1 = min(n, r0 + ROW_BLOCK)
        c = _rng(seed_of(cfg_id, ORD_C), b).standard_normal((r1 - r0, cfg.k))
        C_true[r0:r1] = c
        blk = as_float(Eb[tok[r0:r1]], cfg.dtype).astype(ft)
        blk += as_float(Pb[pos[r0:r1]], cfg.dtype)
        blk += c.astype(ft) @ U.T
        if sigma > 0:
            eta = _rng(seed_of(cfg_id, ORD_NOISE), b).standard_normal((r1 - r0, cfg.d), dtype=ft)
            eta *= ft(sigma)
            eta -= (eta @ U) @ U.T
            noise_sq[b] = float(np.sum(eta.astype(np.float64) ** 2))
            blk += eta
        X[r0:r1] = store(blk, cfg.dtype)

    _parallel(one, _blocks(n))
    return {"X": X, "C_true": C_true, "noise_norm": float(np.sum(noise_sq)) ** 0.5}


def make_gradient(cfg_id: int, n: int | None = None, cfg: Config | None = None) -> np.ndarray:
    cfg = cfg or CONFIGS[cfg_id]
    n = cfg.n_tokens if n is None else n
    return store(gaussian(seed_of(cfg_id, ORD_G), n, cfg.d, cfg.g_std), cfg.dtype)


def make_grad_iteration(cfg_id: int, t: int, n: int | None = None, cfg: Config | None = None,
                        rank: int | None = None, share: float = 0.5) -> np.ndarray:
    """Activation gradient of accumulated iteration t for the subspace update
    (Section 4.5): rows g = g_std (a z V^T + b e) with V (d x rank) a fixed
    orthonormal set of dominant directions, z ~ N(0, I_rank), e ~ N(0, I_d),
    a^2 = share d / rank and b^2 = 1 - share, so a fraction `share` of each
    row's expected energy d g_std^2 lies in span(V).  Gradients concentrated
    in a few directions give the update something to align U with."""
    cfg = cfg or CONFIGS[cfg_id]
    if not 0 <= t < 20:
        raise ValueError("t must be in [0, 20)")
    n = cfg.n_tokens if n is None else n
    rank = cfg.k if rank is None else rank
    ft = np.float64 if cfg.dtype == "f32" else np.float32
    V = orthonormal_basis(seed_of(cfg_id, ORD_GV), cfg.d, rank).astype(ft)
    a = ft((share * cfg.d / rank) ** 0.5)
    b = ft((1.0 - share) ** 0.5)
    out = np.empty((n, cfg.d), dtype=np.float32 if cfg.dtype == "f32" else np.uint16)
    seed = seed_of(cfg_id, ORD_GT + t)

    def one(item):
        blk_i, r0 = item
        r1 = min(n, r0 + ROW_BLOCK)
        rng = _rng(seed, blk_i)
        z = rng.standard_normal((r1 - r0, rank), dtype=ft)
        e = rng.standard_normal((r1 - r0, cfg.d), dtype=ft)
        g = (a * z) @ V.T
        g += b * e
        g *= ft(cfg.g_std)
        out[r0:r1] = store(g, cfg.dtype)

    _parallel(one, _blocks(n))
    return out


def make_adamw_state(cfg_id: int, rows: int, cols: int, scale: float = 1e-3) -> dict:
    """Float32 AdamW moments of a weight mid-training: M ~ N(0, scale^2) and
    V = (|N(0, 1)| scale + scale / 10)^2 (positive, varying across entries)."""
    M = gaussian(seed_of(cfg_id, ORD_AM), rows, cols, scale)
    a = gaussian(seed_of(cfg_id, ORD_AV), rows, cols, scale)
    V = (np.abs(a) + np.float32(scale / 10)) ** 2
    return {"M": M, "V": V.astype(np.float32)}


def make_weight_grad(cfg_id: int, t: int, rows: int, cols: int, cfg: Config | None = None,
                     scale: float = 1e-3, basis: np.ndarray | None = None) -> np.ndarray:
    """Weight gradient of optimizer step t, N(0, scale^2) with a per-column
    scale in [0.1, 10] (uneven second moments across columns), stored in the
    config's dtype; with `basis` (d x k, float64) the columns are projected
    onto its span first (gradients confined to S, Sec. 5 and App. A)."""
    cfg = cfg or CONFIGS[cfg_id]
    if not 0 <= t < 6:
        raise ValueError("t must be in [0, 6)")
    g = gaussian(seed_of(cfg_id, ORD_AG + t), rows, cols, scale).astype(np.float64)
    g *= _rng(seed_of(cfg_id, ORD_AG + t), 1 << 20).uniform(0.1, 10.0, size=(1, cols))
    if basis is not None:
        g = basis @ (basis.T @ g)
    return store(g, cfg.dtype)


def make_weight(cfg_id: int, index: int, rows: int, cols: int,
                cfg: Config | None = None) -> np.ndarray:
    cfg = cfg or CONFIGS[cfg_id]
    return store(gaussian(seed_of(cfg_id, ORD_W + index), rows, cols, 0.02), cfg.dtype)


def device_weight(cfg_id: int, index: int, rows: int, cols: int, std: float = 0.02,
                  device: str = "cuda"):
    """A bf16 N(0, std^2) weight matrix drawn directly on the device with torch's
    seeded generator (for sweeps too large to draw on the host)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed_of(cfg_id, ORD_W + index))
    w = torch.randn(rows, cols, generator=gen, device=device, dtype=torch.float32)
    return (w * std).to(torch.bfloat16)


def make_workload(cfg_id: int, n: int | None = None, sigma: float | None = None) -> dict:
    """Everything a config needs except weights (drawn on demand: they are big)."""
    cfg = CONFIGS[cfg_id]
    basis = make_basis(cfg_id)
    emb = make_embeddings(cfg_id)
    ids = make_ids(cfg_id, n)
    act = make_activations(cfg_id, basis, emb, ids, sigma)
    out = {"cfg": cfg, **basis, **emb, **ids, **act}
    out["G"] = make_gradient(cfg_id, ids["tok"].shape[0])
    return out

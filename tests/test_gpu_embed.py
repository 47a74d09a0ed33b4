"""GPU parity of the low-rank token table (Sec. 4.3.1) through the C ABI
against the CPU oracle.

Forward X0 = P + T_fixed[t] + C_S[t] U^T: the decompress criterion (rtol 1e-5
for float32, 2e-2 for bf16 outputs, per element against max(|ref|, row rms)).
Backward gC_S += scatter of dX0 U: float32 output, rtol 1e-5 against
max(|ref|, rms of the ref's row); rows of ids that do not occur are untouched
(bit-exact), and the result is bitwise the same on every run.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import embed as em
import synth
import paper_2506_01260_amd as sn
from gpu_helpers import assert_parity, dev, host, ids, log

pytestmark = pytest.mark.gpu


def _setup(cfg, cfg_id=0):
    b = synth.make_basis(cfg_id, cfg)
    emb = synth.make_embeddings(cfg_id, cfg)
    idx = synth.make_ids(cfg_id, None, cfg)
    dec = (lambda a: oracle.decode_bf16(a, np.float32)) if cfg.dtype == "bf16" else \
        (lambda a: np.asarray(a, np.float32))
    return b, emb, idx, dec


SHAPES = [("f32", 256, 8, 300, 4, 128), ("bf16", 512, 40, 1000, 8, 512),
          ("bf16", 320, 20, 500, 1, 777), ("bf16", 1024, 82, 2000, 2, 1000)]


@pytest.mark.parametrize("dtype,d,k,vocab,batch,seq", SHAPES)
def test_forward_matches_oracle(dtype, d, k, vocab, batch, seq):
    log(f"[embed forward] {dtype} d={d} k={k} vocab={vocab} N={batch * seq}")
    cfg = synth.Config("embed", dtype, d, k, vocab, batch, seq, True, 0.0, 1e-2)
    b, emb, idx, dec = _setup(cfg)
    U, E, P = dec(b["U"]).astype(np.float64), dec(emb["E"]), dec(emb["P"])
    CS = oracle.round_to(em.lowrank_init(E, U), dtype)   # C_S = T_fixed U, stored in the dtype
    CSs = synth.store(CS, dtype)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    tok = ids(idx["tok"])
    X0 = sn.sn_embed_lowrank_forward(basis, dev(CSs, dtype), tok, E=dev(emb["E"], dtype),
                                     P=dev(emb["P"], dtype), seq_len=seq)
    torch.cuda.synchronize()
    ref = oracle.round_to(em.lowrank_forward(dec(CSs), U, idx["tok"], E, P, seq_len=seq), dtype)
    assert_parity(host(X0), ref, dtype, "X0")
    # no fixed table: the T_S rows alone, in S
    X1 = sn.sn_embed_lowrank_forward(basis, dev(CSs, dtype), tok)
    torch.cuda.synchronize()
    ref1 = oracle.round_to(em.lowrank_forward(dec(CSs), U, idx["tok"]), dtype)
    assert_parity(host(X1), ref1, dtype, "X0 without tables")


@pytest.mark.parametrize("dtype,d,k,vocab,batch,seq", SHAPES)
def test_backward_matches_oracle(dtype, d, k, vocab, batch, seq):
    log(f"[embed backward] {dtype} d={d} k={k} vocab={vocab} N={batch * seq}")
    cfg = synth.Config("embed", dtype, d, k, vocab, batch, seq, True, 0.0, 1e-2)
    b, emb, idx, dec = _setup(cfg)
    U = dec(b["U"]).astype(np.float64)
    G = synth.make_gradient(0, batch * seq, cfg)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    init = (np.random.default_rng(1).standard_normal((vocab, k)) * 1e-3).astype(np.float32)
    gCS = torch.from_numpy(init.copy()).cuda()
    sn.sn_embed_lowrank_backward(basis, dev(G, dtype), ids(idx["tok"]), gCS)
    torch.cuda.synchronize()
    grad = em.lowrank_grad(dec(G), U, idx["tok"], vocab)
    ref = oracle.round_f32(init.astype(np.float64) + grad)
    got = host(gCS)
    present = np.zeros(vocab, bool)
    present[idx["tok"]] = True
    assert np.array_equal(got[~present], init[~present].astype(np.float64))
    # the scatter's own values, with the accumulated start removed exactly in float64
    assert_parity(got[present] - init[present], grad[present], "f32", "scatter of dX0 U")
    assert_parity(got, ref, "f32", "gC_S accumulated")


@pytest.mark.parametrize("pattern", ["one_id", "long_runs"])
def test_backward_long_runs(pattern):
    """Rows of one id that fill whole token blocks (runs crossing every wave
    of a block, and every block), and an id that returns after a long run of
    another: the per-id sums must still take every row exactly once."""
    dtype, d, k, vocab, N = "bf16", 512, 40, 64, 3000  # last block partial
    log(f"[embed backward] {pattern} N={N}")
    cfg = synth.Config("embed", dtype, d, k, vocab, 1, N, True, 0.0, 1e-2)
    b, _, _, dec = _setup(cfg)
    U = dec(b["U"]).astype(np.float64)
    if pattern == "one_id":
        tok = np.full(N, 7, np.int32)
    else:
        tok = np.concatenate([np.full(1100, 3), np.full(900, 40), (np.arange(300) % 5) + 58,
                              np.full(700, 3)]).astype(np.int32)
    G = synth.make_gradient(0, N, cfg)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    outs = []
    for _ in range(2):
        gCS = torch.zeros(vocab, k, device="cuda")
        sn.sn_embed_lowrank_backward(basis, dev(G, dtype), ids(tok), gCS)
        torch.cuda.synchronize()
        outs.append(host(gCS))
    assert np.array_equal(outs[0], outs[1]), "bitwise the same on every run"
    grad = em.lowrank_grad(dec(G), U, tok, vocab)
    present = np.zeros(vocab, bool)
    present[tok] = True
    assert np.all(outs[0][~present] == 0.0)
    assert_parity(outs[0][present], grad[present], "f32", f"scatter of dX0 U, {pattern}")


def test_backward_large_vocab():
    """A Llama-3-sized vocabulary (128256 ids: 2004 id ranges in each block's
    range index) with Zipf ids over 5 blocks and a partial sixth."""
    dtype, d, k, vocab, N = "bf16", 256, 82, 128256, 2900
    log(f"[embed backward] large vocab {vocab} k={k} N={N}")
    cfg = synth.Config("embed", dtype, d, k, vocab, 1, N, True, 0.0, 1e-2)
    b = synth.make_basis(0, cfg)
    dec = lambda a: oracle.decode_bf16(a, np.float32)  # noqa: E731
    U = dec(b["U"]).astype(np.float64)
    tok = synth.make_ids(0, None, cfg)["tok"]
    G = synth.make_gradient(0, N, cfg)
    basis = sn.sn_basis_pack(dev(b["U"], dtype))
    gCS = torch.zeros(vocab, k, device="cuda")
    sn.sn_embed_lowrank_backward(basis, dev(G, dtype), ids(tok), gCS)
    torch.cuda.synchronize()
    got = host(gCS)
    grad = em.lowrank_grad(dec(G), U, tok, vocab)
    present = np.zeros(vocab, bool)
    present[tok] = True
    assert np.all(got[~present] == 0.0)
    assert_parity(got[present], grad[present], "f32", "scatter of dX0 U, large vocabulary")


def test_backward_config2_zipf_deterministic():
    """Config 2's token stream (N = 32768, vocab 32000, Zipf(1.1)): one id
    holds ~14 % of the tokens; every row of the gradient, and two runs
    bitwise equal."""
    cfg = synth.CONFIGS[2]
    log("[embed backward] config 2")
    b = synth.make_basis(2)
    U = oracle.decode_bf16(b["U"], np.float32).astype(np.float64)
    idx = synth.make_ids(2)
    G = synth.make_gradient(2)
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    Gd, tok = dev(G, "bf16"), ids(idx["tok"])
    outs = []
    for _ in range(2):
        gCS = torch.zeros(cfg.vocab, cfg.k, device="cuda")
        sn.sn_embed_lowrank_backward(basis, Gd, tok, gCS)
        torch.cuda.synchronize()
        outs.append(gCS.cpu())
    assert torch.equal(outs[0], outs[1])
    Gf = oracle.decode_bf16(G, np.float32)
    ref = oracle.embed.lowrank_grad(Gf, U, idx["tok"], cfg.vocab)
    got = outs[0].numpy().astype(np.float64)
    present = np.bincount(idx["tok"], minlength=cfg.vocab) > 0
    assert np.all(got[~present] == 0.0), "rows of absent ids stay zero"
    assert_parity(got[present], ref[present], "f32", "gC_S, every row of a present id")


def test_out_of_range_ids_are_clamped_and_flagged():
    log("[embed] out-of-range ids")
    cfg = synth.Config("embed", "bf16", 256, 8, 50, 1, 64, False, 0.0, 1e-2)
    b, emb, idx, dec = _setup(cfg)
    t = idx["tok"].copy()
    t[3], t[10] = -2, 50
    basis = sn.sn_basis_pack(dev(b["U"], "bf16"))
    CS = dev(synth.store(np.ones((50, 8), np.float32), "bf16"), "bf16")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    sn.sn_embed_lowrank_forward(basis, CS, ids(t), err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) & 1
    flag.zero_()
    gCS = torch.zeros(50, 8, device="cuda")
    sn.sn_embed_lowrank_backward(basis, dev(synth.make_gradient(0, 64, cfg), "bf16"), ids(t), gCS,
                                 err_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) & 1

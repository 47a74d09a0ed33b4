"""The seeded input generator (no GPU): reproducibility, shapes, and the
distributions the workloads are meant to have.

* the same configuration and seed give bit-identical arrays; different
  tensor ordinals give different streams;
* token ids follow the truncated Zipf(1.1) law: the share of the most
  frequent ranks is the law's probability within sampling error, and the
  number of distinct ids matches its expectation sum_r 1 - (1 - p_r)^N;
* uniform ids (config 0) cover the vocabulary evenly (chi-square);
* default positions are those of a row-major [batch, seq] layout;
* every configuration's arrays have the stated shapes and storage types.
"""
import numpy as np
import pytest

import synth


def _zipf_p(vocab, a=1.1):
    p = np.arange(1, vocab + 1, dtype=np.float64) ** (-a)
    return p / p.sum()


def test_same_seed_same_bits():
    a = synth.make_workload(0)
    b = synth.make_workload(0)
    for name in ("U", "E", "P", "X", "G", "tok"):
        assert np.array_equal(a[name], b[name]), name
    x1 = synth.make_ids(2, 5000)["tok"]
    x2 = synth.make_ids(2, 5000)["tok"]
    assert np.array_equal(x1, x2)


def test_ordinals_and_configs_give_distinct_streams():
    s = {synth.seed_of(c, o) for c in range(5) for o in range(8)}
    assert len(s) == 40
    g1 = synth.gaussian(synth.seed_of(1, synth.ORD_E), 64, 64, 1.0)
    g2 = synth.gaussian(synth.seed_of(1, synth.ORD_P), 64, 64, 1.0)
    assert not np.array_equal(g1, g2)


@pytest.mark.parametrize("cid", [1, 2, 4])
def test_zipf_head_and_distinct_count(cid):
    cfg = synth.CONFIGS[cid]
    tok = synth.make_ids(cid)["tok"]
    n = tok.shape[0]
    assert n == cfg.n_tokens and tok.dtype == np.int32
    assert tok.min() >= 0 and tok.max() < cfg.vocab
    p = _zipf_p(cfg.vocab)
    counts = np.bincount(tok, minlength=cfg.vocab)
    for r in range(5):  # the head of the law, within 5 binomial standard deviations
        sd = np.sqrt(n * p[r] * (1 - p[r]))
        assert abs(counts[r] - n * p[r]) <= 5 * sd, (r, counts[r], n * p[r])
    expected_distinct = np.sum(1.0 - (1.0 - p) ** n)
    distinct = np.count_nonzero(counts)
    assert abs(distinct - expected_distinct) <= 0.03 * expected_distinct, (
        distinct, expected_distinct)


def test_uniform_ids_cover_vocabulary():
    cfg = synth.CONFIGS[0]
    tok = synth.make_ids(0, 200_000)["tok"]
    counts = np.bincount(tok, minlength=cfg.vocab)
    e = tok.shape[0] / cfg.vocab
    chi2 = np.sum((counts - e) ** 2 / e)
    dof = cfg.vocab - 1
    assert abs(chi2 - dof) <= 6 * np.sqrt(2 * dof)


def test_default_positions_row_major():
    pos = synth.default_positions(10, 4)
    assert pos.tolist() == [0, 1, 2, 3, 0, 1, 2, 3, 0, 1]
    ids = synth.make_ids(2, 3 * 4096 + 5)
    assert ids["pos"][4096] == 0 and ids["pos"][4095] == 4095 and ids["pos"][-1] == 4


@pytest.mark.parametrize("cid", [0, 1, 2, 4])
def test_shapes_and_storage(cid):
    cfg = synth.CONFIGS[cid]
    n = 48
    w = synth.make_workload(cid, n)
    st = np.float32 if cfg.dtype == "f32" else np.uint16
    assert w["U"].shape == (cfg.d, cfg.k) and w["U"].dtype == st
    assert w["E"].shape == (cfg.vocab, cfg.d) and w["E"].dtype == st
    assert w["P"].shape == (cfg.seq, cfg.d) and w["P"].dtype == st
    assert w["X"].shape == (n, cfg.d) and w["X"].dtype == st
    assert w["G"].shape == (n, cfg.d) and w["G"].dtype == st
    assert w["tok"].shape == (n,)
    # the stored basis is orthonormal to its storage precision
    U = synth.as_float(w["U"], cfg.dtype).astype(np.float64)
    tol = 1e-5 if cfg.dtype == "f32" else 2e-2
    assert np.abs(U.T @ U - np.eye(cfg.k)).max() < tol


def test_gaussian_scale():
    g = synth.gaussian(12345, 512, 512, 0.02)
    assert abs(g.std() - 0.02) < 0.02 * 0.01
    assert abs(g.mean()) < 0.02 * 0.01

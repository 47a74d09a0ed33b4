"""Benchmark of the stage-boundary subspace codec on one MI355X.

One step = the whole hot path for one batch at d=4096, k=40, N=32768 tokens
(8 x 4096), bf16, vocab 32000 with Zipf(1.1) ids:

  compress      C  = (X - P[pos] - E[tok]) U
  decompress    X' = C U^T + P[pos] + E[tok]
  grad compress Cg = G U
  grad decomp.  G' = Cg U^T
  projection    Wo (4096 x 4096) and W2 (4096 x 14336) <- U (U^T W), in place

Inputs are resident in HBM before timing; X, G, the outputs and the weights
rotate over several buffer sets so no step finds its data in the 256 MB
Infinity Cache.  Prints one JSON line.  ``value`` is the step's algorithmic
bytes (each op's inputs and outputs, each unique gathered embedding row once,
U once per op) over the step time.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--rotate", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=32768,
                    help="tokens in the oracle's timed sample")
    return ap.parse_args()


def to_dev(a, bf16=True):
    import torch
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def cpu_baseline(w, weights, rows: int):
    """The oracle, as it stands, on a bounded sample of the same step: the
    first `rows` tokens through compress, decompress, grad compress and grad
    decompress, plus the projection of every weight matrix of the step."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    cfg = w["cfg"]
    dec = lambda a: oracle.decode_bf16(a, np.float32)  # noqa: E731
    U = dec(w["U"]).astype(np.float64)
    E, P = dec(w["E"]), dec(w["P"])
    X, G = dec(w["X"][:rows]), dec(w["G"][:rows])
    tok = w["tok"][:rows]
    Ws = [dec(Wb) for Wb in weights]
    t0 = time.perf_counter()
    C = oracle.round_bf16(oracle.compress(X, U, tok, E, P, seq_len=cfg.seq))
    oracle.round_bf16(oracle.decompress(C, U, tok, E, P, seq_len=cfg.seq))
    Cg = oracle.round_bf16(oracle.grad_compress(G, U))
    oracle.round_bf16(oracle.grad_decompress(Cg, U))
    for Wf in Ws:
        oracle.round_bf16(oracle.project_weights(Wf, U))
    dt = time.perf_counter() - t0
    frac = rows / cfg.n_tokens
    return {"value": rows / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{rows} of {cfg.n_tokens} tokens through compress, decompress, grad "
                      f"compress and grad decompress, plus the projection of Wo and W2 "
                      f"({dt:.2f} s of CPU time; the sample is {frac:.0%} of the step's tokens "
                      f"and all of its weights)",
            "seconds": dt}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2506_01260_amd as sn

    cfg_id = 2
    w = synth.make_workload(cfg_id)
    cfg = w["cfg"]
    N, d, k = cfg.n_tokens, cfg.d, cfg.k
    print(f"[bench] inputs generated: N={N} d={d} k={k}", file=sys.stderr, flush=True)

    U = to_dev(w["U"])
    basis = sn.sn_basis_pack(U)
    E, P = to_dev(w["E"]), to_dev(w["P"])
    tok = torch.from_numpy(w["tok"]).cuda()
    R = max(1, args.rotate)
    Xs = [to_dev(w["X"]) for _ in range(R)]
    Gs = [to_dev(w["G"]) for _ in range(R)]
    Cs = [torch.empty(N, k, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Cgs = [torch.empty(N, k, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Xrs = [torch.empty(N, d, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Grs = [torch.empty(N, d, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    weights, host_weights = [], []
    for i, (rows, cols) in enumerate(cfg.weights):
        wb = synth.make_weight(cfg_id, i, rows, cols)
        host_weights.append(wb)
        base = to_dev(wb)
        weights.append([base.clone() for _ in range(R)])
        del base
    ws_bytes = max(sn.sn_project_weights_workspace_bytes(d, k, sn.SN_BF16, c)
                   for _, c in cfg.weights)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

    # algorithmic bytes per op
    es = 2
    uniq_e = len(np.unique(w["tok"])) * d * es
    uniq_p = min(cfg.seq, N) * d * es
    xb, cb, ub = N * d * es, N * k * es, d * k * es
    op_bytes = {
        "compress": xb + cb + uniq_e + uniq_p + ub,
        "decompress": cb + xb + uniq_e + uniq_p + ub,
        "grad_compress": xb + cb + ub,
        "grad_decompress": cb + xb + ub,
    }
    for i, (rows, cols) in enumerate(cfg.weights):
        op_bytes[f"project_W{i}"] = 2 * rows * cols * es

    def op(name, i):
        j = i % R
        if name == "compress":
            sn.sn_compress(basis, Xs[j], tok=tok, E=E, P=P, seq_len=cfg.seq, out=Cs[j])
        elif name == "decompress":
            sn.sn_decompress(basis, Cs[j], tok=tok, E=E, P=P, seq_len=cfg.seq, out=Xrs[j])
        elif name == "grad_compress":
            sn.sn_grad_compress(basis, Gs[j], out=Cgs[j])
        elif name == "grad_decompress":
            sn.sn_decompress(basis, Cgs[j], out=Grs[j])
        else:
            wi = int(name[len("project_W"):])
            sn.sn_project_weights(basis, weights[wi][j], workspace=ws)

    names = list(op_bytes)
    stream = torch.cuda.current_stream()

    def step(i, evs=None):
        for nm in names:
            if evs is not None:
                evs[nm][0].record(stream)
            op(nm, i)
            if evs is not None:
                evs[nm][1].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    K = args.steps
    evs = [{nm: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for nm in names} for _ in range(K)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(K):
        step(args.warmup + i, evs[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / K
    op_ms = {nm: float(np.mean([e[nm][0].elapsed_time(e[nm][1]) for e in evs])) for nm in names}
    print(f"[bench] timed {K} steps: {ms_step:.4f} ms/step", file=sys.stderr, flush=True)

    step_bytes = sum(op_bytes.values())
    value = step_bytes / (ms_step * 1e-3) / 1e9
    ops = {nm: {"ms": round(op_ms[nm], 5), "bytes": op_bytes[nm],
                "GBps": round(op_bytes[nm] / (op_ms[nm] * 1e-3) / 1e9, 1),
                "frac_hbm": round(op_bytes[nm] / (op_ms[nm] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
           for nm in names}
    pair_ms = op_ms["compress"] + op_ms["decompress"]
    pair_bytes = op_bytes["compress"] + op_bytes["decompress"]
    pair_gbs = pair_bytes / (pair_ms * 1e-3) / 1e9
    dom = max(names, key=lambda nm: op_ms[nm])
    dom_gbs = op_bytes[dom] / (op_ms[dom] * 1e-3) / 1e9

    out = {
        "metric": "codec GB/s & % HBM peak (compress+decompress) at d=4096,k=40; tokens/s",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "stage-boundary codec step: compress, decompress, grad compress, "
                               "grad decompress at d=4096 k=40 N=32768 (8x4096) vocab=32000 "
                               "Zipf(1.1) + in-place projection of Wo 4096x4096 and "
                               "W2 4096x14336, bf16",
                   "d": d, "k": k, "tokens": N, "seq_len": cfg.seq, "vocab": cfg.vocab,
                   "rotate_buffers": R},
        "tokens_per_s": round(N / (ms_step * 1e-3), 1),
        "codec_pair": {"ops": "compress+decompress", "ms": round(pair_ms, 5),
                       "GBps": round(pair_gbs, 1), "frac_hbm": round(pair_gbs / HBM_PEAK_GBS, 4),
                       "tokens_per_s": round(N / (pair_ms * 1e-3), 1),
                       "x_c_only_GBps": round(2 * (xb + cb) / (pair_ms * 1e-3) / 1e9, 1)},
        "ops": ops,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(dom_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dom_gbs / HBM_PEAK_GBS, 4), "traffic": None},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        cb_ = cpu_baseline(w, host_weights, min(args.cpu_rows, N))
        out["cpu_baseline"] = {kk: (round(v, 3) if isinstance(v, float) else v)
                               for kk, v in cb_.items()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

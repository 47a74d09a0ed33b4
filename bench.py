"""Benchmark of the stage-boundary subspace codec on one MI355X.

One step = the whole hot path for one batch at d=4096, k=40, N=32768 tokens
(8 x 4096), bf16, vocab 32000 with Zipf(1.1) ids:

  compress      C  = (X - P[pos] - E[tok]) U      gather + subtract + projection, one kernel
  decompress    X' = C U^T + P[pos] + E[tok]
  grad compress Cg = G U
  grad decomp.  G' = Cg U^T
  projection    Wo (4096 x 4096) and W2 (4096 x 14336) <- U (U^T W), in place, one call

Inputs are resident in HBM before timing; X, G, the outputs and the weights
rotate over several buffer sets so no step finds its data in the 256 MB
Infinity Cache.  Prints one JSON line.  ``value`` is the headline metric:
compress + decompress back to back, the pair's algorithmic bytes (X and C of
both ops, each unique gathered embedding row once per op, U once per op) over
the pair time; ``step`` is the whole step (ms_per_step is its time).
``cold_GBps`` is the same pair after a 512 MB fill that evicts every cache.

Also reported, outside the step: the same compress computed against
projected tables (sn_embed_project once per basis, then
sn_compress_projected), the path to use while U is fixed between subspace
updates.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
    python bench.py --profile-pass                    # short run for rocprofv3 counters
    python bench.py --traffic-summary FETCH_DIR WRITE_DIR   # writes profiles/traffic_*.json/.md
    python bench.py --counter-summary BUSY_DIR        # writes profiles/busy_*.md
    python bench.py --trace-summary TRACE_DIR BENCH_LOG     # writes profiles/*_kernel_stats.md
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
CFG_ID = 2
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_codec_step_d4096_k40.json")
CALIB_BYTES = 256 * 1024 * 1024   # plain copy used to scale the HBM counters

# rocprofv3 kernel names of each op (substring match on the demangled name)
OP_KERNELS = {
    "compress": ["compress_kernel<3, true, true, 8, 8, 0>"],
    "decompress": ["decompress_cb_kernel<2, true, true, 0, false>"],
    "grad_compress": ["compress_kernel<3, false, false, 1, 8, 0>"],
    "grad_decompress": ["decompress_cb_kernel<2, false, false, 0, false>"],
    "compress_projected": ["compress_kernel<3, false, false, 1, 8, 1>"],
    # subspace update: its compress pass and its contraction over tokens
    "grassmann_compress": ["compress_kernel<3, false, false, 1, 8, 3>"],
    "grassmann_tokens": ["project_pass1_kernel<5, true, 8>"],
    # the weight projection of Wo and W2 (one call, three launches)
    "project_pass1": ["project_pass1_kernel<3, false, 8>"],
    "project_pass2": ["project_pass2_rfrag_kernel"],
    "project_pass3": ["decompress_cb_kernel<3, false, false, 0, false>"],
}
PROJ_PASSES = ("project_pass1", "project_pass2", "project_pass3")


# kernels that only the subspace update launches
GRASS_KERNELS = ["loss_kernel", "finish_kernel", "gram_partial_kernel", "gram_reduce_kernel",
                 "moments_kernel", "alpha_kernel", "apply_kernel", "gather_rows_kernel",
                 "hist_kernel", "block_prefix_kernel", "tile_scan_kernel",
                 "tiles_scan_kernel", "tile_write_kernel", "place_kernel",
                 "chunk_sum_kernel", "seg_sum_kernel",
                 "update_kernel", "chol_kernel", "tri_apply_kernel", "reset_kernel",
                 "compress_kernel<3, false, false, 1, 8, 3>"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--rotate", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured in a HIP graph and replayed (the "
                         "replays measured no faster than eager launches here)")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the configs 1, 3 and 4 timings and the copy reference")
    ap.add_argument("--profile-pass", action="store_true",
                    help="run a few steps and a plain copy of known size, print nothing")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE)")
    ap.add_argument("--counter-summary", metavar="BUSY_DIR",
                    help="summarise a rocprofv3 --pmc MfmaUtil VALUBusy run of --profile-pass")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "BENCH_LOG"),
                    help="summarise a rocprofv3 --kernel-trace run of this script, split by "
                         "phase, beside the JSON line that run printed")
    return ap.parse_args()


def source_hash() -> str:
    """Hash of the HIP / C++ sources: a traffic figure is valid for one build only."""
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2506_01260_amd", "csrc", "*"))):
        h.update(os.path.basename(p).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def to_dev(a, bf16=True):
    import torch
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _cpu_info() -> dict:
    """Host facts for the CPU baseline: model, core counts, BLAS library."""
    info = {"cpu_model": None, "os_cpu_count": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)), "blas": None, "blas_threads": 1}
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                info["cpu_model"] = line.split(":", 1)[1].strip()
                break
    except OSError:  # pragma: no cover
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if blas:
            info["blas"] = f"{blas[0].get('internal_api')} {blas[0].get('version')}"
            info["blas_threads"] = max(p.get("num_threads", 1) for p in blas)
    except Exception:  # pragma: no cover
        pass
    return info


def cpu_baseline(w, weights) -> dict:
    """The oracle, as it stands (numpy, float64 sums, BLAS on every visible
    core), timed on the host per op and per config on bounded samples:

    * config 2 (the headline workload, this process's own inputs): compress,
      decompress, grad compress and grad decompress on all 32768 tokens,
      median of 3, and the projection of Wo and W2 (4096 of their 18432
      columns, once, scaled: each column is projected on its own);
    * config 1 (d = 2048, k = 20): the four codec ops on all 16384 tokens,
      median of 3; config 0 (tiny fp32): all ops, median of 3;
    * config 4 (d = 8192, k = 82): the four ops on 4096 of the 32768 tokens
      and 4096 of Wo's 8192 columns, once;
    * config 3 (32-layer sweep): 4096 of one layer's 18432 columns, once,
      scaled to the 32 layers.

    Inputs other than config 2's are random arrays of each config's shapes
    (the oracle's time depends on the shapes only).  Rates use the GPU's
    byte accounting for the same sample; ``value`` is the config-2
    compress + decompress rate, the headline metric's CPU counterpart."""
    import oracle
    import synth
    info = _cpu_info()
    rng = np.random.default_rng(7)

    def med(fn, reps):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts))

    def codec_case(n, d, k, vocab, seq, X, G, U, E, P, tok, reps, uniq_rows):
        es = 2
        C = oracle.round_bf16(oracle.compress(X, U, tok, E, P, seq_len=seq))
        Cg = oracle.round_bf16(oracle.grad_compress(G, U))
        t = {"compress": med(lambda: oracle.round_bf16(
                 oracle.compress(X, U, tok, E, P, seq_len=seq)), reps),
             "decompress": med(lambda: oracle.round_bf16(
                 oracle.decompress(C, U, tok, E, P, seq_len=seq)), reps),
             "grad_compress": med(lambda: oracle.round_bf16(oracle.grad_compress(G, U)), reps),
             "grad_decompress": med(lambda: oracle.round_bf16(oracle.grad_decompress(Cg, U)),
                                    reps)}
        xb, cb, ub = n * d * es, n * k * es, d * k * es
        tab = uniq_rows * d * es
        nbytes = {"compress": xb + cb + tab + ub, "decompress": cb + xb + tab + ub,
                  "grad_compress": xb + cb + ub, "grad_decompress": cb + xb + ub}
        out = {op: {"s": round(v, 4), "tokens_per_s": round(n / v, 1),
                    "GBps": round(nbytes[op] / v / 1e9, 4)} for op, v in t.items()}
        pair_s = t["compress"] + t["decompress"]
        out["pair"] = {"s": round(pair_s, 4), "tokens_per_s": round(n / pair_s, 1),
                       "GBps": round((nbytes["compress"] + nbytes["decompress"]) / pair_s / 1e9, 4)}
        return out

    def rand_case(cfg, n, reps):
        d, k = cfg.d, cfg.k
        U = synth.orthonormal_basis(1, d, k)
        X = rng.standard_normal((n, d), dtype=np.float32)
        G = rng.standard_normal((n, d), dtype=np.float32)
        tok = synth.zipf_ids(5, n, cfg.vocab) if cfg.zipf else \
            rng.integers(0, cfg.vocab, n).astype(np.int32)
        # only the rows the sample uses: ids remapped onto a table of its unique ids
        uniq, inv = np.unique(tok, return_inverse=True)
        E = rng.standard_normal((uniq.size, d), dtype=np.float32)
        P = rng.standard_normal((min(cfg.seq, n), d), dtype=np.float32)
        return codec_case(n, d, k, cfg.vocab, min(cfg.seq, n), X, G, U, E, P,
                          inv.astype(np.int32), reps, uniq.size + min(cfg.seq, n))

    def proj_time(d, k, cols, reps, of_cols):
        """seconds for of_cols columns, from a sample of cols columns"""
        U = synth.orthonormal_basis(2, d, k)
        W = rng.standard_normal((d, cols), dtype=np.float32)
        return med(lambda: oracle.round_bf16(oracle.project_weights(W, U)), reps) * of_cols / cols

    per = {}
    t_all = time.perf_counter()
    # config 2: the bench's own inputs, every token
    cfg = w["cfg"]
    n2 = cfg.n_tokens
    dec = lambda a: oracle.decode_bf16(a, np.float32)  # noqa: E731
    U2 = dec(w["U"]).astype(np.float64)
    tok2 = w["tok"][:n2]
    uniq2 = len(np.unique(tok2)) + min(cfg.seq, n2)
    per["cfg2"] = {"tokens": n2, "of_tokens": cfg.n_tokens, "repetitions": 3,
                   **codec_case(n2, cfg.d, cfg.k, cfg.vocab, cfg.seq, dec(w["X"][:n2]),
                                dec(w["G"][:n2]), U2, dec(w["E"]), dec(w["P"]), tok2, 3, uniq2)}
    wcols = sum(Wb.shape[1] for Wb in weights)
    Ws = dec(weights[-1][:, :4096])
    tp = med(lambda: oracle.round_bf16(oracle.project_weights(Ws, U2)), 1) * wcols / 4096
    wbytes = sum(2 * Wb.size * 2 for Wb in weights)
    per["cfg2"]["project_weights_wo_w2"] = {"s": round(tp, 4), "GBps": round(wbytes / tp / 1e9, 4),
                                            "columns_timed": 4096, "of_columns": wcols}
    del Ws
    # configs 1 and 0: every token, median of 3
    per["cfg1"] = {"tokens": synth.CONFIGS[1].n_tokens, "repetitions": 3,
                   **rand_case(synth.CONFIGS[1], synth.CONFIGS[1].n_tokens, 3)}
    c0 = synth.CONFIGS[0]
    per["cfg0"] = {"tokens": c0.n_tokens, "repetitions": 3, **rand_case(c0, c0.n_tokens, 3)}
    # config 4: 4096 of 32768 tokens and 4096 of Wo's columns, once
    c4 = synth.CONFIGS[4]
    per["cfg4"] = {"tokens": 4096, "of_tokens": c4.n_tokens, "repetitions": 1,
                   **rand_case(c4, 4096, 1)}
    t4 = proj_time(8192, 82, 4096, 1, 8192)
    per["cfg4"]["project_wo"] = {"s": round(t4, 4), "GBps": round(2 * 8192 * 8192 * 2 / t4 / 1e9, 4),
                                 "columns_timed": 4096, "of_columns": 8192}
    # config 3: 4096 columns of one layer, scaled to the 32 layers' 32 x 18432
    sweep_cols = 32 * (4096 + 14336)
    tl = proj_time(4096, 40, 4096, 1, sweep_cols)
    sweep_bytes = 2 * 4096 * sweep_cols * 2
    per["cfg3"] = {"columns_timed": 4096, "of_columns": sweep_cols,
                   "sweep_s_estimate": round(tl, 3), "GBps": round(sweep_bytes / tl / 1e9, 4)}
    total = time.perf_counter() - t_all
    head = per["cfg2"]["pair"]
    frac = n2 / cfg.n_tokens
    return {"value": head["GBps"], "unit": "GB/s", "tokens_per_s": head["tokens_per_s"],
            "cores": int(info["blas_threads"]), "kind": "oracle",
            "sample": f"config 2 compress + decompress on {n2} of {cfg.n_tokens} tokens "
                      f"({frac:.0%}), median of 3; per-op and per-config figures in "
                      f"per_config ({total:.1f} s of CPU time in all)",
            "seconds": round(total, 2), **{kk: v for kk, v in info.items() if kk != "blas_threads"},
            "per_config": per}


# --------------------------------------------------------------------------- counters

def _counter_rows(d: str):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    for f in files:
        yield from csv.DictReader(open(f))


def _per_kernel(d: str, counter: str):
    """Mean counter value (KiB per dispatch) per kernel name."""
    acc: dict = {}
    for r in _counter_rows(d):
        if r["Counter_Name"] != counter:
            continue
        acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: float(np.mean(v)) for k, v in acc.items()}


def _short(name: str) -> str:
    """Kernel name without its argument list and namespaces."""
    name = name.replace("void ", "").replace("sn::", "").replace("(anonymous namespace)::", "")
    return name.split(">(")[0] + ">" if ">(" in name else name.split("(")[0]


def traffic_summary(fetch_dir: str, write_dir: str):
    fetch = _per_kernel(fetch_dir, "FETCH_SIZE")
    write = _per_kernel(write_dir, "WRITE_SIZE")

    def find(table, subs, also=None):
        for name, v in table.items():
            if any(s in name for s in subs) and (also is None or also in name):
                return name, v
        return None, None

    # the calibration kernel is the only multiply of the pass
    cname, cf = find(fetch, ["MulFunctor"])
    _, cw = find(write, ["MulFunctor"])
    if cf is None or cw is None:
        raise SystemExit("calibration copy kernel not found in the counter files")
    f_scale = CALIB_BYTES / (cf * 1024.0)
    w_scale = CALIB_BYTES / (cw * 1024.0)
    out = {"source_hash": source_hash(),
           "calibration": {"kernel": cname, "bytes_read": CALIB_BYTES, "bytes_written": CALIB_BYTES,
                           "fetch_kib": cf, "write_kib": cw,
                           "fetch_scale": f_scale, "write_scale": w_scale},
           "ops": {}}
    for op, subs in OP_KERNELS.items():
        name, fv = find(fetch, subs)
        _, wv = find(write, subs)
        if fv is None or wv is None:
            continue
        fb, wb = fv * 1024.0 * f_scale, wv * 1024.0 * w_scale
        out["ops"][op] = {"kernel": _short(name), "fetch_kib": fv, "write_kib": wv,
                          "fetch_bytes": fb, "write_bytes": wb, "traffic_bytes": fb + wb}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    md = TRAFFIC_FILE[:-5] + ".md"
    with open(md, "w") as f:
        f.write("# HBM traffic per launch: codec step at d=4096, k=40, N=32768 (bf16)\n\n")
        f.write("Commands (repository root `$R`, output directory `$OUT`; `cd /tmp && export "
                "TMPDIR=/tmp` first), one counter per run:\n\n```\n"
                "rocprofv3 --pmc FETCH_SIZE -d $OUT/pmc_fetch -o f --output-format csv "
                "-- python3 $R/bench.py --profile-pass\n"
                "rocprofv3 --pmc WRITE_SIZE -d $OUT/pmc_write -o w --output-format csv "
                "-- python3 $R/bench.py --profile-pass\n"
                "python3 $R/bench.py --traffic-summary $OUT/pmc_fetch $OUT/pmc_write\n```\n\n")
        f.write(f"Scale: a streaming kernel (`y = 1.0 * x`, fp32) that reads and writes "
                f"{CALIB_BYTES} bytes (torch `mul` fp32 elementwise kernel) "
                f"reads {cf:.0f} KiB and writes {cw:.0f} KiB per dispatch; counters are "
                f"multiplied by {f_scale:.4f} (fetch) and {w_scale:.4f} (write).\n\n")
        f.write(f"Source hash `{out['source_hash']}`.\n\n")
        f.write("| op | kernel | fetch MB | write MB | traffic MB |\n|---|---|---|---|---|\n")
        for op, v in out["ops"].items():
            f.write(f"| {op} | `{v['kernel']}` | "
                    f"{v['fetch_bytes'] / 1e6:.1f} | {v['write_bytes'] / 1e6:.1f} | "
                    f"{v['traffic_bytes'] / 1e6:.1f} |\n")
    print(json.dumps(out, indent=1))


def counter_summary(busy_dir: str):
    """Summarise one rocprofv3 --pmc run of the profile pass with the derived
    counters MfmaUtil (matrix-core busy cycles / (GPU cycles x SIMDs)) and
    VALUBusy (vector-ALU active cycles / (GPU cycles x CUs)): per kernel of the
    step, the mean over its dispatches, in percent."""
    acc: dict = {}
    for r in _counter_rows(busy_dir):
        acc.setdefault((r["Kernel_Name"], r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    names = sorted({k for k, _ in acc})
    out_md = os.path.join(ROOT, "profiles", "busy_codec_step_d4096_k40.md")
    with open(out_md, "w") as f:
        f.write("# Matrix-core and vector-ALU busy: codec step at d=4096, k=40, N=32768 (bf16)\n\n")
        f.write("Commands (repository root `$R`, output directory `$OUT`; `cd /tmp && export "
                "TMPDIR=/tmp` first):\n\n```\n"
                "rocprofv3 --pmc MfmaUtil VALUBusy -d $OUT/pmc_busy -o b --output-format csv "
                "-- python3 $R/bench.py --profile-pass\n"
                "python3 $R/bench.py --counter-summary $OUT/pmc_busy\n```\n\n")
        f.write(f"Source hash `{source_hash()}`. MfmaUtil = SQ_VALU_MFMA_BUSY_CYCLES / "
                "(GRBM_GUI_ACTIVE x SIMDs); VALUBusy = SQ_ACTIVE_INST_VALU / (GRBM_GUI_ACTIVE x "
                "CUs); both in percent of the kernel's duration, mean over its dispatches in the "
                "profile pass (3 steps).\n\n")
        f.write("| op | kernel | dispatches | MfmaUtil % | VALUBusy % |\n|---|---|---|---|---|\n")
        for op, subs in OP_KERNELS.items():
            name = next((n for n in names if any(sub in n for sub in subs)), None)
            if name is None:
                continue
            mf = acc.get((name, "MfmaUtil"), [])
            va = acc.get((name, "VALUBusy"), [])
            f.write(f"| {op} | `{_short(name)}` | {len(mf)} | "
                    f"{np.mean(mf) if mf else float('nan'):.2f} | "
                    f"{np.mean(va) if va else float('nan'):.2f} |\n")
    print(open(out_md).read())


def trace_summary(trace_dir: str, bench_log: str):
    """Per-kernel durations of a ``rocprofv3 --kernel-trace`` run of this
    script, split into the phases main() runs in order: set-up, the warm-up
    and timed steps, the two back-to-back pair loops, the cold pairs, the
    projected compress alone and the table build.  Only this library's kernels are counted; the
    phases are found from the dispatch order (a step starts at each compress
    launch and has a fixed number of launches)."""
    files = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {trace_dir}")
    rows = [r for f in files for r in csv.DictReader(open(f)) if "sn::" in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    line = next((ln for ln in open(bench_log) if ln.startswith("{\"metric\"")), None)
    if line is None:
        raise SystemExit(f"no JSON line in {bench_log}")
    b = json.loads(line)
    W, K = b["warmup"], b["steps"]
    names = [_short(r["Kernel_Name"]) for r in rows]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    comp = _short(next(r["Kernel_Name"] for r in rows if OP_KERNELS["compress"][0] in r["Kernel_Name"]))
    starts = [i for i, n in enumerate(names) if n == comp]
    s0, per_step = starts[0], starts[1] - starts[0]
    pair = 2 * (3 + 3 * K)  # 3 warm-up pairs, then three timed runs of K pairs
    R = b["config"].get("rotate_buffers", 3)
    cuts = [("set-up", 0, s0),
            ("warm-up steps", s0, s0 + W * per_step),
            ("timed steps", s0 + W * per_step, s0 + (W + K) * per_step)]
    at = s0 + (W + K) * per_step
    if b.get("graph_replay_ms_per_step") is not None:
        cuts += [("graph replays, warm-up", at, at + 2 * R * per_step),
                 ("timed graph replays", at + 2 * R * per_step, at + (2 * R + K) * per_step)]
        at += (2 * R + K) * per_step
    cuts.append(("timed steps, event per op", at, at + K * per_step))
    e = cuts[-1][2]
    e2 = e + 2 * pair
    e3 = e2 + 2 * max(5, K // 2)  # the cold pairs

    def is_build(i):  # the table build: the compress kernel with the fp32-row epilogue
        return names[i].startswith("compress_kernel<") and names[i].endswith(", 2>")

    proj = OP_KERNELS["compress_projected"][0]
    p0 = next((i for i in range(e3, len(rows)) if proj in rows[i]["Kernel_Name"]), None)
    if p0 is None or p0 + K > len(rows) or not all(is_build(i) for i in range(e3, p0)):
        raise SystemExit("dispatch count does not match the bench's phase layout")
    b1 = p0 + K
    while b1 < len(rows) and is_build(b1):
        b1 += 1
    cuts += [("compress+decompress loop, warm-up", e, e + 6),
             ("compress+decompress loop, timed", e + 6, e + pair),
             ("compress_projected+decompress loop, warm-up", e + pair, e + pair + 6),
             ("compress_projected+decompress loop, timed", e + pair + 6, e2),
             ("compress+decompress, cold (512 MB fill before each pair)", e2, e3),
             ("table build, warm-up", e3, p0),
             ("compress_projected alone", p0, p0 + K),
             ("table build", p0 + K, b1)]
    at = b1
    grass = [i for i in range(at, len(rows))
             if names[i] in GRASS_KERNELS or names[i].split("<")[0] in GRASS_KERNELS]
    if grass:
        cuts.append(("subspace update, AdamW, low-rank table (warm-up included)", at,
                     grass[-1] + 1))
        at = grass[-1] + 1
    if at < len(rows):
        cuts.append(("other configs (1, 4, 3-layer sweep; warm-up included)", at, len(rows)))
    out = os.path.join(ROOT, "profiles", "codec_step_d4096_k40_kernel_stats.md")
    with open(out, "w") as f:
        f.write("# Kernel durations: codec step at d=4096, k=40, N=32768 (bf16)\n\n")
        f.write("Commands (repository root `$R`, output directory `$OUT`; `cd /tmp && export "
                "TMPDIR=/tmp` first):\n\n```\n"
                f"rocprofv3 --kernel-trace --stats -d $OUT/prof_step -o step "
                f"--output-format csv -- python3 $R/bench.py --steps {K} --warmup {W} "
                f"--no-cpu-baseline > $OUT/prof_step.log\n"
                "python3 $R/bench.py --trace-summary $OUT/prof_step $OUT/prof_step.log\n"
                "```\n\n")
        f.write(f"Source hash `{source_hash()}`. Durations are rocprofv3's kernel begin/end "
                f"timestamps; the bench's own figures (HIP events around each launch on the "
                f"launch stream, same run) are in the last column where the phase is the one "
                f"they time.\n\n")
        f.write("| phase | kernel | calls | average (us) | min (us) | max (us) | bench event "
                "mean (us) |\n|---|---|---|---|---|---|---|\n")
        for phase, lo, hi in cuts:
            seen = []
            for n in names[lo:hi]:
                if n not in seen:
                    seen.append(n)
            for n in seen:
                ds = [dur[i] for i in range(lo, hi) if names[i] == n]
                ev = ""
                if phase == "timed steps, event per op":
                    ops_here = [op for op, subs in OP_KERNELS.items() if n in subs]
                    if ops_here and ops_here[0] in b["ops"]:
                        ev = f"{b['ops'][ops_here[0]]['ms'] * 1e3:.1f}"
                elif phase == "compress_projected alone":
                    ev = f"{b['codec_pair_projected']['compress_projected_ms'] * 1e3:.1f}"
                elif phase == "table build":
                    ev = f"{b['codec_pair_projected']['embed_project_ms'] * 1e3:.1f} (call)"
                f.write(f"| {phase} | `{n}` | {len(ds)} | {np.mean(ds):.1f} | {np.min(ds):.1f} "
                        f"| {np.max(ds):.1f} | {ev} |\n")
        f.write("\nBench line of the same run (HIP events):\n\n```\n")
        f.write(json.dumps({"value": b["value"], "unit": b["unit"],
                            "ms_per_step": b["ms_per_step"], "roofline": b["roofline"],
                            "codec_pair": b["codec_pair"]}) + "\n```\n")
    print(open(out).read())


def _pair_times(sn, torch, basis, d, k, tok, E, P, seq, steps, R=2, grad=True):
    """Back-to-back compress+decompress (and grad compress+decompress) over R
    rotating buffer sets of device-drawn inputs; ms per pair (median of the
    means of three timed runs)."""
    N = tok.shape[0]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(N * 7 + d)
    Xs = [torch.randn(N, d, device="cuda", generator=gen).to(torch.bfloat16) for _ in range(R)]
    Cs = [torch.empty(N, k, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Os = [torch.empty(N, d, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    stream = torch.cuda.current_stream()

    def loop(fn, blocks=3):
        # median over `blocks` timed runs of `steps` pairs: one host-side
        # stall inside a run (the GPU idles between launches) skews that
        # run's mean, not the figure
        for i in range(3):
            fn(i % R)
        torch.cuda.synchronize()
        means = []
        for _ in range(blocks):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for i in range(steps):
                fn(i % R)
            b.record(stream)
            torch.cuda.synchronize()
            means.append(a.elapsed_time(b) / steps)
        return float(np.median(means))

    def fwd(j):
        sn.sn_compress(basis, Xs[j], tok=tok, E=E, P=P, seq_len=seq, out=Cs[j])
        sn.sn_decompress(basis, Cs[j], tok=tok, E=E, P=P, seq_len=seq, out=Os[j])

    def bwd(j):
        sn.sn_grad_compress(basis, Xs[j], out=Cs[j])
        sn.sn_decompress(basis, Cs[j], out=Os[j])

    out = {"pair_ms": loop(fwd)}
    # the pair's two kernels on their own: an event pair around each launch
    mk = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))  # noqa: E731
    evs = [(mk(), mk()) for _ in range(steps)]
    for i, ((a, b), (c, e)) in enumerate(evs):
        j = i % R
        a.record(stream)
        sn.sn_compress(basis, Xs[j], tok=tok, E=E, P=P, seq_len=seq, out=Cs[j])
        b.record(stream)
        c.record(stream)
        sn.sn_decompress(basis, Cs[j], tok=tok, E=E, P=P, seq_len=seq, out=Os[j])
        e.record(stream)
    torch.cuda.synchronize()
    out["compress_ms"] = float(np.mean([a.elapsed_time(b) for (a, b), _ in evs]))
    out["decompress_ms"] = float(np.mean([c.elapsed_time(e) for _, (c, e) in evs]))
    if grad:
        out["grad_pair_ms"] = loop(bwd)
    del Xs, Cs, Os
    return out


def other_configs(sn, torch, steps: int) -> dict:
    """The forward and gradient pairs at configs 1 and 4 (N = 32768 and the
    ragged 32767), the config-4 Wo projection, the config-3 sweep of 32 x
    (Wo, W2), and a plain device copy for reference.  U and the ids are the
    configs' own; E, P, X and the weights are drawn on the device with the
    configs' shapes and scales (timing does not depend on the values)."""
    import synth
    res = {}

    def rate(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9

    for cid, ns in ((1, (None,)), (4, (None, 32767))):
        cfg = synth.CONFIGS[cid]
        d, k = cfg.d, cfg.k
        U = to_dev(synth.make_basis(cid)["U"])
        basis = sn.sn_basis_pack(U)
        gen = torch.Generator(device="cuda")
        gen.manual_seed(synth.seed_of(cid, synth.ORD_E))
        E = (torch.randn(cfg.vocab, d, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
        P = (torch.randn(cfg.seq, d, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
        entry = {}
        for n in ns:
            ids = synth.make_ids(cid, n)
            tok = torch.from_numpy(ids["tok"]).cuda()
            N = tok.shape[0]
            t = _pair_times(sn, torch, basis, d, k, tok, E, P, cfg.seq, steps)
            uniq = len(np.unique(ids["tok"])) * d * 2 + min(cfg.seq, N) * d * 2
            pair_bytes = 2 * (N * d * 2 + N * k * 2 + uniq + d * k * 2)
            grad_bytes = 2 * (N * d * 2 + N * k * 2 + d * k * 2)
            entry[f"N{N}"] = {
                "pair_ms": round(t["pair_ms"], 5),
                "pair_GBps": round(rate(pair_bytes, t["pair_ms"]), 1),
                "pair_frac_hbm": round(rate(pair_bytes, t["pair_ms"]) / HBM_PEAK_GBS, 4),
                "pair_tokens_per_s": round(N / (t["pair_ms"] * 1e-3), 1),
                "compress_ms": round(t["compress_ms"], 5),
                "decompress_ms": round(t["decompress_ms"], 5),
                "decompress_frac_hbm": round(rate(pair_bytes / 2, t["decompress_ms"])
                                             / HBM_PEAK_GBS, 4),
                "grad_pair_ms": round(t["grad_pair_ms"], 5),
                "grad_pair_GBps": round(rate(grad_bytes, t["grad_pair_ms"]), 1)}
        for i, (rows, cols) in enumerate(cfg.weights if cid == 4 else ()):
            ws = torch.empty(sn.sn_project_weights_workspace_bytes(d, k, sn.SN_BF16, cols),
                             dtype=torch.uint8, device="cuda")
            Wl = [synth.device_weight(cid, i, rows, cols) for _ in range(2)]
            for j in range(3):
                sn.sn_project_weights(basis, Wl[j % 2], workspace=ws)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for j in range(steps):
                sn.sn_project_weights(basis, Wl[j % 2], workspace=ws)
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / steps
            entry[f"project_W{i}_ms"] = round(ms, 5)
            entry[f"project_W{i}_GBps"] = round(rate(2 * rows * cols * 2, ms), 1)
            del Wl, ws
        res[f"cfg{cid}"] = {"d": d, "k": k, **entry}
        del E, P, basis, U
        torch.cuda.empty_cache()
        print(f"[bench] config {cid} timed", file=sys.stderr, flush=True)

    # config 3: one in-place sweep of 32 layers x (Wo, W2)
    cfg = synth.CONFIGS[3]
    U = to_dev(synth.make_basis(3)["U"])
    basis = sn.sn_basis_pack(U)
    mats = [synth.device_weight(3, 2 * layer + i, r, c)
            for layer in range(cfg.layers) for i, (r, c) in enumerate(cfg.weights)]
    group = 16  # matrices per call: 8 layers of (Wo, W2)
    ws = torch.empty(sn.sn_project_weights_multi_workspace_bytes(
        cfg.d, cfg.k, sn.SN_BF16, [Wm.shape[1] for Wm in mats[:group]]),
        dtype=torch.uint8, device="cuda")

    def sweep():
        for g0 in range(0, len(mats), group):
            sn.sn_project_weights_multi(basis, mats[g0:g0 + group], workspace=ws)

    sweep()
    torch.cuda.synchronize()
    reps = 3
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        sweep()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    nbytes = sum(2 * Wm.numel() * 2 for Wm in mats)
    res["cfg3_sweep"] = {"matrices": len(mats), "ms": round(ms, 4),
                         "GBps": round(rate(nbytes, ms), 1),
                         "frac_hbm": round(rate(nbytes, ms) / HBM_PEAK_GBS, 4)}
    del mats, ws, basis, U
    torch.cuda.empty_cache()

    # reference: a plain device-to-device copy of 1 GiB (reads and writes it)
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / 5
    res["device_copy"] = {"bytes_moved": 2 << 30, "ms": round(ms, 4),
                          "GBps": round(rate(2 << 30, ms), 1)}
    del src, dst
    torch.cuda.empty_cache()
    return res


def grassmann_times(sn, torch, basis, Gs, Cgs, d: int, k: int, N: int, steps: int,
                    op_ms: dict) -> dict:
    """The subspace update of Sec. 4.5 at the step's shape: the per-iteration
    accumulation (gradient coefficients for the wire, the off-subspace loss and
    Y += G^T (G U)), the loss monitor alone, and the step with its QR
    retraction.  Mean ms per call over the same rotating gradient buffers."""
    R = len(Gs)
    state = sn.sn_grassmann_state(basis)
    wsb = sn.sn_grassmann_workspace_bytes(d, k, basis.dt, N)
    wsg = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn, reps):
        for i in range(2):
            fn(i)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(reps):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    acc_ms = timed(lambda i: sn.sn_grassmann_accumulate(basis, Gs[i % R], state, out=Cgs[i % R],
                                                        workspace=wsg), steps)
    mon_ms = timed(lambda i: sn.sn_grassmann_accumulate(basis, Gs[i % R], state, with_su=False,
                                                        out=Cgs[i % R], workspace=wsg), steps)
    Un = torch.empty(d, k, dtype=torch.bfloat16, device="cuda")
    step_ms = timed(lambda i: sn.sn_grassmann_step(basis, state, 1e-3, out=Un, workspace=wsg),
                    max(3, steps // 4))
    del wsg
    es = 2
    # what one iteration must move: G once, the wire coefficients, Y read and written, U
    acc_bytes = N * d * es + N * k * es + 2 * d * k * 8 + d * k * es
    mon_bytes = N * d * es + N * k * es + d * k * es

    def rate(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9

    return {
        "accumulate_ms": round(acc_ms, 5),
        "accumulate_bytes": acc_bytes,
        "accumulate_GBps": round(rate(acc_bytes, acc_ms), 1),
        "accumulate_frac_hbm": round(rate(acc_bytes, acc_ms) / HBM_PEAK_GBS, 4),
        "accumulate_reads_of_G": 2,
        "monitor_ms": round(mon_ms, 5),
        "monitor_GBps": round(rate(mon_bytes, mon_ms), 1),
        "grad_compress_ms": round(op_ms["grad_compress"], 5),
        "step_ms": round(step_ms, 5),
        "step_per_iteration_at_500_ms": round(step_ms / 500, 6),
        "su_flops_per_iteration": 4 * N * d * k,
        "paper_s_accumulation_flops_per_iteration": 2 * N * d * d,
        "paper_s_accumulation_ms_at_bf16_peak": round(2 * N * d * d / 2.5e15 * 1e3, 4),
    }


def adamw_times(sn, torch, weights, steps: int) -> dict:
    """The modified AdamW step of Sec. 5 (column-constant rate) and the
    standard one on the step's weight matrices (bf16 W and G, fp32 moments),
    mean ms per call over two rotating sets."""
    out = {}
    for i, Wl in enumerate(weights):
        rows, cols = Wl[0].shape
        gen = torch.Generator(device="cuda")
        gen.manual_seed(7 + i)
        sets = []
        for j in range(2):
            G = (torch.randn(rows, cols, device="cuda", generator=gen) * 1e-3).to(torch.bfloat16)
            M = torch.zeros(rows, cols, device="cuda")
            V = torch.zeros(rows, cols, device="cuda")
            sets.append((Wl[j], G, M, V))
        ws = torch.empty(sn.sn_adamw_workspace_bytes(rows, cols), dtype=torch.uint8,
                         device="cuda")
        stream = torch.cuda.current_stream()
        res = {}
        for name, sub in (("subspace", True), ("standard", False)):
            def call(t):
                W, G, M, V = sets[t % 2]
                sn.sn_adamw_step(W, G, M, V, t + 1, lr=1e-6, weight_decay=0.0, subspace=sub,
                                 workspace=ws)
            for t in range(2):
                call(t)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for t in range(steps):
                call(2 + t)
            b.record(stream)
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / steps
            # read G, M, V, W and write M, V, W once each (the subspace form reads G twice)
            nbytes = rows * cols * (2 + 4 + 4 + 2 + 4 + 4 + 2)
            res[name] = {"ms": round(ms, 5), "bytes": nbytes,
                         "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "frac_hbm": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        out[f"W{i}_{rows}x{cols}"] = res
        del sets, ws
    torch.cuda.empty_cache()
    return out


def embed_times(sn, torch, basis, w, d: int, k: int, N: int, steps: int) -> dict:
    """The low-rank token table of Sec. 4.3.1 at the step's shape: the
    forward X0 = P + T_fixed[t] + C_S[t] U^T and the backward gC_S +=
    scatter(dX0 U), mean ms per call."""
    cfg = w["cfg"]
    E, P = to_dev(w["E"]), to_dev(w["P"])
    tok = torch.from_numpy(w["tok"]).cuda()
    CS = sn.sn_grad_compress(basis, E)                   # C_S = T_fixed U
    X0 = torch.empty(N, d, dtype=torch.bfloat16, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    dX = (torch.randn(N, d, device="cuda", generator=gen) * 1e-2).to(torch.bfloat16)
    gCS = torch.zeros(cfg.vocab, k, device="cuda")
    wsb = sn.sn_embed_lowrank_workspace_bytes(d, k, basis.dt, N, cfg.vocab)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    fwd = timed(lambda: sn.sn_embed_lowrank_forward(basis, CS, tok, E=E, P=P, seq_len=cfg.seq,
                                                    out=X0, workspace=ws))
    bwd = timed(lambda: sn.sn_embed_lowrank_backward(basis, dX, tok, gCS, workspace=ws))
    uniq = len(np.unique(w["tok"]))
    # forward: X0 written, the batch's unique T_fixed rows and C_S rows, P, U once
    fbytes = N * d * 2 + uniq * (d + k) * 2 + min(cfg.seq, N) * d * 2 + d * k * 2
    # backward: dX0 read, the unique gC_S rows read and written, U
    bbytes = N * d * 2 + 2 * uniq * k * 4 + d * k * 2
    del E, P, X0, dX, gCS, ws, CS
    torch.cuda.empty_cache()
    return {"forward_ms": round(fwd, 5), "forward_bytes": fbytes,
            "forward_GBps": round(fbytes / (fwd * 1e-3) / 1e9, 1),
            "backward_ms": round(bwd, 5), "backward_bytes": bbytes,
            "backward_GBps": round(bbytes / (bwd * 1e-3) / 1e9, 1)}


def load_traffic():
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    return t if t.get("source_hash") == source_hash() else None


# --------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.trace_summary:
        trace_summary(*args.trace_summary)
        return
    if args.counter_summary:
        counter_summary(args.counter_summary)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2506_01260_amd as sn

    w = synth.make_workload(CFG_ID)
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
    Cps = [torch.empty(N, k, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Xrs = [torch.empty(N, d, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    Grs = [torch.empty(N, d, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    weights, host_weights = [], []
    for i, (rows, cols) in enumerate(cfg.weights):
        wb = synth.make_weight(CFG_ID, i, rows, cols)
        host_weights.append(wb)
        base = to_dev(wb)
        weights.append([base.clone() for _ in range(R)])
        del base
    ws_bytes = sn.sn_project_weights_multi_workspace_bytes(d, k, sn.SN_BF16,
                                                          [c for _, c in cfg.weights])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

    # algorithmic bytes per op: inputs and outputs, each unique gathered row once, U once
    es = 2
    uniq_tok = len(np.unique(w["tok"]))
    uniq_e = uniq_tok * d * es
    uniq_p = min(cfg.seq, N) * d * es
    xb, cb, ub = N * d * es, N * k * es, d * k * es
    kp = 16 * ((k + 15) // 16)
    op_bytes = {
        "compress": xb + cb + uniq_e + uniq_p + ub,
        "decompress": cb + xb + uniq_e + uniq_p + ub,
        "grad_compress": xb + cb + ub,
        "grad_decompress": cb + xb + ub,
    }
    # the layer's projection matrices (Wo and W2), confined in one call
    op_bytes["project_weights"] = sum(2 * rows * cols * es for rows, cols in cfg.weights)
    # the projected-table compress reads k-wide fp32 projected rows instead of d-wide ones
    alt_bytes = {"compress_projected": xb + cb + ub + (uniq_tok + min(cfg.seq, N)) * kp * 4,
                 "embed_project": (cfg.vocab + cfg.seq) * d * es + (cfg.vocab + cfg.seq) * kp * 4
                 + ub}

    proj = sn.sn_embed_project(basis, E=E, P=P)

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
        elif name == "compress_projected":
            sn.sn_compress_projected(basis, Xs[j], proj, tok=tok, seq_len=cfg.seq, out=Cps[j])
        elif name == "embed_project":
            sn.sn_embed_project(basis, E=E, P=P)
        elif name == "project_weights":
            sn.sn_project_weights_multi(basis, [wl[j] for wl in weights], workspace=ws)
        else:
            raise ValueError(name)

    names = list(op_bytes)
    stream = torch.cuda.current_stream()

    def step(i, evs=None):
        for nm in names:
            if evs is not None:
                evs[nm][0].record(stream)
            op(nm, i)
            if evs is not None:
                evs[nm][1].record(stream)

    if args.profile_pass:
        # plain streaming kernel of known traffic: reads and writes CALIB_BYTES
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        gstate = sn.sn_grassmann_state(basis)
        for i in range(3):
            step(i)
            op("compress_projected", i)
            sn.sn_grassmann_accumulate(basis, Gs[i % R], gstate, out=Cgs[i % R])
        torch.cuda.synchronize()
        print("[bench] profile pass done", file=sys.stderr, flush=True)
        return

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    K = args.steps
    mk = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))  # noqa: E731
    # eager step time: K steps with events only at the two ends
    t_start, t_end = mk()
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(K):
        step(args.warmup + i)
    t_end.record(stream)
    torch.cuda.synchronize()
    eager_ms = t_start.elapsed_time(t_end) / K
    print(f"[bench] timed {K} eager steps: {eager_ms:.4f} ms/step", file=sys.stderr, flush=True)
    # optionally: the same step captured once per buffer set in a HIP graph
    # (every launch of the step, nothing else) and replayed K times
    ms_step = eager_ms
    graph_ms = None
    if args.graph:
        graphs = []
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            for j in range(R):
                gr = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gr, stream=cap):
                    step(j)
                graphs.append(gr)
        stream.wait_stream(cap)
        for i in range(2 * R):
            graphs[i % R].replay()
        torch.cuda.synchronize()
        t_start, t_end = mk()
        t_start.record(stream)
        for i in range(K):
            graphs[(args.warmup + i) % R].replay()
        t_end.record(stream)
        torch.cuda.synchronize()
        graph_ms = t_start.elapsed_time(t_end) / K
        print(f"[bench] timed {K} graph replays: {graph_ms:.4f} ms/step", file=sys.stderr,
              flush=True)
        del graphs
    # per-op times: K more steps with an event pair around every launch (the
    # marker packets add a few microseconds per op, so these sum to more than
    # the step time above)
    evs = [{nm: mk() for nm in names} for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        step(args.warmup + K + i, evs[i])
    torch.cuda.synchronize()
    samples = {nm: np.array([e[nm][0].elapsed_time(e[nm][1]) for e in evs]) for nm in names}
    op_ms = {nm: float(np.mean(v)) for nm, v in samples.items()}
    print(f"[bench] timed {K} steps per op", file=sys.stderr, flush=True)

    # Steady-state codec pair: compress then decompress, back to back over the
    # buffer rotation.  Timing the pair as a whole charges each iteration for
    # the write-backs the previous one left in the caches, which the per-op
    # event times inside the step can shift from one op to the next.
    def pair_loop(cname):
        # median of three timed runs of K pairs (a host stall skews one run)
        for i in range(3):
            op(cname, i)
            op("decompress", i)
        torch.cuda.synchronize()
        means = []
        for _ in range(3):
            a, b = mk()
            a.record(stream)
            for i in range(K):
                op(cname, args.warmup + i)
                op("decompress", args.warmup + i)
            b.record(stream)
            torch.cuda.synchronize()
            means.append(a.elapsed_time(b) / K)
        return float(np.median(means))

    pair_ms = pair_loop("compress")
    ppair_ms = pair_loop("compress_projected")

    # Cold codec pair: before each iteration a 512 MB fill evicts the caches
    # (the 256 MB Infinity Cache included), so compress finds none of X, E, P
    # or U cached.  Median of the per-iteration times.
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = []
    for i in range(max(5, K // 2)):
        flush.fill_(i & 0xFF)
        a, b = mk()
        a.record(stream)
        op("compress", i)
        op("decompress", i)
        b.record(stream)
        cold.append((a, b))
    torch.cuda.synchronize()
    cold_ms = float(np.median([a.elapsed_time(b) for a, b in cold]))
    del flush

    # the projected-table compress, back to back over the same buffer rotation,
    # and the table build (as after a subspace update; two untimed builds
    # first, so the timed ones reuse the allocator's blocks)
    for _ in range(2):
        op("embed_project", 0)
    torch.cuda.synchronize()
    alt_samples = {"compress_projected": [], "embed_project": []}
    for nm in ("compress_projected", "embed_project"):
        for i in range(K):
            a, b = mk()
            a.record(stream)
            op(nm, args.warmup + i)
            b.record(stream)
            alt_samples[nm].append((a, b))
    torch.cuda.synchronize()
    alt_ms = {nm: float(np.mean([a.elapsed_time(b) for a, b in v])) for nm, v in alt_samples.items()}

    step_bytes = sum(op_bytes.values())
    value = step_bytes / (ms_step * 1e-3) / 1e9

    def rate(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9

    ops = {nm: {"ms": round(op_ms[nm], 5), "ms_median": round(float(np.median(samples[nm])), 5),
                "ms_min": round(float(np.min(samples[nm])), 5), "bytes": op_bytes[nm],
                "GBps": round(rate(op_bytes[nm], op_ms[nm]), 1),
                "frac_hbm": round(rate(op_bytes[nm], op_ms[nm]) / HBM_PEAK_GBS, 4)}
           for nm in names}
    pair_bytes = op_bytes["compress"] + op_bytes["decompress"]
    ppair_bytes = alt_bytes["compress_projected"] + op_bytes["decompress"]
    # the roofline is a kernel's: among the ops that are one kernel launch (the
    # projection is three), the one that takes longest; every op of the step
    # is listed beside it with its own fraction, so the op furthest below its
    # roofline is visible whatever its share of the step
    single = [nm for nm in names if nm in OP_KERNELS]
    dom = max(single, key=lambda nm: op_ms[nm])
    dom_gbs = rate(op_bytes[dom], op_ms[dom])
    traffic = load_traffic()

    def traffic_of(nm):
        if traffic and nm in traffic.get("ops", {}):
            return round(traffic["ops"][nm]["traffic_bytes"])
        return None
    dom_traffic = traffic_of(dom)
    kernels = [{"op": nm, "launches": 1 if nm in OP_KERNELS else len(PROJ_PASSES),
                "achieved": round(rate(op_bytes[nm], op_ms[nm]), 1),
                "frac": round(rate(op_bytes[nm], op_ms[nm]) / HBM_PEAK_GBS, 4),
                "traffic": traffic_of(nm) if nm in OP_KERNELS else
                (round(sum(traffic["ops"][p]["traffic_bytes"] for p in PROJ_PASSES))
                 if traffic and all(p in traffic.get("ops", {}) for p in PROJ_PASSES) else None)}
               for nm in names]
    lowest = min(kernels, key=lambda e: e["frac"])

    pair_gbs = rate(pair_bytes, pair_ms)
    out = {
        "metric": "codec GB/s & % HBM peak (compress+decompress) at d=4096,k=40; tokens/s",
        "value": round(pair_gbs, 1),
        "value_is": "codec_pair: compress + decompress back to back (algorithmic bytes of the "
                    "pair / pair time); the whole step (all hot-path ops) is under 'step'",
        "frac_hbm": round(pair_gbs / HBM_PEAK_GBS, 4),
        "frac_is": "algorithmic bytes of the pair / pair time / 8 TB/s (gathered rows largely "
                   "served by the Infinity Cache in the back-to-back loop); cold_GBps is the same "
                   "pair after a 512 MB flush",
        "cold_GBps": round(rate(pair_bytes, cold_ms), 1),
        "cold_frac_hbm": round(rate(pair_bytes, cold_ms) / HBM_PEAK_GBS, 4),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "graph_replay_ms_per_step": None if graph_ms is None else round(graph_ms, 5),
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
                   "unique_tokens": uniq_tok, "rotate_buffers": R},
        "tokens_per_s": round(N / (pair_ms * 1e-3), 1),
        "step": {"ops": names, "ms": round(ms_step, 5), "bytes": step_bytes,
                 "GBps": round(value, 1), "frac_hbm": round(value / HBM_PEAK_GBS, 4),
                 "tokens_per_s": round(N / (ms_step * 1e-3), 1)},
        "codec_pair": {"ops": "compress+decompress, back to back", "ms": round(pair_ms, 5),
                       "in_step_ms": round(op_ms["compress"] + op_ms["decompress"], 5),
                       "GBps": round(rate(pair_bytes, pair_ms), 1),
                       "frac_hbm": round(rate(pair_bytes, pair_ms) / HBM_PEAK_GBS, 4),
                       "tokens_per_s": round(N / (pair_ms * 1e-3), 1),
                       "x_c_only_GBps": round(rate(2 * (xb + cb), pair_ms), 1),
                       "cold_ms_median": round(cold_ms, 5),
                       "cold_GBps": round(rate(pair_bytes, cold_ms), 1)},
        "codec_pair_projected": {
            "ops": "compress_projected+decompress, back to back (tables built once per basis)",
            "ms": round(ppair_ms, 5), "GBps": round(rate(ppair_bytes, ppair_ms), 1),
            "frac_hbm": round(rate(ppair_bytes, ppair_ms) / HBM_PEAK_GBS, 4),
            "tokens_per_s": round(N / (ppair_ms * 1e-3), 1),
            "compress_projected_ms": round(alt_ms["compress_projected"], 5),
            "embed_project_ms": round(alt_ms["embed_project"], 5),
            "embed_project_per_step_at_500_steps_ms": round(alt_ms["embed_project"] / 500, 6)},
        "ops": ops,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(dom_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dom_gbs / HBM_PEAK_GBS, 4), "traffic": dom_traffic,
                     "algorithmic_bytes": op_bytes[dom], "kernels": kernels,
                     "lowest_frac_op": lowest["op"]},
    }
    out["grassmann"] = grassmann_times(sn, torch, basis, Gs, Cgs, d, k, N, K, op_ms)
    print("[bench] subspace update timed", file=sys.stderr, flush=True)
    out["adamw"] = adamw_times(sn, torch, weights, K)
    print("[bench] AdamW timed", file=sys.stderr, flush=True)
    out["embed_lowrank"] = embed_times(sn, torch, basis, w, d, k, N, K)
    print("[bench] low-rank token table timed", file=sys.stderr, flush=True)
    if not args.no_other_configs:
        del Xs, Gs, Cs, Cgs, Cps, Xrs, Grs, weights
        torch.cuda.empty_cache()
        out["other_configs"] = other_configs(sn, torch, K)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, host_weights)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

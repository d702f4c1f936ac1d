"""Benchmark: causal prefill then decode of symmetry-aware Taylor attention on one MI355X.

Workload (d_k = d_v = 32, P = 4, D = 6545 features, bf16 q/k/v, float32 state):
  prefill  B=8, H=32, n=8192 tokens, chunk 64, from an empty state;
  decode   1024 steps for every (b, h), continuing from the prefill state.
One step = one prefill over the batch plus the 1024 decode steps.  Inputs are
seeded synthetic N(0,1) tensors resident in HBM before timing starts.

Prints ONE JSON line.  `value` is whole-job tokens/s: (B*n + B*decode_steps)
tokens per step divided by the step time; the prefill and decode rates are
reported separately next to it.  `roofline` is for the kernel that takes the
largest share of the step (`rooflines` lists both); its achieved rate is the
algorithmic work of one launch divided by the launch's average duration,
measured with HIP events on the stream the kernels run on.  The CPU baseline
leg times the float64 oracle on a sample of the same workload and also checks
the timed GPU output against it on a few rows.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--decode-steps M] [--no-cpu-baseline]

`--workload` selects one of the other workload shapes instead, each printing
its own line in the same form:
  decode_d16  B=64, H=32, d_k=d_v=16, P=4, bf16: 2048-token prefill, then 4096
              decode steps (the decode figure is the one that counts);
  large_d64   B=2, H=8, d_k=d_v=64, P=4 (D=47905), bf16: 4096-token prefill,
              then 1024 decode steps;
  decode_hbm  B=16, H=32, d_k=d_v=32, P=4, bf16: a 256-token prefill, then 1024
              decode steps over 442 MB of state, beyond the 256 MB Infinity
              Cache (the headline's 221 MB fits in it);
  sweep_d16   B=1, H=64, d_k=d_v=16, float32, n=65536: prefill for each P in
              2..6 (the CPU leg also reports the error against softmax);
  error_study one head of 100,000 tokens, float32, for each d_k = d_v in
              {8, 16, 32} with P = 1..6 and d = 64 with P = 1..5: the
              prefill is timed, and the CPU leg measures its output against
              exact float64 softmax attention on sampled rows, overall and by
              token position, in decimal orders of magnitude of the elementwise
              absolute difference (the reconstruction measure of App. A3-A4);
  context_sweep one head per head size d_k = d_v in {8, 16, 32} with
              contexts of 10^3 ... 10^8 tokens (d = 64: up to 10^7), float32,
              P = 4: prefill time and device memory per token, then 64 decode
              steps (per-step time), and the CPU leg checks decoded rows at the
              longest context, far beyond 2^24 tokens, against the oracle
              (Sec. 3.2: cost per token that does not grow with the context);
  backward    B=8, H=32, n=2048, d_k=d_v=32, P=4, bf16: dL/dq, dL/dk, dL/dv
              (float32 arithmetic), checked on two heads against the oracle;
  decode_grouped B=8, 32 query heads, d_k=d_v=32, P=4, bf16: an 8192-token
              prefill of the key/value heads, then 1024 grouped decode steps
              for G = 2, 4, 8 query heads per key/value head (16, 8, 4
              key/value heads); one state read per key/value head serves its
              G query heads.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
# float32 vector peak (packed FMA counted): the bound of the float32 prefill path
PEAK_F32_TFLOPS = 157.3

WORKLOAD_ID = 3
B, H, N, DK, DV, P, CHUNK = 8, 32, 8192, 32, 32, 4, 64


def feature_count(d, p):
    return math.comb(d + p - 1, p - 1)


def prefill_flops_per_head_token(dk, dv, P, C):
    """Algorithmic prefill work per head-token: the two state contractions,
    readout phi(Q_c) S and update phi(K_c)^T [V_c|1], 2*D*(d_v+1) each, plus the
    causal intra-chunk term, on average (C+1)/2 keys per query times
    2*d_k (scores) + 2*(d_v+1) (weights times [v|1])."""
    D = feature_count(dk, P)
    return 4 * D * (dv + 1) + (C + 1) * (dk + dv + 1)


def decode_bytes_per_head_step(dk, dv, P, elem_bytes):
    """Algorithmic decode traffic per head-step: read and write the float32
    state once, D*(d_v+1)*8 bytes, plus q, k, v in and y out."""
    D = feature_count(dk, P)
    return 8 * D * (dv + 1) + elem_bytes * (2 * dk + 2 * dv)


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 summaries.

    Each summary under profiles/ carries a line
      traffic_record: kernel=<name> source=<file> sha256_16=<hash> bytes_per_launch=<bytes>
    with calibrated FETCH_SIZE + WRITE_SIZE counts.  The figure holds only for the
    source it was taken on, so None is returned once that file has changed."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for line in open(path):
            if not line.startswith("traffic_record:"):
                continue
            rec = dict(kv.split("=", 1) for kv in line.split()[1:])
            if rec.get("kernel") != kernel:
                continue
            src = os.path.join(ROOT, rec["source"])
            if not os.path.exists(src):
                return None
            digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
            return int(rec["bytes_per_launch"]) if digest == rec["sha256_16"] else None
    return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--decode-steps", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-heads", type=int, default=48)
    ap.add_argument("--cpu-sample-decode-rows", type=int, default=128)
    ap.add_argument("--workload", default="headline", choices=["headline", "decode_d16", "large_d64", "sweep_d16",
                                                                  "decode_hbm", "error_study", "context_sweep",
                                                                  "decode_grouped", "backward", "feature_map"])
    ap.add_argument("--seq-len", type=int, default=0,
                    help="error_study only: tokens per sequence (default 100000)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, run one device-to-device copy of this many MiB (a kernel of "
                         "known traffic for calibrating hardware byte counters)")
    return ap.parse_args()


def make_inputs(dec_steps):
    import numpy as np
    import torch

    import sata_synth as syn
    n_tot = N + dec_steps
    q = np.empty((B, H, n_tot, DK), np.float32)
    k = np.empty((B, H, n_tot, DK), np.float32)
    v = np.empty((B, H, n_tot, DV), np.float32)
    for b in range(B):
        for h in range(H):
            q[b, h], k[b, h], v[b, h] = syn.make_head(WORKLOAD_ID, b, h, n_tot, DK, DV, "bf16")
    dev = torch.device("cuda:0")

    def up(a):
        return torch.from_numpy(a).to(dev).to(torch.bfloat16)

    pre = [up(np.ascontiguousarray(a[:, :, :N])) for a in (q, k, v)]
    # decode inputs laid out [step][B][H][d] so every step reads a contiguous slice
    dec = [up(np.ascontiguousarray(a[:, :, N:].transpose(2, 0, 1, 3))) for a in (q, k, v)]
    return pre, dec


def blas_threads():
    """Threads of the BLAS library numpy uses (the oracle's matrix products)."""
    try:
        import threadpoolctl
        info = [i for i in threadpoolctl.threadpool_info() if i.get("user_api") == "blas"]
        return {i.get("internal_api", "blas"): i.get("num_threads") for i in info} or None
    except Exception:
        return None


def cpu_baseline(n_heads, dec_rows, y_gpu=None):
    """Times the float64 oracle on a bounded sample of the same workload, and
    checks the GPU prefill output y_gpu ([B, H, n, d_v] on the host) against it
    on a few rows of the first and last head; on those rows it also measures the
    GPU output against exact float64 softmax attention, the paper's measure of
    the approximation (log10 of the elementwise absolute difference)."""
    import numpy as np

    import oracle
    import sata_synth as syn
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    rng = np.random.default_rng(7)
    heads = [(0, 0), (B - 1, H - 1)] + [(int(b), int(h)) for b, h in
                                         zip(rng.integers(0, B, n_heads), rng.integers(0, H, n_heads))]
    heads = heads[:n_heads]
    t_pre = t_dec = 0.0
    for b, h in heads:
        q, k, v = syn.make_head(WORKLOAD_ID, b, h, N + dec_rows, DK, DV, "bf16")
        t0 = time.perf_counter()
        oracle.taylor_attention(q[:N], k[:N], v[:N], P)
        t1 = time.perf_counter()
        oracle.taylor_attention_rows(q, k, v, P, list(range(N, N + dec_rows)))
        t2 = time.perf_counter()
        t_pre += t1 - t0
        t_dec += t2 - t1
    # seconds per head-token, scaled to tokens of the whole batch (H heads per token)
    pre_tok_s = (len(heads) * N) / t_pre / H
    dec_tok_s = (len(heads) * dec_rows) / t_dec / H
    parity = {}
    soft = None
    if y_gpu is not None:
        lds = []
        rows = sorted({0, 63, 64, 4095, N - 1} | set(range(N - 512, N, 16)))
        for (b, h) in ((0, 0), (B - 1, H - 1)):
            q, k, v = syn.make_head(WORKLOAD_ID, b, h, N, DK, DV, "bf16")
            yr, _, kap = oracle.taylor_attention_rows(q, k, v, P, rows)
            err, _ = oracle.max_row_rel_error(y_gpu[b, h, rows], yr, kap)
            parity[f"b{b}h{h}"] = err
            lds.append(oracle.log10_abs_diff(y_gpu[b, h, rows], oracle.softmax_attention_rows(q, k, v, rows)))
        a = np.concatenate([x.ravel() for x in lds])
        soft = {"P": P, "measure": "log10 |y_gpu - y_softmax| elementwise (float64 exact softmax)",
                "rows": f"{len(rows)} rows ({rows[0]}..{rows[-1]}) of heads (0,0) and ({B - 1},{H - 1})",
                "median": float(np.median(a)), "p99": float(np.percentile(a, 99)), "max": float(a.max())}
    return {
        "value": None, "unit": "tokens/s", "cores": threads, "blas_threads": blas_threads(), "kind": "oracle",
        "prefill_tokens_per_s": pre_tok_s, "decode_tokens_per_s": dec_tok_s,
        "sample": (f"{len(heads)} of {B * H} heads: full {N}-token causal prefill by the direct "
                   f"float64 definition, plus {dec_rows} decode rows at positions {N}..{N + dec_rows - 1}; "
                   f"rates scaled to whole-batch tokens (1 token = {H} head-tokens); decode rows near "
                   f"position {N} stand in for all {B}x{H} decode rows"),
        "seconds": t_pre + t_dec,
        "parity_max_row_rel_err": parity,
        "error_vs_softmax": soft,
    }


WORKLOADS = {
    # name: (synthetic stream id, B, H, prefill n, d, P values, dtype, decode steps)
    "decode_d16": (2, 64, 32, 2048, 16, [4], "bf16", 4096),
    "large_d64": (4, 2, 8, 4096, 64, [4], "bf16", 1024),
    "sweep_d16": (5, 1, 64, 65536, 16, [2, 3, 4, 5, 6], "f32", 0),
    # the headline head shape with twice the heads: 442 MB of state, more than
    # the 256 MB Infinity Cache, so every decode step streams it from HBM
    "decode_hbm": (6, 16, 32, 256, 32, [4], "bf16", 1024),
}


def run_workload(args, sata, torch):
    """One of the other workload shapes: prefill (per P) and decode, timed like
    the headline; returns the JSON line."""
    import numpy as np

    import sata_synth as syn
    wid, Bw, Hw, n, d, Ps, dt, n_dec = WORKLOADS[args.workload]
    n_dec = n_dec if args.decode_steps == 1024 else args.decode_steps
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    ebytes = 2 if dt == "bf16" else 4
    q = np.empty((Bw, Hw, n + n_dec, d), np.float32)
    k, v = np.empty_like(q), np.empty_like(q)
    for b in range(Bw):
        for h in range(Hw):
            q[b, h], k[b, h], v[b, h] = syn.make_head(wid, b, h, n + n_dec, d, d, dt)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(tdt)
    pre = [up(a[:, :, :n]) for a in (q, k, v)]
    dec = [up(a[:, :, n:].transpose(2, 0, 1, 3)) for a in (q, k, v)]
    del q, k, v
    y = torch.empty(Bw, Hw, n, d, dtype=tdt, device="cuda")
    ydec = torch.empty(max(n_dec, 1), Bw, Hw, d, dtype=tdt, device="cuda")
    per_P = {}
    t_total = 0.0
    roof_pre = roof_dec = None
    for Pw in Ps:
        D = feature_count(d, Pw)
        S = torch.empty(Bw, Hw, D, d + 1, dtype=torch.float32, device="cuda")

        def step(ev):
            ev[0].record()
            sata.prefill(*pre, Pw, CHUNK, y=y, S=S)
            ev[1].record()
            for t in range(n_dec):
                sata.decode_step(S, dec[0][t], dec[1][t], dec[2][t], Pw, y=ydec[t])
            ev[2].record()
        for _ in range(args.warmup):
            step([torch.cuda.Event(enable_timing=True) for _ in range(3)])
        torch.cuda.synchronize()
        events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for s_ in range(args.steps):
            step(events[s_])
        torch.cuda.synchronize()
        pre_ms = sum(e[0].elapsed_time(e[1]) for e in events) / args.steps
        dec_ms = sum(e[1].elapsed_time(e[2]) for e in events) / args.steps if n_dec else 0.0
        t_total += pre_ms + dec_ms
        flops = prefill_flops_per_head_token(d, d, Pw, CHUNK) * Bw * Hw * n
        # on the matrix cores: bf16 operands (bf16 peak), or float32 inputs as
        # split bf16 pairs (priced at the float32 matrix peak of their dtype)
        ops = sata.prefill_operands(tdt, Bw, Hw, n, d, d, Pw, CHUNK)
        mfma = ops in ("bf16", "split")
        peak = PEAK_BF16_TFLOPS if ops == "bf16" else PEAK_F32_TFLOPS
        ach = flops / (pre_ms * 1e-3) / 1e12
        roof_pre = {"kernel": "sata_prefill (all launches of one call)", "bound": "mfma" if mfma else "alu",
                    "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak, "traffic": None,
                    "work_per_launch": flops}
        entry = {"prefill_ms": pre_ms, "prefill_tokens_per_s": Bw * n / (pre_ms * 1e-3), "prefill_roofline": roof_pre}
        if n_dec:
            dbytes = decode_bytes_per_head_step(d, d, Pw, ebytes) * Bw * Hw
            dach = dbytes / (dec_ms * 1e-3 / n_dec) / 1e9
            roof_dec = {"kernel": "sata_decode_step (all launches of one call)", "bound": "hbm", "achieved": dach,
                        "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": dach / PEAK_HBM_GBS, "traffic": None,
                        "work_per_launch": dbytes}
            entry.update({"decode_ms_per_step": dec_ms / n_dec, "decode_tokens_per_s": Bw * n_dec / (dec_ms * 1e-3),
                          "decode_roofline": roof_dec})
        per_P[str(Pw)] = entry
        del S
    tokens = Bw * (n + n_dec) * len(Ps)
    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": tokens / (t_total * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t_total, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dt, "data": "synthetic",
        "config": {"workload": (f"{args.workload}: causal prefill B={Bw} H={Hw} n={n} d_k=d_v={d} "
                                f"P={'/'.join(map(str, Ps))} {dt} chunk={CHUNK}"
                                + (f" then {n_dec} decode steps" if n_dec else "")),
                   "global_batch": Bw, "seq_len": n, "decode_steps": n_dec, "heads": Hw, "d_k": d, "d_v": d,
                   "P": Ps if len(Ps) > 1 else Ps[0], "chunk": CHUNK, "parallelism": "single GPU"},
        "per_P": per_P,
        "roofline": roof_dec if roof_dec is not None else roof_pre,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_workload(wid, Bw, Hw, n, d, Ps, dt, y if len(Ps) == 1 else None,
                                                     pre if len(Ps) > 1 else None, sata, torch)
        for Pw, e in line["cpu_baseline"]["per_P"].items():
            if "gpu_log10_abs_diff_vs_softmax" in e:
                per_P[Pw]["error_vs_softmax"] = {
                    "measure": "log10 |y_gpu - y_softmax| elementwise (float64 exact softmax)",
                    "rows": line["cpu_baseline"]["sample"], **e["gpu_log10_abs_diff_vs_softmax"]}
    return line


def cpu_baseline_workload(wid, Bw, Hw, n, d, Ps, dt, y_gpu, pre, sata, torch):
    """The oracle on two heads of the workload: its rate on a bounded row sample,
    the GPU output's error against it on those rows and, for the sweep, the
    error against exact softmax attention per P (of the GPU output, and of the
    oracle's float64 P-term output on the same rows)."""
    import numpy as np

    import oracle
    import sata_synth as syn
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    heads = [(0, 0), (Bw - 1, Hw - 1)]
    rows = sorted({0, 63, 64, n // 2, n - 1} | set(range(n - 96, n, 8)))
    out = {"value": None, "unit": "tokens/s", "cores": threads, "blas_threads": blas_threads(), "kind": "oracle",
           "sample": f"rows {rows[0]}..{rows[-1]} ({len(rows)} rows) of heads {heads}, direct float64 definition"}
    t = 0.0
    per_P = {}
    soft = {}  # exact softmax rows per head (independent of P)
    if len(Ps) > 1:
        for (b, h) in heads:
            q, k, v = syn.make_head(wid, b, h, n, d, d, dt)
            soft[(b, h)] = oracle.softmax_attention_rows(q, k, v, rows)
    for Pw in Ps:
        if y_gpu is None:  # the sweep: run each P again to have its output
            yP, _ = sata.prefill(*pre, Pw, CHUNK, want_state=False)
            torch.cuda.synchronize()
        else:
            yP = y_gpu
        yh = yP.float().cpu().numpy()
        errs, lds, lds_gpu = [], [], []
        for (b, h) in heads:
            q, k, v = syn.make_head(wid, b, h, n, d, d, dt)
            t0 = time.perf_counter()
            yr, _, kap = oracle.taylor_attention_rows(q, k, v, Pw, rows)
            t += time.perf_counter() - t0
            errs.append(oracle.max_row_rel_error(yh[b, h, rows], yr, kap)[0])
            if soft:
                lds.append(oracle.log10_abs_diff(yr, soft[(b, h)]))
                lds_gpu.append(oracle.log10_abs_diff(yh[b, h, rows], soft[(b, h)]))
        entry = {"parity_max_row_rel_err": max(errs)}

        def summary(parts):
            a = np.concatenate([x.ravel() for x in parts])
            a = a[np.isfinite(a)]
            return {"median": float(np.median(a)), "p99": float(np.percentile(a, 99)), "max": float(a.max())}
        if lds:
            entry["gpu_log10_abs_diff_vs_softmax"] = summary(lds_gpu)
            entry["log10_abs_diff_vs_softmax"] = summary(lds)
        per_P[str(Pw)] = entry
    out["value"] = len(heads) * len(rows) * len(Ps) / t / Hw
    out["seconds"] = t
    out["per_P"] = per_P
    return out


ERROR_STUDY_CELLS = [(d, p) for d in (8, 16, 32) for p in range(1, 7)] + [(64, p) for p in range(1, 6)]
ERROR_STUDY_N = 100_000


def error_study_rows(n):
    """Query rows the error study samples: log-spaced over the positions (so
    that every decade of context is represented) plus uniformly drawn ones."""
    import numpy as np
    logr = np.unique(np.round(np.logspace(0, math.log10(n), 96)).astype(np.int64) - 1)
    uni = np.random.default_rng(2602).integers(0, n, 64)
    return sorted(set(int(r) for r in logr if 0 <= r < n) | set(int(r) for r in uni))


def run_error_study(args, sata, torch):
    """Prefill of one 100K-token head per (d, P) cell, timed; the CPU leg
    compares the outputs with exact softmax attention (App. A3-A4)."""
    import numpy as np

    import sata_synth as syn
    n = args.seq_len or ERROR_STUDY_N
    cells, outs = {}, {}
    t_total = 0.0
    for d, Pw in ERROR_STUDY_CELLS:
        q, k, v = syn.make_head(600 + d, 0, 0, n, d, d, "f32")
        dev = [torch.from_numpy(a).to("cuda").view(1, 1, n, d) for a in (q, k, v)]
        y = torch.empty(1, 1, n, d, dtype=torch.float32, device="cuda")
        S = torch.empty(1, 1, feature_count(d, Pw), d + 1, dtype=torch.float32, device="cuda")
        for _ in range(args.warmup):
            sata.prefill(*dev, Pw, CHUNK, y=y, S=S)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        ev[0].record()
        for s_ in range(args.steps):
            sata.prefill(*dev, Pw, CHUNK, y=y, S=S)
            ev[s_ + 1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[-1]) / args.steps
        t_total += ms
        flops = prefill_flops_per_head_token(d, d, Pw, CHUNK) * n
        ach = flops / (ms * 1e-3) / 1e12
        cells[f"d{d}_P{Pw}"] = {
            "d": d, "P": Pw, "D": feature_count(d, Pw), "prefill_ms": ms, "prefill_tokens_per_s": n / (ms * 1e-3),
            "prefill_roofline": {"kernel": "sata_prefill (all launches of one call)", "bound": "alu",
                                 "achieved": ach, "peak": PEAK_F32_TFLOPS, "unit": "TFLOP/s",
                                 "frac": ach / PEAK_F32_TFLOPS, "traffic": None, "work_per_launch": flops}}
        outs[(d, Pw)] = y[0, 0].cpu().numpy()
        del dev, y, S
    worst = min(cells.values(), key=lambda c: c["prefill_roofline"]["frac"])
    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": n * len(cells) / (t_total * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t_total, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": (f"error_study: causal prefill of one head, n={n}, float32, chunk={CHUNK}, "
                                f"for d_k=d_v in 8/16/32 with P=1..6 and 64 with P=1..5"),
                   "global_batch": 1, "seq_len": n, "decode_steps": 0, "heads": 1, "chunk": CHUNK,
                   "parallelism": "single GPU"},
        "cells": cells,
        "roofline": worst["prefill_roofline"],
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_error_study(n, outs)
    return line


def cpu_baseline_error_study(n, outs):
    """Per cell, on the sampled rows: the GPU output against the float64 oracle
    (parity), and both against exact float64 softmax attention as
    log10 |difference| per output element: median, 99th percentile and maximum
    overall, and the median per decade of token position."""
    import numpy as np

    import oracle
    import sata_synth as syn
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    rows = error_study_rows(n)
    pos = np.asarray(rows)
    decades = [(0, 10), (10, 100), (100, 1000), (1000, 10000), (10000, n)]
    summary = lambda a: {"median": float(np.median(a)), "p99": float(np.percentile(a, 99)), "max": float(a.max())}
    per_cell = {}
    t = 0.0
    soft = {}
    for (d, Pw), y_gpu in outs.items():
        q, k, v = syn.make_head(600 + d, 0, 0, n, d, d, "f32")
        if d not in soft:
            soft[d] = oracle.softmax_attention_rows(q, k, v, rows)
        t0 = time.perf_counter()
        yr, _, kap = oracle.taylor_attention_rows(q, k, v, Pw, rows)
        t += time.perf_counter() - t0
        lg = oracle.log10_abs_diff(y_gpu[rows], soft[d])
        lo = oracle.log10_abs_diff(yr, soft[d])
        by_pos = {}
        for lo_, hi_ in decades:
            m = (pos >= lo_) & (pos < hi_)
            if m.any():
                by_pos[f"{lo_}-{hi_ - 1}"] = float(np.median(lg[m]))
        per_cell[f"d{d}_P{Pw}"] = {
            "parity_max_row_rel_err": oracle.max_row_rel_error(y_gpu[rows], yr, kap)[0],
            "gpu_vs_softmax_log10": summary(lg.ravel()),
            "oracle_vs_softmax_log10": summary(lo.ravel()),
            "gpu_vs_softmax_median_log10_by_position": by_pos}
    return {"value": len(outs) * len(rows) / t, "unit": "rows/s", "cores": threads, "kind": "oracle",
            "sample": (f"{len(rows)} query rows (96 log-spaced positions and 64 uniform ones) of each cell's "
                       f"{n}-token head, direct float64 definition; the softmax reference on the same rows"),
            "seconds": t, "per_cell": per_cell}


GROUPED_QUERY_HEADS = 32
GROUPED_GS = [2, 4, 8]


def run_decode_grouped(args, sata, torch):
    """Grouped-query decode at the headline head size: prefill the key/value
    heads, then time the decode steps for each G; returns the JSON line."""
    import numpy as np

    import sata_synth as syn
    n_dec = args.decode_steps
    per_G = {}
    t_total = 0.0
    roof = None
    for G in GROUPED_GS:
        Hkv = GROUPED_QUERY_HEADS // G
        q = np.empty((B, GROUPED_QUERY_HEADS, n_dec, DK), np.float32)
        for b in range(B):
            for h in range(GROUPED_QUERY_HEADS):
                q[b, h] = syn.head_stream(900 + G, b, h, syn.TENSOR_Q, (n_dec, DK), "bf16")
        k = np.empty((B, Hkv, N + n_dec, DK), np.float32)
        v = np.empty((B, Hkv, N + n_dec, DV), np.float32)
        for b in range(B):
            for h in range(Hkv):
                k[b, h] = syn.head_stream(900 + G, b, h, syn.TENSOR_K, (N + n_dec, DK), "bf16")
                v[b, h] = syn.head_stream(900 + G, b, h, syn.TENSOR_V, (N + n_dec, DV), "bf16")
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(torch.bfloat16)
        kk, vv = up(k[:, :, :N]), up(v[:, :, :N])
        _, S0 = sata.prefill(kk, kk, vv, P, CHUNK)  # the state does not depend on q
        dq, dk_, dv_ = (up(a.transpose(2, 0, 1, 3)) for a in (q, k[:, :, N:], v[:, :, N:]))
        del q, k, v, kk, vv
        S = torch.empty_like(S0)
        ydec = torch.empty(n_dec, B, GROUPED_QUERY_HEADS, DV, dtype=torch.bfloat16, device="cuda")

        def steps_once():
            for t in range(n_dec):
                sata.decode_step_grouped(S, dq[t], dk_[t], dv_[t], P, y=ydec[t])
        ms = []
        for it in range(args.warmup + args.steps):
            S.copy_(S0)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            steps_once()
            e1.record()
            torch.cuda.synchronize()
            if it >= args.warmup:
                ms.append(e0.elapsed_time(e1))
        step_ms = sum(ms) / len(ms) / n_dec
        t_total += step_ms * n_dec
        D = feature_count(DK, P)
        dbytes = B * Hkv * (8 * D * (DV + 1) + 2 * (DK + DV)) + B * GROUPED_QUERY_HEADS * 2 * (DK + DV)
        ach = dbytes / (step_ms * 1e-3) / 1e9
        r = {"kernel": "decode_grouped_kernel (one launch per step)", "bound": "hbm", "achieved": ach,
             "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": None,
             "work_per_launch": dbytes}
        per_G[str(G)] = {"kv_heads": B * Hkv, "query_heads": B * GROUPED_QUERY_HEADS, "decode_us_per_step": step_ms * 1e3,
                         "decode_tokens_per_s": B / (step_ms * 1e-3),
                         "query_head_tokens_per_s": B * GROUPED_QUERY_HEADS / (step_ms * 1e-3), "roofline": r}
        roof = r if roof is None else roof
        print(f"grouped G={G}: {step_ms * 1e3:.1f} us/step, {ach:.0f} GB/s", file=sys.stderr, flush=True)
        del S, S0, dq, dk_, dv_, ydec
        torch.cuda.empty_cache()
    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": B * n_dec * len(GROUPED_GS) / (t_total * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t_total, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": (f"decode_grouped: B={B}, {GROUPED_QUERY_HEADS} query heads, d_k=d_v={DK}, P={P}, bf16, "
                                f"{N}-token prefill of the key/value heads then {n_dec} grouped decode steps, "
                                f"G={'/'.join(map(str, GROUPED_GS))}"),
                   "global_batch": B, "seq_len": N, "decode_steps": n_dec, "heads": GROUPED_QUERY_HEADS,
                   "d_k": DK, "d_v": DV, "P": P, "parallelism": "single GPU"},
        "per_G": per_G,
        "roofline": roof,
    }
    return line


CONTEXT_SWEEP = [(8, 8), (16, 8), (32, 8), (64, 7)]  # (d, largest power of ten of the context)
CONTEXT_DECODE = 64


def backward_flops_per_head_token(dk, dv, P, C):
    """Algorithmic work of the backward per head-token: the forward readout
    recomputed (2 D (d_v+1)), the forward scan's S h readout and state update
    (2 x 2 D (d_v+1)), the reverse scan's U [v|1] readout, U^T phi(k) and U
    update (2 D (d_v+1) + 2 D d_v + 2 D (d_v+1)), the two Jacobian products of
    the feature map (2 x 2 (P-1) D), and the intra-chunk terms (about
    (C+1)(3 d_k + 2 d_v + 3) per token)."""
    D = feature_count(dk, P)
    E = dv + 1
    return 2 * D * E + 4 * D * E + (4 * D * E + 2 * D * dv) + 4 * (P - 1) * D + (C + 1) * (3 * dk + 2 * dv + 3)


def run_backward(args, sata, torch):
    """sata_backward on B=8, H=32, n=2048, d_k=d_v=32, P=4, bf16 (the
    benchmark's head shape, a quarter of its length); the CPU leg checks two
    heads' gradients against the float64 oracle."""
    import numpy as np

    import sata_synth as syn
    Bw, Hw, n, d, Pw, C, wid = 8, 32, 2048, 32, 4, 64, 7
    arrs = [np.empty((Bw, Hw, n, d), np.float32) for _ in range(4)]
    for b in range(Bw):
        for h in range(Hw):
            arrs[0][b, h], arrs[1][b, h], arrs[2][b, h] = syn.make_head(wid, b, h, n, d, d, "bf16")
            arrs[3][b, h] = syn.head_stream(wid, b, h, 3, (n, d), "bf16")
    dev = [torch.from_numpy(a).to("cuda").to(torch.bfloat16) for a in arrs]
    for _ in range(args.warmup):
        sata.backward(*dev, Pw, C)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(args.steps):
        out = sata.backward(*dev, Pw, C)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / args.steps
    flops = backward_flops_per_head_token(d, d, Pw, C) * Bw * Hw * n
    ach = flops / (ms * 1e-3) / 1e12
    line = {
        "metric": "backward tokens/s (d_k=32,P=4); % float32 roofline",
        "value": Bw * n / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"backward: dL/dq, dL/dk, dL/dv of the causal prefill, B={Bw} H={Hw} n={n} "
                               f"d_k=d_v={d} P={Pw} bf16 chunk={C}, float32 arithmetic",
                   "global_batch": Bw, "seq_len": n, "heads": Hw, "d_k": d, "d_v": d, "P": Pw, "chunk": C,
                   "parallelism": "single GPU"},
        "roofline": {"kernel": "sata_backward (all launches of one call)", "bound": "alu", "achieved": ach,
                     "peak": PEAK_F32_TFLOPS, "unit": "TFLOP/s", "frac": ach / PEAK_F32_TFLOPS, "traffic": None,
                     "work_per_launch": flops},
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
        got = [o.float().cpu().numpy() for o in out]
        errs = {}
        t = 0.0
        for (b, h) in ((0, 0), (Bw - 1, Hw - 1)):
            t0 = time.perf_counter()
            want = oracle.taylor_attention_backward(arrs[0][b, h], arrs[1][b, h], arrs[2][b, h], arrs[3][b, h], Pw)
            t += time.perf_counter() - t0
            for name, g_, w_ in zip(("dq", "dk", "dv"), got, want):
                errs[f"b{b}h{h}_{name}"] = float(np.linalg.norm(g_[b, h] - w_) / np.linalg.norm(w_))
        line["cpu_baseline"] = {"value": 2 * n / t / Hw, "unit": "tokens/s", "cores": threads,
                                "blas_threads": blas_threads(), "kind": "oracle",
                                "sample": f"2 of {Bw * Hw} heads, full {n}-token backward by the direct float64 "
                                          "definition; rate scaled to whole-batch tokens",
                                "seconds": t, "parity_rel_err": errs}
    return line


# feature-map workload: (d, P, rows) with about 1-2 GB of float32 features written per call
FEATURE_MAP_SHAPES = [(16, 4, 262144), (32, 4, 65536), (64, 4, 8192)]


def run_feature_map(args, sata, torch):
    """sata_feature_map alone (Sec. 2.4, "Efficient Computation"): bf16 rows of
    N(0,1) coordinates expanded to their C(d+3, 3) float32 features.  Bound:
    HBM, 4 D + 2 d bytes per row (features written, coordinates read)."""
    import numpy as np

    import sata_synth as syn
    per = {}
    t_total = 0.0
    for (d, P, rows) in FEATURE_MAP_SHAPES:
        D = feature_count(d, P)
        x = torch.from_numpy(syn.head_stream(950 + d, 0, 0, syn.TENSOR_Q, (rows, d), "bf16")).to("cuda").to(
            torch.bfloat16)
        phi = torch.empty(rows, D, dtype=torch.float32, device="cuda")  # one output, reused
        for _ in range(args.warmup):
            sata.feature_map(x, P, phi=phi)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            sata.feature_map(x, P, phi=phi)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        t_total += ms
        nbytes = rows * (4 * D + 2 * d)
        ach = nbytes / (ms * 1e-3) / 1e9
        r = {"kernel": "feature_map_kernel (one launch per call)", "bound": "hbm", "achieved": ach,
             "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": None,
             "work_per_launch": nbytes}
        per[f"d{d}_P{P}"] = {"rows": rows, "D": D, "ms": ms, "rows_per_s": rows / (ms * 1e-3), "roofline": r}
        print(f"feature map d={d} P={P} rows={rows}: {ms:.3f} ms, {ach:.0f} GB/s", file=sys.stderr, flush=True)
        del x, phi
        torch.cuda.empty_cache()
    dom = max(per.values(), key=lambda e: e["ms"])["roofline"]
    total_rows = sum(r for (_, _, r) in FEATURE_MAP_SHAPES)
    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": total_rows / (t_total * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t_total, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "feature_map: bf16 rows -> float32 features, " +
                   ", ".join(f"d={d} P={P} rows={r}" for (d, P, r) in FEATURE_MAP_SHAPES),
                   "parallelism": "single GPU"},
        "per_shape": per, "roofline": dom,
    }
    print(json.dumps(line), flush=True)


def run_context_sweep(args, sata, torch):
    """Prefill of contexts 10^3 ... 10^8 tokens, then decode steps, per head
    size; time and device memory per token.  Inputs: sata_synth.long_head."""
    import numpy as np

    import sata_synth as syn
    Pw = 4
    cells = {}
    keep = {}
    t_total = 0.0
    for d, emax in CONTEXT_SWEEP:
        n_max = 10 ** emax
        q, k, v = syn.long_head(700 + d, n_max + CONTEXT_DECODE, d, d)
        for e in range(3, emax + 1):
            T = 10 ** e
            torch.cuda.synchronize()
            sata.release()  # so that what the library holds afterwards is this call's own
            torch.cuda.reset_peak_memory_stats()
            free0 = torch.cuda.mem_get_info()[0]
            base = torch.cuda.memory_allocated()
            res0 = torch.cuda.memory_reserved()
            dev = [torch.from_numpy(a[:T]).to("cuda").view(1, 1, T, d) for a in (q, k, v)]
            y = torch.empty(1, 1, T, d, dtype=torch.float32, device="cuda")
            S = torch.empty(1, 1, feature_count(d, Pw), d + 1, dtype=torch.float32, device="cuda")
            dq, dk_, dv_ = (torch.from_numpy(np.ascontiguousarray(a[T:T + CONTEXT_DECODE])).to("cuda")
                            .view(CONTEXT_DECODE, 1, 1, d) for a in (q, k, v))
            ydec = torch.empty(CONTEXT_DECODE, 1, 1, d, dtype=torch.float32, device="cuda")
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            torch.cuda.synchronize()
            ev[0].record()
            sata.prefill(*dev, Pw, CHUNK, y=y, S=S)
            ev[1].record()
            for t in range(CONTEXT_DECODE):
                sata.decode_step(S, dq[t], dk_[t], dv_[t], Pw, y=ydec[t])
            ev[2].record()
            torch.cuda.synchronize()
            pre_ms = ev[0].elapsed_time(ev[1])
            dec_ms = ev[1].elapsed_time(ev[2]) / CONTEXT_DECODE
            # device memory: what torch allocated for the call (inputs, outputs,
            # state) plus what the library holds (tables, workspace), read from
            # the device's free memory
            torch_peak = torch.cuda.max_memory_allocated() - base
            lib_held = max(0, (free0 - torch.cuda.mem_get_info()[0]) - (torch.cuda.memory_reserved() - res0))
            t_total += pre_ms + dec_ms * CONTEXT_DECODE
            cells[f"d{d}_T{T}"] = {
                "d": d, "context": T, "prefill_ms": pre_ms, "prefill_ns_per_token": pre_ms * 1e6 / T,
                "decode_us_per_step": dec_ms * 1e3, "state_bytes": S.numel() * 4,
                "device_bytes_peak": int(torch_peak + lib_held),
                "device_bytes_per_token": (torch_peak + lib_held) / T}
            print(f"context d={d} T={T}: prefill {pre_ms:.1f} ms, decode {dec_ms * 1e3:.1f} us/step",
                  file=sys.stderr, flush=True)
            if e == emax:
                keep[d] = ydec[:, 0, 0].cpu().numpy()
            del dev, y, S, dq, dk_, dv_, ydec
            torch.cuda.empty_cache()
        del q, k, v
    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": sum(c["context"] + CONTEXT_DECODE for c in cells.values()) / (t_total * 1e-3),
        "unit": "tokens/s", "n_gpus": 1, "steps": 1, "warmup": 0, "ms_per_step": t_total,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": (f"context_sweep: one head, float32, P={Pw}, chunk={CHUNK}: prefill of 10^3..10^8 "
                                f"tokens (d=64: ..10^7) then {CONTEXT_DECODE} decode steps, d_k=d_v in 8/16/32/64"),
                   "global_batch": 1, "seq_len": 10 ** 8, "decode_steps": CONTEXT_DECODE, "heads": 1, "P": Pw,
                   "chunk": CHUNK, "parallelism": "single GPU"},
        "cells": cells,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_context(keep, Pw)
    return line


def cpu_baseline_context(keep, Pw):
    """The oracle at the longest context of each head size: decoded rows
    0, 31 and 63 (positions just past 10^emax), direct float64 definition."""
    import numpy as np

    import oracle
    import sata_synth as syn
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    out, t = {}, 0.0
    for d, emax in CONTEXT_SWEEP:
        n_max = 10 ** emax
        q, k, v = syn.long_head(700 + d, n_max + CONTEXT_DECODE, d, d)
        steps = [0, CONTEXT_DECODE // 2 - 1, CONTEXT_DECODE - 1]
        print(f"oracle d={d} T={n_max}", file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        yr, _, kap = oracle.taylor_attention_rows(q, k, v, Pw, [n_max + s for s in steps])
        t += time.perf_counter() - t0
        out[f"d{d}_T{n_max}"] = {"decode_rows": steps,
                                 "max_row_rel_err": oracle.max_row_rel_error(keep[d][steps], yr, kap)[0]}
        del q, k, v
    return {"value": sum(3 * (10 ** e + CONTEXT_DECODE) for _, e in CONTEXT_SWEEP) / t, "unit": "keys/s",
            "cores": threads, "kind": "oracle",
            "sample": "3 decoded rows after the longest context of each head size, direct float64 definition",
            "seconds": t, "parity": out}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(heads shard across GPUs with no exchange, so per-GPU throughput is the N=1 figure)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2602_00294_amd as sata
    sata.load_library()
    assert torch.cuda.is_available(), "no GPU"
    if args.workload == "decode_grouped":
        print(json.dumps(run_decode_grouped(args, sata, torch)), flush=True)
        return
    if args.workload == "backward":
        print(json.dumps(run_backward(args, sata, torch)), flush=True)
        return
    if args.workload == "feature_map":
        run_feature_map(args, sata, torch)
        return
    if args.workload == "context_sweep":
        print(json.dumps(run_context_sweep(args, sata, torch)), flush=True)
        return
    if args.workload == "error_study":
        print(json.dumps(run_error_study(args, sata, torch)), flush=True)
        return
    if args.workload != "headline":
        print(json.dumps(run_workload(args, sata, torch)), flush=True)
        return

    pre, dec = make_inputs(args.decode_steps)
    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    D = feature_count(DK, P)
    y = torch.empty(B, H, N, DV, dtype=torch.bfloat16, device="cuda")
    S = torch.empty(B, H, D, DV + 1, dtype=torch.float32, device="cuda")
    ydec = torch.empty(args.decode_steps, B, H, DV, dtype=torch.bfloat16, device="cuda")

    def one_step(ev=None):
        if ev:
            ev[0].record()
        sata.prefill(*pre, P, CHUNK, y=y, S=S)
        if ev:
            ev[1].record()
        for t in range(args.decode_steps):
            sata.decode_step(S, dec[0][t], dec[1][t], dec[2][t], P, y=ydec[t])
        if ev:
            ev[2].record()

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        one_step(events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    pre_ms = sum(e[0].elapsed_time(e[1]) for e in events) / args.steps
    dec_ms = sum(e[1].elapsed_time(e[2]) for e in events) / args.steps
    step_ms = wall * 1e3 / args.steps
    tokens = B * N + B * args.decode_steps
    value = tokens / (step_ms * 1e-3)
    pre_tok_s = B * N / (pre_ms * 1e-3)
    dec_tok_s = B * args.decode_steps / (dec_ms * 1e-3)

    pre_flops = prefill_flops_per_head_token(DK, DV, P, CHUNK) * B * H * N
    pre_ach = pre_flops / (pre_ms * 1e-3) / 1e12
    dec_bytes = decode_bytes_per_head_step(DK, DV, P, 2) * B * H
    dec_ach = dec_bytes / (dec_ms * 1e-3 / args.decode_steps) / 1e9
    t_main, t_fin = measured_traffic("prefill_mfma_main"), measured_traffic("prefill_mfma_finalize")
    pre_traffic = t_main + t_fin if t_main is not None and t_fin is not None else None
    roof_pre = {"kernel": "sata_prefill (all launches of one call)", "bound": "mfma",
                "achieved": pre_ach, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": pre_ach / PEAK_BF16_TFLOPS, "traffic": pre_traffic,
                "work_per_launch": pre_flops}
    roof_dec = {"kernel": "sata_decode_step (all launches of one call)", "bound": "hbm",
                "achieved": dec_ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": dec_ach / PEAK_HBM_GBS, "traffic": measured_traffic("decode_flat_kernel"),
                "work_per_launch": dec_bytes}
    dominant = roof_pre if pre_ms >= dec_ms else roof_dec

    line = {
        "metric": "prefill tokens/s + decode tokens/s (d_k=32,P=4); % MFMA/HBM roofline",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": step_ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": (f"causal prefill B={B} H={H} n={N} d_k=d_v={DK} P={P} (D={D}) bf16 chunk={CHUNK} "
                                f"then {args.decode_steps} decode steps"),
                   "global_batch": B, "seq_len": N, "decode_steps": args.decode_steps, "heads": H,
                   "d_k": DK, "d_v": DV, "P": P, "chunk": CHUNK, "parallelism": "single GPU"},
        "prefill_tokens_per_s": pre_tok_s, "decode_tokens_per_s": dec_tok_s,
        "prefill_ms": pre_ms, "decode_ms_per_step": dec_ms / args.decode_steps,
        "roofline": dominant, "rooflines": {"prefill": roof_pre, "decode": roof_dec},
    }
    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        cb = cpu_baseline(args.cpu_sample_heads, args.cpu_sample_decode_rows, y.float().cpu().numpy())
        whole = tokens / (B * N / cb["prefill_tokens_per_s"] + B * args.decode_steps / cb["decode_tokens_per_s"])
        cb["value"] = whole
        line["error_vs_softmax"] = cb.pop("error_vs_softmax")
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

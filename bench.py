"""Benchmark: log-linear Mamba-2 chunkwise forward on one MI355X.

One step = one ll_mamba2_fwd call over the whole workload (all three kernel stages: tile
states, level scan, tile outputs), inputs already resident in HBM.  Default workload:
B=1, H=16, T=65536, d_k=d_v=128, C=64, bf16 q/k/v with fp32 gates and lambda (17 levels).

Prints ONE JSON line with throughput (tokens/s), TFLOP/s against the bf16 MFMA peak, the
lambda == NULL (Mamba-2) run of the same library, per-stage durations read from HIP events
recorded between the stages of every timed step, the roofline of the dominant kernel and the
float64 oracle timed on the host cores.

FLOP convention (counted, not issued): log-linear Mamba-2
    F = B*H*T*[2C(d_k+d_v) + 2 d_k d_v + d_k d_v log2(T/C)]
(dense C x C intra-chunk blocks, chunk states, one inter-chunk product per (chunk, set bit)),
and for the lambda == NULL Mamba-2 run  F = B*H*T*[2C(d_k+d_v) + 4 d_k d_v].
Algorithmic bytes: q, k, v, log alpha, lambda read once and o written once.
"""

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synthetic import WORKLOADS, generate  # noqa: E402

METRIC = "fwd tokens/sec + TFLOP/s (% bf16 MFMA peak), log-linear Mamba-2, T=64K"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def flops_loglinear(w):
    J = math.log2(w.T // w.C) if w.T > w.C else 0.0
    return w.B * w.H * w.T * (2 * w.C * (w.dk + w.dv) + 2 * w.dk * w.dv + w.dk * w.dv * J)


def flops_mamba2(w):
    return w.B * w.H * w.T * (2 * w.C * (w.dk + w.dv) + 4 * w.dk * w.dv)


STAGES = ["block_state", "block_scan", "tile_out"]
KERNEL_SOURCES = ["paper_2506_04761_amd/csrc/ll_mamba2.hip", "paper_2506_04761_amd/csrc/ll_device.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "tile_out_ll_mamba2_bf16_T65536_hbm_traffic.md")


def stage_figures(w, has_lambda=True):
    """Algorithmic work of one launch of each stage: (bound, amount).  FLOPs for the MFMA
    stages under the convention above; bytes for the scan (HBM-bound, elementwise)."""
    es = 2 if w.dtype == "bf16" else 4
    BH, BHT = w.B * w.H, w.B * w.H * w.T
    SZ = w.dk * w.dv
    J_chunk = math.log2(w.T // w.C) if w.T > w.C else 0.0
    f_state = 2.0 * BHT * w.dk * w.dv
    f_out = BHT * (2 * w.C * (w.dk + w.dv) + (w.dk * w.dv * J_chunk if has_lambda else 2 * w.dk * w.dv))
    R = 4 * w.C                              # tile = 4 chunks
    N = -(-w.T // R)                         # tiles per sequence
    NB = -(-N // 4)                          # 4-tile blocks
    J = (N - 1).bit_length() if N > 1 else 0  # inter-tile levels
    if has_lambda:
        # read: block summaries, tile totals; write: summaries of levels >= 4, gaps (fp32, N x J)
        nup = sum(-(-(N - (1 << (j - 1))) // (1 << j)) for j in range(4, J + 1) if N > (1 << (j - 1)))
        b_scan = BH * ((NB + nup) * SZ * es + N * 4 + N * J * 4)
    else:
        # read: tile states, tile totals; write: running state entering each tile
        b_scan = BH * (2 * N * SZ * es + N * 4)
    return {"block_state": ("mfma", f_state), "block_scan": ("hbm", b_scan), "tile_out": ("mfma", f_out)}


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(workload):
    """HBM bytes per tile_out launch from the committed counter summary (FETCH_SIZE and
    WRITE_SIZE, calibrated against a plain copy), or None when there is none for this workload
    or the kernel sources changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    rec = {}
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            if line.startswith("- ") and ": " in line:
                key, val = line[2:].split(": ", 1)
                rec[key.strip()] = val.strip().strip("`")
    if rec.get("workload") != workload or rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def algorithmic_bytes(w):
    es = 2 if w.dtype == "bf16" else 4
    BTH = w.B * w.T * w.H
    return BTH * ((w.dk * 2 + w.dv) * es + 4 + w.levels * 4 + w.dv * es)


def cpu_baseline(w, budget_s):
    """Time the float64 oracle's per-level recurrent form on a prefix of the workload (all heads),
    growing the prefix until one run takes at least `budget_s` / 4; report tokens/s."""
    from oracle import mamba2
    x = generate(w.with_(T=min(w.T, 4096)))
    L = w.levels
    lam_full = np.zeros(x["lam"].shape[:-1] + (L,), np.float32)
    lam_full[..., :x["lam"].shape[-1]] = x["lam"]
    T = 32
    while True:
        sl = slice(0, T)
        t0, c0 = time.perf_counter(), time.process_time()
        mamba2.recurrent(x["q"][:, sl], x["k"][:, sl], x["v"][:, sl], x["log_alpha"][:, sl], lam_full[:, sl])
        wall, cpu = time.perf_counter() - t0, time.process_time() - c0
        if wall >= budget_s / 4 or T >= x["q"].shape[1]:
            break
        T *= 2
    return {
        "value": w.B * T / wall,
        "unit": "tokens/s",
        "cores": max(1, round(cpu / wall)),
        "host_cores_available": len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": f"float64 per-level recurrent form (Sec. 3.2 states, Eq. 3 output), first {T} tokens of "
                  f"all {w.H} heads, B={w.B}, {L} level states; {wall:.2f} s wall, {cpu:.2f} s CPU",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="ll_mamba2_bf16_T65536")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device-to-device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the operator's "
              "multi-GPU sharding is a design note, not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2506_04761_amd as ll

    w = WORKLOADS[args.workload]
    assert w.variant == "mamba2"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = generate(w)
    d = {n: torch.from_numpy(x[n]).to(dev).to(dt).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev)
    lam = torch.from_numpy(x["lam"]).to(dev)
    del x
    out = torch.empty((w.B, w.T, w.H, w.dv), dtype=dt, device=dev)
    code = ll.LL_BF16 if w.dtype == "bf16" else ll.LL_F32
    ws_bytes = max(ll.ll_workspace_size(ll.LL_MAMBA2, code, w.B, w.T, w.H, w.dk, w.dv, w.C, has_l)
                   for has_l in (0, 1))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def run(lmb):
        ll.ll_mamba2_fwd(d["q"], d["k"], d["v"], la, lmb, w.C, out=out, workspace=ws, stream=stream)

    def timed_plain(lmb, K, W):
        for _ in range(W):
            run(lmb)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(K):
            run(lmb)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    def timed_staged(K, W):
        """K timed steps, each recording HIP events between its kernel stages on the launch
        stream; returns (ms per step over the whole region, mean ms of each stage)."""
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(max(K, 1))]
        for i in range(W):
            ll.ll_mamba2_fwd_staged(d["q"], d["k"], d["v"], la, lam, w.C, evs[i % K], out=out, workspace=ws,
                                    stream=stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(K):
            ll.ll_mamba2_fwd_staged(d["q"], d["k"], d["v"], la, lam, w.C, evs[i], out=out, workspace=ws,
                                    stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        st = np.array([[e[s].elapsed_time(e[s + 1]) for s in range(3)] for e in evs[:K]]).mean(axis=0)
        return e0.elapsed_time(e1) / K, st

    print(f"[bench] {w.name}: warmup {args.warmup}, steps {args.steps}", file=sys.stderr, flush=True)
    ms, stage_ms = timed_staged(args.steps, args.warmup)
    ms_m2 = timed_plain(None, args.steps, args.warmup)
    print(f"[bench] log-linear {ms:.3f} ms/step (stages {', '.join(f'{x:.3f}' for x in stage_ms)}), "
          f"lambda=NULL {ms_m2:.3f} ms/step", file=sys.stderr, flush=True)

    figs = stage_figures(w)
    dom = int(np.argmax(stage_ms))
    bound, amount = figs[STAGES[dom]]
    if bound == "mfma":
        achieved = amount / (stage_ms[dom] * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS
        unit = "TFLOP/s"
    else:
        achieved = amount / (stage_ms[dom] * 1e-3) / 1e9
        peak, unit = PEAK_HBM_GBS, "GB/s"
    traffic = recorded_traffic(w.name) if STAGES[dom] == "tile_out" else None

    F = flops_loglinear(w)
    tflops = F / (ms * 1e-3) / 1e12
    F2 = flops_mamba2(w)
    res = {
        "metric": METRIC,
        "value": w.B * w.T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "variant": "log-linear Mamba-2", "B": w.B, "H": w.H, "T": w.T,
                   "d_k": w.dk, "d_v": w.dv, "C": w.C, "levels": w.levels,
                   "inputs": "bf16 q/k/v, fp32 log-gates and lambda, seeded synthetic (numpy PCG64)"},
        "tflops": tflops,
        "mfma_peak_frac": tflops / (PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS),
        "flop_convention": "B*H*T*[2C(dk+dv) + 2dk*dv + dk*dv*log2(T/C)]",
        "hbm_GBps_algorithmic": algorithmic_bytes(w) / (ms * 1e-3) / 1e9,
        "mamba2_lambda_null": {"ms_per_step": ms_m2, "tokens_per_s": w.B * w.T / (ms_m2 * 1e-3),
                               "tflops": F2 / (ms_m2 * 1e-3) / 1e12},
        "log_factor_overhead": ms / ms_m2,
        "stages_ms": dict(zip(STAGES, [float(x) for x in stage_ms])),
        "roofline": {"kernel": STAGES[dom], "bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": achieved / peak, "traffic": traffic,
                     "algorithmic_per_launch": amount,
                     "traffic_note": "HBM bytes per launch (FETCH_SIZE x 2 + WRITE_SIZE, copy-calibrated)"},
    }
    if args.copy_mib:
        # A plain copy kernel of known size: its FETCH_SIZE / WRITE_SIZE counters calibrate the
        # HBM traffic that the same counters report for the kernels above.
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

"""Benchmark: log-linear Mamba-2 chunkwise forward on one MI355X.

One step = one ll_mamba2_fwd call over the whole workload, inputs already resident in HBM.  For
bf16 with C = 64 that is the single-pass path (tile totals, block sums of the totals, the tile
kernel that forms and consumes the Fenwick nodes); otherwise the three-kernel path (tile states,
the level scan, tile outputs).  Default workload (the headline): B=1, H=16, T=65536,
d_k=d_v=128, C=64, bf16 q/k/v with fp32 gates and lambda (17 levels).

Prints ONE JSON line with throughput (tokens/s), TFLOP/s against the bf16 MFMA peak, the same
kernels with lambda = 1 and the lambda == NULL Mamba-2 path, per-stage durations read from HIP
events recorded between the stages of every timed step, the roofline of the dominant kernel, the
float64 oracle timed on the host cores, and (default run) the other workloads of the scope table
(T = 2048, T = 8192 with its lambda = 1 run, and the Gated DeltaNet forward) as sub-objects.

FLOP convention (counted, not issued): log-linear Mamba-2
    F = B*H*T*[2C(d_k+d_v) + 2 d_k d_v + d_k d_v log2(T/C)]
(dense C x C intra-chunk blocks, chunk states, one inter-chunk product per (chunk, set bit)),
and for Mamba-2 (lambda == NULL)  F = B*H*T*[2C(d_k+d_v) + 4 d_k d_v].
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

from synthetic import WORKLOADS, generate, shared_qk  # noqa: E402

METRIC = "fwd tokens/sec + TFLOP/s (% bf16 MFMA peak), log-linear Mamba-2, T=64K"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def flops_loglinear(w):
    J = math.log2(w.T // w.C) if w.T > w.C else 0.0
    return w.B * w.H * w.T * (2 * w.C * (w.dk + w.dv) + 2 * w.dk * w.dv + w.dk * w.dv * J)


def flops_mamba2(w):
    return w.B * w.H * w.T * (2 * w.C * (w.dk + w.dv) + 4 * w.dk * w.dv)


STAGES = ["block_state", "scan", "tile_out"]
FUSED_STAGES = ["tile_totals", "block_sums", "fused_tile"]
KERNEL_SOURCES = ["paper_2506_04761_amd/csrc/ll_mamba2_fused.hip", "paper_2506_04761_amd/csrc/ll_fast_tile.hpp",
                  "paper_2506_04761_amd/csrc/ll_mamba2_common.hpp", "paper_2506_04761_amd/csrc/ll_device.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fused_tile_ll_mamba2_bf16_T65536_hbm_traffic.md")


def fused_traffic_file(workload):
    """The committed counter summary of the single-pass tile kernel for one workload."""
    return os.path.join(ROOT, "profiles", f"fused_tile_{workload}_hbm_traffic.md")
# the GDN forward's counter record (block tree + read-out stage) and the sources it depends on
GDN_KERNEL_SOURCES = ["paper_2506_04761_amd/csrc/ll_gdn.hip", "paper_2506_04761_amd/csrc/ll_device.hpp",
                      "paper_2506_04761_amd/csrc/ll_launch.hpp"]
GDN_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ll_gdn_bf16_T8192_hbm_traffic.md")


def fused_path(w):
    """Whether ll_mamba2_fwd takes the single-pass kernels for this workload (with or without
    lambda)."""
    return w.dtype == "bf16" and w.C == 64 and w.dk in (64, 128) and w.dv in (64, 128)


def fused_stage_figures(w):
    """Algorithmic work of one launch of each single-pass stage: {stage: (flops, bytes)}.
    tile_totals reads the log-gates and writes one total per tile; block_sums reads and writes the
    block sums of those totals; fused_tile reads q, k, v, the log-gates and lambda and writes o --
    the path's algorithmic bytes -- and does all of the path's FLOPs.  The Fenwick nodes the tiles
    write and read are implementation traffic (see the rocprofv3 counters)."""
    N = -(-w.T // 128)
    BH = w.B * w.H
    b_tot = w.B * w.T * w.H * 4 + BH * N * 4
    b_sum = BH * 2 * N * 4
    return {"tile_totals": (0.0, b_tot), "block_sums": (0.0, b_sum),
            "fused_tile": (flops_loglinear(w), algorithmic_bytes(w))}


def tree_nodes_read(N):
    """Block-tree nodes above the blocks that tiles of a sequence of N tiles read: node (l, k)
    covers blocks [k 2^l, (k+1) 2^l) and is read when k is even and a tile follows its group."""
    nb = -(-N // 4)
    count, l = 0, 1
    while (1 << (l + 2)) < N:
        count += sum(1 for k in range(0, -(-nb // (1 << l)), 2) if ((k + 1) << (l + 2)) < N)
        l += 1
    return count


def stage_figures(w, has_lambda=True):
    """Algorithmic work of one launch of each stage: {stage: (flops, bytes)}.

    FLOPs follow the convention above.  Bytes: block_state reads k, v and the log-gates and
    writes the summaries it produces; scan reads the block summaries and writes the block-tree
    nodes tiles read (lambda == NULL: tile states in, running states out); tile_out reads q, k,
    v, the log-gates and lambda and writes o -- the path's algorithmic bytes.  Summary reads
    inside tile_out are implementation traffic (see the rocprofv3 counters)."""
    es = 2 if w.dtype == "bf16" else 4
    BH, BHT = w.B * w.H, w.B * w.H * w.T
    SZ = w.dk * w.dv
    J_chunk = math.log2(w.T // w.C) if w.T > w.C else 0.0
    R = max(2 * w.C, 64)                     # tile rows
    N = -(-w.T // R)                         # tiles per sequence
    NB = -(-N // 4)                          # 4-tile blocks
    L = w.levels if has_lambda else 0
    f_state = 2.0 * BHT * w.dk * w.dv
    f_out = BHT * (2 * w.C * (w.dk + w.dv) + (w.dk * w.dv * J_chunk if has_lambda else 2 * w.dk * w.dv))
    if has_lambda:
        n_state_out = -(-N // 2) + -(-N // 4) + NB  # even tile states, pair and block summaries
        b_scan = BH * ((NB + tree_nodes_read(N)) * SZ * es + NB * 4)
    else:
        n_state_out = N
        b_scan = BH * (2 * N * SZ * es + N * 4)
    qk = qk_share(w)  # q, k bytes per head relative to one q/k head per head
    b_state = BHT * ((w.dk * qk + w.dv) * es + 4) + BH * (n_state_out * SZ * es + N * 4)
    b_out = BHT * ((2 * w.dk * qk + 2 * w.dv) * es + 4 + L * 4)
    return {"block_state": (f_state, b_state), "scan": (0.0, b_scan), "tile_out": (f_out, b_out)}


def roofline(w, flops, nbytes, ms):
    """Roofline position of one kernel launch: the bound is whichever of the MFMA time and the
    HBM time of its algorithmic work is longer; both fractions are reported."""
    peak_f = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS
    t_f = flops / (peak_f * 1e12)
    t_b = nbytes / (PEAK_HBM_GBS * 1e9)
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = nbytes / (ms * 1e-3) / 1e9
    if t_f >= t_b:
        r = {"bound": "mfma", "achieved": tflops, "peak": peak_f, "unit": "TFLOP/s"}
    else:
        r = {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    r["frac"] = r["achieved"] / r["peak"]
    r["mfma_frac"] = tflops / peak_f
    r["hbm_frac"] = gbs / PEAK_HBM_GBS
    r["algorithmic_flops"] = flops
    r["algorithmic_bytes"] = nbytes
    return r


def kernel_source_hash(sources=None):
    """Hash of the kernel sources (default: the single-pass forward's) with comments and blank
    lines removed (comment edits do not change the kernel)."""
    import hashlib
    h = hashlib.sha256()
    for f in sources or KERNEL_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            for line in fh:
                code = line.split("//", 1)[0].strip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def recorded_traffic(workload, traffic_file=TRAFFIC_FILE, sources=None):
    """HBM bytes per launch (per stage for a multi-kernel stage) from a committed counter summary
    (FETCH_SIZE and WRITE_SIZE, calibrated against a plain copy), or None when there is none for
    this workload or the kernel sources changed since the counters were taken."""
    if not os.path.exists(traffic_file):
        return None
    rec = {}
    with open(traffic_file) as fh:
        for line in fh:
            if line.startswith("- ") and ": " in line:
                key, val = line[2:].split(": ", 1)
                rec[key.strip()] = val.strip().strip("`")
    if rec.get("workload") != workload or rec.get("kernel_source_sha256") != kernel_source_hash(sources):
        return None
    try:
        return float(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def measured_gemm_tflops(torch, dev, n=8192, reps=10):
    """bf16 TFLOP/s of a large plain matrix product (n x n x n through torch, i.e. the vendor BLAS)
    on this GPU: a measured second denominator for the MFMA fraction."""
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    for _ in range(3):
        torch.matmul(a, b)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        torch.matmul(a, b)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2.0 * n ** 3 / (ms * 1e-3) / 1e12


def blas_threads():
    """Threads of the BLAS library NumPy uses (the oracle's matrix products), if it can be read."""
    try:
        import threadpoolctl
        info = [i for i in threadpoolctl.threadpool_info() if i.get("user_api") == "blas"]
        return max(i["num_threads"] for i in info) if info else None
    except Exception:
        return None


def qk_share(w):
    """Query/key heads per head: 1, or H_qk / H when heads share them in groups."""
    return (w.qk_heads or w.H) / w.H


def algorithmic_bytes(w):
    es = 2 if w.dtype == "bf16" else 4
    BTH = w.B * w.T * w.H
    return BTH * ((w.dk * 2 * qk_share(w) + w.dv) * es + 4 + w.levels * 4 + w.dv * es)


def _pool_init():
    """Worker set-up: one BLAS thread per worker process (the workers are the parallelism)."""
    try:
        import threadpoolctl
        threadpoolctl.threadpool_limits(1)
    except Exception:
        pass
    import oracle  # noqa: F401  (imported before the timed calls)


def _pool_ready(_):
    return os.getpid()


def _oracle_part(job):
    """One worker's share of the CPU baseline: the recurrent oracle on a group of heads; returns
    its compute seconds."""
    variant, arrs = job
    from oracle import gdn, mamba2
    t0 = time.perf_counter()
    if variant == "gdn":
        gdn.recurrent(*arrs)
    else:
        mamba2.recurrent(*arrs)
    return time.perf_counter() - t0, os.getpid()


def cpu_baseline(w, budget_s):
    """Time the float64 oracle's per-level recurrent form on a prefix of the workload, all heads:
    the heads are dealt to a pool of worker processes, one per host core (at most 16, the CPU share
    of one GPU), each with one BLAS thread.  The prefix doubles until one run takes at least
    `budget_s` / 2; the time is that of the slowest worker (all run at once)."""
    import concurrent.futures
    import multiprocessing
    x = generate(w.with_(T=min(w.T, 16384)))
    if w.qk_heads:  # the shared q, k repeated to every head of its group: the same computation
        G = w.H // w.qk_heads
        q, k = shared_qk(x, w)
        x["q"], x["k"] = np.repeat(q, G, axis=2), np.repeat(k, G, axis=2)
    L = w.levels
    lam_full = np.zeros(x["lam"].shape[:-1] + (L,), np.float32)
    lam_full[..., :x["lam"].shape[-1]] = x["lam"]
    names = ["q", "k", "v", "log_alpha"] + (["beta"] if w.variant == "gdn" else [])
    arrays = [x[n] for n in names] + [lam_full]
    cores = max(1, min(len(os.sched_getaffinity(0)), 16))
    groups = [g for g in np.array_split(np.arange(w.H), min(cores, w.H)) if len(g)]
    ctx = multiprocessing.get_context("spawn")  # fresh interpreters: nothing of this process's GPU state
    with concurrent.futures.ProcessPoolExecutor(max_workers=len(groups), mp_context=ctx,
                                                initializer=_pool_init) as pool:
        list(pool.map(_pool_ready, range(4 * len(groups))))
        T = 32
        while True:
            jobs = [(w.variant, [a[:, :T, g[0]:g[-1] + 1] for a in arrays]) for g in groups]
            t0 = time.perf_counter()
            parts = list(pool.map(_oracle_part, jobs))
            wall = time.perf_counter() - t0
            compute = max(p[0] for p in parts)
            pids = {p[1] for p in parts}
            if compute >= budget_s / 2 or T >= x["q"].shape[1]:
                break
            T *= 2
    return {
        "value": w.B * T / compute,
        "unit": "tokens/s",
        "cores": len(groups),
        "host_cores_available": len(os.sched_getaffinity(0)), "worker_processes": len(pids),
        "blas_threads": 1,
        "kind": "oracle",
        "sample": f"float64 per-level recurrent form (Sec. 3.2 states, Eq. 3 output, "
                  f"{'gated delta rule' if w.variant == 'gdn' else 'scalar decay'}), first {T} tokens of "
                  f"all {w.H} heads (B={w.B}, {L} level states), heads dealt to {len(groups)} worker "
                  f"processes with one BLAS thread each; slowest worker {compute:.2f} s, "
                  f"{wall:.2f} s wall with the transfers",
    }


CLOCK_SETTLE_S = 0.1
CLOCK_SETTLE_NOTE = ("before its W warm-up steps each workload runs its own step untimed for 0.1 s of wall time: "
                     "after an idle spell (input generation on the host) the GPU starts at low clocks and "
                     "needs ~10-30 ms of load to reach its steady clocks; the K timed steps are unchanged")


def settle_clocks(fn, torch, seconds=CLOCK_SETTLE_S):
    """Runs fn() (one step of the workload) untimed for `seconds` of wall time, synchronising every
    10 calls, so that the timed steps see the GPU's steady clocks rather than its idle ones."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            fn()
        torch.cuda.synchronize()


def measure_mamba2(w, K, W, torch, ll, with_gemm=False, copy_mib=0):
    """Times the log-linear Mamba-2 forward on workload `w` (K timed steps after W warm-up steps,
    HIP events between the kernel stages of every step), the same call with lambda = 1 and the
    lambda == NULL Mamba-2 path; returns the bench line's fields."""
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = generate(w)
    if w.qk_heads:
        x["q"], x["k"] = shared_qk(x, w)
    d = {n: torch.from_numpy(x[n]).to(dev).to(dt).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev)
    lam = torch.from_numpy(x["lam"]).to(dev)
    ones = torch.ones_like(lam)
    del x
    out = torch.empty((w.B, w.T, w.H, w.dv), dtype=dt, device=dev)
    code = ll.LL_BF16 if w.dtype == "bf16" else ll.LL_F32
    ws_bytes = max(ll.ll_workspace_size(ll.LL_MAMBA2, code, w.B, w.T, w.H, w.dk, w.dv, w.C, has_l)
                   for has_l in (0, 1))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    fwd = ll.ll_mamba2_fwd_grouped if w.qk_heads else ll.ll_mamba2_fwd

    def run(lmb):
        fwd(d["q"], d["k"], d["v"], la, lmb, w.C, out=out, workspace=ws, stream=stream)

    def timed_plain(lmb):
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

    def timed_staged():
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

    print(f"[bench] {w.name}: warmup {W}, steps {K}", file=sys.stderr, flush=True)
    settle_clocks(lambda: run(lam), torch)
    ms = timed_plain(lam)
    # the per-kernel durations come from a second pass with events between the kernel stages
    _, stage_ms = timed_staged()
    ms_ones = timed_plain(ones)
    ms_null = timed_plain(None)
    print(f"[bench] {w.name} log-linear {ms:.3f} ms/step (stages {', '.join(f'{x:.3f}' for x in stage_ms)}), "
          f"lambda=1 {ms_ones:.3f}, lambda=NULL {ms_null:.3f} ms/step", file=sys.stderr, flush=True)

    fused = fused_path(w)
    names = FUSED_STAGES if fused else STAGES
    figs = fused_stage_figures(w) if fused else stage_figures(w)
    dom = int(np.argmax(stage_ms))
    roof = roofline(w, *figs[names[dom]], stage_ms[dom])
    traffic = recorded_traffic(w.name, fused_traffic_file(w.name)) if names[dom] == "fused_tile" else None
    F = flops_loglinear(w)
    tflops = F / (ms * 1e-3) / 1e12
    F2 = flops_mamba2(w)
    res = {
        "value": w.B * w.T / (ms * 1e-3),
        "unit": "tokens/s",
        "ms_per_step": ms,
        "dtype": w.dtype,
        "config": {"workload": w.name, "variant": "log-linear Mamba-2", "B": w.B, "H": w.H, "T": w.T,
                   "d_k": w.dk, "d_v": w.dv, "C": w.C, "levels": w.levels,
                   **({"qk_heads": w.qk_heads} if w.qk_heads else {}),
                   "path": "single-pass" if fused else "three-kernel",
                   "inputs": f"{w.dtype} q/k/v, fp32 log-gates and lambda, seeded synthetic (numpy PCG64)"},
        "tflops": tflops,
        "mfma_peak_frac": tflops / (PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS),
        "flop_convention": "B*H*T*[2C(dk+dv) + 2dk*dv + dk*dv*log2(T/C)]",
        "hbm_GBps_algorithmic": algorithmic_bytes(w) / (ms * 1e-3) / 1e9,
        "mamba2_lambda_ones": {"ms_per_step": ms_ones, "tokens_per_s": w.B * w.T / (ms_ones * 1e-3),
                               "note": "the same kernels with every level weight 1 (the output is Mamba-2's)"},
        "mamba2_lambda_null": {"ms_per_step": ms_null, "tokens_per_s": w.B * w.T / (ms_null * 1e-3),
                               "tflops": F2 / (ms_null * 1e-3) / 1e12,
                               "note": ("lambda == NULL: Mamba-2 itself (every level weight 1; the single-pass "
                                        "kernels for bf16 at C = 64, else one running state per tile)")},
        "log_factor_overhead": ms / ms_null,
        "log_factor_overhead_note": "log-linear ms / lambda == NULL Mamba-2 ms",
        "lambda_ones_ratio": ms / ms_ones,
        "clock_settle_s": CLOCK_SETTLE_S, "clock_settle_note": CLOCK_SETTLE_NOTE,
        "stages_ms": dict(zip(names, [float(v) for v in stage_ms])),
        "roofline": {"kernel": names[dom], **roof, "traffic": traffic,
                     "traffic_note": "HBM bytes per launch from rocprofv3 FETCH_SIZE x 2 + WRITE_SIZE x 1 "
                                     "(factors from a 1 GiB copy), null if the kernel changed since"},
    }
    del d, la, lam, ones, out, ws
    torch.cuda.empty_cache()
    if with_gemm:
        # a measured second denominator: a large bf16 matrix product through the vendor BLAS
        res["measured_bf16_gemm_tflops"] = measured_gemm_tflops(torch, dev)
        res["mfma_frac_of_measured_gemm"] = tflops / res["measured_bf16_gemm_tflops"]
    if copy_mib:
        # A plain copy kernel of known size: its FETCH_SIZE / WRITE_SIZE counters calibrate the
        # HBM traffic that the same counters report for the kernels above.
        src = torch.empty(copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    return res


# The other workloads of the scope table, measured in the default run beside the headline.
EXTRA_WORKLOADS = {"ll_mamba2_bf16_T2048": "mamba2", "ll_mamba2_bf16_T8192": "mamba2", "ll_gdn_bf16_T8192": "gdn"}
HEADLINE = "ll_mamba2_bf16_T65536"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None, help=f"one workload only (default: {HEADLINE} plus the others)")
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

    w = WORKLOADS[args.workload or HEADLINE]
    if w.variant == "gdn":
        res = main_gdn(args, w, torch, ll)
        print(json.dumps(res), flush=True)
        return
    if w.variant in ("decode", "gdn_decode"):
        return main_decode(args, w, torch, ll)
    if w.variant == "mamba2_bwd":
        return main_bwd(args, w, torch, ll)
    if w.variant == "mamba2_diag_lambda":
        return main_mlambda(args, w, torch, ll)
    m = measure_mamba2(w, args.steps, args.warmup, torch, ll, with_gemm=True, copy_mib=args.copy_mib)
    res = {"metric": METRIC, "value": m.pop("value"), "unit": m.pop("unit"), "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": m.pop("ms_per_step"), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": m.pop("dtype"), "data": "synthetic",
           "config": m.pop("config"), **m}
    if args.workload is None:
        extra = {}
        for name, kind in EXTRA_WORKLOADS.items():
            we = WORKLOADS[name]
            if kind == "gdn":
                sub = main_gdn(args, we, torch, ll, cpu=False)
            else:
                sub = measure_mamba2(we, args.steps, args.warmup, torch, ll)
            extra[name] = sub
        res["other_workloads"] = extra
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------------------- backward pass

BWD_STAGES = ["fwd_summaries", "rev_summaries", "dq", "dkv"]


def flops_bwd(w):
    """Algorithmic FLOPs of the log-linear Mamba-2 gradient, chunk convention as the forward:
    per chunk the dense C x C products S = Q K^T, G = dO V^T, dq = (W G) K, dk = (W G)^T Q,
    dv = (W S)^T dO; the chunk states of the forward summaries; per (chunk, set bit) the query
    side's two products (dq, and U q for dlambda) and the key-side summary of that level; per
    (chunk, clear bit) the key side's two products (dk, dv)."""
    J = math.log2(w.T // w.C) if w.T > w.C else 0.0
    return w.B * w.H * w.T * (2 * w.C * (3 * w.dk + 2 * w.dv) + 2 * w.dk * w.dv + 5 * w.dk * w.dv * J)


def bwd_stage_figures(w):
    """Work of one launch of each backward stage: {stage: (flops, bytes)}.  dq and dkv each
    recompute S and G for their tile (counted in both).  Bytes: what each stage must read and
    write once (inputs, dO, the summaries it produces, the gradients it writes)."""
    es = 2 if w.dtype == "bf16" else 4
    BH, BHT = w.B * w.H, w.B * w.H * w.T
    SZ = w.dk * w.dv
    J = math.log2(w.T // w.C) if w.T > w.C else 0.0
    L = w.levels
    R = max(2 * w.C, 64)
    N = -(-w.T // R)
    Jt = (N - 1).bit_length() if N > 1 else 0
    n_rev = sum(((N - 1) >> (j - 1)) // 2 + 1 if ((N - 1) >> (j - 1)) >= 1 else 0 for j in range(1, Jt + 1))
    fwd = stage_figures(w)
    f_sum = fwd["block_state"][0]
    b_sum = fwd["block_state"][1] + fwd["scan"][1]
    f_rev = BHT * w.dk * w.dv * J
    b_rev = BHT * ((w.dk + w.dv) * es + 4 * Jt) + BH * n_rev * SZ * es
    f_dq = BHT * (2 * w.C * (2 * w.dk + w.dv) + 2 * w.dk * w.dv * J)
    f_dkv = BHT * (2 * w.C * (2 * w.dk + 2 * w.dv) + 2 * w.dk * w.dv * J)
    b_in = BHT * ((2 * w.dk + 2 * w.dv) * es + 4 + 4 * L)
    b_dq = b_in + BHT * (w.dk * es + 4 * L + 4)
    b_dkv = b_in + BHT * ((w.dk + w.dv) * es + 4 + 4)
    return {"fwd_summaries": (f_sum, b_sum), "rev_summaries": (f_rev, b_rev), "dq": (f_dq, b_dq),
            "dkv": (f_dkv, b_dkv)}


def cpu_baseline_bwd(w, budget_s):
    """The float64 oracle's gradients (quadratic form) on a prefix of the workload, all heads,
    growing the prefix until one run takes at least `budget_s` / 2; tokens/s of that prefix."""
    from oracle import mamba2_grad
    from synthetic import upstream_grad
    x = generate(w)
    if w.qk_heads:  # the shared q, k repeated to every head of its group: the same computation
        G = w.H // w.qk_heads
        q, k = shared_qk(x, w)
        x["q"], x["k"] = np.repeat(q, G, axis=2), np.repeat(k, G, axis=2)
    do = upstream_grad(w)
    T = 64
    while True:
        L = 1 if T == 1 else (T - 1).bit_length() + 1
        args = [np.ascontiguousarray(x[n][:, :T]) for n in ("q", "k", "v", "log_alpha")]
        args += [np.ascontiguousarray(x["lam"][:, :T, :, :L]), np.ascontiguousarray(do[:, :T])]
        t0, c0 = time.perf_counter(), time.process_time()
        mamba2_grad.quadratic_grad(*args)
        wall, cpu = time.perf_counter() - t0, time.process_time() - c0
        # stop at half the budget, or before a doubling (about 4x the work) would overshoot it
        if wall >= budget_s / 2 or 4 * wall > 1.5 * budget_s or 2 * T > w.T:
            break
        T *= 2
    return {
        "value": w.B * T / wall, "unit": "tokens/s", "cores": max(1, round(cpu / wall)),
        "host_cores_available": len(os.sched_getaffinity(0)), "blas_threads": blas_threads(), "kind": "oracle",
        "sample": f"float64 gradients of the quadratic form (chain rule, every input), first {T} tokens "
                  f"of all {w.H} heads, B={w.B}; {wall:.2f} s wall, {cpu:.2f} s CPU (the quadratic form's "
                  f"cost grows with T, so longer prefixes run slower per token)",
    }


def main_bwd(args, w, torch, ll):
    """Log-linear Mamba-2 backward: one step = one ll_mamba2_bwd call (forward summaries,
    key-side summaries, dq and dlambda, dk dv and dlog_alpha), inputs and dO resident."""
    from synthetic import upstream_grad
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = generate(w)
    if w.qk_heads:
        x["q"], x["k"] = shared_qk(x, w)
    d = {n: torch.from_numpy(x[n]).to(dev).to(dt).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev)
    lam = torch.from_numpy(x["lam"]).to(dev)
    del x
    do = torch.from_numpy(upstream_grad(w)).to(dev).to(dt).contiguous()
    ws = ll.ll_mamba2_bwd_workspace(d["q"], d["v"], w.C)
    out = torch.empty((w.B, w.T, w.H, w.dv), dtype=dt, device=dev)
    grads = (torch.empty_like(d["q"]), torch.empty_like(d["k"]), torch.empty_like(d["v"]),
             torch.empty_like(la), torch.empty_like(lam))
    stream = torch.cuda.current_stream()
    K, W = args.steps, args.warmup
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K)]

    def bwd(e=None):
        if e is None:
            ll.ll_mamba2_bwd(d["q"], d["k"], d["v"], la, lam, do, w.C, grads=grads, workspace=ws, stream=stream)
        else:
            ll.ll_mamba2_bwd_staged(d["q"], d["k"], d["v"], la, lam, do, w.C, e, grads=grads, workspace=ws,
                                    stream=stream)

    fwd_call = ll.ll_mamba2_fwd_grouped if w.qk_heads else ll.ll_mamba2_fwd

    def fwd():
        # in the backward's workspace: the backward after it reuses the level summaries
        fwd_call(d["q"], d["k"], d["v"], la, lam, w.C, out=out, workspace=ws, stream=stream)

    def bwd_after_fwd():
        ll.ll_mamba2_bwd_after_fwd(d["q"], d["k"], d["v"], la, lam, do, w.C, ws, grads=grads, stream=stream)

    print(f"[bench] {w.name}: warmup {W}, steps {K}", file=sys.stderr, flush=True)
    for i in range(W):
        bwd(evs[i % K])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(K):
        bwd(evs[i])
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    stage_ms = np.array([[e[s].elapsed_time(e[s + 1]) for s in range(4)] for e in evs]).mean(axis=0)
    # forward + backward, as one training step of the operator would run them (the forward in the
    # backward-sized workspace leaves the level summaries that the backward reuses)
    for _ in range(W):
        fwd()
        bwd_after_fwd()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(K):
        fwd()
        bwd_after_fwd()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_fb = e0.elapsed_time(e1) / K
    print(f"[bench] backward {ms:.3f} ms/step (stages {', '.join(f'{x:.3f}' for x in stage_ms)}), "
          f"forward + backward {ms_fb:.3f} ms", file=sys.stderr, flush=True)

    figs = bwd_stage_figures(w)
    dom = int(np.argmax(stage_ms))
    roof = roofline(w, *figs[BWD_STAGES[dom]], stage_ms[dom])
    F = flops_bwd(w)
    Ff = flops_loglinear(w)
    tflops = F / (ms * 1e-3) / 1e12
    es = 2 if w.dtype == "bf16" else 4
    # read q, k, v, dO, log alpha, lambda; write dq, dk, dv, dlog_alpha, dlambda (q, k, dq, dk at the
    # query/key heads)
    nbytes = w.B * w.T * w.H * ((4 * w.dk * qk_share(w) + 3 * w.dv) * es + 8 + 8 * w.levels)
    res = {
        "metric": "bwd tokens/sec + TFLOP/s (% bf16 MFMA peak), log-linear Mamba-2, T=64K",
        "value": w.B * w.T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "variant": "log-linear Mamba-2 backward", "B": w.B, "H": w.H, "T": w.T,
                   "d_k": w.dk, "d_v": w.dv, "C": w.C, "levels": w.levels,
                   **({"qk_heads": w.qk_heads} if w.qk_heads else {}),
                   "inputs": "bf16 q/k/v/dO, fp32 log-gates and lambda, seeded synthetic (numpy PCG64)"},
        "tflops": tflops,
        "mfma_peak_frac": tflops / (PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS),
        "flop_convention": "B*H*T*[2C(3dk+2dv) + 2dk*dv + 5dk*dv*log2(T/C)]",
        "hbm_GBps_algorithmic": nbytes / (ms * 1e-3) / 1e9,
        "forward_plus_backward": {"ms": ms_fb, "tokens_per_s": w.B * w.T / (ms_fb * 1e-3),
                                  "backward_entry": "ll_mamba2_bwd_after_fwd (level summaries from the forward)",
                                  "tflops": (F + Ff) / (ms_fb * 1e-3) / 1e12},
        "stages_ms": dict(zip(BWD_STAGES, [float(x) for x in stage_ms])),
        "roofline": {"kernel": BWD_STAGES[dom], **roof, "traffic": None,
                     "traffic_note": "counter traffic of the backward kernels in the rocprofv3 summaries"},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline_bwd(w, args.cpu_budget)
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------------------- Gated DeltaNet

def gdn_issued(w, has_lambda=True):
    """MFMA FLOPs the GDN kernels issue, counted from their loop structure, and the algorithmic
    bytes of the whole call.
    gdn_chunk, per chunk: K K^T, Q K^T (C x C x d_k), W = T_G (gamma K), Q~ correction (C x d_k x C),
    U = T_G V, intra output (C x d_v x C), P_G T_G (C x C x C), P_z (d_k x d_k x C), H_z (d_k x d_v x C).
    Block tree, per block of levels 1 .. J-1: T_hi T_lo (d_k x d_k x d_k) and T_hi A_lo
    (d_k x d_v x d_k).  Read-out, per chunk and set bit of its index: q~ A (C x d_v x d_k) and, when
    a higher set bit follows, q~ T (C x d_k x d_k).  lambda == NULL issues the same work."""
    C, dk, dv = w.C, w.dk, w.dv
    N = w.T // C
    J = (N - 1).bit_length() if N > 1 else 0
    f_chunk = 2.0 * (3 * C * C * dk + C * C * dk + 2 * C * C * dv + C ** 3 + dk * dk * C + dk * dv * C)
    f_tree = sum((N >> m) * 2.0 * dk * dk * (dk + dv) for m in range(1, J))
    f_read = 0.0
    for z in range(N):
        nb = bin(z).count("1")
        f_read += nb * 2.0 * C * dk * dv + max(nb - 1, 0) * 2.0 * C * dk * dk
    BH = w.B * w.H
    es = 2 if w.dtype == "bf16" else 4
    L = w.levels if has_lambda else 0
    nbytes = w.B * w.T * w.H * ((2 * dk + 2 * dv) * es + 8 + 4 * L)
    return BH * N * f_chunk, BH * (f_tree + f_read), nbytes


def decode_level_reads(T):
    """Per token t < T: the number of level states (d_v x d_k, fp32) a decode step reads -- the
    nonempty levels >= 1 other than the one it overwrites -- following the Sec. 3.2 occupancy
    (level p+1 filled and levels 1..p emptied at t, p = lssb(t))."""
    occupied, reads = set(), []
    for t in range(T):
        if t == 0:
            reads.append(0)
            continue
        p = (t & -t).bit_length() - 1
        reads.append(len([lv for lv in occupied if lv != p + 1]))
        occupied -= set(range(1, p + 1))
        occupied.add(p + 1)
    return reads


def gdn_decode_level_traffic(T):
    """Per token t < T of Gated DeltaNet decoding: (level states read, level states written).
    Every nonempty level >= 1 after the step (bit l-1 of t set) is rewritten; the merged level
    p+1 (p = lssb(t)) reads the previous levels 1..p, the others read themselves."""
    out = []
    for t in range(T):
        if t == 0:
            out.append((0, 0))
            continue
        p = (t & -t).bit_length() - 1
        n = bin(t).count("1")
        out.append((n - 1 + p, n))
    return out


def main_decode(args, w, torch, ll):
    """Log-linear Mamba-2 or Gated DeltaNet decoding: B sequences, one token each per step, timed
    over the last steps before position T (the state then holds up to log2 T levels)."""
    gdn = w.variant == "gdn_decode"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T0 = 1024  # distinct token inputs, cycled
    L = w.levels
    x = generate(w.with_(T=T0))
    dt = torch.bfloat16
    per_t = {n: torch.from_numpy(x[n]).to(dev).to(dt).transpose(0, 1).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev).transpose(0, 1).contiguous()
    beta = torch.from_numpy(x["beta"]).to(dev).transpose(0, 1).contiguous() if gdn else None
    lam = torch.zeros((T0, w.B, w.H, L), dtype=torch.float32, device=dev)
    lam[..., :x["lam"].shape[-1]] = torch.from_numpy(x["lam"]).to(dev).transpose(0, 1)
    del x
    state = torch.empty(ll.ll_decode_state_bytes(w.B, w.H, w.dk, w.dv, L), dtype=torch.uint8, device=dev)
    out = torch.empty((w.B, w.H, w.dv), dtype=dt, device=dev)
    stream = torch.cuda.current_stream()
    M = min(args.steps * 50, w.T // 2)  # timed tokens: the last M positions before T

    def step(t, lmb=True):
        i = t % T0
        if gdn:
            ll.ll_gdn_decode_step(per_t["q"][i], per_t["k"][i], per_t["v"][i], la[i], beta[i],
                                  lam[i] if lmb else None, state, t, L, out=out, stream=stream)
        else:
            ll.ll_mamba2_decode_step(per_t["q"][i], per_t["k"][i], per_t["v"][i], la[i], lam[i] if lmb else None,
                                     state, t, L, out=out, stream=stream)

    def run(lmb):
        (ll.ll_gdn_decode_init if gdn else ll.ll_mamba2_decode_init)(state, w.B, w.H, w.dk, w.dv, L, dt,
                                                                     stream=stream)
        for t in range(w.T - M):
            step(t, lmb)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for t in range(w.T - M, w.T):
            step(t, lmb)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / M

    print(f"[bench] {w.name}: {w.T - M} untimed tokens, {M} timed", file=sys.stderr, flush=True)
    ms = run(True)
    ms_null = run(False)
    print(f"[bench] decode {ms * 1e3:.1f} us/token-step (lambda), {ms_null * 1e3:.1f} (lambda=NULL)",
          file=sys.stderr, flush=True)
    BH = w.B * w.H
    SZ4 = w.dk * w.dv * 4
    token_bytes = BH * ((2 * w.dk + 2 * w.dv) * 2 + 4 + 4 * L + 2 * (w.dv + w.dk) * 4 + (4 if gdn else 0))
    if gdn:
        rw = np.array(gdn_decode_level_traffic(w.T)[w.T - M:], dtype=np.float64)
        per_step = BH * (rw[:, 0].mean() + rw[:, 1].mean()) * SZ4 + token_bytes
        note = ("per head: the level states read (the carried levels and the merged level's inputs) and every "
                "nonempty level rewritten by the delta-rule transition, fp32, means over the timed positions, plus "
                "the token's inputs and output; states partly served by the 256 MB Infinity Cache")
    else:
        reads = decode_level_reads(w.T)[w.T - M:]
        per_step = BH * (np.mean(reads) + 1) * SZ4 + token_bytes
        note = ("per head: the nonempty level states read (mean over the timed positions) and the merged one "
                "written, fp32, plus the token's inputs and output; the states re-read every token are partly "
                "served by the 256 MB Infinity Cache, so the rate can exceed the HBM peak")
    gbs = per_step / (ms * 1e-3) / 1e9
    name = "Gated DeltaNet" if gdn else "Mamba-2"
    res = {
        "metric": f"decode tokens/sec (one token per sequence per step), log-linear {name}",
        "value": w.B / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": M, "warmup": w.T - M, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "variant": f"log-linear {name} decoding", "B": w.B, "H": w.H,
                   "positions": f"{w.T - M}..{w.T - 1}", "d_k": w.dk, "d_v": w.dv, "levels": L,
                   "inputs": f"bf16 q/k/v, fp32 log-gates{', beta' if gdn else ''} and lambda, the seeded "
                             f"T={T0} draw cycled"},
        ("gated_deltanet_lambda_null" if gdn else "mamba2_lambda_null"):
            {"ms_per_step": ms_null, "tokens_per_s": w.B / (ms_null * 1e-3)},
        "roofline": {"kernel": "gdn_decode_step" if gdn else "decode_step", "bound": "hbm", "achieved": gbs,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "traffic": None,
                     "algorithmic_bytes_per_step": per_step, "bytes_note": note},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w.with_(variant="gdn" if gdn else "mamba2", B=1), args.cpu_budget)
        res["cpu_baseline"]["sample"] += " (the oracle's recurrent form is itself token-by-token decoding)"
    print(json.dumps(res), flush=True)


def main_gdn(args, w, torch, ll, cpu=True):
    """Log-linear Gated DeltaNet forward: same line format, issued-FLOP convention; returns the
    line's fields (with the CPU baseline when `cpu`)."""
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    x = generate(w)
    d = {n: torch.from_numpy(x[n]).to(dev).to(torch.bfloat16).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev)
    beta = torch.from_numpy(x["beta"]).to(dev)
    lam = torch.from_numpy(x["lam"]).to(dev)
    del x
    out = torch.empty((w.B, w.T, w.H, w.dv), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(ll.ll_workspace_size(ll.LL_GDN, ll.LL_BF16, w.B, w.T, w.H, w.dk, w.dv, w.C, 1),
                     dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    K, W = args.steps, args.warmup
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]

    def step(lmb, e=None):
        if e is None:
            ll.ll_gdn_fwd(d["q"], d["k"], d["v"], la, beta, lmb, w.C, out=out, workspace=ws, stream=stream)
        else:
            ll.ll_gdn_fwd_staged(d["q"], d["k"], d["v"], la, beta, lmb, w.C, e, out=out, workspace=ws,
                                 stream=stream)

    print(f"[bench] {w.name}: warmup {W}, steps {K}", file=sys.stderr, flush=True)
    settle_clocks(lambda: step(lam), torch)
    for i in range(W):
        step(lam)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(K):
        step(lam)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    # the per-kernel durations come from a second pass with events between the kernel stages
    for i in range(K):
        step(lam, evs[i])
    torch.cuda.synchronize()
    stage_ms = np.array([[e[s].elapsed_time(e[s + 1]) for s in range(2)] for e in evs]).mean(axis=0)
    for _ in range(W):
        step(None)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(K):
        step(None)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_null = e0.elapsed_time(e1) / K
    print(f"[bench] log-linear GDN {ms:.3f} ms/step (stages {stage_ms[0]:.3f}, {stage_ms[1]:.3f}), "
          f"lambda=NULL {ms_null:.3f} ms/step", file=sys.stderr, flush=True)

    f_chunk, f_scan, nbytes = gdn_issued(w)
    names = ["gdn_chunk", "gdn_tree_read"]
    dom = int(np.argmax(stage_ms))
    # per-stage algorithmic bytes: the chunk kernel reads q, k, v, gates, beta and writes the
    # per-chunk products (Q~, P_z, H_z bf16, intra output fp32); the block tree and the read-out
    # read those and lambda and write o (the tree's own blocks are not counted).
    N = w.T // w.C
    BHN = w.B * w.H * N
    prod = BHN * (w.C * w.dk * 2 + w.dk * w.dk * 2 + w.dk * w.dv * 2 + w.C * w.dv * 4)
    BTH = w.B * w.T * w.H
    b_chunk = BTH * ((2 * w.dk + w.dv) * 2 + 8) + prod
    b_scan = prod + BTH * (4 * w.levels + w.dv * 2)
    figs = {"gdn_chunk": (f_chunk, b_chunk), "gdn_tree_read": (f_scan, b_scan)}
    roof = roofline(w, *figs[names[dom]], stage_ms[dom])
    F = f_chunk + f_scan
    f_n, s_n, _ = gdn_issued(w, has_lambda=False)
    res = {
        "metric": "fwd tokens/sec + TFLOP/s (issued, % bf16 MFMA peak), log-linear Gated DeltaNet",
        "value": w.B * w.T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "variant": "log-linear Gated DeltaNet", "B": w.B, "H": w.H, "T": w.T,
                   "d_k": w.dk, "d_v": w.dv, "C": w.C, "levels": w.levels,
                   "inputs": "bf16 q/k/v (k L2-normalised), fp32 log-gates, beta and lambda, seeded synthetic"},
        "tflops_issued": F / (ms * 1e-3) / 1e12,
        "mfma_peak_frac": F / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "flop_convention": "MFMA FLOPs issued by gdn_chunk, the block tree and the read-out (see gdn_issued)",
        "hbm_GBps_algorithmic": nbytes / (ms * 1e-3) / 1e9,
        "gdn_lambda_null": {"ms_per_step": ms_null, "tokens_per_s": w.B * w.T / (ms_null * 1e-3),
                            "tflops_issued": (f_n + s_n) / (ms_null * 1e-3) / 1e12},
        "log_factor_overhead": ms / ms_null,
        "clock_settle_s": CLOCK_SETTLE_S, "clock_settle_note": CLOCK_SETTLE_NOTE,
        "stages_ms": dict(zip(names, [float(v) for v in stage_ms])),
        "roofline": {"kernel": names[dom], **roof,
                     "traffic": recorded_traffic(w.name, GDN_TRAFFIC_FILE, GDN_KERNEL_SOURCES)
                     if names[dom] == "gdn_tree_read" else None},
    }
    del d, la, beta, lam, out, ws
    torch.cuda.empty_cache()
    if cpu and not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    return res


def lq_level_rows(T, R):
    """Level-query rows the tile kernel needs with matrix-valued weights, summed over a sequence:
    row t (tile u = t // R, tile-local index i) scores its pairs at level 0, at level b + 1 for
    every set bit b of i, and at one inter-tile level per set bit of u."""
    t = np.arange(T)
    pc = lambda x: np.array([bin(int(y)).count("1") for y in x])
    return int(np.sum(1 + pc(t % R) + pc(t // R)))


def main_mlambda(args, w, torch, ll):
    """Log-linear Mamba-2 with diagonal matrix-valued level weights (ll_mamba2_fwd_matrix_lambda).
    One step = the level queries, the tile states, the scan and the tile outputs."""
    from synthetic import level_weight_matrices
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    x = generate(w)
    d = {n: torch.from_numpy(x[n]).to(dev).to(dt).contiguous() for n in ("q", "k", "v")}
    la = torch.from_numpy(x["log_alpha"]).to(dev)
    Lam = torch.from_numpy(level_weight_matrices(w, "diag")).to(dev)
    out = torch.empty((w.B, w.T, w.H, w.dv), dtype=dt, device=dev)
    ws = ll.ll_mamba2_matrix_lambda_workspace(d["q"], d["v"], w.C)
    stream = torch.cuda.current_stream()
    names = ["level_queries", "block_state", "scan", "tile_out"]
    K, W = args.steps, args.warmup
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(max(K, 1))]
    print(f"[bench] {w.name}: warmup {W}, steps {K}", file=sys.stderr, flush=True)
    for i in range(W):
        ll.ll_mamba2_fwd_matrix_lambda_staged(d["q"], d["k"], d["v"], la, Lam, w.C, evs[i % K], out=out,
                                              workspace=ws, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(K):
        ll.ll_mamba2_fwd_matrix_lambda_staged(d["q"], d["k"], d["v"], la, Lam, w.C, evs[i], out=out,
                                              workspace=ws, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    stage_ms = np.array([[e[s].elapsed_time(e[s + 1]) for s in range(4)] for e in evs[:K]]).mean(axis=0)
    print(f"[bench] {ms:.3f} ms/step (stages {', '.join(f'{x:.3f}' for x in stage_ms)})", file=sys.stderr,
          flush=True)

    BHT, L = w.B * w.H * w.T, w.levels
    R = max(2 * w.C, 64)
    base = stage_figures(w)
    lq_rows = w.B * w.H * lq_level_rows(w.T, R)
    figs = {
        # no kernel for diagonal weights
        "level_queries": (0.0, 0.0),
        "block_state": base["block_state"],
        "scan": base["scan"],
        # q, k, v and the log-gates read, the diagonals of the levels each row scores with read,
        # o written; forming the level queries costs L d_k multiplies per row
        "tile_out": (base["tile_out"][0] + BHT * L * w.dk,
                     lq_rows * w.dk * 4 + BHT * ((2 * w.dk + 2 * w.dv) * es + 4)),
    }
    dom = int(np.argmax(stage_ms))
    roof = roofline(w, *figs[names[dom]], stage_ms[dom])
    F = flops_loglinear(w) + BHT * L * w.dk
    tflops = F / (ms * 1e-3) / 1e12
    alg_bytes = BHT * ((2 * w.dk + w.dv) * es + 4 + L * w.dk * 4 + w.dv * es)
    res = {
        "metric": "fwd tokens/sec, log-linear Mamba-2 with diagonal matrix-valued level weights",
        "value": w.B * w.T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "variant": "log-linear Mamba-2, Lambda_t^(l) = diag(lambda_t^(l)) in R^d_k",
                   "B": w.B, "H": w.H, "T": w.T, "d_k": w.dk, "d_v": w.dv, "C": w.C, "levels": L,
                   "inputs": "bf16 q/k/v, fp32 log-gates and diagonal weights [B, T, H, L, d_k], seeded synthetic"},
        "tflops": tflops,
        "mfma_peak_frac": tflops / (PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS),
        "flop_convention": "B*H*T*[2C(dk+dv) + 2dk*dv + dk*dv*log2(T/C)] + B*H*T*L*dk (level queries)",
        "hbm_GBps_algorithmic": alg_bytes / (ms * 1e-3) / 1e9,
        "stages_ms": dict(zip(names, [float(x) for x in stage_ms])),
        "roofline": {"kernel": names[dom], **roof, "traffic": None,
                     "traffic_note": "no counter record for this workload"},
    }
    if not args.no_cpu_baseline:
        from oracle import matrix_lambda
        print("[bench] timing the float64 oracle on the host", file=sys.stderr, flush=True)
        xs = generate(w.with_(T=min(w.T, 4096)))
        lam_h = level_weight_matrices(w.with_(T=min(w.T, 4096)), "diag")
        T = 32
        while True:
            sl = slice(0, T)
            t0, c0 = time.perf_counter(), time.process_time()
            matrix_lambda.recurrent(xs["q"][:, sl], xs["k"][:, sl], xs["v"][:, sl], xs["log_alpha"][:, sl],
                                    lam_h[:, sl])
            wall, cpu = time.perf_counter() - t0, time.process_time() - c0
            if wall >= args.cpu_budget / 2 or T >= xs["q"].shape[1]:
                break
            T *= 2
        res["cpu_baseline"] = {
            "value": w.B * T / wall, "unit": "tokens/s", "cores": max(1, round(cpu / wall)),
            "host_cores_available": len(os.sched_getaffinity(0)), "blas_threads": blas_threads(), "kind": "oracle",
            "sample": f"float64 per-level recurrent form with diagonal level weights, first {T} tokens of "
                      f"all {w.H} heads, B={w.B}; {wall:.2f} s wall, {cpu:.2f} s CPU"}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

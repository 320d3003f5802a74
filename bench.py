#!/usr/bin/env python3
"""Benchmark of the PRQuant MXFP4 + tail-residual hot path on one MI355X.

Default workload: the Qwen3-4B-shaped down_proj at decode (K = 9728 -> N =
2560, k = 256, rows M = 1, 8, 32, 64).  One step = for every M, the fused
activation quantization (prq_quant_act) followed by the augmented MXFP4 GEMM
over K + k (prq_gemm) on one stream, with inputs resident in HBM; the offline
prq_prepare runs once before timing.  Weights are rotated through enough
copies (>= 1 GiB) that every step streams them from HBM rather than from the
256 MB Infinity Cache.

Prints ONE JSON line on stdout (everything else goes to stderr):
  value = algorithmic bytes of one step / step time (GB/s), plus per-M
  kernel times, TFLOP/s, roofline fraction of the dominant kernel (the GEMM)
  from HIP events recorded around each of its launches on its stream, a
  same-shape BF16 torch.matmul for context, and the CPU oracle timed on a
  bounded sample (``cpu_baseline``).

Other workloads (--workload): prefill (M = 512, 2048, 8192), experts (128
expert down_projs 768 -> 2048, k = 64, 64 or 4096 tokens routed top-8, one
grouped launch), layers (the seven linears of a Qwen3-4B-shaped decoder layer
at M = 4096).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

METRIC = "MXFP4+residual GEMM µs/op, TFLOPS & HBM GB/s (% roofline), down_proj shapes"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MXFP4_PEAK_TFLOPS = 10100.0    # MI355X dense FP4 MFMA
ROOT = os.path.dirname(os.path.abspath(__file__))


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="decode",
                   choices=["decode", "prefill", "experts", "experts_prefill", "layers"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-bf16", action="store_true")
    p.add_argument("--rotate-bytes", type=float, default=1.0 * 2 ** 30,
                   help="minimum total bytes of rotated weight copies")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain device copy of known size (for counter scaling)")
    p.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="no run: turn two rocprofv3 --pmc output directories (FETCH_SIZE, "
                        "WRITE_SIZE) into profiles/traffic_<workload>.json")
    p.add_argument("--traffic-command", default="",
                   help="the profiled command, recorded with --traffic-from")
    return p.parse_args(argv)


# ----------------------------------------------------------- workloads ---
def act_bytes(M, K, K_aug):
    return 2 * M * K + M * K_aug * 17 / 32 + 8 * K


def gemm_bytes(M, N, K_aug):
    return (N + M) * K_aug * 17 / 32 + 4 * M * N


def grouped_gemm_bytes(M, E_active, N, K_aug):
    return (E_active * N + M) * K_aug * 17 / 32 + 4 * M * N


class Op:
    """One act-quant + GEMM pair of a step (launch closures bound to buffers)."""

    def __init__(self, name, M, N, K, k, act_fn, gemm_fn, gbytes, abytes, flops):
        self.name, self.M, self.N, self.K, self.k = name, M, N, K, k
        self.act_fn, self.gemm_fn = act_fn, gemm_fn
        self.gemm_bytes, self.act_bytes, self.flops = gbytes, abytes, flops
        self.t_gemm, self.t_act = [], []


def build_dense_ops(torch, prq, layers, M_list, rotate_bytes, stream):
    """layers: list of (name, DenseCase).  Weights rotated, activations per M."""
    ops = []
    for name, c in layers:
        K, k, N = c.K, c.k_tail, c.N
        K_aug = K + k
        t0 = time.perf_counter()
        art = prq.prq_prepare(c.W, c.Xcal, c.alpha, k)
        log(f"[bench] prq_prepare {name}: {time.perf_counter() - t0:.2f} s")
        w_bytes = art["Wq"].nbytes + art["Wsc"].nbytes
        R = max(1, math.ceil(rotate_bytes / w_bytes))
        Wc = prq.prq_pack_weight(torch.from_numpy(art["Wq"]).cuda(), torch.from_numpy(art["Wsc"]).cuda())
        Ws = [prq.PackedWeight(Wc.Wp.clone(), Wc.Wps.clone(), 1, N, K_aug) for _ in range(R)]
        inv = torch.from_numpy(art["inv_scale_pos"]).cuda()
        perm = torch.from_numpy(art["perm"]).cuda()
        X = torch.from_numpy(c.X.view("int16")).cuda()
        for M in M_list:
            Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
            Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")
            Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
            ws_n = prq.prq_gemm_workspace_bytes(M, N, K_aug)
            ws = torch.zeros(max(ws_n, 1), dtype=torch.uint8, device="cuda") if ws_n else None
            Xm = X[:M]
            state = {"r": 0}

            # every per-layer buffer is bound here: a name captured from the
            # enclosing loop would see the last layer's buffers in every op
            def act(Xm=Xm, Aq=Aq, Asc=Asc, K=K, k=k, inv=inv, perm=perm):
                prq.prq_quant_act(Xm, K, k, inv, perm, Aq=Aq, Asc=Asc, stream=stream)

            def gemm(Aq=Aq, Asc=Asc, Y=Y, ws=ws, state=state, R=R, Ws=Ws):
                r = state["r"]
                state["r"] = (r + 1) % R
                prq.prq_gemm(Aq, Asc, Ws[r], Y=Y, workspace=ws, stream=stream)

            ops.append(Op(f"{name}/M={M}", M, N, K, k, act, gemm, gemm_bytes(M, N, K_aug),
                          act_bytes(M, K, K_aug), 2.0 * M * N * K_aug))
        log(f"[bench] {name}: {R} rotated weight copies ({w_bytes / 1e6:.2f} MB each)")
    return ops


def build_expert_ops(torch, np, prq, inputs, tokens, rotate_bytes, stream):
    c = inputs.moe_experts(tokens)
    E, N, K, k = c.E, c.N, c.K, c.k_tail
    K_aug = K + k
    t0 = time.perf_counter()
    arts = [prq.prq_prepare(c.W[e], c.Xcal[e], c.alpha, k) for e in range(E)]
    log(f"[bench] prq_prepare x{E} experts: {time.perf_counter() - t0:.2f} s")
    Wq_h = np.stack([a["Wq"] for a in arts])
    Wsc_h = np.stack([a["Wsc"] for a in arts])
    w_bytes = Wq_h.nbytes + Wsc_h.nbytes
    R = max(1, math.ceil(rotate_bytes / w_bytes))
    Wc = prq.prq_pack_weight(torch.from_numpy(Wq_h).cuda(), torch.from_numpy(Wsc_h).cuda())
    Ws = [prq.PackedWeight(Wc.Wp.clone(), Wc.Wps.clone(), E, N, K_aug) for _ in range(R)]
    inv = torch.from_numpy(np.stack([a["inv_scale_pos"] for a in arts])).cuda()
    perm = torch.from_numpy(np.stack([a["perm"] for a in arts])).cuda()
    off = torch.from_numpy(c.group_offsets).cuda()
    M = int(c.group_offsets[-1])
    X = torch.from_numpy(c.X.view("int16")).cuda()
    Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
    Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    state = {"r": 0}
    e_active = int(np.count_nonzero(np.diff(c.group_offsets)))

    def act():
        prq.prq_quant_act(X, K, k, inv, perm, group_offsets=off, G=E, Aq=Aq, Asc=Asc, stream=stream)

    def gemm():
        r = state["r"]
        state["r"] = (r + 1) % R
        prq.prq_grouped_gemm(Aq, Asc, off, Ws[r], Y=Y, stream=stream)

    log(f"[bench] experts: {M} routed rows, {e_active} active experts, {R} weight copies")
    return [Op(f"experts/{tokens}tok", M, N, K, k, act, gemm,
               grouped_gemm_bytes(M, e_active, N, K_aug), act_bytes(M, K, K_aug) + 8 * K * (E - 1),
               2.0 * M * N * K_aug)]


# -------------------------------------------------------------- timing ---
def run_steps(torch, ops, steps, warmup, stream, record):
    """Run `steps` steps; with `record`, bracket every kernel with events."""
    pairs = []
    for _ in range(warmup):
        for op in ops:
            op.act_fn()
            op.gemm_fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    t0 = time.perf_counter()
    for _ in range(steps):
        for op in ops:
            if record:
                ea0, ea1, eg1 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
                ea0.record(stream)
                op.act_fn()
                ea1.record(stream)
                op.gemm_fn()
                eg1.record(stream)
                pairs.append((op, ea0, ea1, eg1))
            else:
                op.act_fn()
                op.gemm_fn()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for op, ea0, ea1, eg1 in pairs:
        op.t_act.append(ea0.elapsed_time(ea1) * 1e-3)
        op.t_gemm.append(ea1.elapsed_time(eg1) * 1e-3)
    return start.elapsed_time(end) * 1e-3, wall


def bf16_context(torch, layers, M_list, rotate_bytes, steps):
    """Same-shape BF16 torch.matmul (hipBLASLt/rocBLAS), weights rotated."""
    out = {}
    for name, c in layers:
        Wb = torch.from_numpy(c.W.view("int16")).cuda().view(torch.bfloat16)
        R = max(1, math.ceil(rotate_bytes / (Wb.numel() * 2)))
        Ws = [Wb.clone() for _ in range(R)]
        X = torch.from_numpy(c.X.view("int16")).cuda().view(torch.bfloat16)
        for M in M_list:
            Xm = X[:M]
            for r in range(R):
                torch.matmul(Xm, Ws[r].t())
            torch.cuda.synchronize()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            n = max(steps, R)
            s.record()
            for i in range(n):
                torch.matmul(Xm, Ws[i % R].t())
            e.record()
            torch.cuda.synchronize()
            out[f"{name}/M={M}"] = s.elapsed_time(e) * 1e-3 / n   # seconds
        del Ws
    return out


def cpu_baseline(np, layers, M_list, budget_s=12.0):
    """The oracle (as it stands) on the host cores: act-quant + GEMM of every
    (layer, M) pair of one step, repeated until about `budget_s` seconds."""
    from oracle import prquant as pq
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    name, c = layers[0]
    t0 = time.perf_counter()
    art = pq.prepare(c.W, c.Xcal, c.alpha, c.k_tail)
    log(f"[bench] oracle prepare (untimed): {time.perf_counter() - t0:.1f} s")
    K, k, N = c.K, c.k_tail, c.N
    K_aug = K + k
    byts, reps = 0.0, 0
    t0 = time.perf_counter()
    while True:
        for M in M_list:
            Aq, Asc = pq.quant_act(c.X[:M], art["inv_scale"], art["perm"], k)
            pq.gemm(Aq, Asc, art["Wq"], art["Wsc"])
            byts += act_bytes(M, K, K_aug) + gemm_bytes(M, N, K_aug)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 50:
            break
    threads = max(threads, 1)
    return {"value": round(byts / el / 1e9, 4), "unit": "GB/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{reps} passes of oracle act-quant + GEMM at M={list(M_list)} on {name} "
                      f"(N={N}, K={K}, k={k}); {el:.1f} s; host cores visible "
                      f"{len(os.sched_getaffinity(0))}, BLAS threads {threads}"}


CALIB_BYTES = 512 * 2 ** 20
GEMM_SOURCES = ("gemm_stream.hip", "gemm_tile.hip", "mx_device.hpp", "prq_internal.h", "abi.cpp")


def copy_calibration(torch, nbytes=CALIB_BYTES, reps=5):
    """A plain streaming kernel of known traffic (reads and writes `nbytes`),
    for scaling the HBM counters: torch.neg over float32."""
    a = torch.zeros(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    log(f"[bench] copy calibration: {reps} x neg over {nbytes} bytes")


def gemm_source_hash():
    h = hashlib.sha256()
    for name in GEMM_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2609_22106_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def traffic_record(workload):
    """HBM bytes per GEMM launch from committed counter runs, or None when the
    GEMM sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    return rec.get("bytes_per_launch") if rec.get("gemm_src_sha256_16") == gemm_source_hash() else None


def _counter_rows(run_dir, counter):
    """(dispatch id, kernel name, value) of `counter` from a rocprofv3 --pmc
    CSV output directory."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no *counter_collection.csv under {run_dir}")
    per = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r.get("Counter_Name") != counter:
                continue
            key = (f, r["Dispatch_Id"])
            name, v = per.get(key, (r["Kernel_Name"], 0.0))
            per[key] = (name, v + float(r["Counter_Value"]))
    return list(per.values())


def traffic_from_counters(workload, fetch_dir, write_dir, command):
    """Write profiles/traffic_<workload>.json from a FETCH_SIZE run and a
    WRITE_SIZE run of `bench.py --copy-calibration` (KiB per dispatch), each
    scaled by what the same counter reads for the calibration kernel."""
    out = {"workload": workload, "command": command, "calibration_bytes": CALIB_BYTES}
    total = 0.0
    for counter, run_dir in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _counter_rows(run_dir, counter)
        calib = [v for n, v in rows if "neg_kernel" in n]
        gemm = [(n, v) for n, v in rows if "prq" in n and any(
            t in n for t in ("gemm_stream_kernel", "gemm_tile_kernel", "reduce_partials_kernel", "zero_kernel"))]
        launches = [v for n, v in gemm if "gemm_" in n]
        if not calib or not launches:
            raise SystemExit(f"{counter}: calibration or GEMM dispatches missing in {run_dir}")
        scale = CALIB_BYTES / (sorted(calib)[len(calib) // 2] * 1024.0)
        per_launch = sum(v for _, v in gemm) * 1024.0 * scale / len(launches)
        out[counter] = {"calibration_kib_median": sorted(calib)[len(calib) // 2], "scale": scale,
                        "gemm_dispatches": len(launches), "helper_dispatches": len(gemm) - len(launches),
                        "bytes_per_launch": per_launch}
        total += per_launch
    out["bytes_per_launch"] = round(total, 1)
    out["gemm_src_sha256_16"] = gemm_source_hash()
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))
    return 0


# ---------------------------------------------------------------- main ---
def main(argv=None):
    args = parse_args(argv)
    if args.traffic_from:
        return traffic_from_counters(args.workload, *args.traffic_from, args.traffic_command)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "sharding of this path is described in DESIGN.md and not built.", file=sys.stderr)
        return 2
    import numpy as np
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU (torch.cuda.is_available() is False)", file=sys.stderr)
        return 3
    sys.path.insert(0, ROOT)
    from paper_2609_22106_amd import inputs, prq

    stream = torch.cuda.current_stream()
    wl = args.workload
    if wl in ("decode", "prefill"):
        c = inputs.down_proj_decode() if wl == "decode" else inputs.down_proj_prefill()
        layers = [("qwen3_4b_down_proj", c)]
        M_list = list(c.M_list)
        ops = build_dense_ops(torch, prq, layers, M_list, args.rotate_bytes, stream)
        config = {"workload": f"qwen3_4b_down_proj_{wl}", "N": 2560, "K": 9728, "k_tail": 256,
                  "alpha": 0.5, "M": M_list}
    elif wl in ("experts", "experts_prefill"):
        tokens = 64 if wl == "experts" else 4096
        ops = build_expert_ops(torch, np, prq, inputs, tokens, args.rotate_bytes, stream)
        layers, M_list = [], []
        config = {"workload": f"qwen3_30b_a3b_expert_down_proj_{tokens}tok", "E": 128, "N": 2048,
                  "K": 768, "k_tail": 64, "alpha": 0.5, "topk": 8, "routed_rows": ops[0].M}
    else:
        layers = [(n, inputs.layer_case(n)) for n, _, _ in inputs.LAYER_SET]
        M_list = [4096]
        ops = build_dense_ops(torch, prq, layers, M_list, args.rotate_bytes, stream)
        config = {"workload": "qwen3_4b_decoder_linears_prefill", "M": 4096,
                  "layers": {n: {"N": c.N, "K": c.K, "k_tail": c.k_tail} for n, c in layers}}

    if args.copy_calibration:
        copy_calibration(torch)
    # untimed warmup, then the timed region: whole steps, with HIP events on
    # the launch stream around every kernel for the per-kernel durations
    run_steps(torch, ops, 0, args.warmup, stream, record=False)
    t_gpu, t_wall = run_steps(torch, ops, args.steps, 0, stream, record=True)
    ms_per_step = t_gpu / args.steps * 1e3
    step_bytes = sum(op.gemm_bytes + op.act_bytes for op in ops)
    step_flops = sum(op.flops for op in ops)
    value = step_bytes / (t_gpu / args.steps) / 1e9

    detail = {}
    g_bytes = g_time = 0.0
    for op in ops:
        tg = float(np.mean(op.t_gemm))
        ta = float(np.mean(op.t_act))
        g_bytes += op.gemm_bytes
        g_time += tg
        detail[op.name] = {
            "gemm_us": round(tg * 1e6, 3), "act_quant_us": round(ta * 1e6, 3),
            "op_us": round((tg + ta) * 1e6, 3),
            "gemm_GBs": round(op.gemm_bytes / tg / 1e9, 1),
            "gemm_TFLOPs": round(op.flops / tg / 1e12, 2),
            "gemm_hbm_frac": round(op.gemm_bytes / tg / 1e9 / HBM_PEAK_GBS, 4),
            "gemm_mfma_frac": round(op.flops / tg / 1e12 / MXFP4_PEAK_TFLOPS, 4),
            "act_quant_GBs": round(op.act_bytes / ta / 1e9, 1),
        }
    flops_per_byte = step_flops / max(step_bytes, 1)
    bound = "mfma" if flops_per_byte > MXFP4_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"
    g_flops = sum(op.flops for op in ops)
    if bound == "hbm":
        achieved, peak, unit = g_bytes / g_time / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = g_flops / g_time / 1e12, MXFP4_PEAK_TFLOPS, "TFLOP/s"
    roofline = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4), "traffic": traffic_record(wl),
                "kernel": "prq_gemm (augmented MXFP4 GEMM over K+k)",
                "per_launch_bytes": round(g_bytes / len(ops), 1),
                "avg_launch_us": round(g_time / len(ops) * 1e6, 3)}

    if not args.no_bf16 and layers:
        bf = bf16_context(torch, layers, M_list, args.rotate_bytes, args.steps)
        for key, t in bf.items():
            if key in detail:
                detail[key]["bf16_matmul_us"] = round(t * 1e6, 3)
                detail[key]["speedup_op_vs_bf16"] = round(t / (detail[key]["op_us"] * 1e-6), 3)
                detail[key]["speedup_gemm_vs_bf16"] = round(t / (detail[key]["gemm_us"] * 1e-6), 3)

    cpu = None
    if not args.no_cpu_baseline and wl in ("decode",):
        cpu = cpu_baseline(np, layers, M_list)

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "mxfp4", "data": "synthetic", "config": config,
        "tflops": round(step_flops / (t_gpu / args.steps) / 1e12, 3),
        "roofline": roofline, "cpu_baseline": cpu, "detail": detail,
        "wall_s_timed": round(t_wall, 4),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

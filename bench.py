#!/usr/bin/env python3
"""Benchmark of the PRQuant MXFP4 + tail-residual hot path on one MI355X.

Default workload: the Qwen3-4B-shaped down_proj at decode (K = 9728 -> N =
2560, k = 256, rows M = 1, 8, 32, 64).  One step = for every M, the fused
activation quantization (prq_quant_act) followed by the augmented MXFP4 GEMM
over K + k (prq_gemm) on one stream, with inputs resident in HBM; the offline
prq_prepare runs once before timing.  Weights are rotated through enough
copies (>= 1 GiB) that every step streams them from HBM rather than from the
256 MB Infinity Cache.

Timed region: exactly `--steps` whole steps captured into one HIP graph (each
step binding the next rotated weight copy) and replayed once, bracketed by
torch.cuda.synchronize() on both sides and HIP events on the stream -- how a
serving loop launches a step, and free of per-kernel instrumentation.  The
per-kernel durations (detail, roofline) come from a separate pass of the same
steps launched eagerly, queued behind a GPU spin-sleep, with fence-free HIP
events around every kernel; its step time is reported as
``eager_ms_per_step`` (events add ~2-4 us per kernel).  --no-graph times the
eager pass instead.

Prints ONE JSON line on stdout (everything else goes to stderr):
  value = algorithmic bytes of one step / step time (GB/s), plus per-M
  kernel times, TFLOP/s, roofline fraction of the dominant kernel (the GEMM)
  from the events around its launches, a same-shape BF16 torch.matmul for
  context, and the CPU oracle timed on a bounded sample (``cpu_baseline``).

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
import re
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
    p.add_argument("--no-graph", action="store_true", help="skip the graph-replay cross-check")
    p.add_argument("--no-plain", action="store_true", help="skip the plain MXFP4 (k = 0) context")
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


PACKED_MIN_ROWS = 64   # more rows than this: the packed prefill pair
PACKED_MIN_EXPERT_ROWS = 64   # mean routed rows per expert from which experts use it


def build_dense_ops(torch, prq, layers, M_list, rotate_bytes, plain=False):
    """layers: list of (name, DenseCase).  Weights rotated, activations per M.
    plain: the plain MXFP4 baseline (no scaling, no tail: k = 0)."""
    ops = []
    for name, c in layers:
        K, k, N = c.K, (0 if plain else c.k_tail), c.N
        K_aug = K + k
        t0 = time.perf_counter()
        art = prq.prq_prepare(c.W, c.Xcal, c.alpha, k, "none" if plain else "smooth")
        log(f"[bench] prq_prepare {name}: {time.perf_counter() - t0:.2f} s")
        w_bytes = art["Wq"].nbytes + art["Wsc"].nbytes
        R = max(1, math.ceil(rotate_bytes / w_bytes))
        Wc = prq.prq_pack_weight(torch.from_numpy(art["Wq"]).cuda(), torch.from_numpy(art["Wsc"]).cuda())
        Ws = [prq.PackedWeight(Wc.Wp.clone(), Wc.Wps.clone(), 1, N, K_aug) for _ in range(R)]
        inv = torch.from_numpy(art["inv_scale_pos"]).cuda()
        perm = torch.from_numpy(art["perm"]).cuda()
        X = torch.from_numpy(c.X.view("int16")).cuda()
        for M in M_list:
            Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
            Xm = X[:M]
            state = {"r": 0}
            # every per-layer buffer is bound here: a name captured from the
            # enclosing loop would see the last layer's buffers in every op
            if M > PACKED_MIN_ROWS:
                # prefill: the packed pair (activation written in the layout the
                # tile GEMM copies in whole kilobytes)
                A = prq.prq_quant_act_packed(Xm, K, k, inv, perm)
                ws_n = prq.prq_gemm_packed_workspace_bytes(M, N, K_aug)   # split along K
                ws = torch.empty(ws_n, dtype=torch.uint8, device="cuda") if ws_n else None

                def act(Xm=Xm, A=A, K=K, k=k, inv=inv, perm=perm):
                    prq.prq_quant_act_packed(Xm, K, k, inv, perm, out=A)

                def gemm(A=A, Y=Y, ws=ws, state=state, R=R, Ws=Ws):
                    r = state["r"]
                    state["r"] = (r + 1) % R
                    prq.prq_gemm_packed(A, Ws[r], Y=Y, workspace=ws)
            else:
                Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
                Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")
                ws_n = prq.prq_gemm_workspace_bytes(M, N, K_aug)
                ws = torch.zeros(max(ws_n, 1), dtype=torch.uint8, device="cuda") if ws_n else None

                def act(Xm=Xm, Aq=Aq, Asc=Asc, K=K, k=k, inv=inv, perm=perm):
                    prq.prq_quant_act(Xm, K, k, inv, perm, Aq=Aq, Asc=Asc)

                def gemm(Aq=Aq, Asc=Asc, Y=Y, ws=ws, state=state, R=R, Ws=Ws):
                    r = state["r"]
                    state["r"] = (r + 1) % R
                    prq.prq_gemm(Aq, Asc, Ws[r], Y=Y, workspace=ws)

            ops.append(Op(f"{name}/M={M}", M, N, K, k, act, gemm, gemm_bytes(M, N, K_aug),
                          act_bytes(M, K, K_aug), 2.0 * M * N * K_aug))
        log(f"[bench] {name}: {R} rotated weight copies ({w_bytes / 1e6:.2f} MB each)")
    return ops


def build_expert_ops(torch, np, prq, inputs, tokens, rotate_bytes):
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
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    state = {"r": 0}
    e_active = int(np.count_nonzero(np.diff(c.group_offsets)))

    if M >= PACKED_MIN_EXPERT_ROWS * E:
        # prefill: the packed pair (grouped tile GEMM on the packed activation)
        A = prq.prq_quant_act_packed(X, K, k, inv, perm, group_offsets=off, G=E)

        def act():
            prq.prq_quant_act_packed(X, K, k, inv, perm, out=A, group_offsets=off, G=E)

        def gemm():
            r = state["r"]
            state["r"] = (r + 1) % R
            prq.prq_grouped_gemm_packed(A, off, Ws[r], Y=Y)
    else:
        Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device="cuda")
        Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device="cuda")

        def act():
            prq.prq_quant_act(X, K, k, inv, perm, group_offsets=off, G=E, Aq=Aq, Asc=Asc)

        def gemm():
            r = state["r"]
            state["r"] = (r + 1) % R
            prq.prq_grouped_gemm(Aq, Asc, off, Ws[r], Y=Y)

    log(f"[bench] experts: {M} routed rows, {e_active} active experts, {R} weight copies")
    return [Op(f"experts/{tokens}tok", M, N, K, k, act, gemm,
               grouped_gemm_bytes(M, e_active, N, K_aug), act_bytes(M, K, K_aug) + 8 * K * (E - 1),
               2.0 * M * N * K_aug)]


# -------------------------------------------------------------- timing ---
def step_once(ops):
    for op in ops:
        op.act_fn()
        op.gemm_fn()


def sleep_rate(torch, stream):
    """GPU spin-sleep cycles per second (torch.cuda._sleep), measured."""
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(100_000)
    a.record(stream)
    torch.cuda._sleep(4_000_000)
    b.record(stream)
    torch.cuda.synchronize()
    return 4_000_000 / (a.elapsed_time(b) * 1e-3)


class HipTimer:
    """Timing events made through the HIP runtime that torch has loaded (found
    in /proc/self/maps, so it is the same runtime instance), created with
    hipEventDisableSystemFence: recording such an event skips the system-scope
    cache writeback/invalidate that a default event performs, which would
    otherwise add microseconds to every bracketed kernel of a few
    microseconds."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        path = next(line.split()[-1] for line in open("/proc/self/maps") if "libamdhip64" in line)
        self.ct = ctypes
        self.hip = ctypes.CDLL(path)
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.path = path

    def _ok(self, err, what):
        if err != 0:
            raise RuntimeError(f"{what} failed with HIP error {err}")

    def event(self):
        e = self.ct.c_void_p()
        self._ok(self.hip.hipEventCreateWithFlags(self.ct.byref(e), self.DISABLE_SYSTEM_FENCE),
                 "hipEventCreateWithFlags")
        return e

    def record(self, e, stream):
        self._ok(self.hip.hipEventRecord(e, self.ct.c_void_p(stream.cuda_stream)), "hipEventRecord")

    def seconds(self, a, b):
        ms = self.ct.c_float()
        self._ok(self.hip.hipEventElapsedTime(self.ct.byref(ms), a, b), "hipEventElapsedTime")
        return ms.value * 1e-3

    def destroy(self, events):
        for e in events:
            self.hip.hipEventDestroy(e)


def run_steps(torch, ops, steps, warmup, stream):
    """Warmup, then the timed region: `steps` whole steps with HIP events on
    the launch stream around every kernel.  The launches are queued behind a
    GPU spin-sleep long enough for the host to enqueue all of them, so the
    region measures the GPU executing the steps back to back, not the host's
    per-launch cost (which a serving loop hides with a graph; see
    graph_step_time)."""
    for _ in range(warmup):
        step_once(ops)
    torch.cuda.synchronize()
    rate = sleep_rate(torch, stream)
    t0 = time.perf_counter()
    step_once(ops)                                   # host enqueue cost of a step
    host_step = time.perf_counter() - t0
    torch.cuda.synchronize()
    # events add host time per launch too: budget 2x the measured step, +5 ms
    hold_s = min(2.0, steps * host_step * 2.0 + 5e-3)
    timer = HipTimer()
    start, end = timer.event(), timer.event()
    pairs = [(op, timer.event(), timer.event(), timer.event()) for _ in range(steps) for op in ops]
    torch.cuda._sleep(int(hold_s * rate))
    timer.record(start, stream)
    t0 = time.perf_counter()
    for op, ea0, ea1, eg1 in pairs:
        timer.record(ea0, stream)
        op.act_fn()
        timer.record(ea1, stream)
        op.gemm_fn()
        timer.record(eg1, stream)
    timer.record(end, stream)
    enqueue_s = time.perf_counter() - t0
    torch.cuda.synchronize()
    for op, ea0, ea1, eg1 in pairs:
        op.t_act.append(timer.seconds(ea0, ea1))
        op.t_gemm.append(timer.seconds(ea1, eg1))
    gpu_s = timer.seconds(start, end)
    timer.destroy([start, end] + [e for p in pairs for e in p[1:]])
    return gpu_s, {"host_enqueue_s": round(enqueue_s, 5), "gpu_hold_s": round(hold_s, 5),
                   "queued_ahead": bool(enqueue_s < hold_s)}


def graph_step_time(torch, ops, steps):
    """Exactly `steps` steps captured into one HIP graph and replayed once
    (after one untimed replay), bracketed by synchronize: (GPU seconds per
    step from events around the replay, host wall seconds of the replay)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step_once(ops)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    # all `steps` steps in one graph: each captured step binds the next
    # rotated weight copy, so replays stream the same >= 1 GiB of weights as
    # the eager region (a short graph would cycle through few enough copies to
    # be served from the Infinity Cache)
    per_graph = max(1, steps)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(per_graph):
            step_once(ops)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    a.record()
    g.replay()
    b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    del g
    return a.elapsed_time(b) * 1e-3 / per_graph, wall


def copy_context(torch, prq, layers, M_list, reps=50):
    """Activation side, online copy (gather by perm, scale, quantize, copy the
    tail blocks) against offline copy (the expanded producer already emitted
    [Z~, Z~_tail]: a plain quantizer over K + k), both launched back to back
    on warm inputs (seconds per launch)."""
    out = {}
    for name, c in layers:
        K, k = c.K, c.k_tail
        art = prq.prq_prepare(c.W, c.Xcal, c.alpha, k)
        inv = torch.from_numpy(art["inv_scale_pos"]).cuda()
        perm = torch.from_numpy(art["perm"]).cuda()
        X = torch.from_numpy(c.X.view("int16")).cuda()
        g = torch.Generator(device="cpu").manual_seed(0)
        Zaug = (torch.randn((max(M_list), K + k), generator=g) * 2).to(torch.bfloat16).cuda()
        for M in M_list:
            res = {}
            if M > PACKED_MIN_ROWS:     # the quantizer the step uses: packed output
                A = prq.prq_quant_act_packed(X[:M], K, k, inv, perm)
                fns = (("online", lambda: prq.prq_quant_act_packed(X[:M], K, k, inv, perm, out=A)),
                       ("offline", lambda: prq.prq_quant_act_packed(Zaug[:M], K + k, 0, out=A)))
            else:
                Aq = torch.empty((M, (K + k) // 2), dtype=torch.uint8, device="cuda")
                Asc = torch.empty((M, (K + k) // 32), dtype=torch.uint8, device="cuda")
                fns = (("online", lambda: prq.prq_quant_act(X[:M], K, k, inv, perm, Aq=Aq, Asc=Asc)),
                       ("offline", lambda: prq.prq_quant_act(Zaug[:M], K + k, 0, Aq=Aq, Asc=Asc)))
            for label, fn in fns:
                for _ in range(3):
                    fn()
                torch.cuda.synchronize()
                torch.cuda._sleep(20_000_000)
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(reps):
                    fn()
                b.record()
                torch.cuda.synchronize()
                res[label] = a.elapsed_time(b) * 1e-3 / reps
            out[f"{name}/M={M}"] = res
    return out


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
GEMM_SOURCES = ("gemm_decode.hip", "gemm_stream.hip", "gemm_streamk.hip", "gemm_tile.hip", "mx_device.hpp",
                "prq_internal.h", "abi.cpp")


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
    """HBM bytes per GEMM call from committed counter runs, or None when the
    GEMM sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    return rec.get("bytes_per_call") if rec.get("gemm_src_sha256_16") == gemm_source_hash() else None


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


# GEMM calls per step of each workload (one per op; a call may be several
# dispatches, e.g. the two column regions of a planned tile GEMM).
GEMM_OPS_PER_STEP = {"decode": 4, "prefill": 3, "experts": 1, "experts_prefill": 1, "layers": 7}


def _steps_run(command):
    """Steps a counter run executed: --warmup + --steps + the one step that
    measures the host enqueue cost (bench.py defaults when absent)."""
    def opt(name, default):
        m = re.search(rf"--{name}\s+(\d+)", command)
        return int(m.group(1)) if m else default
    return opt("warmup", 10) + opt("steps", 50) + 1


def traffic_from_counters(workload, fetch_dir, write_dir, command):
    """Write profiles/traffic_<workload>.json from a FETCH_SIZE run and a
    WRITE_SIZE run of `bench.py --copy-calibration` (KiB per dispatch), each
    scaled by what the same counter reads for the calibration kernel.  The
    record is HBM bytes per GEMM call (all of a call's dispatches), the unit of
    the roofline's algorithmic bytes."""
    out = {"workload": workload, "command": command, "calibration_bytes": CALIB_BYTES}
    calls = _steps_run(command) * GEMM_OPS_PER_STEP[workload]
    out["gemm_calls"] = calls
    total = 0.0
    for counter, run_dir in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _counter_rows(run_dir, counter)
        calib = [v for n, v in rows if "neg_kernel" in n]
        gemm = [(n, v) for n, v in rows if "prq" in n and any(
            t in n for t in ("gemm_decode_kernel", "gemm_stream_kernel", "gemm_tile_kernel", "gemm_grouped_persist_kernel",
                             "reduce_partials_kernel", "zero_kernel", "splitk_reduce_kernel"))]
        launches = [v for n, v in gemm if "gemm_" in n]
        if not calib or not launches:
            raise SystemExit(f"{counter}: calibration or GEMM dispatches missing in {run_dir}")
        scale = CALIB_BYTES / (sorted(calib)[len(calib) // 2] * 1024.0)
        per_call = sum(v for _, v in gemm) * 1024.0 * scale / calls
        out[counter] = {"calibration_kib_median": sorted(calib)[len(calib) // 2], "scale": scale,
                        "gemm_dispatches": len(launches), "helper_dispatches": len(gemm) - len(launches),
                        "bytes_per_call": per_call}
        total += per_call
    out["bytes_per_call"] = round(total, 1)
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
              "sharding of this path is not built.", file=sys.stderr)
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
        ops = build_dense_ops(torch, prq, layers, M_list, args.rotate_bytes)
        config = {"workload": f"qwen3_4b_down_proj_{wl}", "N": 2560, "K": 9728, "k_tail": 256,
                  "alpha": 0.5, "M": M_list}
    elif wl in ("experts", "experts_prefill"):
        tokens = 64 if wl == "experts" else 4096
        ops = build_expert_ops(torch, np, prq, inputs, tokens, args.rotate_bytes)
        layers, M_list = [], []
        config = {"workload": f"qwen3_30b_a3b_expert_down_proj_{tokens}tok", "E": 128, "N": 2048,
                  "K": 768, "k_tail": 64, "alpha": 0.5, "topk": 8, "routed_rows": ops[0].M}
    else:
        layers = [(n, inputs.layer_case(n)) for n, _, _ in inputs.LAYER_SET]
        M_list = [4096]
        ops = build_dense_ops(torch, prq, layers, M_list, args.rotate_bytes)
        config = {"workload": "qwen3_4b_decoder_linears_prefill", "M": 4096,
                  "layers": {n: {"N": c.N, "K": c.K, "k_tail": c.k_tail} for n, c in layers}}

    if args.copy_calibration:
        copy_calibration(torch)
    # untimed warmup, then the timed region: whole steps, with HIP events on
    # the launch stream around every kernel for the per-kernel durations
    t_gpu, queue_info = run_steps(torch, ops, args.steps, args.warmup, stream)
    t_eager_step = t_gpu / args.steps
    if args.no_graph:
        t_step, t_wall = t_eager_step, None
    else:
        t_step, t_wall = graph_step_time(torch, ops, args.steps)
    ms_per_step = t_step * 1e3
    step_bytes = sum(op.gemm_bytes + op.act_bytes for op in ops)
    step_flops = sum(op.flops for op in ops)
    value = step_bytes / t_step / 1e9

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
    # the GEMM's own arithmetic intensity decides which roof bounds it
    g_flops = sum(op.flops for op in ops)
    bound = "mfma" if g_flops / max(g_bytes, 1) > MXFP4_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"
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

    if layers and not args.no_plain:
        # plain MXFP4 (k = 0, no scaling) through the same kernels and timing
        plain_ops = build_dense_ops(torch, prq, layers, M_list, args.rotate_bytes, plain=True)
        t_plain, _ = run_steps(torch, plain_ops, args.steps, args.warmup, stream)
        for op in plain_ops:
            if op.name in detail:
                tg, ta = float(np.mean(op.t_gemm)), float(np.mean(op.t_act))
                d = detail[op.name]
                d["plain_mxfp4_gemm_us"] = round(tg * 1e6, 3)
                d["plain_mxfp4_op_us"] = round((tg + ta) * 1e6, 3)
                d["op_over_plain_mxfp4"] = round(d["op_us"] / ((tg + ta) * 1e6), 3)
        del plain_ops
    if layers and wl in ("decode", "prefill"):
        for key, r in copy_context(torch, prq, layers, M_list).items():
            if key in detail:
                detail[key]["act_quant_online_copy_warm_us"] = round(r["online"] * 1e6, 3)
                detail[key]["act_quant_offline_copy_warm_us"] = round(r["offline"] * 1e6, 3)

    cpu = None
    if not args.no_cpu_baseline and wl in ("decode",):
        cpu = cpu_baseline(np, layers, M_list)

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "mxfp4", "data": "synthetic", "config": config,
        "tflops": round(step_flops / t_step / 1e12, 3),
        "roofline": roofline, "cpu_baseline": cpu, "detail": detail,
        "timing": {
            "method": ("eager: the steps launched directly" if args.no_graph else
                       f"{args.steps} steps in one HIP graph, replayed once between "
                       "torch.cuda.synchronize() calls, HIP events around the replay"),
            "replay_wall_s": None if t_wall is None else round(t_wall, 6),
            "eager_ms_per_step": round(t_eager_step * 1e3, 5),
            "eager_method": "eager launches queued behind a GPU spin-sleep; HIP events "
                            "(hipEventDisableSystemFence) on the launch stream around every kernel",
            **queue_info},
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

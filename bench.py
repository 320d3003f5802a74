#!/usr/bin/env python3
"""Benchmark of the PRQuant MXFP4 + tail-residual hot path on one MI355X.

Headline workload: the Qwen3-4B-shaped down_proj at decode (K = 9728 -> N =
2560, k = 256, rows M = 1, 8, 32, 64).  One step = for every M, the fused
activation quantization (prq_quant_act) followed by the augmented MXFP4 GEMM
over K + k (prq_gemm) on one stream, with inputs resident in HBM; the offline
prq_prepare runs once before timing.  Weights are rotated through enough
copies (>= 1 GiB) that every step streams them from HBM rather than from the
256 MB Infinity Cache.

Timed region: exactly `--steps` whole steps captured into one HIP graph (each
step binding the next rotated weight copy), replayed once untimed and then five
times, each replay bracketed by torch.cuda.synchronize() and HIP events on the
stream; ms_per_step is the median replay over --steps.  Per-kernel launch
durations (detail, roofline) come from batches of back-to-back launches of one
kernel (rotated weights), queued behind a GPU spin-sleep, with fence-free HIP
events around each batch only.

By default (--workload all) the other workloads run after the headline and
appear in ``detail`` (per op) and ``workloads`` (per step, with their GEMM
roofline): prefill (M = 512, 2048, 8192), experts (128 expert down_projs
768 -> 2048, k = 64, 64 tokens routed top-8, one grouped launch),
experts_prefill (4096 tokens), layers (the seven linears of a
Qwen3-4B-shaped decoder layer at M = 4096).  --workload X runs X alone as the
headline.

Prints ONE JSON line on stdout (everything else goes to stderr): value =
algorithmic bytes of one headline step / step time (GB/s), per-kernel times,
TFLOP/s, the GEMM roofline fraction, context timings (same-shape BF16
torch.matmul, plain MXFP4 through the same kernels, the weight-read floor,
hot-cache step), the CPU oracle timed on a bounded sample (``cpu_baseline``),
GPU clocks and ROCm version.

--counters runs --warmup + --steps eager steps of one workload and nothing
else (for rocprofv3 --pmc); --traffic-from turns two such counter runs into
profiles/traffic_<workload>.json.
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
    p.add_argument("--workload", default="all",
                   choices=["all", "decode", "prefill", "experts", "experts_prefill", "layers"],
                   help="all: the decode headline plus every other workload in detail")
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
    p.add_argument("--counters", action="store_true",
                   help="run --warmup + --steps eager steps of --workload and nothing else")
    p.add_argument("--lds-patterns", action="store_true",
                   help="first run the LDS read-pattern probe kernels (reference points for "
                        "the bank-conflict counters); alone, nothing else")
    return p.parse_args(argv)


# ----------------------------------------------------------- workloads ---
def act_bytes(M, K, K_aug):
    return 2 * M * K + M * K_aug * 17 / 32 + 8 * K


def gemm_bytes(M, N, K_aug):
    return (N + M) * K_aug * 17 / 32 + 4 * M * N


def grouped_gemm_bytes(M, E_active, N, K_aug):
    return (E_active * N + M) * K_aug * 17 / 32 + 4 * M * N


# Rows from which a dense op runs the packed pair: one 16-row group or fewer
# run row-major (the packed layout would stage and store a whole 16-row block;
# measured on the down_proj decode rows, back to back, quantizer + GEMM: M = 1
# 7.7 us row-major vs 8.5 packed, M = 8 8.2 vs 8.6, M = 32 10.8 vs 10.5, M = 64
# 14.0 vs 13.5).
PACKED_MIN_ROWS = 17


class Op:
    """One act-quant + GEMM pair of a step (launch closures bound to buffers)."""

    def __init__(self, name, M, N, K, k, act_fn, gemm_fn, gbytes, abytes, flops):
        self.name, self.M, self.N, self.K, self.k = name, M, N, K, k
        self.act_fn, self.gemm_fn = act_fn, gemm_fn
        self.gemm_bytes, self.act_bytes, self.flops = gbytes, abytes, flops
        self.t_gemm = self.t_act = None
        self.weights = None


PACKED_MIN_EXPERT_ROWS = 64   # mean routed rows per expert from which experts use it


def build_dense_ops(torch, prq, layers, M_list, rotate_bytes, plain=False, rowmajor=False):
    """layers: list of (name, DenseCase).  Weights rotated, activations per M.
    From PACKED_MIN_ROWS rows the packed pair (activation written in the layout
    the GEMM copies in whole kilobytes: the whole-K decode kernel up to 64 rows,
    the tile GEMM above), else (or with rowmajor) prq_quant_act + prq_gemm.
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
            if M >= PACKED_MIN_ROWS and not rowmajor:
                A = prq.prq_quant_act_packed(Xm, K, k, inv, perm)
                ws_n = prq.prq_gemm_packed_workspace_bytes(M, N, K_aug)   # split along K
                ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda") if ws_n else None

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
            ops[-1].weights = Ws
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


def time_kernels(torch, ops, reps, warmup, stream):
    """Per-kernel launch durations: for every op, `reps` back-to-back launches
    of its activation quantizer, then `reps` of its GEMM (the GEMM binding the
    next rotated weight copy each time), each batch queued behind a GPU
    spin-sleep long enough for the host to enqueue it and bracketed by two
    fence-free HIP events on the launch stream (after one untimed batch of the
    same launches); per-launch seconds = batch time / reps.  The quantizer's
    inputs are therefore warm here (in a step they follow a weight stream).  No event sits between two launches of a batch, so the figure is
    the kernel's average duration in a stream of launches (gaps included)."""
    for _ in range(warmup):
        step_once(ops)
    torch.cuda.synchronize()
    rate = sleep_rate(torch, stream)
    timer = HipTimer()
    for op in ops:
        for kind, fn in (("act", op.act_fn), ("gemm", op.gemm_fn)):
            t0 = time.perf_counter()
            fn()
            host = time.perf_counter() - t0
            torch.cuda.synchronize()
            hold_s = min(2.0, reps * host * 2.0 + 2e-3)
            a, b = timer.event(), timer.event()
            for timed in (False, True):      # an untimed batch first: clocks and caches settle
                torch.cuda._sleep(int(hold_s * rate))
                timer.record(a, stream)
                for _ in range(reps):
                    fn()
                timer.record(b, stream)
                torch.cuda.synchronize()
            per = timer.seconds(a, b) / reps
            timer.destroy([a, b])
            if kind == "act":
                op.t_act = per
            else:
                op.t_gemm = per


def graph_step_times(torch, ops, steps, replays=5):
    """Exactly `steps` steps captured into one HIP graph (each captured step
    binds the next rotated weight copy, so a replay streams >= 1 GiB of
    weights from HBM, not the 256 MB Infinity Cache), replayed once untimed and
    then `replays` times, each bracketed by torch.cuda.synchronize() and events:
    (GPU seconds per step of each timed replay, host wall seconds of each)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step_once(ops)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(steps):
            step_once(ops)
    g.replay()
    torch.cuda.synchronize()
    gpu, wall = [], []
    for _ in range(replays):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        wall.append(time.perf_counter() - t0)
        gpu.append(a.elapsed_time(b) * 1e-3 / steps)
    del g
    return gpu, wall


def read_floor(torch, prq, W_list, reps=160):
    """The weight-read floor of the decode GEMM (context, committed probe
    kernel of the test library): every byte of a packed weight (codes and
    scales) read with one workgroup per CU, each an equal contiguous share,
    nothing computed; back-to-back launches over the same rotated copies as the
    GEMM, seconds per launch."""
    import ctypes
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.prq_probe_read_floor.argtypes = [P, I, P, I, I, P, P]
    lib.prq_probe_read_floor.restype = I
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.zeros(cus, dtype=torch.int32, device="cuda")
    sp = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    R = len(W_list)

    def launch(i):
        W = W_list[i % R]
        st = lib.prq_probe_read_floor(W.Wp.data_ptr(), W.Wp.numel() // 1024, W.Wps.data_ptr(),
                                      W.Wps.numel() // 1024, cus, out.data_ptr(), sp)
        if st != 0:
            raise RuntimeError(f"prq_probe_read_floor failed ({st})")
    for i in range(5):
        launch(i)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(reps):
        launch(i)
    b.record()
    torch.cuda.synchronize()
    W = W_list[0]
    nbytes = (W.Wp.numel() // 1024 + W.Wps.numel() // 1024) * 1024
    return a.elapsed_time(b) * 1e-3 / reps, nbytes


def gpu_info(torch):
    """Device, clocks and ROCm versions for the record."""
    import ctypes
    info = {"device": torch.cuda.get_device_name(0),
            "arch": getattr(torch.cuda.get_device_properties(0), "gcnArchName", None),
            "cus": torch.cuda.get_device_properties(0).multi_processor_count,
            "torch_hip": torch.version.hip}
    try:
        info["rocm"] = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        info["rocm"] = None
    try:
        path = next(line.split()[-1] for line in open("/proc/self/maps") if "libamdhip64" in line)
        hip = ctypes.CDLL(path)
        v = ctypes.c_int()
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 5, 0) == 0:       # clock rate, kHz
            info["max_sclk_mhz"] = v.value // 1000
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 60, 0) == 0:      # memory clock, kHz
            info["max_mclk_mhz"] = v.value // 1000
    except Exception as e:  # pragma: no cover
        info["clock_error"] = str(e)
    try:
        import subprocess
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=20)
        info["rocm_smi_clocks"] = [ln.strip() for ln in r.stdout.splitlines()
                                   if "clk" in ln.lower() and "level" in ln.lower()][:6]
    except Exception as e:  # pragma: no cover
        info["rocm_smi_clocks"] = f"unavailable: {e}"
    return info


def copy_context(torch, prq, layers, M_list, reps=50):
    """Activation side, online copy (gather by perm, scale, quantize, copy the
    tail blocks) against offline copy (the expanded producer already emitted
    [Z~, Z~_tail]: a plain quantizer over K + k), and the offline copy's
    producer side from the expanded gate/up outputs: the fused SiLU(gate) * up
    quantization against torch's SiLU and product (bf16 Z) followed by the
    plain quantizer; all launched back to back on warm inputs (seconds per
    launch)."""
    out = {}
    for name, c in layers:
        K, k = c.K, c.k_tail
        art = prq.prq_prepare(c.W, c.Xcal, c.alpha, k)
        inv = torch.from_numpy(art["inv_scale_pos"]).cuda()
        perm = torch.from_numpy(art["perm"]).cuda()
        X = torch.from_numpy(c.X.view("int16")).cuda()
        g = torch.Generator(device="cpu").manual_seed(0)
        Zaug = (torch.randn((max(M_list), K + k), generator=g) * 2).to(torch.bfloat16).cuda()
        Gaug = (torch.randn((max(M_list), K + k), generator=g) * 4).to(torch.bfloat16).cuda()
        Uaug = torch.randn((max(M_list), K + k), generator=g).to(torch.bfloat16).cuda()
        Zb = torch.empty_like(Zaug)

        def swiglu_then(M, quant):
            torch.mul(torch.nn.functional.silu(Gaug[:M]), Uaug[:M], out=Zb[:M])
            quant(Zb[:M])
        for M in M_list:
            res = {}
            if M >= PACKED_MIN_ROWS:     # the quantizer the step uses: packed output
                A = prq.prq_quant_act_packed(X[:M], K, k, inv, perm)
                fns = (("online", lambda: prq.prq_quant_act_packed(X[:M], K, k, inv, perm, out=A)),
                       ("offline", lambda: prq.prq_quant_act_packed(Zaug[:M], K + k, 0, out=A)),
                       ("fused", lambda: prq.prq_swiglu_quant(Gaug[:M], Uaug[:M], K + k, packed=True,
                                                              out=A)),
                       ("unfused", lambda: swiglu_then(M, lambda Z: prq.prq_quant_act_packed(
                           Z, K + k, 0, out=A))))
            else:
                Aq = torch.empty((M, (K + k) // 2), dtype=torch.uint8, device="cuda")
                Asc = torch.empty((M, (K + k) // 32), dtype=torch.uint8, device="cuda")
                fns = (("online", lambda: prq.prq_quant_act(X[:M], K, k, inv, perm, Aq=Aq, Asc=Asc)),
                       ("offline", lambda: prq.prq_quant_act(Zaug[:M], K + k, 0, Aq=Aq, Asc=Asc)),
                       ("fused", lambda: prq.prq_swiglu_quant(Gaug[:M], Uaug[:M], K + k,
                                                              out=(Aq, Asc))),
                       ("unfused", lambda: swiglu_then(M, lambda Z: prq.prq_quant_act(
                           Z, K + k, 0, Aq=Aq, Asc=Asc))))
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
    M of one step, repeated until about `budget_s` seconds (the value, GB/s of
    the same algorithmic bytes as the GPU step); also the oracle's prepare
    (once), quant_act and gemm timed separately, and quant_act on one core."""
    from oracle import prquant as pq
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threadpool_limits, threads = None, 1
    name, c = layers[0]
    t0 = time.perf_counter()
    art = pq.prepare(c.W, c.Xcal, c.alpha, c.k_tail)
    t_prepare = time.perf_counter() - t0
    log(f"[bench] oracle prepare: {t_prepare:.1f} s")
    K, k, N = c.K, c.k_tail, c.N
    K_aug = K + k
    byts, reps, t_q, t_g = 0.0, 0, 0.0, 0.0
    t0 = time.perf_counter()
    while True:
        for M in M_list:
            ta = time.perf_counter()
            Aq, Asc = pq.quant_act(c.X[:M], art["inv_scale"], art["perm"], k)
            tb = time.perf_counter()
            pq.gemm(Aq, Asc, art["Wq"], art["Wsc"])
            t_q += tb - ta
            t_g += time.perf_counter() - tb
            byts += act_bytes(M, K, K_aug) + gemm_bytes(M, N, K_aug)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 50:
            break
    q1 = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            ta = time.perf_counter()
            for M in M_list:
                pq.quant_act(c.X[:M], art["inv_scale"], art["perm"], k)
            q1 = time.perf_counter() - ta
    return {"value": round(byts / el / 1e9, 4), "unit": "GB/s",
            "cores": int(max(threads, 1)), "kind": "oracle",
            "sample": f"{reps} passes of oracle act-quant + GEMM at M={list(M_list)} on {name} "
                      f"(N={N}, K={K}, k={k}); {el:.1f} s; host cores visible "
                      f"{len(os.sched_getaffinity(0))}, BLAS threads {threads}",
            "prepare_s": round(t_prepare, 2),
            "quant_act_s_per_pass": round(t_q / reps, 4),
            "gemm_s_per_pass": round(t_g / reps, 4),
            "quant_act_s_per_pass_1core": None if q1 is None else round(q1, 4)}


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


def lds_patterns(torch, blocks=1024, iters=2048):
    """One launch of each LDS read-pattern probe kernel (the tile GEMM's
    operand reads, its scale reads without and with the staging swap, one
    dword per bank, the quantizer's 2-byte gather): the same bank-conflict
    counters over them give reference points for the kernels' own ratios."""
    import ctypes
    from paper_2609_22106_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.prq_probe_lds_pattern.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_void_p, ctypes.c_void_p]
    lib.prq_probe_lds_pattern.restype = ctypes.c_int
    out = torch.zeros(blocks * 256, dtype=torch.int32, device="cuda")
    sp = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for mode in range(5):
        st = lib.prq_probe_lds_pattern(mode, blocks, iters, out.data_ptr(), sp)
        if st != 0:
            raise RuntimeError(f"prq_probe_lds_pattern({mode}) failed ({st})")
    torch.cuda.synchronize()
    log(f"[bench] LDS read patterns: 5 kernels x {blocks} workgroups x {iters} reads per wave")


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
    """Steps a --counters run executed: --warmup + --steps (bench.py defaults
    when absent)."""
    def opt(name, default):
        m = re.search(rf"--{name}\s+(\d+)", command)
        return int(m.group(1)) if m else default
    return opt("warmup", 10) + opt("steps", 50)


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
            t in n for t in ("gemm_decode_kernel", "gemm_decode_direct_kernel", "gemm_stream_kernel",
                             "gemm_streamk_kernel",
                             "gemm_tile_kernel", "gemm_grouped_persist_kernel",
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
WORKLOADS = ("decode", "prefill", "experts", "experts_prefill", "layers")


def build_workload(torch, np, prq, inputs, wl, rotate_bytes, plain=False, rowmajor=False):
    """(ops, dense layers or [], M list, config) of one workload."""
    if wl in ("decode", "prefill"):
        c = inputs.down_proj_decode() if wl == "decode" else inputs.down_proj_prefill()
        layers = [("qwen3_4b_down_proj", c)]
        M_list = list(c.M_list)
        ops = build_dense_ops(torch, prq, layers, M_list, rotate_bytes, plain=plain, rowmajor=rowmajor)
        config = {"workload": f"qwen3_4b_down_proj_{wl}", "N": 2560, "K": 9728, "k_tail": 256,
                  "alpha": 0.5, "M": M_list}
    elif wl in ("experts", "experts_prefill"):
        tokens = 64 if wl == "experts" else 4096
        ops = build_expert_ops(torch, np, prq, inputs, tokens, rotate_bytes)
        layers, M_list = [], []
        config = {"workload": f"qwen3_30b_a3b_expert_down_proj_{tokens}tok", "E": 128, "N": 2048,
                  "K": 768, "k_tail": 64, "alpha": 0.5, "topk": 8, "routed_rows": ops[0].M}
    else:
        layers = [(n, inputs.layer_case(n)) for n, _, _ in inputs.LAYER_SET]
        M_list = [4096]
        ops = build_dense_ops(torch, prq, layers, M_list, rotate_bytes, plain=plain)
        config = {"workload": "qwen3_4b_decoder_linears_prefill", "M": 4096,
                  "layers": {n: {"N": c.N, "K": c.K, "k_tail": c.k_tail} for n, c in layers}}
    return ops, layers, M_list, config


def op_detail(op):
    tg, ta = op.t_gemm, op.t_act
    return {"gemm_us": round(tg * 1e6, 3), "act_quant_us": round(ta * 1e6, 3),
            "op_us": round((tg + ta) * 1e6, 3),
            "gemm_GBs": round(op.gemm_bytes / tg / 1e9, 1),
            "gemm_TFLOPs": round(op.flops / tg / 1e12, 2),
            "gemm_hbm_frac": round(op.gemm_bytes / tg / 1e9 / HBM_PEAK_GBS, 4),
            "gemm_mfma_frac": round(op.flops / tg / 1e12 / MXFP4_PEAK_TFLOPS, 4),
            "act_quant_GBs": round(op.act_bytes / ta / 1e9, 1),
            "act_quant_hbm_frac": round(op.act_bytes / ta / 1e9 / HBM_PEAK_GBS, 4)}


def gemm_roofline(ops, wl):
    """Roofline of the workload's dominant kernel, the GEMM: algorithmic bytes
    (or FLOPs) of its launches over their summed launch durations; the bound
    follows the GEMM's own arithmetic intensity against the ridge."""
    g_bytes = sum(op.gemm_bytes for op in ops)
    g_flops = sum(op.flops for op in ops)
    g_time = sum(op.t_gemm for op in ops)
    bound = "mfma" if g_flops / max(g_bytes, 1) > MXFP4_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"
    if bound == "hbm":
        achieved, peak, unit = g_bytes / g_time / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = g_flops / g_time / 1e12, MXFP4_PEAK_TFLOPS, "TFLOP/s"
    traffic = traffic_record(wl)
    return {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic,
            "traffic_over_algorithmic": None if traffic is None else round(traffic / (g_bytes / len(ops)), 3),
            "kernel": "prq_gemm (augmented MXFP4 GEMM over K+k)",
            "per_launch_bytes": round(g_bytes / len(ops), 1),
            "per_launch_flops": round(g_flops / len(ops), 1),
            "avg_launch_us": round(g_time / len(ops) * 1e6, 3)}


def measure_workload(torch, np, prq, inputs, wl, args, stream, contexts=True):
    """Everything measured for one workload: per-kernel launch durations, step
    time (median of graph replays), GEMM roofline and the context timings."""
    ops, layers, M_list, config = build_workload(torch, np, prq, inputs, wl, args.rotate_bytes)
    reps = max(args.steps, 20)
    time_kernels(torch, ops, reps, args.warmup, stream)
    if args.no_graph:
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step_once(ops)
        torch.cuda.synchronize()
        steps_gpu, walls = [(time.perf_counter() - t0) / args.steps], [time.perf_counter() - t0]
    else:
        steps_gpu, walls = graph_step_times(torch, ops, args.steps)
    t_step = float(np.median(steps_gpu))
    step_bytes = sum(op.gemm_bytes + op.act_bytes for op in ops)
    step_flops = sum(op.flops for op in ops)
    detail = {op.name: op_detail(op) for op in ops}
    out = {"config": config, "t_step": t_step, "steps_gpu": steps_gpu, "walls": walls,
           "value": step_bytes / t_step / 1e9, "tflops": step_flops / t_step / 1e12,
           "roofline": gemm_roofline(ops, wl), "detail": detail, "M_list": M_list,
           "layers": layers}
    if contexts and wl == "decode":
        t_floor, nbytes = read_floor(torch, prq, ops[0].weights)
        out["read_floor"] = {"us": round(t_floor * 1e6, 3), "bytes": nbytes,
                             "GBs": round(nbytes / t_floor / 1e9, 1),
                             "hbm_frac": round(nbytes / t_floor / 1e9 / HBM_PEAK_GBS, 4)}
    if contexts and layers and not args.no_bf16:
        for key, t in bf16_context(torch, layers, M_list, args.rotate_bytes, args.steps).items():
            if key in detail:
                d = detail[key]
                d["bf16_matmul_us"] = round(t * 1e6, 3)
                d["speedup_op_vs_bf16"] = round(t / (d["op_us"] * 1e-6), 3)
                d["speedup_gemm_vs_bf16"] = round(t / (d["gemm_us"] * 1e-6), 3)
    if contexts and layers and not args.no_plain and wl in ("decode", "prefill"):
        # plain MXFP4 (k = 0, no scaling) through the same kernels and timing
        plain_ops, _, _, _ = build_workload(torch, np, prq, inputs, wl, args.rotate_bytes, plain=True)
        time_kernels(torch, plain_ops, reps, args.warmup, stream)
        for op in plain_ops:
            if op.name in detail:
                d = detail[op.name]
                d["plain_mxfp4_gemm_us"] = round(op.t_gemm * 1e6, 3)
                d["plain_mxfp4_op_us"] = round((op.t_gemm + op.t_act) * 1e6, 3)
                d["op_over_plain_mxfp4"] = round(d["op_us"] / ((op.t_gemm + op.t_act) * 1e6), 3)
        del plain_ops
    if contexts and layers and wl == "decode":
        # the row-major pair (prq_quant_act + prq_gemm) at every M, same timing
        rm_ops, _, _, _ = build_workload(torch, np, prq, inputs, wl, args.rotate_bytes, rowmajor=True)
        time_kernels(torch, rm_ops, reps, args.warmup, stream)
        for op in rm_ops:
            if op.name in detail:
                d = detail[op.name]
                d["rowmajor_gemm_us"] = round(op.t_gemm * 1e6, 3)
                d["rowmajor_act_quant_us"] = round(op.t_act * 1e6, 3)
                d["rowmajor_op_us"] = round((op.t_gemm + op.t_act) * 1e6, 3)
        del rm_ops
    if contexts and layers and wl in ("decode", "prefill"):
        for key, r in copy_context(torch, prq, layers, M_list).items():
            if key in detail:
                detail[key]["act_quant_online_copy_warm_us"] = round(r["online"] * 1e6, 3)
                detail[key]["act_quant_offline_copy_warm_us"] = round(r["offline"] * 1e6, 3)
                detail[key]["producer_swiglu_quant_fused_warm_us"] = round(r["fused"] * 1e6, 3)
                detail[key]["producer_swiglu_then_quant_warm_us"] = round(r["unfused"] * 1e6, 3)
    if contexts and wl == "decode" and not args.no_graph:
        # hot: the same steps on one weight copy (served from the Infinity Cache)
        hot_ops, _, _, _ = build_workload(torch, np, prq, inputs, wl, 0)
        hot, _ = graph_step_times(torch, hot_ops, args.steps)
        out["hot_ms_per_step"] = round(float(np.median(hot)) * 1e3, 5)
        del hot_ops
    del ops
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


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
    if args.lds_patterns:
        lds_patterns(torch)
        if not args.counters:
            print(json.dumps({"lds_patterns_run": 5}), flush=True)
            return 0
    if args.counters:
        wl = "decode" if args.workload == "all" else args.workload
        if args.copy_calibration:
            copy_calibration(torch)
        ops, _, _, config = build_workload(torch, np, prq, inputs, wl, args.rotate_bytes)
        for _ in range(args.warmup + args.steps):
            step_once(ops)
        torch.cuda.synchronize()
        print(json.dumps({"counters_run": config["workload"], "steps": args.warmup + args.steps,
                          "gemm_calls": (args.warmup + args.steps) * len(ops)}), flush=True)
        return 0
    head_wl = "decode" if args.workload == "all" else args.workload
    others = [w for w in WORKLOADS if w != head_wl] if args.workload == "all" else []
    info = gpu_info(torch)
    if args.copy_calibration:
        copy_calibration(torch)
    res = measure_workload(torch, np, prq, inputs, head_wl, args, stream)
    log(f"[bench] {head_wl}: {res['t_step'] * 1e3:.4f} ms per step")
    detail = dict(res["detail"])
    workloads = {}
    for wl in others:
        r = measure_workload(torch, np, prq, inputs, wl, args, stream)
        log(f"[bench] {wl}: {r['t_step'] * 1e3:.4f} ms per step")
        for key, d in r["detail"].items():
            detail[f"layers/{key}" if wl == "layers" else key] = d
        workloads[r["config"]["workload"]] = {
            "ms_per_step": round(r["t_step"] * 1e3, 5), "value_GBs": round(r["value"], 2),
            "tflops": round(r["tflops"], 3), "roofline": r["roofline"], "config": r["config"]}

    cpu = None
    if not args.no_cpu_baseline and head_wl == "decode":
        cpu = cpu_baseline(np, res["layers"], res["M_list"])

    line = {
        "metric": METRIC, "value": round(res["value"], 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(res["t_step"] * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "mxfp4", "data": "synthetic", "config": res["config"],
        "tflops": round(res["tflops"], 3),
        "roofline": res["roofline"], "cpu_baseline": cpu, "detail": detail,
        "workloads": workloads,
        "context": {k: res[k] for k in ("read_floor", "hot_ms_per_step") if k in res},
        "gpu": info,
        "timing": {
            "method": ("eager: the steps launched directly" if args.no_graph else
                       f"{args.steps} steps in one HIP graph, replayed once untimed and then 5 "
                       "times, each between torch.cuda.synchronize() calls with HIP events "
                       "around the replay; ms_per_step = median replay / steps"),
            "replay_ms_per_step": [round(t * 1e3, 5) for t in res["steps_gpu"]],
            "replay_wall_s": [round(t, 6) for t in res["walls"]],
            "kernel_method": f"per op, {max(args.steps, 20)} back-to-back launches of the "
                             "quantizer and then of the GEMM (rotated weights), queued behind a GPU "
                             "spin-sleep, fence-free HIP events around each batch"},
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

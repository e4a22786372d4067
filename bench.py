"""Benchmark one pass of the MoE-layer hot path on one MI355X.

A step is route -> plan -> forward -> backward (training workload) over one
batch of seeded synthetic input already resident in HBM.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Throughput follows the paper's accounting (§4.1): forward FLOPs
6*T*(k*f + f_shared)*d, backward twice that.  Per-stage times come from HIP
events the library records on the stream the kernels run on.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE layer fwd+bwd TFLOP/s and tokens/s on 1 MI355X; % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, AMD's published figure (2.4 GHz)
PEAK_BF16_TFLOPS_ALT = 2300.0  # the ~2.3 PFLOP/s dense bf16 figure the benchmark spec quotes
PEAK_HBM_GBS = 8000.0
# configurations measured forward-only beside the training step (the paper
# benchmarks its layer at several shapes, §4.1)
FORWARD_CONFIGS = ("tiny", "many_experts", "hot_expert", "large_shared")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """Minimal hipEvent API through ctypes (the library records them itself)."""

    def __init__(self):
        self.h = ctypes.CDLL("libamdhip64.so")
        self.h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                               ctypes.c_void_p]
        self.h.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        assert self.h.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def record(self, e, stream):
        assert self.h.hipEventRecord(e, stream) == 0

    def ms(self, a, b):
        out = ctypes.c_float()
        assert self.h.hipEventElapsedTime(ctypes.byref(out), a, b) == 0
        return out.value

    def sync(self, e):
        assert self.h.hipEventSynchronize(e) == 0

    def destroy(self, e):
        self.h.hipEventDestroy(e)


def dense_routing(w):
    """Every token routes to every local expert (k == E): the library folds
    the combine into the down GEMM (its stage "down_routed" then also holds
    the shared down product, and "down_shared" and "combine" are empty) and
    the reverse combine into one dX GEMM over every expert, the shared expert
    and the router term (stage "dx_shared"; "dx_routed" and
    "reverse_combine" are empty)."""
    return w.k == w.E


def stage_flops(w):
    """Algorithmic FLOPs of each timed stage and launches per stage."""
    R, d, f, fs, T = w.T * w.k, w.d, w.f, w.f_s, w.T
    fwd = {"up_routed": (4.0 * R * d * f, 1), "up_shared": (4.0 * T * d * fs, 1),
           "down_routed": (2.0 * R * f * d, 1), "down_shared": (2.0 * T * fs * d, 1)}
    bwd = {"dgrad_routed": (2.0 * R * d * f, 1), "dx_routed": (4.0 * R * f * d, 1),
           "wgrad_gate_up": (4.0 * R * d * f, 2), "wgrad_down": (2.0 * R * f * d, 1),
           "dgrad_shared": (2.0 * T * d * fs, 1), "dx_shared": (4.0 * T * fs * d, 1),
           "wgrad_shared": (6.0 * T * d * fs, 3)}
    if dense_routing(w):
        fwd["down_routed"] = (2.0 * (R * f + T * fs) * d, 1)
        fwd["down_shared"] = (0.0, 0)
        bwd["dx_shared"] = (4.0 * (R * f + T * fs) * d, 1)
        bwd["dx_routed"] = (0.0, 0)
    return fwd, bwd


# sources the BF16 GEMM kernels are compiled from (device code and helpers)
GEMM_SOURCES = ("gemm.hip", "common.h")


def source_sha256():
    """Hash of the BF16 GEMM kernel sources: a traffic record taken on other
    sources does not describe the kernel being timed."""
    import hashlib
    h = hashlib.sha256()
    for name in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_36070_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch recorded under profiles/ for this kernel and workload.

    Returns None unless the record was taken on the current kernel sources
    (same hash of the BF16 GEMM sources): counters of an older kernel say nothing
    about this one.
    """
    import glob
    for path in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json")):
        with open(path) as fh:
            rec = json.load(fh)
        if rec.get("kernel") == kernel and rec.get("workload") == workload \
                and rec.get("source_sha256") == source_sha256():
            return rec["read_bytes_per_launch"] + rec["write_bytes_per_launch"]
    return None


def schedule_timing(H, stream, reps=20):
    """Multi-rank dispatch schedule (moe_schedule) on each synthetic route table,
    built for rank 0 (which owns the hot expert where there is one); GPU time
    per call from a graph of back-to-back calls."""
    import torch
    from paper_2609_36070_amd import binding as B
    from paper_2609_36070_amd.workloads import ROUTE_TABLES, make_route_table
    res = {}
    for name, t in ROUTE_TABLES.items():
        A = torch.from_numpy(make_route_table(t, seed=0)).cuda()
        R, NK, L = t.R, t.NK, t.L
        M = torch.empty(R * L, dtype=torch.int32, device="cuda")
        S = torch.empty(L + 1, dtype=torch.int32, device="cuda")
        phi = torch.empty((R * NK, 2), dtype=torch.int32, device="cuda")
        ws = torch.empty(B.moe_schedule_workspace_bytes(R, NK, L), dtype=torch.uint8, device="cuda")
        for _ in range(3):
            B.moe_schedule(R, NK, L, 0, A, M, S, phi, R * NK, ws)
        torch.cuda.synchronize()
        # reps calls captured in one HIP graph, so host launch cost is not timed
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(reps):
                B.moe_schedule(R, NK, L, 0, A, M, S, phi, R * NK, ws)
        graph.replay()
        torch.cuda.synchronize()
        a, b = H.create(), H.create()
        H.record(a, stream)
        graph.replay()
        H.record(b, stream)
        H.sync(b)
        us = 1e3 * H.ms(a, b) / reps
        P = int(S[L].item())
        nbytes = 2 * 4 * R * NK + 8 * P + 4 * R * L      # A read twice, schedule rows, M
        res[name] = {"R": R, "N": t.N, "K": t.K, "L": L, "rank": 0, "routes_received": P,
                     "us": round(us, 2), "GB/s": round(nbytes / (us * 1e-6) / 1e9, 1)}
        H.destroy(a)
        H.destroy(b)
        del A, phi, ws
    return res


def mx_forward_timing(H, stream, inputs, steps, warmup):
    """route + plan + moe_forward_mx on the forward layer of the benchmark
    workload (routed experts in MXFP8, shared expert BF16), with per-stage
    events; the routed weights are pre-quantised once, outside the timing."""
    import torch
    from paper_2609_36070_amd import binding as B
    from paper_2609_36070_amd.layer import DeviceLayer
    from paper_2609_36070_amd.workloads import WORKLOADS
    w = WORKLOADS["large_shared"]
    L = DeviceLayer(w, inputs, with_backward=False, mx=True)
    for _ in range(warmup):
        L.step_mx()
    torch.cuda.synchronize()
    nf = len(B.FWD_STAGES) + 1
    per = []
    a, b = H.create(), H.create()
    H.record(a, stream)
    for _ in range(steps):
        ev = [H.create() for _ in range(nf)]
        fe = B.MoeStageEvents()
        for i, e in enumerate(ev):
            fe.ev[i] = e
        start = H.create()
        H.record(start, stream)
        L.route()
        L.plan()
        L.forward_mx(events=fe)
        per.append((start, ev))
    H.record(b, stream)
    H.sync(b)
    ms = H.ms(a, b) / steps
    fwd_fl, _ = stage_flops(w)
    stages = {}
    for start, ev in per:
        stages["route+plan"] = stages.get("route+plan", 0.0) + H.ms(start, ev[0])
        for i, name in enumerate(B.FWD_STAGES):
            stages[name] = stages.get(name, 0.0) + H.ms(ev[i], ev[i + 1])
    out = {"workload": w.name, "ms_per_step": round(ms, 4),
           "tflops": round(w.fwd_flops() / (ms * 1e-3) / 1e12, 2), "stages": {}}
    for name, t in stages.items():
        t /= steps
        out["stages"][name] = {"ms": round(t, 4)}
        if name in fwd_fl:
            out["stages"][name]["tflops"] = round(fwd_fl[name][0] / (t * 1e-3) / 1e12, 1)
    del L
    torch.cuda.synchronize()
    return out


def mx_training_timing(H, stream, inputs, steps, warmup):
    """route + plan + moe_forward_mx (pre-activations kept) + moe_backward_mx
    on the training workload, with the weight gradients in BF16 and, on the
    same layer, in MXFP8 (wgrad_mxfp8), in alternating blocks of `steps`
    steps; the routed weights are pre-quantised once (both layouts), outside
    the step, and that requantisation is timed on its own."""
    import torch
    from paper_2609_36070_amd.layer import DeviceLayer
    from paper_2609_36070_amd.workloads import WORKLOADS
    w = WORKLOADS["large_shared_train"]
    L = DeviceLayer(w, inputs, mx=True, mx_wgrad=True)
    for wg in (False, True):
        L.mx_wgrad = wg
        for _ in range(warmup):
            L.step_mx()
    torch.cuda.synchronize()
    a, m, b = H.create(), H.create(), H.create()
    tot = {False: [0.0, 0.0, 0], True: [0.0, 0.0, 0]}
    for wg in (False, True, False, True):
        L.mx_wgrad = wg
        for _ in range(steps):
            H.record(a, stream)
            L.route()
            L.plan()
            L.forward_mx()
            H.record(m, stream)
            L.backward_mx()
            H.record(b, stream)
            H.sync(b)
            tot[wg][0] += H.ms(a, m)
            tot[wg][1] += H.ms(m, b)
            tot[wg][2] += 1
    # both MXFP8 layouts of the routed weights, remade after every weight update
    H.record(a, stream)
    for _ in range(steps):
        L.quantize_mx()
    H.record(b, stream)
    H.sync(b)
    wq = H.ms(a, b) / steps
    for e in (a, m, b):
        H.destroy(e)
    flops = w.fwd_flops() + w.bwd_flops()

    def entry(wg):
        fwd, bwd, n = tot[wg]
        fwd, bwd = fwd / n, bwd / n
        return {"forward_ms": round(fwd, 4), "backward_ms": round(bwd, 4),
                "ms_per_step": round(fwd + bwd, 4),
                "tflops": round(flops / ((fwd + bwd) * 1e-3) / 1e12, 2)}
    out = {"workload": w.name, **entry(False), "wgrad_mxfp8": entry(True),
           "weight_quant_ms": round(wq, 4), "error_word": L.error_word()}
    del L
    torch.cuda.synchronize()
    return out


def fused_forward_timing(H, stream, L, steps):
    """route + plan + forward with the separate launches against the same with
    the fused persistent forward, on the benchmark layer (A and B saved when
    it trains), in two alternating blocks of `steps` steps."""
    import torch

    def block(fused):
        a, b = H.create(), H.create()
        H.record(a, stream)
        for _ in range(steps):
            L.route()
            L.plan()
            if fused:
                L.forward_fused()
            else:
                L.forward()
        H.record(b, stream)
        H.sync(b)
        ms = H.ms(a, b) / steps
        H.destroy(a)
        H.destroy(b)
        return ms

    block(True)                      # warm-up of the fused launch
    torch.cuda.synchronize()
    res = {"separate": 0.0, "fused": 0.0}
    for _ in range(2):
        res["separate"] += block(False) / 2
        res["fused"] += block(True) / 2
    err = L.error_word()
    return {"separate_ms": round(res["separate"], 4), "fused_ms": round(res["fused"], 4),
            "speedup": round(res["separate"] / res["fused"], 4), "error_word": err}


def ring_timing(H, stream, w, inputs, L_full, steps, warmup):
    """Bounded-memory execution against the one-pass path on the benchmark
    workload: a ring holding half of the routed rows (the comparison the
    paper makes for its macrobatch ring) versus buffers for every route.
    Both are timed in two alternating blocks of `steps` whole steps; the
    forward (route + plan + forward) and backward parts are timed apart."""
    import torch
    from paper_2609_36070_amd.layer import DeviceLayer
    R = w.T * w.k
    ring_rows = R // 2
    L_ring = DeviceLayer(w, inputs, ring_rows=ring_rows)
    for _ in range(warmup):
        L_ring.step()
    torch.cuda.synchronize()

    def block(L):
        marks = [(H.create(), H.create(), H.create()) for _ in range(steps)]
        for a, m, b in marks:
            H.record(a, stream)
            L.route()
            L.plan()
            L.forward()
            H.record(m, stream)
            if w.backward:
                L.backward()
            H.record(b, stream)
        H.sync(marks[-1][2])
        f = sum(H.ms(a, m) for a, m, _ in marks) / steps
        bw = sum(H.ms(m, b) for _, m, b in marks) / steps
        for e in marks:
            for x in e:
                H.destroy(x)
        return f, bw

    res = {"full": [0.0, 0.0], "ring": [0.0, 0.0]}
    for _ in range(2):
        for name, L in (("full", L_full), ("ring", L_ring)):
            f, bw = block(L)
            res[name][0] += f / 2
            res[name][1] += bw / 2
    full_ms, ring_ms = sum(res["full"]), sum(res["ring"])
    out = {"ring_rows": ring_rows, "routes": R, "windows": -(-R // ring_rows),
           "workspace_gib_full": round(L_full.ws.numel() / 2 ** 30, 3),
           "workspace_gib_ring": round(L_ring.ws.numel() / 2 ** 30, 3),
           "full_ms": {"forward": round(res["full"][0], 4), "backward": round(res["full"][1], 4),
                       "step": round(full_ms, 4)},
           "ring_ms": {"forward": round(res["ring"][0], 4), "backward": round(res["ring"][1], 4),
                       "step": round(ring_ms, 4)},
           "overhead_pct": {"forward": round(100 * (res["ring"][0] / res["full"][0] - 1), 2),
                            "step": round(100 * (ring_ms / full_ms - 1), 2)}}
    if w.backward:
        out["overhead_pct"]["backward"] = round(100 * (res["ring"][1] / res["full"][1] - 1), 2)
    del L_ring
    torch.cuda.synchronize()
    return out


def hbm_bytes(w):
    """Algorithmic HBM bytes per launch of the memory-bound kernels (each
    tensor read or written once)."""
    T, d, E, k, R = w.T, w.d, w.E, w.k, w.T * w.k
    sh = 1 if w.f_s else 0
    out = {
        # X, W_r read; logits, top-k ids and weights written
        "route": 2 * T * d + 2 * d * E + 4 * T * E + 8 * T * k,
        # Yexp rows, Ysh read; Y written; route positions and weights read
        "combine": 2 * R * d + 2 * T * d * sh + 2 * T * d + 8 * R,
    }
    if w.backward:
        # dXperm rows, dXsh, dZ, W_r read; dX written; route positions read
        out["reverse_combine"] = 2 * R * d + 2 * T * d * sh + 4 * T * E + 2 * d * E + 2 * T * d + 4 * R
        # X and dZ read, dW_r written
        out["dw_router"] = 2 * T * d + 4 * T * E + 4 * d * E
    return out


STEP_OUTPUTS = ("logits", "topk_idx", "topk_w", "counts", "offsets", "perm", "route_pos", "Y", "dX",
                "dZ", "dW_r", "dW_gate", "dW_up", "dW_down", "dWg_s", "dWu_s", "dWd_s")


def determinism_check(L, reps=2):
    """Every output of the step (routing, plan, Y, and with a backward dX
    and every gradient) after `reps` more whole steps on the same inputs,
    compared bitwise with its value after the timed steps."""
    import torch
    torch.cuda.synchronize()
    first = {n: getattr(L, n).clone() for n in STEP_OUTPUTS if getattr(L, n, None) is not None}
    differ = set()
    for _ in range(reps):
        L.step()
        torch.cuda.synchronize()
        differ |= {n for n, t in first.items() if not torch.equal(getattr(L, n), t)}
    return {"runs": reps + 1, "bitwise_identical": not differ, "outputs": len(first),
            "differing": sorted(differ)}


def copy_ceiling(H, stream, mib=2048, reps=5):
    """The practical HBM ceiling of this GPU (bytes read + bytes written per
    second) from two plain streaming kernels over `mib` MiB of fp32: torch's
    device-to-device copy and an elementwise kernel (`dst = src * 1`).  Each
    runs `reps` times back to back between one pair of events, so the GPU
    stays busy and no host-side launch latency enters the time; the faster of
    the two is the ceiling."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    nbytes = 2 * mib * (1 << 20)
    out = {"bytes": nbytes}
    for name, fn in (("copy", lambda: dst.copy_(src)),
                     ("elementwise", lambda: torch.mul(src, 1.0, out=dst))):
        fn()
        torch.cuda.synchronize()
        a, b = H.create(), H.create()
        H.record(a, stream)
        for _ in range(reps):
            fn()
        H.record(b, stream)
        H.sync(b)
        ms = H.ms(a, b) / reps
        H.destroy(a)
        H.destroy(b)
        out[name] = {"ms": round(ms, 4), "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1)}
    del src, dst
    torch.cuda.synchronize()
    best = max(("copy", "elementwise"), key=lambda k: out[k]["GB/s"])
    out.update({"kernel": best, "ms": out[best]["ms"], "GB/s": out[best]["GB/s"]})
    return out


def route_time(H, stream, L, reps=20):
    """moe_route alone, `reps` calls back to back between one pair of events
    (a lone call between events is padded by the events' own gaps)."""
    a, b = H.create(), H.create()
    L.route()
    H.record(a, stream)
    for _ in range(reps):
        L.route()
    H.record(b, stream)
    H.sync(b)
    ms = H.ms(a, b) / reps
    H.destroy(a)
    H.destroy(b)
    return ms


def hbm_report(w, stages, copy_gbs):
    """GB/s of the memory-bound kernels from their stage times."""
    names = {"route": "route", "combine": "fwd.combine", "reverse_combine": "bwd.reverse_combine",
             "dw_router": "bwd.dw_router"}
    out = {}
    folded = ("combine", "reverse_combine") if dense_routing(w) else ()
    for k, nb in hbm_bytes(w).items():
        ms = stages.get(names[k])
        if not ms or k in folded:       # dense routing folds the combines into GEMMs
            continue
        gbs = nb / (ms * 1e-3) / 1e9
        out[k] = {"bytes": nb, "ms": round(ms, 4), "GB/s": round(gbs, 1),
                  "frac_of_8TBs": round(gbs / PEAK_HBM_GBS, 3),
                  "frac_of_copy": round(gbs / copy_gbs, 3) if copy_gbs else None}
    if "plan" in stages:
        out["plan"] = {"us": round(1e3 * stages["plan"], 2), "bound": "latency"}
    return out


def expert_roofline_ms(w, counts):
    """Sum over experts of max(FLOPs / peak, bytes / HBM) for the routed
    up/gate and down GEMMs of a forward: FLOPs 6 M_e d f; bytes the expert's
    three bf16 weight matrices plus its rows (X read, H written and read,
    Yexp written).  Small experts are bound by reading their weights."""
    d, f = w.d, w.f
    t = 0.0
    for m in counts:
        m = int(m)
        if m == 0:
            continue
        fl = 6.0 * m * d * f
        by = 6.0 * d * f + m * (2.0 * d + 4.0 * f + 2.0 * d)
        t += max(fl / (PEAK_BF16_TFLOPS * 1e12), by / (PEAK_HBM_GBS * 1e9))
    return 1e3 * t


def forward_config_timing(H, stream, name, steps, warmup, copy_gbs, inputs=None):
    """route + plan + forward of one forward configuration: per-stage times
    (from steps with events at every stage boundary), then `steps` timed
    passes with events only around each pass; median and mean."""
    import numpy as np
    import torch
    from paper_2609_36070_amd import binding as B
    from paper_2609_36070_amd.layer import DeviceLayer
    from paper_2609_36070_amd.workloads import WORKLOADS, make_inputs
    w = WORKLOADS[name]
    if inputs is None:
        inputs = make_inputs(w, seed=0)
    L = DeviceLayer(w, inputs, with_backward=False)
    for _ in range(warmup):
        L.route()
        L.plan()
        L.forward()
    torch.cuda.synchronize()
    nf = len(B.FWD_STAGES) + 1
    stages = {}
    route_ms = route_time(H, stream, L)
    nstage = 3
    for _ in range(nstage):
        e0, e1 = H.create(), H.create()
        ev = [H.create() for _ in range(nf)]
        fe = B.MoeStageEvents()
        for i, e in enumerate(ev):
            fe.ev[i] = e
        H.record(e0, stream)
        L.route()
        H.record(e1, stream)
        L.plan()
        L.forward(events=fe)
        H.sync(ev[-1])
        stages["route"] = stages.get("route", 0.0) + H.ms(e0, e1) / nstage
        stages["plan"] = stages.get("plan", 0.0) + H.ms(e1, ev[0]) / nstage
        for i, st in enumerate(B.FWD_STAGES):
            stages["fwd." + st] = stages.get("fwd." + st, 0.0) + H.ms(ev[i], ev[i + 1]) / nstage
        for e in [e0, e1] + ev:
            H.destroy(e)
    marks = [(H.create(), H.create()) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in marks:
        H.record(a, stream)
        L.route()
        L.plan()
        L.forward()
        H.record(b, stream)
    H.sync(marks[-1][1])
    times = sorted(H.ms(a, b) for a, b in marks)
    for a, b in marks:
        H.destroy(a)
        H.destroy(b)
    med = times[len(times) // 2]
    mean = sum(times) / len(times)
    fl = w.fwd_flops()
    fwd_fl, _ = stage_flops(w)
    counts = L.counts.cpu().numpy()
    out = {"workload": name, "T": w.T, "d": w.d, "E": w.E, "k": w.k, "f": w.f, "f_shared": w.f_s,
           "passes": "fwd", "step": "route+plan+forward", "steps": steps,
           "ms_median": round(med, 4), "ms_mean": round(mean, 4),
           "tflops": round(fl / (med * 1e-3) / 1e12, 2),
           "tokens_per_s": round(w.T / (med * 1e-3), 1),
           "frac_of_bf16_peak": round(fl / (med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "frac_of_2300": round(fl / (med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS_ALT, 4),
           "expert_load": {"min": int(counts.min()), "mean": round(float(counts.mean()), 1),
                           "max": int(counts.max())},
           "stages": {}}
    for st, ms in stages.items():
        out["stages"][st] = {"ms": round(ms, 4)}
        key = st.split(".", 1)[-1]
        if st.startswith("fwd.") and key in fwd_fl and ms > 0 and fwd_fl[key][0] > 0:
            out["stages"][st]["tflops"] = round(fwd_fl[key][0] / (ms * 1e-3) / 1e12, 1)
    # routed expert GEMMs (with dense routing the folded down GEMM also holds
    # the shared expert's down product: its share of the time is left in)
    gemm_ms = sum(stages.get("fwd." + k, 0.0) for k in ("up_routed", "down_routed"))
    roof = expert_roofline_ms(w, counts)
    out["routed_expert_gemms"] = {"ms": round(gemm_ms, 4), "roofline_ms": round(roof, 4),
                                  "frac_of_roofline": round(roof / gemm_ms, 4) if gemm_ms else None}
    out["hbm"] = hbm_report(w, dict(stages, route=route_ms), copy_gbs)
    del L
    torch.cuda.synchronize()
    return out


def graph_step_timing(H, stream, L, reps):
    """The whole step captured in one HIP graph and replayed `reps` times,
    with an event pair around each replay; median and mean of the replays."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        L.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.step()
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    marks = [(H.create(), H.create()) for _ in range(reps)]
    for a, b in marks:
        H.record(a, stream)
        graph.replay()
        H.record(b, stream)
    H.sync(marks[-1][1])
    times = sorted(H.ms(a, b) for a, b in marks)
    for a, b in marks:
        H.destroy(a)
        H.destroy(b)
    del graph
    torch.cuda.synchronize()
    return {"replays": reps, "ms_median": round(times[len(times) // 2], 4),
            "ms_mean": round(sum(times) / len(times), 4), "ms_min": round(times[0], 4)}


def host_info():
    """CPU model, usable cores and the BLAS numpy calls into."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = f"{i.get('internal_api')} {i.get('version')} ({i.get('num_threads')} threads)"
                break
    except Exception:  # pragma: no cover
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0)), "blas": blas}


def cpu_baseline(w, inputs, sample_tokens):
    """Time the CPU oracle on the first `sample_tokens` tokens of the workload."""
    import numpy as np
    from oracle import moe_oracle as O
    info = host_info()
    cores = info["affinity_cores"]
    try:
        from threadpoolctl import threadpool_info
        used = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        if used:
            cores = min(cores, max(used))   # the BLAS threads the oracle's products ran on
    except Exception:  # pragma: no cover
        pass
    n = min(sample_tokens, w.T)
    X = inputs["X"][:n]
    W = {key: inputs.get(key) for key in ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")}
    t0 = time.perf_counter()
    Z = O.router_logits(X, inputs["W_r"], inputs.get("bias"))
    idx = O.topk_select(Z, w.k)
    wts = O.gate_weights(Z, idx)
    O.plan(idx, w.E)
    O.moe_forward(X, W, idx, wts)
    flops = w.scaled(T=n).fwd_flops()
    if w.backward:
        O.moe_backward(X, inputs["W_r"], W, idx, wts, inputs["dY"][:n])
        flops += w.scaled(T=n).bwd_flops()
    dt = time.perf_counter() - t0
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {n} of {w.T} tokens, all {w.k} routes each, full weights; "
                      f"route+plan+forward{'+backward' if w.backward else ''} in fp64 numpy; "
                      f"{dt:.1f} s",
            "seconds": round(dt, 2), "tokens_per_s": round(n / dt, 1), **info}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large_shared_train")
    ap.add_argument("--cpu-sample-tokens", type=int, default=4096)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-schedule", action="store_true",
                    help="skip timing the multi-rank dispatch schedule")
    ap.add_argument("--no-mx", action="store_true", help="skip timing the MXFP8 forward")
    ap.add_argument("--no-ring", action="store_true",
                    help="skip the bounded-memory (half-capacity ring) comparison")
    ap.add_argument("--no-fused", action="store_true",
                    help="skip timing the fused persistent forward")
    ap.add_argument("--ring-only", type=int, default=0, metavar="ROWS",
                    help="time only steps in bounded-memory execution with a ring of ROWS rows "
                         "(for kernel traces of that mode); prints its own JSON line")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the forward-only configurations measured beside the step")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (the reference "
                         "kernel for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the layer only (got --gpus {args.gpus}); "
              f"there is no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_36070_amd import binding as B
    from paper_2609_36070_amd.layer import DeviceLayer
    from paper_2609_36070_amd.workloads import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    log(f"[bench] workload {w.name}: T={w.T} d={w.d} E={w.E} k={w.k} f={w.f} f_s={w.f_s} "
        f"backward={w.backward}")
    t_in = time.perf_counter()
    inputs = make_inputs(w, seed=0)
    log(f"[bench] inputs drawn in {time.perf_counter() - t_in:.1f} s")
    stream = torch.cuda.current_stream().cuda_stream
    H = HipEvents()
    if args.ring_only:
        L = DeviceLayer(w, inputs, ring_rows=args.ring_only)
        for _ in range(args.warmup):
            L.step()
        torch.cuda.synchronize()
        a, b = H.create(), H.create()
        H.record(a, stream)
        for _ in range(args.steps):
            L.step()
        H.record(b, stream)
        H.sync(b)
        ms = H.ms(a, b) / args.steps
        step_flops = w.fwd_flops() + (w.bwd_flops() if w.backward else 0.0)
        print(json.dumps({"mode": "bounded_memory", "workload": w.name,
                          "ring_rows": args.ring_only, "steps": args.steps,
                          "ms_per_step": round(ms, 4),
                          "tflops": round(step_flops / (ms * 1e-3) / 1e12, 2),
                          "workspace_gib": round(L.ws.numel() / 2 ** 30, 3)}), flush=True)
        return
    L = DeviceLayer(w, inputs)

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calibrate_copy_mib} MiB done")
        del src, dst

    for i in range(args.warmup):
        L.step()
    torch.cuda.synchronize()
    log(f"[bench] {args.warmup} warm-up steps done")

    nf, nb = len(B.FWD_STAGES) + 1, len(B.BWD_STAGES) + 1

    def run_steps(n, fwd_slots, bwd_slots, stage_marks):
        """n steps; events at the listed forward / backward stage boundaries
        (and, with stage_marks, before route, plan and after each step).
        Returns the events and the total GPU time of the n steps."""
        evs = []
        for _ in range(n):
            evs.append({"route": H.create() if stage_marks else None,
                        "plan": H.create() if stage_marks else None,
                        "fwd": {i: H.create() for i in fwd_slots},
                        "bwd": {i: H.create() for i in bwd_slots} if w.backward else {}})
        t0, t1 = H.create(), H.create()
        torch.cuda.synchronize()
        H.record(t0, stream)
        for ev in evs:
            fe = B.MoeStageEvents() if ev["fwd"] else None
            for i, e in ev["fwd"].items():
                fe.ev[i] = e
            be = B.MoeStageEvents() if ev["bwd"] else None
            for i, e in ev["bwd"].items():
                be.ev[i] = e
            if stage_marks:
                H.record(ev["route"], stream)
            L.route()
            if stage_marks:
                H.record(ev["plan"], stream)
            L.plan()
            L.forward(events=fe)
            if w.backward:
                L.backward(events=be)
        H.record(t1, stream)
        H.sync(t1)
        torch.cuda.synchronize()
        return evs, H.ms(t0, t1)

    # Per-stage breakdown, from steps with an event at every stage boundary.
    # Each recorded event leaves the GPU idle for a few microseconds, so
    # these steps are not the timed ones.
    staged, _ = run_steps(max(2, min(5, args.steps)), range(nf), range(nb) if w.backward else [], True)
    stages = {"route": 0.0, "plan": 0.0}
    for ev in staged:
        stages["route"] += H.ms(ev["route"], ev["plan"])
        stages["plan"] += H.ms(ev["plan"], ev["fwd"][0])
        for i, name in enumerate(B.FWD_STAGES):
            stages["fwd." + name] = stages.get("fwd." + name, 0.0) + H.ms(ev["fwd"][i], ev["fwd"][i + 1])
        if w.backward:
            for i, name in enumerate(B.BWD_STAGES):
                stages["bwd." + name] = stages.get("bwd." + name, 0.0) + H.ms(ev["bwd"][i], ev["bwd"][i + 1])
    stages = {k: v / len(staged) for k, v in stages.items()}

    fwd_fl, bwd_fl = stage_flops(w)
    # kernels that run as exactly one instance per launch shape: (phase, first
    # stage, end stage, launches, FLOPs per launch)
    fi, bi = B.FWD_STAGES.index, B.BWD_STAGES.index
    dense = dense_routing(w)
    kern = {
        "gemm up/gate+SwiGLU (routed)": ("fwd", fi("up_routed"), fi("up_routed") + 1, 1,
                                         fwd_fl["up_routed"][0]),
        ("gemm down + combine (all experts)" if dense else "gemm down (routed)"):
            ("fwd", fi("down_routed"), fi("down_routed") + 1, 1, fwd_fl["down_routed"][0]),
    }
    if w.backward:
        kern["gemm dgrad+SwiGLU bwd (routed)"] = ("bwd", bi("dgrad_routed"), bi("dgrad_routed") + 1, 1,
                                                  bwd_fl["dgrad_routed"][0])
        if dense:
            kern["gemm dX + reverse combine (all experts)"] = ("bwd", bi("dx_shared"), bi("dx_shared") + 1,
                                                               1, bwd_fl["dx_shared"][0])
        else:
            kern["gemm dX (routed)"] = ("bwd", bi("dx_routed"), bi("dx_routed") + 1, 1,
                                        bwd_fl["dx_routed"][0])
        kern["gemm weight grad (routed)"] = ("bwd", bi("wgrad_gate_up"), bi("wgrad_down") + 1, 3,
                                             2.0 * w.T * w.k * w.d * w.f)

    def stage_span(k):
        ph, i0, i1 = kern[k][:3]
        names = B.FWD_STAGES if ph == "fwd" else B.BWD_STAGES
        return sum(stages[ph + "." + names[i]] for i in range(i0, i1))

    dom = max(kern, key=stage_span)
    ph, i0, i1, n_launch, fl = kern[dom]

    # Timed steps: events only around the dominant kernel.
    slots = [i0, i1]
    timed, ms_total = run_steps(args.steps, slots if ph == "fwd" else [],
                                slots if ph == "bwd" else [], False)
    ms_step = ms_total / args.steps
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step (events)")
    t_ms = sum(H.ms(ev[ph][i0], ev[ph][i1]) for ev in timed) / args.steps
    avg_ms = t_ms / n_launch
    achieved = fl / (avg_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(dom, w.name),
                "avg_launch_ms": round(avg_ms, 4), "flops_per_launch": fl,
                "frac_of_2300": round(achieved / PEAK_BF16_TFLOPS_ALT, 4)}

    step_flops = w.fwd_flops() + (w.bwd_flops() if w.backward else 0.0)
    value = step_flops / (ms_step * 1e-3) / 1e12
    determinism = determinism_check(L)
    log(f"[bench] determinism: {determinism}")
    stage_report = {}
    for name, ms in stages.items():
        key = name.split(".", 1)[-1]
        fl = (fwd_fl if name.startswith("fwd.") else bwd_fl).get(key, (0.0, 1))[0] \
            if "." in name else 0.0
        stage_report[name] = {"ms": round(ms, 4)}
        if fl:
            stage_report[name]["tflops"] = round(fl / (ms * 1e-3) / 1e12, 1) if ms > 0 else None
    for name, v in stage_report.items():
        log(f"   {name:28s} {v['ms']:9.4f} ms  {v.get('tflops', '')}")

    copy = copy_ceiling(H, stream)
    log(f"[bench] HBM ceiling: copy {copy['copy']['GB/s']} GB/s, elementwise "
        f"{copy['elementwise']['GB/s']} GB/s (read + write)")
    hbm = hbm_report(w, dict(stages, route=route_time(H, stream, L)), copy["GB/s"])
    for name, v in hbm.items():
        log(f"   hbm {name:18s} {v}")

    graph = graph_step_timing(H, stream, L, max(5, args.steps))
    log(f"[bench] graph-replayed step: median {graph['ms_median']:.3f} ms over {graph['replays']} replays")

    configs = None
    if not args.no_configs:
        configs = {}
        for cname in FORWARD_CONFIGS:
            t_c = time.perf_counter()
            same = cname == "large_shared" and w.name == "large_shared_train"
            c = forward_config_timing(H, stream, cname, max(5, args.steps), 2, copy["GB/s"],
                                      inputs=inputs if same else None)
            configs[cname] = c
            log(f"[bench] config {cname}: {c['ms_median']:.3f} ms median, {c['tflops']} TFLOP/s, "
                f"{c['tokens_per_s']:.0f} tok/s, routed GEMMs {c['routed_expert_gemms']} "
                f"({time.perf_counter() - t_c:.1f} s)")

    mxf = None
    if not args.no_mx and w.name in ("large_shared", "large_shared_train"):
        mxf = mx_forward_timing(H, stream, inputs, max(3, args.steps // 2), 2)
        bf16_fwd = stages["route"] + stages["plan"] + sum(
            v for k, v in stages.items() if k.startswith("fwd."))
        mxf["bf16_forward_ms"] = round(bf16_fwd, 4)
        mxf["speedup_vs_bf16_forward"] = round(bf16_fwd / mxf["ms_per_step"], 3)
        log(f"[bench] MXFP8 forward: {mxf['ms_per_step']:.3f} ms ({mxf['tflops']} TFLOP/s), "
            f"BF16 forward {bf16_fwd:.3f} ms")
        for name, v in mxf["stages"].items():
            log(f"   mx.{name:25s} {v['ms']:9.4f} ms  {v.get('tflops', '')}")

    mxt = None
    if not args.no_mx and w.name == "large_shared_train":
        mxt = mx_training_timing(H, stream, inputs, max(3, args.steps // 2), 2)
        mxt["speedup_vs_bf16_step"] = round(ms_step / mxt["ms_per_step"], 3)
        mw = mxt["wgrad_mxfp8"]
        mw["speedup_vs_bf16_step"] = round(ms_step / mw["ms_per_step"], 3)
        log(f"[bench] MXFP8 training step: {mxt['ms_per_step']:.3f} ms (forward {mxt['forward_ms']:.3f}, "
            f"backward {mxt['backward_ms']:.3f}; {mxt['tflops']} TFLOP/s), BF16 step {ms_step:.3f} ms")
        log(f"[bench]   with MXFP8 weight gradients: {mw['ms_per_step']:.3f} ms (backward "
            f"{mw['backward_ms']:.3f}; {mw['tflops']} TFLOP/s, {mw['speedup_vs_bf16_step']}x the BF16 step)")
        log(f"[bench]   weight requantisation after an update (both layouts): {mxt['weight_quant_ms']:.3f} ms")

    fused = None
    if not args.no_fused:
        fused = fused_forward_timing(H, stream, L, max(5, args.steps))
        log(f"[bench] forward (route+plan+forward): separate launches {fused['separate_ms']:.3f} ms, "
            f"fused persistent {fused['fused_ms']:.3f} ms ({fused['speedup']}x)")

    ring = None
    if not args.no_ring:
        ring = ring_timing(H, stream, w, inputs, L, max(3, args.steps // 2), 2)
        log(f"[bench] ring of {ring['ring_rows']} rows ({ring['windows']} windows, "
            f"{ring['workspace_gib_ring']} GiB vs {ring['workspace_gib_full']} GiB): "
            f"step {ring['ring_ms']['step']:.3f} ms vs {ring['full_ms']['step']:.3f} ms, "
            f"overhead {ring['overhead_pct']}")

    sched = None
    if not args.no_schedule:
        sched = schedule_timing(H, stream)
        for name, v in sched.items():
            log(f"   schedule {name:8s} R={v['R']:3d} L={v['L']:3d} {v['us']:8.2f} us "
                f"({100.0 * v['us'] * 1e-3 / ms_step:.3f}% of the layer step)")

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a token sample ...")
        cpu = cpu_baseline(w, inputs, args.cpu_sample_tokens)
        log(f"[bench] cpu baseline {cpu}")

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "T": w.T, "d": w.d, "E": w.E, "k": w.k, "f": w.f,
                   "f_shared": w.f_s, "passes": "fwd+bwd" if w.backward else "fwd",
                   "step": "route+plan+forward" + ("+backward" if w.backward else "")},
        "tokens_per_s": round(w.T / (ms_step * 1e-3), 1),
        "frac_of_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "frac_of_2300": round(value / PEAK_BF16_TFLOPS_ALT, 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "graph_replay": graph,
        "determinism": determinism,
        "hbm_copy": copy,
        "hbm_kernels": hbm,
        "stages": stage_report,
        "forward_configs": configs,
        "schedule": sched,
        "mxfp8_forward": mxf,
        "mxfp8_training_step": mxt,
        "fused_forward": fused,
        "bounded_memory": ring,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

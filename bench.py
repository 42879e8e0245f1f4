#!/usr/bin/env python3
"""DeaMoE MoE-layer decode benchmark on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--batch T]

A step is one pass of the whole layer (router product, route/plan, gate/up,
down, combine) over one batch of T synthetic tokens, through the C ABI.
Weights are resident in HBM before timing; every step uses the next of R
identical weight copies (R * layer bytes >> 256 MB of last-level cache) and
the next of 8 token batches, so no step is served from a cache that the
previous one filled.  Prints one JSON line (stdout); progress goes to stderr.

value = algorithmic HBM bytes of the steps / their time (GB/s), where the
algorithmic bytes of a step are the weights of every department and expert
its routing touched, the router, the shared expert, x read and y written
(deamoe_loaded_bytes on the step's own routing counts).
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer decode latency (µs) + achieved HBM GB/s, batch 1–64, vs vanilla MoE"
HBM_PEAK_GBPS = 8000.0
# Figures of the gate/up kernel at 16 tokens taken with rocprofv3 on the
# library sources whose digest follows (a mismatch reports them as null):
#  - HBM bytes per launch from FETCH_SIZE and WRITE_SIZE passes, scaled by
#    what the same counters read for a plain device copy (x2.0 and x1.0);
#  - the average launch duration from a kernel-trace run of the default
#    command (profiles/gate_up_dsv3_bf16_T16_kernel_trace.md), which excludes
#    the launch gap that the benchmark's own events include.
TRAFFIC_BYTES = 2341123891
PROFILED_GATE_UP_US = 339.66
TRAFFIC_SOURCES_SHA256 = "642b1e82bc6283e4a1c664beac1f39abd57d15368ba13a966b2f9276ae23cdce"


def library_sources_digest() -> str:
    import glob
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    files = sorted(glob.glob(os.path.join(root, "paper_2608_14385_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(root, "paper_2608_14385_amd", "csrc", "*.h")))
    files.append(os.path.join(root, "include", "deamoe.h"))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profiled_figures(cfg, T: int):
    """(traffic bytes, profiled average launch us) of the gate/up kernel for
    the workload and sources they were taken on, else (None, None)."""
    if cfg.name != "dsv3_bf16" or T != 16 or library_sources_digest() != TRAFFIC_SOURCES_SHA256:
        return None, None
    return TRAFFIC_BYTES, PROFILED_GATE_UP_US


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=2000)
    ap.add_argument("--workload", default="dsv3_bf16")
    ap.add_argument("--batch", type=int, default=16)
    ap.add_argument("--sweep", default="1,2,4,8,16,32,64",
                    help="comma-separated batches for the latency sweep ('' to skip)")
    ap.add_argument("--sweep-steps", type=int, default=50)
    ap.add_argument("--no-baseline", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--copies", type=int, default=0, help="weight copies (0: automatic)")
    ap.add_argument("--no-stages", action="store_true", help="skip the per-kernel event timing")
    ap.add_argument("--layers", type=int, default=0,
                    help="also time a decode step through this many distinct layers in one graph")
    ap.add_argument("--no-stream", action="store_true",
                    help="skip the read-bandwidth probe (libdeamoe_probe.so)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy 5 times (counter calibration)")
    return ap.parse_args()


class Hip:
    """The few HIP runtime calls the benchmark needs for raw events."""

    def __init__(self):
        self.lib = C.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.lib.hipEventDestroy.argtypes = [C.c_void_p]

    def event(self) -> int:
        e = C.c_void_p()
        assert self.lib.hipEventCreate(C.byref(e)) == 0
        return e.value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = C.c_float()
        assert self.lib.hipEventElapsedTime(C.byref(ms), C.c_void_p(a), C.c_void_p(b)) == 0
        return float(ms.value)

    def destroy(self, e: int):
        self.lib.hipEventDestroy(C.c_void_p(e))


class LayerRun:
    """R weight copies, token batches and workspace of one layer on the GPU."""

    def __init__(self, cfg, max_tokens: int, copies: int, baseline: bool, seed=0, bias=None):
        import torch
        from paper_2608_14385_amd import deamoe as D
        from paper_2608_14385_amd import workloads as W
        self.D, self.W, self.torch = D, W, torch
        self.cfg, self.baseline = cfg, baseline
        self.bias = bias   # optional fp32 router bias [n] on the device (skewed routing)
        self.bias_ptr = bias.data_ptr() if bias is not None else None
        t0 = time.time()
        w0 = W.make_weights(cfg, seed, device="cuda")
        self.copies = [w0] + [{k: v.clone() for k, v in w0.items()} for _ in range(copies - 1)]
        self.structs = [D.make_weights(w) for w in self.copies]
        self.layer_bytes = sum(t.numel() * t.element_size() for t in w0.values())
        self.c = D.make_config(cfg, max_tokens)
        self.ws = D.alloc_workspace(self.c)
        self.fn = D.lib().deamoe_baseline_forward if baseline else D.lib().deamoe_layer_forward
        self.traced = D.lib().deamoe_layer_forward_traced
        torch.cuda.synchronize()
        log(f"[bench] {cfg.name}: {copies} copies x {self.layer_bytes / 1e9:.2f} GB generated "
            f"in {time.time() - t0:.1f}s")
        self.xs, self.y, self.T = [], None, 0

    def set_batch(self, T: int, n_x: int = 8):
        W, torch = self.W, self.torch
        self.T = T
        self.xs = [W.make_tokens(self.cfg, T, 100 + i, device="cuda") for i in range(n_x)]
        self.y = torch.empty_like(self.xs[0])
        # algorithmic bytes of every token batch from its own routing
        self.bytes = []
        for x in self.xs:
            rt = self.D.Routing.alloc(self.cfg, T)
            self.D.deamoe_layer_forward(self.c, x, self.structs[0], self.y, self.ws,
                                        router_bias=self.bias, routing=rt) \
                if not self.baseline else \
                self.D.deamoe_baseline_forward(self.c, x, self.structs[0], self.y, self.ws,
                                               router_bias=self.bias, routing=rt)
            h = rt.host()
            wb, tb = self.D.deamoe_loaded_bytes(self.c, T, h["dept_count"], h["exp_count"])
            self.bytes.append((wb, tb, h["dept_count"], h["exp_count"]))
        torch.cuda.synchronize()

    def step(self, i: int):
        x = self.xs[i % len(self.xs)]
        W = self.structs[i % len(self.structs)]
        s = self.torch.cuda.current_stream().cuda_stream
        rc = self.fn(C.byref(self.c), self.T, x.data_ptr(), C.byref(W), None, self.bias_ptr, None,
                     self.y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), s)
        if rc:
            raise RuntimeError(f"layer call failed: {self.D.status_string(rc)}")

    def step_bytes(self, i: int) -> int:
        return self.bytes[i % len(self.xs)][1]

    def routing_stats(self) -> dict:
        """Realised routing of the token batches (mean over batches): tokens
        of the busiest department, departments and experts touched."""
        dc = [np.asarray(b[2]) for b in self.bytes]
        ec = [np.asarray(b[3]) for b in self.bytes]
        return {"max_dept_tokens": round(float(np.mean([d.max() for d in dc])), 2),
                "departments": round(float(np.mean([(d > 0).sum() for d in dc])), 2),
                "experts": round(float(np.mean([(e > 0).sum() for e in ec])), 2)}

    def time_direct(self, steps: int, warmup: int) -> float:
        torch = self.torch
        for i in range(warmup):
            self.step(i)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            self.step(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    def time_each(self, steps: int, warmup: int) -> np.ndarray:
        """Per-step latencies (ms): an event before every step and one after
        the last, all on the launch stream, steps launched back to back."""
        torch = self.torch
        for i in range(warmup):
            self.step(i)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        for i in range(steps):
            evs[i].record()
            self.step(i)
        evs[steps].record()
        torch.cuda.synchronize()
        return np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(steps)])

    def time_graph(self, steps: int, warmup: int) -> float:
        """Steps captured in one hipGraph (8 steps per graph), replayed."""
        torch = self.torch
        per = 8
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for i in range(per):
                self.step(i)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            for i in range(per):
                self.step(i)
        reps = max(1, math.ceil(steps / per))
        for _ in range(max(1, warmup // per)):
            g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / (reps * per)

    def time_stages(self, hip: Hip, steps: int, n_ev: int | None = None) -> list:
        """Per-kernel durations (ms) from HIP events recorded between the
        kernels on the launch stream; returns one list of durations per step."""
        torch = self.torch
        if n_ev is None:
            n_ev = self.D.deamoe_trace_points(self.c, self.T)
        evs = [[hip.event() for _ in range(n_ev)] for _ in range(steps)]
        torch.cuda.synchronize()
        for i in range(steps):
            x = self.xs[i % len(self.xs)]
            W = self.structs[i % len(self.structs)]
            arr = (C.c_void_p * n_ev)(*evs[i])
            s = torch.cuda.current_stream().cuda_stream
            rc = self.traced(C.byref(self.c), self.T, x.data_ptr(), C.byref(W), None, self.bias_ptr,
                             None,
                             self.y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), s, arr, n_ev)
            assert rc == 0, rc
        torch.cuda.synchronize()
        out = [[hip.elapsed_ms(e[q], e[q + 1]) for q in range(n_ev - 1)] for e in evs]
        for e in evs:
            for q in e:
                hip.destroy(q)
        return out


class StackRun:
    """A decode step through L distinct layers: layer i reads layer i - 1's
    output (the attention and other non-MoE parts of a block are left out),
    and the L calls are captured in one HIP graph and replayed."""

    def __init__(self, cfg, L: int, T: int, baseline: bool, seed=0):
        import torch
        from paper_2608_14385_amd import deamoe as D
        from paper_2608_14385_amd import workloads as W
        self.D, self.torch, self.cfg, self.L, self.T = D, torch, cfg, L, T
        self.weights = [W.make_weights(cfg, seed + 7919 * i, device="cuda") for i in range(L)]
        self.structs = [D.make_weights(w) for w in self.weights]
        self.c = D.make_config(cfg, T)
        self.ws = D.alloc_workspace(self.c)
        self.fn = D.lib().deamoe_baseline_forward if baseline else D.lib().deamoe_layer_forward
        x0 = W.make_tokens(cfg, T, 500, device="cuda")
        self.acts = [x0] + [torch.empty_like(x0) for _ in range(L)]
        self.rts = [D.Routing.alloc(cfg, T) for _ in range(L)]
        self.rstructs = [r.struct() for r in self.rts]

    def step(self):
        s = self.torch.cuda.current_stream().cuda_stream
        for i in range(self.L):
            rc = self.fn(C.byref(self.c), self.T, self.acts[i].data_ptr(), C.byref(self.structs[i]),
                         None, None, C.byref(self.rstructs[i]), self.acts[i + 1].data_ptr(),
                         self.ws.data_ptr(), self.ws.numel(), s)
            if rc:
                raise RuntimeError(f"layer call failed: {self.D.status_string(rc)}")

    def step_bytes(self) -> int:
        self.step()
        self.torch.cuda.synchronize()
        total = 0
        for r in self.rts:
            h = r.host()
            total += self.D.deamoe_loaded_bytes(self.c, self.T, h["dept_count"], h["exp_count"])[1]
        return total

    def time_graph(self, reps: int, warmup: int) -> float:
        torch = self.torch
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            self.step()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            self.step()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps


def multi_layer(cfg, base_cfg, L: int, T: int, reps: int) -> dict:
    """DeaMoE and vanilla stacks of L layers at batch T (one after the other,
    so only one stack's weights are resident at a time)."""
    import torch
    out = {"layers": L, "batch_tokens": T, "timing": "one HIP graph per decode step, replayed"}
    for name, c, base in (("deamoe", cfg, False), ("vanilla", base_cfg, True)):
        st = StackRun(c, L, T, base)
        nbytes = st.step_bytes()
        ms = st.time_graph(reps, 3)
        out[name] = {"step_us": round(ms * 1e3, 2), "per_layer_us": round(ms * 1e3 / L, 2),
                     "bytes_per_step": int(nbytes), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1)}
        log(f"[bench] {L}-layer {name} T={T}: {out[name]}")
        del st
        torch.cuda.empty_cache()
    out["speedup"] = round(out["vanilla"]["step_us"] / out["deamoe"]["step_us"], 3)
    return out


def routes_in_first_stage(cfg, T: int) -> bool:
    """Batches of at most 4 tokens with routers of at most 1024 experts route
    inside the first expert stage's launch (no separate route/plan kernel)."""
    return T <= 4 and cfg.n_experts <= 1024


def stage_names(cfg, T: int, n_stages: int) -> list:
    """Names of the traced call's stages (between its recorded events)."""
    small = routes_in_first_stage(cfg, T)
    if cfg.form == "slice":
        names = ["router_gemv"] + (["route_gate_up"] if small else ["route_plan", "gate_up"])
        fused = len(names) + 1 == n_stages   # down projections and combine in one kernel
        return names + (["down_combine"] if fused else ["down", "combine"])
    names = ["router_gemv"] + (["route_dept_gate_up"] if small else ["route_plan", "dept_gate_up"])
    names += ["priv_gate_up", "priv_down", "z_collect"]
    fused = len(names) + 1 == n_stages
    return names + (["dept_down_combine"] if fused else ["dept_down", "combine"])


def gate_up_bytes(cfg, T: int, dept_count, exp_count) -> int:
    """Algorithmic bytes of the gate/up kernel: the gate and up matrices of
    every touched department, expert and the shared expert, plus x."""
    wb = {"f32": 4, "bf16": 2, "fp8": 1}[cfg.w_dtype]
    ab = 4 if cfg.act_dtype == "f32" else 2
    h = cfg.hidden

    def mat(R, Cc):
        b = R * Cc * wb
        if cfg.w_dtype == "fp8":
            b += -(-R // 128) * -(-Cc // 128) * 4
        return b
    nd = int((np.asarray(dept_count) > 0).sum())
    ne = int((np.asarray(exp_count) > 0).sum())
    b = nd * 2 * mat(cfg.d_shared, h) + T * h * ab
    if cfg.form == "slice" and cfg.d_private > 0:
        b += ne * 2 * mat(cfg.d_private, h)
    if cfg.d_shared_expert > 0:
        b += 2 * mat(cfg.d_shared_expert, h)
    return b


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_single_core(run: LayerRun, T: int, hw: dict, min_seconds: float = 3.0) -> dict:
    """The oracle on one thread, on single tokens of the step's token batches
    (its cost is per token and expert), scaled to whole steps."""
    import oracle
    threads = oracle.num_threads()
    bias = run.bias.cpu() if run.bias is not None else None
    oracle.set_num_threads(1)
    try:
        done, t0 = 0, time.perf_counter()
        while done < 4 * T and (done == 0 or time.perf_counter() - t0 < min_seconds):
            i, t = (done // T) % len(run.xs), done % T
            oracle.layer(run.cfg, run.xs[i].cpu(), hw, bias=bias, tokens=[t])
            done += 1
        dt = time.perf_counter() - t0
    finally:
        oracle.set_num_threads(threads)
    step_s = dt / done * T
    return {"value": float(np.mean([run.step_bytes(i) for i in range(len(run.xs))])) / step_s / 1e9,
            "unit": "GB/s", "cores": 1, "sample": f"{done} single tokens at one thread, "
            f"{dt:.1f}s, scaled to {T}-token steps", "seconds_per_step": step_s}


def stream_read_peak(nbytes: int = 4 << 30, reps: int = 10) -> float:
    """GB/s of the read probe (libdeamoe_probe.so) streaming a 4 GiB buffer."""
    import torch
    from paper_2608_14385_amd import build as B
    lib = C.CDLL(B.PROBE_LIB)
    lib.deamoe_probe_read.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_int, C.c_void_p]
    bufs = [torch.ones(nbytes, dtype=torch.uint8, device="cuda") for _ in range(2)]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream

    def go(i):
        rc = lib.deamoe_probe_read(bufs[i % 2].data_ptr(), nbytes, sink.data_ptr(), 8192, s)
        assert rc == 0, rc
    for i in range(3):
        go(i)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(reps):
        go(i)
    b.record()
    torch.cuda.synchronize()
    gbps = nbytes * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del bufs
    torch.cuda.empty_cache()
    return gbps


def cpu_baseline(run: LayerRun, T: int, min_seconds: float = 10.0) -> dict:
    """The oracle on whole steps of the same workload (successive token
    batches) until at least `min_seconds` of CPU work, at most 16 steps."""
    import oracle
    threads = oracle.num_threads()
    hw = {k: v.cpu() for k, v in run.copies[0].items()}
    bias = run.bias.cpu() if run.bias is not None else None
    done, nbytes, t0 = 0, 0, time.perf_counter()
    while done < 16 and (done == 0 or time.perf_counter() - t0 < min_seconds):
        i = done % len(run.xs)
        oracle.layer(run.cfg, run.xs[i].cpu(), hw, bias=bias)
        nbytes += run.step_bytes(i)
        done += 1
    dt = time.perf_counter() - t0
    out = {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
           "sample": f"{done} whole {run.cfg.name} steps of {T} tokens (successive token "
                     f"batches), naive fp64 per-token per-expert loop, {dt:.1f}s",
           "seconds_per_step": dt / done, "cpu_model": cpu_model(),
           "affinity_cores": len(os.sched_getaffinity(0))}
    out["single_core"] = cpu_single_core(run, T, hw)
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log("bench.py measures one GPU: the DeaMoE decode layer runs on a single MI355X and this "
            "build has no multi-GPU path; run with --gpus 1.")
        sys.exit(2)
    import torch
    from paper_2608_14385_amd import deamoe as D
    from paper_2608_14385_amd import workloads as W
    D.lib()   # fails loudly when the HIP library is missing
    torch.cuda.set_device(0)
    wl = W.PRESETS[args.workload]
    cfg, bcfg = wl.layer, wl.baseline
    sweep = [int(s) for s in args.sweep.split(",") if s.strip()]
    max_T = max([args.batch] + sweep)
    hip = Hip()

    def copies_for(nbytes):
        if args.copies:
            return args.copies
        return max(2, math.ceil(4 * 256e6 / nbytes))

    layer_bytes = sum(math.prod(s) for s in W.weight_shapes(cfg).values()) * \
        {"f32": 4, "bf16": 2, "fp8": 1}[cfg.w_dtype]
    # skewed routing: one per-expert router bias for both layers, so that the
    # vanilla layer sees the same logits distribution
    bias = W.make_zipf_bias(cfg).cuda() if wl.routing == "zipf_bias" else None
    run = LayerRun(cfg, max_T, copies_for(layer_bytes), baseline=False, bias=bias)
    T = args.batch
    run.set_batch(T)
    step_bytes = [run.step_bytes(i) for i in range(args.steps)]
    log(f"[bench] timing {cfg.name} T={T}: {args.warmup} warmup + {args.steps} steps")
    ms = run.time_direct(args.steps, args.warmup)
    gbps = sum(step_bytes) / (ms * 1e-3 * args.steps) / 1e9
    result = {"metric": METRIC, "value": round(gbps, 1), "unit": "GB/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
              "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.w_dtype,
              "data": "synthetic (seeded gaussian weights and tokens, resident in HBM)"}
    if cfg.form == "slice":
        shape = f"department slice {cfg.d_shared} + private slice {cfg.d_private}"
    else:
        shape = f"FACTORED (Eq. 4), d={cfg.d_shared}, top-{cfg.top_k_dept} departments"
    result["config"] = {
        "workload": f"{cfg.name}: DeaMoE layer, h={cfg.hidden}, {cfg.n_experts} experts in "
                    f"{cfg.n_depts} departments, top-{cfg.top_k} {cfg.score}, {shape}, "
                    f"{cfg.w_dtype} weights",
        "batch_tokens": T, "weight_copies": len(run.copies), "token_batches": len(run.xs),
        "routing": wl.routing, "realised_routing": run.routing_stats(),
        "timing": "direct launches on one stream, torch.cuda events around all steps"}
    result["latency_us"] = round(ms * 1e3, 2)
    each = run.time_each(args.steps, 5) * 1e3
    result["latency_percentiles_us"] = {"p10": round(float(np.percentile(each, 10)), 2),
                                        "p50": round(float(np.percentile(each, 50)), 2),
                                        "p90": round(float(np.percentile(each, 90)), 2),
                                        "timing": "an event before every step, steps back to back"}
    result["bytes_per_step"] = int(np.mean(step_bytes))
    result["hbm_frac"] = round(gbps / HBM_PEAK_GBPS, 4)
    log(f"[bench] {cfg.name} T={T}: {ms * 1e3:.1f} us/step, {gbps:.0f} GB/s")

    if not args.no_graph:
        gms = run.time_graph(args.steps, args.warmup)
        result["graph"] = {"latency_us": round(gms * 1e3, 2),
                           "GBps": round(sum(step_bytes) / (gms * 1e-3 * args.steps) / 1e9, 1)}
        log(f"[bench] graph replay: {gms * 1e3:.1f} us/step")

    # per-kernel durations (HIP events on the launch stream, same region shape)
    if not args.no_stages:
        stages = run.time_stages(hip, args.steps)
        names = stage_names(cfg, T, len(stages[0]))
        mean = np.mean(np.asarray(stages), axis=0)
        result["kernels_us"] = {n: round(float(v) * 1e3, 2) for n, v in zip(names, mean)}
        dom = [i for i, n in enumerate(names) if n.endswith("gate_up") and "priv" not in n][0]
        gu = [gate_up_bytes(cfg, T, b[2], b[3]) for b in run.bytes]
        gu_bytes = float(np.mean([gu[i % len(gu)] for i in range(args.steps)]))
        achieved = gu_bytes / (mean[dom] * 1e-3) / 1e9
        traffic, prof_us = profiled_figures(cfg, T)
        result["roofline"] = {"kernel": f"{names[dom]} stage", "bound": "hbm",
                              "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                              "frac": round(achieved / HBM_PEAK_GBPS, 4),
                              "traffic": traffic,
                              "bytes_per_launch": int(gu_bytes),
                              "avg_launch_us": round(float(mean[dom]) * 1e3, 2),
                              "timing": "HIP events before and after the launch on its stream "
                                        "(they include the launch gap)"}
        if prof_us is not None:
            pa = gu_bytes / (prof_us * 1e-6) / 1e9
            result["roofline"]["profiled"] = {
                "avg_launch_us": prof_us, "achieved": round(pa, 1),
                "frac": round(pa / HBM_PEAK_GBPS, 4),
                "source": "rocprofv3 kernel trace, profiles/gate_up_dsv3_bf16_T16_kernel_trace.md"}
        log(f"[bench] kernels (us): {result['kernels_us']}")

    # vanilla-MoE comparator and the batch sweep
    sweep_rows = []
    brun = b16run = None
    if not args.no_baseline:
        bbytes = sum(math.prod(s) for s in W.weight_shapes(bcfg).values()) * \
            {"f32": 4, "bf16": 2, "fp8": 1}[bcfg.w_dtype]
        brun = LayerRun(bcfg, max_T, copies_for(bbytes), baseline=True, bias=bias)
        if bcfg.w_dtype == "fp8":   # also the vanilla layer with bf16 weights
            b16 = bcfg.replace(name=bcfg.name.replace("fp8", "bf16"), w_dtype="bf16")
            b16run = LayerRun(b16, max_T, copies_for(2 * bbytes), baseline=True, bias=bias)
    for Tb in sweep:
        row = {"batch": Tb}
        for name, r in (("deamoe", run), ("vanilla", brun), ("vanilla_bf16", b16run)):
            if r is None:
                continue
            r.set_batch(Tb)
            k = args.sweep_steps
            m = r.time_direct(k, max(5, k // 5))
            by = float(np.mean([r.step_bytes(i) for i in range(k)]))
            row[name] = {"latency_us": round(m * 1e3, 2), "bytes": int(by),
                         "GBps": round(by / (m * 1e-3) / 1e9, 1), "routing": r.routing_stats()}
            if not args.no_graph:
                gm = r.time_graph(k, 8)
                row[name]["graph_latency_us"] = round(gm * 1e3, 2)
        if brun is not None:
            row["speedup"] = round(row["vanilla"]["latency_us"] / row["deamoe"]["latency_us"], 3)
            row["byte_ratio"] = round(row["deamoe"]["bytes"] / row["vanilla"]["bytes"], 4)
        if b16run is not None:
            row["speedup_vs_bf16_vanilla"] = round(
                row["vanilla_bf16"]["latency_us"] / row["deamoe"]["latency_us"], 3)
        log(f"[bench] sweep {row}")
        sweep_rows.append(row)
    if sweep_rows:
        result["sweep"] = sweep_rows
        head = [r for r in sweep_rows if r["batch"] == T]
        if head and "speedup" in head[0]:
            result["speedup_vs_vanilla"] = head[0]["speedup"]
        if head and "speedup_vs_bf16_vanilla" in head[0]:
            result["speedup_vs_bf16_vanilla"] = head[0]["speedup_vs_bf16_vanilla"]

    if args.layers > 0:
        result["multi_layer"] = multi_layer(cfg, wl.baseline, args.layers, T, max(5, args.steps // 10))

    if not args.no_stream:
        peak = stream_read_peak()
        result["stream_read_peak"] = {
            "GBps": round(peak, 1), "frac_of_peak": round(peak / HBM_PEAK_GBPS, 4),
            "probe": "libdeamoe_probe.so: 4 GiB read once, 16-byte non-temporal loads, "
                     "8192 workgroups of 256 lanes, 10 passes"}
        if "roofline" in result:
            result["stream_read_peak"]["gate_up_frac_of_stream"] = round(
                result["roofline"]["achieved"] / peak, 4)
        log(f"[bench] read probe: {peak:.0f} GB/s")

    if args.copy_probe:
        src = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy probe: 5 x 1073741824-byte device copies")
        del src, dst

    if not args.no_cpu:
        run.set_batch(T)
        result["cpu_baseline"] = cpu_baseline(run, T)
        log(f"[bench] cpu oracle: {result['cpu_baseline']}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

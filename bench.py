#!/usr/bin/env python3
"""Throughput of one GPU's MoE layer (route + source x expert counts +
dispatch + SwiGLU expert FFN + combine) on MI355X.

    python bench.py [--steps K] [--warmup W] [--config NAME]

A step is one moe_forward over one batch of the workload, inputs and bf16
weights resident in HBM.  The default workload is the largest that one GPU
holds: one expert-parallel rank's share of a DeepSeek-V3-shaped layer (16384
tokens from 8 sources, hidden 7168, top-8 of 256 experts of which 32 are
hosted here, intermediate 2048, one shared expert).  Each timed step is cold:
a 1 GiB read before it evicts the L2s and the Infinity Cache.  Prints one JSON
line: whole-job tokens/s, per-stage kernel times measured live with HIP
events on the launch stream, the roofline position of the dominant stage (and
the same figure from the committed kernel trace), back-to-back (warm) steps
as a secondary figure, and the CPU oracle's throughput on a bounded sample of
the same workload.

With a placement workload (--config place_*), a step is instead one
moe_place_experts call: the source-aware greedy expert placement of every MoE
layer of a model from its window statistics, inputs resident in HBM.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/sec on 1 MI355X; expert-FFN % MFMA peak; route/permute % HBM BW"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, vendor figure
STAGES = ("route", "permute", "ffn_up", "ffn_down", "combine")


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--config", default="ep_share_dsv3")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="budget of the CPU-oracle baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--gpu-metrics", action="store_true",
                   help="sample the shader clock and socket power with amd-smi during the run")
    p.add_argument("--fenced-events", action="store_true",
                   help="time with default (system-fenced) HIP events instead of timing-only ones")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="also run a plain device copy of this size (HBM counter calibration)")
    return p.parse_args(argv)


# Timing-only events: no system-scope fence (cache writeback and invalidate)
# when the event is recorded, so recording one does not stall the stream; the
# host reads the times only after a device-wide synchronisation.
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class HipEvents:
    """hipEvent_t handles from the HIP runtime the process already uses."""

    def __init__(self, n: int, flags: int = HIP_EVENT_DISABLE_SYSTEM_FENCE):
        import torch  # noqa: F401  (loads torch's HIP runtime first)
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            rc = self.hip.hipEventCreateWithFlags(ctypes.byref(e), flags)
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            self.ev.append(e.value)

    def record(self, i: int, stream: int) -> None:
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        rc = self.hip.hipEventRecord(self.ev[i], stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), self.ev[a], self.ev[b])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(e)


def stage_work(cfg, R: int, active: int) -> dict:
    """Algorithmic bytes and FLOPs of one launch of each stage (what the
    method must move or compute: active experts' weights only, each tensor
    read or written once)."""
    T, H, E, k, I, S = cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.S
    n_sh, I_sh = cfg.n_shared, (cfg.I_shared if cfg.n_shared else 0)
    bf = 2
    w = {}
    # the statistics (src read, counts read and written) go with the stage
    # that counts them: the router for batches it dispatches itself (at most
    # 512 pairs), else the dispatch's count pass
    stats_bytes = T * 4 + 2 * S * E * 8
    stats_in_route = T * k <= 512
    w["route"] = dict(bytes=T * E * 4 + T * k * 8 + (stats_bytes if stats_in_route else 0), flops=0)
    # the dispatch sort only: the token rows are read by the gate/up GEMM
    # through perm_token (counted there as R*H*bf), never copied
    w["permute"] = dict(bytes=T * k * 4 + (cfg.E_local + 1) * 4 + R * 4 + T * k * 4
                        + (0 if stats_in_route else stats_bytes), flops=0)
    w["ffn_up"] = dict(bytes=active * 2 * I * H * bf + n_sh * 2 * I_sh * H * bf + R * H * bf
                       + (T * H * bf if n_sh else 0) + R * I * bf + T * n_sh * I_sh * bf,
                       flops=2 * 2 * H * I * R + 2 * 2 * H * n_sh * I_sh * T)
    w["ffn_down"] = dict(bytes=active * H * I * bf + n_sh * H * I_sh * bf + R * I * bf
                         + T * n_sh * I_sh * bf + R * H * bf + (T * H * bf if n_sh else 0),
                         flops=2 * H * I * R + 2 * H * n_sh * I_sh * T)
    w["combine"] = dict(bytes=R * H * bf + (T * H * bf if n_sh else 0) + T * k * 8 + T * H * bf, flops=0)
    return w


# The sources of the layer's kernels: a profile's counters stay valid while
# these are unchanged (placement and diagnostics kernels do not run in a step).
LAYER_SOURCES = ("common.h", "ffn_impl.h", "dispatch_impl.h", "route.hip", "permute.hip", "ffn_skinny.hip",
                 "ffn_tiled.hip", "combine.hip")


def source_digest(names=LAYER_SOURCES) -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_15177_amd", "csrc")
    for name in sorted(names):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(stage: str, workload: str):
    """HBM bytes of a stage per layer call (all of the stage's launches) from a
    committed rocprofv3 --pmc summary of this workload, if it was taken on the
    current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", f"pmc_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"source_digest:\s*([0-9a-f]+)", text)
    m_b = re.search(rf"hbm_bytes_per_call_{stage}:\s*([0-9.eE+]+)", text)
    if not m_src or not m_b or m_src.group(1) != source_digest():
        return None
    return float(m_b.group(1))


# The kernels of each stage, as named in a rocprofv3 kernel trace.
STAGE_KERNELS = {
    "route": ("route_kernel<", "stats_kernel"),
    "permute": ("perm_count_kernel", "perm_scan_kernel", "perm_scatter_kernel", "perm_single_kernel"),
    "ffn_up": ("tiled_kernel<true", "skinny_kernel<true"),
    "ffn_down": ("tiled_kernel<false", "skinny_kernel<false"),
    "combine": ("combine_kernel",),
}


def _profile_rows(path: str):
    """(source digest, [(kernel name, cells...)]) of a committed profile
    summary, or None when it is missing or was taken on other sources."""
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"source_digest:\s*([0-9a-f]+)", text)
    if not m_src or m_src.group(1) != source_digest():
        return None
    rows = []
    for line in text.splitlines():
        m = re.match(r"\|\s*`([^`]*)`\s*\|(.*)\|\s*$", line)
        if m:
            rows.append((m.group(1), [c.strip() for c in m.group(2).split("|")]))
    return rows


def profiled_stage_ms(stage: str, workload: str):
    """The stage's time per layer call in the committed kernel trace of this
    workload (the sum of its kernels' average durations; each runs once per
    call), if the trace was taken on the current kernel sources."""
    rows = _profile_rows(os.path.join(ROOT, "profiles", f"kernel_trace_{workload}.md"))
    if rows is None:
        return None
    us = [float(c[1]) for name, c in rows if any(k in name for k in STAGE_KERNELS[stage])]
    return sum(us) * 1e-3 if us else None


def profiled_clock(stage: str, workload: str):
    """Shader clock and MFMA busy fraction of the stage's kernels from the
    committed MFMA counter summary of this workload (current sources only)."""
    rows = _profile_rows(os.path.join(ROOT, "profiles", f"pmc_mfma_{workload}.md"))
    if rows is None:
        return None
    out = []
    for name, c in rows:
        if any(k in name for k in STAGE_KERNELS[stage]):
            out.append({"kernel": name.split("::")[-1].split("(")[0], "avg_us": float(c[2]),
                        "clock_ghz": float(c[3]), "mfma_busy": round(float(c[4].rstrip("%")) / 100, 4)})
    return out or None


def cpu_identity() -> dict:
    """The host CPU's model name and logical core count."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "cpu_count": os.cpu_count()}


class GpuMetricsWatch:
    """amd-smi clock and power samples of GPU 0, once a second, for the whole
    run.  The watcher is started as a child process before this process
    touches the GPU (a process that has initialised the GPU must not start
    programs), so it is opt-in (--gpu-metrics) and refused under a profiler,
    whose preloaded library initialises the GPU before the program starts."""

    def __init__(self):
        import subprocess
        if any("rocprof" in v for k, v in os.environ.items() if k in ("LD_PRELOAD", "HSA_TOOLS_LIB")):
            raise SystemExit("--gpu-metrics cannot run under a profiler")
        self.proc = subprocess.Popen(["amd-smi", "metric", "-c", "-p", "--json", "-g", "0", "-w", "1"],
                                     stdout=subprocess.PIPE, stderr=subprocess.DEVNULL, text=True)

    def stop(self) -> dict:
        self.proc.terminate()
        try:
            text, _ = self.proc.communicate(timeout=10)
        except Exception:  # noqa: BLE001 - a watcher that hangs only loses its samples
            self.proc.kill()
            return {}
        sclk = [int(m) for m in re.findall(r'"gfx_0":\s*\{\s*"clk":\s*\{\s*"value":\s*(\d+)', text)]
        power = [int(m) for m in re.findall(r'"socket_power":\s*\{\s*"value":\s*(\d+)', text)]
        if not sclk:
            return {}
        return {"samples": len(sclk), "sclk_mhz_max": max(sclk), "sclk_mhz_min": min(sclk),
                "socket_power_w_max": max(power) if power else None}


def pinned_core():
    """Pin the calling thread to one core of its allowed set (the last one)
    and return (core, the previous set), or (None, None) where affinity
    cannot be set."""
    try:
        allowed = os.sched_getaffinity(0)
        core = max(allowed)
        os.sched_setaffinity(0, {core})
        return core, allowed
    except (AttributeError, OSError):
        return None, None


def cpu_baseline(cfg, wl, budget_s: float) -> dict:
    """The CPU oracle (plain C, fp64, single thread pinned to one core) on a
    bounded sample of the same workload: the first n tokens, n sized to the
    time budget."""
    from oracle import oracle
    oracle.lib()
    core, allowed = pinned_core()
    try:
        gate = dict(gate=cfg.gate, bias=wl.get("gate_bias"), scale=cfg.routed_scale, n_group=cfg.n_group,
                    topk_group=cfg.topk_group)
        n0 = min(cfg.T, 8)    # a few tokens size the sample (their expert counts vary)
        t0 = time.perf_counter()
        oracle.forward_tokens(cfg.dims, list(range(n0)), wl["logits"], wl["x"], wl["local_experts"], wl, **gate)
        per_tok = max(time.perf_counter() - t0, 1e-6) / n0
        n = int(max(1, min(cfg.T, budget_s / per_tok)))
        toks = list(range(n))
        t0 = time.perf_counter()
        oracle.forward_tokens(cfg.dims, toks, wl["logits"], wl["x"], wl["local_experts"], wl, **gate)
        dt = time.perf_counter() - t0
    finally:
        if allowed is not None:
            os.sched_setaffinity(0, allowed)
    return {"value": n / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of {cfg.T} tokens of {cfg.name}: per-token routing + "
                      f"SwiGLU experts + combine, fp64, single thread ({dt:.1f} s)",
            "pinned_core": core, **cpu_identity()}


def bench_place(args) -> int:
    """Latency of one placement call over all layers of the workload."""
    import numpy as np
    import torch

    from paper_2606_15177_amd import moe
    from paper_2606_15177_amd import workloads as W

    cfg = W.PLACE_CONFIGS[args.config]
    torch.cuda.set_device(0)
    print(f"[bench] generating {cfg.name} (seed {args.seed})", file=sys.stderr, flush=True)
    p = W.make_place_inputs(cfg, args.seed)
    A = torch.from_numpy(p["A"]).cuda()
    D = torch.from_numpy(p["D"]).cuda()
    x0 = torch.from_numpy(p["x0"]).cuda()
    pd = moe.place_dims(cfg.L, cfg.S, cfg.E, cfg.G, *moe.PAPER_PLACE_WEIGHTS, cfg.m_uniform)
    slots = moe.place_slots(pd, p["cap"])
    x = torch.empty((cfg.L, cfg.E), dtype=torch.int32, device="cuda")
    rank_experts = torch.empty((cfg.L, cfg.G, slots), dtype=torch.int32, device="cuda")
    cost = torch.empty((cfg.L, 3), dtype=torch.float64, device="cuda")

    def call():
        moe.place_experts(pd, p["cap"], A, D, x0, x, rank_experts=rank_experts, cost=cost)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream().cuda_stream
    events = HipEvents(2 * args.steps)
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        events.record(2 * i, stream)
        call()
        events.record(2 * i + 1, stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kernel_ms = sum(events.elapsed_ms(2 * i, 2 * i + 1) for i in range(args.steps)) / args.steps
    events.close()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    moved = float((x.cpu().numpy() != p["x0"]).mean())

    # what the window's statistics say before and after: the share of traffic
    # that leaves its source's rank, and the spread of the engines' MoE pressure
    home = torch.from_numpy((np.arange(cfg.S) * cfg.G // cfg.S).astype(np.int32)).cuda()
    wd = moe.MoeWindowDims(cfg.L, cfg.S, cfg.E, cfg.G, cfg.G)

    def window(placement):
        remote = torch.empty((cfg.L, cfg.S), dtype=torch.int64, device="cuda")
        total = torch.empty_like(remote)
        rank_load = torch.empty((cfg.L, cfg.G), dtype=torch.int64, device="cuda")
        pressure = torch.empty((cfg.G,), dtype=torch.float64, device="cuda")
        moe.window_stats(wd, A, placement, home, remote, total, rank_load, pressure=pressure)
        torch.cuda.synchronize()
        return {"remote_fraction": round(float(remote.sum()) / max(float(total.sum()), 1.0), 4),
                "max_rank_load_over_mean": round(float((rank_load.double().max(dim=1).values /
                                                        rank_load.double().mean(dim=1)).mean()), 4),
                "pressure_max": round(float(pressure.max()), 4), "pressure_min": round(float(pressure.min()), 4)}

    diagnostics = {"before": window(x0), "after": window(x)}
    result = {
        "metric": "expert placement: MoE layers placed per second on 1 MI355X",
        "value": round(cfg.L / (ms_per_step * 1e-3), 1),
        "unit": "layers/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": cfg.name, "L": cfg.L, "S": cfg.S, "E": cfg.E, "G": cfg.G, "k": cfg.k,
                   "tokens_per_source": cfg.tokens_per_source, "weights": list(moe.PAPER_PLACE_WEIGHTS),
                   "parallelism": "single GPU"},
        # one workgroup per layer, every layer at once: the critical path is
        # the E dependent placement steps of one layer
        "roofline": {"bound": "latency", "kernel": "place", "kernel_ms": round(kernel_ms, 4),
                     "ns_per_expert_step": round(kernel_ms * 1e6 / cfg.E, 1)},
        "moved_fraction": round(moved, 4),
        "window": diagnostics,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        from oracle import oracle
        oracle.lib()
        n, t_cpu = 0, 0.0
        while t_cpu < min(args.cpu_seconds, 5.0) and n < 1000:
            c0 = time.perf_counter()
            oracle.place_greedy(p["A"], p["D"], p["x0"], p["cap"], m_uniform=cfg.m_uniform)
            t_cpu += time.perf_counter() - c0
            n += 1
        result["cpu_baseline"] = {
            "value": round(n * cfg.L / t_cpu, 1), "unit": "layers/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} whole calls ({cfg.L} layers each) of the C oracle's greedy, fp64, single thread"}
    print(json.dumps(result), flush=True)
    return 0


def main(argv=None) -> int:
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU's MoE layer; --gpus {args.gpus} is not supported "
              "(this build runs on a single GPU)", file=sys.stderr)
        return 2
    if args.config.startswith("place_"):
        return bench_place(args)
    return bench_layer(args, GpuMetricsWatch() if args.gpu_metrics else None)  # watcher before any GPU use


def bench_layer(args, watch) -> int:
    """Throughput of moe_forward on a layer workload (one JSON line)."""
    import numpy as np
    import torch

    from paper_2606_15177_amd import moe
    from paper_2606_15177_amd import workloads as W

    cfg = W.CONFIGS[args.config]
    torch.cuda.set_device(0)
    print(f"[bench] generating {cfg.name} (seed {args.seed})", file=sys.stderr, flush=True)
    wl = W.make_workload(cfg, args.seed)

    def dev(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(a).cuda()

    d = moe.dims_of(cfg)
    weights = {k: dev(wl[k]) for k in ("w_gate", "w_up", "w_down", "sh_gate", "sh_up", "sh_down")
               if k in wl}
    local = None if wl["local_experts"] is None else dev(wl["local_experts"])
    gate_bias = None if wl.get("gate_bias") is None else dev(wl["gate_bias"])
    gating = moe.gating(gate_bias, cfg.routed_scale, cfg.n_group, cfg.topk_group) if cfg.gated else None
    layer = moe.MoeLayer(d, weights, local, gating=gating)
    logits, src, x = dev(wl["logits"]), dev(wl["src"]), dev(wl["x"])
    counts = torch.zeros((cfg.S, cfg.E), dtype=torch.int64, device="cuda")
    out = torch.empty((cfg.T, cfg.H), dtype=torch.bfloat16, device="cuda")
    offsets = torch.empty((cfg.E_local + 1,), dtype=torch.int32, device="cuda")

    n_ev = 2 * len(STAGES)
    plain_taps = moe.make_taps(offsets=offsets)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        layer.forward(logits, src, x, counts, out, plain_taps)
    torch.cuda.synchronize()

    # Stage breakdown from an untimed probe with an event pair around every
    # stage (ten event records cost several percent of a decode step, so the
    # timed steps carry only the dominant kernel's pair).
    n_probe = max(3, min(args.steps, 20))
    ev_flags = 0 if args.fenced_events else HIP_EVENT_DISABLE_SYSTEM_FENCE
    # Probe i runs the layer twice: with the source x expert statistics
    # (events i), then without them (events n_probe + i); alternating keeps
    # the two sets under the same clocks.  Route + permute of the first
    # against the second is the cost of collecting A (counted in the route
    # kernel, or in the dispatch's count pass when the dispatch takes several
    # blocks).
    probe_ev = HipEvents(2 * n_ev * n_probe, ev_flags)
    for i in range(n_probe):
        for j, cts in ((i, counts), (n_probe + i, None)):
            layer.forward(logits, src, x, cts, out,
                          moe.make_taps(offsets=offsets, events=probe_ev.ev[j * n_ev:(j + 1) * n_ev]))
    torch.cuda.synchronize()
    stage_ms = {}
    for s_i, name in enumerate(STAGES):
        vals = [probe_ev.elapsed_ms(i * n_ev + 2 * s_i, i * n_ev + 2 * s_i + 1) for i in range(n_probe)]
        stage_ms[name] = sum(vals) / len(vals)
    # GPU time of each probe step: first stage's start to the last stage's end
    probe_steps = sorted(probe_ev.elapsed_ms(i * n_ev, i * n_ev + n_ev - 1) for i in range(n_probe))

    def route_permute_ms(j):
        return probe_ev.elapsed_ms(j * n_ev, j * n_ev + 3)
    rp_with = [route_permute_ms(i) for i in range(n_probe)]
    rp_without = [route_permute_ms(n_probe + i) for i in range(n_probe)]
    rp_stats = sum(rp_with) / n_probe
    rp_no_stats = sum(rp_without) / n_probe
    # the cost of the statistics: median over the probes of (with - without)
    # of one probe, each pair run back to back; an event pair's own jitter of
    # about a microsecond makes the mean of a few samples wander
    rp_diffs = sorted(a - b for a, b in zip(rp_with, rp_without))
    rp_overhead = rp_diffs[len(rp_diffs) // 2]
    probe_ev.close()
    dom = max(STAGES, key=lambda n: stage_ms[n])
    dom_i = STAGES.index(dom)

    # Timed steps (primary): cold.  Before each step a 1 GiB read evicts the
    # L2s and the 256 MB Infinity Cache (a read leaves no dirty lines to be
    # written back during the step), so every input and weight comes from
    # HBM.  Each step carries two timing-only events, around its first and
    # last kernels.  The dominant stage is timed in K further cold steps
    # that carry its event pair instead (an event record leaves a gap of a
    # few microseconds in the stream, so the pair stays out of the steps
    # that give the value).
    flush = torch.zeros(1 << 28, dtype=torch.float32, device="cuda")    # 1 GiB
    flush_sum = torch.zeros((), dtype=torch.float32, device="cuda")
    ev_step = HipEvents(2 * args.steps, ev_flags)
    ev_dom = HipEvents(2 * args.steps, ev_flags)
    step_taps, dom_taps = [], []
    for i in range(args.steps):
        ev = [None] * n_ev
        ev[0], ev[n_ev - 1] = ev_step.ev[2 * i], ev_step.ev[2 * i + 1]
        step_taps.append(moe.make_taps(offsets=offsets, events=ev))
        ev = [None] * n_ev
        ev[2 * dom_i], ev[2 * dom_i + 1] = ev_dom.ev[2 * i], ev_dom.ev[2 * i + 1]
        dom_taps.append(moe.make_taps(offsets=offsets, events=ev))

    print(f"[bench] timing {args.steps} cold steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        torch.sum(flush, dim=0, out=flush_sum)
        layer.forward(logits, src, x, counts, out, step_taps[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cold_wall_ms = (t1 - t0) * 1e3 / args.steps
    cold = [ev_step.elapsed_ms(2 * i, 2 * i + 1) for i in range(args.steps)]
    ms_per_step = sum(cold) / len(cold)
    cold_sorted = sorted(cold)

    print(f"[bench] timing the {dom} stage over {args.steps} cold steps", file=sys.stderr, flush=True)
    for i in range(args.steps):
        torch.sum(flush, dim=0, out=flush_sum)
        layer.forward(logits, src, x, counts, out, dom_taps[i])
    torch.cuda.synchronize()
    # the dominant stage's average duration over these steps
    stage_ms[dom] = sum(ev_dom.elapsed_ms(2 * i, 2 * i + 1) for i in range(args.steps)) / args.steps
    ev_step.close()
    ev_dom.close()
    del flush

    # Secondary: warm steps, back to back with no events, wall clock.
    print(f"[bench] timing {args.steps} warm steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        layer.forward(logits, src, x, counts, out, plain_taps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    warm_ms = (t1 - t0) * 1e3 / args.steps

    off = offsets.cpu().numpy()
    R = int(off[-1])
    active = int((np.diff(off) > 0).sum())
    work = stage_work(cfg, R, active)
    ridge = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    stages = {}
    for name in STAGES:
        t = stage_ms[name] * 1e-3
        b, f = work[name]["bytes"], work[name]["flops"]
        gbs = b / t / 1e9 if t > 0 else 0.0
        tfl = f / t / 1e12 if t > 0 else 0.0
        stages[name] = {"ms": round(stage_ms[name], 4), "bytes": b, "flops": f,
                        "GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                        "TFLOP/s": round(tfl, 1), "frac_mfma": round(tfl / MFMA_BF16_PEAK_TFLOPS, 4),
                        "bound": "mfma" if f > ridge * b else "hbm"}
    ds = stages[dom]
    if ds["bound"] == "mfma":
        roof = {"bound": "mfma", "achieved": ds["TFLOP/s"], "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": ds["frac_mfma"]}
    else:
        roof = {"bound": "hbm", "achieved": ds["GB/s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": ds["frac_hbm"]}
    roof["traffic"] = measured_traffic(dom, cfg.name)
    roof["kernel"] = dom
    roof["ms"] = round(stage_ms[dom], 4)
    # the same figure from the committed rocprofv3 kernel trace of this
    # workload (sum of the stage's kernels' average durations), when it was
    # taken on the current kernel sources
    prof_ms = profiled_stage_ms(dom, cfg.name)
    if prof_ms:
        if ds["bound"] == "mfma":
            prof_frac = ds["flops"] / (prof_ms * 1e-3) / (MFMA_BF16_PEAK_TFLOPS * 1e12)
        else:
            prof_frac = ds["bytes"] / (prof_ms * 1e-3) / (HBM_PEAK_GBS * 1e9)
        roof["profile"] = {"ms": round(prof_ms, 4), "frac": round(prof_frac, 4),
                           "source": f"profiles/kernel_trace_{cfg.name}.md"}
    else:
        roof["profile"] = None
    roof["clock"] = profiled_clock(dom, cfg.name)
    ffn_ms = stage_ms["ffn_up"] + stage_ms["ffn_down"]
    ffn_flops = work["ffn_up"]["flops"] + work["ffn_down"]["flops"]
    ffn_frac_mfma = ffn_flops / (ffn_ms * 1e-3) / (MFMA_BF16_PEAK_TFLOPS * 1e12) if ffn_ms > 0 else 0.0
    ffn_bytes = work["ffn_up"]["bytes"] + work["ffn_down"]["bytes"]
    ffn_frac_hbm = ffn_bytes / (ffn_ms * 1e-3) / (HBM_PEAK_GBS * 1e9) if ffn_ms > 0 else 0.0


    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20)
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    result = {
        "metric": METRIC,
        "value": round(cfg.T / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "timing": "cold steps (1 GiB read before each); GPU time of each step from events around its first "
                  "and last kernels; ms_per_step is their mean; the dominant stage is timed over as many further "
                  "cold steps carrying its own event pair",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg.name, "T": cfg.T, "H": cfg.H, "E": cfg.E, "k": cfg.k, "I": cfg.I,
                   "S": cfg.S, "E_local": cfg.E_local, "n_shared": cfg.n_shared,
                   "I_shared": cfg.I_shared if cfg.n_shared else 0, "parallelism": "single GPU",
                   **({"router": {"gate": ["softmax_topk", "softmax", "sigmoid"][cfg.gate],
                                  "routed_scale": cfg.routed_scale, "n_group": cfg.n_group,
                                  "topk_group": cfg.topk_group, "selection_bias": cfg.gate_bias_std > 0}}
                      if cfg.gated else {})},
        "roofline": roof,
        "expert_ffn": {"ms": round(ffn_ms, 4), "frac_mfma": round(ffn_frac_mfma, 4),
                       "frac_hbm": round(ffn_frac_hbm, 4)},
        "route_permute_frac_hbm": {"route": stages["route"]["frac_hbm"],
                                   "permute": stages["permute"]["frac_hbm"],
                                   "combine": stages["combine"]["frac_hbm"]},
        "stages": stages,
        "cold": {"median_ms": round(cold_sorted[len(cold_sorted) // 2], 4), "min_ms": round(cold_sorted[0], 4),
                 "max_ms": round(cold_sorted[-1], 4), "wall_ms_per_step_with_flush": round(cold_wall_ms, 4)},
        "warm": {"ms_per_step": round(warm_ms, 4), "tokens_per_s": round(cfg.T / (warm_ms * 1e-3), 1),
                 "note": "back-to-back steps, wall clock"},
        "step_gpu_ms_warm_probe": {"median": round(probe_steps[len(probe_steps) // 2], 4),
                                   "min": round(probe_steps[0], 4), "samples": len(probe_steps)},
        "stats_collection": {"route_permute_ms_with_counts": round(rp_stats, 4),
                             "route_permute_ms_without_counts": round(rp_no_stats, 4),
                             "overhead_ms": round(rp_overhead, 4),
                             "overhead_ms_of_means": round(rp_stats - rp_no_stats, 4), "samples": n_probe,
                             "counted_in": "route" if cfg.T * cfg.k <= 512 else "dispatch count pass"},
        **({"gpu_metrics": watch.stop()} if watch else {}),
        "rows_local": R,
        "active_experts": active,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

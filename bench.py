#!/usr/bin/env python3
"""WHTMix forward throughput on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--op OP]

A step is one whtmix_forward call (every kernel of the plan) over one batch of
the workload (default: stereo64k_bf16, B=4, N=65536, C=128, bf16 in/out,
float32 gain and arithmetic).  --op separable / backward / backward_separable
/ module / module_separable / module_backward time the other entry points the
same way (module: the whole block with its W_in / W_out projections, eqs.
(1)-(4)).  Inputs are resident in HBM before timing; the calls run on a
stream of their own (default priority).

Steps rotate over input/output sets whose total footprint is at least twice
the 256 MB Infinity Cache, so every step reads its inputs from HBM (cold).

Prints one JSON line:
- value: GB/s of ideal traffic (read x + read G once + write y) per second of
  wall time over the K timed steps (which carry no HIP events: each event
  record costs the stream about 3 us); tokens/s; fraction of the 8 TB/s peak;
- per_call: median / p10 / p90 of >= 100 further calls, each between two
  HIP events the library records on the launch stream before its first and
  after its last kernel, rotating over the sets (`rotating`), and again with
  a 1 GiB scrub written before each call outside its events (`cold`);
- roofline: the whole call (every kernel of the plan) as the unit: ideal
  bytes over the mean rotating call time; `traffic` is the whole call's
  rocprofv3 FETCH_SIZE + WRITE_SIZE bytes (committed counter record, null when
  taken on other kernel sources) and `traffic_ratio` that over the ideal bytes;
- floor_ms: the three-pass plan's x, float32-workspace and y traffic moved by
  plain PyTorch kernels of the same shapes (widen x, scale the workspace in
  place, narrow into y), without the gain read;
- kernels: each kernel's average time (events between kernels, which add
  about 3 us each) and rate on its own design bytes (x, y, the gain and the
  float32 workspace round trips), not ideal bytes;
- cpu_baseline: the float64 CPU oracle on a bounded sample, on all host cores
  and on one core, with the host CPU model.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0       # MI355X HBM3E peak, GB/s
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense matrix-core peaks
METRIC = "WHTMix forward GB/s and tokens/s at 1 MI355X; % of HBM roofline"
MALL_BYTES = 256 * 1024 * 1024
SCRUB_BYTES = 1 << 30
MAX_SETS = 2048


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Sources the kernels of each path are compiled from: a counter record taken
# on other sources is not reported.
FORWARD_SOURCES = ("whtmix_kernels.hip", "whtmix_tile.h", "whtmix_plan.h", "whtmix_launch.h",
                   "whtmix_wave.hip")
MODULE_SOURCES = FORWARD_SOURCES + ("whtmix_module.hip", "whtmix_module.h")


def kernel_source_hash(files=FORWARD_SOURCES) -> str:
    h = hashlib.sha256()
    for name in sorted(files):
        with open(os.path.join(ROOT, "paper_2607_25234_amd", "csrc", name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def kernel_names(plan: str) -> list[str]:
    return {"three_pass": ["outer_fwd", "middle", "outer_inv"],
            "wave_tiles": ["wave_pass1", "wave_middle", "wave_pass3"],
            "two_pass": ["fold_pass", "wave_pass3"],
            "fused": ["fused"], "small": ["small"], "one_launch": ["one_launch"]}[plan]


def algorithmic_bytes(plan: str, B: int, N: int, C: int, s: int, gbytes: int) -> list[int]:
    """Design bytes each kernel of the forward plan moves (N here is the
    padded token count; gbytes: bytes of the gain read once).  The one-launch
    plan runs all three passes in one kernel, so its design bytes are the
    three-pass plan's summed."""
    L = N * C
    if plan in ("fused", "small"):
        return [B * L * 2 * s + gbytes]
    three = [B * L * (s + 4),           # read x, write float32 workspace
             B * L * 8 + gbytes,        # read + write workspace, read the gain once
             B * L * (4 + s)]           # read workspace, write y
    if plan == "two_pass":
        # the fold pass reads the slice once from memory (its workgroups'
        # re-reads hit L2), reads the gain, writes the workspace
        return [B * L * (s + 4) + gbytes, three[2]]
    return [sum(three)] if plan == "one_launch" else three   # three_pass and wave_tiles


def backward_plan(plan: dict) -> str:
    """The plan the backward pass and the block run for a forward plan: slices
    of 2^16 and more take the three-pass plan, smaller wave-tile shapes the
    one-workgroup plan (the library's rule)."""
    p = plan["plan"]
    if p in ("wave_tiles", "one_launch", "two_pass"):
        return "three_pass" if plan["log2_slice"] >= 16 or p == "one_launch" else "fused"
    if p == "fused" and plan["log2_slice"] >= 16:
        return "three_pass"
    return p


OPS = ("forward", "separable", "backward", "backward_separable", "module", "module_separable",
       "module_backward")


def module_kernels(plan: str, path: str) -> list[str]:
    """Kernels between the events of a whtmix_module_forward call (the weight
    repacking kernel runs before the first event); path: the library's
    module_path for the shape ("small", "mfma" or "unfused")."""
    if plan == "small" or path == "small":
        return ["module_small"]
    if path != "mfma":
        return ["unfused"]
    return ["module_outer_fwd", "middle", "module_outer_inv"] if plan == "three_pass" \
        else ["module_fused"]


def module_algorithmic(names: list[str], B: int, N: int, P: int, C: int, s: int,
                       gbytes: int) -> tuple[list[int], list[int]]:
    """(bytes, MFMA-eligible flops) each kernel of the block must move / do by
    its definition: x, the workspace, y, the gain and each weight matrix once;
    2 N C^2 flops per slice and projection over the real rows."""
    L = P * C
    wb = C * C * s
    proj = 2 * B * N * C * C
    if names == ["module_outer_fwd", "middle", "module_outer_inv"]:
        return ([B * N * C * s + B * L * 4 + wb, B * L * 8 + gbytes, B * L * 4 + B * N * C * s + wb],
                [proj, 0, proj])
    return [2 * B * N * C * s + 2 * wb + gbytes], [2 * proj]


def ideal_bytes(op: str, B: int, N: int, P: int, C: int, s: int) -> int:
    """Ideal HBM bytes of one call: every input read once, every output
    written once (P: padded token count, the gains' extent)."""
    xy = B * N * C * s
    if op == "forward":
        return 2 * xy + 4 * P * C
    if op == "separable":
        return 2 * xy + 4 * (P + C)
    if op == "backward":            # read x, dy, G; write dx, dG
        return 3 * xy + 8 * P * C
    if op == "backward_separable":
        return 3 * xy + 8 * (P + C)
    wb = 2 * C * C * s              # module: also read W_in and W_out
    if op == "module":
        return 2 * xy + 4 * P * C + wb
    if op == "module_backward":     # read x, dy, G, weights; write dx, dG, both dW (f32)
        return 3 * xy + 8 * P * C + wb + 2 * C * C * 4
    return 2 * xy + 4 * (P + C) + wb  # module_separable


def input_sets(footprint: int) -> int:
    """Sets to rotate over so that their total footprint is at least twice
    the Infinity Cache (capped for tiny workloads)."""
    return max(2, min(MAX_SETS, -(-2 * MALL_BYTES // max(1, footprint)) + 1))


def percentiles(v: list[float]) -> dict:
    import numpy as np
    a = np.asarray(v, dtype=np.float64)
    return {"median_ms": round(float(np.median(a)), 5), "p10_ms": round(float(np.percentile(a, 10)), 5),
            "p90_ms": round(float(np.percentile(a, 90)), 5), "calls": int(a.size)}


TRAFFIC_PATH = os.path.join(ROOT, "profiles", "traffic.json")


def load_traffic(kernel: str, workload: str, op: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    path = TRAFFIC_PATH
    if not os.path.exists(path) or op not in ("forward", "module"):
        return None
    with open(path) as f:
        data = json.load(f)
    files = FORWARD_SOURCES if op == "forward" else MODULE_SOURCES
    hashes = data.get("source_hash")
    if not isinstance(hashes, dict) or hashes.get(op) != kernel_source_hash(files):
        return None
    entry = data.get("workloads", {}).get(workload, {}).get(op, {}).get(kernel)
    return None if not isinstance(entry, dict) else entry.get("hbm_bytes_per_launch")


def call_traffic(names: list[str], workload: str, op: str):
    """The whole call's counter bytes: the sum over its kernels, or None when
    any kernel has no current record."""
    parts = [load_traffic(n, workload, op) for n in names]
    return None if any(p is None for p in parts) else int(sum(parts))


class HipEvents:
    """HIP events through the runtime torch already loaded (same soname)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                 ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.events = []

    def create(self) -> int:
        ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")
        self.events.append(ev.value)
        return ev.value

    def record(self, ev: int, stream: int):
        rc = self.hip.hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def destroy(self):
        for ev in self.events:
            self.hip.hipEventDestroy(ev)
        self.events = []


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(w, op: str, host0, io_bytes: int, seconds: float) -> dict:
    """The float64 CPU oracle, as it stands, on one batch slice of the same
    operation, repeated until about `seconds` of work, on all host cores and
    then on one core; scaled to the whole workload's ideal bytes."""
    from oracle import oracle as oracle_mod
    orc = oracle_mod.Oracle()
    x, g, gt, gc, dy, wi, wo = host0
    call = {
        "forward": lambda: orc.whtmix(x, g),
        "separable": lambda: orc.whtmix_separable(x, gt, gc),
        "backward": lambda: orc.whtmix_grad(x, dy, g),
        "backward_separable": lambda: orc.whtmix_grad_separable(x, dy, gt, gc),
        "module": lambda: orc.whtmix_module(x, wi, g, wo),
        "module_backward": lambda: orc.whtmix_module_grad(x, wi, g, wo, dy),
        "module_separable": lambda: orc.whtmix_module_separable(x, wi, gt, gc, wo),
    }[op]

    def timed(budget: float):
        runs, t_total = 0, 0.0
        while runs == 0 or (t_total < budget and runs < 1000):
            t0 = time.perf_counter()
            call()
            t_total += time.perf_counter() - t0
            runs += 1
        t_workload = t_total / runs * w.B
        return runs, t_total, t_workload

    threads = orc.threads()
    runs, t_total, t_wl = timed(seconds * 0.6)
    # one core: skipped when a single run would take far beyond its share
    # of the budget (perfect scaling would make it threads x slower)
    est1 = t_total / runs * threads
    single = None
    if est1 <= 4 * seconds * 0.4:
        prev = orc.set_threads(1)
        runs1, t_total1, t_wl1 = timed(seconds * 0.4)
        orc.set_threads(prev)
        single = {"value": round(io_bytes / t_wl1 / 1e9, 4), "unit": "GB/s",
                  "tokens_per_s": round(w.B * w.N / t_wl1, 1), "cores": 1,
                  "sample": f"{runs1} run(s) of one slice, {t_total1:.1f} s total"}
    else:
        single = {"value": None, "cores": 1,
                  "sample": f"skipped: one run of one slice would take about {est1:.0f} s on one core"}
    return {
        "value": round(io_bytes / t_wl / 1e9, 4),
        "unit": "GB/s",
        "tokens_per_s": round(w.B * w.N / t_wl, 1),
        "cores": threads,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "host_cpus": os.cpu_count(),
        "sample": (f"{runs} run(s) of one of the {w.B} batch slices ({w.N}x{w.C}), "
                   f"{t_total:.1f} s total, float64 C oracle with OpenMP on {threads} threads; "
                   f"rate scaled to the whole {w.B}-slice workload"),
        "single_core": single,
    }


def copy_floor(torch, w, sets, P: int, hip, stream_ptr: int, reps: int = 20) -> dict:
    """The three-pass plan's x, workspace and y traffic done by plain PyTorch
    kernels on buffers of the same shapes: x widened into a float32 buffer,
    that buffer scaled in place, then narrowed into y (medians).  The gain's
    read (4 N_pad C bytes once) is not in it."""
    ws = torch.empty((w.B, P, w.C), dtype=torch.float32, device=sets[0]["x"].device)
    n = w.N
    ev = [hip.create() for _ in range(4)]
    acc = [[], [], []]
    for r in range(reps):
        t = sets[r % len(sets)]
        hip.record(ev[0], stream_ptr)
        ws[:, :n].copy_(t["x"])
        hip.record(ev[1], stream_ptr)
        ws.mul_(1.5)
        hip.record(ev[2], stream_ptr)
        t["y"].copy_(ws[:, :n])
        hip.record(ev[3], stream_ptr)
        torch.cuda.synchronize()
        for j in range(3):
            acc[j].append(hip.elapsed_ms(ev[j], ev[j + 1]))
    import numpy as np
    med = [float(np.median(a)) for a in acc]
    del ws
    return {"floor_ms": round(sum(med), 5),
            "parts_ms": {"widen_copy": round(med[0], 5), "inplace_scale": round(med[1], 5),
                         "narrow_copy": round(med[2], 5)},
            "note": "PyTorch copy_ / mul_ kernels moving x, the float32 workspace and y as the "
                    "three passes do, without the gain read"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--plan", default="auto")
    ap.add_argument("--op", default="forward", choices=OPS,
                    help="forward (joint gain, the default), separable (log gains), "
                         "backward, backward_separable, module (the block with its "
                         "projections), module_separable, module_backward")
    ap.add_argument("--sets", type=int, default=0,
                    help="input/output sets rotated over the steps (0 = auto)")
    ap.add_argument("--event-every", type=int, default=4,
                    help="record per-kernel HIP events on every n-th timed step")
    ap.add_argument("--calls", type=int, default=100,
                    help="per-call event pairs for the distribution (at least 100)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=14.0)
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the WHTMix path here is built and "
              "timed on a single MI355X (batch slices would shard across GPUs with "
              "no communication). Run with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2607_25234_amd import whtmix, workloads

    name = args.workload or workloads.BENCH_WORKLOAD
    w = workloads.WORKLOADS[name]
    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    whtmix.lib()
    s = 2 if w.dtype == "bf16" else 4
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dt_code = whtmix.DTYPE_BF16 if w.dtype == "bf16" else whtmix.DTYPE_F32
    plan = whtmix.plan_describe(w.B, w.N, w.C, w.dtype, args.plan)
    P = plan["padded_tokens"]
    op = args.op
    io_bytes = ideal_bytes(op, w.B, w.N, P, w.C, s)
    nsets = args.sets or input_sets(io_bytes)
    ndrawn = min(nsets, 4)
    log(f"workload {name}: B={w.B} N={w.N} C={w.C} {w.dtype}; op {op}; plan {plan}; "
        f"{nsets} input sets ({ndrawn} drawn, the rest device copies)")

    wi_h, wo_h = workloads.draw_weights(w.C, w.dtype, w.seed + 50)
    w_in = torch.from_numpy(wi_h).to(dev).to(tdt)
    w_out = torch.from_numpy(wo_h).to(dev).to(tdt)
    sets = []
    for i in range(nsets):
        if i >= ndrawn:
            sets.append({k: v.clone() for k, v in sets[i % ndrawn].items()})
            continue
        if i == 0:
            x, g = workloads.inputs(w)
        else:
            x, g = workloads.draw(w.B, w.N, w.C, w.dtype, w.seed + 1000 * i, w.x_dist)
        gt, gc = workloads.draw_log_gains(P, w.C, w.seed + 1000 * i + 1)
        dy = None
        if "backward" in op:
            dy, _ = workloads.draw(w.B, w.N, w.C, w.dtype, w.seed + 1000 * i + 2)
        t = {"x": torch.from_numpy(x).to(dev).to(tdt), "g": torch.from_numpy(g).to(dev),
             "gt": torch.from_numpy(gt).to(dev), "gc": torch.from_numpy(gc).to(dev)}
        t["y"] = torch.empty_like(t["x"])
        if dy is not None:
            t["dy"] = torch.from_numpy(dy).to(dev).to(tdt)
            t["dg"] = torch.empty_like(t["g"])
            t["dgt"], t["dgc"] = torch.empty_like(t["gt"]), torch.empty_like(t["gc"])
        if op == "module_backward":
            t["dwi"] = torch.empty((w.C, w.C), device=dev)
            t["dwo"] = torch.empty((w.C, w.C), device=dev)
        sets.append(t)
        if i == 0:
            host0 = (x[0].copy(), g.copy(), gt, gc, None if dy is None else dy[0].copy(),
                     wi_h, wo_h)
        del x, g
    torch.cuda.synchronize()

    # A stream of its own (default priority): every call, event, scrub and
    # floor kernel below is ordered on it.
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.set_stream(stream)
    sptr = stream.cuda_stream
    hip = HipEvents()
    if op.startswith("backward"):
        nk, names = 2, (["fwd_transforms_gain_gradient", "dx_outer_inv"]
                        if backward_plan(plan) == "three_pass" else ["gain_gradient", "dx"])
    elif op == "module_backward":
        nk, names = 3, (["transforms_and_gain_gradient", "z_prime_and_dw_out", "dx_and_dw_in"]
                        if plan["module_backward_fused"] else
                        ["recompute_and_dw_out", "mixer_gradients", "dx_and_dw_in"])
    elif op.startswith("module"):
        # the block runs 2^16-element slices with the three-pass plan even
        # where the mixer's forward takes another plan
        names = module_kernels("three_pass" if plan["module_outer_bits"] else backward_plan(plan),
                               plan["module_path"])
        nk = len(names)
    else:
        nk, names = plan["kernels"], kernel_names(plan["plan"])

    # device addresses resolved once per set, as a serving loop holds them
    ptrs = [{k: v.data_ptr() for k, v in t.items()} for t in sets]
    p_in, p_out = w_in.data_ptr(), w_out.data_ptr()

    def step(i, events=None):
        t = ptrs[i % nsets]
        B, N, C = w.B, w.N, w.C
        if op == "forward":
            st = whtmix.forward_raw(t["x"], t["g"], t["y"],
                                    B, N, C, dt_code, sptr, args.plan, events)
        elif op == "separable":
            st = whtmix.forward_separable_raw(t["x"], t["gt"],
                                              t["gc"], t["y"], B, N, C,
                                              dt_code, sptr, args.plan, events)
        elif op == "backward":
            st = whtmix.backward_raw(t["x"], t["dy"], t["g"],
                                     t["y"], t["dg"], B, N, C, dt_code,
                                     sptr, args.plan, events)
        elif op == "module":
            st = whtmix.module_forward_raw(t["x"], p_in, t["g"],
                                           p_out, t["y"], B, N, C,
                                           dt_code, sptr, args.plan, events)
        elif op == "module_backward":
            st = whtmix.module_backward_raw(
                t["x"], p_in, t["g"], p_out,
                t["dy"], t["y"], t["dwi"], t["dwo"],
                t["dg"], B, N, C, dt_code, sptr, args.plan, events)
        elif op == "module_separable":
            st = whtmix.module_forward_separable_raw(
                t["x"], p_in, t["gt"], t["gc"],
                p_out, t["y"], B, N, C, dt_code, sptr, args.plan, events)
        else:
            st = whtmix.backward_separable_raw(
                t["x"], t["dy"], t["gt"], t["gc"],
                t["y"], t["dgt"], t["dgc"], B, N, C, dt_code,
                sptr, args.plan, events)
        if st != whtmix.SUCCESS:
            raise whtmix.WhtmixError(st, f"whtmix {op}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Timed steps: no HIP events inside them (each event record costs the
    # stream about 3 us, measured), only the host clock around the K steps.
    torch.cuda.synchronize()            # barrier (one rank) + device sync
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # Per-call distribution: >= 100 further calls on the same stream and sets,
    # each between two HIP events the library records before its first and
    # after its last kernel; then the same with a 1 GiB scrub written before
    # each call, outside its events (cold caches).
    ncalls = max(100, args.calls)
    base = args.warmup + args.steps
    pairs = [[hip.create()] + [None] * (nk - 1) + [hip.create()] for _ in range(ncalls)]
    for i in range(ncalls):
        step(base + i, pairs[i])
    torch.cuda.synchronize()
    rotating = [hip.elapsed_ms(e[0], e[nk]) for e in pairs]
    scrub = torch.empty(SCRUB_BYTES, dtype=torch.uint8, device=dev)
    cold_pairs = [[hip.create()] + [None] * (nk - 1) + [hip.create()] for _ in range(ncalls)]
    for i in range(ncalls):
        scrub.fill_(i & 0xff)
        step(base + ncalls + i, cold_pairs[i])
    torch.cuda.synchronize()
    cold = [hip.elapsed_ms(e[0], e[nk]) for e in cold_pairs]
    del scrub
    avg_call = float(np.mean(rotating))

    # Per-kernel split: events between the kernels on a sample of calls
    # (--event-every of them out of 4x as many); each inner event adds about
    # 3 us to the kernel after it, so these sum above the call time.
    every = max(1, args.event_every)
    kev = [[hip.create() for _ in range(nk + 1)] if i % every == 0 else None
           for i in range(4 * every * 8)]
    for i, e in enumerate(kev):
        step(base + 2 * ncalls + i, e)
    torch.cuda.synchronize()
    sampled = [e for e in kev if e is not None]
    per_kernel = [float(np.mean([hip.elapsed_ms(e[j], e[j + 1]) for e in sampled]))
                  for j in range(nk)]

    floor = None
    if op == "forward" and plan["plan"] in ("three_pass", "one_launch", "wave_tiles", "two_pass"):
        floor = copy_floor(torch, w, sets, P, hip, sptr)
    hip.destroy()

    ms_per_step = wall * 1e3 / args.steps
    gbs = io_bytes / (ms_per_step * 1e-3) / 1e9
    tokens = w.B * w.N / (ms_per_step * 1e-3)
    flops = None
    if op in ("forward", "separable"):
        gbytes = 4 * P * w.C if op == "forward" else 4 * (P + w.C)
        alg = algorithmic_bytes(plan["plan"], w.B, P, w.C, s, gbytes)
    elif op == "module_backward":
        alg = [0] * nk      # phases recompute design-specific float32 intermediates
    elif op.startswith("module"):
        gbytes = 4 * P * w.C if op == "module" else 4 * (P + w.C)
        alg, flops = module_algorithmic(names, w.B, w.N, P, w.C, s, gbytes)
    elif backward_plan(plan) == "three_pass":
        # fused three-pass gradients: phase 1 = OUTER_FWD of x and dy (read
        # both, write two float32 workspaces) + the middle pass (read both
        # workspaces and the gain, write dY's back and the gain gradient);
        # phase 2 = OUTER_INV of dY's workspace into dx
        gb = 4 * P * w.C if op == "backward" else 4 * (P + w.C)
        L = P * w.C
        xb = w.B * w.N * w.C * s
        alg = [2 * xb + 8 * w.B * L + 12 * w.B * L + gb + 4 * L, 4 * w.B * L + xb]
    else:
        # gain-gradient phase: read x and dy, write the gain gradient;
        # dx phase: the forward mixer applied to dy
        gb = 4 * P * w.C if op == "backward" else 4 * (P + w.C)
        alg = [2 * w.B * w.N * w.C * s + gb, 2 * w.B * w.N * w.C * s + gb]

    achieved = io_bytes / (avg_call * 1e-3) / 1e9
    traffic = call_traffic(names, name, op)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "op": op, "B": w.B, "N": w.N, "C": w.C,
                   "io_dtype": w.dtype, "gain_dtype": "f32", "plan": plan["plan"],
                   "input_sets": nsets},
        "tokens_per_s": round(tokens, 1),
        "hbm_peak_frac": round(gbs / PEAK_HBM_GBS, 4),
        "roofline": {"bound": "hbm", "kernel": "whole call (" + " + ".join(names) + ")",
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "alg_bytes": io_bytes, "avg_call_ms": round(avg_call, 5),
                     "traffic": traffic,
                     "traffic_ratio": None if traffic is None else round(traffic / io_bytes, 3)},
        "per_call": {"rotating": percentiles(rotating), "cold": percentiles(cold)},
        "timing": "timed steps carry no events; the call time is the mean of the rotating "
                  "per-call event pairs; kernel times come from separate calls with events "
                  "between their kernels (about 3 us each)",
        "floor_ms": None if floor is None else floor["floor_ms"],
        "floor": floor,
        "event_sampled_steps": len(sampled),
        "kernels": [{"name": n, "avg_ms": round(t, 5), "design_bytes": b,
                     "design_GBs": round(b / (t * 1e-3) / 1e9, 1) if b else None}
                    for n, t, b in zip(names, per_kernel, alg)],
        "matrix_core": None if flops is None else {
            "alg_TFLOPs_per_kernel": [round(f / (t * 1e-3) / 1e12, 2)
                                      for f, t in zip(flops, per_kernel)],
            "peak_TFLOPs": PEAK_MFMA_TFLOPS[w.dtype],
            "note": "projection flops (2 N C^2 per slice each) over the kernel time; "
                    "the kernels stay HBM-bound"},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on one batch slice ...")
        out["cpu_baseline"] = cpu_baseline(w, op, host0, io_bytes, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

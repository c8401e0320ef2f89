"""Benchmark of the AGS step + gradient statistics on one MI355X.

Workload: ResNet-50 ImageNet layout (161 tensors, 25,557,032 parameters),
K = 16 bf16 replica gradients, fp32 weights and momentum, AGS mode.  A step
is one full pass of the hot path: replica mean, per-layer statistics,
decision and update (the step kernel, the finalize kernel and the correction
pass, which exits at once when the sensitive bit was predicted right, on one
stream).  Inputs are seeded and
synthetic and already resident in HBM when timing starts; the timed steps
reuse one generated gradient set.

Prints one JSON line (last line of stdout):
  value          algorithmic GB/s of the whole step: (K*2 + 16) bytes per
                 parameter per step (each replica read once, w and m read and
                 written once) over the measured step time
  roofline       the dominant kernel's algorithmic bytes per launch over its
                 average duration (start and stop events of its own dispatch
                 on the launch stream), against
                 the 8 TB/s HBM peak; traffic = HBM bytes per launch from
                 rocprofv3 FETCH_SIZE/WRITE_SIZE (committed summary), or null
                 when the kernels changed since it was taken; also as a
                 fraction of two ceilings measured on this GPU by the
                 package's hbm_probe (random data): a read-only stream, and
                 the step's own byte pattern with trivial arithmetic
  hbm_probe      those measured ceilings (and a copy), GB/s
  cold_cache     single steps after a 1 GiB read evicts the caches
  sensitive_phase_steps, mispredicted_steps
                 steps whose decisions are all sensitive (predicted from the
                 last decision, so corrected only once) and alternate (every
                 step corrected: the worst case)
  cpu_baseline   the float64 oracle on the host on whole steps of the same
                 workload (a reported baseline, not a target): on every host
                 core (the layers split into one group per core, each group
                 stepped by the unchanged single-threaded oracle on a thread
                 of its own), and on one thread
  configs        the other configurations in AGS mode (tiny CNN K=4 fp32,
                 ResNet-18 CIFAR K=8 fp32, VGG-16 K=8 fp32, the ResNet-50
                 sweep K=1..64 bf16): microseconds per step warm and cold,
                 GB/s and fraction of peak for both, the kernel split

With --elementwise the scale of Algorithm 1 is kept per parameter element
(AGS mode): a step also reads the scales in force and writes the refreshed
ones, (K*2 + 24) bytes per parameter.

Usage: python bench.py [--gpus 1] [--steps 200] [--warmup 20]
                       [--no-cpu-baseline] [--no-probe] [--no-configs] [--copy-probe]
                       [--elementwise]
                       [--delta-scope global|layer] [--mode ags|sgd|lars|static]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
#: name -> (layout, K, gradient dtype, description).  The default is the
#: headline workload; the others are the remaining configurations.
WORKLOADS = {
    "resnet50_k16_bf16": ("resnet50", 16, "bf16",
                          "ResNet-50 ImageNet layout (161 tensors, 25,557,032 params), K=16 bf16"),
    "tiny_cnn_k4_f32": ("tiny_cnn", 4, "f32", "tiny CNN layout (8 tensors, 24,234 params), K=4 fp32"),
    "resnet18_cifar_k8_f32": ("resnet18_cifar", 8, "f32",
                              "ResNet-18 CIFAR layout (62 tensors, 11,173,962 params), K=8 fp32"),
    "vgg16_k8_f32": ("vgg16", 8, "f32", "VGG-16 layout (32 tensors, 138,357,544 params), K=8 fp32"),
}
for _k in (1, 2, 4, 8, 32, 64):
    WORKLOADS[f"resnet50_k{_k}_bf16"] = ("resnet50", _k, "bf16",
                                         f"ResNet-50 ImageNet layout, K={_k} bf16 (batch sweep)")
WORKLOAD = "resnet50_k16_bf16"
K = 16
E_G = 2  # bytes per gradient element of the selected workload
HYPER = dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8, s_max=0.0,
             trust_coef=1e-3, refresh_every=1, small_replica=0)
KERNEL_SOURCE = os.path.join(ROOT, "paper_2603_18112_amd", "csrc", "ags_kernels.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for p in (KERNEL_SOURCE, os.path.join(ROOT, "paper_2603_18112_amd", "csrc", "ags_internal.h")):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(n_params: int, mode: str = "ags", elementwise: bool = False,
                      reuse_w_norms: bool = True):
    """Per-launch algorithmic bytes of each kernel and of the whole step.

    A step reads every replica once and reads and writes w and m once:
    (K * e_g + 16) bytes per parameter.  AGS and SGD steps do all of it in
    the step kernel; the finalize kernel moves only per-tile partials, and
    the correction pass moves nothing on the steps timed here, whose
    sensitive bit is predicted right.  A LARS step reads the replicas and w
    in the step kernel (and writes the replica mean when K * e_g > 8), then
    reads w, m and the mean (or the replicas again) and writes w, m in the
    update pass; with reuse_w_norms (the steps timed here) the first pass
    takes the weight norms from the update pass before it and does not read
    w.  Element scales add a 4-byte read of the scale in force and
    a 4-byte write of the refreshed one per parameter (refresh every step,
    scales applied: the steps timed here)."""
    step = n_params * (K * E_G + 16 + (8 if elementwise else 0))
    if mode != "lars":
        return {"step": step, "finalize": 0, "second_pass": 0, "whole_step": step}
    mat = K * E_G > 8
    k0 = n_params * (K * E_G + (0 if reuse_w_norms else 4) + (4 if mat else 0))
    k2 = n_params * ((4 if mat else K * E_G) + 16)
    return {"step": k0, "finalize": 0, "second_pass": k2, "whole_step": step}


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")


def workload_key(workload: str, elementwise: bool, delta_scope: str = "global",
                 mode: str = "ags") -> str:
    """Name of the committed counter summary for a run.  SGD and static
    steps run the AGS step kernel (only the coefficients differ), so they
    share its summary; LARS runs other kernels and has its own."""
    return (workload + ("_elementwise" if elementwise else "")
            + ("_layer_delta" if delta_scope == "layer" else "")
            + ("_lars" if mode == "lars" else ""))


def read_traffic(workload: str, kernel: str):
    """HBM bytes per launch of ``kernel`` from the committed counter summary
    of ``workload``, if it was taken on the current kernel source."""
    try:
        kv = {}
        with open(traffic_file(workload)) as f:
            for line in f:
                if "=" in line and not line.lstrip().startswith("#"):
                    k, v = line.split("=", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("kernel_source_sha") != kernel_source_sha():
            return None
        v = kv.get(f"{kernel}_hbm_bytes_per_launch")
        return float(v) if v else None
    except OSError:
        return None


def hbm_probe(K: int, grad_dtype: str, n_elements: int, elementwise: bool = False):
    """Streaming-bandwidth ceilings of this GPU from the package's hbm_probe
    program (random data: read-only, copy, and the step's own byte pattern
    for K replica rows of grad_dtype over n_elements with trivial
    arithmetic, with the element-scale streams when elementwise), run as a
    child process before this process touches the GPU; None if it is not
    built."""
    from paper_2603_18112_amd import _build
    import subprocess
    if not os.path.exists(_build.PROBE):
        return None
    cmd = [_build.PROBE, str(K), grad_dtype, str(n_elements)] + (["ew"] if elementwise else [])
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=180)
    if r.returncode != 0:
        log(f"hbm_probe failed: {r.stderr.strip()}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def copy_probe(torch, nbytes=1 << 30, reps=20):
    """Device-to-device copy bandwidth (read + write bytes / time)."""
    n = nbytes // 4
    a = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2 * n * 4 / (ms * 1e-3) / 1e9


def host_cores() -> int:
    """Host cores this process may run on (its affinity mask)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def split_layers(numels, parts):
    """Layers into at most ``parts`` groups of nearly equal element counts
    (largest first onto the lightest group); groups keep layer order."""
    import heapq
    parts = max(1, min(parts, len(numels)))
    heap = [(0, i) for i in range(parts)]
    groups = [[] for _ in range(parts)]
    for l in sorted(range(len(numels)), key=lambda l: -int(numels[l])):
        load, i = heapq.heappop(heap)
        groups[i].append(l)
        heapq.heappush(heap, (load + int(numels[l]), i))
    return [sorted(g) for g in groups if g]


def cpu_baseline_parallel(layout, w0, grads_np, cores, budget_s=15.0, max_steps=30):
    """The float64 oracle as it stands, on all host cores: the layers are
    split into ``cores`` groups of nearly equal size, each group is a model
    of its own (its layers packed end to end, with its share of every
    replica), and one thread per group runs the unchanged single-threaded
    oracle on it; the oracle is C called through ctypes, which releases the
    interpreter lock, so the groups' steps run in parallel.  A group takes
    its own Delta and decision over its layers (O(layers) work); the
    per-element work of a step is the whole model's.  Returns the median
    wall time of a whole parallel step, the steps timed and the threads."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    from oracle import OracleAGS
    table = layout.table()
    groups = split_layers([n for _, n, _ in table], cores)
    oracles, gsub = [], []
    for grp in groups:
        sub, o = [], 0
        for l in grp:
            n = table[l][1]
            sub.append((o, n, table[l][2]))
            o += (n + 7) // 8 * 8
        w_sub = np.zeros(o, np.float32)
        g_sub = np.zeros((grads_np.shape[0], o), grads_np.dtype)
        for (so, n, _), l in zip(sub, grp):
            lo = table[l][0]
            w_sub[so:so + n] = w0[lo:lo + n]
            g_sub[:, so:so + n] = grads_np[:, lo:lo + n]
        oracles.append(OracleAGS(sub, o, K, w_sub, grad_dtype="bf16" if E_G == 2 else "f32",
                                 **HYPER))
        gsub.append(g_sub)
    times = []
    with ThreadPoolExecutor(len(groups)) as ex:
        t_start = time.time()
        while len(times) < max_steps and (time.time() - t_start) < budget_s:
            t0 = time.perf_counter()
            list(ex.map(lambda i: oracles[i].step(gsub[i]), range(len(groups))))
            times.append(time.perf_counter() - t0)
    return sorted(times)[len(times) // 2], len(times), len(groups)


def cpu_baseline(layout, w0, grads_np, budget_s=20.0, max_steps=30):
    """The float64 oracle as it stands, single-threaded, on whole steps."""
    from oracle import OracleAGS
    o = OracleAGS(layout.table(), layout.n_flat, K, w0, grad_dtype="bf16" if E_G == 2 else "f32",
                  **HYPER)
    times = []
    t_start = time.time()
    while len(times) < max_steps and (time.time() - t_start) < budget_s:
        t0 = time.perf_counter()
        o.step(grads_np)
        times.append(time.perf_counter() - t0)
    sec = sorted(times)[len(times) // 2]
    return sec, len(times)


def time_config(h, g, stream, torch, steps, warmup, flush, n_cold=20):
    """Whole-step times of one handle: warm (back-to-back steps, mean over
    ``steps``), cold (median of single steps, each after ``flush`` is read
    with ordinary loads, which evicts the L2s and the Infinity Cache), and
    each kernel's average duration from its own dispatch events."""
    for _ in range(warmup):
        h.step(g, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        h.step(g, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    warm = e0.elapsed_time(e1) / steps
    h.set_profiling(True)
    h.kernel_times()
    for _ in range(steps):
        h.step(g, stream)
    torch.cuda.synchronize()
    kms, ncalls = h.kernel_times()
    h.set_profiling(False)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n_cold)]
    for a0, a1 in ev:
        flush.sum()
        a0.record(stream)
        h.step(g, stream)
        a1.record(stream)
    torch.cuda.synchronize()
    cold = sorted(a0.elapsed_time(a1) for a0, a1 in ev)[n_cold // 2]
    from paper_2603_18112_amd import ags
    return warm, cold, {n: round(kms[i] / ncalls * 1e3, 2) for i, n in enumerate(ags.KERNEL_NAMES)}


def measure_configs(torch, np, stream, steps, warmup):
    """Every configuration besides the headline, in AGS mode: the tiny CNN
    (K = 4 fp32), ResNet-18 CIFAR (K = 8 fp32), VGG-16 (K = 8 fp32) and the
    ResNet-50 batch-size sweep (K = 1..64 bf16; the first K replicas of one
    K = 64 draw, which are the bytes a K-replica draw gives).  Per
    configuration: whole-step microseconds warm and cold, algorithmic GB/s
    and fraction of the 8 TB/s peak for both, steps/s, the per-kernel split;
    for the sweep also the median over layers of >= 1000 elements of the
    noise ratio V_l / G_l against its expectation c^2 (K-1) / (K + c^2)
    under the generator (c = 0.5)."""
    from paper_2603_18112_amd import ags, layouts, synth
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    out = {}

    def run(name, lay, k, gdt, g, noise_check=False):
        w = torch.from_numpy(synth.init_weights(lay, 0)).cuda()
        m = torch.zeros_like(w)
        h = ags.AGS(lay.table(), w, m, k, grad_dtype=gdt, mode="ags",
                    **{**HYPER, "elementwise": False, "delta_scope": "global"})
        warm, cold, ksplit = time_config(h, g, stream, torch, steps, warmup, flush)
        nbytes = lay.n_params * (k * (2 if gdt == "bf16" else 4) + 16)
        rec = {"K": k, "grad_dtype": gdt, "params": lay.n_params, "bytes_per_step": nbytes,
               "us_warm": round(warm * 1e3, 2), "us_cold": round(cold * 1e3, 2),
               "GBps_warm": round(nbytes / (warm * 1e-3) / 1e9, 1),
               "GBps_cold": round(nbytes / (cold * 1e-3) / 1e9, 1),
               "peak_frac_warm": round(nbytes / (warm * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
               "peak_frac_cold": round(nbytes / (cold * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
               "steps_per_s": round(1e3 / warm, 1), "kernel_us": ksplit}
        if noise_check:
            big = np.array([n >= 1000 for _, n, _ in lay.table()])
            rho = np.asarray(h.read_stats().layer["noise_ratio"])[big]
            rec["noise_ratio_median"] = round(float(np.median(rho)), 6)
            rec["noise_ratio_expected"] = round(0.25 * (k - 1) / (k + 0.25), 6)
        h.close()
        del w, m
        out[name] = rec
        log(f"config {name}: {rec['us_warm']} us warm, {rec['us_cold']} us cold "
            f"({rec['peak_frac_warm']:.3f} / {rec['peak_frac_cold']:.3f} of peak)")

    for name, lname, k, gdt in (("tiny_cnn_k4_f32", "tiny_cnn", 4, "f32"),
                                ("resnet18_cifar_k8_f32", "resnet18_cifar", 8, "f32"),
                                ("vgg16_k8_f32", "vgg16", 8, "f32")):
        lay = layouts.get_layout(lname)
        g_np = synth.replica_grads(lay, k, 0, 0, dtype=gdt, stride=layouts.replica_stride(lay))
        g = torch.from_numpy(g_np).cuda()
        del g_np
        run(name, lay, k, gdt, g)
        del g
    lay = layouts.get_layout("resnet50")
    g_np = synth.replica_grads(lay, max(PLAN_KS), 0, 0, dtype="bf16",
                               stride=layouts.replica_stride(lay))
    g_all = torch.from_numpy(g_np.view(np.int16)).cuda()
    del g_np
    for k in PLAN_KS:
        run(f"resnet50_k{k}_bf16", lay, k, "bf16", g_all[:k], noise_check=True)
    del g_all, flush
    return out


PLAN_KS = (1, 2, 4, 8, 16, 32, 64)
PLAN_NOISES = (0.1, 0.5, 2.0)


def run_plan(args, torch, np):
    """The planner on this library's own step times: ResNet-50 layout, bf16
    replicas, AGS, K = 1..64.  On one GPU the K replicas stand in for K
    workers and the device reads every worker's gradient, the centralized
    form of Eq. (2c): t(K) = c0 + c_sync K.  Full search fits every K,
    partial search the extremes (K = 1 and 64) only; both predict every K.
    The knee of the time per replica gradient, t(K) / K, over K is where
    more replicas per step stop amortising the step's fixed costs.

    The sweep also checks the statistics the step computes: for noise c in
    {0.1, 0.5, 2.0} (per-replica noise std in units of the layer's sigma)
    and every K, the per-layer noise ratio rho_l = V_l / G_l of an ags_stats
    call against its expectation under the generator, c^2 (K - 1) / (K + c^2)
    (median and largest relative deviation over the layers of at least 1000
    elements)."""
    from paper_2603_18112_amd import ags, layouts, plan, synth
    lay = layouts.get_layout("resnet50")
    N = lay.n_params
    stride = layouts.replica_stride(lay)
    kmax = max(PLAN_KS)
    t0 = time.time()
    g_np = synth.replica_grads(lay, kmax, 0, 0, dtype="bf16", stride=stride)
    g_all = torch.from_numpy(g_np.view(np.int16)).cuda()
    del g_np
    log(f"plan: {kmax} bf16 replicas generated in {time.time() - t0:.1f}s")
    w0 = synth.init_weights(lay, 0)
    steps = max(20, min(args.steps, 200))
    hyper = dict(HYPER)
    measured = {}
    noise_sets = {}
    for c in PLAN_NOISES:
        if c == 0.5:
            noise_sets[c] = g_all                      # the timing set: synth's default c
        else:
            g_c = synth.replica_grads(lay, kmax, 0, 0, noise=c, dtype="bf16", stride=stride)
            noise_sets[c] = torch.from_numpy(g_c.view(np.int16)).cuda()
            del g_c
    big = np.array([n >= 1000 for _, n, _ in lay.table()])
    rho_rows = []
    for k in PLAN_KS:
        w = torch.from_numpy(w0.copy()).cuda()
        m = torch.zeros_like(w)
        g = g_all[:k]
        h = ags.AGS(lay.table(), w, m, k, grad_dtype="bf16", mode="ags", **hyper)
        stream = torch.cuda.current_stream()
        for _ in range(args.warmup):
            h.step(g, stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            h.step(g, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        measured[k] = e0.elapsed_time(e1) / steps * 1e-3
        for c in PLAN_NOISES:
            h.stats(noise_sets[c][:k], stream)
            rho = np.asarray(h.read_stats().layer["noise_ratio"])[big]
            expect = c * c * (k - 1) / (k + c * c)
            if expect > 0:
                dev = np.abs(rho / expect - 1.0)
                rho_rows.append({"K": k, "c": c, "expected": round(expect, 6),
                                 "median_rho": round(float(np.median(rho)), 6),
                                 "max_rel_dev": round(float(dev.max()), 4)})
            else:
                rho_rows.append({"K": k, "c": c, "expected": 0.0,
                                 "median_rho": round(float(np.median(rho)), 6),
                                 "max_abs": float(np.abs(rho).max())})
        h.close()
        del w, m
        log(f"plan: K={k}: {measured[k] * 1e6:.1f} us/step")
    samples = [(k, 0.0, measured[k]) for k in PLAN_KS]
    terms = plan.AGS_PLAN_INTERCEPT | plan.AGS_PLAN_SYNC
    tf = time.perf_counter()
    full = plan.ags_plan_fit(samples, "ps", terms)
    fit_us = (time.perf_counter() - tf) * 1e6
    part = plan.ags_plan_fit([s for s in samples if s[0] in (PLAN_KS[0], PLAN_KS[-1])], "ps", terms)

    def report(model):
        rows, worst = [], 0.0
        for k in PLAN_KS:
            pred = plan.ags_plan_step_time(model, k, 0.0)
            err = pred / measured[k] - 1.0
            worst = max(worst, abs(err))
            rows.append({"K": k, "measured_us": round(measured[k] * 1e6, 2),
                         "predicted_us": round(pred * 1e6, 2), "rel_err": round(err, 4)})
        return {"c0_us": round(model.c0 * 1e6, 3), "c_sync_us_per_replica": round(model.c_sync * 1e6, 3),
                "rms_residual_us": round(model.rms_residual * 1e6, 3),
                "max_abs_rel_err": round(worst, 4), "per_K": rows}

    ks = np.array(PLAN_KS, dtype=np.float64)
    per_rep = np.array([measured[k] / k for k in PLAN_KS])
    knee = plan.ags_plan_knee(ks, per_rep, "convex_dec", 1.0)
    bytes_per_step = {k: N * (k * 2 + 16) for k in PLAN_KS}
    out = {
        "metric": "planner step-time model on measured AGS steps (ResNet-50 layout, bf16, K sweep)",
        "unit": "relative error",
        "value": round(report(part)["max_abs_rel_err"], 4),
        "higher_is_better": False,
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "data": "synthetic",
        "config": {"workload": "resnet50_bf16_ksweep", "K": list(PLAN_KS), "mode": "ags",
                   "model": "t(K) = c0 + c_sync * K (Eq. (2), centralized sync term)"},
        "full_search": report(full),
        "partial_search": report(part),
        "knee": {"K": None if knee is None else PLAN_KS[knee],
                 "curve": "seconds per replica gradient t(K)/K over K (Kneedle, convex decreasing)",
                 "per_replica_us": [round(x * 1e6, 2) for x in per_rep]},
        "algorithmic_GBps": {str(k): round(bytes_per_step[k] / measured[k] / 1e9, 1) for k in PLAN_KS},
        "noise_ratio": {"expected": "c^2 (K - 1) / (K + c^2)", "layers": int(big.sum()),
                        "per_K_and_c": rho_rows},
        "fit_call_us": round(fit_us, 2),
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default=WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--mode", default="ags", choices=["ags", "sgd", "lars", "static"])
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured once in a HIP graph and replayed")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the hbm_probe child process (for runs under a profiler, whose "
                         "preloaded library has already initialised the GPU in this process)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run the 1 GiB device copy (counter calibration)")
    ap.add_argument("--elementwise", action="store_true",
                    help="AGS with one scale per parameter element")
    ap.add_argument("--delta-scope", default="global", choices=["global", "layer"],
                    help="variability measure that decides a layer: global Delta or Delta_l")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the timing of the other configurations (tiny CNN, ResNet-18, "
                         "VGG-16, the ResNet-50 K sweep) that the default run reports")
    ap.add_argument("--plan", action="store_true",
                    help="time the ResNet-50 bf16 step for K = 1..64 and fit the planner's "
                         "step-time model to it (full and partial search), then its knee")
    args = ap.parse_args()
    if args.elementwise and args.mode != "ags":
        print("--elementwise needs --mode ags", file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the hot path measured here is the "
              f"single-GPU AGS step (got --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2603_18112_amd import ags, layouts, synth

    probe = None
    if not (args.copy_probe or args.plan or args.no_probe):
        p_lay, p_k, p_dt, _ = WORKLOADS[args.workload]
        probe = hbm_probe(p_k, p_dt, layouts.get_layout(p_lay).n_params, bool(args.elementwise))
    if probe:
        log(f"hbm probe (random data): read {probe['read_GBps']} GB/s, copy {probe['copy_GBps']} GB/s, "
            f"the step's byte pattern {probe['step_pattern_GBps']} GB/s "
            f"(cold {probe.get('step_pattern_cold_GBps')} GB/s)")

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_probe:
        bw = copy_probe(torch)
        log(f"copy probe: {bw:.1f} GB/s")
        print(json.dumps({"copy_probe_GBps": round(bw, 1), "bytes_per_copy": 2 * (1 << 30)}))
        return

    if args.plan:
        run_plan(args, torch, np)
        return

    global K, E_G
    layout_name, K, gdt, desc = WORKLOADS[args.workload]
    E_G = 2 if gdt == "bf16" else 4
    HYPER["elementwise"] = bool(args.elementwise)
    if args.mode == "lars":
        HYPER["reuse_w_norms"] = True   # the weight norms carried from the update pass
    HYPER["delta_scope"] = args.delta_scope
    wkey = workload_key(args.workload, args.elementwise, args.delta_scope, args.mode)
    lib = ags.load_library()
    log(f"libags: {ags.library_path()}")
    lay = layouts.get_layout(layout_name)
    N = lay.n_params
    t0 = time.time()
    w0 = synth.init_weights(lay, 0)
    stride = layouts.replica_stride(lay)
    g_np = synth.replica_grads(lay, K, 0, 0, dtype=gdt, stride=stride)
    log(f"inputs generated in {time.time() - t0:.1f}s: {desc} "
        f"({g_np.nbytes / 1e9:.2f} GB of gradients)")

    w = torch.from_numpy(w0.copy()).cuda()
    m = torch.zeros_like(w)
    g = torch.from_numpy(g_np.view(np.int16) if gdt == "bf16" else g_np).cuda()
    stream = torch.cuda.current_stream()
    h = ags.AGS(lay.table(), w, m, K, grad_dtype=gdt, mode=args.mode, **HYPER)

    for _ in range(args.warmup):
        h.step(g, stream)
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")

    # Timed region: K steps between two events on the launch stream.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        h.step(g, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    log(f"timed {args.steps} steps: {ms_step * 1e3:.1f} us/step")

    # Per-kernel durations: the same K steps again with the library's HIP
    # events around every kernel, on the same stream (the events add a few
    # microseconds per step, so the step time above is taken without them).
    h.set_profiling(True)
    h.kernel_times()  # reset
    for _ in range(args.steps):
        h.step(g, stream)
    torch.cuda.synchronize()
    kms, ncalls = h.kernel_times()
    h.set_profiling(False)
    log("per kernel (us): " + ", ".join(f"{n} {kms[i] / ncalls * 1e3:.1f}"
                                         for i, n in enumerate(ags.KERNEL_NAMES)))

    # Cold-cache steps: a 1 GiB read evicts the caches (L2 and the 256 MB
    # Infinity Cache) between steps, as the forward and backward passes of a
    # training step would; each step is timed on its own with two events.
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    cold_ms = []
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(min(args.steps, 100))]
    for a0, a1 in ev:
        flush.sum()
        a0.record(stream)
        h.step(g, stream)
        a1.record(stream)
    torch.cuda.synchronize()
    cold_ms = sorted(a0.elapsed_time(a1) for a0, a1 in ev)
    cold_step = cold_ms[len(cold_ms) // 2]
    del flush
    log(f"cold-cache steps: median {cold_step * 1e3:.1f} us")
    # The coefficient prediction (sensitive iff the last step was) in a
    # sensitive phase and in its worst case.  Gradient sets g and 2g in
    # turn make every step sensitive (Delta = 3, then 0.75): predicted right
    # from the second step on.  The sets g, g, 2g, 2g, ... alternate the
    # decision (Delta = 0, 3, 0, 0.75, ...): every step is applied with the
    # other coefficients and corrected by the second pass.
    g2 = g.view(torch.bfloat16).mul(2).view(g.dtype) if gdt == "bf16" else g * 2
    nmis = min(args.steps, 100)

    def timed(pick):
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(nmis):
            h.step(pick(i), stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / nmis, h.read_stats().glob["sensitive"]

    sens_ms, sens_last = timed(lambda i: g2 if i % 2 == 0 else g)
    mis_ms, mis_sens = timed(lambda i: g2 if (i // 2) % 2 == 1 else g)
    del g2
    log(f"sensitive phase: {sens_ms * 1e3:.1f} us/step; every step mispredicted: "
        f"{mis_ms * 1e3:.1f} us/step")

    graph_ms = None
    if args.graph:
        # One step captured in a HIP graph (kernels only), replayed K times.
        cap = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            h.step(g)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        graph_ms = e0.elapsed_time(e1) / args.steps
        log(f"graph replay: {graph_ms * 1e3:.1f} us/step")
    s = h.read_stats()

    ab = algorithmic_bytes(N, args.mode, args.elementwise)
    value = ab["whole_step"] / (ms_step * 1e-3) / 1e9
    avg_ms = {n: kms[i] / ncalls for i, n in enumerate(ags.KERNEL_NAMES)}
    dom = max(avg_ms, key=avg_ms.get)
    achieved = ab[dom] / (avg_ms[dom] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "frac_of_measured_read_ceiling": (round(achieved / probe["read_GBps"], 4)
                                                  if probe else None),
                "frac_of_measured_step_pattern": (round(achieved / probe["step_pattern_GBps"], 4)
                                                  if probe else None),
                "traffic": read_traffic(wkey, dom),
                "algorithmic_bytes_per_launch": ab[dom],
                "avg_launch_us": round(avg_ms[dom] * 1e3, 2)}

    copy_bw = copy_probe(torch)
    log(f"device copy: {copy_bw:.1f} GB/s")

    configs = None
    if not args.no_configs and wkey == WORKLOAD and args.mode == "ags":
        h.close()
        h = None
        configs = measure_configs(torch, np, stream, args.steps, args.warmup)

    cpu = None
    if not args.no_cpu_baseline:
        cores = host_cores()
        log(f"cpu baseline: oracle on whole steps, {cores} threads ...")
        psec, pn, threads = cpu_baseline_parallel(lay, w0, g_np, cores)
        log(f"cpu baseline: {psec:.3f} s/step on {threads} threads; 1 thread ...")
        sec, n = cpu_baseline(lay, w0, g_np)
        cpu = {"value": round(ab["whole_step"] / psec / 1e9, 3), "unit": "GB/s", "cores": threads,
               "kind": "oracle", "sec_per_step": round(psec, 4),
               "host_cores": cores,
               "sample": (f"median of {pn} whole steps of {wkey}, float64, the layers split into "
                          f"{threads} groups of nearly equal size, one thread per group running "
                          f"the unchanged single-threaded oracle"),
               "single_thread": {"value": round(ab["whole_step"] / sec / 1e9, 3), "unit": "GB/s",
                                 "cores": 1, "sec_per_step": round(sec, 3),
                                 "sample": f"median of {n} whole steps of {wkey}, float64, "
                                           f"1 thread"}}
        log(f"cpu baseline: {sec:.2f} s/step on 1 thread")

    headline = wkey == WORKLOAD and args.mode == "ags"
    mode_note = "" if args.mode == "ags" else f", {args.mode.upper()} mode"
    cold_value = ab["whole_step"] / (cold_step * 1e-3) / 1e9
    out = {
        "metric": ("AGS step+stats GB/s & % HBM peak (ResNet-50 layout, K=16); steps/s"
                   if headline else
                   f"AGS step+stats GB/s ({desc}{', elementwise scales' if args.elementwise else ''}"
                   f"{', per-layer Delta' if args.delta_scope == 'layer' else ''}{mode_note})"),
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "steps_per_s": round(1e3 / ms_step, 1),
        "hbm_peak_frac": round(value / HBM_PEAK_GBPS, 4),
        "hbm_peak_frac_cold": round(cold_value / HBM_PEAK_GBPS, 4),
        "value_basis": ("warm: back-to-back steps reusing one gradient set, so w and m (16 B per "
                        "parameter) can stay in the 256 MB Infinity Cache between steps; "
                        "hbm_peak_frac_cold and cold_cache give the step after the caches are "
                        "evicted, as after a forward and backward pass"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # arithmetic: fp32 (statistics in fp64); gradients stored as grad_dtype
        "data": "synthetic",
        "config": {"workload": wkey, "layout": layout_name, "tensors": lay.n_layers,
                   "params": N, "K": K, "grad_dtype": gdt, "param_dtype": "f32",
                   "mode": args.mode, "elementwise": bool(args.elementwise),
                   "delta_scope": args.delta_scope,
                   "algorithmic_bytes_per_step": ab["whole_step"],
                   "parallelism": "single GPU (K replicas stand in for K data-parallel workers)"},
        "kernel_us": {n: round(v * 1e3, 2) for n, v in avg_ms.items()},
        "cold_cache": {"ms_per_step": round(cold_step, 5),
                       "value": round(cold_value, 1),
                       "hbm_peak_frac": round(cold_value / HBM_PEAK_GBPS, 4),
                       "frac_of_measured_cold_step_pattern": (
                           round(cold_value / probe["step_pattern_cold_GBps"], 4)
                           if probe and "step_pattern_cold_GBps" in probe else None),
                       "note": "median of single whole steps after a 1 GiB read evicts the "
                               "caches; the fraction is against hbm_probe's step pattern "
                               "timed the same way"},
        "replica_stride": stride,
        "sensitive_phase_steps": {"ms_per_step": round(sens_ms, 5), "last_sensitive": sens_last,
                                  "note": "every step sensitive: predicted from the last "
                                          "decision, so applied directly from the second on"},
        "mispredicted_steps": {"ms_per_step": round(mis_ms, 5), "last_sensitive": mis_sens,
                               "note": "decisions alternating (not sensitive, sensitive, ...): "
                                       "every step applied with the other coefficients, then "
                                       "corrected (AGS); SGD never corrects"},
        "graph_replay_ms_per_step": None if graph_ms is None else round(graph_ms, 5),
        "device_copy_GBps": round(copy_bw, 1),
        "hbm_probe": probe,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "configs": configs,
        "last_step": {"delta": s.glob["delta"], "sensitive": s.glob["sensitive"],
                      "step": s.glob["step"]},
    }
    if h is not None:
        h.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

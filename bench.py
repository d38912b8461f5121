"""Throughput of the exact factored output-layer step on one GPU, with its roofline,
the naive O(D d) path and the fp64 CPU oracle as baselines.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
    python bench.py --sweep        # factored vs naive over the D x d sweep, JSON lines

A step is one pass of the whole factored step (dense contractions, sparse
gather, loss and grad_H, the m x m Woodbury block, the U / U^{-T} / Q updates
and the V scatter: five kernel launches) over one minibatch already resident in
HBM.  Prints one JSON line: the headline workload (squared error, D=200k, d=500,
m=128, K=5) with its roofline and baselines, and beside it the spherical-softmax
and D=800k workloads and a compact D x d sweep with the measured crossover.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 matrix (and vector) peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
METRIC = "examples/s exact loss+grad+update, D=200k d=500 m=128; speedup vs naive O(Dd)"


def phase_work(w, idx_pool):
    """Algorithmic work per launch of each of the step's five launches: (bound, amount,
    unit of amount).

    bound "mfma": dense contractions, flops against the fp32 matrix peak; "hbm": the
    sparse V traffic, bytes against HBM bandwidth.  Launch 2 (gather) also carries three
    small products (H H^^T, E^2, E Xs: 2 (2 m^2 d + m^3) flops) beside the per-example
    gather; its figure is the gather's bytes only.
    """
    m, d, K = w.m, w.d, w.K
    uniq = float(np.mean([len(np.unique(i[i >= 0])) for i in idx_pool]))
    return {
        # H^, H~, X = {Q, U, U^-T} H (3 m d^2) and N = H H^T (m^2 d)
        "contract": ("mfma", 2.0 * (3 * m * d * d + m * m * d), "flop"),
        # the m x K target rows of V and the m rows of H~ read; G and 2 eta D H~ written
        "gather": ("hbm", 4.0 * (m * K * d + 3 * m * d), "byte"),
        # Z^ = G U (m d^2), H~ G^T, E^2 Xs, E^2 W1 (m^2 d each), E^4 (m^3)
        "zgrad": ("mfma", 2.0 * (m * d * d + 3 * m * m * d + m ** 3), "flop"),
        # (eta^2/2) M H - eta grad_H and R X (m^2 d each), the U update (m d^2)
        "mid": ("mfma", 2.0 * (2 * m * m * d + m * d * d), "flop"),
        # the U^-T update (m d^2) and the Q update (2 m d^2); the V scatter's read-modify-write
        # of the distinct target rows rides in the same launch
        "update": ("mfma", 2.0 * 3 * m * d * d, "flop"),
        "scatter_bytes": ("hbm", 4.0 * (2 * uniq * d + m * K * d), "byte"),
    }


def kernel_table(phases, work):
    """Per-phase average duration and, where a roofline applies, its fraction."""
    out = {}
    for name, (bound, amount, unit) in work.items():
        cnt, ms = phases.get("update" if name == "scatter_bytes" else name, (0, 0.0))
        if not cnt:
            continue
        avg_s = ms / cnt / 1e3
        row = {"bound": bound, "avg_us": round(avg_s * 1e6, 3), "work_per_launch": amount,
               "work_unit": unit}
        if bound == "mfma":
            row.update(achieved=round(amount / avg_s / 1e12, 4), peak=PEAK_FP32_TFLOPS,
                       unit="TFLOP/s", frac=round(amount / avg_s / 1e12 / PEAK_FP32_TFLOPS, 5))
        elif bound == "hbm":
            row.update(achieved=round(amount / avg_s / 1e9, 2), peak=PEAK_HBM_GBS, unit="GB/s",
                       frac=round(amount / avg_s / 1e9 / PEAK_HBM_GBS, 5))
        out[name] = row
    return out


TRAFFIC_MD = os.path.join(ROOT, "profiles", "factored_step_sq_D200k_d500_m128_K5_pmc_traffic.md")


def load_traffic():
    """Per-launch HBM bytes measured by hardware counters (the JSON block of the traffic
    summary under profiles/, written by bench_pmc.py), per phase, kept only while the
    kernel's sources are unchanged since the counters were taken."""
    from bench_pmc import read_traffic_block, source_sha

    if not os.path.exists(TRAFFIC_MD):
        return {}
    out = {}
    for phase, r in read_traffic_block(TRAFFIC_MD).items():
        try:
            same = source_sha(r["source"]) == r["source_sha256"]
        except OSError:
            same = False
        if same:
            out[phase] = int(r["fetch_bytes"]) + int(r["write_bytes"])
    return out


def roofline_for(table, traffic=None):
    """The dominant kernel: the longest of the step's launches."""
    name = max((k for k in table if k != "scatter_bytes" and table[k]["bound"] in ("mfma", "hbm")),
               key=lambda k: table[k]["avg_us"])
    r = table[name]
    return {"kernel_phase": name, "bound": r["bound"], "achieved": r["achieved"], "peak": r["peak"],
            "unit": r["unit"], "frac": r["frac"], "traffic": (traffic or {}).get(name),
            "avg_launch_us": r["avg_us"], "algorithmic_per_launch": r["work_per_launch"]}


def attainable_peaks(dev):
    """Measured ceilings on this GPU beside the spec peaks: a 1 GiB device-to-device
    copy (bytes read + written per second) and a 8192^3 fp32 matmul through torch's
    BLAS (fp32 matrix cores; TF32 is off in torch by default)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(10):
        dst.copy_(src)
    ev[1].record()
    torch.cuda.synchronize()
    hbm = 10 * 2 * src.numel() * 4 / (ev[0].elapsed_time(ev[1]) / 1e3) / 1e9
    del src, dst
    n = 8192
    a_ = torch.randn(n, n, device=dev)
    b_ = torch.randn(n, n, device=dev)
    torch.matmul(a_, b_)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(5):
        torch.matmul(a_, b_)
    ev[1].record()
    torch.cuda.synchronize()
    mm = 5 * 2.0 * n ** 3 / (ev[0].elapsed_time(ev[1]) / 1e3) / 1e12
    del a_, b_
    torch.cuda.empty_cache()
    return {"hbm_GBs": round(hbm, 1), "fp32_matrix_TFLOPs": round(mm, 2),
            "how": "1 GiB device copy x10 (read+write bytes); 8192^3 fp32 torch.matmul x5"}


def cpu_baseline(w, V0, pool, seconds, threads=None):
    """The fp64 dense oracle on the host: examples/s over a bounded sample."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import dense_step

    with threadpool_limits(limits=threads, user_api="blas"):
        W = V0.astype(np.float64)
        H, idx, val = pool[0]
        dense_step(W, H, idx, val, np.float32(w.lr), w.loss, np.float32(w.eps))  # warm-up
        n = 0
        t0 = time.perf_counter()
        while True:
            H, idx, val = pool[(n + 1) % len(pool)]
            W = dense_step(W, H, idx, val, np.float32(w.lr), w.loss, np.float32(w.eps)).W_new
            n += 1
            el = time.perf_counter() - t0
            if (el >= seconds and n >= 2) or n >= 200:
                break
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = int(blas[0]["num_threads"]) if blas else 1
    return {"value": round(w.m * n / el, 3), "unit": "examples/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{n} dense fp64 steps of {w.name} (D={w.D}, d={w.d}, m={w.m}) after 1 "
                      f"warm-up step, {el:.1f} s; nproc={os.cpu_count()}, "
                      f"affinity={len(os.sched_getaffinity(0))}"}


def device_stream(w, dev, n, seed):
    """V0 and n minibatches of a workload, on the device: V0 and H drawn on the GPU
    (torch's generator, seeded: these legs are timed, not compared with the oracle),
    the targets by the workload's own index and value laws (numpy PCG64, seeded)."""
    import torch

    from workloads import ZipfSampler, make_targets

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    V0 = torch.randn((w.D, w.d), device=dev, generator=g).mul_(float(1.0 / np.sqrt(w.d)))
    rng = np.random.default_rng(seed)
    zipf = ZipfSampler(w.D, w.zipf_s) if w.index_dist == "zipf" else None
    batches, idxs = [], []
    for _ in range(n):
        H = torch.randn((w.m, w.d), device=dev, generator=g).mul_(float(1.0 / np.sqrt(w.d)))
        idx, val = make_targets(rng, w, None, zipf)
        idxs.append(idx)
        batches.append((H.contiguous(), torch.from_numpy(idx).to(dev), torch.from_numpy(val).to(dev)))
    return V0, batches, idxs


def timed(step, batches, n, warm, lr, grad):
    """ms per step over n steps (HIP events on the current stream) after warm steps."""
    import torch

    for t in range(warm):
        step(*batches[t % len(batches)], lr, grad_H=grad)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for t in range(n):
        step(*batches[t % len(batches)], lr, grad_H=grad)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def factored_vs_naive(w, dev, seed, steps, naive_steps, profile=False):
    """Factored and naive ms/step on the same device-drawn batches of workload w."""
    import torch

    import paper_1606_08061_amd as lst

    V0, batches, idxs = device_stream(w, dev, 8, seed)
    grad = torch.empty((w.m, w.d), dtype=torch.float32, device=dev)
    eps = float(np.float32(w.eps))
    f = lst.Factored(w.D, w.d, w.m, w.K, w.loss, eps, device=dev)
    f.init(V0)
    fms = timed(f.step, batches, steps, 8, w.lr, grad)
    f.check(f"factored steps of {w.name}")
    row = {"workload": w.name, "loss": w.loss, "D": w.D, "d": w.d, "m": w.m, "K": w.K,
           "index_dist": w.index_dist, "factored_ms_per_step": round(fms, 5),
           "examples_per_s": round(w.m / (fms / 1e3), 1)}
    if profile:
        f.profile(True)
        for t in range(steps):
            f.step(*batches[t % len(batches)], w.lr, grad_H=grad)
        table = kernel_table(f.profile_read(), phase_work(w, idxs))
        f.profile(False)
        f.check(f"profiled steps of {w.name}")
        r = roofline_for(table)
        row["roofline"] = {k: r[k] for k in ("kernel_phase", "bound", "achieved", "peak", "unit",
                                                 "frac", "avg_launch_us")}
        row["phases_us"] = {k: v["avg_us"] for k, v in table.items() if k != "scatter_bytes"}
    f.close()
    n = lst.Naive(w.D, w.d, w.m, w.K, w.loss, eps, device=dev)
    n.init(V0)
    nms = timed(n.step, batches, naive_steps, 2, w.lr, grad)
    n.check(f"naive steps of {w.name}")
    n.close()
    del V0, batches, f, n
    torch.cuda.empty_cache()
    row.update(naive_ms_per_step=round(nms, 4), speedup_vs_naive=round(nms / fms, 2),
               D_over_4d=round(w.D / (4 * w.d), 1))
    return row


def sweep_rows(fsteps, nsteps, emit=None):
    """Factored vs naive over the D x d sweep (squared error, m = 512, K = 5) and the
    measured crossover (speedup 1, log-linear between the bracketing D) per d.  The rows
    of the largest D also carry the per-launch times and the longest launch's roofline."""
    from workloads import sweep_workloads

    import torch

    dev = torch.device("cuda:0")
    res = []
    ws = sweep_workloads()
    dmax = max(w.D for w in ws)
    for w in ws:
        r = factored_vs_naive(w, dev, w.D * 7 + w.d, fsteps, nsteps, profile=w.D == dmax)
        row = {"D": w.D, "d": w.d, "factored_ms": r["factored_ms_per_step"],
               "naive_ms": r["naive_ms_per_step"], "speedup": r["speedup_vs_naive"],
               "D_over_4d": r["D_over_4d"]}
        if "roofline" in r:
            row["roofline"] = r["roofline"]
            row["phases_us"] = r["phases_us"]
        res.append(row)
        if emit:
            emit(row)
    cross = {}
    for d in sorted({r["d"] for r in res}):
        pts = sorted((r["D"], r["speedup"]) for r in res if r["d"] == d)
        c = None
        for (D0, s0), (D1, s1) in zip(pts, pts[1:]):
            if s0 < 1.0 <= s1:
                t = (0.0 - np.log(s0)) / (np.log(s1) - np.log(s0))
                c = float(np.exp(np.log(D0) + t * (np.log(D1) - np.log(D0))))
                break
        if c is None and pts and pts[0][1] >= 1.0:
            c = f"below {pts[0][0]}"
        cross[str(d)] = c if not isinstance(c, float) else round(c, 1)
    return res, cross


def run_sweep(args):
    """The sweep as JSON lines: one per configuration, then the crossover per d."""
    res, cross = sweep_rows(args.sweep_steps, max(2, args.sweep_steps // 4),
                            emit=lambda r: print(json.dumps(r), flush=True))
    print(json.dumps({"sweep_crossover_D": cross, "m": 512, "K": 5}), flush=True)


def vendor_gemms(w, dev, H) -> dict:
    """The naive path's three fp32 products through torch (the ROCm BLAS libraries),
    as context for the naive path's own GEMM kernels: O = W H^T, grad_H = O^T W and
    W += -lr O H, each timed over 10 calls on torch's current stream."""
    import torch

    torch.backends.cuda.matmul.allow_tf32 = False
    W = torch.randn(w.D, w.d, device=dev) * 0.1
    O = torch.randn(w.D, w.m, device=dev)
    out = {}
    calls = {
        "naive_fwd": lambda: torch.mm(W, H.t()),
        "naive_grad": lambda: torch.mm(O.t(), W),
        "naive_update": lambda: W.addmm_(O, H, alpha=-w.lr),
    }
    for name, fn in calls.items():
        for _ in range(2):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(10):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name] = round(a.elapsed_time(b) / 10 * 1e3, 2)
    del W, O
    torch.cuda.empty_cache()
    return out


def stabilize_leg(f, w, dev, reps=5):
    """Section 5 operations on the benchmark's state after its steps (V of D x d): each
    timed with HIP events on the context's stream over reps calls.  The pristine restore
    is an O(D d^2) product (2 D d^2 flops, bound by the matrix cores); the fix of one
    singular value passes once over V (2 D d 4 bytes read and written, bound by HBM)."""
    import torch

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, n=reps):
        fn()  # warm-up call
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        f.check("stabilize leg")
        return e0.elapsed_time(e1) / n * 1e3  # us per call

    g = torch.Generator(device=dev).manual_seed(17)
    u0 = torch.randn(w.d, generator=g, device=dev)
    u = u0 / u0.norm()
    sig = torch.tensor(0.5, device=dev)
    out = {}
    out["fix_us"] = timed(lambda: f.fix_singular_value(u, sig, 1.0))
    out["power_iteration_us"] = timed(lambda: f.power_iteration("smallest", 7, u0))
    out["refresh_us"] = timed(lambda: f.refresh_uinvt(2))
    out["restore_us"] = timed(lambda: f.restore_pristine())
    h0 = time.perf_counter()
    n_fix, sigmas = f.singular_stabilize(u0, 1e-3, 100.0, 7, 8)
    out["check_ms_wall"] = (time.perf_counter() - h0) * 1e3
    out["check_result"] = {"fixes": list(n_fix), "sigma_min": sigmas[0], "sigma_max": sigmas[1]}
    restore_flops = 2.0 * w.D * w.d * w.d
    fix_bytes = 2.0 * w.D * w.d * 4
    out["restore_roofline"] = {"bound": "mfma", "achieved": round(restore_flops / out["restore_us"] / 1e6, 2),
                               "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                               "frac": round(restore_flops / out["restore_us"] / 1e6 / PEAK_FP32_TFLOPS, 4),
                               "algorithmic_per_launch": restore_flops}
    out["fix_roofline"] = {"bound": "hbm", "achieved": round(fix_bytes / out["fix_us"] / 1e3, 1),
                           "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": round(fix_bytes / out["fix_us"] / 1e3 / PEAK_HBM_GBS, 4),
                           "algorithmic_per_launch": fix_bytes}
    for k in ("fix_us", "power_iteration_us", "refresh_us", "restore_us", "check_ms_wall"):
        out[k] = round(out[k], 2)
    return out


def online_leg(w, dev, V0, gpool, steps=2000, general_steps=300):
    """The online step (m = 1, squared error, Algorithm 2) on the benchmark's V: the first
    example of each pooled minibatch, through the single launch with its bounded grid barrier
    and through the general step path (LST_OPT_ONLINE_KERNEL = 0).  Algorithmic bytes per
    step: Q, U, U^{-T} read and written once (6 d^2 floats; the K target rows of V add 8 K d)."""
    import torch

    import paper_1606_08061_amd as lst

    ex = [[t[:1].contiguous() for t in b] for b in gpool]
    grad = torch.empty((1, w.d), dtype=torch.float32, device=dev)
    out = {}
    for name, n, online in (("fused", steps, 1), ("general", general_steps, 0)):
        f = lst.Factored(w.D, w.d, 1, w.K, "squared", device=dev)
        f.set_option(lst.LST_OPT_ONLINE_KERNEL, online)
        f.init(V0)
        for t in range(64):
            f.step(*ex[t % len(ex)], w.lr, grad_H=grad)
        f.check("online warm-up")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for t in range(n):
            f.step(*ex[t % len(ex)], w.lr, grad_H=grad)
        e1.record()
        torch.cuda.synchronize()
        f.check("online steps")
        us = e0.elapsed_time(e1) / n * 1e3
        h0 = time.perf_counter()
        for t in range(n):
            f.step(*ex[t % len(ex)], w.lr, grad_H=grad)
        host_us = (time.perf_counter() - h0) / n * 1e6
        torch.cuda.synchronize()
        # GPU time of the step's kernels (launch-attached HIP events per phase)
        f.profile(True)
        for t in range(n):
            f.step(*ex[t % len(ex)], w.lr, grad_H=grad)
        ph = f.profile_read()
        f.profile(False)
        kern_us = sum(v[1] for v in ph.values()) / n * 1e3
        out[name] = {"us_per_example": round(us, 2), "examples_per_s": round(1e6 / us, 1),
                     "host_enqueue_us": round(host_us, 2), "kernel_us": round(kern_us, 2)}
        f.close()
    byt = 6.0 * w.d * w.d * 4 + 8.0 * w.K * w.d
    us = out["fused"]["us_per_example"]
    out["roofline"] = {"bound": "hbm", "achieved": round(byt / us / 1e3, 1), "peak": PEAK_HBM_GBS,
                       "unit": "GB/s", "frac": round(byt / us / 1e3 / PEAK_HBM_GBS, 4),
                       "algorithmic_per_launch": byt}
    out["speedup_fused_vs_general"] = round(out["general"]["us_per_example"] / us, 2)
    return out


def input_layer_leg(w, dev, D_in=200_000, K_in=4, reps=200):
    """The sparse input layer of section 2.2 at the benchmark's d and m: K_in-sparse inputs
    over D_in rows (Zipf, seeded), forward A = X W1 and update W1 -= eta X^T grad_A, each
    timed with HIP events over reps calls.  Bytes: forward m K_in d 4 read + m d 4 written;
    update: the distinct named rows read and written, grad_A read."""
    import torch

    import paper_1606_08061_amd as lst

    rng = np.random.default_rng(23)
    W1 = torch.from_numpy((rng.standard_normal((D_in, w.d)) / np.sqrt(w.d * K_in))
                          .astype(np.float32)).to(dev)
    p = 1.0 / np.arange(1, D_in + 1) ** 1.1
    idx = rng.choice(D_in, size=(w.m, K_in), p=p / p.sum()).astype(np.int32)
    val = rng.standard_normal((w.m, K_in)).astype(np.float32)
    gA = torch.from_numpy(rng.standard_normal((w.m, w.d)).astype(np.float32) * 1e-3).to(dev)
    idx_d, val_d = torch.from_numpy(idx).to(dev), torch.from_numpy(val).to(dev)
    layer = lst.SparseInput(W1)
    A = torch.empty((w.m, w.d), dtype=torch.float32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {"D_in": D_in, "K_in": K_in}
    for name, fn in (("forward", lambda: layer.forward(idx_d, val_d, out=A)),
                     ("update", lambda: layer.update(idx_d, val_d, gA, 1e-3))):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name + "_us"] = round(e0.elapsed_time(e1) / reps * 1e3, 2)
    layer.check()
    u = len(np.unique(idx))
    fb = 4.0 * w.m * w.d * (K_in + 1)
    ub = 4.0 * (2 * u * w.d + w.m * w.d)
    out["forward_GBs"] = round(fb / out["forward_us"] / 1e3, 1)
    out["update_GBs"] = round(ub / out["update_us"] / 1e3, 1)
    out["distinct_rows"] = u
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=128)
    ap.add_argument("--workload", default="sq_D200k_d500_m128_K5")
    ap.add_argument("--pool", type=int, default=64, help="distinct minibatches cycled through")
    ap.add_argument("--naive-steps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-online", action="store_true",
                    help="skip the timing of the one-example (m = 1) online step")
    ap.add_argument("--no-stabilize", action="store_true",
                    help="skip the timing of the section 5 stabilisation operations")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured copy and matmul ceilings (also skipped with --copy-calib)")
    ap.add_argument("--sweep", action="store_true",
                    help="factored vs naive over the D x d sweep instead of the default line")
    ap.add_argument("--sweep-steps", type=int, default=20)
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the spherical-softmax, D=800k and sweep legs")
    ap.add_argument("--copy-calib", type=int, default=0, metavar="MIB",
                    help="also run one plain device copy of MIB MiB (hardware-counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the factored step is measured on one GPU's "
              "share (multi-GPU sharding of V by rows is described but not built)",
              file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        import torch

        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible")
        run_sweep(args)
        return

    import torch

    import paper_1606_08061_amd as lst
    from workloads import WORKLOADS, Stream

    if not torch.cuda.is_available():
        raise RuntimeError("no GPU visible")
    lst.lib()  # fails loudly when the HIP library is not built
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")

    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    s = Stream(w)
    pool = [s.batch() for _ in range(args.pool)]
    gpool = [[torch.from_numpy(a).to(dev) for a in b] for b in pool]
    V0 = torch.from_numpy(s.V0).to(dev)

    # ---- factored path ----
    f = lst.Factored(w.D, w.d, w.m, w.K, w.loss, float(np.float32(w.eps)), device=dev)
    f.init(V0)
    grad = torch.empty((w.m, w.d), dtype=torch.float32, device=dev)
    # Warm-up with exactly the timed calls (the step's descriptors for this m are
    # built and copied on the first call).
    for t in range(max(args.warmup, len(gpool))):
        f.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
    f.check("warm-up")
    print("[bench] factored timed region", file=sys.stderr, flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    h0 = time.perf_counter()
    for t in range(args.steps):
        f.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
    host_us = (time.perf_counter() - h0) / args.steps * 1e6
    e1.record()
    torch.cuda.synchronize()
    ms_total = e0.elapsed_time(e1)
    f.check("timed steps")
    ms_step = ms_total / args.steps
    value = w.m * args.steps / (ms_total / 1e3)

    # per-phase HIP events over a second region of the same length
    f.profile(True)
    for t in range(args.steps):
        f.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
    phases = f.profile_read()
    f.profile(False)
    f.check("profiled steps")
    work = phase_work(w, [b[1] for b in pool])
    table = kernel_table(phases, work)
    traffic = load_traffic()
    for k, v in traffic.items():
        if k in table:
            table[k]["traffic_bytes"] = v
    roof = roofline_for(table, traffic)
    stab = None
    if not args.no_stabilize:
        print("[bench] stabilisation operations", file=sys.stderr, flush=True)
        stab = stabilize_leg(f, w, dev)
        stab["restore_roofline"]["traffic"] = traffic.get("restore")
        stab["fix_roofline"]["traffic"] = traffic.get("fix_v")
    f.close()
    del f

    if args.copy_calib:
        # A copy of known size: its FETCH_SIZE / WRITE_SIZE counters scale the
        # counters of the step's kernels to bytes.
        src = torch.ones(args.copy_calib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    inp = None
    if not args.no_online:
        print("[bench] sparse input layer", file=sys.stderr, flush=True)
        inp = input_layer_leg(w, dev)
    online = None
    if not args.no_online and w.loss == "squared":
        print("[bench] online (m = 1) steps", file=sys.stderr, flush=True)
        online = online_leg(w, dev, V0, gpool)

    # ---- naive O(D d) path on the same batches ----
    naive = None
    if not args.no_naive:
        print("[bench] naive timed region", file=sys.stderr, flush=True)
        n = lst.Naive(w.D, w.d, w.m, w.K, w.loss, float(np.float32(w.eps)), device=dev)
        n.init(V0)
        for t in range(2):
            n.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
        torch.cuda.synchronize()
        e0.record()
        for t in range(args.naive_steps):
            n.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
        e1.record()
        torch.cuda.synchronize()
        n.check("naive steps")
        nms = e0.elapsed_time(e1) / args.naive_steps
        n.profile(True)
        for t in range(args.naive_steps):
            n.step(*gpool[t % len(gpool)], w.lr, grad_H=grad)
        nph = n.profile_read()
        n.close()
        del n
        naive = {"value": round(w.m / (nms / 1e3), 2), "unit": "examples/s",
                 "ms_per_step": round(nms, 4),
                 "phases_us": {k: round(v[1] / max(v[0], 1) * 1e3, 2)
                               for k, v in nph.items() if v[0] and k.startswith("naive")},
                 "vendor_gemm_us": vendor_gemms(w, dev, gpool[0][0])}

    del V0, gpool
    torch.cuda.empty_cache()
    secondary = sweep = None
    if not args.no_secondary:
        from workloads import WORKLOADS as WL

        secondary = {}
        for name in ("sphsm_D200k_d500_m128_zipf", "sq_D800k_d512_m256_K10_zipf",
                     "taylor_D200k_d500_m128_zipf"):
            print(f"[bench] secondary workload {name}", file=sys.stderr, flush=True)
            secondary[name] = factored_vs_naive(WL[name], dev, 11, 300, 8, profile=True)
        print("[bench] D x d sweep", file=sys.stderr, flush=True)
        pts, cross = sweep_rows(10, 3)
        sweep = {"m": 512, "K": 5, "loss": "squared", "points": pts, "crossover_D": cross}
    att = None
    if not (args.no_peaks or args.copy_calib):  # counter runs take the copy as their scale
        att = attainable_peaks(dev)
        roof["attainable_peak"] = (att["hbm_GBs"] if roof["bound"] == "hbm"
                                   else att["fp32_matrix_TFLOPs"])
        roof["frac_attainable"] = round(roof["achieved"] / roof["attainable_peak"], 5)
    cpu = cpu1 = None
    if not args.no_cpu:
        print("[bench] cpu baseline (fp64 oracle)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, s.V0, pool, args.cpu_seconds)
        cpu1 = cpu_baseline(w, s.V0, pool, args.cpu_seconds / 2, threads=1)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "examples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "loss": w.loss, "D": w.D, "d": w.d, "m": w.m, "K": w.K,
                   "index_dist": w.index_dist, "lr": w.lr, "distinct_batches": args.pool},
        "roofline": roof,
        "cpu_baseline": cpu,
        "cpu_baseline_1core": cpu1,
        "naive": naive,
        "speedup_vs_naive": round(value / naive["value"], 2) if naive else None,
        "speedup_model_D_over_4d": round(w.D / (4 * w.d), 1),
        "host_enqueue_us_per_step": round(host_us, 2),
        "kernels": table,
        "attainable": att,
        "stabilize": stab,
        "online": online,
        "input_layer": inp,
        "secondary": secondary,
        "sweep": sweep,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

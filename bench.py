"""Benchmark: batched entropy-regularised Sinkhorn forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4]

The default workload is the largest one that fits one GPU: the grid
(B=64, d1=d2=4096, lambda=1e-3, 500 iterations, tol=1e-6); --config 1..6
selects the others.

One step = the whole hot path over one batch: sinkhorn_forward (all
iterations, loss and marginal error) followed by sinkhorn_backward
(grad_mu, grad_nu; plus grad_C for the point-cloud workload).  Inputs are
synthetic (seeded, see workloads/) and resident in HBM before timing starts.

Prints ONE JSON line.  value = cell-updates/s = sum_b d1*d2*iters_b per step
divided by the step time.  The roofline object refers to the dominant kernel
and is measured live with events on the stream the library launches on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
# v_exp_f32 issues a wave64 in 8 cycles per SIMD (half rate; measured 28.9 of
# 32 per clock per CU in a pure-exp loop): 256 CUs x 4 SIMDs x 8 lanes/clk x 2.4 GHz
PEAK_EXP_TS = 256 * 4 * 8 * 2.4e9 / 1e12
# MI355X published dense fp32 vector peak (TFLOP/s).
PEAK_FP32_VALU = 157.3

# Resident kernels: the first choice for a shape and the source it is built
# from, both the plain form on the vector ALU with K in registers.  A shared
# symmetric cost with d1 = d2 <= 104: the symmetric kernel; any other cost
# (shared or per sample): the general kernel.
RESIDENT_KERNELS = {
    "sym": ("sk_resident_sym_kernel", ("sk_resident_sym.hip", "sk_resident_gen.h", "sk_resident_log.h"), "alu",
            PEAK_FP32_VALU),
    "shared": ("sk_resident_gen_kernel", ("sk_resident_gen.hip", "sk_resident_gen.h", "sk_resident_log.h"), "alu",
               PEAK_FP32_VALU),
    "batched": ("sk_resident_gen_kernel", ("sk_resident_gen.hip", "sk_resident_gen.h", "sk_resident_log.h"), "alu",
                PEAK_FP32_VALU),
}


def resident_kind(prob):
    if prob.c_batched:
        return "batched"
    C = prob.C[0]
    if prob.d1 == prob.d2 <= 104 and np.array_equal(C.view(np.uint32), C.T.view(np.uint32)):
        return "sym"
    return "shared"

WORKLOAD_NAMES = {
    1: "tiny: B=4, d1=d2=10, shared 1-D squared cost, lambda=0.1, 100 iterations + backward",
    2: "label: B=1024, d1=d2=100, shared squared-distance cost of 100 embeddings, lambda=0.05, "
       "200 iterations + backward",
    3: "image: B=256, d1=d2=784 (28x28), blob histograms, shared squared grid cost, lambda=0.01, "
       "300 iterations + backward",
    4: "grid: B=64, d1=d2=4096 (64x64), blob histograms, shared squared grid cost, lambda=1e-3, "
       "500 iterations, tol=1e-6 + backward",
    5: "clouds: B=32, d1=1024, d2=2048, per-sample squared-distance cost [32,1024,2048], lambda=0.05, "
       "100 iterations + backward with grad_C",
    6: "clouds from points: the clouds workload with the cost recreated from the 3-D coordinates in the sweep "
       "(no cost matrix), B=32, d1=1024, d2=2048, lambda=0.05, 100 iterations + backward with grad_X, grad_Y",
}


def code_text(src):
    """Source text without comments, trailing blanks and empty lines: what
    compiles into the kernel (string literals in these files hold no comment
    markers)."""
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    lines = (re.sub(r"//.*$", "", l).rstrip() for l in src.splitlines())
    return "\n".join(l for l in lines if l)


def kernel_source_hash(files):
    """Hash of the kernel sources' code (comments and blank lines excluded), the
    key under which a committed counter summary holds for the current kernel."""
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_1907_01729_amd", "csrc", f)) as fh:
            h.update(code_text(fh.read()).encode())
    return h.hexdigest()[:16]


def stored_counters(profile_name, src_hash):
    """The JSON block of a committed rocprofv3 --pmc summary, if it was taken
    on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", profile_name)
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\s*(\{.*?\})\s*```", open(path).read(), re.S)
    if not m:
        return None
    d = json.loads(m.group(1))
    return d if d.get("source_hash") == src_hash else None


def stored_traffic(profile_name, src_hash):
    """HBM bytes per launch from a committed counter summary (None if stale)."""
    d = stored_counters(profile_name, src_hash)
    return d.get("hbm_bytes_per_launch") if d else None


def counter_fields(profile_name, src_hash):
    """Issue utilisation of the dominant kernel from its committed counter
    summary (None if stale): the share of the SIMDs' cycles spent issuing
    vector instructions (4 cycles per fp32 wave64 instruction, 8 per
    transcendental one), and the exp issue rate against 19.66 Texp/s."""
    d = stored_counters(profile_name, src_hash)
    if not d:
        return dict(valu_busy=None, exp_issue_frac=None)
    return dict(valu_busy=d.get("valu_busy_est"), exp_issue_frac=d.get("exp_issue_frac"))


# The oracle's baseline repeats whole passes of its sample until at least this
# much host time has gone by, so the rate is not one short pass's noise.
CPU_BASELINE_MIN_S = 10.0
CPU_BASELINE_MAX_PASSES = 64


def _timed_passes(one_pass):
    """Run one_pass() until CPU_BASELINE_MIN_S has elapsed (or the pass cap is
    reached); return (seconds, passes, last pass's result)."""
    passes, dt, out = 0, 0.0, None
    while passes < CPU_BASELINE_MAX_PASSES and (passes == 0 or dt < CPU_BASELINE_MIN_S):
        t0 = time.perf_counter()
        out = one_pass()
        dt += time.perf_counter() - t0
        passes += 1
    return dt, passes, out


def cpu_baseline(prob, grad_C, sharp=False):
    """The fp64 oracle, as it stands, on the host cores: the same step
    (forward + backward) on the whole batch, repeated for at least
    CPU_BASELINE_MIN_S seconds."""
    import oracle

    def one_pass():
        o = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter, tol=prob.tol)
        if sharp:
            oracle.sharp_gradient(np.ones(prob.B), prob.mu, prob.nu, prob.C, prob.lam, o["alpha"], o["beta"])
        else:
            oracle.backward(np.ones(prob.B), prob.mu, prob.nu, prob.C, prob.lam, o["alpha"], o["beta"],
                            grad_C=grad_C)
        return o

    dt, passes, o = _timed_passes(one_pass)
    cells = passes * float(np.sum(o["iters"].astype(np.float64))) * prob.d1 * prob.d2
    return dict(value=cells / dt, unit="cell-updates/s", cores=oracle.num_threads(), kind="oracle",
                sample=f"whole batch of workload {prob.name} (B={prob.B}), one forward+backward"
                       f"{' (gradient of E^0, dense solve)' if sharp else ''}, {passes} passes, {dt:.2f} s")


def cpu_baseline_sampled(prob, grad_C, n_samples, sharp=False, n_iter=None):
    """The oracle on the first n_samples problems, at most n_iter of their
    iterations (one grid problem's 500 take ~35 s on 16 host threads)."""
    import workloads

    idx = np.arange(n_samples)
    C = prob.C[idx] if prob.c_batched else prob.C
    its = prob.n_iter if n_iter is None else min(n_iter, prob.n_iter)
    sub = workloads.Problem(prob.name, prob.mu[idx], prob.nu[idx], C, prob.lam, its, prob.tol, grad_C)
    r = cpu_baseline(sub, grad_C, sharp=sharp)
    part = f", the first {its} of its {prob.n_iter} iterations" if its != prob.n_iter else ""
    r["sample"] = (f"first {n_samples} of {prob.B} problems of workload {prob.name}{part}, one forward+backward "
                   f"({', '.join(r['sample'].split(', ')[-2:])})")
    return r


def cpu_baseline_points(prob, n_samples):
    """The oracle on the first problems of a point-cloud workload: the cost from
    the coordinates, forward, backward and the point gradients."""
    import oracle

    idx = np.arange(n_samples)

    def one_pass():
        C = oracle.cost_from_points(prob.X[idx], prob.Y[idx])
        o = oracle.forward(prob.mu[idx], prob.nu[idx], C, prob.lam, prob.n_iter, tol=prob.tol)
        r = oracle.backward(np.ones(n_samples), prob.mu[idx], prob.nu[idx], C, prob.lam, o["alpha"], o["beta"],
                            grad_C=True)
        oracle.points_grads(r["grad_C"], prob.X[idx], prob.Y[idx])
        return o

    dt, passes, o = _timed_passes(one_pass)
    cells = passes * float(np.sum(o["iters"].astype(np.float64))) * prob.d1 * prob.d2
    return dict(value=cells / dt, unit="cell-updates/s", cores=oracle.num_threads(), kind="oracle",
                sample=f"first {n_samples} of {prob.B} problems of workload {prob.name}, cost from the points, "
                       f"one forward+backward with point gradients, {passes} passes, {dt:.2f} s")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=4, choices=[1, 2, 3, 4, 5, 6])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's batch size (same generator); the line then names the override")
    ap.add_argument("--n-iter", type=int, default=None,
                    help="override the workload's iteration count (short runs under a profiler); the line names it")
    ap.add_argument("--tol", type=float, default=None,
                    help="override the workload's early-stop tolerance on the marginal L1 error")
    ap.add_argument("--select", default="default", choices=["default", "log", "plain", "nosym", "nocompact"],
                    help="forward through sinkhorn_forward_select with these kernels pinned (resident shapes: "
                         "'log' times the log-domain kernel alone); the line names it")
    ap.add_argument("--sharp", action="store_true",
                    help="backward = gradient of E^0 itself (implicit differentiation, conjugate gradients; "
                         "configs 1, 2 and 3)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy 3 times (scales rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: measures one GPU only (the batch is embarrassingly parallel; "
              "multi-GPU sharding is design-only). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = 64 << 20  # 64 Mi floats = 256 MiB read + 256 MiB written per copy
        x = torch.ones(n, device="cuda:0", dtype=torch.float32)
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "copies": 3}), flush=True)
        return

    import paper_1907_01729_amd as sk
    import workloads

    points = args.config == 6
    if args.sharp and args.config not in (1, 2, 3):
        print("bench.py: --sharp takes configs 1, 2 and 3", file=sys.stderr)
        sys.exit(2)
    over = {"B": args.batch} if args.batch else {}
    prob = workloads.clouds_points(**over) if points else workloads.make_config(args.config, **over)
    if args.tol is not None:
        prob.tol = args.tol
    if args.n_iter is not None:
        prob.n_iter = args.n_iter
    grad_C = bool(prob.grad_points) if points else bool(prob.grad_C)
    dev = torch.device("cuda:0")
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    mu, nu = t(prob.mu), t(prob.nu)
    g = torch.ones(prob.B, device=dev, dtype=torch.float32)
    if points:
        X, Y = t(prob.X), t(prob.Y)
        nws = sk.sinkhorn_points_workspace_bytes(prob.B, prob.d1, prob.d2, int(prob.c_batched), prob.D, prob.lam,
                                                 prob.n_iter, prob.tol)
        ws = torch.empty((max(nws, 1),), device=dev, dtype=torch.uint8)

        def fwd(n):
            return sk.sinkhorn_forward_points(mu, nu, X, Y, prob.lam, n, prob.tol, workspace=ws)

        def bwd(out):
            return sk.sinkhorn_backward_points(g, mu, nu, X, Y, prob.lam, out["alpha"], out["beta"],
                                               grad_points=grad_C)
    else:
        C = t(prob.C)
        nws = sk.sinkhorn_workspace_bytes(prob.B, prob.d1, prob.d2, int(prob.c_batched), prob.lam, prob.n_iter,
                                          prob.tol)
        ws = torch.empty((max(nws, 1),), device=dev, dtype=torch.uint8)

        def fwd(n):
            if args.select != "default":
                return sk.sinkhorn_forward_select(args.select, mu, nu, C, prob.lam, n, prob.tol, workspace=ws)
            return sk.sinkhorn_forward(mu, nu, C, prob.lam, n, prob.tol, workspace=ws)

        def bwd(out):
            if args.sharp:
                return sk.sinkhorn_backward_sharp(g, mu, nu, C, prob.lam, out["alpha"], out["beta"])
            return sk.sinkhorn_backward(g, mu, nu, C, prob.lam, out["alpha"], out["beta"], grad_C=grad_C)
    regime = sk.sinkhorn_regime(prob.B, prob.d1, prob.d2, int(prob.c_batched), prob.lam, prob.n_iter, prob.tol)

    def step():
        out = fwd(prob.n_iter)
        bwd(out)
        return out

    for _ in range(args.warmup):
        out = step()
    torch.cuda.synchronize()
    iters = out["iters"].cpu().numpy().astype(np.float64)
    cells_per_step = float(iters.sum()) * prob.d1 * prob.d2

    stream = torch.cuda.current_stream(dev)
    # The timed region: K steps back to back, bracketed by one event pair
    # (events between the steps would add their own time to every step).
    e_all0, e_all1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e_all0.record(stream)
    for k in range(args.steps):
        out = step()
    e_all1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = e_all0.elapsed_time(e_all1) / args.steps
    # The forward / backward split, from a second pass with events around
    # each half (reported beside the step time, not used for it).
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    bev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for k in range(args.steps):
        ev[k][0].record(stream)
        o = fwd(prob.n_iter)
        ev[k][1].record(stream)
        bev[k][0].record(stream)
        bwd(o)
        bev[k][1].record(stream)
    torch.cuda.synchronize()
    fwd_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    bwd_ms = float(np.mean([a.elapsed_time(b) for a, b in bev]))

    # Roofline of the dominant kernel.
    if regime == 1 and args.select == "log":
        # The log-domain kernel alone: one launch per forward.  Algorithmic
        # work: one exp2 per cell per iteration, plus the first (exact)
        # v-update and the closing measurement: (iters + 2) d1 d2 per problem.
        kname = "sk_resident_log_kernel"
        kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for k in range(args.steps):
            kev[k][0].record(stream)
            fwd(prob.n_iter)
            kev[k][1].record(stream)
        torch.cuda.synchronize()
        kernel_ms = float(np.mean([a.elapsed_time(b) for a, b in kev]))
        exps = float(np.sum(iters + 2.0)) * prob.d1 * prob.d2
        achieved = exps / (kernel_ms * 1e-3) / 1e12
        src = kernel_source_hash(["sk_resident.hip", "sk_resident_log.h", "sk_resident_gen.h", "sk_device.h"])
        roof = dict(bound="alu", achieved=round(achieved, 4), peak=round(PEAK_EXP_TS, 4), unit="Texp/s",
                    frac=round(achieved / PEAK_EXP_TS, 4),
                    traffic=stored_traffic(f"{kname}_{prob.name}_counters.md", src),
                    **counter_fields(f"{kname}_{prob.name}_counters.md", src), kernel=kname,
                    kernel_ms=round(kernel_ms, 5), work="exp2 per launch = (iters + 2)*d1*d2 per problem")
    elif regime == 1:
        # Resident regime: the first-choice plain-form kernel solves every
        # problem (the fallbacks launched after it find nothing to do).  Its
        # duration alone is taken with events around launches of that kernel
        # only, on the stream the library launches on.  Algorithmic work: two
        # matrix-vector products (4*d1*d2 flops) per iteration, plus the first
        # v-update and the three products of the closing measurement (6*d1*d2).
        kname, kfiles, bound, peak = RESIDENT_KERNELS[resident_kind(prob)]
        kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for k in range(args.steps):
            kev[k][0].record(stream)
            kout = sk.sinkhorn_forward_select("plain", mu, nu, C, prob.lam, prob.n_iter, prob.tol, workspace=ws)
            kev[k][1].record(stream)
        torch.cuda.synchronize()
        if not bool((kout["iters"] >= 0).all()):
            raise RuntimeError("the plain-form kernel left problems to the fallback; its roofline does not apply")
        kernel_ms = float(np.mean([a.elapsed_time(b) for a, b in kev]))
        flops = float(np.sum(4.0 * iters + 6.0)) * prob.d1 * prob.d2
        achieved = flops / (kernel_ms * 1e-3) / 1e12
        src = kernel_source_hash([*kfiles, "sk_device.h"])
        traffic = stored_traffic(f"{kname}_{prob.name}_counters.md", src)
        roof = dict(bound=bound, achieved=round(achieved, 3), peak=peak, unit="TFLOP/s",
                    frac=round(achieved / peak, 4), traffic=traffic,
                    **counter_fields(f"{kname}_{prob.name}_counters.md", src), kernel=kname,
                    kernel_ms=round(kernel_ms, 5),
                    work="fp32 flops per launch = (4*iters + 6)*d1*d2 per problem")
    else:
        # Tiled regime: the dominant kernel is the sweep (one pass over the
        # cost per iteration; all other launches of a forward are fixed
        # costs).  Its average duration is taken live on the library's stream
        # from forwards at n and n/2 iterations, whose difference cancels the
        # fixed launches exactly.  Shared cost: exp bound, one exp2 per cell
        # per sweep.  Per-sample cost: HBM bound, the cost read once per sweep.
        n_hi, n_lo = prob.n_iter, max(prob.n_iter // 2, 1)
        tfwd = {}
        for n in (n_lo, n_hi):
            fwd(n)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = max(2, args.steps // 2)
            e0.record(stream)
            for _ in range(reps):
                o = fwd(n)
            e1.record(stream)
            torch.cuda.synchronize()
            tfwd[n] = (e0.elapsed_time(e1) / reps, float(o["iters"].cpu().numpy().astype(np.float64).sum()))
        sweeps = (tfwd[n_hi][1] - tfwd[n_lo][1]) / prob.B  # sweeps per problem between the two runs
        kernel_ms = (tfwd[n_hi][0] - tfwd[n_lo][0]) / max(sweeps, 1.0)
        cells = float(prob.B) * prob.d1 * prob.d2
        src = kernel_source_hash(["sk_tiled.hip", "sk_device.h"])
        if points:
            # The cost is recreated from the coordinates: nothing streams, the
            # sweep is bound by one exp2 per cell (plus the distance arithmetic);
            # timed with its merge, like the shared-cost sweep.
            kname = "sk_tiled_sweep_points"
            achieved = cells / (kernel_ms * 1e-3) / 1e12
            roof = dict(bound="alu", achieved=round(achieved, 4), peak=round(PEAK_EXP_TS, 4), unit="Texp/s",
                        frac=round(achieved / PEAK_EXP_TS, 4), kernel=kname + " + sk_tiled_merge_cols",
                        kernel_ms=round(kernel_ms, 5), work="exp2 per iteration = B*d1*d2 (one per cell)")
        elif prob.c_batched:
            kname = "sk_tiled_sweep_stream"
            nbytes = 4.0 * cells
            achieved = nbytes / (kernel_ms * 1e-3) / 1e9
            roof = dict(bound="hbm", achieved=round(achieved, 2), peak=PEAK_HBM_GBS, unit="GB/s",
                        frac=round(achieved / PEAK_HBM_GBS, 4), kernel=kname, kernel_ms=round(kernel_ms, 5),
                        work="cost bytes read per sweep = 4*B*d1*d2")
        else:
            # A shared cost's iteration is the sweep plus the merge of its
            # row-block partials (a short launch that also takes the stop
            # test): timed and reported as the pair.
            kname = "sk_tiled_sweep_shared"
            achieved = cells / (kernel_ms * 1e-3) / 1e12
            roof = dict(bound="alu", achieved=round(achieved, 4), peak=round(PEAK_EXP_TS, 4), unit="Texp/s",
                        frac=round(achieved / PEAK_EXP_TS, 4), kernel=kname + " + sk_tiled_merge_cols",
                        kernel_ms=round(kernel_ms, 5), work="exp2 per iteration = B*d1*d2 (one per cell)")
        roof["traffic"] = stored_traffic(f"{kname}_{prob.name}_counters.md", src)
        roof.update(counter_fields(f"{kname}_{prob.name}_counters.md", src))
        roof["sweep_timing"] = f"(t_fwd(n={n_hi}) - t_fwd(n={n_lo})) / {sweeps:g} sweeps, events on the library stream"

    res = {
        "metric": "Sinkhorn cell-updates/s (B*d1*d2*iters/s) fwd+bwd",
        "value": cells_per_step / (ms_per_step * 1e-3),
        "unit": "cell-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "wall_ms_per_step": wall / args.steps * 1e3,
        "fwd_ms": fwd_ms,
        "bwd_ms": bwd_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": WORKLOAD_NAMES[args.config],
            "B": prob.B, "d1": prob.d1, "d2": prob.d2, "lambda": prob.lam, "n_iter": prob.n_iter,
            "tol": prob.tol, "c_batched": bool(prob.c_batched), "iters_done_mean": float(iters.mean()),
            **({"D": prob.D, "cost": "from points"} if points else {}),
            **({"backward": "sharp: gradient of E^0 by implicit differentiation (conjugate gradients)"}
               if args.sharp else {}),
            **({"select": args.select} if args.select != "default" else {}),
            **({"overrides": {k: v for k, v in (("B", args.batch or None), ("tol", args.tol),
                                                 ("n_iter", args.n_iter)) if v is not None}}
               if (args.batch or args.tol is not None or args.n_iter is not None) else {}),
            "regime": {1: "resident", 2: "tiled"}.get(regime, "?"),
        },
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        if points:
            res["cpu_baseline"] = cpu_baseline_points(prob, 2)
        elif args.config in (1, 2):
            res["cpu_baseline"] = cpu_baseline(prob, grad_C, sharp=args.sharp)
        else:
            res["cpu_baseline"] = cpu_baseline_sampled(prob, grad_C, {3: 2 if args.sharp else 16, 4: 1, 5: 2}[args.config],
                                                       sharp=args.sharp, n_iter=300 if args.config == 4 else None)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

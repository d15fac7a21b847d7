#!/usr/bin/env python3
"""Benchmark of the fused FlashNorm norm-then-project path on one MI355X.

A step is one pass of the hot path over one batch of synthetic input: one call
of the fused op (kernel selection + one kernel launch) on inputs and a folded
weight already resident in HBM.  The fold (W* = diag(g) W, done once at load
time) is outside the timed region.  Several independent input/weight/output
sets are rotated so the working set exceeds the 256 MB Infinity Cache and every
step streams its operands from HBM.  The same-library unfused baseline
(normalisation kernel -> the same matrix-multiply kernel) is timed the same way.

Prints ONE JSON line (rank 0) with the throughput, the roofline of the fused
kernel (algorithmic FLOPs or bytes per launch / measured launch time) and the
fp64 CPU oracle timed on a bounded sample of the same workload.

  python bench.py [--steps 100] [--warmup 20] [--workload llama7b_qkv_prefill] [--variant folded]

The default workload is the largest single-GPU configuration, the Llama-7B-scale
fused QKV prefill (a[4096, 4096] -> 12288 columns, bf16).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused RMSNorm+proj TFLOP/s (prefill), HBM GB/s (decode), % of MI355X peak"
# MI355X published peaks: dense bf16 matrix cores 2.5 PFLOP/s (256 CU x 2.4 GHz x
# 4096 FLOP/clk), fp32 vector 157.3 TFLOP/s, HBM3E 8 TB/s.
PEAK_BF16_TFLOPS = 2516.6
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
CACHE_BYTES = 256 * 2 ** 20  # Infinity Cache; the rotation keeps >= 2x this resident


def parse_args():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="llama7b_qkv_prefill",
                   choices=["tiny_fp32", "smollm2_prefill", "llama7b_qkv_prefill", "llama7b_swiglu_decode",
                            "layernorm_linear", "mla_kv_down"])
    p.add_argument("--decode-m", type=int, default=16, choices=[1, 4, 16])
    p.add_argument("--variant", default="folded", choices=["folded", "unfolded", "qkv_rope", "qkv_headnorm", "mla"],
                   help="folded: W* = diag(g) W folded offline (the default path); unfolded: g applied at "
                        "run time to an unfolded W (linear and GLU workloads); qkv_rope: the projection as "
                        "fused Q|K|V heads with RoPE on Q and K; qkv_headnorm: the same with QK-norm (per-head "
                        "RMSNorm of Q and K, Prop. 3) before RoPE (linear workloads); mla: the projection as an MLA "
                        "latent (RMS-normalised, Prop. 3) plus a 64-wide rotary key (--workload mla_kv_down)")
    p.add_argument("--rope-h", type=int, default=0,
                   help="qkv_rope head width (default 128 for Llama-7B, else 64); Hq = Hkv = N / (3 h)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--repeats", type=int, default=5,
                   help="further timed passes after the reported one, for the spread across passes")
    p.add_argument("--no-unfused", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle timing sample")
    p.add_argument("--eager", action="store_true",
                   help="launch every step from Python instead of replaying a captured HIP graph")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 256 MiB device copy (known traffic) for counter calibration")
    return p.parse_args()


class Setup:
    """GPU-resident rotating operand sets and the closures that run one step."""

    def __init__(self, name, decode_m, variant="folded", rope_h=0):
        import torch
        from paper_2407_09577_amd import flashnorm as fn
        from paper_2407_09577_amd import workloads

        self.fn = fn
        self.torch = torch
        gen = workloads.WORKLOADS[name]
        self.w = w = gen(M=decode_m) if name == "llama7b_swiglu_decode" else gen()
        dev = torch.device("cuda:0")
        self.kind = w.kind
        M, K = w.M, w.K
        ncols = w.out_features
        es = w.a.element_size()
        layout = fn.FN_LAYOUT_GLU if w.kind == "glu" else fn.FN_LAYOUT_LINEAR
        a0 = w.a.to(dev)
        W0 = w.W.to(dev)
        g0 = w.g.to(dev)
        beta0 = w.beta.to(dev) if w.beta is not None else None
        ln = w.kind == "layernorm"
        Ws0, cs0, cb0 = fn.fold_weights(W0, g0, beta=beta0, layout=layout, colsum=ln, c_star=ln)
        Wp0, _, _ = fn.fold_weights(W0, None, layout=layout)  # unfolded, for the baseline
        del W0
        self.ws_bytes = Ws0.numel()
        set_bytes = a0.numel() * es + self.ws_bytes + M * ncols * es
        self.nsets = max(2, -(-2 * CACHE_BYTES // set_bytes))
        self.sets = []
        for i in range(self.nsets):
            a = a0 if i == 0 else a0.clone()
            Ws = Ws0 if i == 0 else Ws0.clone()
            Wp = Wp0 if i == 0 else Wp0.clone()
            y = torch.empty(M, ncols, dtype=w.a.dtype, device=dev)
            x = torch.empty_like(a)
            self.sets.append((a, Ws, Wp, y, x))
        self.g, self.beta, self.cs, self.cb = g0, beta0, cs0, cb0
        self.M, self.K, self.ncols, self.es = M, K, ncols, es
        self.N = w.N
        self.settle_s = 0.25
        self.variant = variant
        if variant == "unfolded" and w.kind == "layernorm":
            raise SystemExit("--variant unfolded covers the RMSNorm workloads")
        if variant in ("qkv_rope", "qkv_headnorm"):
            if w.kind != "linear":
                raise SystemExit(f"--variant {variant} covers the linear workloads")
            h = rope_h or (128 if name == "llama7b_qkv_prefill" else 64)
            if w.N % (3 * h):
                raise SystemExit(f"N = {w.N} is not 3 x heads x {h}")
            self.rope = (w.N // (3 * h), w.N // (3 * h), h)  # Hq, Hkv, h
            cos, sin = workloads.rope_tables(4096, h)
            self.rope_cos, self.rope_sin = cos.to(dev), sin.to(dev)
            self.rope_pos_cpu = workloads.positions(M, 2048)  # sequences of 2048 tokens
            self.rope_pos = self.rope_pos_cpu.to(dev)
            self.rope_qs = h ** -0.5
            gen_hn = torch.Generator().manual_seed(1)
            self.hn_gq_cpu = torch.rand(h, generator=gen_hn) + 0.5  # per-head norm weights
            self.hn_gk_cpu = torch.rand(h, generator=gen_hn) + 0.5
            self.hn_gq, self.hn_gk = self.hn_gq_cpu.to(dev), self.hn_gk_cpu.to(dev)

        if variant == "mla":
            if w.kind != "linear":
                raise SystemExit("--variant mla covers the linear workloads")
            R = rope_h or 64
            if w.N <= R or (w.N - R) % 8 or w.N - R > 2048:
                raise SystemExit(f"N = {w.N} is not a latent (multiple of 8, <= 2048) plus {R} rotary columns")
            self.mla = (w.N - R, R)  # L, R
            cos, sin = workloads.rope_tables(4096, R)
            self.rope_cos, self.rope_sin = cos.to(dev), sin.to(dev)
            self.rope_pos_cpu = workloads.positions(M, 2048)
            self.rope_pos = self.rope_pos_cpu.to(dev)
            gen_l = torch.Generator().manual_seed(2)
            self.g_lat_cpu = torch.rand(w.N - R, generator=gen_l) + 0.5  # latent norm weight
            self.g_lat = self.g_lat_cpu.to(dev)
            self.mla_inv = torch.empty(M, dtype=torch.float32, device=dev)

    def run(self, i):
        fn, w = self.fn, self.w
        a, Ws, Wp, y, _ = self.sets[i % self.nsets]
        if self.variant == "unfolded":
            if self.kind == "glu":
                fn.flashnorm_glu_unfolded(a, self.g, Wp, self.ncols, w.eps, out=y)
            else:
                fn.flashnorm_linear_unfolded(a, self.g, Wp, self.ncols, w.eps, out=y)
        elif self.variant == "qkv_rope":
            Hq, Hkv, h = self.rope
            fn.flashnorm_qkv_rope(a, Ws, Hq, Hkv, h, w.eps, self.rope_pos, self.rope_cos, self.rope_sin,
                                  self.rope_qs, out=y)
        elif self.variant == "qkv_headnorm":
            Hq, Hkv, h = self.rope
            fn.flashnorm_qkv_headnorm(a, Ws, Hq, Hkv, h, w.eps, self.hn_gq, self.hn_gk, None, 1e-6,
                                      positions=self.rope_pos, cos_tab=self.rope_cos, sin_tab=self.rope_sin,
                                      q_scale=self.rope_qs, out=y)
        elif self.variant == "mla":
            L, R = self.mla
            fn.flashnorm_mla_latent(a, Ws, L, R, self.g_lat, 1e-6, w.eps, self.rope_pos, self.rope_cos,
                                    self.rope_sin, out=y, inv_rms=self.mla_inv)
        elif self.kind == "glu":
            fn.flashnorm_glu(a, Ws, self.ncols, w.eps, out=y)
        elif self.kind == "layernorm":
            fn.flashnorm_layernorm_linear(a, Ws, self.cs, self.cb, self.ncols, w.eps, out=y)
        else:
            fn.flashnorm_linear(a, Ws, self.ncols, w.eps, out=y)

    def run_unfused(self, i):
        fn, w = self.fn, self.w
        a, _, Wp, y, x = self.sets[i % self.nsets]
        if self.kind == "glu":
            fn.baseline_rmsnorm_glu(a, self.g, Wp, self.ncols, w.eps, x_ws=x, out=y)
        elif self.kind == "layernorm":
            fn.baseline_layernorm_linear(a, self.g, self.beta, Wp, self.ncols, w.eps, x_ws=x, out=y)
        else:
            fn.baseline_rmsnorm_linear(a, self.g, Wp, self.ncols, w.eps, x_ws=x, out=y)
        if self.variant == "qkv_rope":
            Hq, Hkv, h = self.rope
            fn.baseline_rope(y, Hq, Hkv, h, self.rope_pos, self.rope_cos, self.rope_sin, self.rope_qs)
        elif self.variant == "qkv_headnorm":
            Hq, Hkv, h = self.rope
            fn.baseline_qkv_headnorm(y, Hq, Hkv, h, self.hn_gq, self.hn_gk, None, 1e-6, self.rope_pos,
                                     self.rope_cos, self.rope_sin, self.rope_qs)
        elif self.variant == "mla":
            L, R = self.mla
            fn.baseline_mla_latent(y, L, R, self.g_lat, 1e-6, self.rope_pos, self.rope_cos, self.rope_sin)

    def flops(self):
        return 2.0 * self.M * self.K * self.N

    def alg_bytes(self):
        """Read a once, read W* once, write the output once."""
        return self.M * self.K * self.es + self.ws_bytes + self.M * self.ncols * self.es

    def time_steps(self, fn_step, steps, warmup, graph=True, repeats=0):
        """Average ms per step over `steps` steps, HIP events on the launch stream.
        graph=True captures the steps into one HIP graph and times its replay, so
        small kernels are not limited by Python launch overhead.  With repeats > 0 the
        timed region is followed by `repeats` more timed passes, whose per-step averages
        are returned as well (the spread across passes)."""
        torch = self.torch
        for i in range(warmup):
            fn_step(i)
        torch.cuda.synchronize()
        g = None
        if graph:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(steps):
                    fn_step(warmup + i)
            g.replay()  # warm replay
            torch.cuda.synchronize()
        # Untimed: keep the GPU busy with the same work for a moment so that the
        # timed region runs at the settled clock, not the idle-to-busy ramp.
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < self.settle_s:
            if g is not None:
                g.replay()
            else:
                for i in range(steps):
                    fn_step(warmup + i)
            torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(stream)
        if g is not None:
            g.replay()
        else:
            for i in range(steps):
                fn_step(warmup + i)
        end.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / steps  # ms per step
        if not repeats:
            return ms
        more = []
        for _ in range(repeats):
            start.record(stream)
            if g is not None:
                g.replay()
            else:
                for i in range(steps):
                    fn_step(warmup + i)
            end.record(stream)
            torch.cuda.synchronize()
            more.append(start.elapsed_time(end) / steps)
        return ms, more


def cpu_baseline(w, unit, target_s, flops_per_row, bytes_total, s=None):
    """Time the fp64 oracle (as it stands) on a bounded sample of rows of the same workload."""
    import numpy as np
    import oracle

    a = w.a.double().numpy()
    g, W = w.g.double().numpy(), w.W.double().numpy()
    beta = w.beta.double().numpy() if w.beta is not None else None
    rope = s is not None and s.variant in ("qkv_rope", "qkv_headnorm")
    if rope:
        Hq, Hkv, h = s.rope
        rope_args = (Hq, Hkv, h, s.rope_pos_cpu.numpy(), s.rope_cos.cpu(), s.rope_sin.cpu(), s.rope_qs)

    def call(rows):
        if s is not None and s.variant == "mla":
            L, R = s.mla
            oracle.rmsnorm_mla_latent(a, g, W, w.eps, L, s.g_lat_cpu, 1e-6, s.rope_pos_cpu.numpy(), s.rope_cos.cpu(),
                                      s.rope_sin.cpu(), rows=rows)
        elif rope and s.variant == "qkv_headnorm":
            Hq, Hkv, h, pos, cos, sin, qs = rope_args
            oracle.rmsnorm_qkv_headnorm(a, g, W, w.eps, Hq, Hkv, h, s.hn_gq_cpu, s.hn_gk_cpu, None, 1e-6, pos=pos,
                                        cos_tab=cos, sin_tab=sin, q_scale=qs, rows=rows)
        elif rope:
            oracle.rmsnorm_qkv_rope(a, g, W, w.eps, *rope_args, rows=rows)
        elif w.kind == "glu":
            oracle.rmsnorm_swiglu(a, g, W, w.eps, rows=rows)
        elif w.kind == "layernorm":
            oracle.layernorm_linear(a, g, beta, W, w.eps, rows=rows)
        else:
            oracle.rmsnorm_linear(a, g, W, w.eps, rows=rows)

    probe = np.arange(min(w.M, max(4, oracle.num_threads())))
    call(probe)  # warm (page-in, thread pool)
    t0 = time.perf_counter()
    call(probe)
    per_row = (time.perf_counter() - t0) / probe.size
    n = int(max(probe.size, min(w.M, target_s / max(per_row, 1e-9))))
    rows = np.arange(n)
    reps = 0
    t0 = time.perf_counter()
    while True:  # the whole workload may take far less than the target: repeat it
        call(rows)
        reps += 1
        if n < w.M or time.perf_counter() - t0 >= target_s:
            break
    t = (time.perf_counter() - t0) / reps
    if unit == "TFLOP/s":
        value = flops_per_row * n / t / 1e12
    else:  # whole-op bytes over the time the oracle would take for all M rows
        value = bytes_total / (t * w.M / n) / 1e9
    what = f"all {w.M} rows, {reps} repetitions" if n == w.M else f"rows 0..{n - 1} of {w.M}"
    return {"value": value, "unit": unit, "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"fp64 oracle (standard form) on {what} of the same workload, {t * reps:.1f} s wall"}


def copy_calibration():
    """A plain device copy of known size: FETCH_SIZE/WRITE_SIZE read for it calibrate the counters."""
    import torch
    n = 256 * 2 ** 20
    x = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "dispatches": 5}), flush=True)


def main():
    args = parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); "
              "the FlashNorm path here is a single-GPU kernel library", file=sys.stderr)
        sys.exit(2)
    import torch
    import __graft_entry__ as graft

    graft.ensure_built()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    s = Setup(args.workload, args.decode_m, args.variant, args.rope_h)
    w = s.w
    decode = args.workload == "llama7b_swiglu_decode"
    fp32 = w.a.dtype == torch.float32

    torch.cuda.synchronize()
    graph = not args.eager
    timed = s.time_steps(s.run, args.steps, args.warmup, graph, repeats=args.repeats)
    ms, passes = timed if isinstance(timed, tuple) else (timed, [])
    ms_unf = None if args.no_unfused else s.time_steps(s.run_unfused, args.steps, args.warmup, graph)

    t = ms * 1e-3
    if decode:
        unit = "GB/s"
        value = s.alg_bytes() / t / 1e9
        roof = {"bound": "hbm", "achieved": value, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": value / PEAK_HBM_GBS, "traffic": None}
    else:
        unit = "TFLOP/s"
        value = s.flops() / t / 1e12
        peak = PEAK_F32_TFLOPS if fp32 else PEAK_BF16_TFLOPS
        roof = {"bound": "alu" if fp32 else "mfma", "achieved": value, "peak": peak, "unit": "TFLOP/s",
                "frac": value / peak, "traffic": None}

    # HBM traffic per launch from the committed rocprofv3 counter summary of this
    # workload, only if it was taken with the current kernel sources.
    from paper_2407_09577_amd import profiling
    prof_key = args.workload if not decode else f"{args.workload}_m{args.decode_m}"
    if args.variant != "folded":
        prof_key += f"_{args.variant}"
    prof = profiling.read_summary(prof_key)
    if prof is not None:
        roof["traffic"] = float(prof["traffic_bytes_per_launch"])

    cpu = None
    if not args.no_cpu_baseline:
        per_row = 2.0 * w.K * w.N
        cpu = cpu_baseline(w, unit, args.cpu_seconds, per_row, s.alg_bytes(), s)

    config = {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "out_features": s.ncols, "eps": w.eps,
              "op": {"glu": "flashnorm_glu", "layernorm": "flashnorm_layernorm_linear"}.get(w.kind, "flashnorm_linear"),
              "variant": args.variant,
              "step": "one fused call on HBM-resident inputs; weight fold done once before timing",
              "launch": "HIP graph replay of the timed steps" if graph else "eager launches from Python",
              "rotating_sets": s.nsets, "alg_flops_per_step": s.flops(), "alg_bytes_per_step": s.alg_bytes(),
              "parallelism": "single GPU"}
    if args.variant == "unfolded":
        config["op"] = config["op"].replace("flashnorm_linear", "flashnorm_linear_unfolded").replace(
            "flashnorm_glu", "flashnorm_glu_unfolded")
    elif args.variant in ("qkv_rope", "qkv_headnorm"):
        Hq, Hkv, h = s.rope
        config.update(op="flashnorm_" + args.variant, heads={"Hq": Hq, "Hkv": Hkv, "h": h},
                      positions="sequences of 2048 tokens")
    elif args.variant == "mla":
        L, R = s.mla
        config.update(op="flashnorm_mla_latent", mla={"L": L, "R": R, "eps_lat": 1e-6},
                      positions="sequences of 2048 tokens",
                      kernels_per_step="2 (fused projection, latent pass); roofline.achieved uses the whole step")
    if prof is not None:
        config["traffic_profile"] = prof["path"]
        if "kernel_timed_avg_duration_us" in prof:
            config["profile_kernel_timed_avg_us"] = float(prof["kernel_timed_avg_duration_us"])
    if passes:
        allp = sorted([ms] + passes)
        pick = lambda q: allp[min(len(allp) - 1, int(round(q * (len(allp) - 1))))]
        config["us_per_step_passes"] = {"passes": len(allp), "median": pick(0.5) * 1e3, "min": allp[0] * 1e3,
                                        "p90": pick(0.9) * 1e3, "max": allp[-1] * 1e3,
                                        "mean": sum(allp) / len(allp) * 1e3}
    if ms_unf is not None:
        config["unfused_ms_per_step"] = ms_unf
        config["unfused_over_fused"] = ms_unf / ms  # speedup of the fused op (x)
        config["fused_latency_reduction"] = (ms_unf - ms) / ms_unf  # the paper's (t_base - t) / t_base
    out = {"metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32" if fp32 else "bf16", "data": "synthetic",
           "config": config, "roofline": roof, "cpu_baseline": cpu}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

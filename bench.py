"""Throughput of one decoder-layer training step on one MI355X.

Workload: the 8B-shape decoder layer (micro-batch 1 x seq 4096, hidden 4096,
32 query / 8 kv heads of 128, SwiGLU FFN 14336, RoPE base 5e5), bf16 with
fp32 gradient accumulation. One step = layer forward + layer backward + fused
clip/AdamW/bf16 write-back over all 218 M parameters of the layer (flat fp32
master, moments and gradient), on synthetic seeded inputs resident in HBM.

Prints one JSON line: model TFLOP/s (App. C count of the layer fwd+bwd, the
optimizer adds time but no model FLOPs), MFU against the MI355X dense bf16
peak, tokens/s, the roofline of the dominant kernel (measured here with HIP
events on the stream it runs on) and the fp64 CPU oracle's rate on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# BLAS threads for the CPU-baseline leg: every core this process may use
_CORES = len(os.sched_getaffinity(0))
os.environ.setdefault("OPENBLAS_NUM_THREADS", str(_CORES))
os.environ.setdefault("OMP_NUM_THREADS", str(_CORES))

import numpy as np  # noqa: E402

import forge_inputs as fi  # noqa: E402
from paper_2609_13645_amd import flops  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA (published)
MFU_PEAK_TFLOPS = 2516.6           # 256 CU x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0
METRIC = "model TFLOP/s and MFU (%) per fwd+bwd+AdamW step, tokens/s, 1×MI355X"
WORKLOAD = "llama8b_layer"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seq", type=int, default=4096,
                    help="tokens of the CPU-baseline sample")
    ap.add_argument("--kernel-reps", type=int, default=20)
    return ap.parse_args()


def gpu_step_bench(cfg, steps, warmup, kernel_reps):
    import torch
    from paper_2609_13645_amd import _lib, runtime

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    inp = fi.layer_inputs(cfg)
    flat = runtime.FlatParams(runtime.layer_shapes(cfg))
    layer = runtime.Layer(cfg, inp["weights"], flat=flat, stream=stream)
    x = runtime.to_device_bf16(inp["x"])
    dy = runtime.to_device_bf16(inp["dy"])
    out = torch.empty_like(x)
    dx = torch.empty_like(x)
    hp = _lib.AdamwHparams(cfg["beta1"], cfg["beta2"], cfg["adam_eps"], cfg["weight_decay"])
    scal = torch.zeros(4, dtype=torch.float32, device="cuda")
    host_scal = torch.zeros(4, dtype=torch.float32).pin_memory()
    step_no = [0]

    def step():
        step_no[0] += 1
        t = step_no[0]
        host_scal.copy_(torch.tensor([cfg["lr"], 1 - cfg["beta1"] ** t,
                                      1 - cfg["beta2"] ** t, 1.0]))
        scal.copy_(host_scal, non_blocking=True)
        flat.grad.zero_()
        layer.fwd(x, out)
        layer.bwd(x, dy, dx)
        _lib.forge_adamw_step(flat.master, flat.param, flat.grad, flat.m, flat.v, flat.n,
                              hp, scal, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    assert torch.isfinite(out.float()).all() and torch.isfinite(flat.master).all()

    # phase split (separate pass, not part of the headline number)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    phases = {"fwd": 0.0, "bwd": 0.0, "adamw": 0.0}
    reps = max(3, min(steps, 10))
    for _ in range(reps):
        flat.grad.zero_()
        ev[0].record(stream)
        layer.fwd(x, out)
        ev[1].record(stream)
        layer.bwd(x, dy, dx)
        ev[2].record(stream)
        _lib.forge_adamw_step(flat.master, flat.param, flat.grad, flat.m, flat.v, flat.n,
                              hp, scal, stream)
        ev[3].record(stream)
        torch.cuda.synchronize()
        phases["fwd"] += ev[0].elapsed_time(ev[1]) / reps
        phases["bwd"] += ev[1].elapsed_time(ev[2]) / reps
        phases["adamw"] += ev[2].elapsed_time(ev[3]) / reps

    # dominant kernel: the gate/up projection GEMM (largest single launch of
    # the step, y = b W_gu^T, M = T, N = 2f, K = h), run alone on the step's
    # stream on buffers of its shape
    T, h, f = fi.tokens(cfg), cfg["hidden"], cfg["ffn"]
    A = torch.randn((T, h), device="cuda").to(torch.bfloat16)
    C = torch.empty((T, 2 * f), dtype=torch.bfloat16, device="cuda")
    Wgu = layer.w["w_gate_up"]

    def gemm():
        _lib.forge_gemm(_lib.GEMM_KC, _lib.GEMM_KC, _lib.EPI_STORE_BF16, A, Wgu, C, None,
                        T, 2 * f, h, h, h, 2 * f, 0, stream)

    for _ in range(3):
        gemm()
    e0.record(stream)
    for _ in range(kernel_reps):
        gemm()
    e1.record(stream)
    torch.cuda.synchronize()
    k_ms = e0.elapsed_time(e1) / kernel_reps
    k_flop = 2.0 * T * (2 * f) * h
    kernel = {"name": "gemm_kernel<256,256,4,2,KC,KC,StoreBF16> (gate/up fwd)",
              "shape": f"M={T} N={2 * f} K={h}", "avg_us": k_ms * 1e3,
              "flop_per_launch": k_flop}
    return ms, phases, kernel, flat.n


def cpu_baseline(cfg, seq):
    """The fp64 oracle (as it stands) on a bounded sample of the workload."""
    from oracle import dense, adamw as oadam
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = _CORES
    c = dict(cfg, seq=seq)
    inp = fi.layer_inputs(c)
    W = {k: fi.bf16_bits_to_f64(v) for k, v in inp["weights"].items()}
    x = fi.bf16_bits_to_f64(inp["x"])
    dy = fi.bf16_bits_to_f64(inp["dy"])
    frac = seq / cfg["seq"]
    t0 = time.perf_counter()
    out, cache = dense.layer_fwd(x, W, c)
    _, grads = dense.layer_bwd(cache, W, c, dy)
    # the optimizer over the same fraction of the parameters (a prefix of them)
    budget = int(round(frac * sum(w.size for w in W.values())))
    n_opt = 0
    for name, g in grads.items():
        if budget <= 0:
            break
        k = min(budget, g.size)
        p, gg = W[name].reshape(-1)[:k], g.reshape(-1)[:k]
        oadam.adamw_step(p, gg, np.zeros_like(p), np.zeros_like(p), cfg["lr"], cfg["beta1"],
                         cfg["beta2"], cfg["adam_eps"], cfg["weight_decay"], 1)
        budget -= k
        n_opt += k
    dt = time.perf_counter() - t0
    model_flop = flops.step_flops(c)
    return {"value": model_flop / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"fp64 oracle, {frac:.3f} of one step of the same 8B-shape layer: "
                       f"fwd+bwd over the first {seq} of the 4096 tokens, AdamW over "
                       f"{n_opt / 1e6:.1f}M of the 218.1M params; {dt:.1f} s for "
                       f"{model_flop / 1e12:.3f} TFLOP of model work"),
            "seconds": dt}


def summarize_profile(db_path, out=sys.stdout):
    """Per-kernel, per-grid dispatch statistics from a rocprofv3 (rocpd) database."""
    import collections
    import re
    import sqlite3
    con = sqlite3.connect(db_path)
    rows = con.execute("select name, grid_x, grid_y, grid_z, workgroup_x, workgroup_y, "
                       "workgroup_z, duration from kernels").fetchall()
    agg = collections.defaultdict(list)
    for name, gx, gy, gz, wx, wy, wz, dur in rows:
        short = name.replace("forge::(anonymous namespace)::", "").replace("void ", "")
        short = re.sub(r"\(.*", "", short)
        grid = f"{gx // max(wx, 1)}x{gy // max(wy, 1)}x{gz // max(wz, 1)}"
        agg[(short[:72], grid, wx * wy * wz)].append(dur / 1e3)
    total = sum(sum(v) for v in agg.values())
    print("| kernel | workgroups | threads/WG | calls | avg us | min us | max us | "
          "total ms | share |", file=out)
    print("|---|---|---|---|---|---|---|---|---|", file=out)
    for (n, g, th), d in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{n}` | {g} | {th} | {len(d)} | {sum(d) / len(d):.1f} | {min(d):.1f} | "
              f"{max(d):.1f} | {sum(d) / 1e3:.3f} | {100 * sum(d) / total:.1f}% |", file=out)


def main():
    if len(sys.argv) == 3 and sys.argv[1] == "--summarize":
        summarize_profile(sys.argv[2])
        return
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build runs one decoder-layer step on one "
              "MI355X and has no multi-GPU path (--gpus must be 1).", file=sys.stderr)
        sys.exit(2)
    cfg = fi.config(args.workload)
    T = fi.tokens(cfg)
    step_flop = flops.step_flops(cfg)
    print(f"[bench] workload {args.workload}: T={T} h={cfg['hidden']} f={cfg['ffn']} "
          f"warmup={args.warmup} steps={args.steps}", file=sys.stderr, flush=True)
    ms, phases, kernel, nparams = gpu_step_bench(cfg, args.steps, args.warmup,
                                                 args.kernel_reps)
    tflops = step_flop / (ms * 1e-3) / 1e12
    print(f"[bench] {ms:.3f} ms/step, {tflops:.1f} TFLOP/s; phases {phases}",
          file=sys.stderr, flush=True)
    k_tf = kernel["flop_per_launch"] / (kernel["avg_us"] * 1e-6) / 1e12
    res = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "mfu_pct": round(100.0 * tflops / MFU_PEAK_TFLOPS, 2),
        "mfu_fwd_bwd_pct": round(100.0 * step_flop / ((phases["fwd"] + phases["bwd"]) * 1e-3)
                                 / 1e12 / MFU_PEAK_TFLOPS, 2),
        "tokens_per_s": round(T / (ms * 1e-3), 1),
        "phases_ms": {k: round(v, 4) for k, v in phases.items()},
        "config": {"workload": args.workload, "batch": cfg["batch"], "seq": cfg["seq"],
                   "hidden": cfg["hidden"], "n_heads": cfg["n_heads"],
                   "n_kv_heads": cfg["n_kv_heads"], "head_dim": cfg["head_dim"],
                   "ffn": cfg["ffn"], "params": nparams,
                   "model_flop_per_step": step_flop},
        "roofline": {"bound": "mfma", "kernel": kernel["name"], "shape": kernel["shape"],
                     "achieved": round(k_tf, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(k_tf / PEAK_BF16_TFLOPS, 4),
                     "avg_us": round(kernel["avg_us"], 2), "traffic": None},
    }
    if not args.no_cpu_baseline:
        print(f"[bench] cpu baseline: oracle on {args.cpu_seq} tokens ...", file=sys.stderr,
              flush=True)
        cb = cpu_baseline(cfg, args.cpu_seq)
        res["cpu_baseline"] = {k: (round(v, 6) if isinstance(v, float) else v)
                               for k, v in cb.items() if k != "seconds"}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

"""Throughput of one training step on one MI355X.

Default workload: the 8B-shape decoder layer (micro-batch 1 x seq 4096,
hidden 4096, 32 query / 8 kv heads of 128, SwiGLU FFN 14336, RoPE base 5e5),
bf16 with fp32 gradient accumulation. One step = layer forward + layer
backward + fused clip/AdamW/bf16 write-back over all 218 M parameters of the
layer (flat fp32 master, moments and gradient; the backward writes this
step's gradients rather than accumulating into zeroed ones), on synthetic
seeded inputs resident in HBM. A layer workload's backward and optimizer are
one call (forge_layer_bwd_adamw): each weight's update starts once its
gradient is final, overlapping the rest of the backward; the clip
coefficient is 1 (no clipping), as in every step here. Other workloads (--workload): the same layer at seq 16384
with attention recomputed in the backward, the 64-expert top-8 MoE layer,
the 16-layer tied-head model (embedding, layers, LM head + cross-entropy;
each layer's weights updated inside its backward, the embedding and final
norm after the embedding backward) and the tiny one-layer model (one AdamW
over all parameters after the backward).

Prints one JSON line: model TFLOP/s (App. C count of the fwd+bwd; the
optimizer adds time but no model FLOPs), MFU against the MI355X dense bf16
peak, tokens/s, the roofline of the dominant kernel (timed here with HIP
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
METRIC = "model TFLOP/s and MFU (%) per fwd+bwd+AdamW step, tokens/s, 1×MI355X"
WORKLOAD = "llama8b_layer"
DESCRIPTION = {
    "tiny": "tiny decoder layer + untied LM head + CE + AdamW (B1 S128 h256)",
    "llama8b_layer": "Llama-8B-shape decoder layer fwd+bwd+AdamW (B1 S4096 h4096)",
    "dense1b": "16-layer dense model, tied LM head + CE + AdamW (B4 S2048 h2048 V32000)",
    "dense1b_streaming_ce": "the 16-layer dense model with the streaming CE head (2048-token "
                            "chunks: 2048 x 32000 logits at a time)",
    "llama8b_layer_16k": "Llama-8B-shape layer at S16384, attention recomputed in bwd",
    "moe_layer": "MoE decoder layer, 64 experts top-8, fe 1408 (B2 S4096 h2048)",
    "qwen3_layer": "Qwen3-0.6B-shape layer with per-head QK-Norm (B4 S4096 h1024, 16/8 x 128, "
                   "f3072)",
    "minicpm5_moe_layer": "MiniCPM5-16B-A3B-shape MoE layer: 160 experts top-16 fe 512 + shared "
                          "expert 512, muP branch scale (B4 S4096 h2048, 32/2 x 128)",
    "packed_docs_layer": "the 8B-shape layer over rows packed with documents (mean length "
                         "512), RoPE positions restarting per document",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=WORKLOAD, choices=sorted(DESCRIPTION))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step into a HIP graph and time replays of it "
                         "(measured slower than issuing the calls on ROCm 7.2 for these "
                         "workloads, so not the default)")
    ap.add_argument("--cpu-seq", type=int, default=4096,
                    help="tokens of the CPU-baseline sample (layer workloads)")
    ap.add_argument("--kernel-reps", type=int, default=20)
    ap.add_argument("--kernel-rooflines", action="store_true",
                    help="time every kernel of a dense layer's step alone and print its "
                         "roofline fraction (markdown table + JSON), then exit")
    ap.add_argument("--traffic-run", action="store_true",
                    help="run only the dominant kernel and a 1 GiB device copy (for "
                         "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE passes), then exit")
    return ap.parse_args()


def is_model(cfg):
    return cfg["vocab"] > 0


def kc_kernel_name(M, N, suffix):
    """Kernel(s) and tile the library's dispatch picks for a plain GEMM with
    both operands K-contiguous (for labelling the roofline kernel only): full
    256 x 256 tiles on the ring pipeline, with a last round at most half full
    run as 256 x 128 halves in a second launch; 256 x 192 when that fills the
    last wave of workgroups better; smaller tiles for small problems.
    `suffix` closes each template argument list."""
    big = -(-M // 256) * -(-N // 256)
    mid = -(-M // 256) * -(-N // 128)
    if big >= 256:
        tail = big % 256
        if big > 256 and 0 < tail <= 128:
            return f"ring_kernel<256,256,2,4{suffix} + ring_kernel<256,128,2,4{suffix}"
        t192 = -(-M // 256) * -(-N // 192)
        c256 = -(-big // 256) * 256.0
        c192 = -(-t192 // 256) * 192.0 / 0.74
        head = "gemm_kernel<256,192,4,2" if c192 < c256 else "ring_kernel<256,256,2,4"
    else:
        head = "gemm_kernel<256,128,2,2" if mid >= 256 else "gemm_kernel<128,128,2,2"
    return head + suffix


class Step:
    """Buffers and calls of one training step; every call goes to libforge."""

    def __init__(self, cfg, stream):
        import torch
        from paper_2609_13645_amd import _lib, runtime
        self.cfg, self.stream, self.lib = cfg, stream, _lib
        if is_model(cfg):
            inp = fi.model_inputs(cfg)
            self.model = runtime.Model(cfg, inp, stream=stream)
            self.flat = self.model.flat
            self.overlapped = runtime.uses_side_streams(cfg)
        else:
            inp = fi.layer_inputs(cfg)
            self.flat = runtime.FlatParams(runtime.layer_shapes(cfg))
            self.layer = runtime.Layer(cfg, inp["weights"], flat=self.flat, stream=stream)
            self.x = runtime.to_device_bf16(inp["x"])
            self.dy = runtime.to_device_bf16(inp["dy"])
            self.out = torch.empty_like(self.x)
            self.dx = torch.empty_like(self.x)
        self.hp = _lib.AdamwHparams(cfg["beta1"], cfg["beta2"], cfg["adam_eps"],
                                    cfg["weight_decay"])
        # step scalars {lr, 1 - b1^t, 1 - b2^t, clip = 1} advanced on the
        # device each step, so the step needs no host writes (graph replay)
        self.scal = torch.tensor([0.0, 0.0, 0.0, 1.0], dtype=torch.float32, device="cuda")
        self.dstep = torch.zeros(1, dtype=torch.int32, device="cuda")

    def zero(self):
        # gradients are written, not accumulated, by the backward (one
        # micro-batch per step): only the MoE aux scalar starts from zero
        if self.cfg["n_experts"] and not is_model(self.cfg):
            self.layer.aux.zero_()

    def fwd(self):
        if is_model(self.cfg):
            # the head fuses loss fwd and bwd; layers write their gradients,
            # the head / embedding gradients are zeroed first
            self.model.forward_backward(accumulate=False)
        else:
            self.layer.fwd(self.x, self.out)

    def bwd(self):
        if not is_model(self.cfg):
            self.layer.bwd(self.x, self.dy, self.dx, overwrite=True)

    def _scalars(self):
        c = self.cfg
        self.lib.forge_adamw_advance(self.scal, self.dstep, c["lr"], c["beta1"], c["beta2"],
                                     self.stream)

    def adamw(self):
        self._scalars()
        f = self.flat
        self.lib.forge_adamw_step(f.master, f.param, f.grad, f.m, f.v, f.n, self.hp,
                                  self.scal, self.stream)

    def bwd_adamw(self):
        """Layer backward and every weight's update in one call, the updates
        overlapping the rest of the backward."""
        self._scalars()
        self.layer.bwd_adamw(self.x, self.dy, self.dx, self.flat, self.hp, self.scal,
                             overwrite=True)

    def __call__(self):
        self.zero()
        if is_model(self.cfg) and self.overlapped:
            # each layer's update inside its backward, overlapping the
            # backward of the layers below; head and embedding updates last
            self.model.train_step_overlapped()
        elif is_model(self.cfg):
            self.fwd()
            self.adamw()
        else:
            self.fwd()
            self.bwd_adamw()

    def finite(self):
        import torch
        ok = bool(torch.isfinite(self.flat.master).all())
        if is_model(self.cfg):
            return ok and bool(torch.isfinite(self.model.loss).all())
        return ok and bool(torch.isfinite(self.out.float()).all())


def dominant_kernel(cfg, stream, step, reps):
    """The largest single launch of the step, run alone on the step's stream:
    the gate/up projection GEMM of a dense layer, the grouped gate/up GEMM of
    the MoE layer over the routed rows, the LM-head logits GEMM of a model."""
    import torch
    from paper_2609_13645_amd import _lib
    T, h = fi.tokens(cfg), cfg["hidden"]
    if cfg["n_experts"]:
        E, k, fe = cfg["n_experts"], cfg["top_k"], cfg["expert_ffn"]
        # routed row groups from the workload's N(0, 1) router logits
        lg = torch.from_numpy(fi.router_logits(T, E, seed=cfg["seed"])).cuda()
        d = lambda shape, dt: torch.empty(shape, dtype=dt, device="cuda")
        idx, gates, probs = d((T, k), torch.int32), d((T, k), torch.float32), d((T, E), torch.float32)
        counts, offsets, perm = d(E, torch.int32), d(E + 1, torch.int32), d(T * k, torch.int32)
        ws = d(_lib.forge_moe_route_workspace_bytes(T, E, k), torch.uint8)
        _lib.forge_moe_route(lg, T, E, k, idx, gates, probs, counts, offsets, perm, ws, stream)
        rows = T * k
        A = torch.randn((rows, h), device="cuda").to(torch.bfloat16)
        C = torch.empty((rows, 2 * fe), dtype=torch.bfloat16, device="cuda")
        W = step.layer.w["w_gate_up_e"]

        def launch():
            _lib.forge_gemm_grouped_rows(_lib.GEMM_KC, A, W, C, offsets, E, rows, 2 * fe, h,
                                         h, h, 2 * fe, 2 * fe * h, stream)
        flop = 2.0 * rows * 2 * fe * h
        name = "ring_kernel<256,256,4,2,KC,KC,StoreBF16,grouped rows> (expert gate/up fwd)"
        shape = f"rows={rows} E={E} N={2 * fe} K={h}"
    elif is_model(cfg):
        V = cfg["vocab"]
        A = torch.randn((T, h), device="cuda").to(torch.bfloat16)
        C = torch.empty((T, V), dtype=torch.bfloat16, device="cuda")
        W = step.model.w_lm(step.flat.param)

        def launch():
            _lib.forge_gemm(_lib.GEMM_KC, _lib.GEMM_KC, _lib.EPI_STORE_BF16, A, W, C, None,
                            T, V, h, h, h, V, 0, stream)
        flop = 2.0 * T * V * h
        name = f"{kc_kernel_name(T, V, ',KC,KC,StoreBF16>')} (LM-head logits)"
        shape = f"M={T} N={V} K={h}"
    else:
        f = cfg["ffn"]
        A = torch.randn((T, h), device="cuda").to(torch.bfloat16)
        C = torch.empty((T, 2 * f), dtype=torch.bfloat16, device="cuda")
        W = step.layer.w["w_gate_up"]

        def launch():
            _lib.forge_gemm(_lib.GEMM_KC, _lib.GEMM_KC, _lib.EPI_STORE_BF16, A, W, C, None,
                            T, 2 * f, h, h, h, 2 * f, 0, stream)
        flop = 2.0 * T * 2 * f * h
        name = f"{kc_kernel_name(T, 2 * f, ',KC,KC,StoreBF16>')} (gate/up fwd)"
        shape = f"M={T} N={2 * f} K={h}"
    for _ in range(3):
        launch()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        launch()
    e1.record(stream)
    torch.cuda.synchronize()
    return {"name": name, "shape": shape, "avg_us": e0.elapsed_time(e1) / reps * 1e3,
            "flop_per_launch": flop}


def kernel_rooflines(cfg, reps, out=sys.stdout):
    """Every kernel of a dense layer's step run alone on one stream (HIP
    events around `reps` launches after 3 warm-up ones), with its algorithmic
    work per launch and the fraction of its roofline: bf16 MFMA peak for the
    products, HBM bandwidth for the elementwise kernels and AdamW. The
    products are the layer's twelve GEMMs with the layouts and epilogues the
    layer uses; attention backward is the dQ kernel plus the dV and dK passes
    (a kernel trace of this run splits it)."""
    import torch
    from paper_2609_13645_amd import _lib, runtime
    assert not cfg["n_experts"] and not is_model(cfg), "dense layer workloads only"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    T, h, f = fi.tokens(cfg), cfg["hidden"], cfg["ffn"]
    d, nh, nkv = cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"]
    hq, hkv = nh * d, nkv * d
    qkv_w = hq + 2 * hkv
    KC, MC = _lib.GEMM_KC, _lib.GEMM_MC
    bf = lambda *shape: (torch.randn(shape, device="cuda") * 0.5).to(torch.bfloat16)
    f32 = lambda *shape: torch.zeros(shape, dtype=torch.float32, device="cuda")
    rows = []

    def timed(label, kernel, launch, work, unit):
        for _ in range(3):
            launch()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            launch()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        if unit == "TFLOP/s":
            achieved, peak = work / us * 1e-6, PEAK_BF16_TFLOPS
        else:
            achieved, peak = work / us * 1e-3, 8000.0
        rows.append({"step": label, "kernel": kernel, "avg_us": round(us, 1),
                     "work": work, "unit": unit, "achieved": round(achieved, 1),
                     "peak": peak, "frac": round(achieved / peak, 3)})

    # the twelve products: (label, layouts, epilogue, M, N, K)
    x_h, x_hq, x_f, x_2f, x_qkv = bf(T, h), bf(T, hq), bf(T, f), bf(T, 2 * f), bf(T, qkv_w)
    w_qkv, w_o, w_gu, w_d = bf(qkv_w, h), bf(h, hq), bf(2 * f, h), bf(h, f)
    c_bf = torch.empty(T * max(qkv_w, 2 * f, f, h), dtype=torch.bfloat16, device="cuda")
    c_f32 = torch.empty(max(qkv_w, 2 * f, h) * max(h, f, hq), dtype=torch.float32, device="cuda")
    gemms = [
        ("QKV fwd", KC, KC, _lib.EPI_STORE_BF16, x_h, w_qkv, c_bf, None, T, qkv_w, h, h, h, qkv_w),
        ("O fwd + residual", KC, KC, _lib.EPI_RESID_BF16, x_hq, w_o, c_bf, x_h, T, h, hq, hq, hq, h),
        ("gate/up fwd", KC, KC, _lib.EPI_STORE_BF16, x_h, w_gu, c_bf, None, T, 2 * f, h, h, h, 2 * f),
        ("down fwd + residual", KC, KC, _lib.EPI_RESID_BF16, x_f, w_d, c_bf, x_h, T, h, f, f, f, h),
        ("down dgrad", KC, MC, _lib.EPI_STORE_BF16, x_h, w_d, c_bf, None, T, f, h, h, f, f),
        ("gate/up dgrad", KC, MC, _lib.EPI_STORE_BF16, x_2f, w_gu, c_bf, None, T, h, 2 * f, 2 * f, h, h),
        ("O dgrad", KC, MC, _lib.EPI_STORE_BF16, x_h, w_o, c_bf, None, T, hq, h, h, hq, hq),
        ("QKV dgrad", KC, MC, _lib.EPI_STORE_BF16, x_qkv, w_qkv, c_bf, None, T, h, qkv_w, qkv_w, h, h),
        ("down wgrad", MC, MC, _lib.EPI_STORE_F32, x_h, x_f, c_f32, None, h, f, T, h, f, f),
        ("gate/up wgrad", MC, MC, _lib.EPI_STORE_F32, x_2f, x_h, c_f32, None, 2 * f, h, T, 2 * f, h, h),
        ("O wgrad", MC, MC, _lib.EPI_STORE_F32, x_h, x_hq, c_f32, None, h, hq, T, h, hq, hq),
        ("QKV wgrad", MC, MC, _lib.EPI_STORE_F32, x_qkv, x_h, c_f32, None, qkv_w, h, T, qkv_w, h, h),
    ]
    lay = {KC: "KC", MC: "MC"}
    epi = {0: "StoreBF16", 1: "ResidBF16", 2: "AccF32", 3: "StoreF32"}
    for (label, la, lb, ep, A, B, C, R, M, N, K, lda, ldb, ldc) in gemms:
        suffix = f",{lay[la]},{lay[lb]},{epi[ep]}>"
        name = (kc_kernel_name(M, N, suffix) if (la, lb) == (KC, KC)
                else "ring_kernel<256,256,2,4" + suffix)
        timed(f"{label} (M={M} N={N} K={K})", name,
              lambda la=la, lb=lb, ep=ep, A=A, B=B, C=C, R=R, M=M, N=N, K=K, lda=lda, ldb=ldb,
              ldc=ldc: _lib.forge_gemm(la, lb, ep, A, B, C, R, M, N, K, lda, ldb, ldc,
                                       ldc if R is not None else 0, stream),
              2.0 * M * N * K, "TFLOP/s")

    # attention: App. C's count, 4 d FLOP per unmasked (query, key) pair and
    # head forward, twice that backward
    S, B = cfg["seq"], cfg["batch"]
    pairs = B * nh * S * (S + 1) / 2.0
    ac = _lib.attn_cfg(cfg)
    o, lse = bf(T, hq), f32(B * nh * S)
    _lib.forge_attention_fwd(ac, x_qkv, o, lse, stream)
    dqkv = torch.empty_like(x_qkv)
    aws = torch.empty(_lib.forge_attention_bwd_workspace_bytes(ac), dtype=torch.uint8, device="cuda")
    timed("attention fwd", f"attn_fwd_k<{d}>",
          lambda: _lib.forge_attention_fwd(ac, x_qkv, o, lse, stream), 4.0 * d * pairs, "TFLOP/s")
    timed("attention bwd (counted: 2x fwd)",
          f"attn_bwd_prep_k<{d}> + attn_bwd_dv_k<{d}> + attn_bwd_dk_k<{d}> + attn_bwd_dq_k<{d}>",
          lambda: _lib.forge_attention_bwd(ac, x_qkv, o, lse, x_hq, dqkv, aws, stream),
          8.0 * d * pairs, "TFLOP/s")

    # elementwise kernels: algorithmic HBM bytes (each input read once, each
    # output written once)
    g = bf(h)
    y, rstd = torch.empty_like(x_h), f32(T)
    timed(f"RMSNorm fwd (T={T} h={h})", "rmsnorm_fwd_k",
          lambda: _lib.forge_rmsnorm_fwd(x_h, g, y, rstd, T, h, cfg["rms_eps"], stream),
          4.0 * T * h + 4.0 * T + 2.0 * h, "GB/s")
    rws = torch.empty(_lib.forge_rmsnorm_bwd_workspace_bytes(T, h), dtype=torch.uint8, device="cuda")
    dgain, dxn, res = f32(h), torch.empty_like(x_h), bf(T, h)
    timed(f"RMSNorm bwd + residual (T={T} h={h})", "rmsnorm_bwd_k + dg_reduce_k",
          lambda: _lib.forge_rmsnorm_bwd(x_h, g, rstd, y, res, dxn, dgain, False, T, h, rws,
                                         stream),
          8.0 * T * h + 4.0 * T + 6.0 * h, "GB/s")
    cos_t, sin_t = f32(S * d // 2), f32(S * d // 2)
    _lib.forge_rope_table(S, d, cfg["rope_base"], cos_t, sin_t, stream)
    timed(f"RoPE (q and k heads, T={T})", "rope_apply_k",
          lambda: _lib.forge_rope_apply(x_qkv, qkv_w, cos_t, sin_t, None, T, S, nh + nkv, d,
                                        False, stream),
          4.0 * T * (hq + hkv), "GB/s")
    a_out, dgu = torch.empty_like(x_f), torch.empty_like(x_2f)
    timed(f"SwiGLU fwd (T={T} f={f})", "swiglu_fwd_k",
          lambda: _lib.forge_swiglu_fwd(x_2f, a_out, T, f, stream), 6.0 * T * f, "GB/s")
    timed(f"SwiGLU bwd (T={T} f={f})", "swiglu_bwd_k",
          lambda: _lib.forge_swiglu_bwd(x_2f, x_f, dgu, T, f, stream), 10.0 * T * f, "GB/s")
    flat = runtime.FlatParams(runtime.layer_shapes(cfg))
    hp = _lib.AdamwHparams(cfg["beta1"], cfg["beta2"], cfg["adam_eps"], cfg["weight_decay"])
    scal = torch.tensor([1e-4, 0.1, 0.05, 1.0], dtype=torch.float32, device="cuda")
    n_par = sum(int(np.prod(v)) for v in runtime.layer_shapes(cfg).values())
    timed(f"AdamW over the layer ({n_par / 1e6:.1f} M params)", "adamw_k",
          lambda: _lib.forge_adamw_step(flat.master, flat.param, flat.grad, flat.m, flat.v,
                                        flat.n, hp, scal, stream), 30.0 * n_par, "GB/s")

    # a plain 1 GiB device copy three times: calibrates the FETCH_SIZE /
    # WRITE_SIZE counters of a --pmc pass over this run (rooflines_traffic)
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"| step | kernel | avg us | algorithmic work | achieved | peak | frac |", file=out)
    print("|---|---|---|---|---|---|---|", file=out)
    for r in rows:
        w = f"{r['work'] / 1e9:.1f} GFLOP" if r["unit"] == "TFLOP/s" else f"{r['work'] / 1e6:.1f} MB"
        print(f"| {r['step']} | `{r['kernel']}` | {r['avg_us']} | {w} | {r['achieved']} {r['unit']} "
              f"| {r['peak']:.0f} | {r['frac']:.3f} |", file=out)
    print(json.dumps({"workload": cfg["name"], "reps": reps, "kernels": rows}), file=out, flush=True)


COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dominant_kernel_traffic.json")
GEMM_SOURCE = os.path.join(ROOT, "paper_2609_13645_amd", "csrc", "gemm.hip")


def source_digest():
    import hashlib
    with open(GEMM_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_run(cfg, reps):
    """The dominant kernel alone, then a plain device-to-device copy of
    COPY_BYTES, each a few times: the counter passes read both, and the copy
    converts the counters' units into bytes."""
    import torch
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    step = Step(cfg, stream)
    kernel = dominant_kernel(cfg, stream, step, reps)
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"kernel": kernel["name"], "shape": kernel["shape"],
                      "copy_bytes": COPY_BYTES}), flush=True)


def traffic_from_counters(fetch_csv, write_csv, kernel_grid, out=TRAFFIC_FILE):
    """Per-launch HBM bytes of the dominant kernel from the two counter
    passes: each counter's average over the kernel's dispatches, scaled by
    (bytes the copy moves) / (what the counter reads for the copy)."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals = {"kernel": [], "copy": []}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name, grid = r["Kernel_Name"], int(r["Grid_Size"])
            if ("gemm_kernel" in name or "ring_kernel" in name) and grid == kernel_grid:
                vals["kernel"].append(float(r["Counter_Value"]))
            elif "copyBuffer" in name or ("copy" in name.lower() and "gemm" not in name):
                vals["copy"].append(float(r["Counter_Value"]))
        return statistics.median(vals["kernel"]), max(vals["copy"])

    kf, cf = per_kernel(fetch_csv, "FETCH_SIZE")
    kw, cw = per_kernel(write_csv, "WRITE_SIZE")
    res = {"source_sha256": source_digest(), "counters_kib": {"fetch": kf, "write": kw},
           "copy_counters_kib": {"fetch": cf, "write": cw}, "copy_bytes": COPY_BYTES,
           "bytes_per_fetch_kib": COPY_BYTES / cf, "bytes_per_write_kib": COPY_BYTES / cw,
           "fetch_bytes": kf * COPY_BYTES / cf, "write_bytes": kw * COPY_BYTES / cw}
    res["traffic_bytes"] = res["fetch_bytes"] + res["write_bytes"]
    with open(out, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


def rooflines_traffic(fetch_csv, write_csv, out=sys.stdout):
    """HBM bytes per dispatch of every kernel in a --kernel-rooflines run,
    from one FETCH_SIZE and one WRITE_SIZE counter pass: the median over the
    dispatches of each (kernel, grid), converted to bytes by what the same
    counter reads for the run's 1 GiB device copy. Products that share a
    kernel and grid (the dgrad shapes) share a row."""
    import csv
    import statistics
    from collections import defaultdict

    def read(path, counter):
        vals, copy = defaultdict(list), []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name, grid = r["Kernel_Name"], int(r["Grid_Size"])
            if "copyBuffer" in name:
                copy.append(float(r["Counter_Value"]))
            elif not name.startswith("at::") and "rocclr" not in name:
                vals[(name, grid)].append(float(r["Counter_Value"]))
        return vals, max(copy)

    fv, fc = read(fetch_csv, "FETCH_SIZE")
    wv, wc = read(write_csv, "WRITE_SIZE")
    print(f"copy calibration: FETCH_SIZE {fc:.0f} KiB, WRITE_SIZE {wc:.0f} KiB for "
          f"{COPY_BYTES} bytes", file=out)
    print("| kernel | grid (threads) | dispatches | fetch MB | write MB | HBM MB |", file=out)
    print("|---|---|---|---|---|---|", file=out)
    for key in sorted(fv, key=lambda k: -statistics.median(fv[k])):
        fb = statistics.median(fv[key]) * COPY_BYTES / fc / 1e6
        wb = statistics.median(wv.get(key, [0.0])) * COPY_BYTES / wc / 1e6
        name = key[0] if len(key[0]) < 90 else key[0][:87] + "..."
        print(f"| `{name}` | {key[1]} | {len(fv[key])} | {fb:.1f} | {wb:.1f} | {fb + wb:.1f} |",
              file=out)


def recorded_traffic():
    """HBM bytes per launch of the dominant kernel, if the recorded counter
    runs were taken on the current GEMM source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    return rec["traffic_bytes"] if rec.get("source_sha256") == source_digest() else None


def gpu_step_bench(cfg, steps, warmup, kernel_reps, graph=False):
    """Time `steps` training steps after `warmup` eager ones. With `graph`,
    one step is captured into a HIP graph (every libforge call is
    capturable: no allocation, memset or host synchronisation inside; the
    side streams join the capture through events; the AdamW step scalars
    advance on the device) and the timed steps are replays of it."""
    import torch
    torch.cuda.set_device(0)
    stream = torch.cuda.Stream() if graph else torch.cuda.current_stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        step = Step(cfg, stream)
        for _ in range(warmup):
            step()
    torch.cuda.synchronize()
    run = step
    if graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        torch.cuda.synchronize()
        run = g.replay
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        e0.record(stream)
        for _ in range(steps):
            run()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    assert step.finite(), "non-finite output or master weights"
    with torch.cuda.stream(stream):
        phases, kernel = _phases_and_kernel(cfg, stream, step, steps, kernel_reps)
    return ms, phases, kernel, step.flat.n


def _phases_and_kernel(cfg, stream, step, steps, kernel_reps):
    import torch

    # phase split (separate pass, not part of the headline number); a model's
    # forward and backward are one call (the loss head fuses them)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    phases = {"fwd": 0.0, "bwd": 0.0, "adamw": 0.0}
    reps = max(3, min(steps, 10))
    for _ in range(reps):
        step.zero()
        ev[0].record(stream)
        step.fwd()
        ev[1].record(stream)
        step.bwd()
        ev[2].record(stream)
        step.adamw()
        ev[3].record(stream)
        torch.cuda.synchronize()
        phases["fwd"] += ev[0].elapsed_time(ev[1]) / reps
        phases["bwd"] += ev[1].elapsed_time(ev[2]) / reps
        phases["adamw"] += ev[2].elapsed_time(ev[3]) / reps
    if is_model(cfg):
        phases = {"fwd_bwd": phases["fwd"] + phases["bwd"], "adamw": phases["adamw"]}
    else:
        # the step's own order: backward and updates in one overlapped call
        phases["bwd_adamw_overlapped"] = 0.0
        for _ in range(reps):
            step.zero()
            step.fwd()
            ev[1].record(stream)
            step.bwd_adamw()
            ev[2].record(stream)
            torch.cuda.synchronize()
            phases["bwd_adamw_overlapped"] += ev[1].elapsed_time(ev[2]) / reps
    return phases, dominant_kernel(cfg, stream, step, kernel_reps)


def cpu_baseline(cfg, seq, reps=3):
    """The fp64 oracle (as it stands) on a bounded sample of the workload,
    timed `reps` times (the median is reported)."""
    from oracle import dense, moe, head, adamw as oadam
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = _CORES
    f64 = fi.bf16_bits_to_f64
    if is_model(cfg):
        # one layer of the model at one sequence of the batch (plus the full head)
        c = dict(cfg, n_layers=1, batch=1)
        inp = fi.model_inputs(c)
        P = {"embedding": f64(inp["embedding"]), "final_norm": f64(inp["final_norm"]),
             "w_lm": None if inp["w_lm"] is None else f64(inp["w_lm"]),
             "layers": [{k: f64(v) for k, v in W.items()} for W in inp["layers"]]}
        n_params = sum(v.size for v in P["layers"][0].values()) + P["embedding"].size

        def fwd_bwd():
            _, grads = head.model_fwd_bwd(P, inp["ids"], inp["targets"], c)
            flat_p = [P["embedding"]] + list(P["layers"][0].values())
            flat_g = [grads["embedding"]] + [grads["layers"][0][k] for k in P["layers"][0]]
            return flat_p, flat_g
        sample = (f"fp64 oracle: 1 of {cfg['n_layers']} layers, 1 of {cfg['batch']} "
                  f"sequences ({c['seq']} tokens), full LM head and CE, AdamW over that "
                  f"layer and the embedding")
    else:
        seq = min(seq, cfg["seq"])
        c = dict(cfg, seq=seq, batch=1)
        if cfg.get("positions") is not None:
            c["positions"] = cfg["positions"][:seq]
        inp = fi.layer_inputs(c)
        W = {k: f64(v) for k, v in inp["weights"].items()}
        x, dy = f64(inp["x"]), f64(inp["dy"])
        n_params = sum(w.size for w in W.values())

        def fwd_bwd():
            if cfg["n_experts"]:
                _, _, cache = moe.layer_fwd(x, W, c)
                _, grads = moe.layer_bwd(cache, W, c, dy)
            else:
                _, cache = dense.layer_fwd(x, W, c)
                _, grads = dense.layer_bwd(cache, W, c, dy)
            return list(W.values()), [grads[k] for k in W]
        sample = (f"fp64 oracle: fwd+bwd of the same layer shapes over {seq} tokens "
                  f"(one sequence; the workload has {cfg['batch']} x {cfg['seq']})")
    # the optimizer over the same fraction of the parameters as the sample's
    # share of the step's tokens
    frac = fi.tokens(c) / fi.tokens(cfg)

    def once():
        t0 = time.perf_counter()
        flat_p, flat_g = fwd_bwd()
        budget = int(round(frac * n_params))
        n_opt = 0
        for p, g in zip(flat_p, flat_g):
            if budget <= 0:
                break
            k = min(budget, g.size)
            pp, gg = p.reshape(-1)[:k], g.reshape(-1)[:k]
            oadam.adamw_step(pp, gg, np.zeros_like(pp), np.zeros_like(pp), cfg["lr"],
                             cfg["beta1"], cfg["beta2"], cfg["adam_eps"], cfg["weight_decay"], 1)
            budget -= k
            n_opt += k
        return time.perf_counter() - t0, n_opt

    runs = [once() for _ in range(max(1, reps))]
    times = sorted(t for t, _ in runs)
    dt, n_opt = times[len(times) // 2], runs[0][1]
    model_flop = flops.step_flops(c)
    return {"value": model_flop / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"{sample}; AdamW over {n_opt / 1e6:.1f}M params; median of "
                       f"{len(times)} runs ({', '.join(f'{t:.2f}' for t in times)} s) for "
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


def step_timeline(db_path, which=2, out=sys.stdout):
    """One layer step of a traced bench run in time order: start and duration
    (us) from the step's first kernel, the gap to the latest end so far
    (negative: overlapping earlier work on another stream), the stream and
    the workgroup count. A step starts with the attention RMSNorm, the QKV
    product (one or two launches) and RoPE; `which` picks the traced step by
    its index (default 2: the second timed step after one warm-up step)."""
    import re
    import sqlite3
    con = sqlite3.connect(db_path)
    rows = []
    for name, gx, start, end, stream, wx in con.execute(
            "select name, grid_x, start, end, stream_id, workgroup_x from kernels order by start"):
        short = re.sub(r"\(.*", "", name.replace("void ", "").replace(
            "forge::(anonymous namespace)::", ""))
        rows.append((short, gx // max(1, wx), start, end, stream))
    gemm, rope = ("gemm_kernel", "ring_kernel"), ("rope_apply", "qknorm_rope")
    # the QKV product is one launch, or two when its last round runs as halves
    starts = [i for i in range(len(rows) - 3) if rows[i][0].startswith("rmsnorm_fwd")
              and rows[i + 1][0].startswith(gemm)
              and (rows[i + 2][0].startswith(rope)
                   or (rows[i + 2][0].startswith(gemm) and rows[i + 3][0].startswith(rope)))]
    i0 = starts[which]
    nxt = [j for j in starts if j > i0]
    i1 = (nxt[0] if nxt else len(rows)) - 1
    while i1 > i0 and (rows[i1][0].startswith("at::") or "rocclr" in rows[i1][0]):
        i1 -= 1   # torch's checks and copies after the step
    t0 = prev_end = end = rows[i0][2]
    print("| start us | duration us | gap us | stream | kernel | workgroups |", file=out)
    print("|---|---|---|---|---|---|", file=out)
    for name, grid, st, en, stream in rows[i0:i1 + 1]:
        print(f"| {(st - t0) / 1e3:.1f} | {(en - st) / 1e3:.1f} | {(st - prev_end) / 1e3:.1f} | "
              f"s{stream} | `{name[:60]}` | {grid} |", file=out)
        prev_end = max(prev_end, en)
        end = max(end, en)
    print(f"\nstep span {(end - t0) / 1e3:.1f} us", file=out)


def summarize_counters(csv_paths, out=sys.stdout):
    """Mean per dispatch of every counter, per kernel (libforge's GEMM and
    attention kernels), from rocprofv3 --pmc counter_collection CSV files."""
    import collections
    import csv
    import re
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for path in csv_paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                m = re.search(r"((?:ring_kernel|gemm_kernel|attn_\w+)<[^()]*>|attn_\w+)",
                              r["Kernel_Name"])
                if m:
                    agg[m.group(1)][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for cs in agg.values() for c in cs})
    print("| kernel | " + " | ".join(names) + " |", file=out)
    print("|---" * (len(names) + 1) + "|", file=out)
    for k in sorted(agg):
        vals = [agg[k].get(c) for c in names]
        cells = [f"{sum(v) / len(v):.4g}" if v else "" for v in vals]
        print(f"| `{k}` | " + " | ".join(cells) + " |", file=out)


def main():
    if len(sys.argv) >= 3 and sys.argv[1] == "--counters-summarize":
        summarize_counters(sys.argv[2:])
        return
    if len(sys.argv) in (3, 4) and sys.argv[1] == "--timeline":
        step_timeline(sys.argv[2], *(int(a) for a in sys.argv[3:]))
        return
    if len(sys.argv) == 3 and sys.argv[1] == "--summarize":
        summarize_profile(sys.argv[2])
        return
    if len(sys.argv) == 4 and sys.argv[1] == "--rooflines-traffic":
        rooflines_traffic(sys.argv[2], sys.argv[3])
        return
    if len(sys.argv) == 5 and sys.argv[1] == "--traffic-summarize":
        traffic_from_counters(sys.argv[2], sys.argv[3], int(sys.argv[4]))
        return
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library runs the training step on one "
              "MI355X and has no multi-GPU path (--gpus must be 1).", file=sys.stderr)
        sys.exit(2)
    cfg = fi.config(args.workload)
    if args.traffic_run:
        traffic_run(cfg, args.kernel_reps)
        return
    if args.kernel_rooflines:
        kernel_rooflines(cfg, args.kernel_reps)
        return
    T = fi.tokens(cfg)
    step_flop = flops.step_flops(cfg)
    print(f"[bench] workload {args.workload}: {DESCRIPTION[args.workload]}; "
          f"warmup={args.warmup} steps={args.steps}", file=sys.stderr, flush=True)
    ms, phases, kernel, nparams = gpu_step_bench(cfg, args.steps, args.warmup, args.kernel_reps,
                                                 args.graph)
    tflops = step_flop / (ms * 1e-3) / 1e12
    print(f"[bench] {ms:.3f} ms/step, {tflops:.1f} TFLOP/s; phases {phases}",
          file=sys.stderr, flush=True)
    fb_ms = sum(v for k, v in phases.items() if k in ("fwd", "bwd", "fwd_bwd"))
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
        "mfu_fwd_bwd_pct": round(100.0 * step_flop / (fb_ms * 1e-3) / 1e12 / MFU_PEAK_TFLOPS, 2),
        "tokens_per_s": round(T / (ms * 1e-3), 1),
        "phases_ms": {k: round(v, 4) for k, v in phases.items()},
        "launch": "graph replay of one captured step" if args.graph else "eager",
        "config": {"workload": args.workload, "description": DESCRIPTION[args.workload],
                   "batch": cfg["batch"], "seq": cfg["seq"], "hidden": cfg["hidden"],
                   "n_heads": cfg["n_heads"], "n_kv_heads": cfg["n_kv_heads"],
                   "head_dim": cfg["head_dim"], "ffn": cfg["ffn"], "params": nparams,
                   "model_flop_per_step": step_flop},
        "roofline": {"bound": "mfma", "kernel": kernel["name"], "shape": kernel["shape"],
                     "achieved": round(k_tf, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(k_tf / PEAK_BF16_TFLOPS, 4),
                     "avg_us": round(kernel["avg_us"], 2),
                     "traffic": (recorded_traffic() if args.workload == WORKLOAD else None)},
    }
    if cfg["n_experts"]:
        res["config"].update(n_experts=cfg["n_experts"], top_k=cfg["top_k"],
                             expert_ffn=cfg["expert_ffn"], aux_coef=cfg["aux_coef"])
    for key in ("qk_norm", "shared_ffn", "branch_scale", "packed_docs", "dense_first_layers",
                "embed_scale", "logit_scale"):
        if cfg.get(key):
            res["config"][key] = cfg[key]
    if is_model(cfg):
        res["config"].update(n_layers=cfg["n_layers"], vocab=cfg["vocab"], tied=cfg["tied"])
    if cfg["recompute_attn"]:
        hw = step_flop + flops.recompute_flops(cfg)
        res["hfu_pct"] = round(100.0 * hw / (ms * 1e-3) / 1e12 / MFU_PEAK_TFLOPS, 2)
        res["config"]["recompute_attn"] = 1
    if not args.no_cpu_baseline:
        print(f"[bench] cpu baseline: oracle sample ...", file=sys.stderr, flush=True)
        cb = cpu_baseline(cfg, args.cpu_seq)
        res["cpu_baseline"] = {k: (round(v, 6) if isinstance(v, float) else v)
                               for k, v in cb.items() if k != "seconds"}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

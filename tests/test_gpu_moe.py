"""GPU parity of the MoE path: routing (bit-exact integers), layer fwd/bwd.

Routing is checked on identical fp32 logits given to both sides, so the
integer outputs (top-k indices, counts, offsets, permutation) must match
bit for bit, ties included. The layer is checked against the fp64 oracle's
MoE layer (the oracle takes its top-k decision on logits rounded to fp32).

Inside the layer the two sides do not see identical logits: the GPU routes
on its bf16 activations, whose logits differ from the oracle's by about
2.5e-3 of the logit RMS (rounding of b to bf16 plus the bf16 error of h1).
A token whose k-th and (k+1)-th logits lie closer than that can go either
way, and both answers are correct. Such tokens (oracle margin below
TIE_BAND times the logit RMS, about 8 standard deviations of the difference
of two perturbed logits) are "ambiguous": their output rows are not
compared and their dy rows are zero, so no expert weight gradient depends
on their routing. The aux loss still counts them; its tolerance adds the
most that swapping their experts can move it.
"""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import moe as omoe
from gpu_util import rel_fro, dev_bf16, host_f64, banner

pytestmark = pytest.mark.gpu


def gpu_route(l32, k):
    import torch
    from paper_2609_13645_amd import _lib
    T, E = l32.shape
    d = lambda shape, dt: torch.empty(shape, dtype=dt, device="cuda")
    idx, gates, probs = d((T, k), torch.int32), d((T, k), torch.float32), d((T, E), torch.float32)
    counts, offsets, perm = d(E, torch.int32), d(E + 1, torch.int32), d(T * k, torch.int32)
    ws = d(_lib.forge_moe_route_workspace_bytes(T, E, k), torch.uint8)
    _lib.forge_moe_route(torch.from_numpy(l32).cuda(), T, E, k, idx, gates, probs, counts,
                         offsets, perm, ws)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (idx, gates, probs, counts, offsets, perm)]


@pytest.mark.parametrize("T,E,k,ties", [(8192, 64, 8, True), (37, 8, 3, True), (1000, 16, 16, False),
                                        (5, 64, 1, False)])
def test_route_bit_exact(T, E, k, ties):
    banner(f"moe route T={T} E={E} k={k}")
    l32 = fi.router_logits(T, E, seed=5 + T)
    if ties:   # exact ties inside and at the top-k boundary
        l32[:, 3] = l32[:, 7 % E]
        l32[::3, 1] = l32[::3, 0]
        l32[5] = 0.25
    got = gpu_route(l32, k)
    idx, gates, p, counts, offsets, perm = omoe.route(l32, k)
    assert np.array_equal(got[0], idx)
    assert np.array_equal(got[3], counts)
    assert np.array_equal(got[4], offsets)
    assert np.array_equal(got[5], perm)
    assert rel_fro(got[1], gates) <= 1e-6
    assert rel_fro(got[2], p) <= 1e-6


def _moe_weights_f64(w):
    return {k: fi.bf16_bits_to_f64(v) for k, v in w.items()}


TIE_BAND = 3e-2


def ambiguous(l, k):
    """Tokens whose oracle top-k margin is within the bf16 perturbation band."""
    return omoe.topk_margin(l, k) < TIE_BAND * np.sqrt(np.mean(np.square(l)))


def run_moe_layer(cfg, seed=None):
    import torch
    from paper_2609_13645_amd import runtime
    inp = fi.layer_inputs(cfg, seed)
    W = _moe_weights_f64(inp["weights"])
    ref_out, aux, cache = omoe.layer_fwd(fi.bf16_bits_to_f64(inp["x"]), W, cfg)
    amb = ambiguous(cache["moe"]["l"], cfg["top_k"])
    dy_bits = inp["dy"].copy()
    dy_bits[amb] = 0
    ref_dx, ref_g = omoe.layer_bwd(cache, W, cfg, fi.bf16_bits_to_f64(dy_bits))
    layer = runtime.Layer(cfg, inp["weights"])
    x, dy = dev_bf16(inp["x"]), dev_bf16(dy_bits)
    out, dx = torch.empty_like(x), torch.empty_like(x)
    layer.fwd(x, out)
    layer.bwd(x, dy, dx)
    torch.cuda.synchronize()
    got = {"out": host_f64(out)[~amb], "dx": host_f64(dx), "aux": float(layer.aux.item())}
    for n in layer.names:
        got[n] = host_f64(layer.g["d_" + n])
    ref = {"out": ref_out[~amb], "dx": ref_dx, "aux": aux}
    ref.update(ref_g)
    # swapping one slot from expert a to b moves the aux loss by
    # alpha E (P_b - P_a) / (T k); an ambiguous token swaps at most k slots
    P = cache["moe"]["p"].mean(0)
    T = len(amb)
    ref["aux_slack"] = cfg["aux_coef"] * cfg["n_experts"] * amb.sum() * (P.max() - P.min()) / T
    banner(f"  {amb.sum()} of {T} tokens within the tie band")
    return got, ref, layer


def check_moe(got, ref):
    errs = {k: rel_fro(got[k], ref[k]) for k in ref if k not in ("aux", "aux_slack")}
    banner(f"  aux {got['aux']:.6e} vs {ref['aux']:.6e} (slack {ref['aux_slack']:.1e}); errors "
           f"{({k: f'{v:.1e}' for k, v in errs.items()})}")
    assert abs(got["aux"] - ref["aux"]) <= 1e-4 * abs(ref["aux"]) + ref["aux_slack"] + 1e-9
    assert errs["out"] <= 2e-2 and errs["dx"] <= 2e-2
    for k, e in errs.items():
        assert e <= 3e-2, k
    for k, v in got.items():
        assert np.all(np.isfinite(v)), k


def test_moe_layer_mini():
    cfg = fi.config("tiny", batch=2, seq=96, ffn=0, n_experts=16, top_k=4, expert_ffn=128,
                    aux_coef=0.05, seed=41)
    banner("moe layer mini (E 16, k 4, fe 128)")
    got, ref, _ = run_moe_layer(cfg)
    check_moe(got, ref)


def test_moe_layer_large_aux_unambiguous_routing():
    """A large aux coefficient makes the router gradient depend on every
    expert count, so a single ambiguous token would move it: these seeded
    inputs have every token's margin above the tie band (asserted), so the
    routing, the counts and the aux gradient are unique."""
    cfg = fi.config("tiny", batch=1, seq=64, ffn=0, n_experts=8, top_k=2, expert_ffn=64,
                    aux_coef=0.5, seed=489)
    banner("moe layer, aux 0.5, unambiguous routing")
    got, ref, _ = run_moe_layer(cfg)
    assert ref["aux_slack"] == 0.0
    check_moe(got, ref)


def test_moe_layer_full_geometry_short_seq():
    # the MoE workload's widths (h 2048, 16/4 heads of 128, 64 experts top-8,
    # fe 1408) at 320 tokens: ragged expert groups of ~40 rows
    cfg = fi.config("moe_layer", batch=1, seq=320)
    banner("moe layer full geometry, seq 320")
    got, ref, _ = run_moe_layer(cfg, seed=51)
    check_moe(got, ref)


def test_moe_layer_long_sequence_split_router_gradient():
    # 2048 tokens: the router weight gradient (16 x 256 outputs) is reduced
    # over the tokens in four slices whose partial sums are added in order
    cfg = fi.config("tiny", batch=1, seq=2048, ffn=0, n_experts=16, top_k=2, expert_ffn=64,
                    aux_coef=0.05, seed=61)
    banner("moe layer seq 2048 (router gradient split over tokens)")
    got, ref, _ = run_moe_layer(cfg)
    check_moe(got, ref)


def test_moe_layer_is_deterministic():
    cfg = fi.config("tiny", seq=128, ffn=0, n_experts=8, top_k=2, expert_ffn=64, aux_coef=0.01)
    banner("moe determinism")
    a, _, _ = run_moe_layer(cfg, seed=3)
    b, _, _ = run_moe_layer(cfg, seed=3)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_moe_layer_full_size_sampled_rows_and_causality():
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("moe_layer", aux_coef=0.0)   # aux couples all tokens: off here
    T = fi.tokens(cfg)
    t0 = 6000
    banner("moe layer full size (B2 S4096): sampled rows + backward causality")
    inp = fi.layer_inputs(cfg)
    dyb = inp["dy"].copy()
    dyb[t0:] = 0
    layer = runtime.Layer(cfg, inp["weights"])
    x, dy = dev_bf16(inp["x"]), dev_bf16(dyb)
    out, dx = torch.empty_like(x), torch.empty_like(x)
    layer.fwd(x, out)
    layer.bwd(x, dy, dx)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 2, 3, 127, 128, 511, 1000, 2047, 2048, 3001, 4095,
                     4096, 4097, 4098, 5000, 5999, 6000, 6001, 7000, 7777, 8000, 8190, T - 1])
    W = _moe_weights_f64(inp["weights"])
    ref, l = omoe.layer_fwd_rows(fi.bf16_bits_to_f64(inp["x"]), W, cfg, rows, with_logits=True)
    keep = ~ambiguous(l, cfg["top_k"])
    got = host_f64(out)[rows]
    e = rel_fro(got[keep], ref[keep])
    banner(f"  sampled-row forward error {e:.2e} over {keep.sum()} unambiguous rows of {len(rows)}")
    assert keep.sum() >= len(rows) // 2
    assert e <= 2e-2
    g = host_f64(dx)
    # batch row 0 is tokens 0..4095 and row 1 is 4096..8191: with dy zero from
    # t0 = 6000 on, dx is exactly zero there
    assert np.all(g[t0:] == 0.0)
    assert np.count_nonzero(g[:t0]) > 0.99 * g[:t0].size

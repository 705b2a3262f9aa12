"""GPU checks at the full workload sizes, in the launch configuration the bench times.

* 8B-shape layer (seq 4096): full parity of the layer forward and backward
  against the fp64 oracle (the oracle finishes in seconds on the host).
* 8B-shape layer at seq 16384 with attention recompute: the oracle evaluates
  sampled output rows one by one (all keys, selected queries); the backward is
  checked through a property that holds at any size: with the upstream
  gradient zero from token t0 on, the input gradient is exactly zero there
  (every token only feeds later tokens) and nonzero before.
"""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import dense
from gpu_util import rel_fro, dev_bf16, host_f64, banner

pytestmark = pytest.mark.gpu

NAMES = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


def _run(cfg, dy_bits=None):
    import torch
    from paper_2609_13645_amd import runtime
    inp = fi.layer_inputs(cfg)
    layer = runtime.Layer(cfg, inp["weights"])
    x = dev_bf16(inp["x"])
    dy = dev_bf16(inp["dy"] if dy_bits is None else dy_bits)
    out, dx = torch.empty_like(x), torch.empty_like(x)
    layer.fwd(x, out)
    layer.bwd(x, dy, dx)
    torch.cuda.synchronize()
    return inp, layer, out, dx


def test_llama8b_layer_full_size_parity():
    cfg = fi.config("llama8b_layer")
    banner("full-size 8B-shape layer (T 4096) fwd+bwd vs fp64 oracle")
    inp, layer, out, dx = _run(cfg)
    W = {k: fi.bf16_bits_to_f64(v) for k, v in inp["weights"].items()}
    ref_out, cache = dense.layer_fwd(fi.bf16_bits_to_f64(inp["x"]), W, cfg)
    ref_dx, ref_g = dense.layer_bwd(cache, W, cfg, fi.bf16_bits_to_f64(inp["dy"]))
    errs = {"out": rel_fro(host_f64(out), ref_out), "dx": rel_fro(host_f64(dx), ref_dx)}
    for n in NAMES:
        errs[n] = rel_fro(host_f64(layer.g["d_" + n]), ref_g[n])
    banner(f"  errors {({k: f'{v:.2e}' for k, v in errs.items()})}")
    assert errs["out"] <= 2e-2 and errs["dx"] <= 2e-2
    for n in NAMES:
        assert errs[n] <= 3e-2, n


def test_llama8b_16k_layer_sampled_rows_and_backward_causality():
    cfg = fi.config("llama8b_layer_16k")
    S = cfg["seq"]
    t0 = 12000
    inp = fi.layer_inputs(cfg)
    dyb = inp["dy"].copy()
    dyb[t0:] = 0
    banner("full-size 16K layer with attention recompute: sampled rows + causality")
    inp, layer, out, dx = _run(cfg, dyb)
    rows = np.array([0, 1, 127, 128, 4095, 8191, 11999, 12000, 16000, S - 1])
    W = {k: fi.bf16_bits_to_f64(v) for k, v in inp["weights"].items()}
    ref = dense.layer_fwd_rows(fi.bf16_bits_to_f64(inp["x"]), W, cfg, rows)
    got = host_f64(out)[rows]
    e = rel_fro(got, ref)
    banner(f"  sampled-row forward error {e:.2e}")
    assert e <= 2e-2
    for r in range(len(rows)):
        assert rel_fro(got[r], ref[r]) <= 3e-2, rows[r]
    g = host_f64(dx)
    assert np.all(g[t0:] == 0.0)
    assert np.count_nonzero(g[:t0]) > 0.99 * g[:t0].size
    assert np.all(np.isfinite(g))

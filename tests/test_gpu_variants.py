"""GPU parity of the model variants (App. B, App. A step 23) against the
fp64 oracle: per-head QK-Norm, document-aware RoPE positions, the muP
residual-branch scale, the shared expert of the 160-expert top-16 sparse
model, and a whole muP model (embedding and logit scales) whose first layer
is dense and the others routed. Tolerances as everywhere: 2e-2 for
activations and input gradients, 3e-2 for weight gradients.
"""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import dense, head as ohead
from gpu_util import rel_fro, dev_bf16, host_f64, banner
from test_gpu_moe import run_moe_layer, check_moe

pytestmark = pytest.mark.gpu


def _perturb_gains(inp, rng):
    for n in ("q_norm", "k_norm"):
        if n in inp["weights"]:
            d = inp["weights"][n].size
            inp["weights"][n] = fi.to_bf16_bits(
                (1.0 + 0.2 * rng.standard_normal(d)).astype(np.float32))


def run_dense(cfg, seed):
    import torch
    from paper_2609_13645_amd import runtime
    inp = fi.layer_inputs(cfg, seed)
    _perturb_gains(inp, np.random.default_rng(seed))
    layer = runtime.Layer(cfg, inp["weights"])
    x, dy = dev_bf16(inp["x"]), dev_bf16(inp["dy"])
    out, dx = torch.empty_like(x), torch.empty_like(x)
    layer.fwd(x, out)
    layer.bwd(x, dy, dx)
    torch.cuda.synchronize()
    W = {k: fi.bf16_bits_to_f64(v) for k, v in inp["weights"].items()}
    ref_out, cache = dense.layer_fwd(fi.bf16_bits_to_f64(inp["x"]), W, cfg)
    ref_dx, ref_g = dense.layer_bwd(cache, W, cfg, fi.bf16_bits_to_f64(inp["dy"]))
    errs = {"out": rel_fro(host_f64(out), ref_out), "dx": rel_fro(host_f64(dx), ref_dx)}
    for n in layer.names:
        errs[n] = rel_fro(host_f64(layer.g["d_" + n]), ref_g[n])
    banner(f"  errors {({k: f'{v:.1e}' for k, v in errs.items()})}")
    assert errs["out"] <= 2e-2 and errs["dx"] <= 2e-2
    for n in layer.names:
        assert errs[n] <= 3e-2, n
    return errs


@pytest.mark.parametrize("name,over", [
    ("tiny", dict(qk_norm=1, seq=160)),
    ("tiny", dict(qk_norm=1, head_dim=128, n_heads=2, n_kv_heads=1, batch=2, seq=77)),
    ("tiny", dict(packed_docs=20, batch=2, seq=96)),
    ("tiny", dict(branch_scale=1.4 / 24 ** 0.5, qk_norm=1, packed_docs=30, seq=128)),
    ("qwen3_layer", dict(batch=1, seq=320)),
    ("packed_docs_layer", dict(seq=320, packed_docs=60)),
])
def test_dense_variant_layer_vs_oracle(name, over):
    cfg = fi.config(name, **over)
    banner(f"variant layer {name} {over}")
    assert cfg.get("positions") is None or len(cfg["positions"]) == fi.tokens(cfg)
    run_dense(cfg, seed=17 + cfg["seq"])


def test_positions_are_taken_by_the_gpu():
    """Positions that differ from the row index change the result (a path
    that ignored them would not); positions equal to the row index give the
    default bit for bit."""
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("tiny", seq=96)
    inp = fi.layer_inputs(cfg, 5)
    outs = []
    for pos in (None, np.arange(96, dtype=np.int32), fi.doc_positions(1, 96, 16, 3)):
        c = dict(cfg, positions=pos)
        layer = runtime.Layer(c, inp["weights"])
        x = dev_bf16(inp["x"])
        out = torch.empty_like(x)
        layer.fwd(x, out)
        torch.cuda.synchronize()
        outs.append(host_f64(out))
    assert np.array_equal(outs[0], outs[1])
    assert not np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("name,over", [
    ("tiny", dict(batch=1, seq=256, ffn=0, n_experts=32, top_k=4, expert_ffn=64,
                  shared_ffn=96, aux_coef=0.05, branch_scale=0.6)),
    ("minicpm5_moe_layer", dict(batch=1, seq=256)),
])
def test_moe_shared_expert_layer_vs_oracle(name, over):
    cfg = fi.config(name, **over)
    banner(f"moe layer with shared expert {name} {over}")
    got, ref, _ = run_moe_layer(cfg, seed=29)
    check_moe(got, ref)


def test_mup_model_with_dense_first_layer_vs_oracle():
    """Embedding scale, logit scale, branch scale; layer 0 dense, layer 1
    routed with a shared expert; tied head."""
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("tiny", n_layers=2, tied=True, batch=1, seq=192, vocab=512, ffn=344,
                    n_experts=16, top_k=4, expert_ffn=64, shared_ffn=64, aux_coef=0.01,
                    dense_first_layers=1, embed_scale=12.0, logit_scale=256.0 / 1024.0,
                    branch_scale=1.4 / 2 ** 0.5, seed=39)
    banner("muP model: dense first layer, MoE + shared expert, tied head")
    inp = fi.model_inputs(cfg)
    model = runtime.Model(cfg, inp)
    model.flat.grad.zero_()
    loss = float(model.forward_backward().item())
    aux = float(model.aux.item())
    torch.cuda.synchronize()
    f64 = fi.bf16_bits_to_f64
    P = {"embedding": f64(inp["embedding"]), "final_norm": f64(inp["final_norm"]), "w_lm": None,
         "layers": [{k: f64(v) for k, v in W.items()} for W in inp["layers"]]}
    # the routed layer's choice near ties may differ: the oracle runs with the
    # GPU's routing once the oracle's own logits show it is a valid top-k
    from test_gpu_moe import saved_routing, check_routing
    from oracle import moe as omoe
    gidx = saved_routing(model.layers[1])
    loss_ref, g = ohead.model_fwd_bwd(P, inp["ids"], inp["targets"], cfg, route_idx={1: gidx})
    x = ohead.embed_fwd(inp["ids"], P["embedding"], cfg["embed_scale"])
    x, _ = dense.layer_fwd(x, P["layers"][0], ohead.layer_cfg(cfg, 0))
    _, _, c1 = omoe.layer_fwd(x, P["layers"][1], cfg, idx=gidx)
    check_routing(gidx, c1["moe"]["l"], cfg["top_k"])
    banner(f"  loss+aux {loss + aux:.6f} vs oracle {loss_ref:.6f}")
    assert abs((loss + aux) - loss_ref) / loss_ref <= 2e-3
    errs = {"embedding": rel_fro(host_f64(model.flat.view(model.flat.grad, "embedding")),
                                 g["embedding"]),
            "final_norm": rel_fro(host_f64(model.flat.view(model.flat.grad, "final_norm")),
                                  g["final_norm"])}
    for i, gl in enumerate(g["layers"]):
        for n, v in gl.items():
            errs[f"{i}.{n}"] = rel_fro(host_f64(model.flat.view(model.flat.grad, f"{i}.{n}")), v)
    banner(f"  grad errors {({k: f'{v:.1e}' for k, v in errs.items()})}")
    for k, e in errs.items():
        assert e <= 3e-2, k

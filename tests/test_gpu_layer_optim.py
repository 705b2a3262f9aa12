"""forge_layer_bwd_adamw against its definition: forge_layer_bwd followed by
forge_adamw_step. Both run the same kernels per element, so every parameter,
master weight, moment, gradient and the input gradient must agree bit for
bit, over consecutive steps (the second step's forward reads the updated
weights). The weight matrices are updated in the epilogues of their gradient products
(the standalone update's arithmetic per element); layers from 2^20 token x
hidden elements run those products on the library's side stream and the
small updates on its optimizer stream while the backward continues; smaller
layers run everything in order.
"""
import pytest

import forge_inputs as fi
from gpu_util import dev_bf16, banner

pytestmark = pytest.mark.gpu

CASES = {
    "dense_tiny": lambda: fi.config("tiny", batch=2, seq=72, seed=17),
    "dense_8b_geometry": lambda: fi.config("llama8b_layer", seq=512, seed=23),
    "moe": lambda: fi.config("tiny", batch=1, seq=1024, ffn=0, n_experts=16, top_k=2,
                             expert_ffn=64, aux_coef=0.05, seed=61),
    # 512 x 2048 token x hidden elements: the expert updates overlap the
    # attention backward on the library's streams
    "moe_overlapped": lambda: fi.config("moe_layer", batch=1, seq=512, n_experts=16, top_k=2,
                                        expert_ffn=256, seed=67),
    # model variants: QK-Norm with document positions and a branch scale (side
    # streams on), and the shared expert of the 160-expert top-16 layer
    "qk_norm_packed": lambda: fi.config("qwen3_layer", batch=1, seq=1024, packed_docs=100,
                                        branch_scale=0.5, seed=71),
    "moe_shared_expert": lambda: fi.config("minicpm5_moe_layer", batch=1, seq=512, seed=73),
    # the benchmarked workloads at full size, in the bench's launch configuration
    "llama8b_layer_full": lambda: fi.config("llama8b_layer"),
    "moe_layer_full": lambda: fi.config("moe_layer"),
}
FULL = ("llama8b_layer_full", "moe_layer_full")


def run(cfg, inp, fused, steps=2, overwrite=True):
    import torch
    from paper_2609_13645_amd import _lib, runtime
    flat = runtime.FlatParams(runtime.layer_shapes(cfg))
    layer = runtime.Layer(cfg, inp["weights"], flat=flat)
    # nonzero moments inside every weight (the alignment gaps stay zero),
    # drawn on the device from a seeded generator (same values for both runs)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    for n in layer.names:
        mv = flat.view(flat.m, n)
        mv.copy_(torch.randn(mv.shape, generator=gen, device="cuda") * 1e-3)
        vv = flat.view(flat.v, n)
        vv.copy_(torch.rand(vv.shape, generator=gen, device="cuda") * 1e-6)
    hp = _lib.AdamwHparams(0.9, 0.95, 1e-8, 0.1)
    scal = torch.tensor([3e-3, 0.19, 0.0975, 0.7], dtype=torch.float32, device="cuda")
    x, dy = dev_bf16(inp["x"]), dev_bf16(inp["dy"])
    out, dx = torch.empty_like(x), torch.empty_like(x)
    for _ in range(steps):
        if cfg.get("n_experts", 0):
            layer.aux.zero_()
        layer.fwd(x, out)
        if fused:
            layer.bwd_adamw(x, dy, dx, flat, hp, scal, overwrite=overwrite)
        else:
            layer.bwd(x, dy, dx, overwrite=overwrite)
            _lib.forge_adamw_step(flat.master, flat.param, flat.grad, flat.m, flat.v, flat.n,
                                  hp, scal)
    torch.cuda.synchronize()
    res = {"out": out.clone(), "dx": dx.clone()}
    for n in layer.names:
        for buf in ("param", "master", "m", "v", "grad"):
            res[f"{buf}:{n}"] = flat.view(getattr(flat, buf), n).clone()
    return res


@pytest.mark.parametrize("case,overwrite", [(c, o) for c in CASES for o in (True, False)
                                            if o or c not in FULL])
def test_layer_bwd_adamw_equals_bwd_then_adamw(case, overwrite):
    """overwrite=False: the gradients accumulate over the two steps (and the
    fused epilogues update from the accumulated gradient)."""
    import torch
    cfg = CASES[case]()
    banner(f"layer bwd+adamw fused vs sequential ({case}, overwrite={overwrite})")
    inp = fi.layer_inputs(cfg)
    want = run(cfg, inp, fused=False, overwrite=overwrite)
    got = run(cfg, inp, fused=True, overwrite=overwrite)
    for k, v in want.items():
        assert torch.equal(got[k], v), k
    # the updates moved the weights
    one = run(cfg, inp, fused=True, steps=1)
    assert not torch.equal(got["master:w_qkv"], one["master:w_qkv"])

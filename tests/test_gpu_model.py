"""GPU parity of the whole-model training step (embedding, layers, head, AdamW).

The oracle runs the same step in fp64 from the same seeded inputs. Loss and
every gradient are compared directly (2e-2 / 3e-2). The optimizer update is
compared twice: on the GPU's own gradients (identical optimizer inputs, the
1e-5 bar), and from the oracle's gradients where they stand well clear of the
GPU gradient's noise: AdamW's first step is lr * g / (|g| + eps), so an entry
whose gradient is within noise of zero can legitimately flip sign.
The bf16 parameters must equal the round-to-nearest-even of the GPU master.
"""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import head as ohead, adamw as oadam
from gpu_util import rel_fro, host_f64, banner

pytestmark = pytest.mark.gpu

LAYER_NAMES = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


def run_model(cfg):
    import torch
    from paper_2609_13645_amd import runtime
    inp = fi.model_inputs(cfg)
    model = runtime.Model(cfg, inp)
    model.flat.grad.zero_()
    loss = model.forward_backward()
    torch.cuda.synchronize()
    got = {"loss": float(loss.item()),
           "grads": {k: host_f64(model.flat.view(model.flat.grad, k)) for k in model.flat.offsets},
           "master0": {k: host_f64(model.flat.view(model.flat.master, k)) for k in model.flat.offsets}}
    model.optimizer_step()
    torch.cuda.synchronize()
    got["master1"] = {k: host_f64(model.flat.view(model.flat.master, k)) for k in model.flat.offsets}
    got["param1_bits"] = runtime.to_host_bits(model.flat.param)
    got["master1_flat"] = model.flat.master.detach().cpu().numpy()
    f64 = fi.bf16_bits_to_f64
    P = {"embedding": f64(inp["embedding"]), "final_norm": f64(inp["final_norm"]),
         "w_lm": None if inp["w_lm"] is None else f64(inp["w_lm"]),
         "layers": [{k: f64(v) for k, v in W.items()} for W in inp["layers"]]}
    loss_ref, g = ohead.model_fwd_bwd(P, inp["ids"], inp["targets"], cfg)
    ref = {"embedding": g["embedding"], "final_norm": g["final_norm"]}
    if g["w_lm"] is not None:
        ref["w_lm"] = g["w_lm"]
    for i, gl in enumerate(g["layers"]):
        for n in LAYER_NAMES:
            ref[f"{i}.{n}"] = gl[n]
    return got, loss_ref, ref


def check_model(cfg):
    got, loss_ref, ref = run_model(cfg)
    banner(f"  loss {got['loss']:.6f} vs oracle {loss_ref:.6f}")
    assert abs(got["loss"] - loss_ref) / loss_ref <= 2e-3
    errs = {k: rel_fro(got["grads"][k], ref[k]) for k in ref}
    banner(f"  grad errors {({k: f'{v:.1e}' for k, v in errs.items()})}")
    for k, e in errs.items():
        assert e <= 3e-2, k
    f32 = lambda x: float(np.float32(x))    # the hyperparameters as the GPU holds them
    for k, g in ref.items():
        p0 = got["master0"][k]
        # the optimizer isolated: AdamW step 1 on the GPU's own gradients
        p1, _, _ = oadam.adamw_step(p0, got["grads"][k], 0 * g, 0 * g, f32(cfg["lr"]),
                                    f32(cfg["beta1"]), f32(cfg["beta2"]), f32(cfg["adam_eps"]),
                                    f32(cfg["weight_decay"]), 1)
        # (compared with the oracle's result rounded to the fp32 master's
        # precision: for a norm gain near 1 one fp32 step is 1e-4 of the update)
        assert rel_fro(got["master1"][k] - p0, p1.astype(np.float32) - p0) <= 1e-5, k
        # the whole step: AdamW step 1 from the oracle's gradients, on the
        # entries whose gradient stands well clear of the GPU's gradient noise
        # (the first update is about lr * sign(g): within the noise of zero
        # either sign is correct)
        p1, _, _ = oadam.adamw_step(p0, g, 0 * g, 0 * g, cfg["lr"], cfg["beta1"], cfg["beta2"],
                                    cfg["adam_eps"], cfg["weight_decay"], 1)
        # (the noise is taken per row: an embedding row of a frequent token
        # carries both large gradients and large rounding errors)
        err2 = np.square(got["grads"][k] - g)
        noise = np.sqrt(np.mean(err2, axis=-1, keepdims=True)) if g.ndim == 2 else np.sqrt(np.mean(err2))
        conf = np.abs(g) > np.maximum(0.1 * np.sqrt(np.mean(g * g)), 6.0 * noise)
        d_got, d_ref = (got["master1"][k] - p0)[conf], (p1 - p0)[conf]
        assert rel_fro(d_got, d_ref) <= 2e-2, k
        assert np.all(np.abs(got["master1"][k] - p0) <= cfg["lr"] * (1 + cfg["weight_decay"] * np.abs(p0)) * 1.001)
    assert np.array_equal(got["param1_bits"], fi.to_bf16_bits(got["master1_flat"]))


def test_tiny_model_step_untied():
    cfg = fi.config("tiny")
    banner("model step tiny (1 layer, untied head, V 1024)")
    check_model(cfg)


def test_two_layer_tied_model_step():
    cfg = fi.config("tiny", n_layers=2, tied=True, batch=2, seq=96, vocab=512, seed=31)
    banner("model step 2 layers, tied head, batch 2")
    check_model(cfg)


def test_model_step_is_deterministic_except_embedding_scatter():
    """Two runs give bit-identical loss and gradients; only the embedding
    gradient, summed by fp32 atomics over repeated token ids, may differ in
    its last bits."""
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("tiny", n_layers=2, seq=64)
    banner("model determinism (two runs)")
    inp = fi.model_inputs(cfg)
    res = []
    for _ in range(2):
        model = runtime.Model(cfg, inp)
        model.flat.grad.zero_()
        loss = float(model.forward_backward().item())
        torch.cuda.synchronize()
        res.append((loss, {k: host_f64(model.flat.view(model.flat.grad, k))
                           for k in model.flat.offsets}))
    assert res[0][0] == res[1][0]
    for k in res[0][1]:
        if k == "embedding":
            assert rel_fro(res[0][1][k], res[1][1][k]) <= 1e-6
        else:
            assert np.array_equal(res[0][1][k], res[1][1][k]), k


def test_model_step_without_accumulation_matches_zeroed_accumulation():
    """forward_backward(accumulate=False) gives this step's gradients whatever
    the gradient buffer held: layers overwrite, head / embedding are zeroed."""
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("tiny", n_layers=2, tied=True, seq=64, vocab=512, seed=33)
    banner("model step without accumulation")
    inp = fi.model_inputs(cfg)
    model = runtime.Model(cfg, inp)
    model.flat.grad.zero_()
    l1 = float(model.forward_backward().item())
    torch.cuda.synchronize()
    ref = model.flat.grad.clone()
    model.flat.grad.fill_(float("nan"))
    l2 = float(model.forward_backward(accumulate=False).item())
    torch.cuda.synchronize()
    assert l1 == l2
    pad = torch.isnan(model.flat.grad) & (ref == 0)   # alignment gaps are never written
    got = torch.where(pad, torch.zeros_like(ref), model.flat.grad)
    assert torch.equal(got[:model.head_grad_elems] != 0, ref[:model.head_grad_elems] != 0)
    assert rel_fro(got[:model.head_grad_elems].cpu().numpy(),
                   ref[:model.head_grad_elems].cpu().numpy()) <= 1e-6
    assert torch.equal(got[model.head_grad_elems:], ref[model.head_grad_elems:])


def test_dense1b_widths_two_layer_model_step():
    # the 16-layer model's widths (h 2048, 32/8 heads of 64, f 8192, V 32000,
    # tied head) with 2 layers at 512 tokens; T x h = 2^20, so the layer
    # backward runs its weight gradients on the side stream as in the model
    cfg = fi.config("dense1b", n_layers=2, batch=1, seq=512, seed=35)
    banner("model step at the 1B model's widths, 2 layers, 512 tokens, tied head")
    check_model(cfg)

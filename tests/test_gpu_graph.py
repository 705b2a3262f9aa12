"""Whole training steps captured into a HIP graph and replayed.

Every libforge call is capturable (no allocation, memset, copy or host
synchronisation inside; the layer backward's side streams join the capture
through events); the AdamW step scalars advance on the device. A captured
step is replayed several times, with unrelated eager work and host
synchronisations between replays, and after every replay its state is
compared with the same number of eager steps from the same start.
"""
import numpy as np
import pytest

import forge_inputs as fi
from gpu_util import dev_bf16, banner

pytestmark = pytest.mark.gpu


def test_adamw_advance_matches_host_bias_corrections():
    import torch
    from paper_2609_13645_amd import _lib
    banner("adamw_advance: device step scalars")
    b1, b2, lr = 0.9, 0.95, 3e-4
    sc = torch.tensor([0.0, 0.0, 0.0, 0.625], dtype=torch.float32, device="cuda")
    step = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = []
    for _ in range(300):
        _lib.forge_adamw_advance(sc, step, lr, b1, b2)
        got.append(sc.clone())
    step.fill_(9999)
    _lib.forge_adamw_advance(sc, step, lr, b1, b2)
    got.append(sc.clone())
    torch.cuda.synchronize()
    ts = list(range(1, 301)) + [10000]
    assert int(step.item()) == 10000
    for t, g in zip(ts, got):
        want = np.array([lr, 1.0 - np.float64(b1) ** t, 1.0 - np.float64(b2) ** t, 0.625],
                        dtype=np.float32)
        assert np.array_equal(g.cpu().numpy(), want), t


class LayerStep:
    """fwd + backward with overlapped AdamW, scalars advanced on the device."""

    def __init__(self, cfg, inp, stream):
        import torch
        from paper_2609_13645_amd import _lib, runtime
        self.cfg, self.stream, self.lib = cfg, stream, _lib
        self.flat = runtime.FlatParams(runtime.layer_shapes(cfg))
        self.layer = runtime.Layer(cfg, inp["weights"], flat=self.flat, stream=stream)
        self.x, self.dy = dev_bf16(inp["x"]), dev_bf16(inp["dy"])
        self.out, self.dx = torch.empty_like(self.x), torch.empty_like(self.x)
        self.hp = _lib.AdamwHparams(0.9, 0.95, 1e-8, 0.1)
        self.scal = torch.tensor([0.0, 0.0, 0.0, 1.0], dtype=torch.float32, device="cuda")
        self.dstep = torch.zeros(1, dtype=torch.int32, device="cuda")

    def __call__(self):
        self.layer.fwd(self.x, self.out)
        self.lib.forge_adamw_advance(self.scal, self.dstep, 1e-3, 0.9, 0.95, self.stream)
        self.layer.bwd_adamw(self.x, self.dy, self.dx, self.flat, self.hp, self.scal)

    def state(self):
        f = self.flat
        return {"out": self.out, "dx": self.dx, "param": f.param, "master": f.master,
                "m": f.m, "v": f.v, "grad": f.grad, "step": self.dstep}


def _eager_noise():
    import torch
    a = torch.randn(512, 512, device="cuda")
    (a @ a).sum().item()


def test_layer_step_graph_replays_match_eager():
    """8B-geometry layer at seq 256 (2^20 token x hidden elements: the side
    streams are used), bit for bit over three replays."""
    import torch
    cfg = fi.config("llama8b_layer", seq=256, seed=29)
    banner("graph replay of a layer step (side streams)")
    inp = fi.layer_inputs(cfg)
    s_eager = torch.cuda.Stream()
    s_graph = torch.cuda.Stream()
    with torch.cuda.stream(s_eager):
        eager = LayerStep(cfg, inp, s_eager)
    with torch.cuda.stream(s_graph):
        graphed = LayerStep(cfg, inp, s_graph)
        graphed()                      # eager first step: creates the side streams
    with torch.cuda.stream(s_eager):
        eager()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s_graph):
        graphed()
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(s_graph):
            g.replay()
        with torch.cuda.stream(s_eager):
            eager()
        torch.cuda.synchronize()
        _eager_noise()
        a, b = eager.state(), graphed.state()
        for k in a:
            assert torch.equal(a[k], b[k]), (rep, k)


@pytest.mark.parametrize("max_norm", [None, 1e-3])
def test_model_step_graph_replays_match_eager(max_norm):
    """Tiny model (embedding, layer, LM head + CE, flat AdamW), with the clip
    coefficient fixed at 1 or from the gradient norm on the device; its
    embedding backward uses fp32 atomics, so the comparison has a
    tolerance."""
    import torch
    from paper_2609_13645_amd import runtime
    cfg = fi.config("tiny")
    banner(f"graph replay of a model step (max_norm {max_norm})")
    inp = fi.model_inputs(cfg)
    s_eager, s_graph = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s_eager):
        eager = runtime.Model(cfg, inp, stream=s_eager)
    with torch.cuda.stream(s_graph):
        graphed = runtime.Model(cfg, inp, stream=s_graph)
        graphed.train_step(max_norm)
    with torch.cuda.stream(s_eager):
        eager.train_step(max_norm)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s_graph):
        graphed.train_step(max_norm)
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(s_graph):
            g.replay()
        with torch.cuda.stream(s_eager):
            eager.train_step(max_norm)
        torch.cuda.synchronize()
        _eager_noise()
        if max_norm is not None:
            # the coefficient both paths used: min(1, max_norm / (||g|| + eps))
            for m in (eager, graphed):
                norm = float(torch.linalg.vector_norm(m.flat.grad.double()))
                want = min(1.0, max_norm / (norm + 1e-6))
                assert want < 1.0
                assert abs(float(m.scalars[3]) - want) <= 1e-5 * want, rep
        assert int(eager.dev_step.item()) == int(graphed.dev_step.item()) == rep + 2
        assert torch.allclose(graphed.loss, eager.loss, rtol=1e-5, atol=0), rep
        for buf in ("master", "m", "v"):
            a, b = getattr(eager.flat, buf), getattr(graphed.flat, buf)
            assert torch.allclose(b, a, rtol=1e-4, atol=1e-7), (rep, buf)

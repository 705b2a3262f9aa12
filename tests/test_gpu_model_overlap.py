"""Model step with each layer's AdamW update inside its backward
(Model.train_step_overlapped) against the plain step (train_step: the
backward of every layer, then one AdamW over all parameters).

The layer gradients do not depend on the embedding gradient (the only one
summed with atomics), so after one step every layer's parameter, master
weight and moments agree bit for bit; the embedding state agrees to fp32
rounding. The second step starts from those embeddings and is compared with
a tolerance.
"""
import pytest

import forge_inputs as fi
from gpu_util import banner

pytestmark = pytest.mark.gpu

CASES = {
    # layers below 2^20 token x hidden elements: everything in order
    "tiny_untied": lambda: fi.config("tiny", n_layers=2, seed=41),
    # 512 x 2048: side streams and the optimizer stream, tied head
    "two_layers_tied": lambda: fi.config("dense1b", batch=1, seq=512, vocab=1024, n_layers=2,
                                         seed=43),
}


def _layer_names(flat):
    return [n for n in flat.offsets if "." in n]


@pytest.mark.parametrize("case", list(CASES))
def test_overlapped_model_step_equals_plain_step(case):
    import torch
    from paper_2609_13645_amd import runtime
    cfg = CASES[case]()
    banner(f"model step: per-layer overlapped updates vs one AdamW ({case})")
    inp = fi.model_inputs(cfg)
    plain = runtime.Model(cfg, inp)
    over = runtime.Model(cfg, inp)
    plain.train_step()
    over.train_step_overlapped()
    torch.cuda.synchronize()
    assert torch.equal(plain.loss, over.loss)
    for n in _layer_names(plain.flat):
        for buf in ("param", "master", "m", "v", "grad"):
            a = plain.flat.view(getattr(plain.flat, buf), n)
            b = over.flat.view(getattr(over.flat, buf), n)
            assert torch.equal(a, b), (n, buf)
    for buf in ("master", "m", "v"):
        a = plain.flat.view(getattr(plain.flat, buf), "embedding")
        b = over.flat.view(getattr(over.flat, buf), "embedding")
        assert torch.allclose(b, a, rtol=1e-5, atol=1e-9), buf
    plain.train_step()
    over.train_step_overlapped()
    torch.cuda.synchronize()
    assert int(plain.dev_step.item()) == int(over.dev_step.item()) == 2
    assert torch.allclose(over.loss, plain.loss, rtol=1e-4, atol=0)
    for buf in ("master", "m", "v"):
        a, b = getattr(plain.flat, buf), getattr(over.flat, buf)
        assert torch.allclose(b, a, rtol=1e-3, atol=1e-6), buf
    # the update moved the weights
    assert not torch.equal(over.flat.master, runtime.Model(cfg, inp).flat.master)

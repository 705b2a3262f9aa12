"""GPU parity of the fused clip + AdamW + bf16 write-back, gradient norm and clip.

The optimizer is isolated: both sides get the same fp32 master / grad / m / v
from the seeded generator, so the fp32 AdamW master-weight update can be held
to 1e-5 relative Frobenius error on the update itself (p_new - p_old, taken in
fp64). The bf16 parameter must be the round-to-nearest-even of the GPU's own
new master, bit for bit.
"""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import adamw as oadam
from gpu_util import rel_fro, banner

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, wd=0.1)


def _adamw_gpu(st, step, clip=1.0, lr=HP["lr"]):
    import torch
    from paper_2609_13645_amd import _lib
    n = st["master"].size
    dev = {k: torch.from_numpy(v.copy()).cuda() for k, v in st.items()}
    param = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    bc1, bc2 = oadam.bias_corrections(HP["beta1"], HP["beta2"], step)
    sc = torch.tensor([lr, bc1, bc2, clip], dtype=torch.float32, device="cuda")
    hp = _lib.AdamwHparams(HP["beta1"], HP["beta2"], HP["eps"], HP["wd"])
    _lib.forge_adamw_step(dev["master"], param, dev["grad"], dev["m"], dev["v"], n, hp, sc)
    torch.cuda.synchronize()
    out = {k: dev[k].cpu().numpy() for k in ("master", "m", "v")}
    out["param"] = param.view(torch.int16).cpu().numpy().view(np.uint16)
    return out


@pytest.mark.parametrize("n,step,clip", [(1_000_003, 1, 1.0), (65_536, 5, 0.37), (3, 2, 1.0),
                                         (1, 1, 1.0)])
def test_adamw_matches_oracle(n, step, clip):
    banner(f"adamw n={n} step={step} clip={clip}")
    st = fi.optimizer_inputs(n, seed=n % 1000 + step, step=step)
    got = _adamw_gpu(st, step, clip)
    f32 = lambda x: float(np.float32(x))    # the hyperparameters as the GPU holds them
    p, m, v = oadam.adamw_step(st["master"], st["grad"], st["m"], st["v"], f32(HP["lr"]),
                               f32(HP["beta1"]), f32(HP["beta2"]), f32(HP["eps"]),
                               f32(HP["wd"]), step, f32(clip))
    p0 = st["master"].astype(np.float64)
    assert rel_fro(got["master"].astype(np.float64) - p0, p - p0) <= 1e-5
    assert rel_fro(got["m"], m) <= 1e-5
    assert rel_fro(got["v"], v) <= 1e-5
    assert np.array_equal(got["param"], fi.to_bf16_bits(got["master"]))


def test_adamw_is_deterministic_and_resumable():
    """N + M steps in one go on the device equal N steps, a save of master,
    m and v to the host, a restore into fresh device buffers and M more
    steps, bit for bit; the step scalars advance on the device
    (forge_adamw_advance) and each step has its own gradient."""
    import torch
    from paper_2609_13645_amd import _lib
    banner("adamw determinism / save-restore resume over 3 + 2 steps")
    n, N, M = 100_003, 3, 2
    st = fi.optimizer_inputs(n, seed=9, step=1)
    rng = np.random.default_rng(10)
    grads = [(rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)) for _ in range(N + M)]
    hp = _lib.AdamwHparams(HP["beta1"], HP["beta2"], HP["eps"], HP["wd"])

    def fresh(state, step0):
        dev = {k: torch.from_numpy(np.ascontiguousarray(state[k]).copy()).cuda()
               for k in ("master", "m", "v")}
        dev["param"] = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        dev["sc"] = torch.tensor([0.0, 0.0, 0.0, 1.0], dtype=torch.float32, device="cuda")
        dev["step"] = torch.tensor([step0], dtype=torch.int32, device="cuda")
        return dev

    def steps(dev, gs):
        for g in gs:
            gd = torch.from_numpy(g).cuda()
            _lib.forge_adamw_advance(dev["sc"], dev["step"], HP["lr"], HP["beta1"], HP["beta2"])
            _lib.forge_adamw_step(dev["master"], dev["param"], gd, dev["m"], dev["v"], n, hp,
                                  dev["sc"])
        torch.cuda.synchronize()
        out = {k: dev[k].cpu().numpy() for k in ("master", "m", "v")}
        out["param"] = dev["param"].view(torch.int16).cpu().numpy().view(np.uint16)
        out["step"] = int(dev["step"].item())
        return out

    whole = steps(fresh(st, 0), grads)
    again = steps(fresh(st, 0), grads)
    for k in whole:
        assert np.array_equal(whole[k], again[k]), k
    first = steps(fresh(st, 0), grads[:N])
    saved = {k: first[k].copy() for k in ("master", "m", "v")}     # host checkpoint
    resumed = steps(fresh(saved, first["step"]), grads[N:])
    assert resumed["step"] == whole["step"] == N + M
    for k in ("master", "m", "v", "param"):
        assert np.array_equal(resumed[k], whole[k]), k
    # and the whole run matches the oracle's N + M steps from the same state
    p, m, v = (st[k].astype(np.float64) for k in ("master", "m", "v"))
    f32 = lambda x: float(np.float32(x))
    for t, g in enumerate(grads, start=1):
        p, m, v = oadam.adamw_step(p, g, m, v, f32(HP["lr"]), f32(HP["beta1"]),
                                   f32(HP["beta2"]), f32(HP["eps"]), f32(HP["wd"]), t)
    p0 = st["master"].astype(np.float64)
    assert rel_fro(whole["master"].astype(np.float64) - p0, p - p0) <= 1e-5


def test_grad_norm_and_clip_coeff():
    import torch
    from paper_2609_13645_amd import _lib
    banner("grad norm + clip")
    rng = np.random.default_rng(4)
    g1 = rng.standard_normal(3_000_001).astype(np.float32) * 1e-2
    g2 = rng.standard_normal(17).astype(np.float32)
    acc = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = torch.empty(_lib.GRAD_NORM_WORKSPACE_FLOATS, dtype=torch.float32, device="cuda")
    for g in (g1, g2):
        _lib.forge_grad_norm_sq(torch.from_numpy(g).cuda(), g.size, acc, ws)
    sc = torch.tensor([1e-3, 1.0, 1.0, -1.0], dtype=torch.float32, device="cuda")
    _lib.forge_clip_coeff(acc, 1.0, 1e-6, sc)
    torch.cuda.synchronize()
    ref = oadam.grad_norm_sq([g1, g2])
    got = float(acc.item())
    assert abs(got - ref) / ref <= 1e-5
    assert abs(float(sc[3].item()) - oadam.clip_coeff(ref, 1.0, 1e-6)) <= 1e-6
    # repeat: fixed summation order gives identical bits
    acc2 = torch.zeros(1, dtype=torch.float32, device="cuda")
    for g in (g1, g2):
        _lib.forge_grad_norm_sq(torch.from_numpy(g).cuda(), g.size, acc2, ws)
    torch.cuda.synchronize()
    assert acc2.item() == got

"""GPU parity of the output head (final norm + LM head + CE) and the embedding."""
import numpy as np
import pytest

import forge_inputs as fi
from oracle import head as ohead
from gpu_util import rel_fro, dev_bf16, host_f64, banner

pytestmark = pytest.mark.gpu


def run_head(T, h, V, seed, chunk=0):
    import torch
    from paper_2609_13645_amd import _lib
    rng = np.random.default_rng(seed)
    xb = fi.to_bf16_bits(rng.standard_normal((T, h), dtype=np.float32))
    gb = fi.to_bf16_bits(1.0 + 0.1 * rng.standard_normal(h, dtype=np.float32))
    wb = fi.to_bf16_bits(0.02 * rng.standard_normal((V, h), dtype=np.float32))
    tg = rng.integers(0, V, size=T, dtype=np.int32)
    cfg = _lib.HeadCfg(T, h, V, 1e-5)
    nws = (_lib.forge_loss_chunked_workspace_bytes(cfg, chunk) if chunk
           else _lib.forge_loss_workspace_bytes(cfg))
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    loss = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda")
    dx = torch.empty((T, h), dtype=torch.bfloat16, device="cuda")
    dg = torch.full((h,), 0.25, dtype=torch.float32, device="cuda")
    dw = torch.full((V, h), -0.125, dtype=torch.float32, device="cuda")
    args = (dev_bf16(xb), dev_bf16(gb), dev_bf16(wb), torch.from_numpy(tg).cuda(), loss, dx,
            dg, dw, ws)
    if chunk:
        _lib.forge_loss_fwd_bwd_chunked(cfg, chunk, *args)
    else:
        _lib.forge_loss_fwd_bwd(cfg, *args)
    torch.cuda.synchronize()
    r_loss, r_dx, r_dg, r_dw = ohead.head_fwd_bwd(
        fi.bf16_bits_to_f64(xb), fi.bf16_bits_to_f64(gb), fi.bf16_bits_to_f64(wb), tg, 1e-5)
    return dict(loss=(loss.item(), r_loss), dx=(host_f64(dx), r_dx),
                dg=(host_f64(dg) - 0.25, r_dg), dw=(host_f64(dw) + 0.125, r_dw))


@pytest.mark.parametrize("T,h,V", [(128, 256, 1024), (200, 64, 1032), (64, 2048, 32000)])
def test_head_parity(T, h, V):
    banner(f"head T={T} h={h} V={V}")
    r = run_head(T, h, V, seed=T + V)
    gl, rl = r["loss"]
    assert abs(gl - rl) / abs(rl) <= 2e-3
    errs = {k: rel_fro(*r[k]) for k in ("dx", "dg", "dw")}
    banner(f"  loss {gl:.6f} vs {rl:.6f}; errors {errs}")
    assert errs["dx"] <= 2e-2
    assert errs["dg"] <= 3e-2 and errs["dw"] <= 3e-2


@pytest.mark.parametrize("T,h,V,chunk", [(200, 64, 1032, 48), (128, 256, 1024, 1),
                                         (64, 2048, 32000, 24), (96, 128, 1024, 4096)])
def test_streaming_head_parity(T, h, V, chunk):
    """Chunked head (a ragged last chunk, one-row chunks, a chunk above T)
    against the oracle, and against the unchunked head: the same loss and
    input gradient up to the logits GEMM's tile choice, d_w_lm summed in
    chunk order."""
    banner(f"streaming head T={T} h={h} V={V} chunk={chunk}")
    r = run_head(T, h, V, seed=T + V, chunk=chunk)
    p = run_head(T, h, V, seed=T + V)
    gl, rl = r["loss"]
    assert abs(gl - rl) / abs(rl) <= 2e-3
    errs = {k: rel_fro(*r[k]) for k in ("dx", "dg", "dw")}
    banner(f"  loss {gl:.6f} vs {rl:.6f}; errors {errs}")
    assert errs["dx"] <= 2e-2
    assert errs["dg"] <= 3e-2 and errs["dw"] <= 3e-2
    assert abs(gl - p["loss"][0]) <= 1e-5 * abs(gl)
    for k in ("dx", "dg", "dw"):
        assert rel_fro(r[k][0], p[k][0]) <= 1e-2, k


def test_uniform_logits_loss_is_log_vocab_on_gpu():
    # zero LM head: every logit is 0, the loss is exactly ln V up to fp32 rounding
    import torch
    from paper_2609_13645_amd import _lib
    banner("head uniform logits")
    T, h, V = 64, 128, 1024
    cfg = _lib.HeadCfg(T, h, V, 1e-5)
    ws = torch.empty(_lib.forge_loss_workspace_bytes(cfg), dtype=torch.uint8, device="cuda")
    x = torch.randn((T, h), device="cuda").to(torch.bfloat16)
    g = torch.ones(h, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((V, h), dtype=torch.bfloat16, device="cuda")
    tg = torch.randint(0, V, (T,), dtype=torch.int32, device="cuda")
    loss = torch.empty(1, dtype=torch.float32, device="cuda")
    dx = torch.empty((T, h), dtype=torch.bfloat16, device="cuda")
    dg = torch.zeros(h, dtype=torch.float32, device="cuda")
    dw = torch.zeros((V, h), dtype=torch.float32, device="cuda")
    _lib.forge_loss_fwd_bwd(cfg, x, g, w, tg, loss, dx, dg, dw, ws)
    torch.cuda.synchronize()
    assert abs(loss.item() - 6.931471805599453) < 1e-5
    assert torch.all(dx.float() == 0)


def test_embedding_fwd_bwd():
    import torch
    from paper_2609_13645_amd import _lib
    banner("embedding fwd/bwd")
    rng = np.random.default_rng(2)
    T, h, V = 1000, 256, 64           # many repeated ids
    eb = fi.to_bf16_bits(rng.standard_normal((V, h), dtype=np.float32))
    ids = rng.integers(0, V, size=T, dtype=np.int32)
    ids[5] = -1
    ids[7] = V                         # out of range: zero row / skipped
    x = torch.empty((T, h), dtype=torch.bfloat16, device="cuda")
    ids_d = torch.from_numpy(ids).cuda()
    _lib.forge_embed_fwd(ids_d, dev_bf16(eb), x, T, h, V)
    dxb = fi.to_bf16_bits(rng.standard_normal((T, h), dtype=np.float32))
    dE = torch.zeros((V, h), dtype=torch.float32, device="cuda")
    _lib.forge_embed_bwd(ids_d, dev_bf16(dxb), dE, T, h, V)
    torch.cuda.synchronize()
    E = fi.bf16_bits_to_f64(eb)
    got = host_f64(x)
    valid = (ids >= 0) & (ids < V)
    assert np.array_equal(got[valid], ohead.embed_fwd(ids[valid], E))
    assert np.all(got[~valid] == 0)
    ref = ohead.embed_bwd(ids[valid], fi.bf16_bits_to_f64(dxb)[valid], V)
    assert rel_fro(host_f64(dE), ref) <= 1e-6

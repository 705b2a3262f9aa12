"""forge_moe_route_noalloc (routing with the library's fixed scratch, no
workspace argument) against forge_moe_route on the same logits: two calls in
a row, the second smaller, every output bit for bit (requests beyond the
fixed scratch are refused on the host: test_abi)."""
import numpy as np
import pytest

import forge_inputs as fi
from gpu_util import banner

pytestmark = pytest.mark.gpu


def _route(fn_name, l32, k, with_ws):
    import torch
    from paper_2609_13645_amd import _lib
    T, E = l32.shape
    d = lambda shape, dt: torch.full(shape, -7, dtype=dt, device="cuda")
    out = [d((T, k), torch.int32), d((T, k), torch.float32), d((T, E), torch.float32),
           d((E,), torch.int32), d((E + 1,), torch.int32), d((T * k,), torch.int32)]
    logits = torch.from_numpy(l32).cuda()
    if with_ws:
        ws = torch.empty(_lib.forge_moe_route_workspace_bytes(T, E, k), dtype=torch.uint8,
                         device="cuda")
        _lib.forge_moe_route(logits, T, E, k, *out, ws)
    else:
        _lib.forge_moe_route_noalloc(logits, T, E, k, *out)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out]


@pytest.mark.parametrize("T,E,k", [(32768, 160, 16), (1000, 64, 8)])
def test_noalloc_route_equals_route(T, E, k):
    from paper_2609_13645_amd import _lib
    assert T * k <= _lib.MOE_ROUTE_NOALLOC_MAX_ENTRIES
    banner(f"moe route without workspace T={T} E={E} k={k}")
    l32 = fi.router_logits(T, E, seed=900 + T)
    l32[:, 2] = l32[:, 5]          # exact ties
    l32[7] = 0.5
    ref = _route("forge_moe_route", l32, k, True)
    got = _route("forge_moe_route_noalloc", l32, k, False)
    for name, a, b in zip(("idx", "gates", "probs", "counts", "offsets", "perm"), got, ref):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), name

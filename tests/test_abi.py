"""CPU checks of the C ABI: the library loads, exports every declared symbol,
answers size queries, and rejects bad arguments before touching the device."""
import ctypes

import pytest

import forge_inputs as fi
from paper_2609_13645_amd import _lib


def test_library_exports_every_header_function():
    L = _lib.load()
    names = _lib.header_functions()
    assert len(names) >= 15
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    for n in ("forge_layer_fwd", "forge_layer_bwd", "forge_loss_fwd_bwd", "forge_adamw_step"):
        assert n in names


def test_status_strings_and_version():
    assert _lib.status_name(0) == "FORGE_OK"
    assert _lib.status_name(3) == "FORGE_ERR_ALIGNMENT"
    assert _lib.status_name(99) == "FORGE_ERR_UNKNOWN"
    assert "gfx950" in _lib.forge_version()


def test_size_queries_are_consistent():
    c2 = _lib.layer_cfg(fi.config("llama8b_layer"))
    T, h, f = 4096, 4096, 14336
    saved = _lib.forge_layer_saved_bytes(c2)
    # a, qkv, o, h1, b, gu, act (bf16) + rstd x2, lse (fp32), 256-byte aligned pieces
    lower = 2 * T * (h + 6144 + 4096 + h + h + 2 * f + f) + 4 * (2 * T + 32 * T)
    assert lower <= saved <= lower + 256 * 12
    rec = _lib.layer_cfg(fi.config("llama8b_layer_16k"))
    rec_nokeep = _lib.layer_cfg(dict(fi.config("llama8b_layer_16k"), recompute_attn=0))
    assert _lib.forge_layer_saved_bytes(rec) < _lib.forge_layer_saved_bytes(rec_nokeep)
    assert _lib.forge_layer_workspace_bytes(rec) > _lib.forge_layer_workspace_bytes(rec_nokeep)
    hc = _lib.HeadCfg(8192, 2048, 32000, 1e-5)
    assert _lib.forge_loss_workspace_bytes(hc) >= 8192 * 32000 * 2
    # the streaming head holds chunk x V logits; chunk >= T is the plain head
    plain = _lib.forge_loss_workspace_bytes(hc)
    assert _lib.forge_loss_chunked_workspace_bytes(hc, 2048) <= plain - 6144 * 32000 * 2
    assert _lib.forge_loss_chunked_workspace_bytes(hc, 8192) == plain
    assert _lib.forge_loss_chunked_workspace_bytes(hc, 1 << 30) == plain
    with pytest.raises(_lib.ForgeError):
        _lib.forge_loss_chunked_workspace_bytes(hc, 0)


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), _lib.FORGE_ERR_UNSUPPORTED),
    (dict(n_heads=6, n_kv_heads=4), _lib.FORGE_ERR_INVALID_ARG),
    (dict(hidden=260), _lib.FORGE_ERR_INVALID_ARG),
    (dict(ffn=690), _lib.FORGE_ERR_INVALID_ARG),
    (dict(seq=0), _lib.FORGE_ERR_INVALID_ARG),
    (dict(n_experts=264, top_k=8, expert_ffn=1408), _lib.FORGE_ERR_UNSUPPORTED),
    (dict(n_experts=100, top_k=8, expert_ffn=1408), _lib.FORGE_ERR_UNSUPPORTED),
    (dict(n_experts=64, top_k=0, expert_ffn=1408), _lib.FORGE_ERR_INVALID_ARG),
    (dict(n_experts=64, top_k=8, expert_ffn=1404), _lib.FORGE_ERR_INVALID_ARG),
])
def test_bad_configs_rejected(change, status):
    c = _lib.layer_cfg(dict(fi.config("tiny"), **change))
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_layer_saved_bytes(c)
    assert e.value.status == status


def test_null_and_misaligned_pointers_rejected_before_launch():
    c = _lib.layer_cfg(fi.config("tiny"))
    w = _lib.LayerWeights(*([0x1000] * 8 + [0, 0, 0]))
    with pytest.raises(_lib.ForgeError) as e:      # x_in NULL
        _lib.forge_layer_fwd(c, w, None, 0x2000, 0x3000, 0x4000, None, 0)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG
    with pytest.raises(_lib.ForgeError) as e:      # misaligned x_out
        _lib.forge_layer_fwd(c, w, 0x2000, 0x2008, 0x3000, 0x4000, None, 0)
    assert e.value.status == _lib.FORGE_ERR_ALIGNMENT
    with pytest.raises(_lib.ForgeError) as e:      # x_out overlaps x_in
        _lib.forge_layer_fwd(c, w, 0x200000, 0x200000 + 4096, 0x3000, 0x4000, None, 0)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG
    w_bad = _lib.LayerWeights(*([0x1000] * 7 + [0, 0, 0, 0]))   # rope_sin NULL
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_layer_fwd(c, w_bad, 0x2000, 0x900000, 0x3000, 0x4000, None, 0)
    assert "rope_sin" in str(e.value)


def test_gemm_argument_rules():
    with pytest.raises(_lib.ForgeError) as e:      # (MC, KC) is not a supported combination
        _lib.forge_gemm(1, 0, 0, 0x1000, 0x2000, 0x3000, None, 8, 8, 8, 8, 8, 8, 0, 0)
    assert e.value.status == _lib.FORGE_ERR_UNSUPPORTED
    with pytest.raises(_lib.ForgeError) as e:      # K-contiguous A with K % 8 != 0
        _lib.forge_gemm(0, 0, 0, 0x1000, 0x2000, 0x3000, None, 8, 8, 12, 16, 16, 8, 0, 0)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG
    with pytest.raises(_lib.ForgeError) as e:      # residual epilogue without R
        _lib.forge_gemm(0, 0, 1, 0x1000, 0x2000, 0x3000, None, 8, 8, 8, 8, 8, 8, 8, 0)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG
    # empty problems return OK without launching
    _lib.forge_gemm(0, 0, 0, None, None, None, None, 0, 8, 8, 8, 8, 8, 0, 0)


def test_grouped_gemm_argument_rules():
    def status(fn, *a):
        with pytest.raises(_lib.ForgeError) as e:
            fn(*a)
        return e.value.status
    rows, wgrad = _lib.forge_gemm_grouped_rows, _lib.forge_gemm_grouped_wgrad
    P = (0x1000, 0x2000, 0x3000, 0x4000)
    assert status(rows, 2, *P, 4, 64, 16, 16, 16, 16, 16, 256, 0) == _lib.FORGE_ERR_INVALID_ARG
    assert status(rows, 0, *P, 4, 64, 16, 12, 12, 12, 16, 192, 0) == _lib.FORGE_ERR_INVALID_ARG
    assert status(rows, 1, *P, 4, 64, 12, 16, 16, 16, 16, 192, 0) == _lib.FORGE_ERR_INVALID_ARG
    assert status(rows, 0, 0x1000, 0x2008, 0x3000, 0x4000, 4, 64, 16, 16, 16, 16, 16, 256,
                  0) == _lib.FORGE_ERR_ALIGNMENT
    assert status(rows, 0, *P, 4, 64, 16, 16, 16, 16, 16, 252, 0) == _lib.FORGE_ERR_INVALID_ARG
    # per-group outputs may not overlap
    assert status(wgrad, *P, 4, 16, 16, 16, 16, 16, 128, 0) == _lib.FORGE_ERR_INVALID_ARG
    assert status(wgrad, *P, 4, 12, 16, 16, 16, 16, 256, 0) == _lib.FORGE_ERR_INVALID_ARG
    assert status(wgrad, 0x1000, None, 0x3000, 0x4000, 4, 16, 16, 16, 16, 16, 256,
                  0) == _lib.FORGE_ERR_INVALID_ARG
    # nothing to do: OK without launching
    rows(0, None, None, None, None, 0, 64, 16, 16, 16, 16, 16, 256, 0)
    wgrad(None, None, None, None, 4, 0, 16, 16, 16, 16, 256, 0)


def test_optimizer_argument_rules():
    hp = _lib.AdamwHparams(0.9, 1.5, 1e-8, 0.1)
    with pytest.raises(_lib.ForgeError):
        _lib.forge_adamw_step(0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 10, hp, 0x6000, 0)
    ok = _lib.AdamwHparams(0.9, 0.95, 1e-8, 0.1)
    _lib.forge_adamw_step(None, None, None, None, None, 0, ok, None, 0)   # n = 0: no-op
    with pytest.raises(_lib.ForgeError):
        _lib.forge_loss_workspace_bytes(_lib.HeadCfg(16, 64, 1001, 1e-5))  # vocab % 8


def test_layer_bwd_adamw_argument_rules():
    """The fused backward + update checks its optimizer arguments before any
    launch: every used weight's state present and aligned, param the very
    weight pointer, valid hyper-parameters, non-NULL device scalars."""
    c = _lib.layer_cfg(fi.config("tiny"))
    ptrs = [0x10000 * (i + 1) for i in range(8)]
    w = _lib.LayerWeights(*(ptrs + [0, 0, 0]))
    g = _lib.LayerGrads(*([0x900000 + 0x1000 * i for i in range(6)] + [0, 0, 0]), 1)
    names = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")

    def optim(**change):
        t = {n: dict(master=0xA00000 + 0x1000 * i, param=ptrs[i], m=0xB00000 + 0x1000 * i,
                     v=0xC00000 + 0x1000 * i) for i, n in enumerate(names)}
        for k, v in change.items():
            n, field = k.split("__")
            t[n][field] = v
        o = _lib.LayerOptim()
        for n, d in t.items():
            setattr(o, n, _lib.AdamwTensor(d["master"], d["param"], d["m"], d["v"]))
        return o

    hp = _lib.AdamwHparams(0.9, 0.95, 1e-8, 0.1)
    args = (c, w, 0x2000, 0x3000, 0x4000, 0x5000, g)

    def status(o, h=hp, sc=0x6000):
        try:
            _lib.forge_layer_bwd_adamw(*args, o, h, sc, 0x7000, 0)
        except _lib.ForgeError as e:
            return e.status
        return _lib.FORGE_OK

    assert status(optim(w_o__param=ptrs[1])) == _lib.FORGE_ERR_INVALID_ARG   # not the weight
    assert status(optim(w_down__m=0)) == _lib.FORGE_ERR_INVALID_ARG
    assert status(optim(w_qkv__v=0xC01008)) == _lib.FORGE_ERR_ALIGNMENT
    assert status(optim(), h=_lib.AdamwHparams(0.9, 1.0, 1e-8, 0.1)) == _lib.FORGE_ERR_INVALID_ARG
    assert status(optim(), sc=None) == _lib.FORGE_ERR_INVALID_ARG


def test_moe_layer_sizes():
    c5 = fi.config("moe_layer")
    cfg = _lib.layer_cfg(c5)
    T, k, h, fe = 8192, 8, 2048, 1408
    saved = _lib.forge_layer_saved_bytes(cfg)
    # routed rows xs, G|U, A, ys dominate the saved activations
    assert saved >= 2 * T * k * (h + 2 * fe + fe + h)
    assert _lib.forge_layer_workspace_bytes(cfg) >= 2 * T * k * (2 * h + 3 * fe)
    assert _lib.forge_moe_route_workspace_bytes(T, 64, 8) >= T * 8 * 4
    assert _lib.forge_moe_route_workspace_bytes(T, 160, 16) >= T * 16 * 4
    with pytest.raises(_lib.ForgeError):
        _lib.forge_moe_route_workspace_bytes(T, 257, 8)
    # the routing items lie inside the saved buffer and do not overlap
    items = sorted(_lib.forge_layer_saved_item(cfg, i) for i in range(6))
    sizes = dict(zip(range(6), [T * k * 4, T * k * 4, T * 64 * 4, 64 * 4, 65 * 4, T * k * 4]))
    assert sorted(n for _, n in items) == sorted(sizes.values())
    for (o1, n1), (o2, _) in zip(items, items[1:]):
        assert o1 + n1 <= o2
    assert items[-1][0] + items[-1][1] <= saved
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_layer_saved_item(cfg, 6)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_layer_saved_item(_lib.layer_cfg(fi.config("tiny")), 0)
    assert e.value.status == _lib.FORGE_ERR_UNSUPPORTED


def test_moe_route_noalloc_refuses_requests_beyond_its_scratch():
    # host-side limits of the fixed scratch: refused before any launch
    big = _lib.MOE_ROUTE_NOALLOC_MAX_ENTRIES // 16 + 1
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_moe_route_noalloc(16, big, 64, 16, 16, 16, 16, 16, 16, 16, stream=0)
    assert e.value.status == _lib.FORGE_ERR_UNSUPPORTED
    with pytest.raises(_lib.ForgeError) as e:   # histogram limit: blocks * experts
        _lib.forge_moe_route_noalloc(16, 128 * 1024, 256, 1, 16, 16, 16, 16, 16, 16, stream=0)
    assert e.value.status == _lib.FORGE_ERR_UNSUPPORTED
    with pytest.raises(_lib.ForgeError) as e:
        _lib.forge_moe_route_noalloc(16, 100, 64, 8, 0, 16, 16, 16, 16, 16, stream=0)
    assert e.value.status == _lib.FORGE_ERR_INVALID_ARG


def test_binding_structs_match_the_c_header(tmp_path):
    """Every struct of include/forge.h as the C compiler lays it out (size and
    each member's offset) equals the ctypes mirror in the binding."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"forge_layer_cfg": _lib.LayerCfg, "forge_layer_weights": _lib.LayerWeights,
               "forge_layer_grads": _lib.LayerGrads, "forge_head_cfg": _lib.HeadCfg,
               "forge_adamw_hparams": _lib.AdamwHparams, "forge_adamw_tensor": _lib.AdamwTensor,
               "forge_layer_optim": _lib.LayerOptim, "forge_attn_cfg": _lib.AttnCfg}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{_lib.HEADER_PATH}"',
             "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    got = {}
    for line in out.splitlines():
        cname, field, val = line.split()
        got[(cname, field)] = int(val)
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_elementwise_building_block_argument_rules():
    E = _lib.ForgeError
    bad = [
        lambda: _lib.forge_rmsnorm_fwd(0x1000, 0x2000, 0x3000, 0x4000, 4, 12, 1e-5, 0),   # h % 8
        lambda: _lib.forge_rmsnorm_fwd(0x1000, 0x2000, 0x3000, 0x4000, 4, 16384, 1e-5, 0),
        lambda: _lib.forge_rmsnorm_fwd(0x1000, 0x2000, 0x1010, 0x4000, 4, 16, 1e-5, 0),  # y overlaps x
        lambda: _lib.forge_rmsnorm_fwd(0x1000, 0x2000, 0x3000, 0x4000, 4, 16, -1.0, 0),
        lambda: _lib.forge_rmsnorm_bwd(0x1000, 0x2000, 0x3000, 0x4000, None, 0x4000, 0x5000, 0,
                                       4, 16, 0x6000, 0),                                # dx aliases dy
        lambda: _lib.forge_rope_apply(0x1000, 60, 0x2000, 0x3000, None, 4, 4, 2, 32, 0, 0),  # ld % 8
        lambda: _lib.forge_rope_apply(0x1000, 64, 0x2000, 0x3000, None, 4, 4, 3, 32, 0, 0),  # heads > ld
        lambda: _lib.forge_rope_apply(0x1000, 64, 0x2000, 0x3000, None, 4, 4, 2, 24, 0, 0),  # d % 16
        lambda: _lib.forge_swiglu_fwd(0x1000, 0x1040, 4, 16, 0),                          # a inside gu
        lambda: _lib.forge_swiglu_bwd(0x1000, 0x9000, 0x1000, 4, 16, 0),                  # dgu is gu
        lambda: _lib.forge_swiglu_fwd(0x1000, 0x9000, 4, 12, 0),
    ]
    for i, call in enumerate(bad):
        with pytest.raises(E) as e:
            call()
        assert e.value.status == _lib.FORGE_ERR_INVALID_ARG, i
    with pytest.raises(E) as e:                                                    # misaligned
        _lib.forge_rmsnorm_fwd(0x1008, 0x2000, 0x3000, 0x4000, 4, 16, 1e-5, 0)
    assert e.value.status == _lib.FORGE_ERR_ALIGNMENT
    with pytest.raises(E) as e:                                                    # positions
        _lib.forge_rope_apply(0x1000, 64, 0x2000, 0x3000, 0x4002, 4, 4, 2, 32, 0, 0)
    assert e.value.status == _lib.FORGE_ERR_ALIGNMENT
    # no rows: OK without a launch
    _lib.forge_rmsnorm_fwd(None, None, None, None, 0, 16, 1e-5, 0)
    _lib.forge_rmsnorm_bwd(None, 0x2000, None, None, None, None, 0x5000, 1, 0, 16, None, 0)
    _lib.forge_swiglu_fwd(None, None, 0, 16, 0)
    _lib.forge_rope_apply(None, 64, None, None, None, 0, 4, 2, 32, 0, 0)
    assert _lib.forge_rmsnorm_bwd_workspace_bytes(4096, 4096) % (4096 * 4) == 0

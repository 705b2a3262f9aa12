"""ctypes binding of libforge (include/forge.h): same names, argument marshalling only.

Every function takes device pointers as ints or as objects with a
``data_ptr()`` method (torch tensors), and a stream handle (an int, a
``torch.cuda.Stream``, or None for torch's current stream). A non-OK status
raises ForgeError with the library's message. Nothing here computes: every
step of the path runs in the HIP kernels of libforge.so, and importing this
module fails loudly when that library has not been built.
"""
from __future__ import annotations

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libforge.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "forge.h")

FORGE_OK = 0
FORGE_ERR_INVALID_ARG = 1
FORGE_ERR_UNSUPPORTED = 2
FORGE_ERR_ALIGNMENT = 3
FORGE_ERR_HIP = 4
GRAD_NORM_WORKSPACE_FLOATS = 1024

# routing items of a MoE layer's saved buffer (forge_layer_saved_item)
SAVED_ROUTE_IDX, SAVED_ROUTE_GATES, SAVED_ROUTE_PROBS = 0, 1, 2
SAVED_ROUTE_COUNTS, SAVED_ROUTE_OFFSETS, SAVED_ROUTE_PERM = 3, 4, 5

# GEMM operand layouts and epilogues (forge_gemm)
GEMM_KC, GEMM_MC = 0, 1
EPI_STORE_BF16, EPI_RESID_BF16, EPI_ACC_F32, EPI_STORE_F32 = 0, 1, 2, 3


class ForgeError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__(f"{status_name(status)}: {message}")


class LayerCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "seq", "hidden", "n_heads", "n_kv_heads", "head_dim", "ffn")] + [
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
        ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
        ("expert_ffn", ctypes.c_int32), ("aux_coef", ctypes.c_float),
        ("recompute_attn", ctypes.c_int32), ("qk_norm", ctypes.c_int32),
        ("branch_scale", ctypes.c_float), ("shared_ffn", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down",
                 "rope_cos", "rope_sin", "w_router", "w_gate_up_e", "w_down_e",
                 "q_norm", "k_norm", "positions", "w_gate_up_s", "w_down_s")]


class LayerGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("d_attn_norm", "d_w_qkv", "d_w_o", "d_ffn_norm", "d_w_gate_up",
                 "d_w_down", "d_w_router", "d_w_gate_up_e", "d_w_down_e", "d_q_norm",
                 "d_k_norm", "d_w_gate_up_s", "d_w_down_s")] + \
        [("overwrite", ctypes.c_int32)]


class HeadCfg(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("logit_scale", ctypes.c_float)]


class AdamwHparams(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class AdamwTensor(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("master", "param", "m", "v")]


class LayerOptim(ctypes.Structure):
    _fields_ = [(n, AdamwTensor) for n in
                ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down",
                 "w_router", "w_gate_up_e", "w_down_e", "q_norm", "k_norm", "w_gate_up_s",
                 "w_down_s")]


class AttnCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "seq", "n_heads", "n_kv_heads", "head_dim")]


_lib = None


def load():
    """Load libforge.so; raises ImportError if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"libforge.so not found at {LIB_PATH}: build it first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    SZ = ctypes.POINTER(ctypes.c_size_t)
    sigs = {
        "forge_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "forge_last_error": (ctypes.c_char_p, []),
        "forge_version": (ctypes.c_char_p, []),
        "forge_layer_saved_bytes": (ctypes.c_int, [ctypes.POINTER(LayerCfg), SZ]),
        "forge_layer_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(LayerCfg), SZ]),
        "forge_layer_saved_item": (ctypes.c_int, [ctypes.POINTER(LayerCfg), I32, SZ, SZ]),
        "forge_rope_table": (ctypes.c_int, [I32, I32, F32, P, P, P]),
        "forge_layer_fwd": (ctypes.c_int, [ctypes.POINTER(LayerCfg),
                                           ctypes.POINTER(LayerWeights), P, P, P, P, P, P]),
        "forge_layer_bwd": (ctypes.c_int, [ctypes.POINTER(LayerCfg),
                                           ctypes.POINTER(LayerWeights), P, P, P, P,
                                           ctypes.POINTER(LayerGrads), P, P]),
        "forge_loss_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(HeadCfg), SZ]),
        "forge_loss_chunked_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(HeadCfg), I32,
                                                               SZ]),
        "forge_loss_fwd_bwd_chunked": (ctypes.c_int, [ctypes.POINTER(HeadCfg), I32, P, P, P, P,
                                                      P, P, P, P, P, P]),
        "forge_loss_fwd_bwd": (ctypes.c_int, [ctypes.POINTER(HeadCfg), P, P, P, P, P, P,
                                              P, P, P, P]),
        "forge_embed_fwd": (ctypes.c_int, [P, P, P, I32, I32, I32, F32, P]),
        "forge_rmsnorm_fwd": (ctypes.c_int, [P, P, P, P, I32, I32, F32, P]),
        "forge_rmsnorm_bwd_workspace_bytes": (ctypes.c_int, [I32, I32, ctypes.POINTER(ctypes.c_size_t)]),
        "forge_rmsnorm_bwd": (ctypes.c_int, [P, P, P, P, P, P, P, I32, I32, I32, P, P]),
        "forge_rope_apply": (ctypes.c_int, [P, I64, P, P, P, I32, I32, I32, I32, I32, P]),
        "forge_swiglu_fwd": (ctypes.c_int, [P, P, I32, I32, P]),
        "forge_swiglu_bwd": (ctypes.c_int, [P, P, P, I32, I32, P]),
        "forge_embed_bwd": (ctypes.c_int, [P, P, P, I32, I32, I32, F32, P]),
        "forge_adamw_step": (ctypes.c_int, [P, P, P, P, P, I64,
                                            ctypes.POINTER(AdamwHparams), P, P]),
        "forge_layer_bwd_adamw": (ctypes.c_int, [ctypes.POINTER(LayerCfg),
                                                 ctypes.POINTER(LayerWeights), P, P, P, P,
                                                 ctypes.POINTER(LayerGrads),
                                                 ctypes.POINTER(LayerOptim),
                                                 ctypes.POINTER(AdamwHparams), P, P, P]),
        "forge_adamw_advance": (ctypes.c_int, [P, P, F32, ctypes.c_double, ctypes.c_double, P]),
        "forge_grad_norm_sq": (ctypes.c_int, [P, I64, P, P, P]),
        "forge_clip_coeff": (ctypes.c_int, [P, F32, F32, P, P]),
        "forge_gemm": (ctypes.c_int, [I32, I32, I32, P, P, P, P, I32, I32, I32,
                                      I64, I64, I64, I64, P]),
        "forge_gemm_grouped_rows": (ctypes.c_int, [I32, P, P, P, P, I32, I32, I32, I32,
                                                   I64, I64, I64, I64, P]),
        "forge_gemm_grouped_wgrad": (ctypes.c_int, [P, P, P, P, I32, I32, I32, I64, I64,
                                                    I64, I64, P]),
        "forge_attention_fwd": (ctypes.c_int, [ctypes.POINTER(AttnCfg), P, P, P, P]),
        "forge_attention_bwd_workspace_bytes": (ctypes.c_int,
                                                [ctypes.POINTER(AttnCfg), SZ]),
        "forge_attention_bwd": (ctypes.c_int, [ctypes.POINTER(AttnCfg), P, P, P, P, P,
                                               P, P]),
        "forge_moe_route_workspace_bytes": (ctypes.c_int, [I32, I32, I32, SZ]),
        "forge_moe_route": (ctypes.c_int, [P, I32, I32, I32, P, P, P, P, P, P, P, P]),
        "forge_moe_route_noalloc": (ctypes.c_int, [P, I32, I32, I32, P, P, P, P, P, P, P]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def header_functions(path: str = HEADER_PATH):
    """Names of the functions include/forge.h declares."""
    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(forge_[a-z0-9_]+)\s*\(", src)))


def status_name(status: int) -> str:
    return load().forge_status_string(status).decode()


def _check(status: int):
    if status != FORGE_OK:
        raise ForgeError(status, load().forge_last_error().decode())


def _ptr(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream
    return int(s)


def layer_cfg(c: dict) -> LayerCfg:
    return LayerCfg(c["batch"], c["seq"], c["hidden"], c["n_heads"], c["n_kv_heads"],
                    c["head_dim"], c.get("ffn", 0), c["rope_base"], c["rms_eps"],
                    c.get("n_experts", 0), c.get("top_k", 0), c.get("expert_ffn", 0),
                    c.get("aux_coef", 0.0), c.get("recompute_attn", 0), c.get("qk_norm", 0),
                    c.get("branch_scale", 0.0), c.get("shared_ffn", 0))


def layer_weights(w: dict) -> LayerWeights:
    return LayerWeights(*[_ptr(w.get(n)) for n, _ in LayerWeights._fields_])


def layer_grads(g: dict, overwrite: bool = False) -> LayerGrads:
    return LayerGrads(*[_ptr(g.get(n)) for n, _ in LayerGrads._fields_[:-1]], int(overwrite))


def layer_optim(t: dict) -> LayerOptim:
    """t: weight name -> dict(master=, param=, m=, v=) of device tensors."""
    o = LayerOptim()
    for name, _ in LayerOptim._fields_:
        if name in t:
            setattr(o, name, AdamwTensor(*[_ptr(t[name][k]) for k in ("master", "param", "m", "v")]))
    return o


def attn_cfg(c: dict) -> AttnCfg:
    return AttnCfg(c["batch"], c["seq"], c["n_heads"], c["n_kv_heads"], c["head_dim"])


# ---------------------------------------------------------------- calls ----

def forge_version() -> str:
    return load().forge_version().decode()


def forge_layer_saved_bytes(cfg: LayerCfg) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_layer_saved_bytes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def forge_layer_workspace_bytes(cfg: LayerCfg) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_layer_workspace_bytes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def forge_layer_saved_item(cfg: LayerCfg, item: int):
    """(byte offset, bytes) of a routing item within a MoE layer's saved buffer."""
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().forge_layer_saved_item(ctypes.byref(cfg), int(item), ctypes.byref(off),
                                         ctypes.byref(n)))
    return off.value, n.value


def forge_rope_table(seq, head_dim, base, cos_out, sin_out, stream=None):
    _check(load().forge_rope_table(seq, head_dim, base, _ptr(cos_out), _ptr(sin_out),
                                   _stream(stream)))


def forge_layer_fwd(cfg, weights, x_in, x_out, saved, workspace, aux_loss=None,
                    stream=None):
    _check(load().forge_layer_fwd(ctypes.byref(cfg), ctypes.byref(weights), _ptr(x_in),
                                  _ptr(x_out), _ptr(saved), _ptr(workspace),
                                  _ptr(aux_loss), _stream(stream)))


def forge_layer_bwd(cfg, weights, saved, x_in, d_out, d_in, grads, workspace, stream=None):
    _check(load().forge_layer_bwd(ctypes.byref(cfg), ctypes.byref(weights), _ptr(saved),
                                  _ptr(x_in), _ptr(d_out), _ptr(d_in), ctypes.byref(grads),
                                  _ptr(workspace), _stream(stream)))


def forge_loss_workspace_bytes(cfg: HeadCfg) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_loss_workspace_bytes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def forge_loss_fwd_bwd(cfg, x_L, final_norm, w_lm, targets, loss_out, d_x_L, d_final_norm,
                       d_w_lm, workspace, stream=None):
    _check(load().forge_loss_fwd_bwd(ctypes.byref(cfg), _ptr(x_L), _ptr(final_norm),
                                     _ptr(w_lm), _ptr(targets), _ptr(loss_out), _ptr(d_x_L),
                                     _ptr(d_final_norm), _ptr(d_w_lm), _ptr(workspace),
                                     _stream(stream)))


def forge_loss_chunked_workspace_bytes(cfg: HeadCfg, chunk: int) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_loss_chunked_workspace_bytes(ctypes.byref(cfg), int(chunk),
                                                     ctypes.byref(n)))
    return n.value


def forge_loss_fwd_bwd_chunked(cfg, chunk, x_L, final_norm, w_lm, targets, loss_out, d_x_L,
                               d_final_norm, d_w_lm, workspace, stream=None):
    _check(load().forge_loss_fwd_bwd_chunked(ctypes.byref(cfg), int(chunk), _ptr(x_L),
                                             _ptr(final_norm), _ptr(w_lm), _ptr(targets),
                                             _ptr(loss_out), _ptr(d_x_L), _ptr(d_final_norm),
                                             _ptr(d_w_lm), _ptr(workspace), _stream(stream)))


def forge_embed_fwd(ids, emb, x0, tokens, hidden, vocab, scale=1.0, stream=None):
    _check(load().forge_embed_fwd(_ptr(ids), _ptr(emb), _ptr(x0), tokens, hidden, vocab,
                                  float(scale), _stream(stream)))


def forge_rmsnorm_fwd(x, g, y, rstd, tokens, hidden, eps, stream=None):
    _check(load().forge_rmsnorm_fwd(_ptr(x), _ptr(g), _ptr(y), _ptr(rstd), tokens, hidden,
                                    float(eps), _stream(stream)))


def forge_rmsnorm_bwd_workspace_bytes(tokens, hidden) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_rmsnorm_bwd_workspace_bytes(tokens, hidden, ctypes.byref(n)))
    return n.value


def forge_rmsnorm_bwd(x, g, rstd, dy, resid, dx, dg, accumulate, tokens, hidden, workspace,
                      stream=None):
    _check(load().forge_rmsnorm_bwd(_ptr(x), _ptr(g), _ptr(rstd), _ptr(dy), _ptr(resid),
                                    _ptr(dx), _ptr(dg), int(bool(accumulate)), tokens, hidden,
                                    _ptr(workspace), _stream(stream)))


def forge_rope_apply(qkv, ld, rope_cos, rope_sin, positions, tokens, seq, n_rot, head_dim,
                     inverse=False, stream=None):
    _check(load().forge_rope_apply(_ptr(qkv), int(ld), _ptr(rope_cos), _ptr(rope_sin),
                                   _ptr(positions), tokens, seq, n_rot, head_dim,
                                   int(bool(inverse)), _stream(stream)))


def forge_swiglu_fwd(gu, a, tokens, ffn, stream=None):
    _check(load().forge_swiglu_fwd(_ptr(gu), _ptr(a), tokens, ffn, _stream(stream)))


def forge_swiglu_bwd(gu, da, dgu, tokens, ffn, stream=None):
    _check(load().forge_swiglu_bwd(_ptr(gu), _ptr(da), _ptr(dgu), tokens, ffn, _stream(stream)))


def forge_embed_bwd(ids, dx0, d_emb, tokens, hidden, vocab, scale=1.0, stream=None):
    _check(load().forge_embed_bwd(_ptr(ids), _ptr(dx0), _ptr(d_emb), tokens, hidden, vocab,
                                  float(scale), _stream(stream)))


def forge_adamw_step(master, param, grad, m, v, n, hparams: AdamwHparams, dev_scalars,
                     stream=None):
    _check(load().forge_adamw_step(_ptr(master), _ptr(param), _ptr(grad), _ptr(m), _ptr(v),
                                   int(n), ctypes.byref(hparams), _ptr(dev_scalars),
                                   _stream(stream)))


def forge_layer_bwd_adamw(cfg, weights, saved, x_in, d_out, d_in, grads, optim: LayerOptim,
                          hparams: AdamwHparams, dev_scalars, workspace, stream=None):
    _check(load().forge_layer_bwd_adamw(ctypes.byref(cfg), ctypes.byref(weights), _ptr(saved),
                                        _ptr(x_in), _ptr(d_out), _ptr(d_in),
                                        ctypes.byref(grads), ctypes.byref(optim),
                                        ctypes.byref(hparams), _ptr(dev_scalars),
                                        _ptr(workspace), _stream(stream)))


def forge_adamw_advance(dev_scalars, dev_step, lr, beta1, beta2, stream=None):
    _check(load().forge_adamw_advance(_ptr(dev_scalars), _ptr(dev_step), lr, beta1, beta2,
                                      _stream(stream)))


def forge_grad_norm_sq(g, n, accum, workspace, stream=None):
    _check(load().forge_grad_norm_sq(_ptr(g), int(n), _ptr(accum), _ptr(workspace),
                                     _stream(stream)))


def forge_clip_coeff(norm_sq, max_norm, eps, dev_scalars, stream=None):
    _check(load().forge_clip_coeff(_ptr(norm_sq), max_norm, eps, _ptr(dev_scalars),
                                   _stream(stream)))


def forge_gemm(layout_a, layout_b, epilogue, A, B, C, R, M, N, K, lda, ldb, ldc, ldr=0,
               stream=None):
    _check(load().forge_gemm(layout_a, layout_b, epilogue, _ptr(A), _ptr(B), _ptr(C),
                             _ptr(R), M, N, K, lda, ldb, ldc, ldr, _stream(stream)))


def forge_gemm_grouped_rows(layout_b, A, B, C, offsets, groups, rows, N, K, lda, ldb, ldc,
                            stride_b, stream=None):
    _check(load().forge_gemm_grouped_rows(layout_b, _ptr(A), _ptr(B), _ptr(C), _ptr(offsets),
                                          groups, rows, N, K, lda, ldb, ldc, stride_b,
                                          _stream(stream)))


def forge_gemm_grouped_wgrad(A, B, C, offsets, groups, M, N, lda, ldb, ldc, stride_c,
                             stream=None):
    _check(load().forge_gemm_grouped_wgrad(_ptr(A), _ptr(B), _ptr(C), _ptr(offsets), groups,
                                           M, N, lda, ldb, ldc, stride_c, _stream(stream)))


def forge_attention_fwd(cfg: AttnCfg, qkv, o, lse, stream=None):
    _check(load().forge_attention_fwd(ctypes.byref(cfg), _ptr(qkv), _ptr(o), _ptr(lse),
                                      _stream(stream)))


def forge_attention_bwd_workspace_bytes(cfg: AttnCfg) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_attention_bwd_workspace_bytes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def forge_attention_bwd(cfg: AttnCfg, qkv, o, lse, d_o, d_qkv, workspace, stream=None):
    _check(load().forge_attention_bwd(ctypes.byref(cfg), _ptr(qkv), _ptr(o), _ptr(lse),
                                      _ptr(d_o), _ptr(d_qkv), _ptr(workspace),
                                      _stream(stream)))


def forge_moe_route_workspace_bytes(tokens, n_experts, top_k) -> int:
    n = ctypes.c_size_t()
    _check(load().forge_moe_route_workspace_bytes(tokens, n_experts, top_k, ctypes.byref(n)))
    return n.value


def forge_moe_route(logits, tokens, n_experts, top_k, idx, gates, probs, counts, offsets, perm,
                    workspace, stream=None):
    _check(load().forge_moe_route(_ptr(logits), tokens, n_experts, top_k, _ptr(idx), _ptr(gates),
                                  _ptr(probs), _ptr(counts), _ptr(offsets), _ptr(perm),
                                  _ptr(workspace), _stream(stream)))


MOE_ROUTE_NOALLOC_MAX_ENTRIES = 1 << 19
MOE_ROUTE_NOALLOC_MAX_HIST = 1 << 17


def forge_moe_route_noalloc(logits, tokens, n_experts, top_k, idx, gates, probs, counts, offsets,
                            perm, stream=None):
    _check(load().forge_moe_route_noalloc(_ptr(logits), tokens, n_experts, top_k, _ptr(idx),
                                          _ptr(gates), _ptr(probs), _ptr(counts), _ptr(offsets),
                                          _ptr(perm), _stream(stream)))

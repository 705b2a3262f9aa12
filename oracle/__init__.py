"""fp64 CPU oracle for one decoder-layer training step.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check of the entry module
and the bench's CPU-baseline leg may import this package. The GPU library
never calls it, and it shares no code with the GPU path: no kernels, headers,
helpers, tables or constants. The one thing both sides see is the seeded
input generator, which holds none of the method's arithmetic.

What it computes is the plain definition of the training step of a
decoder-only transformer with grouped-query attention, SwiGLU feed-forward
blocks, pre-normalisation RMSNorm and RoPE (App. B "Model Architectures"),
trained in bf16 with fp32 weight-gradient accumulation (Sec. 4.2.2, Table
"Forged-kernel throughput", caption), with the fused clip + AdamW + bf16
write-back update of App. F ("Vertical integration") and the device-side clip
coefficient of App. F ("Deep customization"). The method only reaches this
definition faster, so the oracle is the definition written out: naive
full-matrix causal attention, hand-derived backward formulas, fp64 throughout
on the exact values of the bf16/fp32 inputs, nothing rounded in between.

Modules
  dense   RMSNorm, RoPE, causal GQA attention, SwiGLU, dense layer fwd/bwd
  moe     top-k softmax routing, canonical permutation, expert FFN, aux loss
  head    embedding, final norm + LM head + softmax cross-entropy, model step
  adamw   AdamW with clip coefficient, gradient norm, bf16 rounding

Where the paper is silent the readings are fixed in each function's docstring
(rotate-half RoPE, contiguous GQA groups, mean CE over all tokens, top-k ties
to the lower expert id, no top-k renormalisation, Switch-style aux loss).

Parity status: every function here is pinned by a CPU test against closed
forms, invariants, brute force or central finite differences, except the
whole-step values at the large workload sizes, which no source fixes
("parity unpinned" beyond the per-function pins).
"""
from . import dense, moe, head, adamw  # noqa: F401

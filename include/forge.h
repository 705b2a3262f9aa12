/*
 * forge.h — C ABI of libforge: one decoder-layer training step on MI355X.
 *
 * The library runs one training step of a decoder-only transformer of the
 * kind the paper's engines train (App. B "Model Architectures": grouped-query
 * attention, SwiGLU feed-forward, pre-normalisation RMSNorm, RoPE), in bf16
 * with fp32 weight-gradient accumulation (Sec. 4.2.2, Table "Forged-kernel
 * throughput", caption), as hand-written HIP kernels for gfx950. Calls follow
 * the paper's direct-dispatch model: raw device pointers plus a stream, no
 * framework types (App. J, "Direct dispatch").
 *
 * Conventions (every entry point):
 *   - Pointers are device memory owned by the caller unless a parameter says
 *     "host". The library allocates no device memory and keeps no state
 *     beyond a per-device property cache and, per device, the side streams
 *     and events of the layer backward (created on first use).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *     default stream). Nothing synchronises with the host.
 *   - Arguments are validated on the host before anything is launched; a
 *     failed check returns a status and launches nothing. A failed launch
 *     returns FORGE_ERR_HIP. forge_last_error() gives a message for the last
 *     failing call on the calling thread.
 *   - Base pointers of tensors must be 16-byte aligned (FORGE_ERR_ALIGNMENT).
 *   - bf16 is carried as its 16-bit pattern (forge_bf16).
 *   - Matrices are row-major. Weights follow the nn.Linear convention
 *     [out_features, in_features], y = x W^T.
 *   - Gradient outputs documented as "+=" are accumulated into; the caller
 *     zeroes them before the first accumulation.
 *   - Results are deterministic (bit-identical across runs on one device)
 *     except where a function says otherwise.
 *   - Calls on one stream are ordered; concurrent calls on different streams
 *     must not share workspace, saved or output buffers.
 *   - Every call can be captured into a HIP graph on `stream` (App. E,
 *     "Whole-forward graph capture", extended here to the whole step): no
 *     allocation, memset, copy or host synchronisation happens inside; the
 *     layer backward's side streams join the capture through events recorded
 *     on `stream` and are joined back before the call returns. Run one
 *     forge_layer_bwd / forge_layer_bwd_adamw on the device eagerly before
 *     the first capture (it creates the side streams); keep step-dependent
 *     scalars on the device (forge_adamw_advance, forge_clip_coeff).
 */
#ifndef FORGE_H
#define FORGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t forge_bf16;
typedef void* forge_stream;

typedef enum {
  FORGE_OK = 0,
  FORGE_ERR_INVALID_ARG = 1,   /* null pointer, bad size, aliasing          */
  FORGE_ERR_UNSUPPORTED = 2,   /* valid request the library does not handle */
  FORGE_ERR_ALIGNMENT = 3,     /* base pointer not 16-byte aligned          */
  FORGE_ERR_HIP = 4            /* a HIP runtime call or launch failed       */
} forge_status;

/* Static string naming a status. Never NULL. */
const char* forge_status_string(forge_status s);

/* Message describing the last non-OK status returned on this thread
 * (empty string if none). Valid until the next call on this thread. */
const char* forge_last_error(void);

/* Library version string, e.g. "forge 0.1 gfx950". */
const char* forge_version(void);

/* ------------------------------------------------------------------------ */
/* Layer configuration                                                      */
/* ------------------------------------------------------------------------ */

/*
 * Shape and hyperparameters of one decoder layer (App. B). T = batch * seq
 * tokens, stored batch-row major. hq = n_heads * head_dim,
 * hkv = n_kv_heads * head_dim; query head n uses key/value head
 * n / (n_heads / n_kv_heads) (contiguous GQA groups).
 *
 * n_experts == 0 selects the dense SwiGLU FFN of width `ffn`. n_experts > 0
 * selects the routed MoE FFN of the paper's sparse model (App. B, Table "H100
 * architecture configurations": routed experts, top-k): every token goes to
 * its top_k experts (dropless, no capacity), each a SwiGLU FFN of width
 * expert_ffn; the router is a softmax over all experts of fp32 logits
 * b w_router^T, a token's experts are its top_k logits (ties to the lower
 * expert id), each weighted by its softmax probability (no renormalisation);
 * the load-balance loss aux_coef * E * sum_e f_e P_e (f_e = share of routed
 * slots, a constant; P_e = mean router probability) is added to aux_loss.
 * MoE limits: n_experts a multiple of 8 and <= 256, 1 <= top_k <= min(E, 16),
 * expert_ffn a multiple of 8.
 *
 * recompute_attn != 0: the forward does not keep the attention output and
 * its row statistics; the backward re-runs the attention forward (a
 * recomputation policy, Sec. 3.3, "Surpass" stage).
 *
 * Model variants of App. B (all off when zero):
 *   qk_norm != 0: per-head QK-Norm (Qwen3): every q and k head vector is
 *     RMS-normalised over head_dim (eps = rms_eps) with the gains q_norm /
 *     k_norm [head_dim] before RoPE.
 *   branch_scale: both residual branches are multiplied by it (MiniCPM's
 *     muP scale_depth / sqrt(n_layers)): h1 = x + s Attn, out = h1 + s FFN;
 *     0 means 1.
 *   shared_ffn (MoE layers): width of an always-on shared SwiGLU expert
 *     added to the routed experts' sum (MiniCPM5 16B-A3B's 512-wide shared
 *     expert); a multiple of 8, 0 for none.
 *
 * Supported: head_dim in {64, 128}; n_heads % n_kv_heads == 0;
 * hidden, ffn, hq multiples of 8; seq >= 1; batch >= 1.
 */
typedef struct {
  int32_t batch, seq, hidden, n_heads, n_kv_heads, head_dim, ffn;
  float rope_base, rms_eps;
  int32_t n_experts, top_k, expert_ffn;
  float aux_coef;
  int32_t recompute_attn;
  int32_t qk_norm;
  float branch_scale;
  int32_t shared_ffn;
} forge_layer_cfg;

/*
 * Layer weights (bf16, caller-owned, read only).
 *   attn_norm [h]            RMSNorm gain before attention
 *   w_qkv     [hq+2hkv, h]   rows: q heads, then k heads, then v heads;
 *                            each head's head_dim rows contiguous
 *   w_o       [h, hq]
 *   ffn_norm  [h]
 *   w_gate_up [2f, h]        rows: gate (f rows), then up (f rows)
 *   w_down    [h, f]
 *   rope_cos, rope_sin [seq, head_dim/2] fp32 tables from forge_rope_table
 *   MoE only (unused when n_experts == 0):
 *   w_router [E, h], w_gate_up_e [E, 2fe, h], w_down_e [E, h, fe]
 *   qk_norm only: q_norm [head_dim], k_norm [head_dim]
 *   shared_ffn only: w_gate_up_s [2fs, h] (gate rows, then up rows), w_down_s [h, fs]
 *   positions: device int32 [T], the RoPE position of every token (document-
 *     aware RoPE, App. A step 23: e.g. each token's offset inside its
 *     document of a packed row), in [0, seq) (values outside are clamped);
 *     NULL: a token's position is its index in its batch row. Attention
 *     stays causal over the whole batch row either way.
 */
typedef struct {
  const forge_bf16* attn_norm;
  const forge_bf16* w_qkv;
  const forge_bf16* w_o;
  const forge_bf16* ffn_norm;
  const forge_bf16* w_gate_up;
  const forge_bf16* w_down;
  const float* rope_cos;
  const float* rope_sin;
  const forge_bf16* w_router;
  const forge_bf16* w_gate_up_e;
  const forge_bf16* w_down_e;
  const forge_bf16* q_norm;
  const forge_bf16* k_norm;
  const int32_t* positions;
  const forge_bf16* w_gate_up_s;
  const forge_bf16* w_down_s;
} forge_layer_weights;

/*
 * Weight gradients, fp32, same shapes as the weights. With overwrite == 0
 * they are accumulated (+=, micro-batch accumulation: the caller zeroes them
 * before the first micro-batch); with overwrite != 0 every one is written
 * (=), the same values as accumulating into zeros, without the zeroing pass
 * or the read of the old contents.
 */
typedef struct {
  float* d_attn_norm;
  float* d_w_qkv;
  float* d_w_o;
  float* d_ffn_norm;
  float* d_w_gate_up;
  float* d_w_down;
  float* d_w_router;
  float* d_w_gate_up_e;
  float* d_w_down_e;
  float* d_q_norm;
  float* d_k_norm;
  float* d_w_gate_up_s;
  float* d_w_down_s;
  int32_t overwrite;
} forge_layer_grads;

/* Bytes of the `saved` buffer that forge_layer_fwd fills and
 * forge_layer_bwd reads (activations kept for the backward). Host only. */
forge_status forge_layer_saved_bytes(const forge_layer_cfg* cfg, size_t* bytes);

/* Bytes of the scratch `workspace` of forge_layer_fwd / forge_layer_bwd.
 * Host only. The contents need not be preserved between calls. Includes the
 * attention backward's dS scratch: batch * n_heads * 4096 * t (t + 1) / 2
 * bf16 for t = ceil(seq / 64) 64-key tiles (the causal half of each head's
 * seq x seq score gradient; 545 MB at 32 heads and seq 4096). */
forge_status forge_layer_workspace_bytes(const forge_layer_cfg* cfg, size_t* bytes);

/* Items of a MoE layer's saved buffer that forge_layer_saved_item locates:
 * the routing decision of the forward (App. B, routed experts with top-k
 * selection), as the backward reads it. */
#define FORGE_SAVED_ROUTE_IDX 0      /* int32 [T, top_k]: chosen experts, descending logit */
#define FORGE_SAVED_ROUTE_GATES 1    /* fp32 [T, top_k]: their router probabilities */
#define FORGE_SAVED_ROUTE_PROBS 2    /* fp32 [T, E]: router softmax over all experts */
#define FORGE_SAVED_ROUTE_COUNTS 3   /* int32 [E]: routed (token, slot) entries per expert */
#define FORGE_SAVED_ROUTE_OFFSETS 4  /* int32 [E + 1]: exclusive scan of the counts */
#define FORGE_SAVED_ROUTE_PERM 5     /* int32 [T * top_k]: flat entries, expert-major order */

/* Byte offset and size, within the `saved` buffer that forge_layer_fwd fills
 * for this configuration, of one routing item above (valid after the
 * forward has completed on its stream, unchanged by the backward). Host
 * only. UNSUPPORTED for a dense layer; INVALID_ARG for an unknown item. */
forge_status forge_layer_saved_item(const forge_layer_cfg* cfg, int32_t item, size_t* offset,
                                    size_t* bytes);

/*
 * RoPE tables: for position s < seq and pair index i < head_dim/2,
 * angle = s * base^(-2i/head_dim) (rotate-half pairing (i, i + head_dim/2)),
 * cos_out[s*head_dim/2 + i] = cos(angle), sin_out[...] = sin(angle), computed
 * in fp64 on the device and stored as fp32. Position restarts at 0 in every
 * batch row. Fill once per (seq, head_dim, base).
 */
forge_status forge_rope_table(int32_t seq, int32_t head_dim, float base,
                              float* cos_out, float* sin_out, forge_stream stream);

/* ------------------------------------------------------------------------ */
/* Elementwise steps of the layer as building blocks (the same kernels the  */
/* layer calls; for per-kernel measurement and per-step parity tests)       */
/* ------------------------------------------------------------------------ */

/*
 * RMSNorm forward (App. B pre-normalisation; the layer's two norms): per row
 * t, rstd[t] = 1 / sqrt(mean_j x[t,j]^2 + eps) in fp32, y[t,j] =
 * bf16(x[t,j] * rstd[t] * g[j]). x, y [T, h] bf16 (y must not overlap x),
 * g [h] bf16, rstd [T] fp32. 8 <= h <= 8192, h % 8 == 0.
 */
forge_status forge_rmsnorm_fwd(const forge_bf16* x, const forge_bf16* g, forge_bf16* y,
                               float* rstd, int32_t tokens, int32_t hidden, float eps,
                               forge_stream stream);

/* Scratch bytes of forge_rmsnorm_bwd (per-block gain-gradient partials).
 * Host only. */
forge_status forge_rmsnorm_bwd_workspace_bytes(int32_t tokens, int32_t hidden, size_t* bytes);

/*
 * RMSNorm backward: with y = RMSNorm(x; g) as above and dy [T, h] bf16,
 * dx = d<y, dy>/dx (+ resid when resid is non-NULL: a residual stream's
 * gradient passing the norm), written as bf16 [T, h]; the gain gradient
 * sum_t dy*x*rstd is added to dg [h] fp32 (accumulate != 0) or stored
 * (accumulate == 0), summed over fixed row blocks in a fixed order. rstd is
 * the forward's. dx must not overlap x, dy or resid. Limits as the forward.
 */
forge_status forge_rmsnorm_bwd(const forge_bf16* x, const forge_bf16* g, const float* rstd,
                               const forge_bf16* dy, const forge_bf16* resid, forge_bf16* dx,
                               float* dg, int32_t accumulate, int32_t tokens, int32_t hidden,
                               void* workspace, forge_stream stream);

/*
 * RoPE (App. B), in place on the first n_rot heads of each row of a fused
 * qkv buffer [T, ld] bf16 (head r at columns r*head_dim ..): rotate-half
 * pairs (i, i + head_dim/2) of token t rotated by the angle of its position
 * (positions[t] when non-NULL, clamped to [0, seq); else t mod seq), from the
 * forge_rope_table tables [seq, head_dim/2]; inverse != 0 rotates back (the
 * backward). head_dim % 16 == 0, ld % 8 == 0, n_rot * head_dim <= ld;
 * positions (int32 [T]) 4-byte aligned.
 */
forge_status forge_rope_apply(forge_bf16* qkv, int64_t ld, const float* rope_cos,
                              const float* rope_sin, const int32_t* positions, int32_t tokens,
                              int32_t seq, int32_t n_rot, int32_t head_dim, int32_t inverse,
                              forge_stream stream);

/*
 * SwiGLU (App. B): gu [T, 2f] bf16 holds the gate G (columns 0..f-1) and up
 * U (columns f..2f-1) of each row; a [T, f] bf16 = bf16(silu(G) * U) with
 * silu(z) = z / (1 + exp(-z)) in fp32. f % 8 == 0; a must not overlap gu.
 */
forge_status forge_swiglu_fwd(const forge_bf16* gu, forge_bf16* a, int32_t tokens, int32_t ffn,
                              forge_stream stream);

/*
 * SwiGLU backward: from da [T, f] bf16, writes dgu [T, 2f] bf16 = [dG | dU]
 * with dG = da * U * silu'(G), dU = da * silu(G) (fp32 math, one rounding).
 * dgu must not overlap gu or da.
 */
forge_status forge_swiglu_bwd(const forge_bf16* gu, const forge_bf16* da, forge_bf16* dgu,
                              int32_t tokens, int32_t ffn, forge_stream stream);

/*
 * One decoder layer forward (App. B):
 *   a  = RMSNorm(x; attn_norm)        qkv = a w_qkv^T, RoPE on q and k
 *   o  = causal GQA attention(q,k,v)  h1  = x + o w_o^T
 *   b  = RMSNorm(h1; ffn_norm)        x_out = h1 + (silu(b Wg^T) * (b Wu^T)) w_down^T
 * x_in, x_out: [T, h] bf16; x_out must not overlap x_in.
 * For a MoE layer the FFN branch is h1 + sum_j gate_j FFN_{e_j}(b) instead.
 * saved: forge_layer_saved_bytes bytes, written here, read by the backward.
 * workspace: forge_layer_workspace_bytes bytes of scratch (may be NULL for a
 * dense layer without recompute_attn).
 * aux_loss: device fp32 scalar, MoE only: += the layer's load-balance loss;
 * may be NULL (the loss is then not reported; the backward still includes
 * its gradient).
 */
forge_status forge_layer_fwd(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                             const forge_bf16* x_in, forge_bf16* x_out,
                             void* saved, void* workspace, float* aux_loss,
                             forge_stream stream);

/*
 * Backward of forge_layer_fwd for upstream gradient d_out [T, h] (bf16):
 * writes d_in [T, h] (bf16, may alias d_out) and accumulates every weight
 * gradient into `grads` (fp32 +=, or = when grads->overwrite is set). x_in and saved must be those of the
 * matching forward. Weight gradients are the data-gradient / weight-gradient
 * product pair of every projection (App. C). For a MoE layer the objective
 * is <x_out, d_out> + aux: the router gradient includes the load-balance
 * term, and expert weights that received no tokens get no contribution.
 * MoE results are deterministic; d_w_router goes through a bf16 rounding of
 * the router logit gradient.
 */
forge_status forge_layer_bwd(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                             const void* saved, const forge_bf16* x_in,
                             const forge_bf16* d_out, forge_bf16* d_in,
                             const forge_layer_grads* grads, void* workspace,
                             forge_stream stream);

/* ------------------------------------------------------------------------ */
/* Output head: final RMSNorm + LM head + softmax cross-entropy            */
/* ------------------------------------------------------------------------ */

/* logit_scale: the logits are multiplied by it before the softmax (MiniCPM's
 * muP: the final hidden state divided by hidden / dim_model_base); 0 means 1. */
typedef struct {
  int32_t tokens, hidden, vocab;
  float rms_eps;
  float logit_scale;
} forge_head_cfg;

/* Scratch bytes for forge_loss_fwd_bwd (holds the [T, V] bf16 logits). */
forge_status forge_loss_workspace_bytes(const forge_head_cfg* cfg, size_t* bytes);

/*
 * Fused output head, forward and backward in one call (the fused fp32
 * cross-entropy of App. A (framework-level trajectory) and App. G (fused
 * FP32 cross-entropy)):
 *   xn = RMSNorm(x_L; final_norm), z = xn w_lm^T (bf16 logits, [T, V]),
 *   u = logit_scale z, loss = (1/T) sum_t (logsumexp(u_t) - u_t[targets_t]),
 *   softmax in fp32, then dz = logit_scale (softmax(u) - onehot) / T and the
 *   gradients.
 * x_L [T, h] bf16; final_norm [h] bf16; w_lm [V, h] bf16 (the embedding
 * matrix when the head is tied); targets [T] int32 in [0, V) (checked on the
 * device: an out-of-range target contributes nothing and sets loss to NaN).
 * Outputs: loss_out device fp32 scalar (=); d_x_L [T, h] bf16 (=);
 * d_final_norm [h] fp32 (+=); d_w_lm [V, h] fp32 (+=).
 */
forge_status forge_loss_fwd_bwd(const forge_head_cfg* cfg, const forge_bf16* x_L,
                                const forge_bf16* final_norm, const forge_bf16* w_lm,
                                const int32_t* targets, float* loss_out,
                                forge_bf16* d_x_L, float* d_final_norm, float* d_w_lm,
                                void* workspace, forge_stream stream);

/* Scratch bytes for forge_loss_fwd_bwd_chunked: as forge_loss_workspace_bytes
 * with min(chunk, T) rows of logits instead of T. chunk >= 1. */
forge_status forge_loss_chunked_workspace_bytes(const forge_head_cfg* cfg, int32_t chunk,
                                                size_t* bytes);

/*
 * forge_loss_fwd_bwd over token chunks of `chunk` rows (the chunked / streaming
 * cross-entropy of App. G): per chunk, its logits, their cross-entropy
 * forward and backward in place, the chunk's rows of the input gradient and
 * its share of d_w_lm; only chunk x V logits exist at a time. Same arguments,
 * ownership and accumulation rules as forge_loss_fwd_bwd (the loss is still
 * the mean over all T tokens); d_w_lm gains the chunks' shares one after
 * another, so its fp32 sums are ordered by chunk (equal to the unchunked
 * result up to fp32 rounding). Costs one fp32 read-modify-write of d_w_lm
 * per chunk. chunk >= 1; chunk >= T is the unchunked head.
 */
forge_status forge_loss_fwd_bwd_chunked(const forge_head_cfg* cfg, int32_t chunk,
                                        const forge_bf16* x_L, const forge_bf16* final_norm,
                                        const forge_bf16* w_lm, const int32_t* targets,
                                        float* loss_out, forge_bf16* d_x_L,
                                        float* d_final_norm, float* d_w_lm, void* workspace,
                                        forge_stream stream);

/* ------------------------------------------------------------------------ */
/* Embedding                                                                */
/* ------------------------------------------------------------------------ */

/* x0[t, :] = scale * emb[ids[t], :]. ids [T] int32, emb [V, h] bf16, x0
 * [T, h] bf16; scale is MiniCPM's muP scale_emb (App. B), 1 for a plain
 * copy (bit for bit). An id outside [0, V) yields a zero row. */
forge_status forge_embed_fwd(const int32_t* ids, const forge_bf16* emb, forge_bf16* x0,
                             int32_t tokens, int32_t hidden, int32_t vocab, float scale,
                             forge_stream stream);

/* d_emb[ids[t], :] += scale * dx0[t, :] (fp32 +=). Ids outside [0, V) are
 * skipped. Uses fp32 atomics: the summation order over repeated ids varies
 * between runs (not bit-deterministic). */
forge_status forge_embed_bwd(const int32_t* ids, const forge_bf16* dx0, float* d_emb,
                             int32_t tokens, int32_t hidden, int32_t vocab, float scale,
                             forge_stream stream);

/* ------------------------------------------------------------------------ */
/* Optimizer                                                                */
/* ------------------------------------------------------------------------ */

typedef struct {
  float beta1, beta2, eps, weight_decay;
} forge_adamw_hparams;

/*
 * Fused clip + AdamW + bf16 write-back over n elements of flat fp32 buffers
 * (App. F, "Vertical integration"):
 *   g = grad * clip; m = b1 m + (1-b1) g; v = b2 v + (1-b2) g^2
 *   master -= lr * ((m / bc1) / (sqrt(v / bc2) + eps) + wd * master)
 *   param = bf16(master), round to nearest even
 * dev_scalars: device fp32 [4] = {lr, bc1, bc2, clip}, read in the kernel so
 * the host refreshes them once per step without a sync (App. F, "Deep
 * customization"); bc1 = 1 - b1^t, bc2 = 1 - b2^t.
 * master, m, v: updated in place; param: written; grad: read only.
 * n may be 0 (no launch).
 */
forge_status forge_adamw_step(float* master, forge_bf16* param, const float* grad,
                              float* m, float* v, int64_t n,
                              const forge_adamw_hparams* hp, const float* dev_scalars,
                              forge_stream stream);

/* The step scalars of forge_adamw_step kept on the device, so a whole
 * training step needs no host writes and can be captured into a graph and
 * replayed (App. F, "Deep customization": step scalars on the device):
 *   t = ++dev_step[0]; dev_scalars[0] = lr;
 *   dev_scalars[1] = 1 - beta1^t; dev_scalars[2] = 1 - beta2^t
 * (betas and powers in fp64, then rounded to fp32: the bias corrections of
 * the exact betas, not of their fp32 roundings that the moment updates of
 * forge_adamw_hparams use). dev_scalars[3] (the clip
 * coefficient, from forge_clip_coeff or set once by the caller) is left as
 * it is. dev_step: device int32, 0 before the first step. */
forge_status forge_adamw_advance(float* dev_scalars, int32_t* dev_step, float lr, double beta1,
                                 double beta2, forge_stream stream);

/* Floats of scratch that forge_grad_norm_sq needs. */
#define FORGE_GRAD_NORM_WORKSPACE_FLOATS 1024

/* accum[0] += sum_i g[i]^2 over n fp32 elements (device scalar), the first
 * half of the device-side gradient-norm / clip pipeline (App. F, "Deep
 * customization"). workspace: FORGE_GRAD_NORM_WORKSPACE_FLOATS device
 * floats of scratch. The summation order is fixed (deterministic). */
forge_status forge_grad_norm_sq(const float* g, int64_t n, float* accum,
                                float* workspace, forge_stream stream);

/* dev_scalars[3] = min(1, max_norm / (sqrt(max(norm_sq[0], 0)) + eps)), on
 * the device (App. F, "Deep customization"). */
forge_status forge_clip_coeff(const float* norm_sq, float max_norm, float eps,
                              float* dev_scalars, forge_stream stream);

/* Optimizer state of one weight tensor: fp32 master copy, fp32 moments m
 * and v, and the bf16 parameter, all with the weight's element count and
 * 16-byte aligned (device). */
typedef struct {
  float* master;
  forge_bf16* param;
  float* m;
  float* v;
} forge_adamw_tensor;

/* Optimizer state of one layer's weights, named as in forge_layer_weights.
 * Entries of weights the layer does not have (the expert weights of a dense
 * layer, w_gate_up / w_down of a MoE layer) are ignored and may be zero. */
typedef struct {
  forge_adamw_tensor attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down;
  forge_adamw_tensor w_router, w_gate_up_e, w_down_e;
  forge_adamw_tensor q_norm, k_norm, w_gate_up_s, w_down_s;
} forge_layer_optim;

/*
 * forge_layer_bwd followed by forge_adamw_step on every weight of the layer
 * (grad = the matching member of `grads`, n = the weight's element count),
 * with the same results bit for bit (App. F: fused clip + AdamW + bf16
 * write-back). Each weight's update is issued as soon as its gradient is
 * complete and the backward has read the weight for the last time, on a
 * stream of the library's own, so the memory-bound updates of the FFN (or
 * expert and router) weights run while the compute-bound attention backward
 * is in flight (layers of fewer than 2^20 token x hidden elements, where
 * the stream hand-offs would cost more than they save, run the updates in
 * order on `stream`).
 * opt: each used entry's param must be the same pointer as the matching
 *   member of w (the update overwrites the weight in place, after the
 *   backward's last read of it); master, m, v are updated in place.
 * hp, dev_scalars: as forge_adamw_step. dev_scalars (the clip coefficient
 *   included) are read by the update kernels while the call's work runs, so
 *   they must hold their final values by the point of `stream` where the
 *   call is enqueued: clipping by this step's own gradient norm needs
 *   forge_layer_bwd, forge_grad_norm_sq, forge_clip_coeff, forge_adamw_step.
 * grads: as forge_layer_bwd (with overwrite == 0 the update uses the
 *   accumulated gradient, so call this on the last micro-batch only).
 * All other arguments and the errors as forge_layer_bwd, plus
 * INVALID_ARG / ALIGNMENT for opt, hp and dev_scalars. The call's work,
 * updates included, is complete when `stream` reaches the point after it.
 */
forge_status forge_layer_bwd_adamw(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                                   const void* saved, const forge_bf16* x_in,
                                   const forge_bf16* d_out, forge_bf16* d_in,
                                   const forge_layer_grads* grads, const forge_layer_optim* opt,
                                   const forge_adamw_hparams* hp, const float* dev_scalars,
                                   void* workspace, forge_stream stream);

/* ------------------------------------------------------------------------ */
/* Building blocks, exposed for per-kernel measurement and tests            */
/* ------------------------------------------------------------------------ */

/* Operand layouts and epilogues of forge_gemm. */
#define FORGE_GEMM_KC 0            /* contiguous along the reduction dim K  */
#define FORGE_GEMM_MC 1            /* contiguous along the M (or N) dim     */
#define FORGE_EPI_STORE_BF16 0     /* C bf16 = acc                          */
#define FORGE_EPI_RESID_BF16 1     /* C bf16 = acc + R (bf16), one rounding */
#define FORGE_EPI_ACC_F32 2        /* C fp32 += acc                         */
#define FORGE_EPI_STORE_F32 3      /* C fp32 = acc                          */

/*
 * C[m][n] (op)= sum_k A(m,k) B(k,n): bf16 operands, fp32 accumulation, on the
 * MFMA units. These are the three products of every projection of the step:
 * the forward and, in the backward, one data-gradient and one
 * weight-gradient product (App. C).
 *   layout_a KC: A(m,k) = A[m*lda + k]    MC: A(m,k) = A[k*lda + m]
 *   layout_b KC: B(k,n) = B[n*ldb + k]    MC: B(k,n) = B[k*ldb + n]
 * so y = x W^T is (KC, KC), dX = dY W is (KC, MC), dW += dY^T X is (MC, MC).
 * Supported: (KC, KC) with every epilogue; (KC, MC) with STORE_BF16 and
 * RESID_BF16; (MC, MC) with ACC_F32 and STORE_F32 (else UNSUPPORTED).
 * Shape rules (else INVALID_ARG): M, N, K >= 0; a KC operand needs K % 8 == 0,
 * an MC operand needs M % 8 == 0 (A) or N % 8 == 0 (B); every leading
 * dimension is a multiple of 8 and at least the operand's contiguous extent;
 * R (RESID_BF16 only, leading dim ldr) must not overlap C.
 */
forge_status forge_gemm(int32_t layout_a, int32_t layout_b, int32_t epilogue,
                        const forge_bf16* A, const forge_bf16* B, void* C,
                        const forge_bf16* R, int32_t M, int32_t N, int32_t K,
                        int64_t lda, int64_t ldb, int64_t ldc, int64_t ldr,
                        forge_stream stream);

/*
 * Grouped products over row groups: the per-expert projections of a routed
 * mixture-of-experts FFN (App. B, MoE configurations), whose routed rows are
 * stored expert-major so that group e owns rows [offsets[e], offsets[e+1]).
 * offsets: device int32 [groups + 1] with offsets[0] = 0, non-decreasing and
 * offsets[groups] <= rows. The offsets are read on the device and not
 * checked: rows beyond `rows` are not computed, and every operand must hold
 * the rows the offsets name. An empty group contributes nothing.
 *
 * forge_gemm_grouped_rows: for r in group e,
 *   C[r][n] = sum_k A[r][k] B_e(k, n)   (bf16 out, fp32 accumulation)
 * with B_e = B + e * stride_b, layout_b KC: B_e(k,n) = B_e[n*ldb + k]
 * (y = x W_e^T, W_e [N, K]) or MC: B_e(k,n) = B_e[k*ldb + n] (dX = dY W_e).
 * Rules (else INVALID_ARG): K % 8 == 0 (K > 0 for KC); N % 8 == 0 for MC;
 * lda >= K, ldb >= K (KC) or N (MC), ldc >= N; every leading dimension and
 * stride_b a multiple of 8. Pointers 16-byte aligned (ALIGNMENT).
 */
forge_status forge_gemm_grouped_rows(int32_t layout_b, const forge_bf16* A, const forge_bf16* B,
                                     forge_bf16* C, const int32_t* offsets, int32_t groups,
                                     int32_t rows, int32_t N, int32_t K, int64_t lda,
                                     int64_t ldb, int64_t ldc, int64_t stride_b,
                                     forge_stream stream);

/*
 * forge_gemm_grouped_wgrad: the per-expert weight gradients, for each group e
 *   C_e[m][n] += sum over rows r of group e of A[r][m] B[r][n]
 * with A [rows, M] (lda), B [rows, N] (ldb) bf16 and C_e = C + e * stride_c
 * fp32 [M, N] (ldc), accumulated (+=; the caller zeroes). Rules (else
 * INVALID_ARG): M, N multiples of 8; lda >= M, ldb >= N, ldc >= N, all and
 * stride_c multiples of 8; stride_c >= (M - 1) * ldc + N (groups do not
 * overlap). Deterministic (one workgroup owns each output tile).
 */
forge_status forge_gemm_grouped_wgrad(const forge_bf16* A, const forge_bf16* B, float* C,
                                      const int32_t* offsets, int32_t groups, int32_t M,
                                      int32_t N, int64_t lda, int64_t ldb, int64_t ldc,
                                      int64_t stride_c, forge_stream stream);

typedef struct {
  int32_t batch, seq, n_heads, n_kv_heads, head_dim;
} forge_attn_cfg;

/*
 * Causal grouped-query attention forward (App. B; causal as in App. C's
 * attention-core count): q, k, v are the column blocks [0, hq), [hq, hq+hkv),
 * [hq+hkv, hq+2hkv) of the fused qkv buffer [T, hq+2hkv] bf16 (after RoPE);
 * o [T, hq] bf16 = softmax(q k^T / sqrt(d) + causal mask) v per head;
 * lse [batch, n_heads, seq] fp32 = natural-log row log-sum-exp of the scaled
 * scores. head_dim in {64, 128}.
 */
forge_status forge_attention_fwd(const forge_attn_cfg* cfg, const forge_bf16* qkv,
                                 forge_bf16* o, float* lse, forge_stream stream);

/* Scratch bytes of forge_attention_bwd: 2 * batch * n_heads * seq fp32
 * (per-query -rowsum(dO o) and -lse log2 e) and the dS scratch described at
 * forge_layer_workspace_bytes, each rounded up to 256 bytes. Host only. */
forge_status forge_attention_bwd_workspace_bytes(const forge_attn_cfg* cfg, size_t* bytes);

/*
 * Attention backward: from d_o [T, hq] bf16 and the forward's qkv, o, lse,
 * writes d_qkv [T, hq+2hkv] bf16 (=): dq for every query head, dk and dv
 * summed over each kv head's query group. dS = P (dP - rowsum(dO o)) is
 * formed once, rounded to bf16 into the workspace, and dq and dk are
 * products over it (no atomics: bitwise deterministic).
 */
forge_status forge_attention_bwd(const forge_attn_cfg* cfg, const forge_bf16* qkv,
                                 const forge_bf16* o, const float* lse,
                                 const forge_bf16* d_o, forge_bf16* d_qkv,
                                 void* workspace, forge_stream stream);

/* Scratch bytes of forge_moe_route. Host only. */
forge_status forge_moe_route_workspace_bytes(int32_t tokens, int32_t n_experts, int32_t top_k,
                                             size_t* bytes);

/*
 * Token routing of the MoE layer on given fp32 logits [tokens, n_experts]
 * (n_experts <= 256): probs [tokens, E] = softmax over all experts; idx
 * [tokens, top_k] = the top_k experts by descending logit, ties to the lower
 * expert id, -0 equal to +0 and NaN ranked below -inf (so every index lies
 * in [0, E) whatever the logits hold; a NaN logit makes that token's probs
 * and gates NaN); gates [tokens, top_k] = their probabilities; counts [E] slots
 * per expert; offsets [E + 1] = exclusive scan of counts; perm [tokens *
 * top_k] = the flat (token * top_k + slot) entries in expert-major order,
 * tokens ascending within an expert, then slots ascending. Integer outputs
 * are bit-exact and deterministic. All pointers device, 4-byte aligned.
 */
forge_status forge_moe_route(const float* logits, int32_t tokens, int32_t n_experts,
                             int32_t top_k, int32_t* idx, float* gates, float* probs,
                             int32_t* counts, int32_t* offsets, int32_t* perm,
                             void* workspace, forge_stream stream);

/* Limits of forge_moe_route_noalloc's fixed scratch. */
#define FORGE_MOE_ROUTE_NOALLOC_MAX_ENTRIES (1 << 19)  /* tokens * top_k */
#define FORGE_MOE_ROUTE_NOALLOC_MAX_HIST (1 << 17)     /* ceil(tokens / 128) * n_experts */

/*
 * forge_moe_route without the workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation. Same arguments, results (bit for bit)
 * and errors as forge_moe_route otherwise. The counting sort's scratch (per
 * block expert histograms, then the inverse permutation) is a fixed device
 * array inside the library, 2.5 MiB on each GPU the library runs on, held
 * until the process ends; every call writes the parts it reads, so nothing
 * in it needs to start at zero. All calls on one GPU share that array: calls
 * that overlap on one GPU (other streams, other threads) race and must be
 * serialised by the caller. Limits: tokens * top_k <=
 * FORGE_MOE_ROUTE_NOALLOC_MAX_ENTRIES and ceil(tokens / 128) * n_experts <=
 * FORGE_MOE_ROUTE_NOALLOC_MAX_HIST, else FORGE_ERR_UNSUPPORTED before any
 * launch. Allocates nothing (the array's device address is looked up once
 * per GPU on its first call).
 */
forge_status forge_moe_route_noalloc(const float* logits, int32_t tokens, int32_t n_experts,
                                     int32_t top_k, int32_t* idx, float* gates, float* probs,
                                     int32_t* counts, int32_t* offsets, int32_t* perm,
                                     forge_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* FORGE_H */

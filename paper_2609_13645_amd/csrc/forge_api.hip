// C ABI of libforge (include/forge.h): argument validation, the layout of
// the caller-owned saved / workspace buffers, and the launch order of one
// decoder layer's forward and backward, the fused output head, embedding,
// optimizer and gradient-norm calls. Every call only enqueues kernels on the
// caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "../../include/forge.h"
#include "kernels.h"

namespace {

using forge::GemmArgs;

thread_local std::string g_last_error;

forge_status fail(forge_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
forge_status fail(forge_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

forge_status ok() {
  return FORGE_OK;
}

#define FORGE_HIP(call)                                                            \
  do {                                                                             \
    hipError_t e_ = (call);                                                        \
    if (e_ != hipSuccess)                                                          \
      return fail(FORGE_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));   \
  } while (0)

#define FORGE_CHECK(cond, status, ...)             \
  do {                                             \
    if (!(cond)) return fail(status, __VA_ARGS__); \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define FORGE_PTR(p)                                                                     \
  do {                                                                                   \
    FORGE_CHECK((p) != nullptr, FORGE_ERR_INVALID_ARG, "%s is NULL", #p);                \
    FORGE_CHECK(aligned16(p), FORGE_ERR_ALIGNMENT, "%s is not 16-byte aligned", #p);     \
  } while (0)

constexpr size_t kAlign = 256;
size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---- derived sizes --------------------------------------------------------
struct Dims {
  long T, h, hq, hkv, qkv, f, nh, nkv, d, B, S;
  long E, k, fe, R;  // MoE: experts, top-k, expert FFN width, routed rows T*k
  long fs;           // MoE: shared expert width (0: none)
  bool qkn;          // QK-Norm
  float bs;          // residual-branch scale (1 unless set)
};

Dims dims(const forge_layer_cfg& c) {
  Dims d;
  d.B = c.batch;
  d.S = c.seq;
  d.T = (long)c.batch * c.seq;
  d.h = c.hidden;
  d.d = c.head_dim;
  d.nh = c.n_heads;
  d.nkv = c.n_kv_heads;
  d.hq = d.nh * d.d;
  d.hkv = d.nkv * d.d;
  d.qkv = d.hq + 2 * d.hkv;
  d.f = c.ffn;
  d.E = c.n_experts;
  d.k = c.top_k;
  d.fe = c.expert_ffn;
  d.R = d.T * d.k;
  d.fs = c.n_experts > 0 ? c.shared_ffn : 0;
  d.qkn = c.qk_norm != 0;
  d.bs = c.branch_scale == 0.0f ? 1.0f : c.branch_scale;
  return d;
}

constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;

forge_status check_cfg(const forge_layer_cfg* c) {
  FORGE_CHECK(c != nullptr, FORGE_ERR_INVALID_ARG, "cfg is NULL");
  FORGE_CHECK(c->batch >= 1 && c->seq >= 1, FORGE_ERR_INVALID_ARG,
              "batch and seq must be >= 1 (got %d, %d)", c->batch, c->seq);
  FORGE_CHECK(c->hidden >= 8 && c->hidden % 8 == 0, FORGE_ERR_INVALID_ARG,
              "hidden must be a positive multiple of 8 (got %d)", c->hidden);
  FORGE_CHECK(c->hidden <= 8192, FORGE_ERR_UNSUPPORTED, "hidden > 8192 (got %d)", c->hidden);
  FORGE_CHECK(c->n_heads >= 1 && c->n_kv_heads >= 1 && c->n_heads % c->n_kv_heads == 0,
              FORGE_ERR_INVALID_ARG, "n_heads (%d) must be a positive multiple of n_kv_heads (%d)",
              c->n_heads, c->n_kv_heads);
  FORGE_CHECK(c->head_dim == 64 || c->head_dim == 128, FORGE_ERR_UNSUPPORTED,
              "head_dim must be 64 or 128 (got %d)", c->head_dim);
  FORGE_CHECK(c->n_experts >= 0, FORGE_ERR_INVALID_ARG, "n_experts must be >= 0");
  if (c->n_experts == 0) {
    FORGE_CHECK(c->ffn >= 8 && c->ffn % 8 == 0, FORGE_ERR_INVALID_ARG,
                "ffn must be a positive multiple of 8 (got %d)", c->ffn);
  } else {
    FORGE_CHECK(c->n_experts % 8 == 0 && c->n_experts <= kMaxExperts, FORGE_ERR_UNSUPPORTED,
                "n_experts must be a multiple of 8 and <= %d (got %d)", kMaxExperts,
                c->n_experts);
    FORGE_CHECK(c->top_k >= 1 && c->top_k <= c->n_experts && c->top_k <= kMaxTopK,
                FORGE_ERR_INVALID_ARG, "top_k must be in [1, min(n_experts, %d)] (got %d)",
                kMaxTopK, c->top_k);
    FORGE_CHECK(c->expert_ffn >= 8 && c->expert_ffn % 8 == 0, FORGE_ERR_INVALID_ARG,
                "expert_ffn must be a positive multiple of 8 (got %d)", c->expert_ffn);
    FORGE_CHECK(std::isfinite(c->aux_coef), FORGE_ERR_INVALID_ARG, "aux_coef must be finite");
  }
  FORGE_CHECK(c->rms_eps >= 0.0f && std::isfinite(c->rms_eps), FORGE_ERR_INVALID_ARG,
              "rms_eps must be finite and >= 0");
  FORGE_CHECK(c->branch_scale >= 0.0f && std::isfinite(c->branch_scale), FORGE_ERR_INVALID_ARG,
              "branch_scale must be finite and >= 0 (0 means 1)");
  FORGE_CHECK(c->shared_ffn >= 0 && c->shared_ffn % 8 == 0, FORGE_ERR_INVALID_ARG,
              "shared_ffn must be a non-negative multiple of 8 (got %d)", c->shared_ffn);
  FORGE_CHECK(c->shared_ffn == 0 || c->n_experts > 0, FORGE_ERR_INVALID_ARG,
              "shared_ffn needs a MoE layer (n_experts > 0)");
  FORGE_CHECK(c->rope_base > 0.0f && std::isfinite(c->rope_base), FORGE_ERR_INVALID_ARG,
              "rope_base must be finite and > 0");
  const Dims d = dims(*c);
  const long widest = std::max(std::max(d.qkv, 2 * d.f), std::max(d.h, 2 * d.fs));
  FORGE_CHECK(d.T * widest < (1L << 31), FORGE_ERR_UNSUPPORTED,
              "a [T, width] activation exceeds 2^31 elements");
  FORGE_CHECK(d.E == 0 || d.R * std::max(2 * d.fe, d.h) < (1L << 31), FORGE_ERR_UNSUPPORTED,
              "a [T * top_k, width] routed activation exceeds 2^31 elements");
  return FORGE_OK;
}

// ---- saved buffer ----------------------------------------------------------
// Everything the backward reads. Dense FFN: b, G|U, A. MoE FFN: b, router
// probabilities, routing (idx, gates, counts, offsets, perm, pos_of), the
// routed rows xs, G|U, A and the expert outputs ys.
struct Saved {
  size_t a, rstd1, qkv, o, lse, h1, rstd2, b, gu, act;
  size_t probs, idx, gates, counts, offsets, perm, pos_of, xs, ys;
  size_t qk_raw, rstd_qk, gu_s, act_s;  // QK-Norm; shared expert
  size_t total;
};

Saved saved_layout(const forge_layer_cfg& c) {
  const Dims d = dims(c);
  Saved s{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += up(bytes); return o; };
  s.a = take(d.T * d.h * 2);
  s.rstd1 = take(d.T * 4);
  s.qkv = take(d.T * d.qkv * 2);
  if (d.qkn) {
    s.qk_raw = take(d.T * (d.hq + d.hkv) * 2);
    s.rstd_qk = take(d.T * (d.nh + d.nkv) * 4);
  }
  const bool keep = c.recompute_attn == 0;
  s.o = keep ? take(d.T * d.hq * 2) : 0;
  s.lse = keep ? take(d.B * d.nh * d.S * 4) : 0;
  s.h1 = take(d.T * d.h * 2);
  s.rstd2 = take(d.T * 4);
  s.b = take(d.T * d.h * 2);
  if (d.E == 0) {
    s.gu = take(d.T * 2 * d.f * 2);
    s.act = take(d.T * d.f * 2);
  } else {
    s.probs = take(d.T * d.E * 4);
    s.idx = take(d.R * 4);
    s.gates = take(d.R * 4);
    s.counts = take(d.E * 4);
    s.offsets = take((d.E + 1) * 4);
    s.perm = take(d.R * 4);
    s.pos_of = take(d.R * 4);
    s.xs = take(d.R * d.h * 2);
    s.gu = take(d.R * 2 * d.fe * 2);
    s.act = take(d.R * d.fe * 2);
    s.ys = take(d.R * d.h * 2);
    if (d.fs) {
      s.gu_s = take(d.T * 2 * d.fs * 2);
      s.act_s = take(d.T * d.fs * 2);
    }
  }
  s.total = off;
  return s;
}

// ---- workspace -------------------------------------------------------------
struct Work {
  size_t dA, dgu, db, dh1, dO, delta, ds, dqkv, da, dg, o, lse;
  size_t logits, blk, colsum, dys, dxs, dgate, dl, dbs, wpart;  // MoE
  size_t qk_dg, h1s, dA_s, dgu_s, db1;  // QK-Norm; shared expert
  size_t total;
};

forge::AttnArgs attn_args(const Dims& d, const uint16_t* qkv);

Work work_layout(const forge_layer_cfg& c) {
  const Dims d = dims(c);
  Work w{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += up(bytes); return o; };
  if (d.E == 0) {
    w.dA = take(d.T * d.f * 2);
    w.dgu = take(d.T * 2 * d.f * 2);
  } else {
    w.dA = take(d.R * d.fe * 2);
    w.dgu = take(d.R * 2 * d.fe * 2);
    w.logits = take(d.T * d.E * 4);
    w.blk = take((size_t)forge::moe_sort_blocks((int)d.T) * d.E * 4);
    w.colsum = take((1 + (size_t)forge::moe_aux_blocks((int)d.T)) * d.E * 4);
    w.dys = take(d.R * d.h * 2);
    w.dxs = take(d.R * d.h * 2);
    w.dgate = take(d.R * 4);
    w.dl = take(d.T * d.E * 2);
    w.dbs = take(d.T * d.h * 2);
    const int rs = forge::splitk_splits((int)d.E, (int)d.h, (int)d.T);
    w.wpart = rs > 1 ? take((size_t)rs * d.E * d.h * 4) : 0;
    if (d.fs) {
      w.h1s = take(d.T * d.h * 2);
      w.dA_s = take(d.T * d.fs * 2);
      w.dgu_s = take(d.T * 2 * d.fs * 2);
      w.db1 = take(d.T * d.h * 2);
    }
  }
  if (d.qkn)
    w.qk_dg = take((size_t)2 * forge::qknorm_bwd_blocks((int)d.T, (int)(d.nh + d.nkv), (int)d.d) *
                   d.d * 4);
  w.db = take(d.T * d.h * 2);
  w.dh1 = take(d.T * d.h * 2);
  w.dO = take(d.T * d.hq * 2);
  w.delta = take(2 * d.B * d.nh * d.S * 4);   // delta, then -lse log2(e)
  w.ds = take(forge::attn_bwd_ds_bytes(attn_args(d, nullptr)));   // dS, causal half
  w.dqkv = take(d.T * d.qkv * 2);
  w.da = take(d.T * d.h * 2);
  w.dg = take((size_t)forge::rmsnorm_bwd_blocks((int)d.T) * d.h * 4);
  const bool rec = c.recompute_attn != 0;
  w.o = rec ? take(d.T * d.hq * 2) : 0;
  w.lse = rec ? take(d.B * d.nh * d.S * 4) : 0;
  w.total = off;
  return w;
}

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}
template <typename T>
const T* at(const void* base, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

GemmArgs gargs(const void* A, long lda, const void* B, long ldb, void* C, long ldc, long M,
               long N, long K, const void* R = nullptr, long ldr = 0) {
  GemmArgs g;
  g.A = static_cast<const uint16_t*>(A);
  g.B = static_cast<const uint16_t*>(B);
  g.C = C;
  g.R = static_cast<const uint16_t*>(R);
  g.M = (int)M;
  g.N = (int)N;
  g.K = (int)K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.ldr = ldr;
  return g;
}

// the same product with every epilogue value multiplied by alpha (a residual
// branch's scale)
GemmArgs scaled(GemmArgs g, float alpha) {
  g.alpha = alpha;
  return g;
}

// weight-gradient epilogue: accumulate, or store when the caller asked for it
forge::GemmEpilogue wgrad_epi(const forge_layer_grads* g) {
  return g->overwrite ? forge::kStoreF32 : forge::kAccF32;
}

GemmArgs grouped(GemmArgs g, const int32_t* off, long E, long strideB, long strideC) {
  g.g_off = off;
  g.groups = (int)E;
  g.strideB = strideB;
  g.strideC = strideC;
  return g;
}

forge::AttnArgs attn_args(const Dims& d, const uint16_t* qkv) {
  forge::AttnArgs a;
  a.q = qkv;
  a.k = qkv + d.hq;
  a.v = qkv + d.hq + d.hkv;
  a.ld_qkv = d.qkv;
  a.batch = (int)d.B;
  a.seq = (int)d.S;
  a.n_heads = (int)d.nh;
  a.n_kv_heads = (int)d.nkv;
  a.d = (int)d.d;
  a.scale = (float)(1.0 / std::sqrt((double)d.d));
  return a;
}

forge_status check_weights(const forge_layer_cfg& c, const forge_layer_weights* w) {
  FORGE_CHECK(w != nullptr, FORGE_ERR_INVALID_ARG, "weights is NULL");
  FORGE_PTR(w->attn_norm);
  FORGE_PTR(w->w_qkv);
  FORGE_PTR(w->w_o);
  FORGE_PTR(w->ffn_norm);
  FORGE_PTR(w->rope_cos);
  FORGE_PTR(w->rope_sin);
  if (c.n_experts == 0) {
    FORGE_PTR(w->w_gate_up);
    FORGE_PTR(w->w_down);
  } else {
    FORGE_PTR(w->w_router);
    FORGE_PTR(w->w_gate_up_e);
    FORGE_PTR(w->w_down_e);
  }
  if (c.qk_norm) {
    FORGE_PTR(w->q_norm);
    FORGE_PTR(w->k_norm);
  }
  if (c.n_experts > 0 && c.shared_ffn > 0) {
    FORGE_PTR(w->w_gate_up_s);
    FORGE_PTR(w->w_down_s);
  }
  FORGE_CHECK((reinterpret_cast<uintptr_t>(w->positions) & 3u) == 0, FORGE_ERR_ALIGNMENT,
              "positions is not 4-byte aligned");
  return FORGE_OK;
}

forge_status check_grads(const forge_layer_cfg& c, const forge_layer_grads* g) {
  FORGE_CHECK(g != nullptr, FORGE_ERR_INVALID_ARG, "grads is NULL");
  FORGE_PTR(g->d_attn_norm);
  FORGE_PTR(g->d_w_qkv);
  FORGE_PTR(g->d_w_o);
  FORGE_PTR(g->d_ffn_norm);
  if (c.n_experts == 0) {
    FORGE_PTR(g->d_w_gate_up);
    FORGE_PTR(g->d_w_down);
  } else {
    FORGE_PTR(g->d_w_router);
    FORGE_PTR(g->d_w_gate_up_e);
    FORGE_PTR(g->d_w_down_e);
  }
  if (c.qk_norm) {
    FORGE_PTR(g->d_q_norm);
    FORGE_PTR(g->d_k_norm);
  }
  if (c.n_experts > 0 && c.shared_ffn > 0) {
    FORGE_PTR(g->d_w_gate_up_s);
    FORGE_PTR(g->d_w_down_s);
  }
  return FORGE_OK;
}

// ---- attention block (shared by the dense and MoE layers) -----------------
// a = RMSNorm(x), qkv = a W_qkv^T, [QK-Norm], RoPE, attention,
// h1 = x + s O W_o^T (s: the branch scale).
forge_status attn_block_fwd(const forge_layer_cfg& c, const Dims& d,
                            const forge_layer_weights* w, const uint16_t* x, uint16_t* a,
                            float* rstd1, uint16_t* qkv, uint16_t* o, float* lse, uint16_t* h1,
                            uint16_t* qk_raw, float* rstd_qk, hipStream_t s) {
  FORGE_HIP(forge::rmsnorm_fwd(x, w->attn_norm, a, rstd1, (int)d.T, (int)d.h, c.rms_eps, s));
  FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kStoreBF16,
                        gargs(a, d.h, w->w_qkv, d.h, qkv, d.qkv, d.T, d.qkv, d.h), s));
  if (d.qkn)
    FORGE_HIP(forge::qknorm_rope_fwd(qkv, d.qkv, qk_raw, rstd_qk, w->q_norm, w->k_norm,
                                     w->rope_cos, w->rope_sin, w->positions, (int)d.T, (int)d.S,
                                     (int)d.nh, (int)d.nkv, (int)d.d, c.rms_eps, s));
  else
    FORGE_HIP(forge::rope_apply(qkv, d.qkv, w->rope_cos, w->rope_sin, w->positions, (int)d.T,
                                (int)d.S, (int)(d.nh + d.nkv), (int)d.d, false, s));
  FORGE_HIP(forge::attn_fwd(attn_args(d, qkv), o, lse, s));
  FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kResidBF16,
                        scaled(gargs(o, d.hq, w->w_o, d.hq, h1, d.h, d.T, d.h, d.hq, x, d.h), d.bs),
                        s));
  return FORGE_OK;
}

// ---- side streams of the layer backward ----------------------------------------
// The dense layer backward (from 2^20 token x hidden elements up) runs its
// four weight-gradient GEMMs on a second stream of the same device, forked from the caller's stream after each one's
// inputs exist and joined back before the call's work ends, so they fill the
// tail waves of the data-gradient GEMMs and the bandwidth-bound kernels in
// between. forge_layer_bwd_adamw adds a third stream for the optimizer
// updates, each forked once its weight's gradient is complete and its
// data-gradient product (the last reader of the weight) has run. Non-blocking
// streams of default priority and their events, one set per device, created
// on first use and kept for the life of the process; launch sequences on one
// device are serialised by a mutex, so concurrent callers do not interleave
// their event records. Each event is recorded once per call and waited on
// right after its record.
constexpr int kMaxDevices = 64;
constexpr int kLaneEvents = 24;
struct SideLane {
  std::mutex mu;
  bool ready = false;
  hipStream_t stream = nullptr;  // weight gradients
  hipStream_t opt = nullptr;     // optimizer updates
  hipEvent_t ev[kLaneEvents] = {};
};
SideLane g_side[kMaxDevices];
std::mutex g_side_init;

// side streams only for layers whose products outlast the event hand-offs
bool use_side_streams(const Dims& d) { return d.T * d.h >= (1L << 20); }

hipError_t side_lane(SideLane** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  SideLane& L = g_side[dev];
  std::lock_guard<std::mutex> lk(g_side_init);
  if (!L.ready) {
    e = hipStreamCreateWithFlags(&L.stream, hipStreamNonBlocking);
    if (e != hipSuccess) return e;
    e = hipStreamCreateWithFlags(&L.opt, hipStreamNonBlocking);
    if (e != hipSuccess) return e;
    for (hipEvent_t& ev : L.ev) {
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e != hipSuccess) return e;
    }
    L.ready = true;
  }
  *out = &L;
  return hipSuccess;
}

// everything enqueued on `from` so far happens before what is enqueued on `to` next
hipError_t link(hipStream_t from, hipStream_t to, hipEvent_t ev) {
  const hipError_t e = hipEventRecord(ev, from);
  return e != hipSuccess ? e : hipStreamWaitEvent(to, ev, 0);
}

// Optimizer updates of forge_layer_bwd_adamw, issued on the lane's optimizer
// stream behind everything enqueued so far on the caller's stream s and the
// weight-gradient stream ws (events 7 onwards; 0..6 are the backward's); a
// layer without a lane issues them in order on s.
struct OptPlan {
  const forge_layer_optim* o;
  const forge_adamw_hparams* hp;
  const float* scalars;
  SideLane* lane;
  int next_ev;
};

hipError_t opt_update(OptPlan* P, hipStream_t s, hipStream_t ws, const forge_adamw_tensor& t,
                      const float* grad, long n) {
  hipStream_t os = s;  // without a lane (small layer): in order on the caller's stream
  if (P->lane) {
    if (P->next_ev + 2 > kLaneEvents) return hipErrorInvalidValue;
    os = P->lane->opt;
    hipError_t e = link(s, os, P->lane->ev[P->next_ev++]);
    if (e == hipSuccess && ws != s) e = link(ws, os, P->lane->ev[P->next_ev++]);
    if (e != hipSuccess) return e;
  }
  return forge::adamw(t.master, reinterpret_cast<uint16_t*>(t.param), grad, t.m, t.v, n,
                      P->hp->beta1, P->hp->beta2, P->hp->eps, P->hp->weight_decay, P->scalars,
                      os);
}

// A weight gradient with the weight's AdamW update in the GEMM epilogue
// (App. F, vertical integration): each tile's gradient is final when the
// tile ends, so the tile updates the same elements of master, m, v and the
// bf16 parameter, exactly as forge_adamw_step would, without another pass
// over the gradient. The weight's data-gradient product must already have
// read the parameter. Used for the MoE expert weights: as a separate pass
// their update (most of an MoE layer's parameters) cannot overlap the rest
// of the backward without holding its kernels off the CUs.
GemmArgs with_adam(GemmArgs a, const OptPlan* P, const forge_adamw_tensor& t) {
  a.o_master = t.master;
  a.o_m = t.m;
  a.o_v = t.v;
  a.o_param = reinterpret_cast<uint16_t*>(t.param);
  a.o_sc = P->scalars;
  a.o_b1 = P->hp->beta1;
  a.o_b2 = P->hp->beta2;
  a.o_eps = P->hp->eps;
  a.o_wd = P->hp->weight_decay;
  return a;
}

forge::GemmEpilogue wgrad_adam_epi(const forge_layer_grads* g) {
  return g->overwrite ? forge::kStoreF32Adam : forge::kAccF32Adam;
}

// the optimizer stream's work happens before what is enqueued on s next
hipError_t opt_join(OptPlan* P, hipStream_t s) {
  if (!P->lane) return hipSuccess;
  if (P->next_ev + 1 > kLaneEvents) return hipErrorInvalidValue;
  return link(P->lane->opt, s, P->lane->ev[P->next_ev++]);
}

// Backward of attn_block_fwd from dh1 (the full gradient at h1, residual
// path included) to d_in.
forge_status attn_block_bwd(const forge_layer_cfg& c, const Dims& d,
                            const forge_layer_weights* w, const forge_layer_grads* g,
                            const uint16_t* x, const uint16_t* a, const float* rstd1,
                            const uint16_t* qkv, const uint16_t* o, const float* lse,
                            const uint16_t* qk_raw, const float* rstd_qk,
                            const uint16_t* dh1, uint16_t* d_in, void* workspace, const Work& wk,
                            hipStream_t s, SideLane* side = nullptr, OptPlan* opt = nullptr,
                            hipEvent_t before_d_in = nullptr) {
  uint16_t* dO = at<uint16_t>(workspace, wk.dO);
  float* delta = at<float>(workspace, wk.delta);
  uint16_t* dqkv = at<uint16_t>(workspace, wk.dqkv);
  uint16_t* da = at<uint16_t>(workspace, wk.da);
  float* dgp = at<float>(workspace, wk.dg);
  const int nblk = forge::rmsnorm_bwd_blocks((int)d.T);
  const forge::AttnArgs aa = attn_args(d, qkv);
  (void)c;
  // weight gradients go to the side stream when there is one (dh1 and o
  // exist: fork now; dqkv after the RoPE backward: fork again)
  hipStream_t ws = side ? side->stream : s;
  if (side) FORGE_HIP(link(s, ws, side->ev[2]));
  FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                        scaled(gargs(dh1, d.h, o, d.hq, g->d_w_o, d.hq, d.h, d.hq, d.T), d.bs),
                        ws));
  FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                        scaled(gargs(dh1, d.h, w->w_o, d.hq, dO, d.hq, d.T, d.hq, d.h), d.bs), s));
  if (opt) FORGE_HIP(opt_update(opt, s, ws, opt->o->w_o, g->d_w_o, d.h * d.hq));
  FORGE_HIP(forge::attn_bwd(aa, o, dO, lse, delta, at<uint16_t>(workspace, wk.ds), dqkv,
                             dqkv + d.hq, dqkv + d.hq + d.hkv, d.qkv, s));
  if (d.qkn) {
    // inverse RoPE and the QK-Norm backward in place; gain gradients
    float* qdg = at<float>(workspace, wk.qk_dg);
    const int nq = forge::qknorm_bwd_blocks((int)d.T, (int)(d.nh + d.nkv), (int)d.d);
    FORGE_HIP(forge::qknorm_rope_bwd(dqkv, d.qkv, qk_raw, rstd_qk, w->q_norm, w->k_norm,
                                     w->rope_cos, w->rope_sin, w->positions, (int)d.T, (int)d.S,
                                     (int)d.nh, (int)d.nkv, (int)d.d, qdg, s));
    FORGE_HIP(forge::rmsnorm_dg_reduce(qdg, nq, g->d_q_norm, (int)d.d, !g->overwrite, s));
    FORGE_HIP(forge::rmsnorm_dg_reduce(qdg + (size_t)nq * d.d, nq, g->d_k_norm, (int)d.d,
                                       !g->overwrite, s));
    if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->q_norm, g->d_q_norm, d.d));
    if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->k_norm, g->d_k_norm, d.d));
  } else {
    FORGE_HIP(forge::rope_apply(dqkv, d.qkv, w->rope_cos, w->rope_sin, w->positions, (int)d.T,
                                (int)d.S, (int)(d.nh + d.nkv), (int)d.d, true, s));
  }
  if (side) FORGE_HIP(link(s, ws, side->ev[3]));
  FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                        gargs(dqkv, d.qkv, a, d.h, g->d_w_qkv, d.h, d.qkv, d.h, d.T), ws));
  FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                        gargs(dqkv, d.qkv, w->w_qkv, d.h, da, d.h, d.T, d.h, d.qkv), s));
  if (opt) FORGE_HIP(opt_update(opt, s, ws, opt->o->w_qkv, g->d_w_qkv, d.qkv * d.h));
  // d_in may alias the layer's upstream gradient, which a side-stream
  // product may still be reading: wait for that product first
  if (before_d_in) FORGE_HIP(hipStreamWaitEvent(s, before_d_in, 0));
  FORGE_HIP(forge::rmsnorm_bwd(x, w->attn_norm, rstd1, da, dh1, d_in, dgp, (int)d.T, (int)d.h, s));
  FORGE_HIP(forge::rmsnorm_dg_reduce(dgp, nblk, g->d_attn_norm, (int)d.h, !g->overwrite, s));
  if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->attn_norm, g->d_attn_norm, d.h));
  if (side) FORGE_HIP(link(ws, s, side->ev[4]));  // join: the call's work ends on s
  if (opt) FORGE_HIP(opt_join(opt, s));
  return FORGE_OK;
}

// ---- MoE FFN ------------------------------------------------------------------
// out = h1 + sum_j gate_j FFN_{e_j}(b), b = RMSNorm(h1) already in saved.b;
// aux (if non-null) += alpha E sum_e f_e P_e.
forge_status moe_ffn_fwd(const forge_layer_cfg& c, const Dims& d, const forge_layer_weights* w,
                         void* saved, const Saved& sv, void* workspace, const Work& wk,
                         const uint16_t* h1, uint16_t* out, float* aux, hipStream_t s) {
  const uint16_t* bn = at<uint16_t>(saved, sv.b);
  float* logits = at<float>(workspace, wk.logits);
  float* probs = at<float>(saved, sv.probs);
  int32_t* idx = at<int32_t>(saved, sv.idx);
  float* gates = at<float>(saved, sv.gates);
  int32_t* counts = at<int32_t>(saved, sv.counts);
  int32_t* offsets = at<int32_t>(saved, sv.offsets);
  int32_t* perm = at<int32_t>(saved, sv.perm);
  int32_t* pos_of = at<int32_t>(saved, sv.pos_of);
  uint16_t* xs = at<uint16_t>(saved, sv.xs);
  uint16_t* gu = at<uint16_t>(saved, sv.gu);
  uint16_t* act = at<uint16_t>(saved, sv.act);
  uint16_t* ys = at<uint16_t>(saved, sv.ys);
  const int T = (int)d.T, E = (int)d.E, k = (int)d.k;
  FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kStoreF32,
                        gargs(bn, d.h, w->w_router, d.h, logits, d.E, d.T, d.E, d.h), s));
  FORGE_HIP(forge::moe_route(logits, T, E, k, idx, gates, probs, s));
  FORGE_HIP(forge::moe_sort(idx, T, E, k, at<int32_t>(workspace, wk.blk), counts, offsets, perm,
                            pos_of, s));
  FORGE_HIP(forge::moe_gather(bn, perm, d.R, (int)d.h, k, xs, s));
  FORGE_HIP(forge::gemm_grouped_m(
      forge::kKC, forge::kStoreBF16,
      grouped(gargs(xs, d.h, w->w_gate_up_e, d.h, gu, 2 * d.fe, d.R, 2 * d.fe, d.h), offsets, E,
              2 * d.fe * d.h, 0), s));
  FORGE_HIP(forge::swiglu_fwd(gu, act, (int)d.R, (int)d.fe, s));
  FORGE_HIP(forge::gemm_grouped_m(
      forge::kKC, forge::kStoreBF16,
      grouped(gargs(act, d.fe, w->w_down_e, d.fe, ys, d.h, d.R, d.h, d.fe), offsets, E,
              d.h * d.fe, 0), s));
  // the shared expert on every token: h1s = h1 + s (silu(b Wg^T) (b Wu^T)) Wd^T,
  // then the routed sum is added on top of it
  const uint16_t* resid = h1;
  if (d.fs) {
    uint16_t* gu_s = at<uint16_t>(saved, sv.gu_s);
    uint16_t* act_s = at<uint16_t>(saved, sv.act_s);
    uint16_t* h1s = at<uint16_t>(workspace, wk.h1s);
    FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kStoreBF16,
                          gargs(bn, d.h, w->w_gate_up_s, d.h, gu_s, 2 * d.fs, d.T, 2 * d.fs, d.h),
                          s));
    FORGE_HIP(forge::swiglu_fwd(gu_s, act_s, (int)d.T, (int)d.fs, s));
    FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kResidBF16,
                          scaled(gargs(act_s, d.fs, w->w_down_s, d.fs, h1s, d.h, d.T, d.h, d.fs,
                                       h1, d.h), d.bs), s));
    resid = h1s;
  }
  FORGE_HIP(forge::moe_combine(ys, gates, pos_of, resid, d.T, (int)d.h, k, d.bs, out, s));
  FORGE_HIP(forge::moe_aux_loss(probs, counts, T, E, k, c.aux_coef,
                                at<float>(workspace, wk.colsum), aux, s));
  return FORGE_OK;
}

// Backward of moe_ffn_fwd for upstream d_out (objective <out, d_out> + aux):
// writes db (the gradient at b) into the workspace.
forge_status moe_ffn_bwd(const forge_layer_cfg& c, const Dims& d, const forge_layer_weights* w,
                         const forge_layer_grads* g, const void* saved, const Saved& sv,
                         void* workspace, const Work& wk, const uint16_t* d_out, uint16_t* db,
                         hipStream_t s, SideLane* side = nullptr, const OptPlan* opt = nullptr) {
  const uint16_t* bn = at<uint16_t>(saved, sv.b);
  const float* probs = at<float>(saved, sv.probs);
  const int32_t* idx = at<int32_t>(saved, sv.idx);
  const float* gates = at<float>(saved, sv.gates);
  const int32_t* counts = at<int32_t>(saved, sv.counts);
  const int32_t* offsets = at<int32_t>(saved, sv.offsets);
  const int32_t* pos_of = at<int32_t>(saved, sv.pos_of);
  const uint16_t* xs = at<uint16_t>(saved, sv.xs);
  const uint16_t* gu = at<uint16_t>(saved, sv.gu);
  const uint16_t* act = at<uint16_t>(saved, sv.act);
  const uint16_t* ys = at<uint16_t>(saved, sv.ys);
  uint16_t* dys = at<uint16_t>(workspace, wk.dys);
  uint16_t* dact = at<uint16_t>(workspace, wk.dA);
  uint16_t* dgu = at<uint16_t>(workspace, wk.dgu);
  uint16_t* dxs = at<uint16_t>(workspace, wk.dxs);
  float* dgate = at<float>(workspace, wk.dgate);
  uint16_t* dl = at<uint16_t>(workspace, wk.dl);
  uint16_t* dbs = at<uint16_t>(workspace, wk.dbs);
  const int T = (int)d.T, E = (int)d.E, k = (int)d.k;
  FORGE_HIP(forge::moe_combine_bwd(ys, gates, pos_of, d_out, d.T, (int)d.h, k, d.bs, dgate, dys,
                                   s));
  // down projection: dgrad into the routed rows, wgrad per expert
  FORGE_HIP(forge::gemm_grouped_m(
      forge::kMC, forge::kStoreBF16,
      grouped(gargs(dys, d.h, w->w_down_e, d.fe, dact, d.fe, d.R, d.fe, d.h), offsets, E,
              d.h * d.fe, 0), s));
  // the expert weight gradients (with updates: in their epilogues, after
  // the data gradient read the weights) go to the side stream when there is
  // one: their operands stay untouched for the rest of the call
  hipStream_t ws = side ? side->stream : s;
  if (side) FORGE_HIP(link(s, ws, side->ev[0]));
  const GemmArgs wd = grouped(gargs(dys, d.h, act, d.fe, g->d_w_down_e, d.fe, d.h, d.fe, 0),
                              offsets, E, 0, d.h * d.fe);
  FORGE_HIP(opt ? forge::gemm_grouped_k(wgrad_adam_epi(g), with_adam(wd, opt, opt->o->w_down_e), ws)
                : forge::gemm_grouped_k(wgrad_epi(g), wd, ws));
  FORGE_HIP(forge::swiglu_bwd(gu, dact, dgu, (int)d.R, (int)d.fe, s));
  FORGE_HIP(forge::gemm_grouped_m(
      forge::kMC, forge::kStoreBF16,
      grouped(gargs(dgu, 2 * d.fe, w->w_gate_up_e, d.h, dxs, d.h, d.R, d.h, 2 * d.fe), offsets,
              E, 2 * d.fe * d.h, 0), s));
  const GemmArgs wgu = grouped(gargs(dgu, 2 * d.fe, xs, d.h, g->d_w_gate_up_e, d.h, 2 * d.fe,
                                     d.h, 0), offsets, E, 0, 2 * d.fe * d.h);
  if (side) FORGE_HIP(link(s, ws, side->ev[1]));
  FORGE_HIP(opt ? forge::gemm_grouped_k(wgrad_adam_epi(g),
                                        with_adam(wgu, opt, opt->o->w_gate_up_e), ws)
                : forge::gemm_grouped_k(wgrad_epi(g), wgu, ws));
  FORGE_HIP(forge::moe_scatter_back(dxs, pos_of, d.T, (int)d.h, k, dbs, s));
  // router: dl through the softmax (gates and aux loss), then its two products
  FORGE_HIP(forge::moe_router_bwd(probs, idx, dgate, counts, T, E, k, c.aux_coef, dl, s));
  uint16_t* db_r = d.fs ? at<uint16_t>(workspace, wk.db1) : db;
  FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kResidBF16,
                        gargs(dl, d.E, w->w_router, d.h, db_r, d.h, d.T, d.h, d.E, dbs, d.h), s));
  if (d.fs) {
    // shared expert: weight gradients beside the rest (side stream when there
    // is one), data gradient added to db
    const uint16_t* gu_s = at<uint16_t>(saved, sv.gu_s);
    const uint16_t* act_s = at<uint16_t>(saved, sv.act_s);
    uint16_t* dA_s = at<uint16_t>(workspace, wk.dA_s);
    uint16_t* dgu_s = at<uint16_t>(workspace, wk.dgu_s);
    if (side) FORGE_HIP(link(s, ws, side->ev[5]));
    FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                          scaled(gargs(d_out, d.h, act_s, d.fs, g->d_w_down_s, d.fs, d.h, d.fs,
                                       d.T), d.bs), ws));
    FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                          scaled(gargs(d_out, d.h, w->w_down_s, d.fs, dA_s, d.fs, d.T, d.fs, d.h),
                                 d.bs), s));
    FORGE_HIP(forge::swiglu_bwd(gu_s, dA_s, dgu_s, (int)d.T, (int)d.fs, s));
    if (side) FORGE_HIP(link(s, ws, side->ev[6]));
    FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                          gargs(dgu_s, 2 * d.fs, bn, d.h, g->d_w_gate_up_s, d.h, 2 * d.fs, d.h,
                                d.T), ws));
    FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kResidBF16,
                          gargs(dgu_s, 2 * d.fs, w->w_gate_up_s, d.h, db, d.h, d.T, d.h, 2 * d.fs,
                                db_r, d.h), s));
  }
  // router weight gradient: 64 x h output tiles over T tokens, split over T
  FORGE_HIP(forge::gemm_wgrad_splitk(gargs(dl, d.E, bn, d.h, g->d_w_router, d.h, d.E, d.h, d.T),
                                     forge::splitk_splits((int)d.E, (int)d.h, (int)d.T),
                                     at<float>(workspace, wk.wpart), !g->overwrite, s));
  return FORGE_OK;
}

}  // namespace

extern "C" {

const char* forge_status_string(forge_status s) {
  switch (s) {
    case FORGE_OK: return "FORGE_OK";
    case FORGE_ERR_INVALID_ARG: return "FORGE_ERR_INVALID_ARG";
    case FORGE_ERR_UNSUPPORTED: return "FORGE_ERR_UNSUPPORTED";
    case FORGE_ERR_ALIGNMENT: return "FORGE_ERR_ALIGNMENT";
    case FORGE_ERR_HIP: return "FORGE_ERR_HIP";
  }
  return "FORGE_ERR_UNKNOWN";
}

const char* forge_last_error(void) { return g_last_error.c_str(); }

const char* forge_version(void) { return "forge 0.2 gfx950"; }

forge_status forge_layer_saved_bytes(const forge_layer_cfg* cfg, size_t* bytes) {
  if (forge_status s = check_cfg(cfg)) return s;
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = saved_layout(*cfg).total;
  return ok();
}

forge_status forge_layer_workspace_bytes(const forge_layer_cfg* cfg, size_t* bytes) {
  if (forge_status s = check_cfg(cfg)) return s;
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = work_layout(*cfg).total;
  return ok();
}

forge_status forge_layer_saved_item(const forge_layer_cfg* cfg, int32_t item, size_t* offset,
                                    size_t* bytes) {
  if (forge_status s = check_cfg(cfg)) return s;
  FORGE_CHECK(offset != nullptr && bytes != nullptr, FORGE_ERR_INVALID_ARG,
              "offset or bytes is NULL");
  FORGE_CHECK(cfg->n_experts > 0, FORGE_ERR_UNSUPPORTED,
              "the saved routing exists for MoE layers only (n_experts == 0)");
  const Saved sv = saved_layout(*cfg);
  const Dims d = dims(*cfg);
  switch (item) {
    case FORGE_SAVED_ROUTE_IDX: *offset = sv.idx; *bytes = d.R * 4; break;
    case FORGE_SAVED_ROUTE_GATES: *offset = sv.gates; *bytes = d.R * 4; break;
    case FORGE_SAVED_ROUTE_PROBS: *offset = sv.probs; *bytes = d.T * d.E * 4; break;
    case FORGE_SAVED_ROUTE_COUNTS: *offset = sv.counts; *bytes = d.E * 4; break;
    case FORGE_SAVED_ROUTE_OFFSETS: *offset = sv.offsets; *bytes = (d.E + 1) * 4; break;
    case FORGE_SAVED_ROUTE_PERM: *offset = sv.perm; *bytes = d.R * 4; break;
    default: return fail(FORGE_ERR_INVALID_ARG, "unknown saved item %d", item);
  }
  return ok();
}

forge_status forge_rope_table(int32_t seq, int32_t head_dim, float base, float* cos_out,
                              float* sin_out, forge_stream stream) {
  FORGE_CHECK(seq >= 1, FORGE_ERR_INVALID_ARG, "seq must be >= 1");
  FORGE_CHECK(head_dim >= 16 && head_dim % 16 == 0, FORGE_ERR_INVALID_ARG,
              "head_dim must be a positive multiple of 16");
  FORGE_CHECK(base > 0.0f && std::isfinite(base), FORGE_ERR_INVALID_ARG, "base must be > 0");
  FORGE_PTR(cos_out);
  FORGE_PTR(sin_out);
  FORGE_HIP(forge::rope_table(seq, head_dim, base, cos_out, sin_out, (hipStream_t)stream));
  return ok();
}

namespace {
forge_status check_rows(int32_t tokens, int32_t hidden) {
  FORGE_CHECK(tokens >= 0, FORGE_ERR_INVALID_ARG, "tokens must be >= 0");
  FORGE_CHECK(hidden >= 8 && hidden <= 8192 && hidden % 8 == 0, FORGE_ERR_INVALID_ARG,
              "hidden must be a multiple of 8 in [8, 8192]");
  return ok();
}
bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return a != nullptr && b != nullptr && x < y + bn && y < x + an;
}
}  // namespace

forge_status forge_rmsnorm_fwd(const forge_bf16* x, const forge_bf16* g, forge_bf16* y,
                               float* rstd, int32_t tokens, int32_t hidden, float eps,
                               forge_stream stream) {
  if (forge_status s = check_rows(tokens, hidden)) return s;
  FORGE_CHECK(eps >= 0.0f && std::isfinite(eps), FORGE_ERR_INVALID_ARG, "eps must be >= 0");
  if (tokens == 0) return ok();
  FORGE_PTR(x);
  FORGE_PTR(g);
  FORGE_PTR(y);
  FORGE_PTR(rstd);
  const size_t n = (size_t)tokens * hidden * 2;
  FORGE_CHECK(!overlap(x, n, y, n), FORGE_ERR_INVALID_ARG, "y overlaps x");
  FORGE_HIP(forge::rmsnorm_fwd(x, g, y, rstd, tokens, hidden, eps, (hipStream_t)stream));
  return ok();
}

forge_status forge_rmsnorm_bwd_workspace_bytes(int32_t tokens, int32_t hidden, size_t* bytes) {
  if (forge_status s = check_rows(tokens, hidden)) return s;
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = (size_t)forge::rmsnorm_bwd_blocks(tokens) * hidden * 4;
  return ok();
}

forge_status forge_rmsnorm_bwd(const forge_bf16* x, const forge_bf16* g, const float* rstd,
                               const forge_bf16* dy, const forge_bf16* resid, forge_bf16* dx,
                               float* dg, int32_t accumulate, int32_t tokens, int32_t hidden,
                               void* workspace, forge_stream stream) {
  if (forge_status s = check_rows(tokens, hidden)) return s;
  FORGE_PTR(g);
  FORGE_PTR(dg);
  hipStream_t st = (hipStream_t)stream;
  if (tokens == 0) {
    // no rows: the gain gradient is an empty sum (a reduction over zero
    // partials, which stores zeros; no memset, so the call stays capturable)
    if (!accumulate) FORGE_HIP(forge::rmsnorm_dg_reduce(nullptr, 0, dg, hidden, false, st));
    return ok();
  }
  FORGE_PTR(x);
  FORGE_PTR(rstd);
  FORGE_PTR(dy);
  FORGE_PTR(dx);
  FORGE_PTR(workspace);
  if (resid) FORGE_PTR(resid);
  const size_t n = (size_t)tokens * hidden * 2;
  FORGE_CHECK(!overlap(dx, n, x, n) && !overlap(dx, n, dy, n) && !overlap(dx, n, resid, n),
              FORGE_ERR_INVALID_ARG, "dx overlaps an input");
  float* part = static_cast<float*>(workspace);
  FORGE_HIP(forge::rmsnorm_bwd(x, g, rstd, dy, resid, dx, part, tokens, hidden, st));
  FORGE_HIP(forge::rmsnorm_dg_reduce(part, forge::rmsnorm_bwd_blocks(tokens), dg, hidden,
                                     accumulate != 0, st));
  return ok();
}

forge_status forge_rope_apply(forge_bf16* qkv, int64_t ld, const float* rope_cos,
                              const float* rope_sin, const int32_t* positions, int32_t tokens,
                              int32_t seq, int32_t n_rot, int32_t head_dim, int32_t inverse,
                              forge_stream stream) {
  FORGE_CHECK(tokens >= 0 && seq >= 1 && n_rot >= 0, FORGE_ERR_INVALID_ARG,
              "bad tokens / seq / n_rot");
  FORGE_CHECK(head_dim >= 16 && head_dim % 16 == 0, FORGE_ERR_INVALID_ARG,
              "head_dim must be a positive multiple of 16");
  FORGE_CHECK(ld % 8 == 0 && (int64_t)n_rot * head_dim <= ld, FORGE_ERR_INVALID_ARG,
              "ld must be a multiple of 8 holding n_rot heads");
  if (tokens == 0 || n_rot == 0) return ok();
  FORGE_PTR(qkv);
  FORGE_PTR(rope_cos);
  FORGE_PTR(rope_sin);
  FORGE_CHECK((reinterpret_cast<uintptr_t>(positions) & 3u) == 0, FORGE_ERR_ALIGNMENT,
              "positions is not 4-byte aligned");
  FORGE_HIP(forge::rope_apply(qkv, ld, rope_cos, rope_sin, positions, tokens, seq, n_rot,
                              head_dim, inverse != 0, (hipStream_t)stream));
  return ok();
}

forge_status forge_swiglu_fwd(const forge_bf16* gu, forge_bf16* a, int32_t tokens, int32_t ffn,
                              forge_stream stream) {
  FORGE_CHECK(tokens >= 0 && ffn >= 8 && ffn % 8 == 0, FORGE_ERR_INVALID_ARG,
              "ffn must be a positive multiple of 8");
  if (tokens == 0) return ok();
  FORGE_PTR(gu);
  FORGE_PTR(a);
  FORGE_CHECK(!overlap(a, (size_t)tokens * ffn * 2, gu, (size_t)tokens * ffn * 4),
              FORGE_ERR_INVALID_ARG, "a overlaps gu");
  FORGE_HIP(forge::swiglu_fwd(gu, a, tokens, ffn, (hipStream_t)stream));
  return ok();
}

forge_status forge_swiglu_bwd(const forge_bf16* gu, const forge_bf16* da, forge_bf16* dgu,
                              int32_t tokens, int32_t ffn, forge_stream stream) {
  FORGE_CHECK(tokens >= 0 && ffn >= 8 && ffn % 8 == 0, FORGE_ERR_INVALID_ARG,
              "ffn must be a positive multiple of 8");
  if (tokens == 0) return ok();
  FORGE_PTR(gu);
  FORGE_PTR(da);
  FORGE_PTR(dgu);
  const size_t n2 = (size_t)tokens * ffn * 4;
  FORGE_CHECK(!overlap(dgu, n2, gu, n2) && !overlap(dgu, n2, da, n2 / 2), FORGE_ERR_INVALID_ARG,
              "dgu overlaps an input");
  FORGE_HIP(forge::swiglu_bwd(gu, da, dgu, tokens, ffn, (hipStream_t)stream));
  return ok();
}

forge_status forge_layer_fwd(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                             const forge_bf16* x_in, forge_bf16* x_out, void* saved,
                             void* workspace, float* aux_loss, forge_stream stream) {
  if (forge_status s = check_cfg(cfg)) return s;
  if (forge_status s = check_weights(*cfg, w)) return s;
  FORGE_PTR(x_in);
  FORGE_PTR(x_out);
  FORGE_PTR(saved);
  const Dims d = dims(*cfg);
  FORGE_CHECK(x_out + d.T * d.h <= x_in || x_in + d.T * d.h <= x_out, FORGE_ERR_INVALID_ARG,
              "x_out overlaps x_in");
  const bool moe = d.E > 0;
  FORGE_CHECK(!(cfg->recompute_attn || moe) || workspace != nullptr, FORGE_ERR_INVALID_ARG,
              "workspace is NULL (needed for recompute_attn and for MoE layers)");
  FORGE_CHECK(aux_loss == nullptr || (reinterpret_cast<uintptr_t>(aux_loss) & 3u) == 0,
              FORGE_ERR_ALIGNMENT, "aux_loss is not 4-byte aligned");
  const Saved sv = saved_layout(*cfg);
  const Work wk = work_layout(*cfg);
  hipStream_t s = (hipStream_t)stream;
  uint16_t* a = at<uint16_t>(saved, sv.a);
  float* rstd1 = at<float>(saved, sv.rstd1);
  uint16_t* qkv = at<uint16_t>(saved, sv.qkv);
  uint16_t* h1 = at<uint16_t>(saved, sv.h1);
  float* rstd2 = at<float>(saved, sv.rstd2);
  uint16_t* bn = at<uint16_t>(saved, sv.b);
  uint16_t* o = cfg->recompute_attn ? at<uint16_t>(workspace, wk.o) : at<uint16_t>(saved, sv.o);
  float* lse = cfg->recompute_attn ? at<float>(workspace, wk.lse) : at<float>(saved, sv.lse);

  uint16_t* qk_raw = d.qkn ? at<uint16_t>(saved, sv.qk_raw) : nullptr;
  float* rstd_qk = d.qkn ? at<float>(saved, sv.rstd_qk) : nullptr;
  if (forge_status e =
          attn_block_fwd(*cfg, d, w, x_in, a, rstd1, qkv, o, lse, h1, qk_raw, rstd_qk, s))
    return e;
  FORGE_HIP(forge::rmsnorm_fwd(h1, w->ffn_norm, bn, rstd2, (int)d.T, (int)d.h, cfg->rms_eps, s));
  if (moe) return moe_ffn_fwd(*cfg, d, w, saved, sv, workspace, wk, h1, x_out, aux_loss, s);
  uint16_t* gu = at<uint16_t>(saved, sv.gu);
  uint16_t* act = at<uint16_t>(saved, sv.act);
  FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kStoreBF16,
                        gargs(bn, d.h, w->w_gate_up, d.h, gu, 2 * d.f, d.T, 2 * d.f, d.h), s));
  FORGE_HIP(forge::swiglu_fwd(gu, act, (int)d.T, (int)d.f, s));
  FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kResidBF16,
                        scaled(gargs(act, d.f, w->w_down, d.f, x_out, d.h, d.T, d.h, d.f, h1, d.h),
                               d.bs), s));
  return ok();
}

namespace {
forge_status check_layer_bwd_args(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                                  const void* saved, const forge_bf16* x_in,
                                  const forge_bf16* d_out, forge_bf16* d_in,
                                  const forge_layer_grads* g, void* workspace) {
  if (forge_status s = check_cfg(cfg)) return s;
  if (forge_status s = check_weights(*cfg, w)) return s;
  FORGE_PTR(saved);
  FORGE_PTR(x_in);
  FORGE_PTR(d_out);
  FORGE_PTR(d_in);
  FORGE_PTR(workspace);
  return check_grads(*cfg, g);
}

// The layer backward; with `opt` (dense layers) each weight's optimizer
// update is issued on the lane's optimizer stream as soon as it is final.
forge_status layer_bwd(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                       const void* saved, const forge_bf16* x_in, const forge_bf16* d_out,
                       forge_bf16* d_in, const forge_layer_grads* g, void* workspace,
                       hipStream_t s, OptPlan* opt) {
  const Dims d = dims(*cfg);
  const Saved sv = saved_layout(*cfg);
  const Work wk = work_layout(*cfg);
  const uint16_t* a = at<uint16_t>(saved, sv.a);
  const float* rstd1 = at<float>(saved, sv.rstd1);
  const uint16_t* qkv = at<uint16_t>(saved, sv.qkv);
  const uint16_t* h1 = at<uint16_t>(saved, sv.h1);
  const float* rstd2 = at<float>(saved, sv.rstd2);
  const uint16_t* bn = at<uint16_t>(saved, sv.b);
  const uint16_t* qk_raw = d.qkn ? at<uint16_t>(saved, sv.qk_raw) : nullptr;
  const float* rstd_qk = d.qkn ? at<float>(saved, sv.rstd_qk) : nullptr;
  uint16_t* db = at<uint16_t>(workspace, wk.db);
  uint16_t* dh1 = at<uint16_t>(workspace, wk.dh1);
  float* dgp = at<float>(workspace, wk.dg);
  const int nblk = forge::rmsnorm_bwd_blocks((int)d.T);

  const uint16_t* o;
  const float* lse;
  if (cfg->recompute_attn) {
    uint16_t* o_w = at<uint16_t>(workspace, wk.o);
    float* lse_w = at<float>(workspace, wk.lse);
    FORGE_HIP(forge::attn_fwd(attn_args(d, qkv), o_w, lse_w, s));
    o = o_w;
    lse = lse_w;
  } else {
    o = at<uint16_t>(saved, sv.o);
    lse = at<float>(saved, sv.lse);
  }

  // FFN branch: gradient at b, then RMSNorm backward plus the residual path
  if (d.E > 0) {
    // expert weight gradients on the side stream (updated in their
    // epilogues), beside the rest of the backward, whose attention weight
    // gradients go there too as in a dense layer
    SideLane* side = nullptr;
    if (use_side_streams(d)) FORGE_HIP(side_lane(&side));
    std::unique_lock<std::mutex> lk;
    if (side) lk = std::unique_lock<std::mutex>(side->mu);
    if (opt) opt->lane = side;
    if (forge_status e =
            moe_ffn_bwd(*cfg, d, w, g, saved, sv, workspace, wk, d_out, db, s, side, opt))
      return e;
    // the router weight is final: its update overlaps the rest
    if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->w_router, g->d_w_router, d.E * d.h));
    if (opt && d.fs) {
      hipStream_t ws = side ? side->stream : s;
      FORGE_HIP(opt_update(opt, s, ws, opt->o->w_down_s, g->d_w_down_s, d.h * d.fs));
      FORGE_HIP(opt_update(opt, s, ws, opt->o->w_gate_up_s, g->d_w_gate_up_s, 2 * d.fs * d.h));
    }
    FORGE_HIP(forge::rmsnorm_bwd(h1, w->ffn_norm, rstd2, db, d_out, dh1, dgp, (int)d.T, (int)d.h, s));
    FORGE_HIP(forge::rmsnorm_dg_reduce(dgp, nblk, g->d_ffn_norm, (int)d.h, !g->overwrite, s));
    if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->ffn_norm, g->d_ffn_norm, d.h));
    return attn_block_bwd(*cfg, d, w, g, x_in, a, rstd1, qkv, o, lse, qk_raw, rstd_qk, dh1, d_in,
                          workspace, wk, s, side, opt);
  } else {
    const uint16_t* gu = at<uint16_t>(saved, sv.gu);
    const uint16_t* act = at<uint16_t>(saved, sv.act);
    uint16_t* dA = at<uint16_t>(workspace, wk.dA);
    uint16_t* dgu = at<uint16_t>(workspace, wk.dgu);
    // weight gradients on the side stream (see SideLane): dW_down as soon
    // as the call starts, dW_gate_up once dgu exists
    // small layers stay on the caller's stream: there the event hand-offs
    // cost more than the overlap gains
    SideLane* side = nullptr;
    if (use_side_streams(d)) FORGE_HIP(side_lane(&side));
    std::unique_lock<std::mutex> lk;
    if (side) lk = std::unique_lock<std::mutex>(side->mu);
    hipStream_t ws = side ? side->stream : s;
    if (opt) opt->lane = side;
    if (side) FORGE_HIP(link(s, ws, side->ev[0]));
    FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                          scaled(gargs(d_out, d.h, act, d.f, g->d_w_down, d.f, d.h, d.f, d.T),
                                 d.bs), ws));
    // the weight-gradient product above is the side stream's only reader of
    // d_out; when d_in overlaps d_out, d_in is written only after it
    hipEvent_t d_out_read = nullptr;
    const bool alias = d_in < d_out + d.T * d.h && d_out < d_in + d.T * d.h;
    if (side && alias) {
      d_out_read = side->ev[5];
      FORGE_HIP(hipEventRecord(d_out_read, ws));
    }
    FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                          scaled(gargs(d_out, d.h, w->w_down, d.f, dA, d.f, d.T, d.f, d.h), d.bs),
                          s));
    FORGE_HIP(forge::swiglu_bwd(gu, dA, dgu, (int)d.T, (int)d.f, s));
    if (side) FORGE_HIP(link(s, ws, side->ev[1]));
    FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, wgrad_epi(g),
                          gargs(dgu, 2 * d.f, bn, d.h, g->d_w_gate_up, d.h, 2 * d.f, d.h, d.T), ws));
    FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                          gargs(dgu, 2 * d.f, w->w_gate_up, d.h, db, d.h, d.T, d.h, 2 * d.f), s));
    // separate updates (dense weights): they start once the gate/up data
    // gradient is done, beside the attention backward; updating in the
    // weight-gradient epilogue instead would order each weight-gradient
    // product after its data gradient and measured slower here
    if (opt) FORGE_HIP(opt_update(opt, s, ws, opt->o->w_down, g->d_w_down, d.h * d.f));
    if (opt) FORGE_HIP(opt_update(opt, s, ws, opt->o->w_gate_up, g->d_w_gate_up, 2 * d.f * d.h));
    FORGE_HIP(forge::rmsnorm_bwd(h1, w->ffn_norm, rstd2, db, d_out, dh1, dgp, (int)d.T, (int)d.h, s));
    FORGE_HIP(forge::rmsnorm_dg_reduce(dgp, nblk, g->d_ffn_norm, (int)d.h, !g->overwrite, s));
    if (opt) FORGE_HIP(opt_update(opt, s, s, opt->o->ffn_norm, g->d_ffn_norm, d.h));
    return attn_block_bwd(*cfg, d, w, g, x_in, a, rstd1, qkv, o, lse, qk_raw, rstd_qk, dh1, d_in,
                          workspace, wk, s, side, opt, d_out_read);
  }
}

// Per-weight optimizer state of the layer's weights: each used entry's
// buffers present and aligned, and param the very weight the layer reads.
forge_status check_optim(const forge_layer_cfg& c, const forge_layer_weights* w,
                         const forge_layer_optim* o) {
  FORGE_CHECK(o != nullptr, FORGE_ERR_INVALID_ARG, "opt is NULL");
  auto one = [&](const forge_adamw_tensor& t, const forge_bf16* weight,
                 const char* name) -> forge_status {
    FORGE_CHECK(t.master && t.param && t.m && t.v, FORGE_ERR_INVALID_ARG,
                "opt->%s has a NULL buffer", name);
    FORGE_CHECK(aligned16(t.master) && aligned16(t.param) && aligned16(t.m) && aligned16(t.v),
                FORGE_ERR_ALIGNMENT, "opt->%s has a buffer that is not 16-byte aligned", name);
    FORGE_CHECK(t.param == weight, FORGE_ERR_INVALID_ARG,
                "opt->%s.param must be the layer's %s weight pointer", name, name);
    return FORGE_OK;
  };
  if (forge_status e = one(o->attn_norm, w->attn_norm, "attn_norm")) return e;
  if (forge_status e = one(o->w_qkv, w->w_qkv, "w_qkv")) return e;
  if (forge_status e = one(o->w_o, w->w_o, "w_o")) return e;
  if (forge_status e = one(o->ffn_norm, w->ffn_norm, "ffn_norm")) return e;
  if (c.n_experts == 0) {
    if (forge_status e = one(o->w_gate_up, w->w_gate_up, "w_gate_up")) return e;
    if (forge_status e = one(o->w_down, w->w_down, "w_down")) return e;
  } else {
    if (forge_status e = one(o->w_router, w->w_router, "w_router")) return e;
    if (forge_status e = one(o->w_gate_up_e, w->w_gate_up_e, "w_gate_up_e")) return e;
    if (forge_status e = one(o->w_down_e, w->w_down_e, "w_down_e")) return e;
    if (c.shared_ffn > 0) {
      if (forge_status e = one(o->w_gate_up_s, w->w_gate_up_s, "w_gate_up_s")) return e;
      if (forge_status e = one(o->w_down_s, w->w_down_s, "w_down_s")) return e;
    }
  }
  if (c.qk_norm) {
    if (forge_status e = one(o->q_norm, w->q_norm, "q_norm")) return e;
    if (forge_status e = one(o->k_norm, w->k_norm, "k_norm")) return e;
  }
  return FORGE_OK;
}

forge_status check_hparams(const forge_adamw_hparams* hp) {
  FORGE_CHECK(hp != nullptr, FORGE_ERR_INVALID_ARG, "hparams is NULL");
  FORGE_CHECK(hp->beta1 >= 0.0f && hp->beta1 < 1.0f && hp->beta2 >= 0.0f && hp->beta2 < 1.0f,
              FORGE_ERR_INVALID_ARG, "betas must be in [0, 1)");
  FORGE_CHECK(hp->eps >= 0.0f && std::isfinite(hp->eps), FORGE_ERR_INVALID_ARG, "bad eps");
  FORGE_CHECK(std::isfinite(hp->weight_decay), FORGE_ERR_INVALID_ARG, "bad weight_decay");
  return FORGE_OK;
}
}  // namespace

forge_status forge_layer_bwd(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                             const void* saved, const forge_bf16* x_in,
                             const forge_bf16* d_out, forge_bf16* d_in,
                             const forge_layer_grads* g, void* workspace,
                             forge_stream stream) {
  if (forge_status e = check_layer_bwd_args(cfg, w, saved, x_in, d_out, d_in, g, workspace))
    return e;
  if (forge_status e = layer_bwd(cfg, w, saved, x_in, d_out, d_in, g, workspace,
                                 (hipStream_t)stream, nullptr))
    return e;
  return ok();
}

forge_status forge_layer_bwd_adamw(const forge_layer_cfg* cfg, const forge_layer_weights* w,
                                   const void* saved, const forge_bf16* x_in,
                                   const forge_bf16* d_out, forge_bf16* d_in,
                                   const forge_layer_grads* g, const forge_layer_optim* opt,
                                   const forge_adamw_hparams* hp, const float* dev_scalars,
                                   void* workspace, forge_stream stream) {
  if (forge_status e = check_layer_bwd_args(cfg, w, saved, x_in, d_out, d_in, g, workspace))
    return e;
  if (forge_status e = check_optim(*cfg, w, opt)) return e;
  if (forge_status e = check_hparams(hp)) return e;
  FORGE_PTR(dev_scalars);
  OptPlan plan{opt, hp, dev_scalars, nullptr, 7};
  if (forge_status e = layer_bwd(cfg, w, saved, x_in, d_out, d_in, g, workspace,
                                 (hipStream_t)stream, &plan))
    return e;
  return ok();
}

// ---- MoE routing building block -----------------------------------------------
namespace {
size_t route_ws_bytes(int32_t tokens, int32_t n_experts, int32_t top_k, size_t* pos_of_off) {
  const size_t hist = up((size_t)forge::moe_sort_blocks(tokens) * n_experts * 4);
  if (pos_of_off) *pos_of_off = hist;
  return hist + up((size_t)tokens * top_k * 4);
}
}  // namespace

forge_status forge_moe_route_workspace_bytes(int32_t tokens, int32_t n_experts, int32_t top_k,
                                             size_t* bytes) {
  FORGE_CHECK(tokens >= 1, FORGE_ERR_INVALID_ARG, "tokens must be >= 1");
  FORGE_CHECK(n_experts >= 1 && n_experts <= kMaxExperts, FORGE_ERR_UNSUPPORTED,
              "n_experts must be in [1, %d]", kMaxExperts);
  FORGE_CHECK(top_k >= 1 && top_k <= n_experts, FORGE_ERR_INVALID_ARG,
              "top_k must be in [1, n_experts]");
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = route_ws_bytes(tokens, n_experts, top_k, nullptr);
  return ok();
}

forge_status forge_moe_route(const float* logits, int32_t tokens, int32_t n_experts,
                             int32_t top_k, int32_t* idx, float* gates, float* probs,
                             int32_t* counts, int32_t* offsets, int32_t* perm, void* workspace,
                             forge_stream stream) {
  FORGE_CHECK(tokens >= 1, FORGE_ERR_INVALID_ARG, "tokens must be >= 1");
  FORGE_CHECK(n_experts >= 1 && n_experts <= kMaxExperts, FORGE_ERR_UNSUPPORTED,
              "n_experts must be in [1, %d]", kMaxExperts);
  FORGE_CHECK(top_k >= 1 && top_k <= n_experts, FORGE_ERR_INVALID_ARG,
              "top_k must be in [1, n_experts]");
  FORGE_CHECK((long)tokens * top_k < (1L << 31), FORGE_ERR_UNSUPPORTED, "tokens * top_k too large");
  for (const void* p : {(const void*)logits, (const void*)idx, (const void*)gates,
                        (const void*)probs, (const void*)counts, (const void*)offsets,
                        (const void*)perm, (const void*)workspace})
    FORGE_CHECK(p != nullptr && (reinterpret_cast<uintptr_t>(p) & 3u) == 0,
                FORGE_ERR_INVALID_ARG, "a pointer argument is NULL or not 4-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  size_t pos_off = 0;
  route_ws_bytes(tokens, n_experts, top_k, &pos_off);
  FORGE_HIP(forge::moe_route(logits, tokens, n_experts, top_k, idx, gates, probs, s));
  FORGE_HIP(forge::moe_sort(idx, tokens, n_experts, top_k, static_cast<int32_t*>(workspace),
                            counts, offsets, perm, at<int32_t>(workspace, pos_off), s));
  return ok();
}

// ---- MoE routing without a workspace argument -------------------------------
// The counting sort's scratch of forge_moe_route_noalloc (block histograms,
// then the inverse permutation) lives in this fixed device array, one copy
// per GPU for the life of the process. In host code its name is not a device
// address: each device's address comes from hipGetSymbolAddress, taken once
// per device with that device current, and only that address reaches the
// kernels.
namespace {
constexpr size_t kRouteScratchEntries = size_t(1) << 19;  // tokens * top_k
constexpr size_t kRouteScratchHist = size_t(1) << 17;     // sort blocks * n_experts
}  // namespace
static __device__ __align__(256) int32_t scratch[kRouteScratchHist + kRouteScratchEntries];

namespace {
int32_t* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;

hipError_t route_scratch(int32_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

forge_status forge_moe_route_noalloc(const float* logits, int32_t tokens, int32_t n_experts,
                                     int32_t top_k, int32_t* idx, float* gates, float* probs,
                                     int32_t* counts, int32_t* offsets, int32_t* perm,
                                     forge_stream stream) {
  FORGE_CHECK(tokens >= 1, FORGE_ERR_INVALID_ARG, "tokens must be >= 1");
  FORGE_CHECK(n_experts >= 1 && n_experts <= kMaxExperts, FORGE_ERR_UNSUPPORTED,
              "n_experts must be in [1, %d]", kMaxExperts);
  FORGE_CHECK(top_k >= 1 && top_k <= n_experts, FORGE_ERR_INVALID_ARG,
              "top_k must be in [1, n_experts]");
  FORGE_CHECK((size_t)tokens * top_k <= kRouteScratchEntries, FORGE_ERR_UNSUPPORTED,
              "tokens * top_k = %lld exceeds the fixed scratch limit %zu",
              (long long)tokens * top_k, kRouteScratchEntries);
  FORGE_CHECK((size_t)forge::moe_sort_blocks(tokens) * n_experts <= kRouteScratchHist,
              FORGE_ERR_UNSUPPORTED,
              "ceil(tokens / 128) * n_experts = %lld exceeds the fixed scratch limit %zu",
              (long long)forge::moe_sort_blocks(tokens) * n_experts, kRouteScratchHist);
  for (const void* p : {(const void*)logits, (const void*)idx, (const void*)gates,
                        (const void*)probs, (const void*)counts, (const void*)offsets,
                        (const void*)perm})
    FORGE_CHECK(p != nullptr && (reinterpret_cast<uintptr_t>(p) & 3u) == 0,
                FORGE_ERR_INVALID_ARG, "a pointer argument is NULL or not 4-byte aligned");
  int32_t* ws = nullptr;
  FORGE_HIP(route_scratch(&ws));
  hipStream_t s = (hipStream_t)stream;
  FORGE_HIP(forge::moe_route(logits, tokens, n_experts, top_k, idx, gates, probs, s));
  FORGE_HIP(forge::moe_sort(idx, tokens, n_experts, top_k, ws, counts, offsets, perm,
                            ws + kRouteScratchHist, s));
  return ok();
}

// ---- output head ----------------------------------------------------------
namespace {
struct HeadWork {
  size_t xn, rstd, z, row_loss, dxn, dg, total;
};
forge_status check_head(const forge_head_cfg* c) {
  FORGE_CHECK(c != nullptr, FORGE_ERR_INVALID_ARG, "cfg is NULL");
  FORGE_CHECK(c->tokens >= 1, FORGE_ERR_INVALID_ARG, "tokens must be >= 1");
  FORGE_CHECK(c->hidden >= 8 && c->hidden % 8 == 0 && c->hidden <= 8192, FORGE_ERR_INVALID_ARG,
              "hidden must be a multiple of 8 in [8, 8192] (got %d)", c->hidden);
  FORGE_CHECK(c->vocab >= 8 && c->vocab % 8 == 0, FORGE_ERR_INVALID_ARG,
              "vocab must be a positive multiple of 8 (got %d)", c->vocab);
  FORGE_CHECK((long)c->tokens * c->vocab < (1L << 31), FORGE_ERR_UNSUPPORTED,
              "tokens * vocab exceeds 2^31");
  FORGE_CHECK(std::isfinite(c->logit_scale) && c->logit_scale >= 0.0f, FORGE_ERR_INVALID_ARG,
              "logit_scale must be finite and >= 0 (0 means 1)");
  return FORGE_OK;
}
// zrows: rows of logits held at once (T, or the chunk of the streaming head)
HeadWork head_layout(const forge_head_cfg& c, long zrows) {
  HeadWork w;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += up(bytes); return o; };
  const long T = c.tokens, h = c.hidden, V = c.vocab;
  w.xn = take(T * h * 2);
  w.rstd = take(T * 4);
  w.z = take(zrows * V * 2);
  w.row_loss = take(T * 4);
  w.dxn = take(T * h * 2);
  w.dg = take((size_t)forge::rmsnorm_bwd_blocks((int)T) * h * 4);
  w.total = off;
  return w;
}
}  // namespace

forge_status forge_loss_workspace_bytes(const forge_head_cfg* cfg, size_t* bytes) {
  if (forge_status s = check_head(cfg)) return s;
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = head_layout(*cfg, cfg->tokens).total;
  return ok();
}

forge_status forge_loss_chunked_workspace_bytes(const forge_head_cfg* cfg, int32_t chunk,
                                                size_t* bytes) {
  if (forge_status s = check_head(cfg)) return s;
  FORGE_CHECK(chunk >= 1, FORGE_ERR_INVALID_ARG, "chunk must be >= 1");
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = head_layout(*cfg, std::min<long>(chunk, std::max(cfg->tokens, 1))).total;
  return ok();
}

namespace {
// The head over token chunks of `chunk` rows: per chunk the logits, the
// cross-entropy forward and backward in place, the input gradient rows and
// the chunk's share of dW_lm (fp32, accumulated); a chunk of T is the plain
// head.
forge_status loss_impl(const forge_head_cfg* cfg, long chunk, const forge_bf16* x_L,
                       const forge_bf16* final_norm, const forge_bf16* w_lm,
                       const int32_t* targets, float* loss_out, forge_bf16* d_x_L,
                       float* d_final_norm, float* d_w_lm, void* workspace,
                       forge_stream stream) {
  if (forge_status s = check_head(cfg)) return s;
  FORGE_PTR(x_L);
  FORGE_PTR(final_norm);
  FORGE_PTR(w_lm);
  FORGE_PTR(targets);
  FORGE_CHECK(loss_out != nullptr, FORGE_ERR_INVALID_ARG, "loss_out is NULL");
  FORGE_PTR(d_x_L);
  FORGE_PTR(d_final_norm);
  FORGE_PTR(d_w_lm);
  FORGE_PTR(workspace);
  const long T = cfg->tokens, h = cfg->hidden, V = cfg->vocab;
  chunk = std::min(chunk, std::max(T, 1L));
  const HeadWork hw = head_layout(*cfg, chunk);
  hipStream_t s = (hipStream_t)stream;
  uint16_t* xn = at<uint16_t>(workspace, hw.xn);
  float* rstd = at<float>(workspace, hw.rstd);
  uint16_t* z = at<uint16_t>(workspace, hw.z);
  float* rl = at<float>(workspace, hw.row_loss);
  uint16_t* dxn = at<uint16_t>(workspace, hw.dxn);
  float* dgp = at<float>(workspace, hw.dg);
  const int nblk = forge::rmsnorm_bwd_blocks((int)T);

  FORGE_HIP(forge::rmsnorm_fwd(x_L, final_norm, xn, rstd, (int)T, (int)h, cfg->rms_eps, s));
  for (long t0 = 0; t0 < T; t0 += chunk) {
    const long n = std::min(chunk, T - t0);
    const uint16_t* xc = xn + t0 * h;
    FORGE_HIP(forge::gemm(forge::kKC, forge::kKC, forge::kStoreBF16,
                          gargs(xc, h, w_lm, h, z, V, n, V, h), s));
    FORGE_HIP(forge::ce_fwd_bwd(z, targets + t0, rl + t0, (int)n, (int)V,
                                (float)(1.0 / (double)T),
                                cfg->logit_scale == 0.0f ? 1.0f : cfg->logit_scale, s));
    FORGE_HIP(forge::gemm(forge::kKC, forge::kMC, forge::kStoreBF16,
                          gargs(z, V, w_lm, h, dxn + t0 * h, h, n, h, V), s));
    FORGE_HIP(forge::gemm(forge::kMC, forge::kMC, forge::kAccF32,
                          gargs(z, V, xc, h, d_w_lm, h, V, h, n), s));
  }
  FORGE_HIP(forge::mean_reduce(rl, (int)T, (float)(1.0 / (double)T), loss_out, s));
  FORGE_HIP(forge::rmsnorm_bwd(x_L, final_norm, rstd, dxn, nullptr, d_x_L, dgp, (int)T, (int)h, s));
  FORGE_HIP(forge::rmsnorm_dg_reduce(dgp, nblk, d_final_norm, (int)h, true, s));
  return ok();
}
}  // namespace

forge_status forge_loss_fwd_bwd(const forge_head_cfg* cfg, const forge_bf16* x_L,
                                const forge_bf16* final_norm, const forge_bf16* w_lm,
                                const int32_t* targets, float* loss_out, forge_bf16* d_x_L,
                                float* d_final_norm, float* d_w_lm, void* workspace,
                                forge_stream stream) {
  FORGE_CHECK(cfg != nullptr, FORGE_ERR_INVALID_ARG, "cfg is NULL");
  return loss_impl(cfg, cfg->tokens, x_L, final_norm, w_lm, targets, loss_out, d_x_L,
                   d_final_norm, d_w_lm, workspace, stream);
}

forge_status forge_loss_fwd_bwd_chunked(const forge_head_cfg* cfg, int32_t chunk,
                                        const forge_bf16* x_L, const forge_bf16* final_norm,
                                        const forge_bf16* w_lm, const int32_t* targets,
                                        float* loss_out, forge_bf16* d_x_L,
                                        float* d_final_norm, float* d_w_lm, void* workspace,
                                        forge_stream stream) {
  FORGE_CHECK(chunk >= 1, FORGE_ERR_INVALID_ARG, "chunk must be >= 1");
  return loss_impl(cfg, chunk, x_L, final_norm, w_lm, targets, loss_out, d_x_L, d_final_norm,
                   d_w_lm, workspace, stream);
}

// ---- embedding --------------------------------------------------------------
forge_status forge_embed_fwd(const int32_t* ids, const forge_bf16* emb, forge_bf16* x0,
                             int32_t tokens, int32_t hidden, int32_t vocab, float scale,
                             forge_stream stream) {
  FORGE_CHECK(tokens >= 0 && vocab >= 1, FORGE_ERR_INVALID_ARG, "bad tokens/vocab");
  FORGE_CHECK(hidden >= 8 && hidden % 8 == 0, FORGE_ERR_INVALID_ARG,
              "hidden must be a positive multiple of 8");
  if (tokens == 0) return ok();
  FORGE_PTR(ids);
  FORGE_PTR(emb);
  FORGE_PTR(x0);
  FORGE_CHECK(std::isfinite(scale), FORGE_ERR_INVALID_ARG, "scale must be finite");
  FORGE_HIP(forge::embed_fwd(ids, emb, x0, tokens, hidden, vocab, scale, (hipStream_t)stream));
  return ok();
}

forge_status forge_embed_bwd(const int32_t* ids, const forge_bf16* dx0, float* d_emb,
                             int32_t tokens, int32_t hidden, int32_t vocab, float scale,
                             forge_stream stream) {
  FORGE_CHECK(tokens >= 0 && vocab >= 1, FORGE_ERR_INVALID_ARG, "bad tokens/vocab");
  FORGE_CHECK(hidden >= 8 && hidden % 8 == 0, FORGE_ERR_INVALID_ARG,
              "hidden must be a positive multiple of 8");
  if (tokens == 0) return ok();
  FORGE_PTR(ids);
  FORGE_PTR(dx0);
  FORGE_PTR(d_emb);
  FORGE_CHECK(std::isfinite(scale), FORGE_ERR_INVALID_ARG, "scale must be finite");
  FORGE_HIP(forge::embed_bwd(ids, dx0, d_emb, tokens, hidden, vocab, scale, (hipStream_t)stream));
  return ok();
}

// ---- optimizer ---------------------------------------------------------------
forge_status forge_adamw_step(float* master, forge_bf16* param, const float* grad, float* m,
                              float* v, int64_t n, const forge_adamw_hparams* hp,
                              const float* dev_scalars, forge_stream stream) {
  FORGE_CHECK(n >= 0, FORGE_ERR_INVALID_ARG, "n must be >= 0");
  if (forge_status e = check_hparams(hp)) return e;
  if (n == 0) return ok();
  FORGE_PTR(master);
  FORGE_PTR(param);
  FORGE_PTR(grad);
  FORGE_PTR(m);
  FORGE_PTR(v);
  FORGE_PTR(dev_scalars);
  FORGE_HIP(forge::adamw(master, param, grad, m, v, n, hp->beta1, hp->beta2, hp->eps,
                         hp->weight_decay, dev_scalars, (hipStream_t)stream));
  return ok();
}

forge_status forge_adamw_advance(float* dev_scalars, int32_t* dev_step, float lr, double beta1,
                                 double beta2, forge_stream stream) {
  FORGE_CHECK(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0,
              FORGE_ERR_INVALID_ARG, "betas must be in [0, 1)");
  FORGE_CHECK(std::isfinite(lr), FORGE_ERR_INVALID_ARG, "bad lr");
  FORGE_PTR(dev_scalars);
  FORGE_CHECK(dev_step != nullptr && (reinterpret_cast<uintptr_t>(dev_step) & 3u) == 0,
              FORGE_ERR_INVALID_ARG, "dev_step is NULL or not 4-byte aligned");
  FORGE_HIP(forge::adamw_advance(dev_scalars, dev_step, lr, beta1, beta2, (hipStream_t)stream));
  return ok();
}

forge_status forge_grad_norm_sq(const float* g, int64_t n, float* accum, float* workspace,
                                forge_stream stream) {
  FORGE_CHECK(n >= 0, FORGE_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return ok();
  FORGE_PTR(g);
  FORGE_CHECK(accum != nullptr, FORGE_ERR_INVALID_ARG, "accum is NULL");
  FORGE_PTR(workspace);
  hipStream_t s = (hipStream_t)stream;
  FORGE_HIP(forge::sumsq_partials(g, n, workspace, s));
  FORGE_HIP(forge::sumsq_finish(workspace, accum, s));
  return ok();
}

forge_status forge_clip_coeff(const float* norm_sq, float max_norm, float eps,
                              float* dev_scalars, forge_stream stream) {
  FORGE_CHECK(norm_sq != nullptr && dev_scalars != nullptr, FORGE_ERR_INVALID_ARG,
              "NULL pointer");
  FORGE_CHECK(max_norm > 0.0f && eps >= 0.0f, FORGE_ERR_INVALID_ARG,
              "max_norm must be > 0 and eps >= 0");
  FORGE_HIP(forge::clip_coeff(norm_sq, max_norm, eps, dev_scalars, (hipStream_t)stream));
  return ok();
}

// ---- building blocks --------------------------------------------------------
forge_status forge_gemm(int32_t layout_a, int32_t layout_b, int32_t epilogue,
                        const forge_bf16* A, const forge_bf16* B, void* C, const forge_bf16* R,
                        int32_t M, int32_t N, int32_t K, int64_t lda, int64_t ldb, int64_t ldc,
                        int64_t ldr, forge_stream stream) {
  FORGE_CHECK((layout_a == 0 || layout_a == 1) && (layout_b == 0 || layout_b == 1) &&
                  epilogue >= 0 && epilogue <= 3,
              FORGE_ERR_INVALID_ARG, "bad layout or epilogue code");
  const bool bf16_out = epilogue == FORGE_EPI_STORE_BF16 || epilogue == FORGE_EPI_RESID_BF16;
  const bool supported = (layout_a == 0 && layout_b == 0) ||
                         (layout_a == 0 && layout_b == 1 && bf16_out) ||
                         (layout_a == 1 && layout_b == 1 && !bf16_out);
  FORGE_CHECK(supported, FORGE_ERR_UNSUPPORTED, "layout/epilogue combination (%d,%d,%d)",
              layout_a, layout_b, epilogue);
  FORGE_CHECK(M >= 0 && N >= 0 && K >= 0, FORGE_ERR_INVALID_ARG, "negative size");
  if (M == 0 || N == 0) return ok();
  FORGE_PTR(C);
  if (K > 0) {
    FORGE_PTR(A);
    FORGE_PTR(B);
  }
  FORGE_CHECK(layout_a == 1 || K % 8 == 0, FORGE_ERR_INVALID_ARG, "K-contiguous A needs K %% 8 == 0");
  FORGE_CHECK(layout_b == 1 || K % 8 == 0, FORGE_ERR_INVALID_ARG, "K-contiguous B needs K %% 8 == 0");
  FORGE_CHECK(layout_a == 0 || M % 8 == 0, FORGE_ERR_INVALID_ARG, "M-contiguous A needs M %% 8 == 0");
  FORGE_CHECK(layout_b == 0 || N % 8 == 0, FORGE_ERR_INVALID_ARG, "N-contiguous B needs N %% 8 == 0");
  FORGE_CHECK(lda % 8 == 0 && ldb % 8 == 0 && ldc % 8 == 0, FORGE_ERR_INVALID_ARG,
              "leading dimensions must be multiples of 8");
  FORGE_CHECK(lda >= (layout_a == 0 ? K : M) && ldb >= (layout_b == 0 ? K : N) && ldc >= N,
              FORGE_ERR_INVALID_ARG, "leading dimension smaller than the contiguous extent");
  if (epilogue == FORGE_EPI_RESID_BF16) {
    FORGE_PTR(R);
    FORGE_CHECK(ldr % 8 == 0 && ldr >= N, FORGE_ERR_INVALID_ARG, "bad ldr");
    const char* c0 = static_cast<const char*>(C);
    const char* c1 = c0 + ((M - 1) * ldc + N) * 2;
    const char* r0 = reinterpret_cast<const char*>(R);
    const char* r1 = r0 + ((M - 1) * ldr + N) * 2;
    FORGE_CHECK(c1 <= r0 || r1 <= c0, FORGE_ERR_INVALID_ARG, "R overlaps C");
  }
  FORGE_CHECK((int64_t)M * ldc < (1LL << 40), FORGE_ERR_INVALID_ARG, "C too large");
  GemmArgs g = gargs(A, lda, B, ldb, C, ldc, M, N, K, R, ldr);
  FORGE_HIP(forge::gemm((forge::GemmLayout)layout_a, (forge::GemmLayout)layout_b,
                        (forge::GemmEpilogue)epilogue, g, (hipStream_t)stream));
  return ok();
}

forge_status forge_gemm_grouped_rows(int32_t layout_b, const forge_bf16* A, const forge_bf16* B,
                                     forge_bf16* C, const int32_t* offsets, int32_t groups,
                                     int32_t rows, int32_t N, int32_t K, int64_t lda,
                                     int64_t ldb, int64_t ldc, int64_t stride_b,
                                     forge_stream stream) {
  FORGE_CHECK(layout_b == FORGE_GEMM_KC || layout_b == FORGE_GEMM_MC, FORGE_ERR_INVALID_ARG,
              "bad layout_b");
  FORGE_CHECK(groups >= 0 && rows >= 0 && N >= 0 && K >= 0, FORGE_ERR_INVALID_ARG,
              "negative size");
  if (groups == 0 || rows == 0 || N == 0) return ok();
  FORGE_PTR(A);
  FORGE_PTR(B);
  FORGE_PTR(C);
  FORGE_PTR(offsets);
  FORGE_CHECK(K % 8 == 0, FORGE_ERR_INVALID_ARG, "K-contiguous A needs K %% 8 == 0");
  FORGE_CHECK(layout_b == FORGE_GEMM_MC || K > 0, FORGE_ERR_INVALID_ARG, "K must be > 0");
  FORGE_CHECK(layout_b == FORGE_GEMM_KC || N % 8 == 0, FORGE_ERR_INVALID_ARG,
              "N-contiguous B needs N %% 8 == 0");
  FORGE_CHECK(lda % 8 == 0 && ldb % 8 == 0 && ldc % 8 == 0 && stride_b % 8 == 0,
              FORGE_ERR_INVALID_ARG, "leading dimensions and stride_b must be multiples of 8");
  FORGE_CHECK(lda >= K && ldb >= (layout_b == FORGE_GEMM_KC ? K : N) && ldc >= N,
              FORGE_ERR_INVALID_ARG, "leading dimension smaller than the contiguous extent");
  FORGE_CHECK(stride_b >= 0, FORGE_ERR_INVALID_ARG, "negative stride_b");
  FORGE_CHECK((int64_t)rows * ldc < (1LL << 40) && (int64_t)rows * lda < (1LL << 40),
              FORGE_ERR_INVALID_ARG, "operand too large");
  GemmArgs g = grouped(gargs(A, lda, B, ldb, C, ldc, rows, N, K), offsets, groups, stride_b, 0);
  FORGE_HIP(forge::gemm_grouped_m((forge::GemmLayout)layout_b, forge::kStoreBF16, g,
                                  (hipStream_t)stream));
  return ok();
}

forge_status forge_gemm_grouped_wgrad(const forge_bf16* A, const forge_bf16* B, float* C,
                                      const int32_t* offsets, int32_t groups, int32_t M,
                                      int32_t N, int64_t lda, int64_t ldb, int64_t ldc,
                                      int64_t stride_c, forge_stream stream) {
  FORGE_CHECK(groups >= 0 && M >= 0 && N >= 0, FORGE_ERR_INVALID_ARG, "negative size");
  if (groups == 0 || M == 0 || N == 0) return ok();
  FORGE_PTR(A);
  FORGE_PTR(B);
  FORGE_PTR(C);
  FORGE_PTR(offsets);
  FORGE_CHECK(M % 8 == 0 && N % 8 == 0, FORGE_ERR_INVALID_ARG, "M and N must be multiples of 8");
  FORGE_CHECK(lda % 8 == 0 && ldb % 8 == 0 && ldc % 8 == 0 && stride_c % 8 == 0,
              FORGE_ERR_INVALID_ARG, "leading dimensions and stride_c must be multiples of 8");
  FORGE_CHECK(lda >= M && ldb >= N && ldc >= N, FORGE_ERR_INVALID_ARG,
              "leading dimension smaller than the contiguous extent");
  FORGE_CHECK(stride_c >= (int64_t)(M - 1) * ldc + N, FORGE_ERR_INVALID_ARG,
              "stride_c smaller than one group's output: groups would overlap");
  FORGE_CHECK((int64_t)groups * stride_c < (1LL << 40), FORGE_ERR_INVALID_ARG, "C too large");
  GemmArgs g = grouped(gargs(A, lda, B, ldb, C, ldc, M, N, 0), offsets, groups, 0, stride_c);
  FORGE_HIP(forge::gemm_grouped_k(forge::kAccF32, g, (hipStream_t)stream));
  return ok();
}

namespace {
forge_status check_attn(const forge_attn_cfg* c) {
  FORGE_CHECK(c != nullptr, FORGE_ERR_INVALID_ARG, "cfg is NULL");
  FORGE_CHECK(c->batch >= 1 && c->seq >= 1, FORGE_ERR_INVALID_ARG, "batch, seq must be >= 1");
  FORGE_CHECK(c->n_heads >= 1 && c->n_kv_heads >= 1 && c->n_heads % c->n_kv_heads == 0,
              FORGE_ERR_INVALID_ARG, "n_heads must be a positive multiple of n_kv_heads");
  FORGE_CHECK(c->head_dim == 64 || c->head_dim == 128, FORGE_ERR_UNSUPPORTED,
              "head_dim must be 64 or 128");
  return FORGE_OK;
}
Dims attn_dims(const forge_attn_cfg& c) {
  forge_layer_cfg l{};
  l.batch = c.batch;
  l.seq = c.seq;
  l.n_heads = c.n_heads;
  l.n_kv_heads = c.n_kv_heads;
  l.head_dim = c.head_dim;
  return dims(l);
}
}  // namespace

forge_status forge_attention_fwd(const forge_attn_cfg* cfg, const forge_bf16* qkv, forge_bf16* o,
                                 float* lse, forge_stream stream) {
  if (forge_status s = check_attn(cfg)) return s;
  FORGE_PTR(qkv);
  FORGE_PTR(o);
  FORGE_PTR(lse);
  const Dims d = attn_dims(*cfg);
  FORGE_HIP(forge::attn_fwd(attn_args(d, qkv), o, lse, (hipStream_t)stream));
  return ok();
}

forge_status forge_attention_bwd_workspace_bytes(const forge_attn_cfg* cfg, size_t* bytes) {
  if (forge_status s = check_attn(cfg)) return s;
  FORGE_CHECK(bytes != nullptr, FORGE_ERR_INVALID_ARG, "bytes is NULL");
  const Dims d = attn_dims(*cfg);
  *bytes = up(2 * (size_t)cfg->batch * cfg->n_heads * cfg->seq * 4) +
           up(forge::attn_bwd_ds_bytes(attn_args(d, nullptr)));
  return ok();
}

forge_status forge_attention_bwd(const forge_attn_cfg* cfg, const forge_bf16* qkv,
                                 const forge_bf16* o, const float* lse, const forge_bf16* d_o,
                                 forge_bf16* d_qkv, void* workspace, forge_stream stream) {
  if (forge_status s = check_attn(cfg)) return s;
  FORGE_PTR(qkv);
  FORGE_PTR(o);
  FORGE_PTR(lse);
  FORGE_PTR(d_o);
  FORGE_PTR(d_qkv);
  FORGE_PTR(workspace);
  const Dims d = attn_dims(*cfg);
  const forge::AttnArgs aa = attn_args(d, qkv);
  hipStream_t s = (hipStream_t)stream;
  float* delta = static_cast<float*>(workspace);
  uint16_t* ds = at<uint16_t>(workspace, up(2 * (size_t)cfg->batch * cfg->n_heads * cfg->seq * 4));
  FORGE_HIP(forge::attn_bwd(aa, o, d_o, lse, delta, ds, d_qkv, d_qkv + d.hq,
                            d_qkv + d.hq + d.hkv, d.qkv, s));
  return ok();
}

}  // extern "C"

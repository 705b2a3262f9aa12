// Internal launchers of libforge's gfx950 kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace forge {

// ---------------------------------------------------------------- GEMM ----
// C[m][n] (op)= sum_k A(m,k) B(k,n), bf16 operands, fp32 accumulation.
//   A layout KC: A(m,k) = A[m*lda + k]     MC: A(m,k) = A[k*lda + m]
//   B layout KC: B(k,n) = B[n*ldb + k]     MC: B(k,n) = B[k*ldb + n]
// so y = x W^T is (KC, KC), dX = dY W is (KC, MC), dW = dY^T X is (MC, MC).
enum GemmLayout { kKC = 0, kMC = 1 };
enum GemmEpilogue {
  kStoreBF16 = 0,     // C bf16 = acc
  kResidBF16 = 1,     // C bf16 = acc + R (bf16), one rounding
  kAccF32 = 2,        // C fp32 += acc
  kStoreF32 = 3,      // C fp32 = acc
  // weight gradient and its AdamW update in one epilogue (per-group weight
  // gradients, gemm_grouped_k): g = acc (kStoreF32Adam) or C + acc
  // (kAccF32Adam) is stored to C and then applied to the optimizer state at
  // the same position
  kStoreF32Adam = 4,
  kAccF32Adam = 5,
};

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  const uint16_t* R;
  int M, N, K;
  long lda, ldb, ldc, ldr;
  // every epilogue takes alpha * acc in place of acc (a residual branch's
  // scale, App. B muP); 1 leaves every result bit-identical
  float alpha = 1.0f;
  // grouped products (MoE experts): g_off[E + 1] device row offsets of the
  // groups; strideB / strideC elements between consecutive groups' B / C.
  const int* g_off = nullptr;
  int groups = 0;
  long strideB = 0, strideC = 0;
  // split last round (GEMM tile order 4): the full 256-wide tiles from this
  // one on in the band order, each run as two BN-wide halves
  int tile_base = 0;
  // AdamW epilogues: fp32 master, moments m and v and the bf16 parameter,
  // laid out like C (leading dimension ldc; grouped: strideC apart), device
  // step scalars {lr, 1 - b1^t, 1 - b2^t, clip} and the hyper-parameters
  float* o_master = nullptr;
  float* o_m = nullptr;
  float* o_v = nullptr;
  uint16_t* o_param = nullptr;
  const float* o_sc = nullptr;
  float o_b1 = 0.0f, o_b2 = 0.0f, o_eps = 0.0f, o_wd = 0.0f;
};

// Host-side shape rules (checked by the caller): K-contiguous operands need
// K % 8 == 0; M/N-contiguous operands need that dimension % 8 == 0; leading
// dimensions % 8 == 0; base pointers 16-byte aligned.
hipError_t gemm(GemmLayout la, GemmLayout lb, GemmEpilogue epi, const GemmArgs& a,
                hipStream_t stream);
// Grouped forms, one product per group e with rows [g_off[e], g_off[e+1]):
//   M-grouped (KC or MC B): C rows g_off[e].. = A rows g_off[e].. x B_e, where
//     B_e = B + e * strideB; M is an upper bound of the total rows (T * k).
//   K-grouped (MC, MC): C_e (+)= sum over rows g_off[e].. of A^T B, C_e = C + e * strideC.
hipError_t gemm_grouped_m(GemmLayout lb, GemmEpilogue epi, const GemmArgs& a, hipStream_t s);
hipError_t gemm_grouped_k(GemmEpilogue epi, const GemmArgs& a, hipStream_t s);
// Weight gradient C += A^T B (or C = A^T B when !accumulate), both operands
// M/N-contiguous, with the reduction split
// into `splits` uniform slices: fp32 partials [splits][M][N] in `partial`,
// then summed in slice order into C. For products with few output tiles and
// a long reduction (N % 4 == 0). splitk_splits picks the split count (1 =
// plain GEMM, no partials needed).
int splitk_splits(int M, int N, int K);
hipError_t gemm_wgrad_splitk(const GemmArgs& a, int splits, float* partial, bool accumulate,
                             hipStream_t s);

// --------------------------------------------------------- elementwise ----
hipError_t rmsnorm_fwd(const uint16_t* x, const uint16_t* g, uint16_t* y, float* rstd,
                       int T, int h, float eps, hipStream_t s);
// dx = RMSNorm backward (+ resid if non-null); dg_partial [nblk, h] per-block
// partial sums of dy*x*rstd, reduced into dg (+=, or = when !accumulate)
// by rmsnorm_dg_reduce.
int rmsnorm_bwd_blocks(int T);
hipError_t rmsnorm_bwd(const uint16_t* x, const uint16_t* g, const float* rstd,
                       const uint16_t* dy, const uint16_t* resid, uint16_t* dx,
                       float* dg_partial, int T, int h, hipStream_t s);
hipError_t rmsnorm_dg_reduce(const float* dg_partial, int nblk, float* dg, int h, bool accumulate,
                             hipStream_t s);
hipError_t rope_table(int seq, int d, float base, float* cos_t, float* sin_t,
                      hipStream_t s);
// pos: RoPE position of every token (NULL: index within its batch row).
hipError_t rope_apply(uint16_t* qkv, long row_stride, const float* cos_t,
                      const float* sin_t, const int32_t* pos, int T, int seq, int n_heads_rot,
                      int d, bool inverse, hipStream_t s);
// QK-Norm then RoPE on the nh q heads and nkv k heads of the qkv buffer, in
// place; raw [T, (nh + nkv) * d] keeps the un-normalised rows, rstd
// [T, nh + nkv] their rstd. The backward turns the post-RoPE gradient rows
// into the pre-norm gradient in place and writes gain-gradient partials
// [2][qknorm_bwd_blocks][d] (q, then k) for rmsnorm_dg_reduce.
hipError_t qknorm_rope_fwd(uint16_t* qkv, long ld, uint16_t* raw, float* rstd, const uint16_t* gq,
                           const uint16_t* gk, const float* cos_t, const float* sin_t,
                           const int32_t* pos, int T, int seq, int nh, int nkv, int d, float eps,
                           hipStream_t s);
int qknorm_bwd_blocks(int T, int nrot, int d);
hipError_t qknorm_rope_bwd(uint16_t* dqkv, long ld, const uint16_t* raw, const float* rstd,
                           const uint16_t* gq, const uint16_t* gk, const float* cos_t,
                           const float* sin_t, const int32_t* pos, int T, int seq, int nh, int nkv,
                           int d, float* dg_partial, hipStream_t s);
hipError_t swiglu_fwd(const uint16_t* gu, uint16_t* a, int T, int f, hipStream_t s);
hipError_t swiglu_bwd(const uint16_t* gu, const uint16_t* da, uint16_t* dgu, int T,
                      int f, hipStream_t s);
hipError_t embed_fwd(const int32_t* ids, const uint16_t* emb, uint16_t* x, int T,
                     int h, int V, float scale, hipStream_t s);
hipError_t embed_bwd(const int32_t* ids, const uint16_t* dx, float* demb, int T,
                     int h, int V, float scale, hipStream_t s);
// In place: z [T, V] bf16 logits -> dz = scale (softmax(scale z) - onehot)
// * inv_T; row_loss[t] of the scaled logits.
hipError_t ce_fwd_bwd(uint16_t* z, const int32_t* targets, float* row_loss, int T,
                      int V, float inv_T, float scale, hipStream_t s);
hipError_t mean_reduce(const float* v, int n, float scale, float* out, hipStream_t s);
hipError_t adamw(float* master, uint16_t* param, const float* grad, float* m, float* v,
                 int64_t n, float b1, float b2, float eps, float wd,
                 const float* scalars, hipStream_t s);
hipError_t adamw_advance(float* scalars, int32_t* step, float lr, double b1, double b2,
                         hipStream_t s);
constexpr int kNormPartials = 1024;
hipError_t sumsq_partials(const float* g, int64_t n, float* partials, hipStream_t s);
hipError_t sumsq_finish(const float* partials, float* accum, hipStream_t s);
hipError_t clip_coeff(const float* norm_sq, float max_norm, float eps, float* scalars,
                      hipStream_t s);

// ----------------------------------------------------------- attention ----
struct AttnArgs {
  const uint16_t* q;    // [T, *] rows, head n at column n*d, row stride ld_qkv
  const uint16_t* k;
  const uint16_t* v;
  long ld_qkv;
  int batch, seq, n_heads, n_kv_heads, d;
  float scale;          // 1/sqrt(d)
};
// o [T, n_heads*d] bf16; lse [batch, n_heads, seq] fp32 (natural log).
hipError_t attn_fwd(const AttnArgs& a, uint16_t* o, float* lse, hipStream_t s);
// Backward. delta: 2 * batch * n_heads * seq fp32 scratch ([b,n,i] =
// -sum_d dO*O, then [b,n,i] = -lse * log2(e)); ds: attn_bwd_ds_bytes scratch
// (dS in bf16, the causal half per (batch, head)). dq [T, n_heads*d] and
// dk, dv [T, n_kv*d] are column blocks of the dqkv buffer (row stride
// ld_dqkv); dk and dv hold each kv head's sums over its GQA group.
size_t attn_bwd_ds_bytes(const AttnArgs& a);
hipError_t attn_bwd(const AttnArgs& a, const uint16_t* o, const uint16_t* dout, const float* lse,
                    float* delta, uint16_t* ds, uint16_t* dq, uint16_t* dk, uint16_t* dv,
                    long ld_dqkv, hipStream_t s);

// ----------------------------------------------------------------- MoE ----
// Routing of fp32 logits [T, E] (E <= 256): idx / gates [T, k], probs [T, E];
// every idx entry lies in [0, E) (NaN logits rank below -inf).
hipError_t moe_route(const float* logits, int T, int E, int k, int32_t* idx, float* gates,
                     float* probs, hipStream_t s);
// Blocks of the counting sort; block_counts needs moe_sort_blocks(T) * E ints.
int moe_sort_blocks(int T);
// counts [E], offsets [E + 1], perm / pos_of [T k] (canonical order).
hipError_t moe_sort(const int32_t* idx, int T, int E, int k, int32_t* block_counts,
                    int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* pos_of,
                    hipStream_t s);
hipError_t moe_gather(const uint16_t* b, const int32_t* perm, long rows, int h, int k,
                      uint16_t* xs, hipStream_t s);
// out = h1 + scale * sum_j gate_j ys_j; backward with the same scale.
hipError_t moe_combine(const uint16_t* ys, const float* gates, const int32_t* pos_of,
                       const uint16_t* h1, long T, int h, int k, float scale, uint16_t* out,
                       hipStream_t s);
hipError_t moe_combine_bwd(const uint16_t* ys, const float* gates, const int32_t* pos_of,
                           const uint16_t* dy, long T, int h, int k, float scale, float* dgate,
                           uint16_t* dys, hipStream_t s);
hipError_t moe_scatter_back(const uint16_t* dxs, const int32_t* pos_of, long T, int h, int k,
                            uint16_t* db, hipStream_t s);
// colsum: E column sums followed by moe_aux_blocks(T) * E block partials.
int moe_aux_blocks(int T);
hipError_t moe_aux_loss(const float* probs, const int32_t* counts, int T, int E, int k,
                        float alpha, float* colsum, float* aux, hipStream_t s);
hipError_t moe_router_bwd(const float* probs, const int32_t* idx, const float* dgate,
                          const int32_t* counts, int T, int E, int k, float alpha, uint16_t* dl,
                          hipStream_t s);

}  // namespace forge

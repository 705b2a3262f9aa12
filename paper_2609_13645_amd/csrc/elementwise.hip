// HBM-bound kernels of the step: RMSNorm fwd/bwd, RoPE, SwiGLU fwd/bwd,
// embedding fwd/bwd, fused softmax cross-entropy, fused clip + AdamW + bf16
// write-back, gradient sum of squares and the device-side clip coefficient.
//
// Every kernel moves 16-byte vectors per lane (8 bf16 or 4 fp32) so each
// wave issues whole 1 KB coalesced transactions; row reductions stay inside
// one 64-lane wavefront (butterfly shuffles), and cross-row reductions
// (norm-gain gradients, loss mean, gradient norm) go through fixed-order
// partial sums so their results are deterministic.
#include "common.h"
#include "kernels.h"

namespace forge {
namespace {

constexpr int kRowsPerBlock = 4;  // forward: one wave per row, 4 waves per block
constexpr int kBwdWaves = 8;      // backward: 8 waves per block, rows strided over the grid
constexpr int kBwdMaxBlocks = 512;

// ------------------------------------------------------------- RMSNorm ----
// y = x * rstd * g with rstd = (mean(x^2) + eps)^(-1/2), fp32 math, one
// rounding to bf16 (App. B: pre-normalisation RMSNorm).
template <int MAXCH>
__global__ __launch_bounds__(256) void rmsnorm_fwd_k(const bf16_t* __restrict__ x,
                                                     const bf16_t* __restrict__ g,
                                                     bf16_t* __restrict__ y,
                                                     float* __restrict__ rstd, int T, int h,
                                                     float eps) {
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= T) return;
  const int nch = h / 8;
  const uint4* xr = reinterpret_cast<const uint4*>(x + row * h);
  uint4 v[MAXCH];
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = lane + i * 64;
    if (c < nch) {
      v[i] = xr[c];
      float f[8];
      unpack8(v[i], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += f[e] * f[e];
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)h + eps);
  if (lane == 0) rstd[row] = r;
  uint4* yr = reinterpret_cast<uint4*>(y + row * h);
  const uint4* gr = reinterpret_cast<const uint4*>(g);
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = lane + i * 64;
    if (c < nch) {
      float f[8], w[8];
      unpack8(v[i], f);
      unpack8(gr[c], w);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = f[e] * r * w[e];
      yr[c] = pack8(f);
    }
  }
}

// dx = r (g dy) - r^3 x sum(g dy x) / h  (+ resid);  per-block partial of
// dg = sum_rows dy x r, reduced across the block's waves through LDS.
template <int MAXCH>
__global__ __launch_bounds__(512) void rmsnorm_bwd_k(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ g,
    const float* __restrict__ rstd, const bf16_t* __restrict__ dy,
    const bf16_t* __restrict__ resid, bf16_t* __restrict__ dx,
    float* __restrict__ dg_partial, int T, int h) {
  __shared__ float red[kBwdWaves][512];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = h / 8;
  const uint4* gr = reinterpret_cast<const uint4*>(g);
  float dga[MAXCH][8];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) dga[i][e] = 0.0f;

  for (long row = (long)blockIdx.x * kBwdWaves + wave; row < T;
       row += (long)gridDim.x * kBwdWaves) {
    const uint4* xr = reinterpret_cast<const uint4*>(x + row * h);
    const uint4* dyr = reinterpret_cast<const uint4*>(dy + row * h);
    const uint4* rr = resid ? reinterpret_cast<const uint4*>(resid + row * h) : nullptr;
    const float r = rstd[row];
    uint4 xv[MAXCH], dv[MAXCH], rv[MAXCH];
    float dot = 0.0f;
    // the residual rows are loaded with x and dy, so their latency overlaps
    // the row's reduction
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = lane + i * 64;
      if (c < nch && rr) rv[i] = rr[c];
    }
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = lane + i * 64;
      if (c < nch) {
        xv[i] = xr[c];
        dv[i] = dyr[c];
        float xf[8], df[8], w[8];
        unpack8(xv[i], xf);
        unpack8(dv[i], df);
        unpack8(gr[c], w);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          dot += w[e] * df[e] * xf[e];
          dga[i][e] += df[e] * xf[e] * r;
        }
      }
    }
    dot = wave_sum(dot);
    const float coef = r * r * r * dot / (float)h;
    uint4* dxr = reinterpret_cast<uint4*>(dx + row * h);
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = lane + i * 64;
      if (c < nch) {
        float xf[8], df[8], w[8], o[8];
        unpack8(xv[i], xf);
        unpack8(dv[i], df);
        unpack8(gr[c], w);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = r * w[e] * df[e] - coef * xf[e];
        if (rr) {
          float rf[8];
          unpack8(rv[i], rf);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] += rf[e];
        }
        dxr[c] = pack8(o);
      }
    }
  }
  // block reduction of dg partials, 512 columns at a time
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][lane * 8 + e] = dga[i][e];
    __syncthreads();
    for (int j = threadIdx.x; j < 512; j += blockDim.x) {
      const int col = i * 512 + j;
      if (col < h) {
        float s = 0.0f;
#pragma unroll
        for (int w = 0; w < kBwdWaves; ++w) s += red[w][j];
        dg_partial[(long)blockIdx.x * h + col] = s;
      }
    }
    __syncthreads();
  }
}

// dg[c] += sum_b part[b][c]: a block covers 64 columns as 16 groups of four
// (16-byte loads); 16 stripes of threads each sum every 16th partial row,
// then the 16 stripe sums of a column are added in stripe order (fixed, so
// deterministic).
template <bool ACC>
__global__ __launch_bounds__(256) void dg_reduce_k(const float* __restrict__ part, int nblk,
                                                   float* __restrict__ dg, int h) {
  __shared__ float4 red[16][16];
  const int cg = threadIdx.x & 15, stripe = threadIdx.x >> 4;
  const int col = blockIdx.x * 64 + cg * 4;
  float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (col < h) {
#pragma unroll 8
    for (int b = stripe; b < nblk; b += 16) {
      const float4 v = *reinterpret_cast<const float4*>(part + (long)b * h + col);
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
  }
  red[stripe][cg] = s;
  __syncthreads();
  if (threadIdx.x < 64) {
    const int c = blockIdx.x * 64 + threadIdx.x;
    if (c < h) {
      const float* rf = reinterpret_cast<const float*>(&red[0][0]);
      float t = 0.0f;
#pragma unroll
      for (int w = 0; w < 16; ++w) t += rf[w * 64 + threadIdx.x];
      dg[c] = ACC ? dg[c] + t : t;
    }
  }
}

// ---------------------------------------------------------------- RoPE ----
// Rotate-half pairs (i, i + d/2) by angle pos * base^(-2i/d); pos restarts
// in each batch row. Table computed once in fp64, stored fp32.
__global__ void rope_table_k(int seq, int d, double base, float* cos_t, float* sin_t) {
  const int half = d / 2;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)seq * half) return;
  const int s = (int)(id / half), i = (int)(id % half);
  const double ang = (double)s * pow(base, -2.0 * (double)i / (double)d);
  cos_t[id] = (float)cos(ang);
  sin_t[id] = (float)sin(ang);
}

// RoPE position of token t: pos[t] (document-aware RoPE, App. A step 23;
// clamped to the table's seq rows) or, without pos, its index in its row.
__device__ __forceinline__ int rope_pos(const int32_t* pos, long t, int seq) {
  return pos ? min(max(pos[t], 0), seq - 1) : (int)(t % seq);
}

// One thread per (token, head, 8-pair chunk), in place.
__global__ void rope_apply_k(bf16_t* __restrict__ qkv, long ld, const float* __restrict__ cos_t,
                             const float* __restrict__ sin_t, const int32_t* __restrict__ pos,
                             int T, int seq, int nrot, int d, int inverse) {
  const int half = d / 2, cpr = half / 8;  // chunks per head
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)T * nrot * cpr) return;
  const int c = (int)(id % cpr);
  const long th = id / cpr;
  const int hd = (int)(th % nrot);
  const long t = th / nrot;
  const int s = rope_pos(pos, t, seq);
  bf16_t* base = qkv + t * ld + (long)hd * d + c * 8;
  uint4* p1 = reinterpret_cast<uint4*>(base);
  uint4* p2 = reinterpret_cast<uint4*>(base + half);
  const float4* cp = reinterpret_cast<const float4*>(cos_t + (long)s * half + c * 8);
  const float4* sp = reinterpret_cast<const float4*>(sin_t + (long)s * half + c * 8);
  float x1[8], x2[8];
  unpack8(*p1, x1);
  unpack8(*p2, x2);
  const float4 c0 = cp[0], c1 = cp[1], s0 = sp[0], s1 = sp[1];
  const float cs[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
  float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  if (inverse) {
#pragma unroll
    for (int e = 0; e < 8; ++e) sn[e] = -sn[e];
  }
  float y1[8], y2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    y1[e] = x1[e] * cs[e] - x2[e] * sn[e];
    y2[e] = x2[e] * cs[e] + x1[e] * sn[e];
  }
  *p1 = pack8(y1);
  *p2 = pack8(y2);
}

// ------------------------------------------------------ QK-Norm + RoPE ----
// Per-head RMSNorm of q and k over head_dim (gains gq / gk [d], shared by the
// heads; Qwen3's QK-Norm, App. B), then RoPE, in place on the qkv buffer.
// d / 8 lanes hold one (token, head) row, eight elements each; the row's sum
// of squares and the rotate-half partner (d / 16 lanes away) stay inside the
// wave. The forward keeps the un-normalised rows (raw [T, nrot * d]) and
// their rstd [T, nrot] for the backward.
template <int D>
__global__ __launch_bounds__(256) void qknorm_rope_fwd_k(
    bf16_t* __restrict__ qkv, long ld, bf16_t* __restrict__ raw, float* __restrict__ rstd,
    const bf16_t* __restrict__ gq, const bf16_t* __restrict__ gk,
    const float* __restrict__ cos_t, const float* __restrict__ sin_t,
    const int32_t* __restrict__ pos, int T, int seq, int nh, int nkv, float eps) {
  constexpr int LPR = D / 8, HALF = LPR / 2;
  const int nrot = nh + nkv;
  const long row = ((long)blockIdx.x * blockDim.x + threadIdx.x) / LPR;
  const int c = threadIdx.x % LPR;
  const bool ok = row < (long)T * nrot;
  const long t = ok ? row / nrot : 0;
  const int hd = ok ? (int)(row % nrot) : 0;
  bf16_t* xr = qkv + t * ld + (long)hd * D + c * 8;
  float x[8];
  uint4 xv = ok ? *reinterpret_cast<const uint4*>(xr) : make_uint4(0, 0, 0, 0);
  unpack8(xv, x);
  float ss = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) ss += x[e] * x[e];
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  const float r = 1.0f / sqrtf(ss / (float)D + eps);
  float g[8], y[8], yp[8];
  unpack8(*reinterpret_cast<const uint4*>((hd < nh ? gq : gk) + c * 8), g);
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = x[e] * r * g[e];
#pragma unroll
  for (int e = 0; e < 8; ++e) yp[e] = __shfl_xor(y[e], HALF, 64);
  const int s = rope_pos(pos, t, seq);
  const float* cp = cos_t + (long)s * (D / 2) + (c % HALF) * 8;
  const float* sp = sin_t + (long)s * (D / 2) + (c % HALF) * 8;
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e)
    o[e] = c < HALF ? y[e] * cp[e] - yp[e] * sp[e] : y[e] * cp[e] + yp[e] * sp[e];
  if (ok) {
    *reinterpret_cast<uint4*>(xr) = pack8(o);
    *reinterpret_cast<uint4*>(raw + (t * nrot + hd) * D + c * 8) = xv;
    if (c == 0) rstd[t * nrot + hd] = r;
  }
}

// Backward in place on the gradient rows: inverse rotation, then the RMSNorm
// backward dx = r (g dn) - x r^3 sum(g dn x) / d; the gain gradients
// sum_rows dn x r go to per-block partials [2][nblk][d] (q heads, then k
// heads), each block summing a fixed set of rows in a fixed order.
constexpr int kQkBlocks = 256;
template <int D>
__global__ __launch_bounds__(256) void qknorm_rope_bwd_k(
    bf16_t* __restrict__ dqkv, long ld, const bf16_t* __restrict__ raw,
    const float* __restrict__ rstd, const bf16_t* __restrict__ gq,
    const bf16_t* __restrict__ gk, const float* __restrict__ cos_t,
    const float* __restrict__ sin_t, const int32_t* __restrict__ pos, int T, int seq, int nh,
    int nkv, float* __restrict__ dg_partial) {
  constexpr int LPR = D / 8, HALF = LPR / 2, RPB = 256 / LPR;
  __shared__ float red[4][2][D];
  const int nrot = nh + nkv;
  const long nrows = (long)T * nrot;
  const int c = threadIdx.x % LPR;
  float accq[8], acck[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) accq[e] = acck[e] = 0.0f;
  for (long row0 = (long)blockIdx.x * RPB; row0 < nrows; row0 += (long)gridDim.x * RPB) {
    const long row = row0 + threadIdx.x / LPR;
    const bool ok = row < nrows;
    const long t = ok ? row / nrot : 0;
    const int hd = ok ? (int)(row % nrot) : 0;
    bf16_t* dr = dqkv + t * ld + (long)hd * D + c * 8;
    float dy[8], dp[8], x[8], g[8], dn[8];
    unpack8(ok ? *reinterpret_cast<const uint4*>(dr) : make_uint4(0, 0, 0, 0), dy);
    unpack8(ok ? *reinterpret_cast<const uint4*>(raw + row * D + c * 8) : make_uint4(0, 0, 0, 0), x);
    unpack8(*reinterpret_cast<const uint4*>((hd < nh ? gq : gk) + c * 8), g);
    const float r = ok ? rstd[row] : 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) dp[e] = __shfl_xor(dy[e], HALF, 64);
    const int s = rope_pos(pos, t, seq);
    const float* cp = cos_t + (long)s * (D / 2) + (c % HALF) * 8;
    const float* sp = sin_t + (long)s * (D / 2) + (c % HALF) * 8;
    float proj = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dn[e] = c < HALF ? dy[e] * cp[e] + dp[e] * sp[e] : dy[e] * cp[e] - dp[e] * sp[e];
      proj += dn[e] * g[e] * x[e];
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) proj += __shfl_xor(proj, o, 64);
    const float k3 = r * r * r * proj / (float)D;
    float dx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dx[e] = r * (dn[e] * g[e]) - x[e] * k3;
      const float dg = dn[e] * x[e] * r;
      if (hd < nh) accq[e] += dg;
      else acck[e] += dg;
    }
    if (ok) *reinterpret_cast<uint4*>(dr) = pack8(dx);
  }
  // lanes of one chunk c: fold within the wave, then the four waves in order
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      accq[e] += __shfl_xor(accq[e], o, 64);
      acck[e] += __shfl_xor(acck[e], o, 64);
    }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < LPR)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      red[wave][0][c * 8 + e] = accq[e];
      red[wave][1][c * 8 + e] = acck[e];
    }
  __syncthreads();
  for (int i = threadIdx.x; i < 2 * D; i += blockDim.x) {
    const int which = i / D, col = i % D;
    dg_partial[((long)which * gridDim.x + blockIdx.x) * D + col] =
        (red[0][which][col] + red[1][which][col]) + (red[2][which][col] + red[3][which][col]);
  }
}

// -------------------------------------------------------------- SwiGLU ----
__device__ __forceinline__ float sigmoidf_(float v) { return 1.0f / (1.0f + __expf(-v)); }

// A = silu(G) * U with G = gu[:, :f], U = gu[:, f:].
__global__ void swiglu_fwd_k(const bf16_t* __restrict__ gu, bf16_t* __restrict__ a, int T,
                             int f) {
  const int cpr = f / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  const uint4 gv = *reinterpret_cast<const uint4*>(gu + t * 2 * f + c * 8);
  const uint4 uv = *reinterpret_cast<const uint4*>(gu + t * 2 * f + f + c * 8);
  float G[8], U[8], o[8];
  unpack8(gv, G);
  unpack8(uv, U);
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = G[e] * sigmoidf_(G[e]) * U[e];
  *reinterpret_cast<uint4*>(a + t * f + c * 8) = pack8(o);
}

// dG = dA U s (1 + G (1 - s)), dU = dA G s, s = sigmoid(G).
__global__ void swiglu_bwd_k(const bf16_t* __restrict__ gu, const bf16_t* __restrict__ da,
                             bf16_t* __restrict__ dgu, int T, int f) {
  const int cpr = f / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  const uint4 gv = *reinterpret_cast<const uint4*>(gu + t * 2 * f + c * 8);
  const uint4 uv = *reinterpret_cast<const uint4*>(gu + t * 2 * f + f + c * 8);
  const uint4 dv = *reinterpret_cast<const uint4*>(da + t * f + c * 8);
  float G[8], U[8], D[8], dG[8], dU[8];
  unpack8(gv, G);
  unpack8(uv, U);
  unpack8(dv, D);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float s = sigmoidf_(G[e]);
    dG[e] = D[e] * U[e] * s * (1.0f + G[e] * (1.0f - s));
    dU[e] = D[e] * G[e] * s;
  }
  *reinterpret_cast<uint4*>(dgu + t * 2 * f + c * 8) = pack8(dG);
  *reinterpret_cast<uint4*>(dgu + t * 2 * f + f + c * 8) = pack8(dU);
}

// ----------------------------------------------------------- embedding ----
// x0 = scale * E[id] (scale: muP's scale_emb; 1 copies the row bit for bit)
__global__ void embed_fwd_k(const int32_t* __restrict__ ids, const bf16_t* __restrict__ emb,
                            bf16_t* __restrict__ x, int T, int h, int V, float scale) {
  const int cpr = h / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  const int v = ids[t];
  uint4 val = make_uint4(0, 0, 0, 0);
  if (v >= 0 && v < V) val = *reinterpret_cast<const uint4*>(emb + (long)v * h + c * 8);
  if (scale != 1.0f) {
    float f[8];
    unpack8(val, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] *= scale;
    val = pack8(f);
  }
  *reinterpret_cast<uint4*>(x + t * h + c * 8) = val;
}

__global__ void embed_bwd_k(const int32_t* __restrict__ ids, const bf16_t* __restrict__ dx,
                            float* __restrict__ demb, int T, int h, int V, float scale) {
  const int cpr = h / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= (long)T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  const int v = ids[t];
  if (v < 0 || v >= V) return;
  float f[8];
  unpack8(*reinterpret_cast<const uint4*>(dx + t * h + c * 8), f);
  float* dst = demb + (long)v * h + c * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) unsafeAtomicAdd(dst + e, f[e] * scale);
}

// ------------------------------------------------------- cross-entropy ----
// One block per row: online max / sum-exp in fp32 over the scaled logits
// u = scale * z (scale: muP's dim_model_base / hidden, 1 otherwise), then
// dz = scale * (exp(u - lse) - [j == y]) * inv_T written over the logits.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __expf(m - mn) + s2 * __expf(m2 - mn);
  m = mn;
}

__global__ __launch_bounds__(256) void ce_k(bf16_t* __restrict__ z,
                                            const int32_t* __restrict__ targets,
                                            float* __restrict__ row_loss, int V, float inv_T,
                                            float scale) {
  __shared__ float sm[4], ss[4];
  const long row = blockIdx.x;
  bf16_t* zr = z + row * V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = V / 8;
  float m = -INFINITY, s = 0.0f;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    float f[8];
    unpack8(*reinterpret_cast<const uint4*>(zr + c * 8), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] *= scale;
    float cm = f[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) cm = fmaxf(cm, f[e]);
    float cs = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) cs += __expf(f[e] - cm);
    lse_merge(m, s, cm, cs);
  }
  for (int j = nch * 8 + threadIdx.x; j < V; j += blockDim.x)
    lse_merge(m, s, bf2f(zr[j]) * scale, 1.0f);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(s, o, 64);
    lse_merge(m, s, m2, s2);
  }
  if (lane == 0) { sm[wave] = m; ss[wave] = s; }
  __syncthreads();
  m = sm[0];
  s = ss[0];
  for (int w = 1; w < 4; ++w) lse_merge(m, s, sm[w], ss[w]);
  const float lse = m + __logf(s);
  const int y = targets[row];
  const bool ok = (y >= 0 && y < V);
  if (threadIdx.x == 0) row_loss[row] = ok ? lse - bf2f(zr[y]) * scale : __builtin_nanf("");
  __syncthreads();  // z[y] read before it is overwritten
  const float gs = inv_T * scale;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    float f[8];
    unpack8(*reinterpret_cast<const uint4*>(zr + c * 8), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = c * 8 + e;
      f[e] = (__expf(f[e] * scale - lse) - (j == y ? 1.0f : 0.0f)) * gs;
    }
    *reinterpret_cast<uint4*>(zr + c * 8) = pack8(f);
  }
  for (int j = nch * 8 + threadIdx.x; j < V; j += blockDim.x)
    zr[j] = f2bf((__expf(bf2f(zr[j]) * scale - lse) - (j == y ? 1.0f : 0.0f)) * gs);
}

// out = scale * sum(v), one block, fixed order.
__global__ __launch_bounds__(1024) void mean_reduce_k(const float* __restrict__ v, int n,
                                                      float scale, float* __restrict__ out) {
  __shared__ float red[16];
  float s = 0.0f;
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += v[i];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w];
    *out = t * scale;
  }
}

// --------------------------------------------------------------- AdamW ----
// adam1 (the per-element update, App. F) lives in common.h: the fused
// weight-gradient epilogue of the GEMM applies the same arithmetic.

// One float4 of parameters per thread and no grid-stride loop: with seven
// streams (read g, p, m, v; write p, m, v and bf16 p) this keeps the most
// independent 16-byte requests in flight. Every stream is touched once, so
// the accesses are nontemporal (no cache allocation): ~8 % faster than
// plain loads and stores on this chip, at copy bandwidth.
__global__ __launch_bounds__(256) void adamw_k(float* __restrict__ master,
                                               bf16_t* __restrict__ param,
                                               const float* __restrict__ grad,
                                               float* __restrict__ mom1,
                                               float* __restrict__ mom2, int64_t n, float b1,
                                               float b2, float eps, float wd,
                                               const float* __restrict__ sc) {
  const float lr = sc[0], ibc1 = 1.0f / sc[1], ibc2 = 1.0f / sc[2], clip = sc[3];
  const int64_t n4 = n / 4;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n4) {
    f32x4_t p = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(master) + i);
    f32x4_t m = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(mom1) + i);
    f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(mom2) + i);
    const f32x4_t g = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(grad) + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float pe = p[e], me = m[e], ve = v[e];
      adam1(pe, me, ve, g[e], b1, b2, eps, wd, lr, ibc1, ibc2, clip);
      p[e] = pe;
      m[e] = me;
      v[e] = ve;
    }
    __builtin_nontemporal_store(p, reinterpret_cast<f32x4_t*>(master) + i);
    __builtin_nontemporal_store(m, reinterpret_cast<f32x4_t*>(mom1) + i);
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(mom2) + i);
    const u32x2_t pb = {pack2(p[0], p[1]), pack2(p[2], p[3])};
    __builtin_nontemporal_store(pb, reinterpret_cast<u32x2_t*>(param) + i);
  } else if (i < n4 + (n - n4 * 4)) {
    // tail: the last n % 4 elements, one per thread
    const int64_t e = n4 * 4 + (i - n4);
    float p = master[e], m = mom1[e], v = mom2[e];
    adam1(p, m, v, grad[e], b1, b2, eps, wd, lr, ibc1, ibc2, clip);
    master[e] = p;
    mom1[e] = m;
    mom2[e] = v;
    param[e] = f2bf(p);
  }
}

// Step scalars of the next AdamW update, kept on the device: t = ++step;
// {lr, 1 - b1^t, 1 - b2^t} into sc[0..2] (betas and powers in fp64, then
// rounded to fp32); sc[3], the clip coefficient, is left as it is. One thread.
__global__ void adamw_advance_k(float* __restrict__ sc, int32_t* __restrict__ step, float lr,
                                double b1, double b2) {
  if (threadIdx.x != 0) return;
  const int32_t t = step[0] + 1;
  step[0] = t;
  sc[0] = lr;
  sc[1] = (float)(1.0 - pow(b1, (double)t));
  sc[2] = (float)(1.0 - pow(b2, (double)t));
}

// ------------------------------------------------ gradient norm, clip ----
// Block b sums the squares of its fixed contiguous slice; then one block
// adds the partials in a fixed tree order.
__global__ __launch_bounds__(256) void sumsq_partials_k(const float* __restrict__ g, int64_t n,
                                                        float* __restrict__ partials) {
  __shared__ float red[4];
  const int64_t per = ((n + gridDim.x - 1) / gridDim.x + 3) / 4 * 4;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  float s = 0.0f;
  if (lo < hi) {
    const int64_t nv = (hi - lo) / 4;
    const float4* g4 = reinterpret_cast<const float4*>(g + lo);
    for (int64_t i = threadIdx.x; i < nv; i += blockDim.x) {
      const float4 x = g4[i];
      s += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    }
    for (int64_t i = lo + nv * 4 + threadIdx.x; i < hi; i += blockDim.x) s += g[i] * g[i];
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) partials[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(1024) void sumsq_finish_k(const float* __restrict__ partials,
                                                       float* __restrict__ accum) {
  __shared__ float red[16];
  float s = partials[threadIdx.x];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int w = 0; w < 16; ++w) t += red[w];
    accum[0] += t;
  }
}

__global__ void clip_coeff_k(const float* __restrict__ nsq, float max_norm, float eps,
                             float* __restrict__ sc) {
  const float norm = sqrtf(fmaxf(nsq[0], 0.0f));
  sc[3] = fminf(1.0f, max_norm / (norm + eps));
}

inline unsigned blocks_for(long work, int threads) {
  return (unsigned)((work + threads - 1) / threads);
}

}  // namespace

// ------------------------------------------------------------ launchers ----
hipError_t rmsnorm_fwd(const uint16_t* x, const uint16_t* g, uint16_t* y, float* rstd, int T,
                       int h, float eps, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const dim3 grid(blocks_for(T, kRowsPerBlock)), block(256);
  const int ch = (h / 8 + 63) / 64;
  if (ch <= 1) hipLaunchKernelGGL(rmsnorm_fwd_k<1>, grid, block, 0, s, x, g, y, rstd, T, h, eps);
  else if (ch <= 2) hipLaunchKernelGGL(rmsnorm_fwd_k<2>, grid, block, 0, s, x, g, y, rstd, T, h, eps);
  else if (ch <= 4) hipLaunchKernelGGL(rmsnorm_fwd_k<4>, grid, block, 0, s, x, g, y, rstd, T, h, eps);
  else if (ch <= 8) hipLaunchKernelGGL(rmsnorm_fwd_k<8>, grid, block, 0, s, x, g, y, rstd, T, h, eps);
  else if (ch <= 16) hipLaunchKernelGGL(rmsnorm_fwd_k<16>, grid, block, 0, s, x, g, y, rstd, T, h, eps);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

int rmsnorm_bwd_blocks(int T) {
  const int need = (T + kBwdWaves - 1) / kBwdWaves;
  return need < kBwdMaxBlocks ? (need > 0 ? need : 1) : kBwdMaxBlocks;
}

hipError_t rmsnorm_bwd(const uint16_t* x, const uint16_t* g, const float* rstd,
                       const uint16_t* dy, const uint16_t* resid, uint16_t* dx, float* dg_partial,
                       int T, int h, hipStream_t s) {
  const dim3 grid(rmsnorm_bwd_blocks(T)), block(64 * kBwdWaves);
  const int ch = (h / 8 + 63) / 64;
#define FORGE_RMSB(N) hipLaunchKernelGGL(rmsnorm_bwd_k<N>, grid, block, 0, s, x, g, rstd, dy, resid, dx, dg_partial, T, h)
  if (ch <= 1) FORGE_RMSB(1);
  else if (ch <= 2) FORGE_RMSB(2);
  else if (ch <= 4) FORGE_RMSB(4);
  else if (ch <= 8) FORGE_RMSB(8);
  else if (ch <= 16) FORGE_RMSB(16);
  else return hipErrorInvalidValue;
#undef FORGE_RMSB
  return hipGetLastError();
}

hipError_t rmsnorm_dg_reduce(const float* dg_partial, int nblk, float* dg, int h, bool accumulate,
                             hipStream_t s) {
  if (accumulate)
    hipLaunchKernelGGL(dg_reduce_k<true>, dim3(blocks_for(h, 64)), dim3(256), 0, s, dg_partial, nblk, dg, h);
  else
    hipLaunchKernelGGL(dg_reduce_k<false>, dim3(blocks_for(h, 64)), dim3(256), 0, s, dg_partial, nblk, dg, h);
  return hipGetLastError();
}

hipError_t rope_table(int seq, int d, float base, float* cos_t, float* sin_t, hipStream_t s) {
  const long n = (long)seq * (d / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, seq, d,
                     (double)base, cos_t, sin_t);
  return hipGetLastError();
}

hipError_t rope_apply(uint16_t* qkv, long ld, const float* cos_t, const float* sin_t,
                      const int32_t* pos, int T, int seq, int nrot, int d, bool inverse,
                      hipStream_t s) {
  const long n = (long)T * nrot * (d / 16);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_apply_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, qkv, ld, cos_t,
                     sin_t, pos, T, seq, nrot, d, inverse ? 1 : 0);
  return hipGetLastError();
}

hipError_t qknorm_rope_fwd(uint16_t* qkv, long ld, uint16_t* raw, float* rstd, const uint16_t* gq,
                           const uint16_t* gk, const float* cos_t, const float* sin_t,
                           const int32_t* pos, int T, int seq, int nh, int nkv, int d, float eps,
                           hipStream_t s) {
  const long n = (long)T * (nh + nkv) * (d / 8);
  if (n == 0) return hipSuccess;
  if (d == 128)
    hipLaunchKernelGGL(qknorm_rope_fwd_k<128>, dim3(blocks_for(n, 256)), dim3(256), 0, s, qkv, ld,
                       raw, rstd, gq, gk, cos_t, sin_t, pos, T, seq, nh, nkv, eps);
  else if (d == 64)
    hipLaunchKernelGGL(qknorm_rope_fwd_k<64>, dim3(blocks_for(n, 256)), dim3(256), 0, s, qkv, ld,
                       raw, rstd, gq, gk, cos_t, sin_t, pos, T, seq, nh, nkv, eps);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

int qknorm_bwd_blocks(int T, int nrot, int d) {
  const long rows = (long)T * nrot, rpb = 256 / (d / 8);
  const long b = (rows + rpb - 1) / rpb;
  return (int)(b < kQkBlocks ? b : kQkBlocks);
}

hipError_t qknorm_rope_bwd(uint16_t* dqkv, long ld, const uint16_t* raw, const float* rstd,
                           const uint16_t* gq, const uint16_t* gk, const float* cos_t,
                           const float* sin_t, const int32_t* pos, int T, int seq, int nh, int nkv,
                           int d, float* dg_partial, hipStream_t s) {
  const int nb = qknorm_bwd_blocks(T, nh + nkv, d);
  if (d == 128)
    hipLaunchKernelGGL(qknorm_rope_bwd_k<128>, dim3(nb), dim3(256), 0, s, dqkv, ld, raw, rstd, gq,
                       gk, cos_t, sin_t, pos, T, seq, nh, nkv, dg_partial);
  else if (d == 64)
    hipLaunchKernelGGL(qknorm_rope_bwd_k<64>, dim3(nb), dim3(256), 0, s, dqkv, ld, raw, rstd, gq,
                       gk, cos_t, sin_t, pos, T, seq, nh, nkv, dg_partial);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t swiglu_fwd(const uint16_t* gu, uint16_t* a, int T, int f, hipStream_t s) {
  const long n = (long)T * (f / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_fwd_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, gu, a, T, f);
  return hipGetLastError();
}

hipError_t swiglu_bwd(const uint16_t* gu, const uint16_t* da, uint16_t* dgu, int T, int f,
                      hipStream_t s) {
  const long n = (long)T * (f / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_bwd_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, gu, da, dgu, T, f);
  return hipGetLastError();
}

hipError_t embed_fwd(const int32_t* ids, const uint16_t* emb, uint16_t* x, int T, int h, int V,
                     float scale, hipStream_t s) {
  const long n = (long)T * (h / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_fwd_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, ids, emb, x, T, h, V,
                     scale);
  return hipGetLastError();
}

hipError_t embed_bwd(const int32_t* ids, const uint16_t* dx, float* demb, int T, int h, int V,
                     float scale, hipStream_t s) {
  const long n = (long)T * (h / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_bwd_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, ids, dx, demb, T, h, V,
                     scale);
  return hipGetLastError();
}

hipError_t ce_fwd_bwd(uint16_t* z, const int32_t* targets, float* row_loss, int T, int V,
                      float inv_T, float scale, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(ce_k, dim3(T), dim3(256), 0, s, z, targets, row_loss, V, inv_T, scale);
  return hipGetLastError();
}

hipError_t mean_reduce(const float* v, int n, float scale, float* out, hipStream_t s) {
  hipLaunchKernelGGL(mean_reduce_k, dim3(1), dim3(1024), 0, s, v, n, scale, out);
  return hipGetLastError();
}

hipError_t adamw(float* master, uint16_t* param, const float* grad, float* m, float* v,
                 int64_t n, float b1, float b2, float eps, float wd, const float* sc,
                 hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t work = n / 4 + (n % 4);
  const int64_t blocks = (work + 255) / 256;
  hipLaunchKernelGGL(adamw_k, dim3((unsigned)blocks), dim3(256), 0, s, master, param, grad, m, v,
                     n, b1, b2, eps, wd, sc);
  return hipGetLastError();
}

hipError_t adamw_advance(float* sc, int32_t* step, float lr, double b1, double b2, hipStream_t s) {
  hipLaunchKernelGGL(adamw_advance_k, dim3(1), dim3(64), 0, s, sc, step, lr, b1, b2);
  return hipGetLastError();
}

hipError_t sumsq_partials(const float* g, int64_t n, float* partials, hipStream_t s) {
  hipLaunchKernelGGL(sumsq_partials_k, dim3(kNormPartials), dim3(256), 0, s, g, n, partials);
  return hipGetLastError();
}

hipError_t sumsq_finish(const float* partials, float* accum, hipStream_t s) {
  hipLaunchKernelGGL(sumsq_finish_k, dim3(1), dim3(kNormPartials), 0, s, partials, accum);
  return hipGetLastError();
}

hipError_t clip_coeff(const float* norm_sq, float max_norm, float eps, float* sc, hipStream_t s) {
  hipLaunchKernelGGL(clip_coeff_k, dim3(1), dim3(1), 0, s, norm_sq, max_norm, eps, sc);
  return hipGetLastError();
}

}  // namespace forge

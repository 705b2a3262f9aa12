// Causal grouped-query flash attention on gfx950 MFMA: forward, and the
// backward as a pre-pass (delta = rowsum(dO * O)) plus two kernels, one that
// owns a key tile and accumulates dK, dV over the queries of its whole GQA
// group, and one that owns a query tile and accumulates dQ over keys. The
// paper's H100 kernel accumulates dQ through a flat global buffer (App. D,
// "Anatomy of a Forged Kernel"); on MI355X the separate dQ kernel costs two
// recomputed products but no fp32 atomics and keeps every output
// deterministic.
//
// Operand layout. The 32x32x16 MFMA gives each lane one column of its 32x32
// result and sixteen rows. Scores are formed with the lane-owned index on the
// column:
//   * forward / dQ: S^T = K Q^T (lane owns a query), so the softmax row
//     statistics, the LSE and delta are lane-local and O^T = V^T P^T,
//     dQ^T = K^T dS^T take P^T / dS^T straight from the accumulators;
//   * dK/dV: S = Q K^T (lane owns a key), so dV^T = dO^T P and dK^T = Q^T dS
//     take P / dS straight from the accumulators.
// Accumulator rows come in groups of four, so the reduction index of those
// register-sourced operands is permuted; the LDS copies of V^T, K^T, Q^T and
// dO^T are stored with the same permutation of their key / query index (each
// 16-byte LDS chunk holds keys {4h..4h+3, 8+4h..8+4h+3} of a 16-key group), so
// every MFMA operand is one 16-byte LDS read. Transposed copies are made in
// registers (8x8 blocks) from the same coalesced loads as the natural copies.
//
// Online softmax runs in the log2 domain (scale * log2 e folded into one
// multiply); the causal mask is only evaluated on tiles that straddle the
// diagonal, and waves whose rows are fully masked skip their MFMAs.
#include "common.h"
#include "kernels.h"

namespace forge {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// [64 rows][D] tile, row-contiguous along D, chunk-swizzled.
template <int D>
__device__ __forceinline__ int nat_idx(int row, int c) {
  constexpr int CPR = D / 8;
  return row * CPR + (c ^ (row & (CPR - 1)));
}
// [D rows][64] tile of a transposed operand: 8 chunks per row, permuted
// 4+4 index order inside each 16-group, chunk-swizzled.
__device__ __forceinline__ int tr_idx(int row, int pc) {
  return row * 8 + (pc ^ ((row ^ (row >> 3)) & 7));
}

__device__ __forceinline__ void load_blk(const bf16_t* __restrict__ base, long ld, int row0,
                                         int lim, int cg, uint4* r) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = row0 + i;
    r[i] = row < lim ? *reinterpret_cast<const uint4*>(base + (long)row * ld + cg * 8)
                     : make_uint4(0, 0, 0, 0);
  }
}

template <int D>
__device__ __forceinline__ void store_nat(uint4* lds, int rg, int cg, const uint4* r) {
#pragma unroll
  for (int i = 0; i < 8; ++i) lds[nat_idx<D>(rg * 8 + i, cg)] = r[i];
}

// Block (rg, cg) of a [64][D] tile -> rows cg*8..+7 of the [D][64] permuted copy.
__device__ __forceinline__ void store_tr(uint4* lds, int rg, int cg, const uint4* r) {
  uint4 t[8];
  transpose8x8(r, t);
  const int a = rg >> 1, odd = rg & 1;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int row = cg * 8 + c;
    uint2* p0 = reinterpret_cast<uint2*>(lds + tr_idx(row, 2 * a)) + odd;
    uint2* p1 = reinterpret_cast<uint2*>(lds + tr_idx(row, 2 * a + 1)) + odd;
    *p0 = make_uint2(t[c].x, t[c].y);
    *p1 = make_uint2(t[c].z, t[c].w);
  }
}

__device__ __forceinline__ bf16x8_t pack_frag(const f32x16_t& v, int s) {
  uint4 u = make_uint4(pack2(v[8 * s + 0], v[8 * s + 1]), pack2(v[8 * s + 2], v[8 * s + 3]),
                       pack2(v[8 * s + 4], v[8 * s + 5]), pack2(v[8 * s + 6], v[8 * s + 7]));
  return __builtin_bit_cast(bf16x8_t, u);
}

__device__ __forceinline__ bf16x8_t ld_frag(const uint4* p) {
  return __builtin_bit_cast(bf16x8_t, *p);
}

__device__ __forceinline__ bf16x8_t gload_frag(const bf16_t* p, bool ok) {
  return __builtin_bit_cast(bf16x8_t, ok ? *reinterpret_cast<const uint4*>(p)
                                         : make_uint4(0, 0, 0, 0));
}

__device__ __forceinline__ void zero(f32x16_t& a) {
#pragma unroll
  for (int e = 0; e < 16; ++e) a[e] = 0.0f;
}

// ------------------------------------------------------------- forward ----
// Block: 128 queries (32 per wave) of one (batch, head); key tiles of 64.
template <int D>
__global__ __launch_bounds__(256, 1) void attn_fwd_k(AttnArgs a, bf16_t* __restrict__ o,
                                                     float* __restrict__ lse) {
  constexpr int BQ = 128, BKV = 64, CPR = D / 8;
  constexpr int NAT = BKV * CPR, TRN = D * 8, NBLK = 8 * CPR;
  __shared__ uint4 smem[2][NAT + TRN];

  const int S = a.seq;
  const int nqt = (S + BQ - 1) / BQ;
  const int qt = nqt - 1 - (int)blockIdx.x;
  const int n = blockIdx.y, b = blockIdx.z;
  const int m = n / (a.n_heads / a.n_kv_heads);
  const long rb = (long)b * S;
  const bf16_t* Qg = a.q + rb * a.ld_qkv + (long)n * D;
  const bf16_t* Kg = a.k + rb * a.ld_qkv + (long)m * D;
  const bf16_t* Vg = a.v + rb * a.ld_qkv + (long)m * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int q0w = qt * BQ + wave * 32;
  const int q = q0w + l32;

  bf16x8_t qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk)
    qf[kk] = gload_frag(Qg + (long)q * a.ld_qkv + kk * 16 + hh * 8, q < S);

  f32x16_t oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) zero(oacc[db]);
  float mrow = -INFINITY, lrow = 0.0f;
  const float c = a.scale * kLog2e;
  const int q_last = min(qt * BQ + BQ, S) - 1;
  const int nkt = q_last / BKV + 1;

  // staging: block t < NBLK -> K block (natural), NBLK <= t < 2 NBLK -> V block (transposed)
  const int tb = threadIdx.x;
  const bool has_blk = tb < 2 * NBLK;
  const bool is_v = tb >= NBLK;
  const int blk = tb % NBLK, rg = blk / CPR, cg = blk % CPR;
  uint4 st[8];
  auto load_tile = [&](int kt) {
    if (has_blk) load_blk(is_v ? Vg : Kg, a.ld_qkv, kt * BKV + rg * 8, S, cg, st);
  };
  auto store_tile = [&](int buf) {
    if (has_blk) {
      if (is_v) store_tr(smem[buf] + NAT, rg, cg, st);
      else store_nat<D>(smem[buf], rg, cg, st);
    }
  };

  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nkt;
    if (more) load_tile(kt + 1);
    const int k0 = kt * BKV;
    if (k0 <= q0w + 31) {
      const uint4* Ks = smem[cur];
      const uint4* Vt = smem[cur] + NAT;
      f32x16_t s[2];
      zero(s[0]);
      zero(s[1]);
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              ld_frag(Ks + nat_idx<D>(kb * 32 + l32, kk * 2 + hh)), qf[kk], s[kb], 0, 0, 0);
      const bool diag = (k0 + BKV - 1 > q0w);
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float t = s[kb][i] * c;
          if (diag) {
            const int key = k0 + kb * 32 + (i >> 2) * 8 + hh * 4 + (i & 3);
            if (key > q) t = -INFINITY;
          }
          s[kb][i] = t;
          mt = fmaxf(mt, t);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      const float mnew = fmaxf(mrow, mt);
      const float alpha = fast_exp2(mrow - mnew);
      lrow *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = fast_exp2(s[kb][i] - mnew);
          s[kb][i] = p;
          lrow += p;
        }
      mrow = mnew;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          const bf16x8_t pf = pack_frag(s[kb], ss);
#pragma unroll
          for (int db = 0; db < D / 32; ++db)
            oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                ld_frag(Vt + tr_idx(db * 32 + l32, kb * 4 + ss * 2 + hh)), pf, oacc[db], 0, 0, 0);
        }
    }
    if (more) store_tile(cur ^ 1);
    __syncthreads();
  }

  lrow += __shfl_xor(lrow, 32, 64);
  if (q < S) {
    const float inv = 1.0f / lrow;
    bf16_t* orow = o + (rb + q) * (long)(a.n_heads * D) + (long)n * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = db * 32 + g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(orow + d) =
            make_uint2(pack2(oacc[db][g * 4 + 0] * inv, oacc[db][g * 4 + 1] * inv),
                       pack2(oacc[db][g * 4 + 2] * inv, oacc[db][g * 4 + 3] * inv));
      }
    if (hh == 0) lse[((long)b * a.n_heads + n) * S + q] = (mrow + log2f(lrow)) * kLn2;
  }
}

// -------------------------------------------------- backward pre-pass ----
// delta[b, n, s] = sum_d dO[t, n, d] O[t, n, d]; one thread per (token, head).
template <int D>
__global__ void attn_bwd_pre_k(AttnArgs a, const bf16_t* __restrict__ o,
                               const bf16_t* __restrict__ dout, float* __restrict__ delta) {
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long T = (long)a.batch * a.seq;
  if (id >= T * a.n_heads) return;
  const long t = id / a.n_heads;
  const int n = (int)(id % a.n_heads);
  const long off = t * (long)(a.n_heads * D) + (long)n * D;
  const uint4* op = reinterpret_cast<const uint4*>(o + off);
  const uint4* dp = reinterpret_cast<const uint4*>(dout + off);
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < D / 8; ++c) {
    float x[8], y[8];
    unpack8(op[c], x);
    unpack8(dp[c], y);
#pragma unroll
    for (int e = 0; e < 8; ++e) s += x[e] * y[e];
  }
  const long b = t / a.seq, i = t % a.seq;
  delta[(b * a.n_heads + n) * a.seq + i] = s;
}

// ------------------------------------------------------ backward dK, dV ----
// Block: 128 keys (32 per wave) of one (batch, kv head); loops over the GQA
// group's query heads and the 64-query tiles at or after its first key.
template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_k(
    AttnArgs a, const bf16_t* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16_t* __restrict__ dk, bf16_t* __restrict__ dv,
    long ld_d) {
  constexpr int BKEY = 128, BQ = 64, CPR = D / 8;
  constexpr int NAT = BQ * CPR, TRN = D * 8, NBLK = 8 * CPR;
  // per stage: Q nat, dO nat, Q^T, dO^T, then lse2[64], delta[64] as floats
  constexpr int STAGE = 2 * NAT + 2 * TRN + 32;
  __shared__ uint4 smem[2][STAGE];

  const int S = a.seq;
  const int kt = blockIdx.x, m = blockIdx.y, b = blockIdx.z;
  const int grp = a.n_heads / a.n_kv_heads;
  const long rb = (long)b * S;
  const long ldo = (long)a.n_heads * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int kw0 = kt * BKEY + wave * 32;
  const int key = kw0 + l32;

  const bf16_t* Kg = a.k + rb * a.ld_qkv + (long)m * D;
  const bf16_t* Vg = a.v + rb * a.ld_qkv + (long)m * D;
  bf16x8_t kf[D / 16], vf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    kf[kk] = gload_frag(Kg + (long)key * a.ld_qkv + kk * 16 + hh * 8, key < S);
    vf[kk] = gload_frag(Vg + (long)key * a.ld_qkv + kk * 16 + hh * 8, key < S);
  }
  f32x16_t dka[D / 32], dva[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    zero(dka[db]);
    zero(dva[db]);
  }
  const float c = a.scale * kLog2e;
  const int nqt = (S + BQ - 1) / BQ;
  const int qt0 = (kt * BKEY) / BQ;
  const int per_head = nqt - qt0;
  const int iters = grp * per_head;

  const int tb = threadIdx.x;
  const bool has_blk = tb < 2 * NBLK;
  const bool is_do = tb >= NBLK;
  const int blk = tb % NBLK, rg = blk / CPR, cg = blk % CPR;
  uint4 st[8];
  float st_l = 0.0f, st_d = 0.0f;
  auto load_tile = [&](int it) {
    const int n = m * grp + it / per_head;
    const int q0 = (qt0 + it % per_head) * BQ;
    if (has_blk) {
      if (is_do) load_blk(dout + rb * ldo + (long)n * D, ldo, q0 + rg * 8, S, cg, st);
      else load_blk(a.q + rb * a.ld_qkv + (long)n * D, a.ld_qkv, q0 + rg * 8, S, cg, st);
    }
    if (tb < BQ) {
      const int qq = q0 + tb;
      const long li = ((long)b * a.n_heads + n) * S + qq;
      st_l = qq < S ? lse[li] * kLog2e : INFINITY;
      st_d = qq < S ? delta[li] : 0.0f;
    }
  };
  auto store_tile = [&](int buf) {
    uint4* base = smem[buf];
    if (has_blk) {
      store_nat<D>(base + (is_do ? NAT : 0), rg, cg, st);
      store_tr(base + 2 * NAT + (is_do ? TRN : 0), rg, cg, st);
    }
    float* stats = reinterpret_cast<float*>(base + 2 * NAT + 2 * TRN);
    if (tb < BQ) {
      stats[tb] = st_l;
      stats[BQ + tb] = st_d;
    }
  };

  if (iters > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  for (int it = 0; it < iters; ++it) {
    const int cur = it & 1;
    const bool more = it + 1 < iters;
    if (more) load_tile(it + 1);
    const int q0 = (qt0 + it % per_head) * BQ;
    if (q0 + BQ - 1 >= kw0) {
      const uint4* base = smem[cur];
      const uint4* Qs = base;
      const uint4* dOs = base + NAT;
      const uint4* Qt = base + 2 * NAT;
      const uint4* dOt = base + 2 * NAT + TRN;
      const float* L2 = reinterpret_cast<const float*>(base + 2 * NAT + 2 * TRN);
      const float* Dl = L2 + BQ;
      f32x16_t s[2], dp[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        zero(s[qb]);
        zero(dp[qb]);
      }
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          s[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              ld_frag(Qs + nat_idx<D>(qb * 32 + l32, kk * 2 + hh)), kf[kk], s[qb], 0, 0, 0);
          dp[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              ld_frag(dOs + nat_idx<D>(qb * 32 + l32, kk * 2 + hh)), vf[kk], dp[qb], 0, 0, 0);
        }
      const bool diag = (q0 < kw0 + 31);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int qi = qb * 32 + (i >> 2) * 8 + hh * 4 + (i & 3);
          float p = fast_exp2(s[qb][i] * c - L2[qi]);
          if (diag && key > q0 + qi) p = 0.0f;
          s[qb][i] = p;
          dp[qb][i] = p * (dp[qb][i] - Dl[qi]);
        }
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          const bf16x8_t pf = pack_frag(s[qb], ss);
          const bf16x8_t df = pack_frag(dp[qb], ss);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const int ti = tr_idx(db * 32 + l32, qb * 4 + ss * 2 + hh);
            dva[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_frag(dOt + ti), pf, dva[db], 0, 0, 0);
            dka[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_frag(Qt + ti), df, dka[db], 0, 0, 0);
          }
        }
    }
    if (more) store_tile(cur ^ 1);
    __syncthreads();
  }

  if (key < S) {
    bf16_t* dkr = dk + (rb + key) * ld_d + (long)m * D;
    bf16_t* dvr = dv + (rb + key) * ld_d + (long)m * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = db * 32 + g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(dkr + d) =
            make_uint2(pack2(dka[db][g * 4 + 0] * a.scale, dka[db][g * 4 + 1] * a.scale),
                       pack2(dka[db][g * 4 + 2] * a.scale, dka[db][g * 4 + 3] * a.scale));
        *reinterpret_cast<uint2*>(dvr + d) =
            make_uint2(pack2(dva[db][g * 4 + 0], dva[db][g * 4 + 1]),
                       pack2(dva[db][g * 4 + 2], dva[db][g * 4 + 3]));
      }
  }
}

// ---------------------------------------------------------- backward dQ ----
// Block: 128 queries (32 per wave) of one (batch, head); key tiles of 64.
template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dq_k(AttnArgs a, const bf16_t* __restrict__ dout,
                                                        const float* __restrict__ lse,
                                                        const float* __restrict__ delta,
                                                        bf16_t* __restrict__ dq, long ld_d) {
  constexpr int BQ = 128, BKV = 64, CPR = D / 8;
  constexpr int NAT = BKV * CPR, TRN = D * 8, NBLK = 8 * CPR;
  __shared__ uint4 smem[2][2 * NAT + TRN];  // K nat, V nat, K^T

  const int S = a.seq;
  const int nqt = (S + BQ - 1) / BQ;
  const int qt = nqt - 1 - (int)blockIdx.x;
  const int n = blockIdx.y, b = blockIdx.z;
  const int m = n / (a.n_heads / a.n_kv_heads);
  const long rb = (long)b * S;
  const long ldo = (long)a.n_heads * D;
  const bf16_t* Qg = a.q + rb * a.ld_qkv + (long)n * D;
  const bf16_t* Kg = a.k + rb * a.ld_qkv + (long)m * D;
  const bf16_t* Vg = a.v + rb * a.ld_qkv + (long)m * D;
  const bf16_t* dOg = dout + rb * ldo + (long)n * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int q0w = qt * BQ + wave * 32;
  const int q = q0w + l32;

  bf16x8_t qf[D / 16], of[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    qf[kk] = gload_frag(Qg + (long)q * a.ld_qkv + kk * 16 + hh * 8, q < S);
    of[kk] = gload_frag(dOg + (long)q * ldo + kk * 16 + hh * 8, q < S);
  }
  const long li = ((long)b * a.n_heads + n) * S + q;
  const float l2 = q < S ? lse[li] * kLog2e : INFINITY;
  const float dl = q < S ? delta[li] : 0.0f;
  f32x16_t dqa[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) zero(dqa[db]);
  const float c = a.scale * kLog2e;
  const int q_last = min(qt * BQ + BQ, S) - 1;
  const int nkt = q_last / BKV + 1;

  const int tb = threadIdx.x;
  const bool has_blk = tb < 2 * NBLK;
  const bool is_v = tb >= NBLK;
  const int blk = tb % NBLK, rg = blk / CPR, cg = blk % CPR;
  uint4 st[8];
  auto load_tile = [&](int kt) {
    if (has_blk) load_blk(is_v ? Vg : Kg, a.ld_qkv, kt * BKV + rg * 8, S, cg, st);
  };
  auto store_tile = [&](int buf) {
    if (has_blk) {
      if (is_v) {
        store_nat<D>(smem[buf] + NAT, rg, cg, st);
      } else {
        store_nat<D>(smem[buf], rg, cg, st);
        store_tr(smem[buf] + 2 * NAT, rg, cg, st);
      }
    }
  };

  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nkt;
    if (more) load_tile(kt + 1);
    const int k0 = kt * BKV;
    if (k0 <= q0w + 31) {
      const uint4* Ks = smem[cur];
      const uint4* Vs = smem[cur] + NAT;
      const uint4* Kt = smem[cur] + 2 * NAT;
      f32x16_t s[2], dp[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        zero(s[kb]);
        zero(dp[kb]);
      }
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              ld_frag(Ks + nat_idx<D>(kb * 32 + l32, kk * 2 + hh)), qf[kk], s[kb], 0, 0, 0);
          dp[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              ld_frag(Vs + nat_idx<D>(kb * 32 + l32, kk * 2 + hh)), of[kk], dp[kb], 0, 0, 0);
        }
      const bool diag = (k0 + BKV - 1 > q0w);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float p = fast_exp2(s[kb][i] * c - l2);
          if (diag) {
            const int key = k0 + kb * 32 + (i >> 2) * 8 + hh * 4 + (i & 3);
            if (key > q) p = 0.0f;
          }
          dp[kb][i] = p * (dp[kb][i] - dl);
        }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          const bf16x8_t df = pack_frag(dp[kb], ss);
#pragma unroll
          for (int db = 0; db < D / 32; ++db)
            dqa[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                ld_frag(Kt + tr_idx(db * 32 + l32, kb * 4 + ss * 2 + hh)), df, dqa[db], 0, 0, 0);
        }
    }
    if (more) store_tile(cur ^ 1);
    __syncthreads();
  }

  if (q < S) {
    bf16_t* dqr = dq + (rb + q) * ld_d + (long)n * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = db * 32 + g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(dqr + d) =
            make_uint2(pack2(dqa[db][g * 4 + 0] * a.scale, dqa[db][g * 4 + 1] * a.scale),
                       pack2(dqa[db][g * 4 + 2] * a.scale, dqa[db][g * 4 + 3] * a.scale));
      }
  }
}

}  // namespace

hipError_t attn_fwd(const AttnArgs& a, uint16_t* o, float* lse, hipStream_t s) {
  const dim3 grid((a.seq + 127) / 128, a.n_heads, a.batch), block(256);
  if (a.d == 128) hipLaunchKernelGGL(attn_fwd_k<128>, grid, block, 0, s, a, o, lse);
  else if (a.d == 64) hipLaunchKernelGGL(attn_fwd_k<64>, grid, block, 0, s, a, o, lse);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t attn_bwd_pre(const AttnArgs& a, const uint16_t* o, const uint16_t* dout, float* delta,
                        hipStream_t s) {
  const long n = (long)a.batch * a.seq * a.n_heads;
  const dim3 grid((unsigned)((n + 255) / 256)), block(256);
  if (a.d == 128) hipLaunchKernelGGL(attn_bwd_pre_k<128>, grid, block, 0, s, a, o, dout, delta);
  else if (a.d == 64) hipLaunchKernelGGL(attn_bwd_pre_k<64>, grid, block, 0, s, a, o, dout, delta);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t attn_bwd_dkdv(const AttnArgs& a, const uint16_t* dout, const float* lse,
                         const float* delta, uint16_t* dk, uint16_t* dv, long ld_d,
                         hipStream_t s) {
  const dim3 grid((a.seq + 127) / 128, a.n_kv_heads, a.batch), block(256);
  if (a.d == 128)
    hipLaunchKernelGGL(attn_bwd_dkdv_k<128>, grid, block, 0, s, a, dout, lse, delta, dk, dv, ld_d);
  else if (a.d == 64)
    hipLaunchKernelGGL(attn_bwd_dkdv_k<64>, grid, block, 0, s, a, dout, lse, delta, dk, dv, ld_d);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t attn_bwd_dq(const AttnArgs& a, const uint16_t* dout, const float* lse,
                       const float* delta, uint16_t* dq, long ld_d, hipStream_t s) {
  const dim3 grid((a.seq + 127) / 128, a.n_heads, a.batch), block(256);
  if (a.d == 128)
    hipLaunchKernelGGL(attn_bwd_dq_k<128>, grid, block, 0, s, a, dout, lse, delta, dq, ld_d);
  else if (a.d == 64)
    hipLaunchKernelGGL(attn_bwd_dq_k<64>, grid, block, 0, s, a, dout, lse, delta, dq, ld_d);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace forge

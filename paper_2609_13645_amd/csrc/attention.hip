// Causal grouped-query flash attention on gfx950 MFMA: forward, and the
// backward as a key-owned kernel that forms S, P, dP and dS once per (key,
// query) block, accumulates dV of a kv head over every query head of its GQA
// group and stores dS, then one key-owned and one query-owned product over
// the stored dS for dK and dQ. The paper's H100 kernel accumulates dQ
// through a flat global buffer (App. D, "Anatomy of a Forged Kernel"); here
// no output takes fp32 atomics, so every output is deterministic.
//
// Operand layout. The 32x32x16 MFMA gives each lane one column of its 32x32
// result and sixteen rows. Scores are formed with the lane-owned index on the
// column:
//   * forward / dQ: S^T = K Q^T (lane owns a query), so the softmax row
//     statistics, the LSE and delta are lane-local, and O^T = V^T P^T,
//     dQ^T = K^T dS^T take P^T / dS^T straight from the accumulators;
//   * dK/dV: S = Q K^T (lane owns a key), so dV^T = dO^T P and dK^T = Q^T dS
//     take P / dS straight from the accumulators.
// Accumulator rows come in groups of four, so the reduction index of those
// register-sourced operands is permuted (keys {4h..4h+3, 8+4h..8+4h+3} of a
// 16-group for lane half h); the matching transposed operand (V^T, K^T, Q^T,
// dO^T) is read with two ds_read_b64_tr_b16 of four consecutive rows each
// from the natural [rows][d] tile, which gives exactly that order.
//
// Every tile is loaded global -> LDS by buffer_load ... lds (no register
// staging); rows past the sequence end read as zeros. The online softmax runs
// in the log2 domain (scale * log2 e folded into one multiply); the causal
// mask is evaluated only on tiles that straddle the diagonal, and waves whose
// rows are fully masked skip their MFMAs.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace forge {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr uint32_t kOOB = 0x80000000u;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7FFFFFF0,
                                           0x00020000);
}
// A buffer of `bytes` bytes: loads at or past the end return zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_n(const void* base, long bytes) {
  const int n = bytes <= 0 ? 0 : (bytes > 0x7FFFFFF0L ? 0x7FFFFFF0 : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t* lds_v4i16_ptr;

// Natural [64 rows][D] bf16 tile in LDS, 16-byte chunk c of row r at slot
// c ^ fsw(r). For D = 128 the swizzle keeps both read patterns on distinct
// banks: 32 rows of one chunk (row-fragment reads) and 4 consecutive rows of
// 4 consecutive chunks (transposed reads).
template <int D>
__device__ __forceinline__ int fsw(int r) {
  return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : (r & 7);
}
template <int D>
__device__ __forceinline__ int slot(int r, int c) {
  return r * (D / 8) + (c ^ fsw<D>(r));
}

// DMA of 64 rows [row0, row0 + 64) of a [*, ld] bf16 matrix (column block at
// base) into a natural tile, 1 KB per wave instruction. The lane's byte
// offsets are computed once per block (dma_offsets; they do not depend on
// the tile); rows at or past `lim` read as zeros, cut off by the buffer's
// size rather than by a per-lane test.
template <int D, int NW>
struct DmaPlan {
  static constexpr int LPR = D / 8, RPI = 64 / LPR, PER = 64 / RPI / NW;
  static_assert(PER * RPI * NW == 64, "tile rows must split over waves");
};
template <int D, int NW>
__device__ __forceinline__ void dma_offsets(long ld, int wave, int lane, uint32_t* off) {
  using P = DmaPlan<D, NW>;
#pragma unroll
  for (int i = 0; i < P::PER; ++i) {
    const int row = (i * NW + wave) * P::RPI + lane / P::LPR;
    const int c = (lane % P::LPR) ^ fsw<D>(row);
    off[i] = (uint32_t)(((long)row * ld + c * 8) * 2);
  }
}
template <int D, int NW>
__device__ __forceinline__ void dma_tile_at(const bf16_t* base, long ld, int row0, int lim,
                                            uint4* lds, int wave, const uint32_t* off) {
  using P = DmaPlan<D, NW>;
  const __amdgpu_buffer_rsrc_t r = rsrc_n(base + (long)row0 * ld, (long)(lim - row0) * ld * 2);
#pragma unroll
  for (int i = 0; i < P::PER; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(lds + (i * NW + wave) * 64), 16, off[i],
                                             0, 0, 0);
}

// Row fragment: rows rb..rb+31 (lane row rb + lane % 32), d = kk*16 +
// 8*(lane/32) .. +7. Transposed fragment: column d = db*32 + lane % 32 of the
// tile, rows (the reduction index) r16 + 4h + {0..3} and r16 + 8 + 4h +
// {0..3}, h = lane/32.
// Both are read from per-lane byte offsets computed once per block
// (frag_offsets) plus a compile-time offset OFF (tensor within the stage,
// first row: a multiple of 16 rows, which leaves the swizzle unchanged), so
// each read is one LDS instruction with an immediate offset and no address
// arithmetic.
template <int D>
__device__ __forceinline__ void frag_offsets(int lane, uint32_t (&ro)[D / 16],
                                             uint32_t (&to)[D / 32][2]) {
  const int hh = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) ro[kk] = slot<D>(l32, kk * 2 + hh) * 16;
  const int g = lane >> 4, i = lane & 15;
  const int r = (g >> 1) * 4 + (i >> 2);
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    const int d = db * 32 + (g & 1) * 16 + 4 * (i & 3);
    to[db][0] = (slot<D>(r, d >> 3) * 8 + (d & 7)) * 2;
    to[db][1] = (slot<D>(r + 8, d >> 3) * 8 + (d & 7)) * 2;
  }
}
template <int OFF>
__device__ __forceinline__ bf16x8_t row_at(const uint4* t, uint32_t ro) {
  return __builtin_bit_cast(bf16x8_t,
                            *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(t) + ro + OFF));
}
template <int OFF>
__device__ __forceinline__ bf16x8_t tr_at(const uint4* t, const uint32_t (&to)[2]) {
  const char* e = reinterpret_cast<const char*>(t) + OFF;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_ptr)(e + to[0]));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_ptr)(e + to[1]));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return __builtin_bit_cast(bf16x8_t, make_uint4(a.x, a.y, b.x, b.y));
}

__device__ __forceinline__ bf16x8_t pack_frag(const f32x16_t& v, int s) {
  uint4 u = make_uint4(pack2(v[8 * s + 0], v[8 * s + 1]), pack2(v[8 * s + 2], v[8 * s + 3]),
                       pack2(v[8 * s + 4], v[8 * s + 5]), pack2(v[8 * s + 6], v[8 * s + 7]));
  return __builtin_bit_cast(bf16x8_t, u);
}

__device__ __forceinline__ bf16x8_t gload_frag(const bf16_t* p, bool ok) {
  return __builtin_bit_cast(bf16x8_t, ok ? *reinterpret_cast<const uint4*>(p)
                                         : make_uint4(0, 0, 0, 0));
}

__device__ __forceinline__ void zero(f32x16_t& a) {
#pragma unroll
  for (int e = 0; e < 16; ++e) a[e] = 0.0f;
}

#define MFMA(a, b, c) __builtin_amdgcn_mfma_f32_32x32x16_bf16((a), (b), (c), 0, 0, 0)

// ------------------------------------------------------------- forward ----
// Block: 128 queries (32 per wave) of one (batch, head); key tiles of 64.
//  * K/V tiles are double-buffered in LDS; each tile ends with an explicit
//    wait + barrier.
//  * All K fragments of a tile are in flight before its 16 score MFMAs, and
//    each MFMA pair waits only for its own fragments; the V^T fragments are
//    read after the row max and land under the exp / row sums. The row
//    max's exchange between the two lane halves is v_permlane32_swap, a
//    VALU operation: as an LDS lane exchange it waited on the lgkm counter,
//    which (saturating at 15) then also waited for every V^T read in flight.
//  * The softmax, not the MFMAs, bounds this kernel on this chip (a wave64
//    VALU op takes 4 cycles, exp more), so the per-tile VALU work is cut to
//    the softmax itself: the scale is folded into the exponent's FMA; the
//    running max (log2 units) is raised only when a tile's max exceeds it by
//    more than 8, so the output rescale runs on few tiles (behind a real
//    branch) and probabilities stay below 2^8 (exact in the final
//    normalisation); the causal mask runs only on the diagonal tile; the row
//    max is a running chain the compiler turns into v_max3 without quieting
//    each operand first; fragment reads are inline asm from per-lane LDS
//    addresses computed once, with the stage, key block and row offsets as
//    immediates (no address arithmetic per read, no compiler wait for the
//    in-flight DMA of the other stage).
//  * Inline asm here only reads LDS into registers and waits; it never reads
//    an MFMA result (the compiler does not insert the wait states an MFMA
//    result needs before an asm consumer).
namespace fa {

__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
template <int OFF>
__device__ __forceinline__ bf16x8_t rd_b128(uint32_t a) {
  uint4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(a), "n"(OFF) : "memory");
  return __builtin_bit_cast(bf16x8_t, r);
}
template <int OFF>
__device__ __forceinline__ bf16x8_t rd_tr(uint32_t lo, uint32_t hi) {
  uint2 x, y;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(x) : "v"(lo), "n"(OFF) : "memory");
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(y) : "v"(hi), "n"(OFF) : "memory");
  return __builtin_bit_cast(bf16x8_t, make_uint4(x.x, x.y, y.x, y.y));
}
// at most N LDS operations of this wave outstanding (the counter saturates
// at 15: a larger N waits for all but 15)
template <int N>
__device__ __forceinline__ void wait_lds() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N < 15 ? N : 15) : "memory");
}
// the value counts as rewritten here, so its uses stay below the wait
template <typename T>
__device__ __forceinline__ void bind(T& x) {
  asm volatile("" : "+v"(x));
}
__device__ __forceinline__ void sync_block() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}
template <int I>
using ic = std::integral_constant<int, I>;
// max / sum of the values of lanes l and l ^ 32, on the VALU
// (v_permlane32_swap): no LDS operation, so no lgkmcnt wait that would also
// cover the fragment reads in flight
// (a = lanes 0..31 in both halves, b = lanes 32..63). Inline asm: through
// the compiler builtin, the second result of the swap was replaced by the
// first in the code generated for a sum of the two (a miscompile seen with
// this toolchain). The leading and trailing s_nop give the wait states
// around a VALU write of the operands and a VALU read of the results.
__device__ __forceinline__ f32x2_t halves(float v) {
  uint32_t a = __builtin_bit_cast(uint32_t, v), b = a;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
  return f32x2_t{__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)};
}
__device__ __forceinline__ float max_xor32(float v) {
  const f32x2_t h = halves(v);
  return fmaxf(h[0], h[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const f32x2_t h = halves(v);
  return h[0] + h[1];
}
}  // namespace fa

template <int D>
__global__ __launch_bounds__(256, 2) void attn_fwd_k(AttnArgs a, bf16_t* __restrict__ o,
                                                         float* __restrict__ lse) {
  constexpr int BQ = 128, BKV = 64, NAT = BKV * D / 8, KK = D / 16, DB = D / 32;
  constexpr int TILE_B = NAT * 16;       // bytes of one K or V tile
  constexpr int HALF_B = TILE_B / 2;     // rows 32..63 of a tile
  constexpr int ROW16_B = 16 * D * 2;    // 16 rows of a tile
  constexpr int V0_B = 2 * TILE_B;       // V slots after the two K slots
  constexpr int KW = 4;                  // K fragment steps (kk) in flight
  // K slots 0, 1 then V slots 0, 1: tile t's K in K slot t & 1, its V in V
  // slot t & 1. K runs one tile ahead of V (S of tile j + 1 is formed while
  // tile j's softmax and P V run), so each slot pair is a double buffer.
  __shared__ uint4 smem[4 * NAT];
  const int S = a.seq;
  const int nqt = (S + BQ - 1) / BQ;
  // Block order: the query tiles with the most keys (the last ones) first,
  // one tile level at a time across every (batch, head), so that the long
  // blocks do not end up in the last round of the grid. Within a level,
  // consecutive blocks go to the 8 XCDs in turn; when the level's count is
  // a multiple of 8, XCD x takes a contiguous range of heads at every level,
  // so the heads that share a kv head keep its K / V in one L2.
  const int W = a.n_heads * a.batch;
  const int id = (int)blockIdx.x;
  const int level = id / W, r = id % W;
  const int L = (W % 8 == 0) ? (r % 8) * (W / 8) + r / 8 : r;
  const int qt = nqt - 1 - level;
  const int n = L % a.n_heads, b = L / a.n_heads;
  const int m = n / (a.n_heads / a.n_kv_heads);
  const long rb = (long)b * S;
  const bf16_t* Qg = a.q + rb * a.ld_qkv + (long)n * D;
  const bf16_t* Kg = a.k + rb * a.ld_qkv + (long)m * D;
  const bf16_t* Vg = a.v + rb * a.ld_qkv + (long)m * D;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hh = lane >> 5, l32 = lane & 31;
  const int q0w = qt * BQ + wave * 32;
  const int q = q0w + l32;
  bf16x8_t qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    qf[kk] = gload_frag(Qg + (long)q * a.ld_qkv + kk * 16 + hh * 8, q < S);
  f32x16_t oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) zero(oacc[db]);
  float mrow = -INFINITY, lrow = 0.0f;
  const float c = a.scale * kLog2e;
  const int q_last = min(qt * BQ + BQ, S) - 1;
  const int nkt = q_last / BKV + 1;
  // the wave's last key tile (its queries end at q0w + 31)
  const int lw = min(q0w + 31, S - 1) / BKV;

  // per-lane byte addresses in K slot 0 / V slot 0: K row fragment of slice
  // kk (rows 0..31), V^T fragment of column block db (rows 0..15, both row
  // quads)
  const uint32_t base = fa::lds_off(smem);
  uint32_t ka[KK], va[DB][2];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) ka[kk] = base + slot<D>(l32, kk * 2 + hh) * 16;
  {
    const int g4 = lane >> 4, i = lane & 15;
    const int r = (g4 >> 1) * 4 + (i >> 2);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int dd = db * 32 + (g4 & 1) * 16 + 4 * (i & 3);
      va[db][0] = base + V0_B + (slot<D>(r, dd >> 3) * 8 + (dd & 7)) * 2;
      va[db][1] = base + V0_B + (slot<D>(r + 8, dd >> 3) * 8 + (dd & 7)) * 2;
    }
  }

  uint32_t doff[DmaPlan<D, 4>::PER];
  dma_offsets<D, 4>(a.ld_qkv, wave, lane, doff);
  auto dma_k = [&](int kt) __attribute__((always_inline)) {
    dma_tile_at<D, 4>(Kg, a.ld_qkv, kt * BKV, S, smem + (kt & 1) * NAT, wave, doff);
  };
  auto dma_v = [&](int kt) __attribute__((always_inline)) {
    dma_tile_at<D, 4>(Vg, a.ld_qkv, kt * BKV, S, smem + (2 + (kt & 1)) * NAT, wave, doff);
  };

  // S^T of a tile (K slot KS) into sc: K fragments KW steps ahead, each MFMA
  // pair waiting for its own two reads; after MFMA step kk, the hook runs
  // (the softmax work of the previous tile, interleaved with these MFMAs)
  auto scores = [&](auto KS, f32x16_t (&sc)[2], auto&& hook) __attribute__((always_inline)) {
    constexpr int KO = decltype(KS)::value * TILE_B;
    bf16x8_t f[KK][2];
#pragma unroll
    for (int kk = 0; kk < KW; ++kk) {
      f[kk][0] = fa::rd_b128<KO>(ka[kk]);
      f[kk][1] = fa::rd_b128<KO + HALF_B>(ka[kk]);
    }
    zero(sc[0]);
    zero(sc[1]);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      // reads issued after step kk's: min(KW - 1, KK - 1 - kk) steps of two
      switch (KK - 1 - kk < KW - 1 ? KK - 1 - kk : KW - 1) {
        case 3: fa::wait_lds<6>(); break;
        case 2: fa::wait_lds<4>(); break;
        case 1: fa::wait_lds<2>(); break;
        default: fa::wait_lds<0>(); break;
      }
      fa::bind(f[kk][0]);
      fa::bind(f[kk][1]);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sc[kb] = MFMA(f[kk][kb], qf[kk], sc[kb]);
      if (kk + KW < KK) {
        f[kk + KW][0] = fa::rd_b128<KO>(ka[kk + KW]);
        f[kk + KW][1] = fa::rd_b128<KO + HALF_B>(ka[kk + KW]);
      }
      hook(kk);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto no_hook = [](int) {};

  // causal mask of a tile that straddles the wave's diagonal, then the row
  // max, the lazy rescale; returns -running max (log2 units)
  auto softmax_head = [&](f32x16_t (&s)[2], int kt) __attribute__((always_inline)) {
    const int k0 = kt * BKV;
    if (k0 + BKV - 1 > q0w) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = k0 + kb * 32 + (i >> 2) * 8 + hh * 4 + (i & 3);
          if (key > q) s[kb][i] = -INFINITY;
        }
    }
    // two running-max chains over the lane's 32 scores (the compiler forms
    // v_max3 without quieting every operand first)
    float mk[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float t = fmaxf(s[kb][0], s[kb][1]);
#pragma unroll
      for (int i = 2; i < 16; ++i) t = fmaxf(t, s[kb][i]);
      mk[kb] = t;
    }
    const float mt = fa::max_xor32(fmaxf(mk[0], mk[1])) * c;
    const bool grow = mt > mrow + 8.0f;
    if (__ballot(grow)) {
      const float mnew = grow ? mt : mrow;
      const float alpha = fast_exp2(mrow - mnew);
      lrow *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
      mrow = mnew;
    }
    return -mrow;
  };
  // probabilities of scores 4 step .. 4 step + 3 (of 32), in place, and
  // their share of the row sum
  auto exp_step = [&](f32x16_t (&s)[2], float nm, int step) __attribute__((always_inline)) {
    const int kb = step >> 2, i0 = (step & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float pp = fast_exp2(__builtin_fmaf(s[kb][i0 + e], c, nm));
      s[kb][i0 + e] = pp;
      lrow += pp;
    }
  };
  // O^T += V^T P^T over the tile in V slot VS (va addresses V slot 0)
  auto pv = [&](auto VS, const f32x16_t (&p)[2]) __attribute__((always_inline)) {
    constexpr int VO = decltype(VS)::value * TILE_B;
    bf16x8_t v[2][2][DB];
    // two (kb, ss) steps of DB fragments in flight
#pragma unroll
    for (int db = 0; db < DB; ++db) v[0][0][db] = fa::rd_tr<VO>(va[db][0], va[db][1]);
#pragma unroll
    for (int db = 0; db < DB; ++db) v[0][1][db] = fa::rd_tr<VO + ROW16_B>(va[db][0], va[db][1]);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int kb = st >> 1, ss = st & 1;
      const bf16x8_t pf = pack_frag(p[kb], ss);
      if (st < 3) fa::wait_lds<2 * DB>();
      else fa::wait_lds<0>();
#pragma unroll
      for (int db = 0; db < DB; ++db) fa::bind(v[kb][ss][db]);
      if (st + 2 < 4) {
        const int s2 = st + 2;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          if (s2 == 2) v[1][0][db] = fa::rd_tr<VO + 2 * ROW16_B>(va[db][0], va[db][1]);
          if (s2 == 3) v[1][1][db] = fa::rd_tr<VO + 3 * ROW16_B>(va[db][0], va[db][1]);
        }
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] = MFMA(v[kb][ss][db], pf, oacc[db]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // iteration j: tile j's softmax, interleaved with the scores of tile
  // j + 1, then tile j's P V. K of tile j + 1 and V of tile j are resident
  // (and fenced by the barrier that opens the iteration); the DMA of K of
  // tile j + 2 and V of tile j + 1 refills the slots that tiles j and j - 1
  // used.
  f32x16_t sa[2], sb[2];
  auto iteration = [&](auto PAR, f32x16_t (&scur)[2], f32x16_t (&snext)[2], int j)
      __attribute__((always_inline)) {
    constexpr int P = decltype(PAR)::value;   // j & 1
    fa::sync_block();
    if (j + 2 < nkt) dma_k(j + 2);
    if (j + 1 < nkt) dma_v(j + 1);
    if (j > lw) return;   // every query of this wave is before the tile
    const float nm = softmax_head(scur, j);
    if (j < lw) {
      // the 8 exp steps of 4 spread over the KK MFMA steps of the next
      // tile's scores
      static_assert(8 % KK == 0, "exp steps per MFMA step");
      scores(fa::ic<P ^ 1>{}, snext, [&](int kk) __attribute__((always_inline)) {
#pragma unroll
        for (int st = kk * (8 / KK); st < (kk + 1) * (8 / KK); ++st) exp_step(scur, nm, st);
      });
    } else {
      // (the binds keep the compiler from hoisting the exp steps of both
      // branches above the branch, which would undo the interleaving)
      fa::bind(scur[0]);
      fa::bind(scur[1]);
#pragma unroll
      for (int st = 0; st < 8; ++st) exp_step(scur, nm, st);
    }
    pv(fa::ic<P>{}, scur);
  };

  dma_k(0);
  dma_v(0);
  if (nkt > 1) dma_k(1);
  fa::sync_block();
  scores(fa::ic<0>{}, sa, no_hook);
  for (int j = 0; j < nkt; j += 2) {
    iteration(fa::ic<0>{}, sa, sb, j);
    if (j + 1 < nkt) iteration(fa::ic<1>{}, sb, sa, j + 1);
  }
  lrow = fa::sum_xor32(lrow);
  if (q < S) {
    const float inv = 1.0f / lrow;
    bf16_t* orow = o + (rb + q) * (long)(a.n_heads * D) + (long)n * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dd = db * 32 + g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(orow + dd) =
            make_uint2(pack2(oacc[db][g * 4 + 0] * inv, oacc[db][g * 4 + 1] * inv),
                       pack2(oacc[db][g * 4 + 2] * inv, oacc[db][g * 4 + 3] * inv));
      }
    if (hh == 0) lse[((long)b * a.n_heads + n) * S + q] = (mrow + log2f(lrow)) * kLn2;
  }
}

// ------------------------------------------------------------ backward ----
// Four launches and five MFMA products in all (S recomputed once), with no
// atomics, so every output is deterministic:
//  1. attn_bwd_prep_k: per query, -delta = -rowsum(dO * O) and
//     -LSE log2(e) (the exponent offset of P = exp(S - LSE) in base 2).
//  2. attn_bwd_dv_k, key-owned (64 keys of a kv head per block):
//     S = Q K^T, P, dP = dO V^T, dS = P (dP - delta); dV = sum P^T dO over
//     the GQA group; dS goes to a scratch buffer in bf16, the precision the
//     dK and dQ products take it in.
//  3. attn_bwd_dk_k, key-owned: dK = scale * sum dS^T Q from the stored dS.
//  4. attn_bwd_dq_k, query-owned: dQ = scale * dS K from the stored dS.
// The paper's H100 kernel accumulates dQ through fp32 atomics in a flat
// buffer (App. D); here dQ is a product of its own over the stored dS, and
// dK no longer needs S and dP formed a second time.
//
// dS layout, per (batch, head): for 64-key tile kt, one 4 KB block per
// 32-query slab j = 2 kt .. NS - 1 (NS = ceil(seq / 32)) in slab order, so
// only the causal half is stored. A block holds its 64 x 32 values in the
// dV pass's accumulator order: value 4 g + e of lane hh * 32 + l32 of key
// block kb, (key 32 kb + l32, query 8 g + 4 hh + e), is element
// 4 (g & 1) + e of the 16-byte piece at
//   kb * 2 KB + u * 1 KB + 512 hh + ((16 l32) ^ (128 hh) ^ (64 u)),  u = g / 2.
// (The LDS serves a 16-byte read 16 lanes at a time from 64 banks: the dK
// pass's B-fragment reads take 16 consecutive keys' pieces, a contiguous
// 256 bytes; the XORs put a key's two lane halves 128 bytes apart and the
// two query halves 64 bytes apart, so the dQ pass's transposed reads cover
// all banks too.)
// Every
// visited block is written whole (zeros where the mask or the sequence end
// removes a score). That order is also the dK pass's B-fragment order
// (loaded straight into registers, 1 KB per wave instruction); the dQ pass
// reads its transpose with ds_read_b64_tr_b16.
struct DsLayout {
  int ns;      // 32-query slabs of the sequence
  long head;   // elements per (batch, head)
  __host__ __device__ explicit DsLayout(int S) {
    ns = (S + 31) / 32;
    const long nkt = (S + 63) / 64;
    head = 2048L * (nkt * ns - nkt * (nkt - 1));
  }
  __host__ __device__ long tile(int kt) const { return 2048L * ((long)kt * ns - (long)kt * (kt - 1)); }
  __host__ __device__ long block(int kt, int j) const { return tile(kt) + 2048L * (j - 2 * kt); }
};

// 1. -delta and -LSE log2(e) of every (batch, head, query): D / 8 lanes per
// (token, head) row of dO and O, 16-byte loads (the heads of a token are
// adjacent rows).
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_prep_k(const bf16_t* __restrict__ o,
                                                       const bf16_t* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       float* __restrict__ delta, long rows,
                                                       int n_heads, int S) {
  constexpr int TPR = D / 8;
  const long r = (long)blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  const int c = threadIdx.x % TPR;
  float s = 0.0f;
  if (r < rows) {
    float x[8], y[8];
    unpack8(*reinterpret_cast<const uint4*>(dout + r * D + c * 8), x);
    unpack8(*reinterpret_cast<const uint4*>(o + r * D + c * 8), y);
#pragma unroll
    for (int e = 0; e < 8; ++e) s = __builtin_fmaf(x[e], y[e], s);
  }
#pragma unroll
  for (int w = TPR / 2; w >= 1; w >>= 1) s += __shfl_xor(s, w, 64);
  if (c == 0 && r < rows) {
    const long t = r / n_heads;
    const int n = (int)(r % n_heads);
    const long li = ((t / S) * n_heads + n) * S + t % S;
    delta[li] = -s;
    delta[rows + li] = -lse[li] * kLog2e;
  }
}

// 2-3. Key-owned blocks: 64 keys [k0, k0 + 64) of one (batch, kv head), four
// waves, one per SIMD. The block's work is every (query head of the GQA
// group, 32-query slab at or after k0) pair; wave w takes pairs w, w + 4,
// ... and accumulates over them for all 64 keys, streaming each pair's
// operands through a private LDS double buffer (no block barrier in the
// loop). At the end the four waves' sums are added through LDS in wave
// order, so the result does not depend on timing, and written as bf16: no
// partials leave the block, and K / V are read once per GQA group.
template <int D>
struct KvPlan {
  static constexpr int BK = 64, BQ = 32;
  static constexpr int SLAB = BQ * D / 8;         // 16-byte chunks of a 32-row tile
  static constexpr int RED = BK * (D + 4) / 4;    // one wave's [64][D + 4] fp32 sums
  static constexpr int LPR = D / 8, RPI = 64 / LPR, PER = BQ / RPI;  // DMA of a slab
};
// dV pass: per-wave buffer (Q, dO slabs, -LSE log2 e | -delta) and its DMA
// instructions per pair
template <int D>
struct KvBuf {
  using P = KvPlan<D>;
  static constexpr int WBUF = 2 * P::SLAB + 16;
  static constexpr int DMA = 2 * P::PER + 1;
  static constexpr int ARR = 4 * WBUF > 2 * P::RED ? 4 * WBUF : 2 * P::RED;
};
// s_waitcnt immediate that waits for vmcnt <= n only (gfx9 encoding: vmcnt
// bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 at their maxima)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

template <int D>
__device__ __forceinline__ void slab_offsets(long ld, int lane, uint32_t (&off)[KvPlan<D>::PER]) {
  using P = KvPlan<D>;
#pragma unroll
  for (int i = 0; i < P::PER; ++i) {
    const int row = i * P::RPI + lane / P::LPR;
    const int c = (lane % P::LPR) ^ fsw<D>(row);
    off[i] = (uint32_t)(((long)row * ld + c * 8) * 2);
  }
}
// 32 rows [row0, row0 + 32) of a [*, ld] bf16 matrix into a natural tile;
// rows at or past lim read as zeros.
template <int D>
__device__ __forceinline__ void dma_slab(const bf16_t* base, long ld, int row0, int lim,
                                         uint4* lds, const uint32_t* off) {
  using P = KvPlan<D>;
  const __amdgpu_buffer_rsrc_t r = rsrc_n(base + (long)row0 * ld, (long)(lim - row0) * ld * 2);
#pragma unroll
  for (int i = 0; i < P::PER; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(lds + i * 64), 16, off[i], 0, 0, 0);
}

// The four waves' [64 keys][D] accumulators (acc[db][kb]: rows d, columns
// keys) summed in wave order through sm0 / sm1, times scale, stored as bf16
// rows out[key][D] (key-major, row stride ld) for the first nkeys keys.
template <int D>
__device__ __forceinline__ void kv_reduce_store(const f32x16_t (&acc)[D / 32][2], uint4* sm0,
                                                uint4* sm1, int wave, int lane, float scale,
                                                bf16_t* out, long ld, int nkeys) {
  using P = KvPlan<D>;
  constexpr int DB = D / 32;
  const int hh = lane >> 5, l32 = lane & 31;
  float* red = reinterpret_cast<float*>((wave < 2 ? sm0 : sm1) + (wave & 1) * P::RED);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // the unused last reload
  __syncthreads();
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<float4*>(red + (kb * 32 + l32) * (D + 4) + db * 32 + g * 8 + hh * 4) =
            make_float4(acc[db][kb][g * 4], acc[db][kb][g * 4 + 1], acc[db][kb][g * 4 + 2],
                        acc[db][kb][g * 4 + 3]);
  __syncthreads();
  // the four threads of a key take interleaved 8-column pieces (columns
  // 32 j + 8 part ..), so eight lanes of a 16-byte read cover all banks
  const int key = threadIdx.x >> 2;
  const int part = threadIdx.x & 3;
  if (key < nkeys) {
    const float* w0 = reinterpret_cast<const float*>(sm0);
    const float* w1 = reinterpret_cast<const float*>(sm0 + P::RED);
    const float* w2 = reinterpret_cast<const float*>(sm1);
    const float* w3 = reinterpret_cast<const float*>(sm1 + P::RED);
    bf16_t* orow = out + (long)key * ld + part * 8;
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
      const int o = key * (D + 4) + j * 32 + part * 8;
      float f[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) f[u] = (((w0[o + u] + w1[o + u]) + w2[o + u]) + w3[o + u]) * scale;
      *reinterpret_cast<uint4*>(orow + j * 32) = pack8(f);
    }
  }
}

// 2. dV pass. Per pair: S and dP (accumulators starting at -delta, so they
// hold dP - delta), P = exp2(S c - LSE log2 e), dS = P (dP - delta) stored,
// dV^T += dO^T P. The wave keeps K and V of its 64 keys in registers as two
// 32-key column blocks, so every Q / dO fragment read from LDS feeds two
// MFMAs.
template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dv_k(AttnArgs a,
                                                       const bf16_t* __restrict__ dout,
                                                       const float* __restrict__ delta,
                                                       bf16_t* __restrict__ ds,
                                                       bf16_t* __restrict__ dv, long ld_d) {
  using P = KvPlan<D>;
  using B = KvBuf<D>;
  constexpr int BK = P::BK, BQ = P::BQ, SLAB = P::SLAB, KK = D / 16, DB = D / 32;
  __shared__ uint4 sm0[B::ARR];
  __shared__ uint4 sm1[B::ARR];

  const int S = a.seq;
  const int grp = a.n_heads / a.n_kv_heads;
  // block order: key tile slowest, so the low key tiles (the most work)
  // are dispatched first
  const int per_kt = a.n_kv_heads * a.batch;
  const int kt = (int)blockIdx.x / per_kt;
  const int m = (int)blockIdx.x % per_kt % a.n_kv_heads;
  const int b = (int)blockIdx.x % per_kt / a.n_kv_heads;
  const int k0 = kt * BK;
  const int j0 = k0 / BQ;                      // first slab holding a query >= k0
  const int ns = (S + BQ - 1) / BQ - j0;       // slabs per query head
  const int total = grp * ns;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hh = lane >> 5, l32 = lane & 31;
  const long rb = (long)b * S;
  const long ldo = (long)a.n_heads * D;
  const long nrows = (long)a.batch * a.n_heads * S;
  const DsLayout L(S);

  // K and V rows of the lane's two keys k0 + l32 and k0 + 32 + l32: the
  // B operands of S and dP
  bf16x8_t kf[2][KK], vf[2][KK];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int key = k0 + kb * 32 + l32;
    const long r = (rb + key) * a.ld_qkv + (long)m * D + hh * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kf[kb][kk] = gload_frag(a.k + r + kk * 16, key < S);
      vf[kb][kk] = gload_frag(a.v + r + kk * 16, key < S);
    }
  }
  f32x16_t acc[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) zero(acc[db][kb]);
  const float c = a.scale * kLog2e;

  uint32_t qoff[P::PER], ooff[P::PER];
  slab_offsets<D>(a.ld_qkv, lane, qoff);
  slab_offsets<D>(ldo, lane, ooff);
  uint32_t ro[KK], to[DB][2];
  frag_offsets<D>(lane, ro, to);
  const __amdgpu_buffer_rsrc_t drs = rsrc(delta);
  // the lane's dS piece (elements) in a 1 KB half; half u adds the XOR u * 32
  const int pc0 = 256 * hh + ((8 * l32) ^ (64 * hh));

  // pair p: query head m * grp + p % grp, slab j0 + ns - 1 - p / grp. Every
  // block of the kv group walks the slabs from the sequence end, head-minor,
  // so the blocks running at once read the same Q / dO slabs (one XCD's L2
  // serves them; block ids cycle through the kv heads, which the dispatcher
  // spreads over the XCDs)
  auto load = [&](int p, uint4* base) __attribute__((always_inline)) {
    const int n = m * grp + p % grp;
    const int q0 = (j0 + ns - 1 - p / grp) * BQ;
    dma_slab<D>(a.q + rb * a.ld_qkv + (long)n * D, a.ld_qkv, q0, S, base, qoff);
    dma_slab<D>(dout + rb * ldo + (long)n * D, ldo, q0, S, base + SLAB, ooff);
    // lanes 0-31: -LSE log2(e) of the slab's queries; lanes 32-63: -delta
    const long li = ((long)b * a.n_heads + n) * S + q0 + l32;
    const uint32_t off = q0 + l32 < S ? (uint32_t)(((hh ? 0 : nrows) + li) * 4) : kOOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(drs, (lds_ptr_t)(base + 2 * SLAB), 4, off, 0, 0, 0);
  };

  auto pair = [&](const uint4* base, int p) __attribute__((always_inline)) {
    // this buffer's DMA has landed once only the other buffer's (issued
    // after it) can still be in flight
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(B::DMA));
    __builtin_amdgcn_sched_barrier(0);
    const int n = m * grp + p % grp;
    const int q0 = (j0 + ns - 1 - p / grp) * BQ;
    const float* Lp = reinterpret_cast<const float*>(base + 2 * SLAB);
    const float* Dl = Lp + BQ;
    f32x16_t sc[2], dp[2];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 dd = *reinterpret_cast<const float4*>(Dl + g * 8 + hh * 4);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        dp[kb][g * 4 + 0] = dd.x;
        dp[kb][g * 4 + 1] = dd.y;
        dp[kb][g * 4 + 2] = dd.z;
        dp[kb][g * 4 + 3] = dd.w;
      }
    }
    // S and dP: each row fragment feeds both key blocks. The fragments of
    // a product are all read at once (inline asm: the compiler would wait
    // for each read before its MFMAs) and each MFMA pair waits only for its
    // own fragment.
    const uint32_t ab = fa::lds_off(base);
    auto rows_product = [&](auto OFF, const bf16x8_t (&bk)[2][KK], f32x16_t (&cc)[2], bool from0)
        __attribute__((always_inline)) {
      constexpr int O = decltype(OFF)::value;
      bf16x8_t f[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) f[kk] = fa::rd_b128<O>(ab + ro[kk]);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        switch (KK - 1 - kk) {
          case 7: fa::wait_lds<7>(); break;
          case 6: fa::wait_lds<6>(); break;
          case 5: fa::wait_lds<5>(); break;
          case 4: fa::wait_lds<4>(); break;
          case 3: fa::wait_lds<3>(); break;
          case 2: fa::wait_lds<2>(); break;
          case 1: fa::wait_lds<1>(); break;
          default: fa::wait_lds<0>(); break;
        }
        fa::bind(f[kk]);
        cc[0] = MFMA(f[kk], bk[0][kk], (kk == 0 && from0) ? f32x16_t{} : cc[0]);
        cc[1] = MFMA(f[kk], bk[1][kk], (kk == 0 && from0) ? f32x16_t{} : cc[1]);
        __builtin_amdgcn_sched_barrier(0);   // keep each pair at its own wait
      }
    };
    rows_product(fa::ic<0>{}, kf, sc, true);
    rows_product(fa::ic<SLAB * 16>{}, vf, dp, false);
    // causal mask and sequence tail (diagonal and last slabs only): -inf
    // scores, so exp2 gives 0
    if (q0 < k0 + BK - 1 || q0 + BQ > S) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int q = q0 + (i >> 2) * 8 + hh * 4 + (i & 3);
          if (k0 + kb * 32 + l32 > q || q >= S) sc[kb][i] = -INFINITY;
        }
    }
    // P into sc, dS into dp
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 ll = *reinterpret_cast<const float4*>(Lp + g * 8 + hh * 4);
      const float lv[4] = {ll.x, ll.y, ll.z, ll.w};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = g * 4 + e;
          const float pr = fast_exp2(__builtin_fmaf(sc[kb][i], c, lv[e]));
          dp[kb][i] = pr * dp[kb][i];
          sc[kb][i] = pr;
        }
    }
    // the pair's dS block, in accumulator order: 16-byte stores, 1 KB per
    // wave instruction; nontemporal, since the block is read back only after
    // the pass (as ordinary stores, the dirty lines the memory-side cache
    // holds at the end are written back while the dK pass reads dS: dK
    // +7 %)
    bf16_t* blk = ds + ((long)b * a.n_heads + n) * L.head + L.block(kt, q0 / BQ);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int u = 0; u < 2; ++u)
        __builtin_nontemporal_store(
            __builtin_bit_cast(u32x4_t, pack_frag(dp[kb], u)),
            reinterpret_cast<u32x4_t*>(blk + kb * 1024 + u * 512 + (pc0 ^ (u * 32))));
    // dV^T += dO^T P, 16 queries at a time; each transposed fragment feeds
    // both key blocks
    auto quarter = [&](auto SS) __attribute__((always_inline)) {
      constexpr int ss = decltype(SS)::value;
      constexpr int T0 = SLAB * 16 + ss * 16 * D * 2;   // dO rows 16 ss ..
      // all transposed fragments of the quarter in flight (inline asm), each
      // MFMA pair waiting only for its own two reads
      bf16x8_t ft[DB];
#pragma unroll
      for (int db = 0; db < DB; ++db) ft[db] = fa::rd_tr<T0>(ab + to[db][0], ab + to[db][1]);
      const bf16x8_t p0 = pack_frag(sc[0], ss), p1 = pack_frag(sc[1], ss);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        switch (DB - 1 - db) {
          case 3: fa::wait_lds<6>(); break;
          case 2: fa::wait_lds<4>(); break;
          case 1: fa::wait_lds<2>(); break;
          default: fa::wait_lds<0>(); break;
        }
        fa::bind(ft[db]);
        acc[db][0] = MFMA(ft[db], p0, acc[db][0]);
        acc[db][1] = MFMA(ft[db], p1, acc[db][1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    quarter(std::integral_constant<int, 0>());
    quarter(std::integral_constant<int, 1>());
  };

  // the wave's pairs through its two buffers (two arrays, so the compiler
  // waits only for the DMA of the buffer being read)
  // Every step issues the same DMA count (past the last pair it reloads the
  // last pair, which is not used), so the wait before reading a buffer can
  // leave the other buffer's DMA in flight.
  uint4* my0 = sm0 + wave * B::WBUF;
  uint4* my1 = sm1 + wave * B::WBUF;
  load(min(wave, total - 1), my0);
  for (int p = wave; p < total; p += 8) {
    load(min(p + 4, total - 1), my1);
    pair(my0, p);
    if (p + 4 >= total) break;
    load(min(p + 8, total - 1), my0);
    pair(my1, p + 4);
  }
  kv_reduce_store<D>(acc, sm0, sm1, wave, lane, 1.0f, dv + (rb + k0) * ld_d + (long)m * D,
                             ld_d, S - k0);
}

// 3. dK pass: dK^T += Q^T dS over the block's pairs. Each pair's Q slab and
// dS block go through the wave's LDS ring by DMA; the A operand is the Q
// slab's transposed fragments (as the dV pass reads dO^T), and the dS block
// is already in B-fragment order, so each B fragment is one 16-byte read
// (1 KB per wave instruction, contiguous). Each wave keeps KR pairs in
// flight: the pass streams dS from HBM with little arithmetic per byte.
template <int D>
struct DkPlan {
  using P = KvPlan<D>;
  static constexpr int KR = 3;                      // ring depth (pairs per wave)
  static constexpr int SLOT = P::SLAB + 256;        // Q slab + 4 KB dS block
  static constexpr int MEM = P::PER + 4;            // DMA instructions per pair
  static constexpr int RING = 4 * KR * SLOT;        // chunks of the four waves' rings
  static constexpr int ARR = RING > 4 * P::RED ? RING : 4 * P::RED;
};

template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dk_k(AttnArgs a, const bf16_t* __restrict__ ds,
                                                       bf16_t* __restrict__ dk, long ld_d) {
  using P = KvPlan<D>;
  using R = DkPlan<D>;
  constexpr int BK = P::BK, BQ = P::BQ, KK = D / 16, DB = D / 32, KR = R::KR;
  constexpr int NR = 2 * DB + 2;   // LDS reads of one 16-query step
  __shared__ uint4 sm[R::ARR];

  const int S = a.seq;
  const int grp = a.n_heads / a.n_kv_heads;
  const int per_kt = a.n_kv_heads * a.batch;
  const int kt = (int)blockIdx.x / per_kt;
  const int m = (int)blockIdx.x % per_kt % a.n_kv_heads;
  const int b = (int)blockIdx.x % per_kt / a.n_kv_heads;
  const int k0 = kt * BK;
  const int j0 = k0 / BQ;
  const int ns = (S + BQ - 1) / BQ - j0;
  const int total = grp * ns;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const long rb = (long)b * S;
  const DsLayout L(S);

  f32x16_t acc[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) zero(acc[db][kb]);

  uint32_t qoff[P::PER];
  slab_offsets<D>(a.ld_qkv, lane, qoff);
  uint32_t ro[KK], to[DB][2];
  frag_offsets<D>(lane, ro, to);
  // the (batch, key tile kt) dS blocks of query head n are consecutive:
  // pair p's block is ns - 1 - p / grp blocks after the tile's first
  const bf16_t* dsk = ds + L.tile(kt);
  uint4* ring = sm + wave * KR * R::SLOT;
  const uint32_t lb = lane * 16;   // the lane's 16 bytes of each 1 KB of a dS block (DMA)
  // the lane's B fragments in a dS block: half ss at ss * 1 KB + (pc ^ ss * 64)
  const uint32_t pc = (uint32_t)(512 * (lane >> 5) + ((16 * (lane & 31)) ^ (128 * (lane >> 5))));

  // pair p into ring slot u: the Q slab, then the dS block (four 1 KB DMA)
  auto load = [&](int p, int u) __attribute__((always_inline)) {
    const int n = m * grp + p % grp;
    const int q0 = (j0 + ns - 1 - p / grp) * BQ;
    uint4* slot = ring + u * R::SLOT;
    dma_slab<D>(a.q + rb * a.ld_qkv + (long)n * D, a.ld_qkv, q0, S, slot, qoff);
    const __amdgpu_buffer_rsrc_t r =
        rsrc(dsk + ((long)b * a.n_heads + n) * L.head + 2048L * (ns - 1 - p / grp));
    // (cache policy 2 = non-temporal: each dS block is read once by this
    // pass, so it need not displace the Q slabs every block re-reads from L2)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(slot + P::SLAB + i * 64), 16,
                                               lb + i * 1024, 0, 0, 2);
  };

  auto pair = [&](int u) __attribute__((always_inline)) {
    // this pair's DMA has landed once only the KR - 1 pairs issued after it
    // can still be in flight
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm((KR - 1) * R::MEM));
    __builtin_amdgcn_sched_barrier(0);
    const uint32_t ab = fa::lds_off(ring + u * R::SLOT);
    // both 16-query steps' fragments in flight; each step's MFMAs wait for
    // its own reads.
    bf16x8_t ft[2][DB], fb[2][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) ft[0][db] = fa::rd_tr<0>(ab + to[db][0], ab + to[db][1]);
    fb[0][0] = fa::rd_b128<P::SLAB * 16>(ab + pc);
    fb[0][1] = fa::rd_b128<P::SLAB * 16 + 2048>(ab + pc);
#pragma unroll
    for (int db = 0; db < DB; ++db)
      ft[1][db] = fa::rd_tr<16 * D * 2>(ab + to[db][0], ab + to[db][1]);
    fb[1][0] = fa::rd_b128<P::SLAB * 16 + 1024>(ab + (pc ^ 64));
    fb[1][1] = fa::rd_b128<P::SLAB * 16 + 2048 + 1024>(ab + (pc ^ 64));
    fa::wait_lds<NR>();
    fa::bind(fb[0][0]);
    fa::bind(fb[0][1]);
#pragma unroll
    for (int db = 0; db < DB; ++db) fa::bind(ft[0][db]);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      acc[db][0] = MFMA(ft[0][db], fb[0][0], acc[db][0]);
      acc[db][1] = MFMA(ft[0][db], fb[0][1], acc[db][1]);
    }
    __builtin_amdgcn_sched_barrier(0);
    fa::wait_lds<0>();
    fa::bind(fb[1][0]);
    fa::bind(fb[1][1]);
#pragma unroll
    for (int db = 0; db < DB; ++db) fa::bind(ft[1][db]);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      acc[db][0] = MFMA(ft[1][db], fb[1][0], acc[db][0]);
      acc[db][1] = MFMA(ft[1][db], fb[1][1], acc[db][1]);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // The wave's pairs p = wave + 4 i; pair i sits in slot i % KR. Every step
  // issues the same number of DMA instructions (past the last pair it
  // reloads the last pair, unused), so the wait count above is exact.
#pragma unroll
  for (int u = 0; u < KR - 1; ++u) load(min(wave + 4 * u, total - 1), u);
  bool done = false;
  for (int p = wave; !done; p += 4 * KR) {
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      if (!done) {
        const int pp = p + 4 * u;
        if (pp >= total) {
          done = true;
        } else {
          load(min(pp + 4 * (KR - 1), total - 1), (u + KR - 1) % KR);
          pair(u);
        }
      }
    }
  }
  kv_reduce_store<D>(acc, sm, sm + 2 * P::RED, wave, lane, a.scale,
                     dk + (rb + k0) * ld_d + (long)m * D, ld_d, S - k0);
}

// 4. dQ: block of 256 queries (32 per wave, eight waves) of one (batch,
// head), 64-key tiles up to the diagonal: dQ^T += K^T dS^T, both operands
// transposed reads from LDS: K^T from the natural K tile [64 keys][D], dS^T
// from the tile's eight dS blocks (wave w's 32 queries are block w), whose
// accumulator order holds four consecutive queries of one key in 8 bytes,
// the row piece ds_read_b64_tr_b16 transposes. Three stages in a ring, each
// tile's DMA issued two tiles ahead, and each wave waits only for the
// oldest stage's DMA. A wave whose queries all precede a tile skips it;
// blocks of a tile that do not exist (queries before the keys) are fetched
// as zeros.
template <int D>
struct DqPlan {
  static constexpr int BQ = 256, BKV = 64, NW = 8, NST = 3;
  static constexpr int NAT = BKV * D / 8;      // K tile chunks
  static constexpr int NDS = BKV * BQ / 8;     // dS tile chunks (eight 4 KB blocks)
  static constexpr int STAGE = NAT + NDS;
  static constexpr int MEM = DmaPlan<D, NW>::PER + NDS / 64 / NW;   // DMA per wave per tile
};

template <int D>
__global__ __launch_bounds__(512, 1) void attn_bwd_dq_k(AttnArgs a, const bf16_t* __restrict__ ds,
                                                       bf16_t* __restrict__ dq, long ld_d) {
  using Q = DqPlan<D>;
  constexpr int BQ = Q::BQ, BKV = Q::BKV, NAT = Q::NAT, NW = Q::NW, NST = Q::NST, DB = D / 32;
  __shared__ uint4 sm[NST * Q::STAGE];
  const int S = a.seq;
  const int nqt = (S + BQ - 1) / BQ;
  // block id: kv head fastest (the dispatcher spreads consecutive ids over
  // the XCDs, so each XCD's L2 holds the K of few kv heads), then the query
  // head within its group, batch, and query tile, largest first
  const int grp = a.n_heads / a.n_kv_heads;
  const int id = (int)blockIdx.x;
  const int m = id % a.n_kv_heads;
  const int n = m * grp + id / a.n_kv_heads % grp;
  const int b = id / a.n_kv_heads / grp % a.batch;
  const int qt = nqt - 1 - id / (a.n_kv_heads * grp * a.batch);
  const long rb = (long)b * S;
  const DsLayout L(S);
  const bf16_t* Kg = a.k + rb * a.ld_qkv + (long)m * D;
  const bf16_t* dsh = ds + ((long)b * a.n_heads + n) * L.head;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hh = lane >> 5, l32 = lane & 31;
  const int qb0 = qt * BQ;
  const int q0w = qb0 + wave * 32;
  const int q = q0w + l32;
  f32x16_t dqa[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) zero(dqa[db]);
  const int q_last = min(qb0 + BQ, S) - 1;
  const int nkt = q_last / BKV + 1;
  uint32_t koff[DmaPlan<D, NW>::PER];
  dma_offsets<D, NW>(a.ld_qkv, wave, lane, koff);
  // dS: instruction t of wave w copies KB c = 8 t + w of the tile, the
  // (c % 4)-th KB of block c / 4 (slab qb0 / 32 + c / 4); blocks past the
  // sequence end lie past the tile's extent and read as zeros
  auto dma = [&](int kt, int st) __attribute__((always_inline)) {
    uint4* stg = sm + st * Q::STAGE;
    dma_tile_at<D, NW>(Kg, a.ld_qkv, kt * BKV, S, stg, wave, koff);
    const int jb = qb0 / 32 - 2 * kt;   // block of slab qb0 / 32 in the tile (>= -6)
    const __amdgpu_buffer_rsrc_t r = rsrc_n(dsh + L.tile(kt), 4096L * (L.ns - 2 * kt));
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int c = t * NW + wave;
      const int blk = jb + c / 4;
      // non-temporal (cache policy 2): dS is read once here; K stays in L2
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (lds_ptr_t)(stg + NAT + c * 64), 16,
          blk < 0 ? kOOB : (uint32_t)((2048 * blk + ((c & 3) * 64 + lane) * 8) * 2), 0, 0, 2);
    }
  };
  // per-lane offsets: K^T fragments of column block db; the wave's dS^T
  // fragment of key step s: lane i of 16-lane group G supplies key
  // kr = 16 s + 4 (G >> 1) + (i >> 2) (+ 8 for the second read) and the four
  // queries 16 (G & 1) + 4 (i & 3) .. + 3, i.e. value quad g = 2 (G & 1) +
  // (i & 3) / 2 of lane half hh = i & 1: half u = G & 1, piece
  // 512 hh + ((16 kr) ^ (128 hh) ^ (64 u)), 8 bytes in at (g & 1) * 8; key step
  // s adds (s / 2) * 2 KB + (s % 2) * 256 B (bit 8: no XOR touches it), the
  // second read's + 8 keys sets bit 7 and so has offsets of its own
  uint32_t ro[D / 16], to[DB][2];
  frag_offsets<D>(lane, ro, to);
  uint32_t ts[2];
  {
    const int G = lane >> 4, i = lane & 15;
    const int kr = 4 * (G >> 1) + (i >> 2);
    const int hh = i & 1, u = G & 1;
#pragma unroll
    for (int hi = 0; hi < 2; ++hi)
      ts[hi] = NAT * 16 + wave * 4096 + u * 1024 + 512 * hh +
               ((16 * (kr + 8 * hi)) ^ (128 * hh) ^ (64 * u)) + ((i & 3) >> 1) * 8;
  }
  const uint32_t smb = fa::lds_off(sm);
  // one key step's fragments: the dS^T fragment, then the DB K^T fragments
  // (2 (DB + 1) LDS reads, inline asm: a C++ read would make the compiler
  // wait for every DMA in flight first)
  auto rd_step = [&](auto SV, uint32_t sb, bf16x8_t& bt, bf16x8_t (&at)[DB])
      __attribute__((always_inline)) {
    constexpr int s = decltype(SV)::value;
    constexpr int SO = (s >> 1) * 2048 + (s & 1) * 256, KO = s * 16 * D * 2;
    bt = fa::rd_tr<SO>(sb + ts[0], sb + ts[1]);
#pragma unroll
    for (int db = 0; db < DB; ++db) at[db] = fa::rd_tr<KO>(sb + to[db][0], sb + to[db][1]);
  };
  auto mfma_step = [&](bf16x8_t& bt, bf16x8_t (&at)[DB]) __attribute__((always_inline)) {
    fa::bind(bt);
#pragma unroll
    for (int db = 0; db < DB; ++db) fa::bind(at[db]);
#pragma unroll
    for (int db = 0; db < DB; ++db) dqa[db] = MFMA(at[db], bt, dqa[db]);
    __builtin_amdgcn_sched_barrier(0);
  };
  auto tile = [&](int kt, int st) __attribute__((always_inline)) {
    if (kt * BKV > q0w + 31) return;   // every query of this wave precedes the tile
    const uint32_t sb = smb + st * Q::STAGE * 16;
    constexpr int NRS = 2 * (DB + 1);   // reads of one key step
    bf16x8_t bt[4], at[4][DB];
    // each step's reads go out before the previous step's MFMAs
    rd_step(fa::ic<0>{}, sb, bt[0], at[0]);
    rd_step(fa::ic<1>{}, sb, bt[1], at[1]);
    fa::wait_lds<NRS>();
    mfma_step(bt[0], at[0]);
    rd_step(fa::ic<2>{}, sb, bt[2], at[2]);
    fa::wait_lds<NRS>();
    mfma_step(bt[1], at[1]);
    rd_step(fa::ic<3>{}, sb, bt[3], at[3]);
    fa::wait_lds<NRS>();
    mfma_step(bt[2], at[2]);
    fa::wait_lds<0>();
    mfma_step(bt[3], at[3]);
  };
  // after the wait, every wave's DMA of the tile about to be read has landed
  // and every wave is done with the stage the next DMA overwrites
  auto sync = [&](bool ahead) __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    if (ahead) __builtin_amdgcn_s_waitcnt(vmcnt_imm(Q::MEM));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  dma(0, 0);
  if (nkt > 1) dma(1, 1);
  sync(nkt > 1);
  int st = 0;
  for (int kt = 0; kt < nkt; ++kt) {
    if (kt + 2 < nkt) dma(kt + 2, st == 0 ? 2 : st - 1);
    tile(kt, st);
    if (kt + 1 < nkt) sync(kt + 2 < nkt);
    st = st == NST - 1 ? 0 : st + 1;
  }
  if (q < S) {
    bf16_t* dqr = dq + (rb + q) * ld_d + (long)n * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
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
  const dim3 grid((unsigned)((a.seq + 127) / 128 * a.n_heads * a.batch)), block(256);
  if (a.d == 128) hipLaunchKernelGGL(attn_fwd_k<128>, grid, block, 0, s, a, o, lse);
  else if (a.d == 64) hipLaunchKernelGGL(attn_fwd_k<64>, grid, block, 0, s, a, o, lse);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

size_t attn_bwd_ds_bytes(const AttnArgs& a) {
  return (size_t)a.batch * a.n_heads * DsLayout(a.seq).head * 2;
}

hipError_t attn_bwd(const AttnArgs& a, const uint16_t* o, const uint16_t* dout, const float* lse,
                    float* delta, uint16_t* ds, uint16_t* dq, uint16_t* dk, uint16_t* dv,
                    long ld_d, hipStream_t s) {
  const long rows = (long)a.batch * a.seq * a.n_heads;
  const dim3 block(256);
  const dim3 kgrid((unsigned)((a.seq + 63) / 64 * a.n_kv_heads * a.batch));
  const dim3 qgrid((unsigned)((a.seq + 255) / 256 * a.n_heads * a.batch));
  if (a.d == 128) {
    const dim3 pgrid((unsigned)((rows + 15) / 16));
    hipLaunchKernelGGL(attn_bwd_prep_k<128>, pgrid, block, 0, s, o, dout, lse, delta, rows,
                       a.n_heads, a.seq);
    hipLaunchKernelGGL(attn_bwd_dv_k<128>, kgrid, block, 0, s, a, dout, delta, ds, dv, ld_d);
    hipLaunchKernelGGL(attn_bwd_dk_k<128>, kgrid, block, 0, s, a, ds, dk, ld_d);
    hipLaunchKernelGGL(attn_bwd_dq_k<128>, qgrid, dim3(512), 0, s, a, ds, dq, ld_d);
  } else if (a.d == 64) {
    const dim3 pgrid((unsigned)((rows + 31) / 32));
    hipLaunchKernelGGL(attn_bwd_prep_k<64>, pgrid, block, 0, s, o, dout, lse, delta, rows,
                       a.n_heads, a.seq);
    hipLaunchKernelGGL(attn_bwd_dv_k<64>, kgrid, block, 0, s, a, dout, delta, ds, dv, ld_d);
    hipLaunchKernelGGL(attn_bwd_dk_k<64>, kgrid, block, 0, s, a, ds, dk, ld_d);
    hipLaunchKernelGGL(attn_bwd_dq_k<64>, qgrid, dim3(512), 0, s, a, ds, dq, ld_d);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace forge

// bf16 GEMM on gfx950 MFMA, fp32 accumulation.
//
// Every projection of the layer is one of three products (App. C: the
// backward of each GEMM is one data-gradient and one weight-gradient
// product): y = x W^T (both operands K-contiguous), dX = dY W (W is
// N-contiguous) and dW += dY^T X (both operands M/N-contiguous, reduction
// over tokens). Two pipelines share tile order, operand layouts and epilogue
// stores:
//
//  * ring_kernel (every layout; all 256 x 256 tiles): v_mfma_f32_16x16x32_bf16
//    over a ring of four 32-deep LDS stages, one MFMA k-step per stage. The
//    barrier that publishes stage s + 1 sits two MFMAs into stage s; after it
//    the fragment reads of stage s + 1 and the DMA of stage s + 4 (into the
//    slot stage s has just released) are spread evenly over the stage's
//    MFMAs, so neither the LDS nor the texture unit sees a burst. Fragment
//    reads are inline asm with explicit lgkmcnt waits: the compiler cannot
//    tell the transposing reads apart from the DMA writes and would otherwise
//    wait for every outstanding DMA before each of them. The 16x16x32 shape
//    does the work of 32x32x16 at the same rate per cycle with less power,
//    which keeps the clock higher under load.
//  * gemm_kernel (K-contiguous 256 x 192 and small tiles): v_mfma_f32_32x32x16
//    over a block tile BM x BN x 64 double-buffered in LDS, one barrier per
//    k-step placed before the step's last 16-deep slice; the barrier also
//    frees the current buffer, which is refilled at once with the step after
//    next.
//  * Tiles are filled by buffer_load ... lds (global to LDS without
//    registers); out-of-range chunks read as zeros through the buffer
//    descriptor's range check, so ragged edges need no branches.
//  * A K-contiguous operand tile keeps 128-byte rows (eight 16-byte chunks,
//    chunk c of row r at c ^ ((r ^ (r >> 3)) & 7)) in gemm_kernel and 64-byte
//    rows (chunk c of row r at c ^ ((r >> 1) & 3)) in a ring stage; either
//    way the eight lanes a 16-byte read serves per cycle cover a 128-byte
//    bank window once (no bank conflicts). Each MFMA operand is one 16-byte
//    LDS read. An operand contiguous along M / N is
//    stored as it lies in HBM (chunks XOR-swizzled per k-row) and read with
//    gfx950's ds_read_b64_tr_b16 transpose reads, so dgrad and wgrad need no
//    transpose pass.
//  * The MFMA computes D = Btile * Atile^T, i.e. C transposed, so each lane's
//    four consecutive accumulator rows are four consecutive n of one row m of
//    C: the epilogue writes 16-byte fp32 vectors, and in the ring kernel
//    lanes l and l ^ 16 swap halves so that each writes eight consecutive
//    bf16 (one 16-byte nontemporal store). The AdamW epilogues of the grouped
//    weight gradients stage the fp32 tile through the free stage ring and
//    stream it by rows through the optimizer state (adam_tile).
//  * Workgroups are dispatched round-robin over the 8 XCDs; the tile order is
//    remapped so each XCD works on a contiguous, M-grouped band of tiles and
//    reuses operands in its own L2.
#include "common.h"
#include "kernels.h"

namespace forge {
namespace {

constexpr int BK = 64;
constexpr int CHUNKS = BK / 8;  // 16-byte chunks per LDS tile row
constexpr int GROUP_M = 8;
constexpr int NUM_XCD = 8;

__device__ __forceinline__ int wave_incl_scan_int(int v) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d, 64);
    if ((int)(threadIdx.x & 63) >= d) v += u;
  }
  return v;
}
__device__ __forceinline__ int wave_sum_int(int v) { return __shfl(wave_incl_scan_int(v), 63, 64); }

__device__ __forceinline__ int swz(int row, int c) {
  return row * CHUNKS + (c ^ ((row ^ (row >> 3)) & 7));
}

// ---- buffer resources ------------------------------------------------------
// Raw buffer loads return zero for an offset past num_records, so every
// out-of-range chunk (ragged M/N edge, K tail) is fetched as zeros without a
// branch: the address of a chunk that is out of range is set to kOOB.
constexpr uint32_t kOOB = 0x80000000u;
constexpr uint32_t kRecords = 0x7FFFFFF0u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)kRecords,
                                           0x00020000);
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// ---- K-contiguous source: global -> LDS directly (no register staging) ----
// Each wave-wide buffer_load_dwordx4 ... lds writes 1 KB of LDS: 8 tile rows
// of 128 bytes, lane l landing at byte 16*l. Lane l therefore fetches the
// logical chunk that the swizzle places at physical slot l % 8 of row l / 8.
template <int ROWS, int NW>
struct KcLoader {
  static constexpr int PER = ROWS / 8 / NW;
  static_assert(PER * 8 * NW == ROWS, "tile rows must split over waves");
  __device__ __forceinline__ void load(const bf16_t* __restrict__ src, long ld, int row0,
                                       int rows_lim, int k0, int K, uint4* lds, int wave,
                                       int lane) const {
    const __amdgpu_buffer_rsrc_t r = rsrc(src + (long)row0 * ld + k0);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int blk = i * NW + wave;
      const int row = blk * 8 + (lane >> 3);
      const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
      const bool ok = (row0 + row < rows_lim) && (k0 + c * 8 < K);
      const uint32_t off = ok ? (uint32_t)(((long)row * ld + c * 8) * 2) : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(lds + blk * 64), 16, off, 0, 0, 0);
    }
  }
};

// Fragment of rows base..base+31 (the lane's row is base + lane % 32) over
// k-slice kk: eight consecutive k starting at kk*16 + 8*(lane / 32).
__device__ __forceinline__ bf16x8_t frag(const uint4* tile, int base, int kk, int lane) {
  return __builtin_bit_cast(bf16x8_t, tile[swz(base + (lane & 31), kk * 2 + (lane >> 5))]);
}

// ---- epilogue: four consecutive n of row m ---------------------------------
// fp32 C (and the C it accumulates into) goes through nontemporal accesses: a
// round of 256 x 256 tiles writes about as much C per XCD as the XCD's L2
// holds, and ordinary stores would evict the operand rows that the next tiles
// read there. bf16 pieces of 8 bytes stay ordinary stores (streaming stores
// that small are slower than the eviction they avoid).
template <int EPI>
__device__ __forceinline__ void store4(const GemmArgs& p, int m, int n, const float* vin) {
  if (m >= p.M) return;
  const bool full = (n + 3 < p.N);
  const float v[4] = {vin[0] * p.alpha, vin[1] * p.alpha, vin[2] * p.alpha, vin[3] * p.alpha};
  if (EPI == kStoreBF16 || EPI == kResidBF16) {
    bf16_t* C = reinterpret_cast<bf16_t*>(p.C) + (long)m * p.ldc + n;
    float x[4] = {v[0], v[1], v[2], v[3]};
    if (EPI == kResidBF16) {
      const bf16_t* R = p.R + (long)m * p.ldr + n;
      if (full) {
        const uint2 r = *reinterpret_cast<const uint2*>(R);
        x[0] += lo_f(r.x); x[1] += hi_f(r.x); x[2] += lo_f(r.y); x[3] += hi_f(r.y);
      } else {
        for (int e = 0; e < 4; ++e)
          if (n + e < p.N) x[e] += bf2f(R[e]);
      }
    }
    if (full) {
      *reinterpret_cast<uint2*>(C) = make_uint2(pack2(x[0], x[1]), pack2(x[2], x[3]));
    } else {
      for (int e = 0; e < 4; ++e)
        if (n + e < p.N) C[e] = f2bf(x[e]);
    }
  } else {
    float* C = reinterpret_cast<float*>(p.C) + (long)m * p.ldc + n;
    if (full) {
      f32x4_t o = {v[0], v[1], v[2], v[3]};
      if (EPI == kAccF32) o += __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(C));
      __builtin_nontemporal_store(o, reinterpret_cast<f32x4_t*>(C));
    } else {
      for (int e = 0; e < 4; ++e)
        if (n + e < p.N) C[e] = (EPI == kAccF32 ? C[e] : 0.0f) + v[e];
    }
  }
}

// ---- epilogue of a 32x32 block: lane holds C[m][n..n+3] for 4 groups ------
template <int EPI, int FN, int FM>
__device__ __forceinline__ void store_tile(const GemmArgs& p, const f32x16_t (&acc)[FN][FM],
                                           int mw, int nw, int lane) {
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int m = mw + j * 32 + (lane & 31);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = nw + i * 32 + g * 8 + (lane >> 5) * 4;
        float v[4] = {acc[i][j][g * 4 + 0], acc[i][j][g * 4 + 1], acc[i][j][g * 4 + 2],
                      acc[i][j][g * 4 + 3]};
        store4<EPI>(p, m, n, v);
      }
    }
}

// Tile of this workgroup (tm, tn) and the group-adjusted arguments; false
// when the workgroup has no tile (M-grouped launches over-provision).
template <int BM, int BN, int EPI, int GROUP>
__device__ __forceinline__ bool tile_setup(GemmArgs& p, int& tm, int& tn) {
  if (GROUP == 0) {
    // ---- tile order: XCD-contiguous bands, GROUP_M rows of tiles per band ----
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int nb = gridDim.x;
    const int bid = blockIdx.x;
    const int nb8 = nb - nb % NUM_XCD;
    const int pid = bid < nb8 ? (bid % NUM_XCD) * (nb8 / NUM_XCD) + bid / NUM_XCD : bid;
    const int in_group = GROUP_M * tiles_n;
    const int first_m = (pid / in_group) * GROUP_M;
    const int gsize = min(tiles_m - first_m, GROUP_M);
    tm = first_m + (pid % in_group) % gsize;
    tn = (pid % in_group) / gsize;
  } else if (GROUP == 1) {
    // M-grouped. The grid is an upper bound (host does not know the group
    // sizes); the real tiles are counted from the device offsets and dealt
    // to the 8 XCDs (workgroup b runs on XCD b % 8) as balanced contiguous
    // ranges. Within a range, group by group, n-tile major with the group's
    // m-tiles consecutive: a B_e column block is reused from L2 by all of the
    // group's m-tiles, an A row block by neighbouring n-tiles.
    const int tiles_n = (p.N + BN - 1) / BN;
    // group sizes in m-tiles, 64 groups per wave-wide step (one coalesced
    // load, a lane per group, prefix sums across the wave)
    const int ln = threadIdx.x & 63;
    int total = 0;
    for (int base = 0; base < p.groups; base += 64) {
      const int g = base + ln;
      const int mt = g < p.groups ? (p.g_off[g + 1] - p.g_off[g] + BM - 1) / BM : 0;
      total += wave_sum_int(mt);
    }
    const int real = total * tiles_n;
    const int per = (real + NUM_XCD - 1) / NUM_XCD;
    const int li = blockIdx.x / NUM_XCD;
    const int pid = (blockIdx.x % NUM_XCD) * per + li;
    if (li >= per || pid >= real) return false;
    int e = 0, acc = 0, mte = 1;
    for (int base = 0; base < p.groups; base += 64) {
      const int g = base + ln;
      const int mt = g < p.groups ? (p.g_off[g + 1] - p.g_off[g] + BM - 1) / BM : 0;
      const int incl = wave_incl_scan_int(mt * tiles_n);
      const int excl = incl - mt * tiles_n;
      const uint64_t hit = __ballot(mt > 0 && pid >= acc + excl && pid < acc + incl);
      if (hit) {
        const int l = __ffsll((unsigned long long)hit) - 1;
        e = base + l;
        mte = __shfl(mt, l, 64);
        acc += __shfl(excl, l, 64);
        break;
      }
      acc += __shfl(incl, 63, 64);
    }
    e = __builtin_amdgcn_readfirstlane(e);
    mte = __builtin_amdgcn_readfirstlane(mte);
    acc = __builtin_amdgcn_readfirstlane(acc);
    tm = (pid - acc) % mte;
    tn = (pid - acc) / mte;
    const long r0 = p.g_off[e];
    p.M = p.g_off[e + 1] - p.g_off[e];
    p.A += r0 * p.lda;  // K-contiguous A: group rows are row blocks
    p.B += (long)e * p.strideB;
    p.C = (char*)p.C + r0 * p.ldc * (EPI == kStoreBF16 || EPI == kResidBF16 ? 2 : 4);
    if (EPI == kResidBF16) p.R += r0 * p.ldr;
  } else if (GROUP == 4) {
    // the last, partial round of a product of 2BN-wide tiles: full tile
    // p.tile_base + i of the band order above runs as two BN-wide halves
    // (workgroups 2i and 2i + 1 after the same XCD remapping), so the round
    // fills twice as many CUs with half as much work each
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + 2 * BN - 1) / (2 * BN);
    const int nb = gridDim.x, bid = blockIdx.x;
    const int nb8 = nb - nb % NUM_XCD;
    const int ph = bid < nb8 ? (bid % NUM_XCD) * (nb8 / NUM_XCD) + bid / NUM_XCD : bid;
    const int pid = p.tile_base + ph / 2;
    const int in_group = GROUP_M * tiles_n;
    const int first_m = (pid / in_group) * GROUP_M;
    const int gsize = min(tiles_m - first_m, GROUP_M);
    tm = first_m + (pid % in_group) % gsize;
    tn = 2 * ((pid % in_group) / gsize) + (ph & 1);
  } else if (GROUP == 3) {
    // uniform split of the reduction: split e covers k rows [e * ks, e * ks + ks)
    // (ks = p.strideB) and stores its partial product to C + e * strideC
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int e = blockIdx.x / (tiles_m * tiles_n);
    const int t = blockIdx.x % (tiles_m * tiles_n);
    tm = t / tiles_n;
    tn = t % tiles_n;
    const long k0 = (long)e * p.strideB;
    p.K = (int)min((long)p.K - k0, p.strideB);
    p.A += k0 * p.lda;  // both operands M/N-contiguous: k rows
    p.B += k0 * p.ldb;
    p.C = (char*)p.C + (long)e * p.strideC * 4;
  } else {
    // K-grouped: one (m, n) tile grid per group, reduction over the group's
    // rows; XCD-contiguous ranges of tiles, group by group
    const int tiles_m = (p.M + BM - 1) / BM;
    const int tiles_n = (p.N + BN - 1) / BN;
    const int nb = gridDim.x, bid = blockIdx.x;
    const int nb8 = nb - nb % NUM_XCD;
    const int pid = bid < nb8 ? (bid % NUM_XCD) * (nb8 / NUM_XCD) + bid / NUM_XCD : bid;
    const int e = pid / (tiles_m * tiles_n);
    const int t = pid % (tiles_m * tiles_n);
    tm = t / tiles_n;
    tn = t % tiles_n;
    const long r0 = p.g_off[e];
    p.K = p.g_off[e + 1] - p.g_off[e];
    p.A += r0 * p.lda;  // both operands M/N-contiguous: group rows are k rows
    p.B += r0 * p.ldb;
    p.C = (char*)p.C + (long)e * p.strideC * 4;
    if (EPI == kStoreF32Adam || EPI == kAccF32Adam) {
      const long off = (long)e * p.strideC;
      p.o_master += off;
      p.o_m += off;
      p.o_v += off;
      p.o_param += off;
    }
  }
  return true;
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int LA, int LB, int EPI, int GROUP = 0>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64, 1) void gemm_kernel(GemmArgs p) {
  static_assert(LA == kKC && LB == kKC, "the double-buffered kernel takes K-contiguous operands");
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int FM = WM / 32, FN = WN / 32;
  static_assert(FM * 32 == WM && FN * 32 == WN, "wave tile must be a multiple of 32");
  constexpr int A_ELEMS = BM * CHUNKS, B_ELEMS = BN * CHUNKS;
  __shared__ uint4 lds[2][A_ELEMS + B_ELEMS];

  int tm, tn;
  if (!tile_setup<BM, BN, EPI, GROUP>(p, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  constexpr int NW = WAVES_M * WAVES_N;

  KcLoader<BM, NW> la;
  KcLoader<BN, NW> lb;

  f32x16_t acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  // ---- main loop: the barrier that publishes tile t+1 sits before the last
  // 16-deep k-slice of tile t, so every wave leaves it with that slice's
  // MFMAs to issue while the first fragments of tile t+1 are read; right
  // after it, tile t+2 is loaded into tile t's buffer.
  const int nk = (p.K + BK - 1) / BK;
  constexpr int KS = BK / 16;
  la.load(p.A, p.lda, m0, p.M, 0, p.K, lds[0], wave, lane);
  lb.load(p.B, p.ldb, n0, p.N, 0, p.K, lds[0] + A_ELEMS, wave, lane);
  __syncthreads();
  bf16x8_t fa[2][FN], fb[2][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i) fa[0][i] = frag(lds[0] + A_ELEMS, wn * WN + i * 32, 0, lane);
#pragma unroll
  for (int j = 0; j < FM; ++j) fb[0][j] = frag(lds[0], wm * WM + j * 32, 0, lane);
  // tile 1 into the second buffer (past the end: zeros into an unused buffer)
  la.load(p.A, p.lda, m0, p.M, BK, p.K, lds[1], wave, lane);
  lb.load(p.B, p.ldb, n0, p.N, BK, p.K, lds[1] + A_ELEMS, wave, lane);

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const uint4* At = lds[cur];
    const uint4* Bt = lds[cur] + A_ELEMS;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int cb = kk & 1, nx = cb ^ 1;
      if (kk + 1 < KS) {
#pragma unroll
        for (int i = 0; i < FN; ++i) fa[nx][i] = frag(Bt, wn * WN + i * 32, kk + 1, lane);
#pragma unroll
        for (int j = 0; j < FM; ++j) fb[nx][j] = frag(At, wm * WM + j * 32, kk + 1, lane);
      } else {
        // publish tile t+1: this wave's DMA has landed and its reads of tile
        // t are complete; after the barrier every wave's are
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        const uint4* An = lds[cur ^ 1];
        const uint4* Bn = lds[cur ^ 1] + A_ELEMS;
#pragma unroll
        for (int i = 0; i < FN; ++i) fa[nx][i] = frag(Bn, wn * WN + i * 32, 0, lane);
#pragma unroll
        for (int j = 0; j < FM; ++j) fb[nx][j] = frag(An, wm * WM + j * 32, 0, lane);
        // every wave's reads of tile t are complete: its buffer takes tile
        // t+2 (all zeros past the end)
        la.load(p.A, p.lda, m0, p.M, (kt + 2) * BK, p.K, lds[cur], wave, lane);
        lb.load(p.B, p.ldb, n0, p.N, (kt + 2) * BK, p.K, lds[cur] + A_ELEMS, wave, lane);
      }
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cb][i], fb[cb][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  __builtin_amdgcn_s_waitcnt(0);  // the last (all-zero) tile loads land before exit
  store_tile<EPI, FN, FM>(p, acc, m0 + wm * WM, n0 + wn * WN, lane);
}

// ---- ring pipeline: four 32-deep stages, 16x16x32 MFMAs ---------------------
// Stage slot = A part then B part. K-contiguous operand: ROWS rows of four
// 16-byte chunks (k 0..31), chunk c of row r at c ^ ((r >> 2) & 3).
// M/N-contiguous operand: 32 k-rows of ROWS elements, 16-byte chunk c of
// k-row k at c ^ ((k & 3) << 2) ^ (((k >> 3) & 1) << 1). A fragment read
// touches k-rows {0..3} and {8..11} (or their +4 / +16 shifts) in one
// half-wave; the two XOR terms put those eight rows' 32-byte pieces on
// distinct banks.
constexpr int SK = 32;

template <int ROWS, int NW>
struct RingPart {
  static constexpr int ELEMS = ROWS * 4;         // 16-byte chunks per stage
  static constexpr int PER = ROWS * 4 / 64 / NW;  // DMA instructions per wave per stage
  static_assert(PER * 64 * NW == ROWS * 4, "stage tile must split over the waves");
};

// K-contiguous stage: 64-byte rows (four 16-byte chunks), two rows per 128-byte
// bank window. A ds_read_b128 serves eight lanes per cycle, here eight
// consecutive rows at one logical chunk: XOR-ing the chunk with (row / 2) % 4
// puts the four rows of each parity on four different slots, so the eight
// reads cover the window once (keying on row / 4 left two rows per slot, a
// two-way conflict on every fragment read).
__device__ __forceinline__ int kc_swz(int row) { return (row >> 1) & 3; }
__device__ __forceinline__ int kc4(int row, int c) { return row * 4 + (c ^ kc_swz(row)); }

__device__ __forceinline__ int mc_swz(int k) { return ((k & 3) << 2) ^ (((k >> 3) & 1) << 1); }

template <int ROWS>
__device__ __forceinline__ int mc_ring_elem(int k, int m) {
  return k * ROWS + (((m >> 3) ^ mc_swz(k)) << 3) + (m & 7);
}

__device__ __forceinline__ uint32_t lds_addr(const void* ptr) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)ptr;
}

// DMA instruction i (of RingPart::PER) of this wave for one operand of a stage.
template <int ROWS, int NW, int LAYOUT>
__device__ __forceinline__ void ring_dma(int i, const bf16_t* __restrict__ src, long ld, int row0,
                                         int rows_lim, int k0, int K, uint4* part, int wave,
                                         int lane) {
  const int blk = i * NW + wave;  // 1 KB block of the stage's part
  if (LAYOUT == kKC) {
    const __amdgpu_buffer_rsrc_t r = rsrc(src + (long)row0 * ld + k0);
    const int row = blk * 16 + (lane >> 2);
    const int c = (lane & 3) ^ kc_swz(row);
    const bool ok = (row0 + row < rows_lim) && (k0 + c * 8 < K);
    const uint32_t off = ok ? (uint32_t)(((long)row * ld + c * 8) * 2) : kOOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(part + blk * 64), 16, off, 0, 0, 0);
  } else {
    constexpr int LPR = ROWS / 8;  // lanes per k-row
    constexpr int RPI = 64 / LPR;  // k-rows per instruction
    static_assert(LPR >= 16, "the swizzle needs at least 16 chunks per k-row");
    const __amdgpu_buffer_rsrc_t r = rsrc(src + (long)k0 * ld + row0);
    const int k = blk * RPI + lane / LPR;
    const int c = (lane % LPR) ^ mc_swz(k);
    const bool ok = (k0 + k < K) && (row0 + c * 8 < rows_lim);
    const uint32_t off = ok ? (uint32_t)(((long)k * ld + c * 8) * 2) : kOOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(part + blk * 64), 16, off, 0, 0, 0);
  }
}

// 16x16x32 operand of rows base..base+15 over a whole stage: the lane holds
// row base + lane % 16, k = 8 (lane / 16) .. + 7. Issued as asm (not tracked
// by the compiler: ring_fence waits for it). M/N-contiguous: two transposing
// reads, lane 4r + j of each 16-lane group pointing at k-row r, elements
// 4j..4j+3 of a 4 x 16 block.
template <int LAYOUT, int ROWS>
__device__ __forceinline__ bf16x8_t ring_frag(const uint4* part, int base, int lane) {
  if (LAYOUT == kKC) {
    const uint32_t a = lds_addr(part + kc4(base + (lane & 15), lane >> 4));
    uint4 r;
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(a) : "memory");
    return __builtin_bit_cast(bf16x8_t, r);
  } else {
    const uint16_t* t = reinterpret_cast<const uint16_t*>(part);
    const int g = lane >> 4, i = lane & 15;
    const int m = base + 4 * (i & 3);
    const int k = g * 8 + (i >> 2);
    const uint32_t a0 = lds_addr(t + mc_ring_elem<ROWS>(k, m));
    const uint32_t a1 = lds_addr(t + mc_ring_elem<ROWS>(k + 4, m));
    uint2 lo, hi;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a0) : "memory");
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(hi) : "v"(a1) : "memory");
    return __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
  }
}

// Wait for every outstanding LDS read; the fragments count as rewritten here,
// so nothing that uses (or reuses the registers of) them moves above the wait.
template <int FN, int FM>
__device__ __forceinline__ void ring_fence(bf16x8_t (&fa)[FN], bf16x8_t (&fb)[FM]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < FN; ++i) asm volatile("" : "+v"(fa[i]));
#pragma unroll
  for (int j = 0; j < FM; ++j) asm volatile("" : "+v"(fb[j]));
}

// At most N DMA instructions of this wave still outstanding.
template <int N>
__device__ __forceinline__ void wait_dma() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---- bf16 epilogue: eight consecutive n of row m ---------------------------
// A full piece is one 16-byte nontemporal store (see store4): with whole
// 16-byte pieces, 64 contiguous bytes per row and instruction, streaming
// stores keep the XCD's L2 for the operand rows.
template <int EPI>
__device__ __forceinline__ void store8_bf16(const GemmArgs& p, int m, int n, float* x) {
  if (m >= p.M) return;
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] *= p.alpha;
  bf16_t* C = reinterpret_cast<bf16_t*>(p.C) + (long)m * p.ldc + n;
  const bool full = (n + 7 < p.N);
  if (EPI == kResidBF16) {
    const bf16_t* R = p.R + (long)m * p.ldr + n;
    if (full) {
      float r[8];
      unpack8(*reinterpret_cast<const uint4*>(R), r);
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] += r[e];
    } else {
      for (int e = 0; e < 8; ++e)
        if (n + e < p.N) x[e] += bf2f(R[e]);
    }
  }
  if (full) {
    __builtin_nontemporal_store(__builtin_bit_cast(f32x4_t, pack8(x)), reinterpret_cast<f32x4_t*>(C));
  } else {
    for (int e = 0; e < 8; ++e)
      if (n + e < p.N) C[e] = f2bf(x[e]);
  }
}

// ---- epilogue of 16x16 blocks: lane holds C[m][n..n+3] ---------------------
// bf16 output: lanes l and l ^ 16 swap halves of two neighbouring blocks so
// that each lane holds eight consecutive n, and a row takes 64 contiguous
// bytes per store instruction.
// AdamW epilogue of C[m][n..n+3] (kStoreF32Adam / kAccF32Adam): the weight
// gradient g (acc, or C + acc, rounded as the plain fp32 epilogues round it)
// is stored to C, then the same elements of the optimizer state are updated
// exactly as the standalone AdamW kernel does (adam1; sc = lr, 1 / bc1,
// 1 / bc2, clip). Every stream is touched once: nontemporal accesses.
struct AdamPiece {
  f32x4_t g, w, m1, m2;
};

template <int EPI>
__device__ __forceinline__ void adam_load(const GemmArgs& p, int m, int n, const float* v,
                                          AdamPiece& a) {
  a.g = f32x4_t{v[0] * p.alpha, v[1] * p.alpha, v[2] * p.alpha, v[3] * p.alpha};
  if (m >= p.M || n + 3 >= p.N) return;  // ragged pieces: adam_store, element by element
  const long i = (long)m * p.ldc + n;
  if (EPI == kAccF32Adam)
    a.g += __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>((float*)p.C + i));
  a.w = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p.o_master + i));
  a.m1 = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p.o_m + i));
  a.m2 = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p.o_v + i));
}

template <int EPI>
__device__ __forceinline__ void adam_store(const GemmArgs& p, const float* sc, int m, int n,
                                           AdamPiece& a) {
  if (m >= p.M) return;
  const long i = (long)m * p.ldc + n;
  float* C = reinterpret_cast<float*>(p.C) + i;
  if (n + 3 < p.N) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float we = a.w[e], me = a.m1[e], ve = a.m2[e];
      adam1(we, me, ve, a.g[e], p.o_b1, p.o_b2, p.o_eps, p.o_wd, sc[0], sc[1], sc[2], sc[3]);
      a.w[e] = we;
      a.m1[e] = me;
      a.m2[e] = ve;
    }
    __builtin_nontemporal_store(a.g, reinterpret_cast<f32x4_t*>(C));
    __builtin_nontemporal_store(a.w, reinterpret_cast<f32x4_t*>(p.o_master + i));
    __builtin_nontemporal_store(a.m1, reinterpret_cast<f32x4_t*>(p.o_m + i));
    __builtin_nontemporal_store(a.m2, reinterpret_cast<f32x4_t*>(p.o_v + i));
    const u32x2_t pb = {pack2(a.w[0], a.w[1]), pack2(a.w[2], a.w[3])};
    __builtin_nontemporal_store(pb, reinterpret_cast<u32x2_t*>(p.o_param + i));
  } else {
    for (int e = 0; e < 4; ++e)
      if (n + e < p.N) {
        const float g = (EPI == kAccF32Adam ? C[e] : 0.0f) + a.g[e];
        C[e] = g;
        float we = p.o_master[i + e], me = p.o_m[i + e], ve = p.o_v[i + e];
        adam1(we, me, ve, g, p.o_b1, p.o_b2, p.o_eps, p.o_wd, sc[0], sc[1], sc[2], sc[3]);
        p.o_master[i + e] = we;
        p.o_m[i + e] = me;
        p.o_v[i + e] = ve;
        p.o_param[i + e] = f2bf(we);
      }
  }
}

template <int EPI, int FN, int FM>
__device__ __forceinline__ void store_tile16(const GemmArgs& p, const f32x4_t (&acc)[FN][FM],
                                             int mw, int nw, int lane) {
  if constexpr (EPI == kStoreBF16 || EPI == kResidBF16) {
    static_assert(FN % 2 == 0, "bf16 epilogue pairs neighbouring n-blocks");
    const int g = lane >> 4;
    const bool even = (g & 1) == 0;
#pragma unroll
    for (int i = 0; i < FN; i += 2)
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        const int m = mw + j * 16 + (lane & 15);
        float x[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float send = even ? acc[i + 1][j][e] : acc[i][j][e];
          const float recv = __shfl_xor(send, 16);
          x[e] = even ? acc[i][j][e] : recv;
          x[4 + e] = even ? recv : acc[i + 1][j][e];
        }
        const int n = nw + (even ? i * 16 + g * 4 : (i + 1) * 16 + (g - 1) * 4);
        store8_bf16<EPI>(p, m, n, x);
      }
  } else {
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        const int m = mw + j * 16 + (lane & 15);
        const int n = nw + i * 16 + (lane >> 4) * 4;
        const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4<EPI>(p, m, n, v);
      }
  }
}

// AdamW epilogue of a whole tile (kStoreF32Adam / kAccF32Adam), through LDS:
// the tile goes to the stage ring (free after the loop) as fp32, half of its
// rows at a time, and comes back row by row, so that each wave streams whole
// tile rows (1 KB per instruction for 256 columns) through the update's
// streams (C, master, m and v in; those and the bf16 parameter out) instead
// of 64-byte pieces of 16 rows, with the loads of U rows issued together.
// Chunks are XOR-swizzled by row so that the column writes of 16 rows and
// the row reads are both free of bank conflicts.
template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI, int FN, int FM>
__device__ __forceinline__ void adam_tile(const GemmArgs& p, const f32x4_t (&acc)[FN][FM],
                                          float* lds, int m0, int n0, int wm, int wn, int wave,
                                          int lane) {
  constexpr int NW = WAVES_M * WAVES_N, WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int HR = BM / 2;            // rows per half
  constexpr int CPR = BN / 4;           // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;         // rows per wave instruction
  constexpr int IT = HR / (NW * RPI);   // row groups per wave and half
  constexpr int U = IT >= 4 ? 4 : IT;   // row groups loaded together
  static_assert(CPR <= 64 && 64 % CPR == 0 && CPR >= 16, "row must split over a wave");
  static_assert(IT * NW * RPI == HR && IT % U == 0, "half tile must split over the waves");
  static_assert(HR % WM == 0, "a wave's rows lie in one half");
  const float sc[4] = {p.o_sc[0], 1.0f / p.o_sc[1], 1.0f / p.o_sc[2], p.o_sc[3]};
  const int c = lane % CPR;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    __syncthreads();  // the ring (or the previous half) is no longer read
    if ((wm * WM) / HR == h) {
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          const int ml = wm * WM + j * 16 + (lane & 15) - h * HR;
          const int cw = (wn * WN + i * 16 + (lane >> 4) * 4) / 4;
          *reinterpret_cast<f32x4_t*>(lds + ml * BN + ((cw ^ (ml & 15)) * 4)) = acc[i][j];
        }
    }
    __syncthreads();
#pragma unroll
    for (int it0 = 0; it0 < IT; it0 += U) {
      AdamPiece a[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = (wave + (it0 + u) * NW) * RPI + lane / CPR;
        const f32x4_t g = *reinterpret_cast<const f32x4_t*>(lds + r * BN + ((c ^ (r & 15)) * 4));
        const float v[4] = {g[0], g[1], g[2], g[3]};
        adam_load<EPI>(p, m0 + h * HR + r, n0 + c * 4, v, a[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = (wave + (it0 + u) * NW) * RPI + lane / CPR;
        adam_store<EPI>(p, sc, m0 + h * HR + r, n0 + c * 4, a[u]);
      }
    }
  }
}

// Each stage is one 16x16x32 k-step. Its fragments were read during the
// previous stage (double-buffered registers); BAR_AT MFMAs into the stage the
// wave waits for its own DMA of the next stage and meets the others at the
// barrier, after which the next stage is readable and the slot of this stage
// (every wave has fenced its reads) takes the stage four ahead. The NF
// fragment reads of the next stage and the D DMA instructions of the stage
// four ahead are then spread evenly over the MFMAs up to TAIL before the end,
// reads and DMAs interleaved in proportion, so that neither the LDS nor the
// texture unit sees a burst.
template <int BM, int BN, int WAVES_M, int WAVES_N, int LA, int LB, int EPI, int GROUP = 0,
          int TAIL = 4>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64, 1) void ring_kernel(GemmArgs p) {
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int FM = WM / 16, FN = WN / 16;
  static_assert(FM * 16 == WM && FN * 16 == WN, "wave tile must be a multiple of 16");
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int AE = RingPart<BM, NW>::ELEMS, BE = RingPart<BN, NW>::ELEMS;
  constexpr int DA = RingPart<BM, NW>::PER, DB = RingPart<BN, NW>::PER;
  constexpr int D = DA + DB;  // DMA instructions per wave per stage
  constexpr int NF = FN + FM, NM = FN * FM;
  constexpr int SLOT = AE + BE;
  constexpr int BAR_AT = 2;   // MFMAs of a stage issued before its barrier
  constexpr int E = NF + D;   // memory instructions spread over a stage
  constexpr int W = NM - BAR_AT - TAIL;
  static_assert(W > 0, "wave tile too small for the barrier placement and tail");
  __shared__ uint4 lds[4 * SLOT];

  int tm, tn;
  if (!tile_setup<BM, BN, EPI, GROUP>(p, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;

  f32x4_t acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.0f;
  const int nst = (p.K + SK - 1) / SK;

  // DMA instruction d (0..D-1) of stage st into slot st % 4 (zeros past K)
  auto dma = [&](int st, int d) {
    uint4* slot = lds + (st & 3) * SLOT;
    if (d < DA) ring_dma<BM, NW, LA>(d, p.A, p.lda, m0, p.M, st * SK, p.K, slot, wave, lane);
    else ring_dma<BN, NW, LB>(d - DA, p.B, p.ldb, n0, p.N, st * SK, p.K, slot + AE, wave, lane);
  };
  // fragment f (B fragments first, then A) of stage st
  auto read = [&](bf16x8_t* fa_, bf16x8_t* fb_, int st, int f) {
    const uint4* slot = lds + (st & 3) * SLOT;
    if (f < FN) fa_[f] = ring_frag<LB, BN>(slot + AE, wn * WN + f * 16, lane);
    else fb_[f - FN] = ring_frag<LA, BM>(slot, wm * WM + (f - FN) * 16, lane);
  };

  // prologue: stages 0..3 in flight; publish stage 0; its fragments
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int d = 0; d < D; ++d) dma(st, d);
  wait_dma<3 * D>();
  __builtin_amdgcn_s_barrier();
  bf16x8_t fa[2][FN], fb[2][FM];
#pragma unroll
  for (int f = 0; f < NF; ++f) read(fa[0], fb[0], 0, f);

  // two stages per iteration, so that the fragment buffers are fixed; past
  // the last stage the ring holds zeros (an odd stage count runs one stage
  // of zeros)
  for (int st = 0; st < nst; st += 2) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int s = st + h;
      bf16x8_t* ca = fa[h];
      bf16x8_t* cb = fb[h];
      bf16x8_t* na = fa[h ^ 1];
      bf16x8_t* nb = fb[h ^ 1];
      ring_fence<FN, FM>(fa[h], fb[h]);
      __builtin_amdgcn_sched_barrier(0);
      int fr = 0, dm = 0;
#pragma unroll
      for (int q = 0; q < NM; ++q) {
        const int i = q / FM, j = q % FM;
        if (q == BAR_AT) {
          // this wave's part of stage s + 1 has landed (s + 2 and s + 3 may
          // still be in flight)
          wait_dma<2 * D>();
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
        }
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ca[i], cb[j], acc[i][j], 0, 0, 0);
        if (q >= BAR_AT) {
          // memory instructions due by the end of MFMA q: event e is a read
          // when the read count steps between e and e + 1
          const int due = q - BAR_AT + 1 >= W ? E : ((q - BAR_AT + 1) * E) / W;
#pragma unroll
          for (int t = 0; t < (E + W - 1) / W + 1; ++t) {
            if (fr + dm < due) {
              const int e = fr + dm;
              const bool is_read = ((e + 1) * NF) / E > (e * NF) / E;
              if ((is_read && fr < NF) || dm >= D) read(na, nb, s + 1, fr++);
              else dma(s + 4, dm++);
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // every DMA has landed and every LDS read returned before the registers of
  // the last (unused) fragments are reused and before the workgroup exits
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  ring_fence<FN, FM>(fa[0], fb[0]);
  if constexpr (EPI == kStoreF32Adam || EPI == kAccF32Adam) {
    static_assert(BM / 2 * BN <= 4 * SLOT * 4, "half a tile must fit the stage ring");
    adam_tile<BM, BN, WAVES_M, WAVES_N, EPI, FN, FM>(p, acc, reinterpret_cast<float*>(lds), m0,
                                                      n0, wm, wn, wave, lane);
  } else {
    store_tile16<EPI, FN, FM>(p, acc, m0 + wm * WM, n0 + wn * WN, lane);
  }
}

// Operands contiguous along M / N and full 256 x 256 tiles run on the ring
// pipeline; the remaining K-contiguous tiles (256 x 192 and the small ones)
// on the double-buffered one.
template <int BM, int BN, int WAVES_M, int WAVES_N, int LA, int LB, int EPI, int GROUP>
void launch_kernel(const GemmArgs& a, long grid, hipStream_t s) {
  if constexpr (LA == kMC || LB == kMC || (BM == 256 && BN == 256) || GROUP == 4)
    hipLaunchKernelGGL((ring_kernel<BM, BN, WAVES_M, WAVES_N, LA, LB, EPI, GROUP>),
                       dim3((unsigned)grid), dim3(WAVES_M * WAVES_N * 64), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_kernel<BM, BN, WAVES_M, WAVES_N, LA, LB, EPI, GROUP>),
                       dim3((unsigned)grid), dim3(WAVES_M * WAVES_N * 64), 0, s, a);
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int LA, int LB, int EPI>
hipError_t launch(const GemmArgs& a, hipStream_t s) {
  const long tiles = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  launch_kernel<BM, BN, WAVES_M, WAVES_N, LA, LB, EPI, 0>(a, tiles, s);
  return hipGetLastError();
}

// M-grouped: at most M / BM + groups m-tiles exist, whatever the group sizes.
template <int BM, int BN, int WAVES_M, int WAVES_N, int LB, int EPI>
hipError_t launch_grouped_m(const GemmArgs& a, hipStream_t s) {
  // real tiles <= (M / BM + groups) * tiles_n; rounded up so that every XCD's
  // share of the workgroups covers ceil(real / 8) tiles
  const long mt = a.M / BM + a.groups;
  const long tiles = ((mt * ((a.N + BN - 1) / BN) + NUM_XCD - 1) / NUM_XCD + 1) * NUM_XCD;
  launch_kernel<BM, BN, WAVES_M, WAVES_N, kKC, LB, EPI, 1>(a, tiles, s);
  return hipGetLastError();
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI>
hipError_t launch_grouped_k(const GemmArgs& a, hipStream_t s) {
  const long tiles = (long)a.groups * ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  launch_kernel<BM, BN, WAVES_M, WAVES_N, kMC, kMC, EPI, 2>(a, tiles, s);
  return hipGetLastError();
}

template <bool ACC>
__global__ __launch_bounds__(256) void splitk_reduce_k(const float* __restrict__ part, int S,
                                                      long stride, int M, int N,
                                                      float* __restrict__ out, long ldo) {
  // out[m][n..n+3] (+)= sum over splits, in split order
  const long q = (long)blockIdx.x * 256 + threadIdx.x;
  const int nq = N / 4;
  if (q >= (long)M * nq) return;
  const int m = (int)(q / nq), n = (int)(q % nq) * 4;
  const float* src = part + (long)m * N + n;
  float4 acc = *reinterpret_cast<const float4*>(src);
  for (int e = 1; e < S; ++e) {
    const float4 v = *reinterpret_cast<const float4*>(src + e * stride);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  float4* o = reinterpret_cast<float4*>(out + (long)m * ldo + n);
  if (ACC) {
    const float4 c = *o;
    acc.x += c.x; acc.y += c.y; acc.z += c.z; acc.w += c.w;
  }
  *o = acc;
}

constexpr int kCUs = 256;

template <int LA, int LB, int EPI>
hipError_t dispatch_tiles(const GemmArgs& a, hipStream_t s) {
  // Large tiles once they fill the chip, smaller ones for small problems.
  const long big = (long)((a.M + 255) / 256) * ((a.N + 255) / 256);
  const long mid = (long)((a.M + 255) / 256) * ((a.N + 127) / 128);
  if constexpr (LA == kKC && LB == kKC) {
    const long tail = big % kCUs;
    if (big > kCUs && tail <= kCUs / 2 && tail > 0) {
      // whole rounds of 256 x 256 tiles, then the last half-empty round's
      // tiles as 256 x 128 halves, twice as many workgroups; only products
      // with both operands K-contiguous (the forward ones, which run alone
      // on the chip; a product that shares the chip with a side stream
      // leaves its partial round to that stream's work)
      launch_kernel<256, 256, 2, 4, LA, LB, EPI, 0>(a, big - tail, s);
      GemmArgs b = a;
      b.tile_base = (int)(big - tail);
      launch_kernel<256, 128, 2, 4, LA, LB, EPI, 4>(b, 2 * tail, s);
      return hipGetLastError();
    }
    if (big >= kCUs) {
      // 256 x 192 tiles when 256 x 256 ones leave the last wave of workgroups
      // partly empty: cost ~ waves x tile area, the narrower (double-buffered)
      // tile being ~26 % less efficient per FLOP than the ring's 256 x 256
      // (measured on the 4096 x 6144 x 4096 product: two rounds of each,
      // 200 us on the ring against 208-212 us)
      const long t192 = (long)((a.M + 255) / 256) * ((a.N + 191) / 192);
      const double c256 = (double)((big + kCUs - 1) / kCUs) * 256.0;
      const double c192 = (double)((t192 + kCUs - 1) / kCUs) * 192.0 / 0.74;
      if (c192 < c256) return launch<256, 192, 4, 2, LA, LB, EPI>(a, s);
    }
  }
  // 8 waves of 64 x 128 (two per SIMD)
  if (big >= 256) {
    // 128 x 64 wave tiles (2 x 4 waves): in a data gradient (B M/N-contiguous,
    // read with the slower transposing reads) they put the transposing reads
    // on the narrow side of the wave tile, half as many per stage as with
    // 64 x 128; the other products measured no slower (slightly faster)
    return launch<256, 256, 2, 4, LA, LB, EPI>(a, s);
  }
  if (mid >= 256) return launch<256, 128, 2, 2, LA, LB, EPI>(a, s);
  return launch<128, 128, 2, 2, LA, LB, EPI>(a, s);
}

}  // namespace

hipError_t gemm_grouped_m(GemmLayout lb, GemmEpilogue epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || a.groups <= 0) return hipSuccess;
  if (lb == kKC && epi == kStoreBF16) return launch_grouped_m<256, 256, 4, 2, kKC, kStoreBF16>(a, s);
  if (lb == kMC && epi == kStoreBF16) return launch_grouped_m<256, 256, 2, 4, kMC, kStoreBF16>(a, s);
  return hipErrorInvalidValue;
}

hipError_t gemm_grouped_k(GemmEpilogue epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || a.groups <= 0) return hipSuccess;
  if (epi == kAccF32) return launch_grouped_k<256, 256, 4, 2, kAccF32>(a, s);
  if (epi == kStoreF32) return launch_grouped_k<256, 256, 4, 2, kStoreF32>(a, s);
  if (epi == kAccF32Adam) return launch_grouped_k<256, 256, 4, 2, kAccF32Adam>(a, s);
  if (epi == kStoreF32Adam) return launch_grouped_k<256, 256, 4, 2, kStoreF32Adam>(a, s);
  return hipErrorInvalidValue;
}

int splitk_splits(int M, int N, int K) {
  const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128);
  if (tiles >= 128 || K < 1024) return 1;
  int S = (int)((256 + tiles - 1) / tiles);
  S = S > K / 512 ? K / 512 : S;
  return S < 1 ? 1 : (S > 32 ? 32 : S);
}

hipError_t gemm_wgrad_splitk(const GemmArgs& a, int splits, float* partial, bool accumulate,
                             hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (splits <= 1 || a.K <= 0) return gemm(kMC, kMC, accumulate ? kAccF32 : kStoreF32, a, s);
  const long ks = ((a.K + splits - 1) / splits + BK - 1) / BK * BK;
  const int S = (int)((a.K + ks - 1) / ks);
  GemmArgs p = a;
  p.C = partial;
  p.ldc = a.N;
  p.strideB = ks;
  p.strideC = (long)a.M * a.N;
  p.groups = S;
  const long tiles = (long)S * ((a.M + 127) / 128) * ((a.N + 127) / 128);
  launch_kernel<128, 128, 2, 2, kMC, kMC, kStoreF32, 3>(p, tiles, s);
  const long n4 = (long)a.M * (a.N / 4);
  const dim3 grid((unsigned)((n4 + 255) / 256));
  if (accumulate)
    hipLaunchKernelGGL(splitk_reduce_k<true>, grid, dim3(256), 0, s, partial, S, (long)a.M * a.N,
                       a.M, a.N, reinterpret_cast<float*>(a.C), a.ldc);
  else
    hipLaunchKernelGGL(splitk_reduce_k<false>, grid, dim3(256), 0, s, partial, S, (long)a.M * a.N,
                       a.M, a.N, reinterpret_cast<float*>(a.C), a.ldc);
  return hipGetLastError();
}

hipError_t gemm(GemmLayout la, GemmLayout lb, GemmEpilogue epi, const GemmArgs& a,
                hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (la == kKC && lb == kKC) {
    switch (epi) {
      case kStoreBF16: return dispatch_tiles<kKC, kKC, kStoreBF16>(a, s);
      case kResidBF16: return dispatch_tiles<kKC, kKC, kResidBF16>(a, s);
      case kAccF32: return dispatch_tiles<kKC, kKC, kAccF32>(a, s);
      case kStoreF32: return dispatch_tiles<kKC, kKC, kStoreF32>(a, s);
      default: break;
    }
  } else if (la == kKC && lb == kMC) {
    switch (epi) {
      case kStoreBF16: return dispatch_tiles<kKC, kMC, kStoreBF16>(a, s);
      case kResidBF16: return dispatch_tiles<kKC, kMC, kResidBF16>(a, s);
      default: break;
    }
  } else if (la == kMC && lb == kMC) {
    switch (epi) {
      case kAccF32: return dispatch_tiles<kMC, kMC, kAccF32>(a, s);
      case kStoreF32: return dispatch_tiles<kMC, kMC, kStoreF32>(a, s);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace forge

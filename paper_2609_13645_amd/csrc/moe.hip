// Routed mixture-of-experts pieces of the layer (the sparse model of App. B,
// Table "H100 architecture configurations": routed experts with top-k
// selection), dropless: every token goes to its top_k experts.
//
//  * route: one wave per token, lane l holds the fp32 logits of experts
//    l, l + 64, l + 128, l + 192 (E <= 256): softmax over all experts, then
//    top_k rounds of wave argmax on a total order of the logits (numeric
//    order, -0 equal to +0, NaN below -inf; ties to the lower expert id), so
//    every index lies in [0, E) whatever the logits hold. Gates are the
//    softmax probabilities of the chosen experts (no renormalisation).
//  * permutation: a counting sort that is deterministic by construction —
//    per-block expert histograms, a fixed-order scan over blocks, then each
//    block assigns ranks in flat (token, slot) order with wave ballots, so
//    the order is expert-major, token ascending, slot ascending.
//  * gather / combine / their backward move whole bf16 rows with 16-byte
//    vectors; every sum over the k slots of a token runs in slot order.
//  * the load-balance auxiliary loss alpha * E * sum_e f_e P_e and its
//    gradient through the softmax (f_e = count_e / (T k) is a constant);
//    the column sums behind P_e are per-block partials summed in block order.
#include <climits>

#include "common.h"
#include "kernels.h"

namespace forge {
namespace {

constexpr int kSortTokens = 128;  // tokens per counting-sort block
constexpr int kMaxE = 256;        // experts (four per lane of a wave)
constexpr int kSlots = kMaxE / 64;

// ------------------------------------------------------------- routing ----
// Order key of a logit for the top-k choice: larger key = preferred. The
// integer image of the float is monotone in its value; -0 is first made +0
// (they compare equal) and NaN gets the lowest key of all.
__device__ __forceinline__ uint32_t order_key(float f) {
  if (f == 0.0f) f = 0.0f;
  const int b = __float_as_int(f);
  const int key = b >= 0 ? b : (b ^ 0x7FFFFFFF);
  return (uint32_t)(f != f ? INT_MIN : key) ^ 0x80000000u;
}
// Candidate word: order key, then the expert id reversed (a lower id wins a
// tie of keys), then a 1 so that every real candidate is above 0, which
// marks an expert that is taken or absent.
__device__ __forceinline__ uint64_t cand_word(float l, int e) {
  return ((uint64_t)order_key(l) << 32) | ((uint64_t)(kMaxE - 1 - e) << 1) | 1ull;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
    const uint64_t w = ((uint64_t)hi << 32) | lo;
    v = w > v ? w : v;
  }
  return v;
}

__global__ __launch_bounds__(256) void route_k(const float* __restrict__ logits, int T, int E,
                                               int k, int32_t* __restrict__ idx,
                                               float* __restrict__ gates,
                                               float* __restrict__ probs) {
  const int lane = threadIdx.x & 63;
  const long t = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  float l[kSlots], p[kSlots];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int e = lane + 64 * i;
    l[i] = e < E ? logits[t * E + e] : -INFINITY;
    mx = fmaxf(mx, l[i]);
  }
  mx = wave_max(mx);
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int e = lane + 64 * i;
    p[i] = e < E ? __expf(l[i] - mx) : 0.0f;
    sum += p[i];
  }
  sum = wave_sum(sum);
  uint64_t cand[kSlots];
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int e = lane + 64 * i;
    p[i] /= sum;
    if (e < E) probs[t * E + e] = p[i];
    cand[i] = e < E ? cand_word(l[i], e) : 0ull;
  }
  for (int j = 0; j < k; ++j) {
    uint64_t best = cand[0];
#pragma unroll
    for (int i = 1; i < kSlots; ++i) best = cand[i] > best ? cand[i] : best;
    best = wave_max_u64(best);
    // k <= E, so a real candidate is left in every round
    const int e = kMaxE - 1 - (int)((best >> 1) & (kMaxE - 1));
    const int owner = e & 63, slot = e >> 6;
    float ps = p[0];
#pragma unroll
    for (int i = 1; i < kSlots; ++i) ps = slot == i ? p[i] : ps;
    const float g = __shfl(ps, owner, 64);
    if (lane == 0) {
      idx[t * k + j] = e;
      gates[t * k + j] = g;
    }
#pragma unroll
    for (int i = 0; i < kSlots; ++i)
      if (lane == owner && slot == i) cand[i] = 0ull;
  }
}

// Per-block expert histogram of the flat (token, slot) entries (entries
// outside [0, E) are not counted).
__global__ __launch_bounds__(256) void sort_count_k(const int32_t* __restrict__ idx, int T, int E,
                                                    int k, int32_t* __restrict__ block_counts) {
  __shared__ int hist[kMaxE];
  hist[threadIdx.x] = 0;
  __syncthreads();
  const long f0 = (long)blockIdx.x * kSortTokens * k;
  const long f1 = min((long)T * k, f0 + (long)kSortTokens * k);
  for (long f = f0 + threadIdx.x; f < f1; f += blockDim.x) {
    const int e = idx[f];
    if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  if (threadIdx.x < E) block_counts[(long)blockIdx.x * E + threadIdx.x] = hist[threadIdx.x];
}

// Fixed-order scan: offsets[e] (exclusive over experts), per-block bases.
// One block of kMaxE threads.
__global__ __launch_bounds__(256) void sort_scan_k(int32_t* __restrict__ block_counts, int nblk,
                                                   int E, int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ offsets) {
  __shared__ int tot[kMaxE];
  const int e = threadIdx.x;
  if (e < E) {
    int run = 0;
    for (int b = 0; b < nblk; ++b) {
      const int c = block_counts[(long)b * E + e];
      block_counts[(long)b * E + e] = run;  // becomes the in-expert base of block b
      run += c;
    }
    tot[e] = run;
    counts[e] = run;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < E; ++i) {
      offsets[i] = acc;
      acc += tot[i];
    }
    offsets[E] = acc;
  }
}

// Ranks within each expert in flat order: one wave per block, 64 entries per
// round; for each expert present in the round, a ballot gives the lanes'
// ranks. perm[pos] = flat entry, pos_of[flat entry] = pos.
__global__ __launch_bounds__(64) void sort_scatter_k(const int32_t* __restrict__ idx, int T, int E,
                                                     int k, const int32_t* __restrict__ block_base,
                                                     const int32_t* __restrict__ offsets,
                                                     int32_t* __restrict__ perm,
                                                     int32_t* __restrict__ pos_of) {
  // One wave walks the block's entries 64 at a time in flat order. The lanes
  // holding the same expert are found with one ballot per bit of the expert
  // id (E <= 256: eight bits), so each lane's rank among the earlier lanes of
  // its expert is a popcount, and the group's lowest lane advances the
  // expert's running position. Entries outside [0, E) are skipped.
  __shared__ int run[kMaxE];
  const int lane = threadIdx.x;
  for (int e = lane; e < E; e += 64)
    run[e] = offsets[e] + block_base[(long)blockIdx.x * E + e];
  __syncthreads();
  const long f0 = (long)blockIdx.x * kSortTokens * k;
  const long f1 = min((long)T * k, f0 + (long)kSortTokens * k);
  const uint64_t below = (1ull << lane) - 1ull;
  for (long base = f0; base < f1; base += 64) {
    const long f = base + lane;
    const int raw = f < f1 ? idx[f] : -1;
    const bool ok = (unsigned)raw < (unsigned)E;
    const int e = ok ? raw : 0;
    uint64_t same = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t ones = __ballot(ok && ((e >> b) & 1));
      same &= ((e >> b) & 1) ? ones : ~ones;
    }
    const int pos = run[e] + __popcll(same & below);  // every lane reads before any update
    __builtin_amdgcn_wave_barrier();
    if (ok) {
      perm[pos] = (int32_t)f;
      pos_of[f] = pos;
      if ((same & below) == 0) run[e] += __popcll(same);
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// xs[pos] = b[perm[pos] / k]; one thread per 8 elements.
__global__ __launch_bounds__(256) void gather_k(const bf16_t* __restrict__ b,
                                                const int32_t* __restrict__ perm, long rows, int h,
                                                int k, bf16_t* __restrict__ xs) {
  const int cpr = h / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= rows * cpr) return;
  const long r = id / cpr;
  const int c = (int)(id % cpr);
  const long t = perm[r] / k;
  reinterpret_cast<uint4*>(xs + r * h)[c] = reinterpret_cast<const uint4*>(b + t * h)[c];
}

// out[t] = h1[t] + scale * sum_j gate[t, j] * ys[pos_of[t k + j]] (fp32,
// slot order; scale: the branch scale of muP, 1 otherwise).
__global__ __launch_bounds__(256) void combine_k(const bf16_t* __restrict__ ys,
                                                 const float* __restrict__ gates,
                                                 const int32_t* __restrict__ pos_of,
                                                 const bf16_t* __restrict__ h1, long T, int h,
                                                 int k, float scale, bf16_t* __restrict__ out) {
  const int cpr = h / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  float acc[8] = {};
  for (int j = 0; j < k; ++j) {
    const float g = gates[t * k + j];
    float y[8];
    unpack8(reinterpret_cast<const uint4*>(ys + (long)pos_of[t * k + j] * h)[c], y);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += g * y[e];
  }
  float r[8];
  unpack8(reinterpret_cast<const uint4*>(h1 + t * h)[c], r);
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] += scale * acc[e];
  reinterpret_cast<uint4*>(out + t * h)[c] = pack8(r);
}

// Backward of combine for one token per block: dgate[t, j] = scale dy_t .
// ys_row and dys_row = scale gate[t, j] dy_t. k <= 16.
__global__ __launch_bounds__(256) void combine_bwd_k(const bf16_t* __restrict__ ys,
                                                     const float* __restrict__ gates,
                                                     const int32_t* __restrict__ pos_of,
                                                     const bf16_t* __restrict__ dy, int h, int k,
                                                     float scale, float* __restrict__ dgate,
                                                     bf16_t* __restrict__ dys) {
  __shared__ float red[4][16];
  const long t = blockIdx.x;
  const int cpr = h / 8;
  float dot[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) dot[j] = 0.0f;
  for (int c = threadIdx.x; c < cpr; c += blockDim.x) {
    float d[8];
    unpack8(reinterpret_cast<const uint4*>(dy + t * h)[c], d);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j < k) {
        const long row = pos_of[t * k + j];
        float y[8], o[8];
        unpack8(reinterpret_cast<const uint4*>(ys + row * h)[c], y);
        const float g = scale * gates[t * k + j];
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s += d[e] * y[e];
          o[e] = g * d[e];
        }
        dot[j] += s;
        reinterpret_cast<uint4*>(dys + row * h)[c] = pack8(o);
      }
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if (j < k) {
      const float s = wave_sum(dot[j]);
      if (lane == 0) red[wave][j] = s;
    }
  }
  __syncthreads();
  if (threadIdx.x < k) {
    const int j = threadIdx.x;
    dgate[t * k + j] = scale * ((red[0][j] + red[1][j]) + (red[2][j] + red[3][j]));
  }
}

// db_s[t] = sum_j dxs[pos_of[t k + j]] (fp32 in slot order, one rounding).
__global__ __launch_bounds__(256) void scatter_back_k(const bf16_t* __restrict__ dxs,
                                                      const int32_t* __restrict__ pos_of, long T,
                                                      int h, int k, bf16_t* __restrict__ db) {
  const int cpr = h / 8;
  const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= T * cpr) return;
  const long t = id / cpr;
  const int c = (int)(id % cpr);
  float acc[8] = {};
  for (int j = 0; j < k; ++j) {
    float y[8];
    unpack8(reinterpret_cast<const uint4*>(dxs + (long)pos_of[t * k + j] * h)[c], y);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += y[e];
  }
  reinterpret_cast<uint4*>(db + t * h)[c] = pack8(acc);
}

// Column sums of the router probabilities over kAuxTokens-token blocks,
// partial[block][e] (thread e sums its expert's column in token order);
// aux_loss_k adds the blocks in block order: P_e = sum_t p[t, e], and
// aux += alpha E sum_e f_e P_e / T.
constexpr int kAuxTokens = 64;
__global__ __launch_bounds__(256) void prob_colsum_k(const float* __restrict__ probs, int T, int E,
                                                     float* __restrict__ partial) {
  const int e = threadIdx.x;
  const long t0 = (long)blockIdx.x * kAuxTokens;
  const long t1 = min((long)T, t0 + kAuxTokens);
  if (e >= E) return;
  float sum = 0.0f;
  for (long t = t0; t < t1; ++t) sum += probs[t * E + e];
  partial[(long)blockIdx.x * E + e] = sum;
}

__global__ __launch_bounds__(256) void aux_loss_k(const float* __restrict__ partial, int nblk,
                                                  const int32_t* __restrict__ counts, int T, int E,
                                                  int k, float alpha, float* __restrict__ colsum,
                                                  float* __restrict__ aux) {
  __shared__ float part[4];
  const int e = threadIdx.x;
  float c = 0.0f;
  if (e < E)
    for (int b = 0; b < nblk; ++b) c += partial[(long)b * E + e];
  if (e < E) colsum[e] = c;
  const float fe = e < E ? (float)counts[e] / ((float)T * k) : 0.0f;
  const float term = wave_sum(fe * c);
  if ((e & 63) == 0) part[e >> 6] = term;
  __syncthreads();
  if (e == 0 && aux) aux[0] += alpha * (float)E * ((part[0] + part[1]) + (part[2] + part[3])) /
                               (float)T;
}

// dl[t, e] = p (dp - sum_e p dp) with dp = dgate on chosen experts plus the
// aux term alpha E f_e / T on every expert; written as bf16 for the router
// data / weight gradient products. One wave per token, lane l holding
// experts l + 64 i.
__global__ __launch_bounds__(256) void router_bwd_k(const float* __restrict__ probs,
                                                    const int32_t* __restrict__ idx,
                                                    const float* __restrict__ dgate,
                                                    const int32_t* __restrict__ counts, int T,
                                                    int E, int k, float alpha,
                                                    bf16_t* __restrict__ dl) {
  const int lane = threadIdx.x & 63;
  const long t = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  float p[kSlots], dp[kSlots];
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int e = lane + 64 * i;
    p[i] = e < E ? probs[t * E + e] : 0.0f;
    dp[i] = e < E ? alpha * (float)E * ((float)counts[e] / ((float)T * k)) / (float)T : 0.0f;
    for (int j = 0; j < k; ++j)
      if (idx[t * k + j] == e) dp[i] += dgate[t * k + j];
    part += p[i] * dp[i];
  }
  const float dot = wave_sum(part);
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int e = lane + 64 * i;
    if (e < E) dl[t * E + e] = f2bf(p[i] * (dp[i] - dot));
  }
}

inline unsigned nblocks(long work, int threads) { return (unsigned)((work + threads - 1) / threads); }

}  // namespace

int moe_sort_blocks(int T) { return (T + kSortTokens - 1) / kSortTokens; }

hipError_t moe_route(const float* logits, int T, int E, int k, int32_t* idx, float* gates,
                     float* probs, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(route_k, dim3(nblocks(T, 4)), dim3(256), 0, s, logits, T, E, k, idx, gates, probs);
  return hipGetLastError();
}

hipError_t moe_sort(const int32_t* idx, int T, int E, int k, int32_t* block_counts,
                    int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* pos_of,
                    hipStream_t s) {
  const int nb = moe_sort_blocks(T);
  hipLaunchKernelGGL(sort_count_k, dim3(nb), dim3(256), 0, s, idx, T, E, k, block_counts);
  hipLaunchKernelGGL(sort_scan_k, dim3(1), dim3(kMaxE), 0, s, block_counts, nb, E, counts, offsets);
  hipLaunchKernelGGL(sort_scatter_k, dim3(nb), dim3(64), 0, s, idx, T, E, k, block_counts, offsets,
                     perm, pos_of);
  return hipGetLastError();
}

hipError_t moe_gather(const uint16_t* b, const int32_t* perm, long rows, int h, int k,
                      uint16_t* xs, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_k, dim3(nblocks(rows * (h / 8), 256)), dim3(256), 0, s, b, perm, rows, h, k, xs);
  return hipGetLastError();
}

hipError_t moe_combine(const uint16_t* ys, const float* gates, const int32_t* pos_of,
                       const uint16_t* h1, long T, int h, int k, float scale, uint16_t* out,
                       hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_k, dim3(nblocks(T * (h / 8), 256)), dim3(256), 0, s, ys, gates, pos_of, h1, T, h, k, scale, out);
  return hipGetLastError();
}

hipError_t moe_combine_bwd(const uint16_t* ys, const float* gates, const int32_t* pos_of,
                           const uint16_t* dy, long T, int h, int k, float scale, float* dgate,
                           uint16_t* dys, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_bwd_k, dim3((unsigned)T), dim3(256), 0, s, ys, gates, pos_of, dy, h, k, scale, dgate, dys);
  return hipGetLastError();
}

hipError_t moe_scatter_back(const uint16_t* dxs, const int32_t* pos_of, long T, int h, int k,
                            uint16_t* db, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(scatter_back_k, dim3(nblocks(T * (h / 8), 256)), dim3(256), 0, s, dxs, pos_of, T, h, k, db);
  return hipGetLastError();
}

int moe_aux_blocks(int T) { return (T + kAuxTokens - 1) / kAuxTokens; }
hipError_t moe_aux_loss(const float* probs, const int32_t* counts, int T, int E, int k, float alpha,
                        float* colsum, float* aux, hipStream_t s) {
  // colsum holds E sums followed by moe_aux_blocks(T) * E block partials
  if (T <= 0) return hipSuccess;
  const int nb = moe_aux_blocks(T);
  float* partial = colsum + E;
  hipLaunchKernelGGL(prob_colsum_k, dim3(nb), dim3(256), 0, s, probs, T, E, partial);
  hipLaunchKernelGGL(aux_loss_k, dim3(1), dim3(256), 0, s, partial, nb, counts, T, E, k, alpha, colsum, aux);
  return hipGetLastError();
}

hipError_t moe_router_bwd(const float* probs, const int32_t* idx, const float* dgate,
                          const int32_t* counts, int T, int E, int k, float alpha, uint16_t* dl,
                          hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(router_bwd_k, dim3(nblocks(T, 4)), dim3(256), 0, s, probs, idx, dgate, counts, T, E, k, alpha, dl);
  return hipGetLastError();
}

}  // namespace forge

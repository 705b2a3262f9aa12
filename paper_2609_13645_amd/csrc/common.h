// Device-side helpers shared by the gfx950 kernels of libforge.
//
// bf16 values travel as uint16_t bit patterns; arithmetic is fp32. The
// float -> bf16 conversion uses the compiler's __bf16 type, which gfx950
// lowers to its native round-to-nearest-even conversion (v_cvt_pk_bf16_f32).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace forge {

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}

__device__ __forceinline__ bf16_t f2bf(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}

// Two floats -> one dword holding two bf16 (lo = a, hi = b), RNE.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2_t f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ float lo_f(uint32_t w) {
  return __builtin_bit_cast(float, w << 16);
}
__device__ __forceinline__ float hi_f(uint32_t w) {
  return __builtin_bit_cast(float, w & 0xFFFF0000u);
}

// 8 bf16 in a uint4 -> 8 floats.
__device__ __forceinline__ void unpack8(const uint4& u, float* f) {
  f[0] = lo_f(u.x); f[1] = hi_f(u.x);
  f[2] = lo_f(u.y); f[3] = hi_f(u.y);
  f[4] = lo_f(u.z); f[5] = hi_f(u.z);
  f[6] = lo_f(u.w); f[7] = hi_f(u.w);
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]),
                    pack2(f[4], f[5]), pack2(f[6], f[7]));
}

// Wave-wide (64 lanes) butterfly reductions.
// One AdamW element (App. F, fused clip + Adam + cast), shared by the
// standalone update and the GEMM's fused weight-gradient epilogue so that
// both give the same bits:
//   g *= clip; m = b1 m + (1-b1) g; v = b2 v + (1-b2) g^2;
//   p -= lr ((m/bc1) / (sqrt(v/bc2) + eps) + wd p); param = bf16(p).
__device__ __forceinline__ void adam1(float& p, float& m, float& v, float g, float b1,
                                      float b2, float eps, float wd, float lr, float ibc1,
                                      float ibc2, float clip) {
  // explicit fused multiply-adds and no other contraction: the kernels that
  // inline this get the same roundings whatever their surroundings
#pragma clang fp contract(off)
  g *= clip;
  m = __builtin_fmaf(b1, m, (1.0f - b1) * g);
  v = __builtin_fmaf(b2, v, ((1.0f - b2) * g) * g);
  const float upd = __builtin_fmaf(wd, p, (m * ibc1) / (sqrtf(v * ibc2) + eps));
  p = __builtin_fmaf(-lr, upd, p);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Transpose an 8x8 block of bf16 held as 8 uint4 rows: in[r] holds elements
// (r, 0..7); out[c] receives elements (0..7, c). Pure register permutes.
__device__ __forceinline__ void transpose8x8(const uint4* in, uint4* out) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(in);  // w[r*4 + j]
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int j = c >> 1;
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t a = w[(2 * p) * 4 + j];
      const uint32_t b = w[(2 * p + 1) * 4 + j];
      o[p] = (c & 1) ? ((a >> 16) | (b & 0xFFFF0000u))
                     : ((a & 0xFFFFu) | (b << 16));
    }
    out[c] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace forge

// Device-side helpers shared by the gfx950 kernels of the conv / BN / SiLU path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace numbat {

typedef uint16_t bf16_t;  // bf16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // 16 bytes as a native vector (loads stay loads)

constexpr int kWave = 64;

// bf16 bits -> fp32 (exact)
__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

// two fp32 -> packed bf16 bits (lo in bits 0..15), round to nearest even, NaN kept
// (quiet): one v_cvt_pk_bf16_f32 on gfx950
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// fp32 -> bf16 bits, round to nearest even, NaN kept (quiet)
__device__ __forceinline__ uint32_t f2bf(float f) { return pack2(f, 0.f) & 0xffffu; }

// unpack a 16-byte vector of 8 bf16 into fp32
__device__ __forceinline__ void unpack8(const uint4& v, float f[8]) {
  f[0] = bf2f(v.x & 0xffffu); f[1] = bf2f(v.x >> 16);
  f[2] = bf2f(v.y & 0xffffu); f[3] = bf2f(v.y >> 16);
  f[4] = bf2f(v.z & 0xffffu); f[5] = bf2f(v.z >> 16);
  f[6] = bf2f(v.w & 0xffffu); f[7] = bf2f(v.w >> 16);
}

__device__ __forceinline__ uint4 pack8(const float f[8]) {
  uint4 v;
  v.x = pack2(f[0], f[1]);
  v.y = pack2(f[2], f[3]);
  v.z = pack2(f[4], f[5]);
  v.w = pack2(f[6], f[7]);
  return v;
}

// Unsigned division by a run-time constant d >= 1 (Granlund-Montgomery), exact for n < 2^31.
struct FastDiv {
  uint32_t d, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  f.shift = s;
  f.mul = (uint32_t)((((1ull << 32) * ((1ull << s) - d)) / d) + 1);
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  uint32_t t = __umulhi(n, f.mul);
  return (t + n) >> f.shift;
}

// 16x16x32 bf16 MFMA, fp32 accumulate: D = A(16x32) * B(32x16) + C.
// Lane l supplies A row (l % 16) and B column (l % 16), each with the 8 reduction
// elements of group (l / 16); it receives D rows 4*(l/16) .. +3 of column (l % 16).
__device__ __forceinline__ f32x4 mfma16x16x32(const uint4& a, const uint4& b, f32x4 c) {
  bf16x8 av, bv;
  __builtin_memcpy(&av, &a, 16);
  __builtin_memcpy(&bv, &b, 16);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

// the same MFMA on native 16-byte vectors
__device__ __forceinline__ f32x4 mfma16x16x32(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

// 32x32x16 bf16 MFMA, fp32 accumulate (full rate on gfx950; the 16x16x32 form issues at
// about half the FLOP rate).  Lane l supplies A row (l % 32) and B column (l % 32), each
// with the 8 reduction elements of group (l / 32); accumulator register r of lane l holds
// D row 8*(r/4) + 4*(l/32) + (r%4), column (l % 32).
__device__ __forceinline__ f32x16 mfma32x32x16(const u32x4& a, const u32x4& b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

// sigmoid with the hardware exp2 and reciprocal (about 1 ulp each)
__device__ __forceinline__ float sigmoidf_fast(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// BN with batch statistics + SiLU of one element as a multiply-add with per-channel folded
// constants: scale = gamma / sqrt(var + eps), shift = beta - mean * scale, z = y scale +
// shift, a = z sigmoid(z).  The BN forward kernel and the conv prologue both use these, so
// they form bit-identical activations.
__device__ __forceinline__ void bn_fold(float gamma, float beta, float mean, float var, float eps, float& sc,
                                        float& sh) {
  sc = gamma * (1.0f / sqrtf(var + eps));
  sh = beta - mean * sc;
}
__device__ __forceinline__ float bn_silu_apply(float y, float sc, float sh) {
  const float z = __builtin_fmaf(y, sc, sh);
  return z * sigmoidf_fast(z);
}

// The backward of the above with batch statistics, for one element, as multiply-adds with
// per-channel folded constants.  With a = gamma rstd, xhat = (y - mean) rstd:
//   z  = y a + b,  b = beta - mean a                  (the forward's z)
//   dz = g sigmoid(z) (1 + z (1 - sigmoid(z)))
//   dy = a (dz - dbeta / m - xhat dgamma / m) = a dz + (y c + d),
//        c = -a rstd dgamma / m,  d = -a dbeta / m - mean c
// The BN backward kernels (the finalize folds the constants once per channel, the apply
// uses them) and the data gradient's prologue both use these, so they form bit-identical dy.
__device__ __forceinline__ void bn_bwd_fold(float gamma, float beta, float mean, float rstd, float dgamma,
                                            float dbeta, int64_t m, float& a, float& b, float& c, float& d) {
  a = gamma * rstd;
  b = beta - mean * a;
  const float gm = (float)((double)dgamma / (double)m), bm = (float)((double)dbeta / (double)m);
  c = -(a * rstd) * gm;
  d = -(a * bm) - mean * c;
}
__device__ __forceinline__ float bn_silu_bwd_apply(float g, float y, float a, float b, float c, float d) {
  const float z = __builtin_fmaf(y, a, b);
  const float sg = sigmoidf_fast(z);
  const float dz = g * sg * (1.0f + z * (1.0f - sg));
  return __builtin_fmaf(a, dz, __builtin_fmaf(y, c, d));
}

// Workgroups are dealt round-robin to the 8 XCDs (linear id L runs on XCD L % 8), and
// each XCD has its own L2.  Tiles that read the same data should share an XCD, so a
// kernel whose consecutive logical tiles share data maps its linear id to the logical
// tile xcd_remap(L, total): XCD x works through the x-th contiguous chunk of logical
// tiles in order.  A bijection on [0, total).
constexpr uint32_t kXcds = 8;
__device__ __forceinline__ uint32_t xcd_remap(uint32_t L, uint32_t total) {
  const uint32_t q = total / kXcds, r = total % kXcds;
  const uint32_t x = L % kXcds, i = L / kXcds;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

}  // namespace numbat

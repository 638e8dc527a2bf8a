// The optimiser step after the weight gradients on gfx950: global-norm gradient clipping
// and SGD with Nesterov momentum over a list of fp32 parameter tensors in parameter
// groups, in two launches over every tensor:
//  1. sumsq: each of kOptBlocks blocks sums g^2 (fp64) over its share of every tensor
//     and writes one partial;
//  2. update: every block adds the kOptBlocks partials in a fixed order (so every block
//     derives the same norm and clip coefficient, and the result is bitwise
//     reproducible), then updates its share of every tensor: d = c g + wd w,
//     buf = mu buf + d, w -= lr (d + mu buf).
// Block b owns elements 4 (b + i kOptBlocks) .. +3 of every tensor (16-byte vectors
// where the tensor's pointers allow, a scalar tail).  The tensor table lives in device
// memory (caller-owned) and is staged in LDS at kernel entry.  HBM-bound: the update
// moves 20 bytes per element (w, g, buf read; w, buf written).
#include "kernels.h"

namespace numbat {

namespace {

constexpr int kOptThreads = 256;

__device__ __forceinline__ void stage_table(const OptTensor* tab, int count, OptTensor* s_tab) {
  const int words = count * (int)(sizeof(OptTensor) / 4);
  const uint32_t* src = reinterpret_cast<const uint32_t*>(tab);
  uint32_t* dst = reinterpret_cast<uint32_t*>(s_tab);
  for (int i = threadIdx.x; i < words; i += kOptThreads) dst[i] = src[i];
  __syncthreads();
}

// the elements of tensor t block b owns: vectors v = b + i * nblk of 4 elements
template <typename F>
__device__ __forceinline__ void for_my_elements(const OptTensor& T, bool vec_ok, F&& f) {
  const int64_t n = T.n;
  const int64_t nv = vec_ok ? n / 4 : 0;
  const int64_t step = (int64_t)gridDim.x * kOptThreads;
  for (int64_t v = (int64_t)blockIdx.x * kOptThreads + threadIdx.x; v < nv; v += step) f(v * 4, 4);
  // scalar tail (or the whole tensor when its pointers are not 16-byte aligned)
  for (int64_t i = nv * 4 + (int64_t)blockIdx.x * kOptThreads + threadIdx.x; i < n; i += step) f(i, 1);
}

__device__ __forceinline__ bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

__global__ __launch_bounds__(kOptThreads) void opt_sumsq_kernel(const OptTensor* tab, int count, double* part) {
  extern __shared__ OptTensor s_tab[];
  __shared__ double s_w[kOptThreads / 64];
  stage_table(tab, count, s_tab);
  double acc = 0.0;
  for (int t = 0; t < count; ++t) {
    const OptTensor T = s_tab[t];
    const bool vec = aligned16(T.g);
    for_my_elements(T, vec, [&](int64_t i, int k) {
      if (k == 4) {
        const float4 g = *reinterpret_cast<const float4*>(T.g + i);
        acc += (double)g.x * g.x + (double)g.y * g.y + (double)g.z * g.z + (double)g.w * g.w;
      } else {
        const float g = T.g[i];
        acc += (double)g * g;
      }
    });
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
}

__global__ __launch_bounds__(kOptThreads) void opt_update_kernel(const OptTensor* tab, int count, OptGroups grp,
                                                                  float momentum, float max_norm, const double* part,
                                                                  float* total_norm) {
  extern __shared__ OptTensor s_tab[];
  __shared__ float s_coef;
  // the norm from the partials, in a fixed order: lane l sums partials l, l + 64, ...,
  // then a fixed butterfly over the wave
  if (threadIdx.x < 64) {
    double s = 0.0;
    for (int i = threadIdx.x; i < (int)gridDim.x; i += 64) s += part[i];
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d);
    if (threadIdx.x == 0) {
      const double total = sqrt(s);
      const double c = (double)max_norm / (total + 1e-6);
      s_coef = (float)(c < 1.0 ? c : 1.0);
      if (blockIdx.x == 0 && total_norm != nullptr) *total_norm = (float)total;
    }
  }
  stage_table(tab, count, s_tab);  // (its barrier also publishes s_coef)
  const float coef = s_coef, mu = momentum;
  for (int t = 0; t < count; ++t) {
    const OptTensor T = s_tab[t];
    if (T.group < 0 || T.group >= grp.count) continue;  // outside the given groups: left unchanged
    const float lr = grp.lr[T.group], wd = grp.wd[T.group];
    const bool vec = aligned16(T.w) && aligned16(T.g) && aligned16(T.mom);
    for_my_elements(T, vec, [&](int64_t i, int k) {
      if (k == 4) {
        float4 w = *reinterpret_cast<const float4*>(T.w + i);
        const float4 g = *reinterpret_cast<const float4*>(T.g + i);
        float4 b = *reinterpret_cast<const float4*>(T.mom + i);
        float* wv = &w.x;
        const float* gv = &g.x;
        float* bv = &b.x;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d = __builtin_fmaf(wd, wv[e], coef * gv[e]);
          bv[e] = __builtin_fmaf(mu, bv[e], d);
          wv[e] = __builtin_fmaf(-lr, __builtin_fmaf(mu, bv[e], d), wv[e]);
        }
        *reinterpret_cast<float4*>(T.w + i) = w;
        *reinterpret_cast<float4*>(T.mom + i) = b;
      } else {
        const float d = __builtin_fmaf(wd, T.w[i], coef * T.g[i]);
        const float b = __builtin_fmaf(mu, T.mom[i], d);
        T.mom[i] = b;
        T.w[i] = __builtin_fmaf(-lr, __builtin_fmaf(mu, b, d), T.w[i]);
      }
    });
  }
}

}  // namespace

hipError_t opt_clip_sgd_launch(const OptTensor* tab, int count, const OptGroups& grp, float momentum, float max_norm,
                               float* total_norm, double* part, hipStream_t s) {
  const size_t smem = (size_t)count * sizeof(OptTensor);
  trace_begin(KC_OPT_SUMSQ);
  NUMBAT_LAUNCH(opt_sumsq_kernel, dim3(kOptBlocks), dim3(kOptThreads), smem, s, tab, count, part);
  trace_end(KC_OPT_SUMSQ);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_begin(KC_OPT_UPDATE);
  NUMBAT_LAUNCH(opt_update_kernel, dim3(kOptBlocks), dim3(kOptThreads), smem, s, tab, count, grp, momentum,
                     max_norm, (const double*)part, total_norm);
  trace_end(KC_OPT_UPDATE);
  return hipGetLastError();
}

}  // namespace numbat

// The optimiser step after the weight gradients on gfx950: global-norm gradient clipping
// and SGD with Nesterov momentum over a list of fp32 parameter tensors in parameter
// groups, in two launches over every tensor:
//  1. sumsq: each of kOptBlocks blocks sums g^2 (fp64) over its share of the elements and
//     writes one partial;
//  2. update: every block adds the kOptBlocks partials in a fixed order (so every block
//     derives the same norm and clip coefficient, and the result is bitwise
//     reproducible), then updates its share: d = c g + wd w, buf = mu buf + d,
//     w -= lr (d + mu buf).
// Work is split evenly whatever the tensor sizes: every tensor is cut into chunks of
// kChunk elements (the last one partial), the chunks of all tensors are numbered in table
// order, and block b takes a contiguous range of them.  Each block stages the tensor table
// (caller-owned device memory) in LDS with the prefix of the tensors' chunk counts, so a
// chunk's tensor is a binary search away.  Within a chunk the threads take 16-byte vectors
// where the tensor's pointers allow (a scalar path otherwise and for the tail).  HBM-bound:
// the update moves 20 bytes per element (w, g, buf read; w, buf written), the sum 4.
#include "kernels.h"

namespace numbat {

namespace {

constexpr int kOptThreads = 256;
constexpr int kChunk = 4096;  // elements per chunk: four rounds of one float4 per thread

// the table in LDS, and s_first[t] = chunks of the tensors before t (s_first[count] = all)
__device__ __forceinline__ void stage_table(const OptTensor* tab, int count, OptTensor* s_tab, int64_t* s_first) {
  __shared__ int64_t s_sum[kOptThreads];
  const int t = threadIdx.x;
  const int words = count * (int)(sizeof(OptTensor) / 4);
  const uint32_t* src = reinterpret_cast<const uint32_t*>(tab);
  uint32_t* dst = reinterpret_cast<uint32_t*>(s_tab);
  for (int i = t; i < words; i += kOptThreads) dst[i] = src[i];
  __syncthreads();
  // thread t counts the chunks of tensors 4t .. 4t + 3 (count <= 4 * kOptThreads)
  int64_t c[4], local = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = 4 * t + j;
    const int64_t n = i < count ? s_tab[i].n : 0;
    c[j] = n > 0 ? (n + kChunk - 1) / kChunk : 0;
    local += c[j];
  }
  s_sum[t] = local;
  __syncthreads();
  // inclusive scan of the threads' counts
  for (int d = 1; d < kOptThreads; d <<= 1) {
    const int64_t v = t >= d ? s_sum[t - d] : 0;
    __syncthreads();
    s_sum[t] += v;
    __syncthreads();
  }
  int64_t run = s_sum[t] - local;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = 4 * t + j;
    if (i < count) s_first[i] = run;
    run += c[j];
  }
  if (t == 0) s_first[count] = s_sum[kOptThreads - 1];
  __syncthreads();
}

__device__ __forceinline__ bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// calls f(T, element index, vector width 4 or 1) for every element of this block's chunks
// that this thread owns, in a fixed order; 16-byte vectors where the gradient (GRAD_ONLY)
// or all three of the tensor's pointers are 16-byte aligned
template <bool GRAD_ONLY, typename F>
__device__ __forceinline__ void for_my_elements(const OptTensor* s_tab, const int64_t* s_first, int count, F&& f) {
  const int64_t total = s_first[count];
  const int64_t per = (total + gridDim.x - 1) / gridDim.x;
  int64_t k = (int64_t)blockIdx.x * per;
  const int64_t kend = k + per < total ? k + per : total;
  if (k >= kend) return;
  // the last tensor whose first chunk is at or before k
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_first[mid] <= k) lo = mid;
    else hi = mid - 1;
  }
  int t = lo;
  const int tid = threadIdx.x;
  for (; k < kend; ++k) {
    while (s_first[t + 1] <= k) ++t;  // (tensors without elements have no chunks)
    const OptTensor& T = s_tab[t];
    const int64_t off = (k - s_first[t]) * kChunk;
    const int64_t len = T.n - off < kChunk ? T.n - off : kChunk;
    const bool vec = GRAD_ONLY ? aligned16(T.g) : (aligned16(T.w) && aligned16(T.g) && aligned16(T.mom));
    if (vec) {
      const int64_t nv = len & ~(int64_t)3;
#pragma unroll
      for (int r = 0; r < kChunk / (4 * kOptThreads); ++r) {
        const int64_t i = 4 * (tid + (int64_t)r * kOptThreads);
        if (i < nv) f(T, off + i, 4);
      }
      if (tid < (int)(len - nv)) f(T, off + nv + tid, 1);
    } else {
      for (int64_t i = tid; i < len; i += kOptThreads) f(T, off + i, 1);
    }
  }
}

__global__ __launch_bounds__(kOptThreads) void opt_sumsq_kernel(const OptTensor* tab, int count, double* part) {
  extern __shared__ unsigned char s_dyn[];
  OptTensor* s_tab = reinterpret_cast<OptTensor*>(s_dyn);
  int64_t* s_first = reinterpret_cast<int64_t*>(s_dyn + (size_t)count * sizeof(OptTensor));
  __shared__ double s_w[kOptThreads / 64];
  stage_table(tab, count, s_tab, s_first);
  double acc = 0.0;
  for_my_elements<true>(s_tab, s_first, count, [&](const OptTensor& T, int64_t i, int k) {
    if (k == 4) {
      const float4 g = *reinterpret_cast<const float4*>(T.g + i);
      acc += (double)g.x * g.x + (double)g.y * g.y + (double)g.z * g.z + (double)g.w * g.w;
    } else {
      const float g = T.g[i];
      acc += (double)g * g;
    }
  });
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
}

__global__ __launch_bounds__(kOptThreads) void opt_update_kernel(const OptTensor* tab, int count, OptGroups grp,
                                                                  float momentum, float max_norm, const double* part,
                                                                  float* total_norm) {
  extern __shared__ unsigned char s_dyn[];
  OptTensor* s_tab = reinterpret_cast<OptTensor*>(s_dyn);
  int64_t* s_first = reinterpret_cast<int64_t*>(s_dyn + (size_t)count * sizeof(OptTensor));
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
  stage_table(tab, count, s_tab, s_first);  // (its barriers also publish s_coef)
  const float coef = s_coef, mu = momentum;
  for_my_elements<false>(s_tab, s_first, count, [&](const OptTensor& T, int64_t i, int k) {
    if (T.group < 0 || T.group >= grp.count) return;  // outside the given groups: left unchanged
    const float lr = grp.lr[T.group], wd = grp.wd[T.group];
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

}  // namespace

hipError_t opt_clip_sgd_launch(const OptTensor* tab, int count, const OptGroups& grp, float momentum, float max_norm,
                               float* total_norm, double* part, hipStream_t s) {
  const size_t smem = (size_t)count * sizeof(OptTensor) + (size_t)(count + 1) * sizeof(int64_t);
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

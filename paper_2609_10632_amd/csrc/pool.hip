// The glue between conv blocks on gfx950: the SPPF block's 5x5 stride-1 max pool (padding
// 2, never winning) and the neck's nearest 2x upsampling, forward and backward, NHWC bf16
// with pixel strides (so inputs and outputs can be channel slices of concatenation
// buffers).  One thread handles 8 channels (16 bytes) of one pixel.  These tensors are
// small (the SPPF's are 20 x 20 x 288 per image): the window re-reads hit the caches.
//
// Max pool forward: the window's first maximum in row-major order wins (a later equal
// value does not replace it); its window position (0 .. 24) is stored per element as one
// byte, and the backward sends each dy to that position.  The backward is a gather: an
// input pixel visits the 25 windows that contain it in a fixed order and adds the dy of
// those whose stored position is its own, in fp32, rounded once (deterministic).
#include "kernels.h"

namespace numbat {

namespace {

constexpr int kPoolThreads = 256;

__global__ __launch_bounds__(kPoolThreads) void maxpool5_fwd_kernel(PoolArgs a, const bf16_t* x, bf16_t* y,
                                                                    uint8_t* idx) {
  const int cv = a.c / 8;
  const int64_t nvec = (int64_t)a.n * a.h * a.w * cv;
  for (int64_t v = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * kPoolThreads) {
    const int64_t pix = v / cv;
    const int ch = (int)(v - pix * cv) * 8;
    const int64_t img = pix / ((int64_t)a.h * a.w);
    const int rem = (int)(pix - img * a.h * a.w);
    const int p = rem / a.w, q = rem - p * a.w;
    float best[8];
    uint32_t at[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      best[e] = -__builtin_huge_valf();
      at[e] = 0;
    }
    for (int r = 0; r < 5; ++r) {
      const int i = p + r - 2;
      if ((unsigned)i >= (unsigned)a.h) continue;
      for (int s = 0; s < 5; ++s) {
        const int j = q + s - 2;
        if ((unsigned)j >= (unsigned)a.w) continue;
        float f[8];
        unpack8(*reinterpret_cast<const uint4*>(x + ((img * a.h + i) * a.w + j) * a.x_pix + ch), f);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool better = f[e] > best[e];
          best[e] = better ? f[e] : best[e];
          at[e] = better ? (uint32_t)(r * 5 + s) : at[e];
        }
      }
    }
    *reinterpret_cast<uint4*>(y + pix * a.y_pix + ch) = pack8(best);  // bf16 values: exact
    if (idx != nullptr) {
      uint2 b;
      b.x = at[0] | (at[1] << 8) | (at[2] << 16) | (at[3] << 24);
      b.y = at[4] | (at[5] << 8) | (at[6] << 16) | (at[7] << 24);
      *reinterpret_cast<uint2*>(idx + pix * a.c + ch) = b;
    }
  }
}

__global__ __launch_bounds__(kPoolThreads) void maxpool5_bwd_kernel(PoolArgs a, const bf16_t* dy, const uint8_t* idx,
                                                                    bf16_t* dx, int accumulate) {
  const int cv = a.c / 8;
  const int64_t nvec = (int64_t)a.n * a.h * a.w * cv;
  for (int64_t v = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * kPoolThreads) {
    const int64_t pix = v / cv;
    const int ch = (int)(v - pix * cv) * 8;
    const int64_t img = pix / ((int64_t)a.h * a.w);
    const int rem = (int)(pix - img * a.h * a.w);
    const int i = rem / a.w, j = rem - i * a.w;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    // window of output (p, q) holds this pixel at position (r, s) = (i - p + 2, j - q + 2)
    for (int r = 0; r < 5; ++r) {
      const int p = i - r + 2;
      if ((unsigned)p >= (unsigned)a.h) continue;
      for (int s = 0; s < 5; ++s) {
        const int q = j - s + 2;
        if ((unsigned)q >= (unsigned)a.w) continue;
        const int64_t op = (img * a.h + p) * a.w + q;
        const uint2 b = *reinterpret_cast<const uint2*>(idx + op * a.c + ch);
        float g[8];
        unpack8(*reinterpret_cast<const uint4*>(dy + op * a.y_pix + ch), g);
        const uint32_t pos = (uint32_t)(r * 5 + s);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = ((e < 4 ? b.x : b.y) >> (8 * (e & 3))) & 0xffu;
          acc[e] += w == pos ? g[e] : 0.f;
        }
      }
    }
    uint4* o = reinterpret_cast<uint4*>(dx + pix * a.x_pix + ch);
    if (accumulate) {
      float f[8];
      unpack8(*o, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += f[e];
    }
    *o = pack8(acc);
  }
}

// nearest 2x: input pixel (i, j) -> output pixels (2i + a, 2j + b)
__global__ __launch_bounds__(kPoolThreads) void upsample2x_fwd_kernel(PoolArgs a, const bf16_t* x, bf16_t* y) {
  const int cv = a.c / 8;
  const int64_t nvec = (int64_t)a.n * a.h * a.w * cv;
  for (int64_t v = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * kPoolThreads) {
    const int64_t pix = v / cv;
    const int ch = (int)(v - pix * cv) * 8;
    const int64_t img = pix / ((int64_t)a.h * a.w);
    const int rem = (int)(pix - img * a.h * a.w);
    const int i = rem / a.w, j = rem - i * a.w;
    const uint4 val = *reinterpret_cast<const uint4*>(x + pix * a.x_pix + ch);
    const int64_t o0 = (img * 2 * a.h + 2 * i) * (2 * (int64_t)a.w) + 2 * j;
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int s = 0; s < 2; ++s)
        *reinterpret_cast<uint4*>(y + (o0 + r * 2 * (int64_t)a.w + s) * a.y_pix + ch) = val;
  }
}

__global__ __launch_bounds__(kPoolThreads) void upsample2x_bwd_kernel(PoolArgs a, const bf16_t* dy, bf16_t* dx,
                                                                      int accumulate) {
  const int cv = a.c / 8;
  const int64_t nvec = (int64_t)a.n * a.h * a.w * cv;
  for (int64_t v = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; v < nvec; v += (int64_t)gridDim.x * kPoolThreads) {
    const int64_t pix = v / cv;
    const int ch = (int)(v - pix * cv) * 8;
    const int64_t img = pix / ((int64_t)a.h * a.w);
    const int rem = (int)(pix - img * a.h * a.w);
    const int i = rem / a.w, j = rem - i * a.w;
    const int64_t o0 = (img * 2 * a.h + 2 * i) * (2 * (int64_t)a.w) + 2 * j;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        float g[8];
        unpack8(*reinterpret_cast<const uint4*>(dy + (o0 + r * 2 * (int64_t)a.w + s) * a.y_pix + ch), g);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += g[e];
      }
    uint4* o = reinterpret_cast<uint4*>(dx + pix * a.x_pix + ch);
    if (accumulate) {
      float f[8];
      unpack8(*o, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += f[e];
    }
    *o = pack8(acc);
  }
}

int pool_blocks(const PoolArgs& a) {
  const int64_t nvec = (int64_t)a.n * a.h * a.w * (a.c / 8);
  int64_t b = (nvec + kPoolThreads - 1) / kPoolThreads;
  if (b > 8192) b = 8192;
  return (int)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t maxpool5_fwd_launch(const PoolArgs& a, const bf16_t* x, bf16_t* y, uint8_t* idx, hipStream_t s) {
  trace_begin(KC_POOL);
  NUMBAT_LAUNCH(maxpool5_fwd_kernel, dim3(pool_blocks(a)), dim3(kPoolThreads), 0, s, a, x, y, idx);
  trace_end(KC_POOL);
  return hipGetLastError();
}

hipError_t maxpool5_bwd_launch(const PoolArgs& a, const bf16_t* dy, const uint8_t* idx, bf16_t* dx, int accumulate,
                               hipStream_t s) {
  trace_begin(KC_POOL);
  NUMBAT_LAUNCH(maxpool5_bwd_kernel, dim3(pool_blocks(a)), dim3(kPoolThreads), 0, s, a, dy, idx, dx, accumulate);
  trace_end(KC_POOL);
  return hipGetLastError();
}

hipError_t upsample2x_fwd_launch(const PoolArgs& a, const bf16_t* x, bf16_t* y, hipStream_t s) {
  trace_begin(KC_POOL);
  NUMBAT_LAUNCH(upsample2x_fwd_kernel, dim3(pool_blocks(a)), dim3(kPoolThreads), 0, s, a, x, y);
  trace_end(KC_POOL);
  return hipGetLastError();
}

hipError_t upsample2x_bwd_launch(const PoolArgs& a, const bf16_t* dy, bf16_t* dx, int accumulate, hipStream_t s) {
  trace_begin(KC_POOL);
  NUMBAT_LAUNCH(upsample2x_bwd_kernel, dim3(pool_blocks(a)), dim3(kPoolThreads), 0, s, a, dy, dx, accumulate);
  trace_end(KC_POOL);
  return hipGetLastError();
}

}  // namespace numbat

// BatchNorm (training mode, batch statistics) + SiLU on gfx950: forward apply,
// standalone statistics, backward reduce / finalize / apply.
//
// These passes are HBM-bound: every thread moves 16-byte vectors (8 channels of one
// pixel) and per-channel constants sit in LDS.  Reductions are per-block partials in
// a fixed row assignment, summed in a fixed order (fp64 for the cross-block step),
// so results are bitwise reproducible.
#include "kernels.h"

namespace numbat {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 4096;
constexpr int kVpt = 4;  // 16-byte vectors in flight per thread in the apply kernels

// rows handled together by one block: thread t works on channel vector t % cv of row t / cv
struct RowLayout {
  int cv, rows_per_iter, active;
};
__device__ __forceinline__ RowLayout row_layout(int c) {
  RowLayout r;
  r.cv = c >> 3;
  r.rows_per_iter = kThreads / r.cv;
  if (r.rows_per_iter < 1) r.rows_per_iter = 1;
  r.active = r.rows_per_iter * r.cv;
  return r;
}

// --- standalone statistics of bf16 y: per-block (mean, M2), shifted sums in fp32
__global__ __launch_bounds__(kThreads) void bn_stats_kernel(const bf16_t* y, int64_t y_pix, int64_t m, int c,
                                                            int64_t rows_per_block, float2* part) {
  extern __shared__ float smem[];  // [rows_per_iter][c][2]
  const RowLayout L = row_layout(c);
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  int64_t r1 = r0 + rows_per_block;
  if (r1 > m) r1 = m;
  const int t = threadIdx.x;
  const int rr = t / L.cv, cvi = t - rr * L.cv;
  // shift: the block's first row (same for every thread of a channel)
  float shift[8], s1[8], s2[8];
  const uint4 sv = *reinterpret_cast<const uint4*>(y + r0 * y_pix + cvi * 8);
  unpack8(sv, shift);
#pragma unroll
  for (int e = 0; e < 8; ++e) s1[e] = s2[e] = 0.f;
  if (t < L.active) {
    int64_t r = r0 + rr;
    for (; r + L.rows_per_iter < r1; r += 2 * L.rows_per_iter) {
      float f[8], h[8];
      const uint4 u0 = *reinterpret_cast<const uint4*>(y + r * y_pix + cvi * 8);
      const uint4 u1 = *reinterpret_cast<const uint4*>(y + (r + L.rows_per_iter) * y_pix + cvi * 8);
      unpack8(u0, f);
      unpack8(u1, h);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = f[e] - shift[e], d2 = h[e] - shift[e];
        s1[e] += d;
        s2[e] += d * d;
        s1[e] += d2;
        s2[e] += d2 * d2;
      }
    }
    if (r < r1) {
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(y + r * y_pix + cvi * 8), f);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = f[e] - shift[e];
        s1[e] += d;
        s2[e] += d * d;
      }
    }
  }
  if (t < L.active) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      smem[(rr * c + cvi * 8 + e) * 2 + 0] = s1[e];
      smem[(rr * c + cvi * 8 + e) * 2 + 1] = s2[e];
    }
  }
  __syncthreads();
  const double n = (double)(r1 - r0);
  for (int ch = t; ch < c; ch += kThreads) {
    float a = 0.f, b = 0.f;
    for (int k = 0; k < L.rows_per_iter; ++k) {
      a += smem[(k * c + ch) * 2 + 0];
      b += smem[(k * c + ch) * 2 + 1];
    }
    const float sh = __uint_as_float(((uint32_t)y[r0 * y_pix + ch]) << 16);
    const double mean_d = (double)a / n;
    const float mean = (float)((double)sh + mean_d);
    const float m2 = (float)((double)b - (double)a * mean_d);
    part[(int64_t)blockIdx.x * c + ch] = make_float2(mean, m2 > 0.f ? m2 : 0.f);
  }
}

// --- forward apply: out = SiLU((y - mean) * gamma * rstd + beta) [+ residual]
__global__ __launch_bounds__(kThreads) void bn_fwd_kernel(BnArgs a, FastDiv div_cv, const bf16_t* y,
                                                          const float* mean_var, const float* gamma,
                                                          const float* beta, const bf16_t* res, bf16_t* out,
                                                          float* save_mean, float* save_rstd, float* run_mean,
                                                          float* run_var) {
  extern __shared__ float smem[];  // mean[c], scale[c], beta[c]
  float* s_mean = smem;
  float* s_scale = smem + a.c;
  float* s_beta = smem + 2 * a.c;
  for (int ch = threadIdx.x; ch < a.c; ch += kThreads) {
    const float mu = mean_var[ch], var = mean_var[a.c + ch];
    const float rstd = 1.0f / sqrtf(var + a.eps);
    s_mean[ch] = mu;
    s_scale[ch] = gamma[ch] * rstd;
    s_beta[ch] = beta[ch];
    if (blockIdx.x == 0) {
      save_mean[ch] = mu;
      save_rstd[ch] = rstd;
      if (run_mean != nullptr) {
        const float mo = a.momentum;
        run_mean[ch] = (1.0f - mo) * run_mean[ch] + mo * mu;
        run_var[ch] = (1.0f - mo) * run_var[ch] + mo * (float)((double)var * (double)a.m / (double)(a.m - 1));
      }
    }
  }
  __syncthreads();
  const uint32_t cv = (uint32_t)(a.c >> 3);
  const int64_t total = a.m * (int64_t)cv;
  for (int64_t base = (int64_t)blockIdx.x * kThreads * kVpt; base < total; base += (int64_t)gridDim.x * kThreads * kVpt) {
    uint4 yv[kVpt], rv[kVpt];
    int64_t rowoff[kVpt];
    int cbs[kVpt];
#pragma unroll
    for (int j = 0; j < kVpt; ++j) {
      const int64_t v = base + threadIdx.x + j * kThreads;
      const uint32_t vv = (uint32_t)(v < total ? v : 0);
      const uint32_t row = fdiv(vv, div_cv);
      rowoff[j] = row;
      cbs[j] = (int)(vv - row * cv) * 8;
      if (v < total) {
        yv[j] = *reinterpret_cast<const uint4*>(y + (int64_t)row * a.y_pix + cbs[j]);
        if (res != nullptr) rv[j] = *reinterpret_cast<const uint4*>(res + (int64_t)row * a.r_pix + cbs[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < kVpt; ++j) {
      const int64_t v = base + threadIdx.x + j * kThreads;
      if (v >= total) continue;
      const int cb = cbs[j];
      float f[8], o[8];
      unpack8(yv[j], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float z = (f[e] - s_mean[cb + e]) * s_scale[cb + e] + s_beta[cb + e];
        o[e] = z * sigmoidf_fast(z);
      }
      if (res != nullptr) {
        float r[8];
        unpack8(rv[j], r);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += r[e];
      }
      *reinterpret_cast<uint4*>(out + rowoff[j] * a.a_pix + cb) = pack8(o);
    }
  }
}

// --- backward reduce: per-block sums of dz and dz * xhat
__global__ __launch_bounds__(kThreads) void bn_bwd_reduce_kernel(BnArgs a, const bf16_t* g, const bf16_t* y,
                                                                 const float* save_mean, const float* save_rstd,
                                                                 const float* gamma, const float* beta,
                                                                 int64_t rows_per_block, float2* part) {
  extern __shared__ float smem[];  // consts [3][c] then partials [rows_per_iter][c][2]
  const int c = a.c;
  float* s_mean = smem;
  float* s_rstd = smem + c;
  float* s_gam = smem + 2 * c;
  float* s_bet = smem + 3 * c;
  float* s_red = smem + 4 * c;
  for (int ch = threadIdx.x; ch < c; ch += kThreads) {
    s_mean[ch] = save_mean[ch];
    s_rstd[ch] = save_rstd[ch];
    s_gam[ch] = gamma[ch];
    s_bet[ch] = beta[ch];
  }
  __syncthreads();
  const RowLayout L = row_layout(c);
  const int t = threadIdx.x;
  const int rr = t / L.cv, cvi = t - rr * L.cv;
  const int cb = cvi * 8;
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  int64_t r1 = r0 + rows_per_block;
  if (r1 > a.m) r1 = a.m;
  float sdz[8], sdx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sdz[e] = sdx[e] = 0.f;
  if (t < L.active) {
    auto accum = [&](const uint4& gu, const uint4& yu) {
      float gy[8], yy[8];
      unpack8(gu, gy);
      unpack8(yu, yy);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xh = (yy[e] - s_mean[cb + e]) * s_rstd[cb + e];
        const float z = s_gam[cb + e] * xh + s_bet[cb + e];
        const float sg = sigmoidf_fast(z);
        const float dz = gy[e] * sg * (1.0f + z * (1.0f - sg));
        sdz[e] += dz;
        sdx[e] += dz * xh;
      }
    };
    int64_t r = r0 + rr;
    for (; r + L.rows_per_iter < r1; r += 2 * L.rows_per_iter) {
      const int64_t r2 = r + L.rows_per_iter;
      const uint4 g0 = *reinterpret_cast<const uint4*>(g + r * a.a_pix + cb);
      const uint4 y0 = *reinterpret_cast<const uint4*>(y + r * a.y_pix + cb);
      const uint4 g1 = *reinterpret_cast<const uint4*>(g + r2 * a.a_pix + cb);
      const uint4 y1 = *reinterpret_cast<const uint4*>(y + r2 * a.y_pix + cb);
      accum(g0, y0);
      accum(g1, y1);
    }
    if (r < r1)
      accum(*reinterpret_cast<const uint4*>(g + r * a.a_pix + cb), *reinterpret_cast<const uint4*>(y + r * a.y_pix + cb));
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s_red[(rr * c + cb + e) * 2 + 0] = sdz[e];
      s_red[(rr * c + cb + e) * 2 + 1] = sdx[e];
    }
  }
  __syncthreads();
  for (int ch = t; ch < c; ch += kThreads) {
    float p = 0.f, q = 0.f;
    for (int k = 0; k < L.rows_per_iter; ++k) {
      p += s_red[(k * c + ch) * 2 + 0];
      q += s_red[(k * c + ch) * 2 + 1];
    }
    part[(int64_t)blockIdx.x * c + ch] = make_float2(p, q);
  }
}

// --- backward finalize: fixed-order fp64 sums over blocks -> dbeta, dgamma and apply coefficients
constexpr int kFinGroups = 16;
__global__ __launch_bounds__(64 * kFinGroups) void bn_bwd_finalize_kernel(const float2* part, int nblocks, int c,
                                                                          int64_t m, const float* save_rstd,
                                                                          const float* gamma, float* dgamma,
                                                                          float* dbeta, float* coef) {
  __shared__ double sa[kFinGroups][64], sb[kFinGroups][64];
  const int cl = threadIdx.x & 63, gidx = threadIdx.x >> 6;
  const int ch = blockIdx.x * 64 + cl;
  double p = 0, q = 0;
  if (ch < c)
    for (int b = gidx; b < nblocks; b += kFinGroups) {
      const float2 v = part[(int64_t)b * c + ch];
      p += v.x;
      q += v.y;
    }
  sa[gidx][cl] = p;
  sb[gidx][cl] = q;
  __syncthreads();
  if (gidx == 0 && ch < c) {
    for (int k = 1; k < kFinGroups; ++k) {
      p += sa[k][cl];
      q += sb[k][cl];
    }
    dbeta[ch] = (float)p;
    dgamma[ch] = (float)q;
    coef[ch] = gamma[ch] * save_rstd[ch];
    coef[c + ch] = (float)(p / (double)m);
    coef[2 * c + ch] = (float)(q / (double)m);
  }
}

// --- backward apply: dy = gamma * rstd * (dz - dbeta/m - xhat * dgamma/m); residual_grad += g
__global__ __launch_bounds__(kThreads) void bn_bwd_apply_kernel(BnArgs a, FastDiv div_cv, const bf16_t* g,
                                                                const bf16_t* y, const float* save_mean,
                                                                const float* save_rstd, const float* gamma,
                                                                const float* beta, const float* coef, bf16_t* dy,
                                                                bf16_t* res_grad) {
  extern __shared__ float smem[];  // mean, rstd, gamma, beta, k1, k2, k3  [7][c]
  const int c = a.c;
  for (int ch = threadIdx.x; ch < c; ch += kThreads) {
    smem[ch] = save_mean[ch];
    smem[c + ch] = save_rstd[ch];
    smem[2 * c + ch] = gamma[ch];
    smem[3 * c + ch] = beta[ch];
    smem[4 * c + ch] = coef[ch];
    smem[5 * c + ch] = coef[c + ch];
    smem[6 * c + ch] = coef[2 * c + ch];
  }
  __syncthreads();
  const uint32_t cv = (uint32_t)(c >> 3);
  const int64_t total = a.m * (int64_t)cv;
  for (int64_t base = (int64_t)blockIdx.x * kThreads * kVpt; base < total; base += (int64_t)gridDim.x * kThreads * kVpt) {
    uint4 gv[kVpt], yv[kVpt], rv[kVpt];
    int64_t rows[kVpt];
    int cbs[kVpt];
#pragma unroll
    for (int j = 0; j < kVpt; ++j) {
      const int64_t v = base + threadIdx.x + j * kThreads;
      const uint32_t vv = (uint32_t)(v < total ? v : 0);
      const uint32_t row = fdiv(vv, div_cv);
      rows[j] = row;
      cbs[j] = (int)(vv - row * cv) * 8;
      if (v < total) {
        gv[j] = *reinterpret_cast<const uint4*>(g + (int64_t)row * a.a_pix + cbs[j]);
        yv[j] = *reinterpret_cast<const uint4*>(y + (int64_t)row * a.y_pix + cbs[j]);
        if (res_grad != nullptr) rv[j] = *reinterpret_cast<const uint4*>(res_grad + (int64_t)row * a.r_pix + cbs[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < kVpt; ++j) {
      const int64_t v = base + threadIdx.x + j * kThreads;
      if (v >= total) continue;
      const int cb = cbs[j];
      float gy[8], yy[8], o[8];
      unpack8(gv[j], gy);
      unpack8(yv[j], yy);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int ch = cb + e;
        const float xh = (yy[e] - smem[ch]) * smem[c + ch];
        const float z = smem[2 * c + ch] * xh + smem[3 * c + ch];
        const float sg = sigmoidf_fast(z);
        const float dz = gy[e] * sg * (1.0f + z * (1.0f - sg));
        o[e] = smem[4 * c + ch] * (dz - smem[5 * c + ch] - xh * smem[6 * c + ch]);
      }
      *reinterpret_cast<uint4*>(dy + rows[j] * a.dy_pix + cb) = pack8(o);
      if (res_grad != nullptr) {
        float r[8];
        unpack8(rv[j], r);
#pragma unroll
        for (int e = 0; e < 8; ++e) r[e] += gy[e];
        *reinterpret_cast<uint4*>(res_grad + rows[j] * a.r_pix + cb) = pack8(r);
      }
    }
  }
}

int grid_for_elems(int64_t vecs) {
  int64_t b = (vecs + kThreads * kVpt - 1) / (kThreads * kVpt);
  if (b > 8192) b = 8192;
  if (b < 1) b = 1;
  return (int)b;
}

size_t reduce_smem(int c) {
  const int cv = c / 8;
  int rpi = kThreads / cv;
  if (rpi < 1) rpi = 1;
  return (size_t)rpi * c * 2 * sizeof(float);
}

}  // namespace

int bn_reduce_blocks(int64_t m, int c) {
  // about 8 vectors of 8 channels per thread
  int64_t b = (m * (c / 8) + kThreads * 8 - 1) / (kThreads * 8);
  if (b > kMaxBlocks) b = kMaxBlocks;
  if (b < 1) b = 1;
  return (int)b;
}

static int64_t rows_per_block(int64_t m, int nblocks) { return (m + nblocks - 1) / nblocks; }

hipError_t bn_stats_launch(const BnArgs& a, const bf16_t* y, float* part3, int nblocks, float* mean_var,
                           hipStream_t s) {
  const int64_t rpb = rows_per_block(a.m, nblocks);
  const int nb = (int)((a.m + rpb - 1) / rpb);
  float2* part = reinterpret_cast<float2*>(part3);
  trace_begin(KC_BN_STATS, s);
  hipLaunchKernelGGL(bn_stats_kernel, dim3(nb), dim3(kThreads), reduce_smem(a.c), s, y, a.y_pix, a.m, a.c, rpb,
                     part);
  trace_end(KC_BN_STATS, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return stats_merge_launch(part, nb, (int)rpb, a.m, a.c, mean_var, s);
}

hipError_t bn_fwd_launch(const BnArgs& a, const bf16_t* y, const float* mean_var, const float* gamma,
                         const float* beta, const bf16_t* res, bf16_t* out, float* save_mean, float* save_rstd,
                         float* run_mean, float* run_var, hipStream_t s) {
  const int64_t vecs = a.m * (a.c / 8);
  const FastDiv d = make_fastdiv((uint32_t)(a.c / 8));
  trace_begin(KC_BN_FWD, s);
  hipLaunchKernelGGL(bn_fwd_kernel, dim3(grid_for_elems(vecs)), dim3(kThreads), 3 * a.c * sizeof(float), s, a, d, y,
                     mean_var, gamma, beta, res, out, save_mean, save_rstd, run_mean, run_var);
  trace_end(KC_BN_FWD, s);
  return hipGetLastError();
}

hipError_t bn_bwd_launch(const BnArgs& a, const bf16_t* g, const bf16_t* y, const float* save_mean,
                         const float* save_rstd, const float* gamma, const float* beta, bf16_t* dy, float* dgamma,
                         float* dbeta, bf16_t* res_grad, float* part2, int nblocks, float* coef, hipStream_t s) {
  const int64_t rpb = rows_per_block(a.m, nblocks);
  const int nb = (int)((a.m + rpb - 1) / rpb);
  float2* part = reinterpret_cast<float2*>(part2);
  trace_begin(KC_BN_BWD_REDUCE, s);
  hipLaunchKernelGGL(bn_bwd_reduce_kernel, dim3(nb), dim3(kThreads), 4 * a.c * sizeof(float) + reduce_smem(a.c), s,
                     a, g, y, save_mean, save_rstd, gamma, beta, rpb, part);
  trace_end(KC_BN_BWD_REDUCE, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_begin(KC_BN_BWD_FINALIZE, s);
  hipLaunchKernelGGL(bn_bwd_finalize_kernel, dim3((a.c + 63) / 64), dim3(64 * kFinGroups), 0, s, part, nb, a.c, a.m,
                     save_rstd, gamma, dgamma, dbeta, coef);
  trace_end(KC_BN_BWD_FINALIZE, s);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t vecs = a.m * (a.c / 8);
  const FastDiv d = make_fastdiv((uint32_t)(a.c / 8));
  trace_begin(KC_BN_BWD_APPLY, s);
  hipLaunchKernelGGL(bn_bwd_apply_kernel, dim3(grid_for_elems(vecs)), dim3(kThreads), 7 * a.c * sizeof(float), s, a,
                     d, g, y, save_mean, save_rstd, gamma, beta, coef, dy, res_grad);
  trace_end(KC_BN_BWD_APPLY, s);
  return hipGetLastError();
}

}  // namespace numbat

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

// --- forward apply: out = SiLU((y - mean) * gamma * rstd + beta) [+ residual].
// Thread t always handles channel vector t % cv, so its per-channel constants sit in
// registers; rows advance by rows_per_iter, four rows in flight.
__global__ __launch_bounds__(kThreads) void bn_fwd_kernel(BnArgs a, const bf16_t* y, const float* mean,
                                                          const float* var_in, const float* gamma, const float* beta,
                                                          const bf16_t* res, bf16_t* out, float* save_mean,
                                                          float* save_rstd, float* run_mean, float* run_var,
                                                          int64_t rows_per_block, int stat_block) {
  const int t = threadIdx.x;
  // the last block (when save_mean is given) only publishes the saved statistics and
  // updates the running ones, in parallel with the row blocks (done by a row block, it
  // would lengthen that block by a round trip to memory)
  if (stat_block && blockIdx.x == gridDim.x - 1) {
    for (int ch = t; ch < a.c; ch += kThreads) {
      const float mu = mean[ch], var = var_in[ch];
      save_mean[ch] = mu;
      save_rstd[ch] = 1.0f / sqrtf(var + a.eps);
      if (run_mean != nullptr) {
        const float mo = a.momentum;
        run_mean[ch] = (1.0f - mo) * run_mean[ch] + mo * mu;
        run_var[ch] = (1.0f - mo) * run_var[ch] + mo * (float)((double)var * (double)a.m / (double)(a.m - 1));
      }
    }
    return;
  }
  const RowLayout L = row_layout(a.c);
  if (t >= L.active) return;
  const int rr = t / L.cv, cb = (t - rr * L.cv) * 8;
  // z = (y - mu) * gamma * rstd + beta, as one multiply-add per element
  float sc[8], bz[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bn_fold(gamma[cb + e], beta[cb + e], mean[cb + e], var_in[cb + e], a.eps, sc[e], bz[e]);
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = r0 + rows_per_block < a.m ? r0 + rows_per_block : a.m;
  const int64_t st = L.rows_per_iter;
  for (int64_t r = r0 + rr; r < r1; r += 4 * st) {
    uint4 yv[4], rv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t rj = r + j * st;
      if (rj < r1) {
        yv[j] = *reinterpret_cast<const uint4*>(y + rj * a.y_pix + cb);
        if (res != nullptr) rv[j] = *reinterpret_cast<const uint4*>(res + rj * a.r_pix + cb);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t rj = r + j * st;
      if (rj >= r1) continue;
      float f[8], o[8];
      unpack8(yv[j], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = bn_silu_apply(f[e], sc[e], bz[e]);
      if (res != nullptr) {
        float q[8];
        unpack8(rv[j], q);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += q[e];
      }
      *reinterpret_cast<uint4*>(out + rj * a.a_pix + cb) = pack8(o);
    }
  }
}

// --- backward reduce: per-block sums of dz and dz * xhat (row layout, constants in registers)
__global__ __launch_bounds__(kThreads) void bn_bwd_reduce_kernel(BnArgs a, const bf16_t* g, const bf16_t* y,
                                                                 const float* save_mean, const float* save_rstd,
                                                                 const float* gamma, const float* beta,
                                                                 int64_t rows_per_block, float2* part) {
  extern __shared__ float s_red[];  // [rows_per_iter][c][2]
  const int c = a.c;
  const RowLayout L = row_layout(c);
  const int t = threadIdx.x;
  const int rr = t / L.cv, cb = (t - rr * L.cv) * 8;
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = r0 + rows_per_block < a.m ? r0 + rows_per_block : a.m;
  float sdz[8], sdx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sdz[e] = sdx[e] = 0.f;
  if (t < L.active) {
    // xhat = (y - mu) * rstd as one multiply-add per element
    float nm[8], rs[8], ga[8], be[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      rs[e] = save_rstd[cb + e];
      nm[e] = -save_mean[cb + e] * rs[e];
      ga[e] = gamma[cb + e];
      be[e] = beta[cb + e];
    }
    const int64_t st = L.rows_per_iter;
    // eight rows in flight per round: with the block count bn_reduce_blocks picks, one
    // full round (more on layers large enough to meet its block cap)
    for (int64_t r = r0 + rr; r < r1; r += 8 * st) {
      uint4 gv[8], yv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int64_t rj = r + j * st;
        if (rj < r1) {
          gv[j] = *reinterpret_cast<const uint4*>(g + rj * a.a_pix + cb);
          yv[j] = *reinterpret_cast<const uint4*>(y + rj * a.y_pix + cb);
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (r + j * st >= r1) continue;
        float gy[8], yy[8];
        unpack8(gv[j], gy);
        unpack8(yv[j], yy);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = __builtin_fmaf(yy[e], rs[e], nm[e]);
          const float z = __builtin_fmaf(ga[e], xh, be[e]);
          const float sg = sigmoidf_fast(z);
          const float dz = gy[e] * sg * (1.0f + z * (1.0f - sg));
          sdz[e] += dz;
          sdx[e] += dz * xh;
        }
      }
    }
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

// --- backward finalize: fixed-order fp64 sums over blocks -> dbeta, dgamma, and the apply's
// folded constants (bn_bwd_fold of the rounded dgamma, dbeta) as coef[4][c].
// 8 channels per block, G groups of partial rows per channel (a few loads in flight per
// lane); the group sums are combined by shuffles within each wave (8 groups) and then the
// G/8 wave sums by a pairwise tree, in a fixed order that depends only on G.
constexpr int kFinCh = 8;
template <int G>
__global__ __launch_bounds__(kFinCh * G) void bn_bwd_finalize_kernel(const float2* part, int nblocks, int c, int64_t m,
                                                                     const float* save_mean, const float* save_rstd,
                                                                     const float* gamma, const float* beta,
                                                                     float* dgamma, float* dbeta, float* coef) {
  constexpr int NWV = G / 8;  // waves
  __shared__ double sa[NWV][kFinCh], sb[NWV][kFinCh];
  const int cl = threadIdx.x % kFinCh, gidx = threadIdx.x / kFinCh;
  const int ch = blockIdx.x * kFinCh + cl;
  double p = 0, q = 0;
  if (ch < c) {
#pragma unroll 4
    for (int b = gidx; b < nblocks; b += G) {
      const float2 v = part[(int64_t)b * c + ch];
      p += v.x;
      q += v.y;
    }
  }
  // lanes 8 apart hold the same channel of neighbouring groups
#pragma unroll
  for (int d = 8; d < 64; d *= 2) {
    p += __shfl_xor(p, d);
    q += __shfl_xor(q, d);
  }
  const int wave = threadIdx.x / 64;
  if ((threadIdx.x & 63) < kFinCh) {
    sa[wave][cl] = p;
    sb[wave][cl] = q;
  }
  __syncthreads();
  if (gidx == 0 && ch < c) {
    double ta[NWV], tb[NWV];
#pragma unroll
    for (int w = 0; w < NWV; ++w) {
      ta[w] = sa[w][cl];
      tb[w] = sb[w][cl];
    }
#pragma unroll
    for (int h = NWV / 2; h >= 1; h /= 2)
#pragma unroll
      for (int w = 0; w < h; ++w) {
        ta[w] += ta[w + h];
        tb[w] += tb[w + h];
      }
    p = ta[0];
    q = tb[0];
    const float db = (float)p, dg = (float)q;
    dbeta[ch] = db;
    dgamma[ch] = dg;
    bn_bwd_fold(gamma[ch], beta[ch], save_mean[ch], save_rstd[ch], dg, db, m, coef[ch], coef[c + ch],
                coef[2 * c + ch], coef[3 * c + ch]);
  }
}

// --- backward apply: dy = gamma * rstd * (dz - dbeta/m - xhat * dgamma/m); residual_grad += g
// (row layout, the finalize's folded constants in registers, four rows in flight)
__global__ __launch_bounds__(kThreads) void bn_bwd_apply_kernel(BnArgs a, const bf16_t* g, const bf16_t* y,
                                                                const float* coef, bf16_t* dy, bf16_t* res_grad,
                                                                int64_t rows_per_block) {
  const int c = a.c;
  const RowLayout L = row_layout(c);
  const int t = threadIdx.x;
  if (t >= L.active) return;
  const int rr = t / L.cv, cb = (t - rr * L.cv) * 8;
  float ka[8], kb[8], kc[8], kd[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    ka[e] = coef[cb + e];
    kb[e] = coef[c + cb + e];
    kc[e] = coef[2 * c + cb + e];
    kd[e] = coef[3 * c + cb + e];
  }
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = r0 + rows_per_block < a.m ? r0 + rows_per_block : a.m;
  const int64_t st = L.rows_per_iter;
  for (int64_t r = r0 + rr; r < r1; r += 4 * st) {
    uint4 gv[4], yv[4], rv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t rj = r + j * st;
      if (rj < r1) {
        gv[j] = *reinterpret_cast<const uint4*>(g + rj * a.a_pix + cb);
        yv[j] = *reinterpret_cast<const uint4*>(y + rj * a.y_pix + cb);
        if (res_grad != nullptr) rv[j] = *reinterpret_cast<const uint4*>(res_grad + rj * a.r_pix + cb);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t rj = r + j * st;
      if (rj >= r1) continue;
      float gy[8], yy[8], o[8];
      unpack8(gv[j], gy);
      unpack8(yv[j], yy);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = bn_silu_bwd_apply(gy[e], yy[e], ka[e], kb[e], kc[e], kd[e]);
      *reinterpret_cast<uint4*>(dy + rj * a.dy_pix + cb) = pack8(o);
      if (res_grad != nullptr) {
        float q[8];
        unpack8(rv[j], q);
#pragma unroll
        for (int e = 0; e < 8; ++e) q[e] += gy[e];
        *reinterpret_cast<uint4*>(res_grad + rj * a.r_pix + cb) = pack8(q);
      }
    }
  }
}

size_t reduce_smem(int c) {
  const int cv = c / 8;
  int rpi = kThreads / cv;
  if (rpi < 1) rpi = 1;
  return (size_t)rpi * c * 2 * sizeof(float);
}

}  // namespace

int bn_reduce_blocks(int64_t m, int c) {
  // 8 rows per active thread, one round: a block covers 8 * rows_per_iter rows (counting
  // all kThreads threads as active gave most layers a nearly empty last round).  Against
  // two rounds of eight (half the blocks and partials) the reduce kernels take 0.875
  // instead of 0.98 ms per step and the two-stream step is unchanged (8.54 ms; with the
  // earlier weight-gradient kernels two rounds were 0.5% faster); four rows per thread
  // were slower.
  int64_t vpt = 8;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_BN_VEC")) vpt = atoi(e);
#endif
  const int cv = c / 8;
  int64_t rpi = cv > 0 ? kThreads / cv : 1;
  if (rpi < 1) rpi = 1;
  int64_t b = (m + rpi * vpt - 1) / (rpi * vpt);
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
  trace_begin(KC_BN_STATS);
  NUMBAT_LAUNCH(bn_stats_kernel, dim3(nb), dim3(kThreads), reduce_smem(a.c), s, y, a.y_pix, a.m, a.c, rpb,
                     part);
  trace_end(KC_BN_STATS);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return stats_merge_launch(part, nb, (int)rpb, a.m, a.c, mean_var, s);
}

// apply kernels: 4 rows of 8 channels per thread, all four loads in flight at once — these
// passes are latency-bound on most layers, so more blocks with one round trip each beat
// fewer blocks that loop (measured over the detector's layers: 16 rows per thread cost
// 0.45 ms more per training step)
static int apply_blocks(int64_t m, int c, int64_t* rows_per_block) {
  const int cv = c / 8;
  int rpi = kThreads / cv;
  if (rpi < 1) rpi = 1;
  int64_t rows = 4;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_BN_ROWS")) rows = atoi(e);
#endif
  int64_t b = (m + (int64_t)rpi * rows - 1) / ((int64_t)rpi * rows);
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  *rows_per_block = (m + b - 1) / b;
  return (int)((m + *rows_per_block - 1) / *rows_per_block);
}

hipError_t bn_fwd_launch(const BnArgs& a, const bf16_t* y, const float* mean, const float* var, const float* gamma,
                         const float* beta, const bf16_t* res, bf16_t* out, float* save_mean, float* save_rstd,
                         float* run_mean, float* run_var, hipStream_t s) {
  int64_t rpb = 0;
  const int nb = apply_blocks(a.m, a.c, &rpb);
  const int stat = save_mean != nullptr ? 1 : 0;
  trace_begin(KC_BN_FWD);
  NUMBAT_LAUNCH(bn_fwd_kernel, dim3(nb + stat), dim3(kThreads), 0, s, a, y, mean, var, gamma, beta, res, out,
                     save_mean, save_rstd, run_mean, run_var, rpb, stat);
  trace_end(KC_BN_FWD);
  return hipGetLastError();
}

hipError_t bn_bwd_launch(const BnArgs& a, const bf16_t* g, const bf16_t* y, const float* save_mean,
                         const float* save_rstd, const float* gamma, const float* beta, bf16_t* dy, float* dgamma,
                         float* dbeta, bf16_t* res_grad, float* part2, int nblocks, float* coef, hipStream_t s) {
  const int64_t rpb = rows_per_block(a.m, nblocks);
  const int nb = (int)((a.m + rpb - 1) / rpb);
  float2* part = reinterpret_cast<float2*>(part2);
  trace_begin(KC_BN_BWD_REDUCE);
  NUMBAT_LAUNCH(bn_bwd_reduce_kernel, dim3(nb), dim3(kThreads), reduce_smem(a.c), s, a, g, y, save_mean,
                     save_rstd, gamma, beta, rpb, part);
  trace_end(KC_BN_BWD_REDUCE);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_begin(KC_BN_BWD_FINALIZE);
  // about eight partial rows per lane
  const dim3 fgrid((a.c + kFinCh - 1) / kFinCh);
  int fg = nb <= 256 ? 32 : nb <= 512 ? 64 : 128;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_BN_FING")) fg = atoi(e);
#endif
  if (fg == 128)
    NUMBAT_LAUNCH(bn_bwd_finalize_kernel<128>, fgrid, dim3(kFinCh * 128), 0, s, part, nb, a.c, a.m, save_mean,
                  save_rstd, gamma, beta, dgamma, dbeta, coef);
  else if (fg == 64)
    NUMBAT_LAUNCH(bn_bwd_finalize_kernel<64>, fgrid, dim3(kFinCh * 64), 0, s, part, nb, a.c, a.m, save_mean,
                  save_rstd, gamma, beta, dgamma, dbeta, coef);
  else
    NUMBAT_LAUNCH(bn_bwd_finalize_kernel<32>, fgrid, dim3(kFinCh * 32), 0, s, part, nb, a.c, a.m, save_mean,
                  save_rstd, gamma, beta, dgamma, dbeta, coef);
  trace_end(KC_BN_BWD_FINALIZE);
  e = hipGetLastError();
  if (e != hipSuccess || dy == nullptr) return e;  // (no dy: the statistics gradients only)
  int64_t arpb = 0;
  const int anb = apply_blocks(a.m, a.c, &arpb);
  trace_begin(KC_BN_BWD_APPLY);
  NUMBAT_LAUNCH(bn_bwd_apply_kernel, dim3(anb), dim3(kThreads), 0, s, a, g, y, (const float*)coef, dy, res_grad,
                arpb);
  trace_end(KC_BN_BWD_APPLY);
  return hipGetLastError();
}

}  // namespace numbat

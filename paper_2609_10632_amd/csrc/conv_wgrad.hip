// Weight gradient dW[o][k] = sum_m dy[m][o] * X[m][k] on gfx950 MFMA, where m runs over
// the n*ho*wo output pixels and X[m][(tap, c)] is the input pixel that tap reads.
//
// In NHWC both operands are contiguous along o / k and strided along the reduction
// dimension m, while an MFMA lane needs 8 consecutive reduction elements.  Each thread
// therefore loads an 8-pixel x 8-channel block (eight 16-byte loads), transposes it in
// registers with byte permutes, and writes eight 16-byte rows of [channel][pixel] into
// LDS.  The reduction over m is split into fixed contiguous ranges, one per
// blockIdx.z, whose fp32 partial sums are added afterwards in split order, so the
// result does not depend on scheduling.
#include "kernels.h"

namespace numbat {

namespace {

constexpr int BR = 64;           // reduction pixels per step
constexpr int LROW = BR + 8;     // bf16 per LDS row (16 B pad)

__device__ __forceinline__ uint32_t lo_pair(uint32_t p0, uint32_t p1) {
  return __builtin_amdgcn_perm(p1, p0, 0x05040100u);  // (p0.lo16, p1.lo16)
}
__device__ __forceinline__ uint32_t hi_pair(uint32_t p0, uint32_t p1) {
  return __builtin_amdgcn_perm(p1, p0, 0x07060302u);  // (p0.hi16, p1.hi16)
}
__device__ __forceinline__ uint32_t word(const uint4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// in: P[j] = 8 channels of pixel j.  out: Q[ch] = 8 pixels of channel ch.
__device__ __forceinline__ void transpose8x8(const uint4 P[8], uint4 Q[8]) {
#pragma unroll
  for (int ch = 0; ch < 8; ++ch) {
    const int wi = ch >> 1;
    uint32_t q[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t a = word(P[2 * k], wi), b = word(P[2 * k + 1], wi);
      q[k] = (ch & 1) ? hi_pair(a, b) : lo_pair(a, b);
    }
    Q[ch] = make_uint4(q[0], q[1], q[2], q[3]);
  }
}

template <int TM, int TN>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a, FastDiv div_wo, FastDiv div_howo) {
  constexpr int BMO = 2 * TM * 16;  // output channels per tile
  constexpr int BNK = 2 * TN * 16;  // k columns per tile
  constexpr int UDY = (BMO / 8) * (BR / 8);
  constexpr int UX = (BNK / 8) * (BR / 8);
  constexpr int UNITS = UDY + UX;
  constexpr int UPT = (UNITS + 255) / 256;  // units per thread

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BMO][LROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNK][LROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int o0 = blockIdx.x * BMO;
  const int k0 = blockIdx.y * BNK;
  const int64_t rbeg = (int64_t)blockIdx.z * a.rows_per_split;
  int64_t rend = rbeg + a.rows_per_split;
  if (rend > a.m) rend = a.m;
  const int nsteps = rend > rbeg ? (int)((rend - rbeg + BR - 1) / BR) : 0;

  // per-unit static description
  int u_isx[UPT], u_grp[UPT], u_pb[UPT];
  int u_dh[UPT], u_dw[UPT], u_c[UPT];
  bool u_ok[UPT];
#pragma unroll
  for (int t = 0; t < UPT; ++t) {
    const int u = tid + 256 * t;
    u_ok[t] = u < UNITS;
    const bool isx = u >= UDY;
    const int v = isx ? u - UDY : u;
    u_isx[t] = isx;
    u_grp[t] = v >> 3;  // channel group (dy) or k group (x)
    u_pb[t] = v & 7;    // pixel block within the step
    u_dh[t] = u_dw[t] = u_c[t] = 0;
    if (isx) {
      const int k = k0 + u_grp[t] * 8;
      const int tap = k / a.ci;
      u_c[t] = k - tap * a.ci;
      u_dh[t] = tap / a.kw - a.ph;
      u_dw[t] = tap % a.kw - a.pw;
    }
  }

  uint4 Q[UPT][8];

  auto load_step = [&](int st) {
    const int64_t pbase = rbeg + (int64_t)st * BR;
#pragma unroll
    for (int t = 0; t < UPT; ++t) {
      uint4 P[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) P[j] = make_uint4(0, 0, 0, 0);
      if (u_ok[t]) {
        const int64_t px0 = pbase + u_pb[t] * 8;
        if (!u_isx[t]) {
          const int o = o0 + u_grp[t] * 8;
          if (o < a.co) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const int64_t px = px0 + j;
              if (px < rend) P[j] = *reinterpret_cast<const uint4*>(a.dy + px * a.dy_pix + o);
            }
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int64_t px = px0 + j;
            if (px >= rend) continue;
            const uint32_t pm = (uint32_t)px;
            const uint32_t img = fdiv(pm, div_howo);
            const uint32_t rem = pm - img * (uint32_t)(a.ho * a.wo);
            const uint32_t p = fdiv(rem, div_wo);
            const uint32_t q = rem - p * (uint32_t)a.wo;
            const int ihb = (int)p * a.sh, iwb = (int)q * a.sw;
            const int64_t ibase = (int64_t)img * a.h;
            {
              const int k = k0 + u_grp[t] * 8;
              const int ih = ihb + u_dh[t], iw = iwb + u_dw[t];
              if (k < a.ktot && (unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w)
                P[j] = *reinterpret_cast<const uint4*>(a.x + ((ibase + ih) * a.w + iw) * a.x_pix + u_c[t]);
            }
          }
        }
      }
      transpose8x8(P, Q[t]);
    }
  };

  auto store_step = [&](int buf) {
#pragma unroll
    for (int t = 0; t < UPT; ++t) {
      if (!u_ok[t]) continue;
      const int row0 = u_grp[t] * 8;
      const int col = u_pb[t] * 8;
      if (!u_isx[t]) {
#pragma unroll
        for (int c = 0; c < 8; ++c) *reinterpret_cast<uint4*>(&As[buf][row0 + c][col]) = Q[t][c];
      } else {
#pragma unroll
        for (int c = 0; c < 8; ++c) *reinterpret_cast<uint4*>(&Bs[buf][row0 + c][col]) = Q[t][c];
      }
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nsteps > 0) {
    load_step(0);
    store_step(0);
    __syncthreads();
  }
  for (int st = 0; st < nsteps; ++st) {
    const int buf = st & 1;
    if (st + 1 < nsteps) load_step(st + 1);
#pragma unroll
    for (int ks = 0; ks < BR / 32; ++ks) {
      const int kc = ks * 32 + (lane >> 4) * 8;
      uint4 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const uint4*>(&As[buf][wm * TM * 16 + i * 16 + (lane & 15)][kc]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const uint4*>(&Bs[buf][wn * TN * 16 + j * 16 + (lane & 15)][kc]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
    }
    if (st + 1 < nsteps) store_step(buf ^ 1);
    __syncthreads();
  }

  // epilogue: rows = output channels, cols = k
  float* out = a.out + (a.splits > 1 ? (int64_t)blockIdx.z * a.co * a.ktot : 0);
  const bool acc_in = a.splits == 1 && a.accumulate;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int o = o0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + e;
      if (o >= a.co) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int k = k0 + wn * TN * 16 + j * 16 + (lane & 15);
        if (k >= a.ktot) continue;
        float* p = out + (int64_t)o * a.ktot + k;
        const float v = acc[i][j][e];
        *p = acc_in ? *p + v : v;
      }
    }
}

template <int TM, int TN>
hipError_t launch_w(const WgradArgs& a, hipStream_t s) {
  constexpr int BMO = 2 * TM * 16, BNK = 2 * TN * 16;
  dim3 grid((a.co + BMO - 1) / BMO, (a.ktot + BNK - 1) / BNK, a.splits);
  const FastDiv dwo = make_fastdiv((uint32_t)a.wo), dhw = make_fastdiv((uint32_t)(a.ho * a.wo));
  trace_begin(KC_WGRAD, s);
  hipLaunchKernelGGL((wgrad_kernel<TM, TN>), grid, dim3(256), 0, s, a, dwo, dhw);
  trace_end(KC_WGRAD, s);
  return hipGetLastError();
}

// dw = [dw +] sum over splits in split order; four consecutive outputs per thread
__global__ void splitk_reduce_kernel(const float4* part, int splits, int64_t count4, float* dw, int accumulate) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count4; i += (int64_t)gridDim.x * blockDim.x) {
    float4 t = part[i];
    int k = 1;
    for (; k + 1 < splits; k += 2) {
      const float4 u = part[(int64_t)k * count4 + i];
      const float4 v = part[(int64_t)(k + 1) * count4 + i];
      t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
      t.x += v.x; t.y += v.y; t.z += v.z; t.w += v.w;
    }
    if (k < splits) {
      const float4 u = part[(int64_t)k * count4 + i];
      t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
    }
    float* o = dw + 4 * i;
    if (accumulate) {
      t.x = o[0] + t.x; t.y = o[1] + t.y; t.z = o[2] + t.z; t.w = o[3] + t.w;
    }
    o[0] = t.x; o[1] = t.y; o[2] = t.z; o[3] = t.w;
  }
}

}  // namespace

int wgrad_pick_splits(int64_t m, int co, int ktot, int64_t* rows_per_split) {
  const int tiles = (int)(((co + 127) / 128) * ((ktot + 127) / 128));
  const int64_t steps = (m + BR - 1) / BR;
  int64_t splits = (512 + tiles - 1) / tiles;
  // at least 16 steps per split, at most 256 splits, partials at most 64 MiB
  const int64_t max_by_steps = steps / 16 > 0 ? steps / 16 : 1;
  if (splits > max_by_steps) splits = max_by_steps;
  if (splits > 256) splits = 256;
  const int64_t part_bytes = (int64_t)co * ktot * 4;
  while (splits > 1 && splits * part_bytes > (64ll << 20)) --splits;
  if (splits < 1) splits = 1;
  const int64_t steps_per = (steps + splits - 1) / splits;
  *rows_per_split = steps_per * BR;
  splits = (int)((m + *rows_per_split - 1) / *rows_per_split);
  return (int)(splits < 1 ? 1 : splits);
}

hipError_t wgrad_launch(const WgradArgs& a, hipStream_t s) { return launch_w<4, 4>(a, s); }

hipError_t splitk_reduce_launch(const float* part, int splits, int64_t count, float* dw, int accumulate,
                                hipStream_t s) {
  // count = c_out * k_total is a multiple of 8 (c_out is)
  const int64_t count4 = count / 4;
  int64_t blocks = (count4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  trace_begin(KC_SPLITK_REDUCE, s);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     reinterpret_cast<const float4*>(part), splits, count4, dw, accumulate);
  trace_end(KC_SPLITK_REDUCE, s);
  return hipGetLastError();
}

}  // namespace numbat

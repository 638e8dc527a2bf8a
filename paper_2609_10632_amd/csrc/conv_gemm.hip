// Implicit-GEMM convolution on gfx950 MFMA, second generation (bf16 in, fp32 accumulate).
//
// Computes the GEMM family described with ConvGemmArgs: the forward convolution (one
// phase) and all stride phases of a data gradient (one launch, blockIdx.z = phase).
//
// Differences from the first kernel, all aimed at keeping the MFMA pipes fed:
//  * 256-row tiles with one 64 x BN wave tile per wave (BN up to 128), so each LDS
//    fragment feeds more MFMAs;
//  * the gather address of an A vector costs a bit test and a 64-bit add: every tile
//    row keeps a pointer to its source pixel and a bitmask of the taps that land inside
//    the image, and the per-tap pixel offsets sit in LDS;
//  * BK = 32 with two LDS stages (about 60 KB), so two blocks share a CU and hide each
//    other's global-load latency;
//  * the epilogue stages fp32 results through LDS and writes whole 16-byte vectors of
//    8 channels (bf16, rounded once, after the optional accumulate).
#include <type_traits>

#include "kernels.h"

namespace numbat {

namespace {

constexpr int GK = 32;          // reduction elements per pipeline step
constexpr int GROW = GK + 8;    // bf16 per LDS row (80 bytes: conflict-free 16-byte fragment reads)

// Sixteen zero bytes in the code object.  Gather lanes that fall on zero padding (or
// past the end of K or N) load from here instead of being predicated off, so every
// step issues the same number of loads and the compiler can wait for exactly the ring
// slot it needs instead of for every outstanding load.
// (Not const: a const object would live in the constant address space, and a select
// between it and a global pointer would degrade every gather load to a flat load.)
__device__ __attribute__((aligned(16))) u32x4 kZero16 = {0u, 0u, 0u, 0u};

template <int V>
using Ic = std::integral_constant<int, V>;

template <int WM, int TM, int TN>
struct GemmShape {
  static constexpr int WN = 4 / WM;
  static constexpr int WTM = TM * 16, WTN = TN * 16;
  static constexpr int BM = WM * WTM, BN = WN * WTN;
  static constexpr int AV = BM / 64;         // A vectors per thread per step
  static constexpr int BV = (BN + 63) / 64;  // B vectors per thread per step
  static constexpr int A_BYTES = 2 * BM * GROW * 2;
  static constexpr int B_BYTES = 2 * BN * GROW * 2;
  static constexpr int STAGE_LD = WTN + 4;                // fp32 per staged row
  static constexpr int STAGE_BYTES = 4 * 16 * STAGE_LD * 4;  // 16 rows per wave
  static constexpr int SMEM = (A_BYTES + B_BYTES) > STAGE_BYTES ? (A_BYTES + B_BYTES) : STAGE_BYTES;
};

__device__ __forceinline__ void grid_pos(uint32_t m, const GemmPhase& P, uint32_t& img, uint32_t& gi, uint32_t& gj) {
  img = fdiv(m, P.div_ghw);
  const uint32_t rem = m - img * (uint32_t)(P.gh * P.gw);
  gi = fdiv(rem, P.div_gw);
  gj = rem - gi * (uint32_t)P.gw;
}

template <int WM, int TM, int TN, int D>
__global__ __launch_bounds__(256) void convgemm_kernel(ConvGemmArgs a) {
  using S = GemmShape<WM, TM, TN>;
  constexpr int BM = S::BM, BN = S::BN, AV = S::AV, BV = S::BV, WTM = S::WTM, WTN = S::WTN;
  static_assert(BM % 64 == 0, "BM multiple of 64");
  static_assert(WM * S::WN == 4, "four waves");

  __shared__ __attribute__((aligned(16))) unsigned char smem[S::SMEM];
  __shared__ int32_t s_toff[kMaxTaps];
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[WM][BN];
  __shared__ float s_mean[BN];
  typedef bf16_t ATile[BM][GROW];
  typedef bf16_t BTile[BN][GROW];
  ATile* As = reinterpret_cast<ATile*>(smem);
  BTile* Bs = reinterpret_cast<BTile*>(smem + S::A_BYTES);
  float* stage = reinterpret_cast<float*>(smem);

  const GemmPhase& P = a.ph[blockIdx.z];
  const int m0 = blockIdx.x * BM;
  if (m0 >= P.m) return;  // this phase has fewer tiles; uniform exit before any barrier
  const int n0 = blockIdx.y * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int cv = tid & 3;   // 16-byte column of the 64-byte tile row
  const int rb = tid >> 2;  // first tile row of this thread

  if (tid < P.taps) {
    const int off = P.off[tid];
    const int dh = (int)(int16_t)(off & 0xffff), dw = off >> 16;
    s_toff[tid] = (dh * a.ws + dw) * (int)a.src_pix;
  }
  for (int r = tid; r < BM; r += 256) {
    const int m = m0 + r;
    int64_t d = -1;
    if (m < P.m) {
      uint32_t img, gi, gj;
      grid_pos((uint32_t)m, P, img, gi, gj);
      d = (((int64_t)img * a.hd + (int)gi * a.dstep_h + P.doff_h) * a.wd + (int)gj * a.dstep_w + P.doff_w) *
          a.dst_pix;
    }
    s_dst[r] = d;
  }

  // A rows: source pixel pointer and the taps that stay inside the image
  const bf16_t* rowp[AV];
  uint32_t rmask[AV];
#pragma unroll
  for (int i = 0; i < AV; ++i) {
    const int m = m0 + rb + 64 * i;
    rowp[i] = a.src;
    rmask[i] = 0;
    if (m < P.m) {
      uint32_t img, gi, gj;
      grid_pos((uint32_t)m, P, img, gi, gj);
      const int ih0 = (int)gi * a.gstride_h, iw0 = (int)gj * a.gstride_w;
      rowp[i] = a.src + ((int64_t)img * a.hs * a.ws + (int64_t)ih0 * a.ws + iw0) * a.src_pix;
      uint32_t mk = 0;
      for (int t = 0; t < P.taps; ++t) {
        const int off = P.off[t];
        const int ih = ih0 + (int)(int16_t)(off & 0xffff), iw = iw0 + (off >> 16);
        if ((unsigned)ih < (unsigned)a.hs && (unsigned)iw < (unsigned)a.ws) mk |= 1u << t;
      }
      rmask[i] = mk;
    }
  }
  // B rows
  const bf16_t* bptr[BV];
  bool bok[BV];
#pragma unroll
  for (int j = 0; j < BV; ++j) {
    const int row = rb + 64 * j;
    const int o = n0 + row;
    bok[j] = row < BN && o < a.nout;
    bptr[j] = P.wt + (int64_t)(bok[j] ? o : 0) * P.ktot + cv * 8;
  }
  int tapA = (cv * 8) / a.cs;
  int cA = cv * 8 - tapA * a.cs;
  const int nk = (P.ktot + GK - 1) / GK;
  __syncthreads();

  static_assert(D >= 1 && D <= 4, "prefetch depth 1..4");
  // D register sets form a ring: the loads of step kt + D are in flight while step kt
  // computes, so D global round trips overlap instead of one per step.
  u32x4 ra[D][AV], rbv[D][BV];
  const bf16_t* zp = reinterpret_cast<const bf16_t*>(&kZero16);
  auto load_tiles = [&](int kt, u32x4 (&xa)[AV], u32x4 (&xb)[BV]) __attribute__((always_inline)) {
    const bool tok = tapA < P.taps;
    const int toff = s_toff[tok ? tapA : 0] + cA;
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const bool ok = tok && ((rmask[i] >> tapA) & 1u);
      xa[i] = *reinterpret_cast<const u32x4*>(ok ? rowp[i] + toff : zp);
    }
    cA += GK;
    if (a.cs >= GK) {
      if (cA >= a.cs) {
        cA -= a.cs;
        ++tapA;
      }
    } else {
      while (cA >= a.cs) {
        cA -= a.cs;
        ++tapA;
      }
    }
    const int kb = kt * GK + cv * 8;
#pragma unroll
    for (int j = 0; j < BV; ++j) {
      const bool ok = bok[j] && kb < P.ktot;
      xb[j] = *reinterpret_cast<const u32x4*>(ok ? bptr[j] + kt * GK : zp);
    }
  };
  auto store_tiles = [&](int buf, const u32x4 (&xa)[AV], const u32x4 (&xb)[BV]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < AV; ++i) *reinterpret_cast<u32x4*>(&As[buf][rb + 64 * i][cv * 8]) = xa[i];
#pragma unroll
    for (int j = 0; j < BV; ++j)
      if (rb + 64 * j < BN) *reinterpret_cast<u32x4*>(&Bs[buf][rb + 64 * j][cv * 8]) = xb[j];
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int kc = (lane >> 4) * 8;
  const int arow = wm * WTM + (lane & 15), brow = wn * WTN + (lane & 15);
  auto compute = [&](int buf) __attribute__((always_inline)) {
    u32x4 af[TM], bfr[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const u32x4*>(&As[buf][arow + i * 16][kc]);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[j] = *reinterpret_cast<const u32x4*>(&Bs[buf][brow + j * 16][kc]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
  };

  // One pipeline step with its ring slot fixed at compile time (u = kt mod D), so every
  // ring access is a register access.
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    constexpr int nxt = (u + 1) % D;  // slot holding step kt + 1
    store_tiles((kt + 1) & 1, ra[nxt], rbv[nxt]);
    load_tiles(kt + 1 + D, ra[nxt], rbv[nxt]);
    compute(kt & 1);
    __syncthreads();
  };
  auto prologue_load = [&](auto dc) __attribute__((always_inline)) {
    constexpr int d = decltype(dc)::value;
    load_tiles(d, ra[d], rbv[d]);
  };

  // prologue: steps 0 .. D-1 in flight, step 0 in LDS, step D in flight in slot 0.
  // Loads past the end of K read zeros, so they are issued unconditionally.
  if (nk > 0) {
    prologue_load(Ic<0>{});
    if constexpr (D > 1) prologue_load(Ic<1>{});
    if constexpr (D > 2) prologue_load(Ic<2>{});
    if constexpr (D > 3) prologue_load(Ic<3>{});
    store_tiles(0, ra[0], rbv[0]);
    load_tiles(D, ra[0], rbv[0]);
    __syncthreads();
  }
  for (int kb = 0; kb < nk; kb += D) {
    step(Ic<0>{}, kb);
    if constexpr (D > 1) {
      if (kb + 1 < nk) step(Ic<1 % D>{}, kb + 1);
    }
    if constexpr (D > 2) {
      if (kb + 2 < nk) step(Ic<2 % D>{}, kb + 2);
    }
    if constexpr (D > 3) {
      if (kb + 3 < nk) step(Ic<3 % D>{}, kb + 3);
    }
  }

  // ---- per-channel (mean, M2) of this tile's rows from the fp32 accumulators (phase 0)
  if (a.stats_part != nullptr && blockIdx.z == 0) {
    const int left = P.m - m0;
    const int count = left < BM ? left : BM;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i) s += (acc[i][j][0] + acc[i][j][1]) + (acc[i][j][2] + acc[i][j][3]);
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (lane < 16) s_red[wm][wn * WTN + j * 16 + lane] = s;
    }
    __syncthreads();
    if (tid < BN) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < WM; ++w) s += s_red[w][tid];
      s_mean[tid] = s / (float)count;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float mu = s_mean[wn * WTN + j * 16 + (lane & 15)];
      float q = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = wm * WTM + i * 16 + 4 * (lane >> 4) + e;
          const float d = acc[i][j][e] - mu;
          q += (row < count) ? d * d : 0.f;
        }
      q += __shfl_xor(q, 16);
      q += __shfl_xor(q, 32);
      if (lane < 16) s_red[wm][wn * WTN + j * 16 + lane] = q;
    }
    __syncthreads();
    if (tid < BN && n0 + tid < a.nout) {
      float q = 0.f;
#pragma unroll
      for (int w = 0; w < WM; ++w) q += s_red[w][tid];
      a.stats_part[(int64_t)blockIdx.x * a.nout + n0 + tid] = make_float2(s_mean[tid], q);
    }
  }

  // ---- output
  if ((a.nout & 7) == 0) {
    // stage 16 rows per wave in LDS as fp32, then write 16-byte vectors of 8 channels
    float* st = stage + wave * 16 * S::STAGE_LD;
    constexpr int VPR = WTN / 8;  // vectors per staged row
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      __syncthreads();
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) st[(4 * (lane >> 4) + e) * S::STAGE_LD + j * 16 + (lane & 15)] = acc[i][j][e];
      __syncthreads();
      for (int v = lane; v < 16 * VPR; v += 64) {
        const int r = v / VPR, c8 = v - r * VPR;
        const int col = n0 + wn * WTN + c8 * 8;
        const int64_t d = s_dst[wm * WTM + i * 16 + r];
        if (col < a.nout && d >= 0) {
          const float4 lo = *reinterpret_cast<const float4*>(&st[r * S::STAGE_LD + c8 * 8]);
          const float4 hi = *reinterpret_cast<const float4*>(&st[r * S::STAGE_LD + c8 * 8 + 4]);
          float f[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          uint4* p = reinterpret_cast<uint4*>(a.dst + d + col);
          if (a.accumulate) {
            float o[8];
            unpack8(*p, o);
#pragma unroll
            for (int e = 0; e < 8; ++e) f[e] += o[e];
          }
          *p = pack8(f);
        }
      }
    }
  } else {
    // channel counts that are not a multiple of 8: scalar stores straight from the accumulators
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t d = s_dst[wm * WTM + i * 16 + 4 * (lane >> 4) + e];
        if (d < 0) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = n0 + wn * WTN + j * 16 + (lane & 15);
          if (col < a.nout) {
            float v = acc[i][j][e];
            if (a.accumulate) v += bf2f(a.dst[d + col]);
            a.dst[d + col] = (bf16_t)f2bf(v);
          }
        }
      }
  }
}

struct GInst {
  int wm, tm, tn, d;  // waves along M, 16-row tiles per wave, 16-col tiles per wave, prefetch depth
};
constexpr GInst kG[] = {
    {4, 4, 8, 2},  // 0: 256 x 128
    {4, 4, 6, 3},  // 1: 256 x 96
    {4, 4, 5, 3},  // 2: 256 x 80
    {4, 4, 4, 4},  // 3: 256 x 64
    {4, 4, 3, 4},  // 4: 256 x 48
    {2, 4, 4, 4},  // 5: 128 x 128
    {2, 4, 3, 4},  // 6: 128 x 96
    {2, 4, 2, 4},  // 7: 128 x 64
    {4, 1, 1, 4},  // 8: 64 x 16
};

template <int I>
hipError_t launch_g(const ConvGemmArgs& a, hipStream_t s) {
  constexpr GInst c = kG[I];
  using Sh = GemmShape<c.wm, c.tm, c.tn>;
  int mmax = 0;
  for (int p = 0; p < a.nphase; ++p) mmax = a.ph[p].m > mmax ? a.ph[p].m : mmax;
  dim3 grid((unsigned)((mmax + Sh::BM - 1) / Sh::BM), (unsigned)((a.nout + Sh::BN - 1) / Sh::BN), (unsigned)a.nphase);
  hipLaunchKernelGGL((convgemm_kernel<c.wm, c.tm, c.tn, c.d>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

TileCfg convgemm_pick(int64_t m_max, int nout) {
  if (nout <= 16) return TileCfg{64, 16, 8};
  // narrowest padding waste on N among the 256-row tiles; ties go to the wider tile
  struct Opt {
    int id, bn;
  };
  const Opt wide[] = {{0, 128}, {1, 96}, {2, 80}, {3, 64}, {4, 48}};
  int best = 0;
  int64_t waste = INT64_MAX;
  for (int i = 0; i < 5; ++i) {
    const int64_t w = ((nout + wide[i].bn - 1) / wide[i].bn) * wide[i].bn - nout;
    if (w < waste) {
      waste = w;
      best = i;
    }
  }
  const int bn = wide[best].bn;
  const int64_t blocks256 = ((m_max + 255) / 256) * ((nout + bn - 1) / bn);
  // few tiles: 128-row tiles (2 x 2 waves) fill the 256 CUs better
  if (blocks256 < 512) {
    if (bn == 128) return TileCfg{128, 128, 5};
    if (bn == 96) return TileCfg{128, 96, 6};
    if (bn == 64) return TileCfg{128, 64, 7};
  }
  return TileCfg{256, bn, wide[best].id};
}

hipError_t convgemm_launch(const ConvGemmArgs& a, const TileCfg& t, hipStream_t s, int cls) {
  trace_begin(cls, s);
  hipError_t e;
  switch (t.id) {
    case 0: e = launch_g<0>(a, s); break;
    case 1: e = launch_g<1>(a, s); break;
    case 2: e = launch_g<2>(a, s); break;
    case 3: e = launch_g<3>(a, s); break;
    case 4: e = launch_g<4>(a, s); break;
    case 5: e = launch_g<5>(a, s); break;
    case 6: e = launch_g<6>(a, s); break;
    case 7: e = launch_g<7>(a, s); break;
    default: e = launch_g<8>(a, s); break;
  }
  trace_end(cls, s);
  return e;
}

}  // namespace numbat

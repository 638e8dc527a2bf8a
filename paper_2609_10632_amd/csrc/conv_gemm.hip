// Implicit-GEMM convolution on gfx950 MFMA, second generation (bf16 in, fp32 accumulate).
//
// Computes the GEMM family described with ConvGemmArgs: the forward convolution (one
// phase) and all stride phases of a data gradient (one launch, blockIdx.z = phase).
//
// Differences from the first kernel, all aimed at keeping the MFMA pipes fed:
//  * the gathered operand A bypasses LDS: each wave loads its own MFMA A fragments
//    (16 contiguous bytes per lane) from global memory into a register ring several
//    steps deep; only the weight tile B, shared by the four waves, goes through LDS;
//  * the gather address of an A fragment costs a bit test and a 64-bit add: every row
//    keeps a pointer to its source pixel and a bitmask of the taps that land inside the
//    image, and the per-tap pixel offsets sit in LDS; padding lanes read a zero constant,
//    so every step issues the same loads and waits are counted exactly;
//  * 32x32x16 MFMAs (the full-rate bf16 form on gfx950) on 256- or 128-row tiles
//    (4 waves) by up to 128 columns;
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

template <int TM, int TN>
struct GemmShape {
  static constexpr int WTM = TM * 32;          // rows per wave
  static constexpr int BM = 4 * WTM, BN = TN * 32;
  static constexpr int BV = (BN + 63) / 64;    // B vectors per thread per step
  static constexpr int B_BYTES = 2 * BN * GROW * 2;
  static constexpr int STAGE_LD = BN + 4;                   // fp32 per staged row
  static constexpr int STAGE_BYTES = 4 * 8 * STAGE_LD * 4;  // 8 rows per wave
  static constexpr int SMEM = B_BYTES > STAGE_BYTES ? B_BYTES : STAGE_BYTES;
};

__device__ __forceinline__ void grid_pos(uint32_t m, const GemmPhase& P, uint32_t& img, uint32_t& gi, uint32_t& gj) {
  img = fdiv(m, P.div_ghw);
  const uint32_t rem = m - img * (uint32_t)(P.gh * P.gw);
  gi = fdiv(rem, P.div_gw);
  gj = rem - gi * (uint32_t)P.gw;
}

// Shared epilogue: per-channel (mean, M2) partials of the tile's rows (phase 0, when
// requested) and the bf16 output, staged through LDS as fp32 and written as 16-byte
// vectors of 8 channels.  Accumulator register r of a lane sits on wave row
// 8*(r/4) + 4*(lane/32) + (r%4) of its 32-row block, column lane%32 of its 32-column block.
template <int TM, int TN>
__device__ __forceinline__ void gemm_epilogue(const ConvGemmArgs& a, const GemmPhase& P, f32x16 (&acc)[TM][TN],
                                              int m0, int n0, unsigned char* smem, const int64_t* s_dst,
                                              float (*s_red)[TN * 32], float* s_mean) {
  using S = GemmShape<TM, TN>;
  constexpr int BM = S::BM, BN = S::BN, WTM = S::WTM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  float* stage = reinterpret_cast<float*>(smem);
  __syncthreads();  // the main loop's last LDS reads are done before staging reuses LDS
  // ---- per-channel (mean, M2) of this tile's rows from the fp32 accumulators (phase 0)
  if (a.stats_part != nullptr && blockIdx.z == 0) {
    const int left = P.m - m0;
    const int count = left < BM ? left : BM;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[i][j][r];
      s += __shfl_xor(s, 32);
      if (lane < 32) s_red[wave][j * 32 + lane] = s;
    }
    __syncthreads();
    if (tid < BN) s_mean[tid] = ((s_red[0][tid] + s_red[1][tid]) + (s_red[2][tid] + s_red[3][tid])) / (float)count;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float mu = s_mean[j * 32 + l32];
      float q = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wave * WTM + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          const float d = acc[i][j][r] - mu;
          q += (row < count) ? d * d : 0.f;
        }
      q += __shfl_xor(q, 32);
      if (lane < 32) s_red[wave][j * 32 + lane] = q;
    }
    __syncthreads();
    if (tid < BN && n0 + tid < a.nout) {
      const float q = (s_red[0][tid] + s_red[1][tid]) + (s_red[2][tid] + s_red[3][tid]);
      a.stats_part[(int64_t)blockIdx.x * a.nout + n0 + tid] = make_float2(s_mean[tid], q);
    }
  }

  // ---- output
  if ((a.nout & 7) == 0) {
    // stage 8 rows per wave in LDS as fp32 (register group g = r/4 of every 32-row block),
    // then write 16-byte vectors of 8 channels
    float* st = stage + wave * 8 * S::STAGE_LD;
    constexpr int VPR = BN / 8;  // vectors per staged row
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        __syncthreads();
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) st[(4 * half + e) * S::STAGE_LD + j * 32 + l32] = acc[i][j][4 * g + e];
        __syncthreads();
        for (int v = lane; v < 8 * VPR; v += 64) {
          const int r = v / VPR, c8 = v - r * VPR;
          const int col = n0 + c8 * 8;
          const int64_t d = s_dst[wave * WTM + i * 32 + 8 * g + r];
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
      for (int r = 0; r < 16; ++r) {
        const int64_t d = s_dst[wave * WTM + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3)];
        if (d < 0) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = n0 + j * 32 + l32;
          if (col < a.nout) {
            float v = acc[i][j][r];
            if (a.accumulate) v += bf2f(a.dst[d + col]);
            a.dst[d + col] = (bf16_t)f2bf(v);
          }
        }
      }
  }
}

// Four waves split the tile's rows; each wave owns TM*32 rows and all BN columns and
// multiplies with 32x32x16 MFMAs.  A (the gathered operand) is never shared between
// waves, and an MFMA lane's A fragment -- 8 consecutive channels of one pixel at one
// tap -- is 16 contiguous bytes in NHWC, so every wave loads its A fragments straight
// from global memory into a register ring.  Only B (the weights, shared by the four
// waves) is staged through LDS.  One pipeline step covers GK = 32 reduction elements,
// i.e. two MFMA k-slices.
template <int TM, int TN, int D>
__global__ __launch_bounds__(256) void convgemm_kernel(ConvGemmArgs a) {
  using S = GemmShape<TM, TN>;
  constexpr int BM = S::BM, BN = S::BN, BV = S::BV, WTM = S::WTM;
  static_assert(D >= 1 && D <= 4, "prefetch depth 1..4");

  __shared__ __attribute__((aligned(16))) unsigned char smem[S::SMEM];
  __shared__ int32_t s_toff[kMaxTaps];
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[4][BN];
  __shared__ float s_mean[BN];
  typedef bf16_t BTile[BN][GROW];
  BTile* Bs = reinterpret_cast<BTile*>(smem);

  const GemmPhase& P = a.ph[blockIdx.z];
  const int m0 = blockIdx.x * BM;
  if (m0 >= P.m) return;  // this phase has fewer tiles; uniform exit before any barrier
  const int n0 = blockIdx.y * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;  // MFMA row / column, k group

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

  // A: this lane's rows (one per 32-row block of the wave) and the taps inside the image
  const bf16_t* rowp[TM];
  uint32_t rmask[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wave * WTM + i * 32 + l32;
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
  // B: cooperative rows of the weight tile
  const int cv = tid & 3, rb = tid >> 2;
  const bf16_t* bptr[BV];
  bool bok[BV];
#pragma unroll
  for (int j = 0; j < BV; ++j) {
    const int row = rb + 64 * j;
    const int o = n0 + row;
    bok[j] = row < BN && o < a.nout;
    bptr[j] = P.wt + (int64_t)(bok[j] ? o : 0) * P.ktot + cv * 8;
  }
  // reduction position of this lane's next A fragment: k = slice * 16 + half * 8
  int tapA = (half * 8) / a.cs;
  int cA = half * 8 - tapA * a.cs;
  const int nk = (P.ktot + GK - 1) / GK;
  __syncthreads();

  const bf16_t* zp = reinterpret_cast<const bf16_t*>(&kZero16);
  // ring slot: TM rows x 2 k-slices of A fragments, BV vectors of B
  u32x4 ra[D][2 * TM], rbv[D][BV];
  auto advance = [&]() __attribute__((always_inline)) {
    cA += 16;
    if (a.cs >= 16) {
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
  };
  auto load_a = [&](u32x4 (&xa)[2 * TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bool tok = tapA < P.taps;
      const int toff = s_toff[tok ? tapA : 0] + cA;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bool ok = tok && ((rmask[i] >> tapA) & 1u);
        xa[ks * TM + i] = *reinterpret_cast<const u32x4*>(ok ? rowp[i] + toff : zp);
      }
      advance();
    }
  };
  auto load_b = [&](int kt, u32x4 (&xb)[BV]) __attribute__((always_inline)) {
    const int kb = kt * GK + cv * 8;
#pragma unroll
    for (int j = 0; j < BV; ++j) {
      const bool ok = bok[j] && kb < P.ktot;
      xb[j] = *reinterpret_cast<const u32x4*>(ok ? bptr[j] + kt * GK : zp);
    }
  };
  auto store_b = [&](int buf, const u32x4 (&xb)[BV]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < BV; ++j)
      if (rb + 64 * j < BN) *reinterpret_cast<u32x4*>(&Bs[buf][rb + 64 * j][cv * 8]) = xb[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf, const u32x4 (&xa)[2 * TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      u32x4 bfr[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const u32x4*>(&Bs[buf][j * 32 + l32][ks * 16 + half * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(xa[ks * TM + i], bfr[j], acc[i][j]);
    }
  };

  // step kt (ring slot u = kt mod D): stage B(kt+1) in LDS, fetch B(kt+1+D), multiply
  // A(kt) with B(kt), then fetch A(kt+D) into the slot just consumed.
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    constexpr int nxt = (u + 1) % D;
    store_b((kt + 1) & 1, rbv[nxt]);
    load_b(kt + 1 + D, rbv[nxt]);
    compute(kt & 1, ra[u]);
    load_a(ra[u]);
    __syncthreads();
  };
  auto prologue = [&](auto dc) __attribute__((always_inline)) {
    constexpr int d = decltype(dc)::value;
    load_a(ra[d]);
    load_b(d, rbv[d]);
  };

  // Loads past the end of K read zeros, so every load is issued unconditionally.
  if (nk > 0) {
    prologue(Ic<0>{});
    if constexpr (D > 1) prologue(Ic<1>{});
    if constexpr (D > 2) prologue(Ic<2>{});
    if constexpr (D > 3) prologue(Ic<3>{});
    store_b(0, rbv[0]);
    load_b(D, rbv[0]);
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

  gemm_epilogue<TM, TN>(a, P, acc, m0, n0, smem, s_dst, s_red, s_mean);
}

// ---------------------------------------------------------------------------
// Fast path for source channel counts that are multiples of 16 (every layer of the
// detector except the 3-channel image).  A 16-wide k-slice then never straddles a tap,
// so the tap of each slice -- and its pixel offset -- is the same for the whole wave:
// tap tracking runs on the scalar unit and the per-tap offset comes from the kernel
// arguments, leaving one bit test and one 64-bit add per A fragment.  One pipeline
// step covers 64 reduction elements (four MFMA k-slices) per barrier.
constexpr int GK16 = 64;
constexpr int GROW16 = GK16 + 8;  // 144-byte LDS rows: 16 lanes reading 16 rows hit 16 distinct bank groups

template <int TM, int TN, int D>
__global__ __launch_bounds__(256) void convgemm16_kernel(ConvGemmArgs a) {
  using S = GemmShape<TM, TN>;
  constexpr int BM = S::BM, BN = S::BN, WTM = S::WTM;
  constexpr int BV = (BN * 8 + 255) / 256;  // 16-byte B chunks per thread per step (BN rows x 8 chunks)
  constexpr int B_BYTES16 = 2 * BN * GROW16 * 2;
  constexpr int SM = B_BYTES16 > S::STAGE_BYTES ? B_BYTES16 : S::STAGE_BYTES;
  static_assert(D >= 1 && D <= 4, "prefetch depth 1..4");

  __shared__ __attribute__((aligned(16))) unsigned char smem[SM];
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[4][BN];
  __shared__ float s_mean[BN];
  typedef bf16_t BTile[BN][GROW16];
  BTile* Bs = reinterpret_cast<BTile*>(smem);

  const GemmPhase& P = a.ph[blockIdx.z];
  const int m0 = blockIdx.x * BM;
  if (m0 >= P.m) return;  // this phase has fewer tiles; uniform exit before any barrier
  const int n0 = blockIdx.y * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

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
  const bf16_t* rowp[TM];
  uint32_t rmask[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wave * WTM + i * 32 + l32;
    rowp[i] = a.src;
    rmask[i] = 0;
    if (m < P.m) {
      uint32_t img, gi, gj;
      grid_pos((uint32_t)m, P, img, gi, gj);
      const int ih0 = (int)gi * a.gstride_h, iw0 = (int)gj * a.gstride_w;
      rowp[i] = a.src + ((int64_t)img * a.hs * a.ws + (int64_t)ih0 * a.ws + iw0) * a.src_pix + half * 8;
      uint32_t mk = 0;
      for (int t = 0; t < P.taps; ++t) {
        const int off = P.off[t];
        const int ih = ih0 + (int)(int16_t)(off & 0xffff), iw = iw0 + (off >> 16);
        if ((unsigned)ih < (unsigned)a.hs && (unsigned)iw < (unsigned)a.ws) mk |= 1u << t;
      }
      rmask[i] = mk;
    }
  }
  const bf16_t* bptr[BV];
  bool bok[BV];
  int brow[BV], bch[BV];
#pragma unroll
  for (int j = 0; j < BV; ++j) {
    const int v = tid + 256 * j;
    brow[j] = v >> 3;
    bch[j] = v & 7;
    const int o = n0 + brow[j];
    bok[j] = brow[j] < BN && o < a.nout;
    bptr[j] = P.wt + (int64_t)(bok[j] ? o : 0) * P.ktot + bch[j] * 8;
  }
  int tapS = 0, cS = 0;  // wave-uniform position of the next A k-slice
  const int nk = (P.ktot + GK16 - 1) / GK16;
  __syncthreads();

  const bf16_t* zp = reinterpret_cast<const bf16_t*>(&kZero16);
  u32x4 ra[D][4 * TM], rbv[D][BV];
  auto load_a = [&](u32x4 (&xa)[4 * TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bool tok = tapS < P.taps;
      int toff = cS;
      if (tok) {
        const int off = P.off[tapS];
        toff += ((int)(int16_t)(off & 0xffff) * a.ws + (off >> 16)) * (int)a.src_pix;
      }
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bool ok = tok && ((rmask[i] >> tapS) & 1u);
        xa[ks * TM + i] = *reinterpret_cast<const u32x4*>(ok ? rowp[i] + toff : zp);
      }
      cS += 16;
      if (cS == a.cs) {
        cS = 0;
        ++tapS;
      }
    }
  };
  auto load_b = [&](int kt, u32x4 (&xb)[BV]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < BV; ++j) {
      const bool ok = bok[j] && kt * GK16 + bch[j] * 8 < P.ktot;
      xb[j] = *reinterpret_cast<const u32x4*>(ok ? bptr[j] + kt * GK16 : zp);
    }
  };
  auto store_b = [&](int buf, const u32x4 (&xb)[BV]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < BV; ++j)
      if (brow[j] < BN) *reinterpret_cast<u32x4*>(&Bs[buf][brow[j]][bch[j] * 8]) = xb[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf, const u32x4 (&xa)[4 * TM]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      u32x4 bfr[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const u32x4*>(&Bs[buf][j * 32 + l32][ks * 16 + half * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(xa[ks * TM + i], bfr[j], acc[i][j]);
    }
  };
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    constexpr int nxt = (u + 1) % D;
    store_b((kt + 1) & 1, rbv[nxt]);
    load_b(kt + 1 + D, rbv[nxt]);
    compute(kt & 1, ra[u]);
    load_a(ra[u]);
    __syncthreads();
  };
  auto prologue = [&](auto dc) __attribute__((always_inline)) {
    constexpr int d = decltype(dc)::value;
    load_a(ra[d]);
    load_b(d, rbv[d]);
  };

  if (nk > 0) {
    prologue(Ic<0>{});
    if constexpr (D > 1) prologue(Ic<1>{});
    if constexpr (D > 2) prologue(Ic<2>{});
    if constexpr (D > 3) prologue(Ic<3>{});
    store_b(0, rbv[0]);
    load_b(D, rbv[0]);
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
  gemm_epilogue<TM, TN>(a, P, acc, m0, n0, smem, s_dst, s_red, s_mean);
}


struct GInst {
  int tm, tn, d;  // 32-row tiles per wave (4 waves along M), 32-col tiles, prefetch depth
};
constexpr GInst kG[] = {
    {2, 4, 2},  // 0: 256 x 128
    {2, 3, 3},  // 1: 256 x 96
    {2, 2, 4},  // 2: 256 x 64
    {2, 1, 4},  // 3: 256 x 32
    {1, 4, 3},  // 4: 128 x 128
    {1, 3, 4},  // 5: 128 x 96
    {1, 2, 4},  // 6: 128 x 64
    {1, 1, 4},  // 7: 128 x 32
};

// prefetch depth of the 64-deep fast path (its ring slots are twice as large)
constexpr int d16(const GInst& c) { return c.tm * c.tn >= 6 ? 2 : 3; }

template <int I>
hipError_t launch_g(const ConvGemmArgs& a, hipStream_t s) {
  constexpr GInst c = kG[I];
  using Sh = GemmShape<c.tm, c.tn>;
  int mmax = 0;
  for (int p = 0; p < a.nphase; ++p) mmax = a.ph[p].m > mmax ? a.ph[p].m : mmax;
  dim3 grid((unsigned)((mmax + Sh::BM - 1) / Sh::BM), (unsigned)((a.nout + Sh::BN - 1) / Sh::BN), (unsigned)a.nphase);
  if (a.cs % 16 == 0)
    hipLaunchKernelGGL((convgemm16_kernel<c.tm, c.tn, d16(c)>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((convgemm_kernel<c.tm, c.tn, c.d>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

TileCfg convgemm_pick(int64_t m_max, int nout) {
  // narrowest padding waste on N (32-column granularity); ties go to the wider tile
  const int bns[4] = {128, 96, 64, 32};
  int bn = 128;
  int64_t waste = INT64_MAX;
  for (int i = 0; i < 4; ++i) {
    const int64_t w = ((nout + bns[i] - 1) / bns[i]) * bns[i] - nout;
    if (w < waste) {
      waste = w;
      bn = bns[i];
    }
  }
  const int ntiles = (nout + bn - 1) / bn;
  const int64_t blocks256 = ((m_max + 255) / 256) * ntiles;
  // few tiles: 128-row tiles fill the 256 CUs better
  const bool small = blocks256 < 512;
  const int id = (small ? 4 : 0) + (bn == 128 ? 0 : bn == 96 ? 1 : bn == 64 ? 2 : 3);
  return TileCfg{small ? 128 : 256, bn, id};
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
    default: e = launch_g<7>(a, s); break;
  }
  trace_end(cls, s);
  return e;
}

}  // namespace numbat

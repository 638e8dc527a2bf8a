// Implicit-GEMM convolution on gfx950 MFMA (bf16 in, fp32 accumulate).
//
// Computes the GEMM family described with ConvGemmArgs: the forward convolution (one
// phase) and all stride phases of a data gradient (one launch, blockIdx.z = phase).
// Kernels:
//  * convdma_kernel, for source channel counts that are multiples of 16 and at least 32
//    (every layer of the detector but the image input): both operands reach LDS through
//    loads that write LDS directly, in 2 or 3 stages (up to 6 supported);
//  * convhalo_kernel, 3x3 stride-1 padding-1 forwards and data gradients: the input halo
//    of a tile is staged once per 32-channel chunk and all nine taps read out of it
//    (linear tiles, or two-dimensional tiles of one image), optionally with the previous
//    layer's BN + SiLU applied to the staged halo (the prologue form);
//  * convgemm_kernel, for any other channel count that is a multiple of 8 (and tiles
//    whose address span exceeds 31 bits): each wave loads its own MFMA A fragments (16
//    contiguous bytes per lane) from global memory into a register ring several steps
//    deep; only the weight tile B, shared by the four waves, goes through LDS;
//  * convstem_kernel, the RGB image layer's forward (3 channels, 3x3, stride 2): a patch's
//    input pixels staged once in LDS;
//  * convnarrow_kernel, forward only, for other inputs of fewer than 8 channels: the
//    reduction (tap, channel) is packed densely and gathered element by element.  Every row keeps a
//    pointer to its source pixel and a bitmask of the taps that land inside the image;
//    padding lanes read a zero constant, so every step issues the same loads and waits
//    are counted exactly.
// All use 32x32x16 MFMAs (the full-rate bf16 form on gfx950) with 4 waves split along M
// (an 8-wave direct-to-LDS variant takes 256-row tiles; the halo kernel's 128-row tiles
// run as two halves of four waves that split the reduction), and share one epilogue:
// optional per-tile batch-statistics partials, then fp32 results staged through LDS and
// written as 16-byte vectors of 8 channels (bf16, rounded once, after the optional
// accumulate, and the inference post-op where asked).
#include <cstdlib>
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

// f(Ic<I>{}), ..., f(Ic<N - 1>{})
template <int I, int N, typename F>
__device__ __forceinline__ void static_for_ic(F&& f) {
  if constexpr (I < N) {
    f(Ic<I>{});
    static_for_ic<I + 1, N>(f);
  }
}

template <int TM, int TN, int NW = 4>
struct GemmShape {
  static constexpr int WTM = TM * 32;          // rows per wave
  static constexpr int BM = NW * WTM, BN = TN * 32;
  static constexpr int BV = (BN + 63) / 64;    // B vectors per thread per step
  static constexpr int B_BYTES = 2 * BN * GROW * 2;
  static constexpr int STAGE_LD = BN + 4;                   // fp32 per staged row
  static constexpr int STAGE_BYTES = NW * 8 * STAGE_LD * 4;  // 8 rows per wave
  static constexpr int SMEM = B_BYTES > STAGE_BYTES ? B_BYTES : STAGE_BYTES;
};

__device__ __forceinline__ void grid_pos(uint32_t m, const GemmPhase& P, uint32_t& img, uint32_t& gi, uint32_t& gj) {
  img = fdiv(m, P.div_ghw);
  const uint32_t rem = m - img * (uint32_t)(P.gh * P.gw);
  gi = fdiv(rem, P.div_gw);
  gj = rem - gi * (uint32_t)P.gw;
}

// logical tile of this block.  With the XCD-aware order: n tile fastest, then m tile,
// then phase, so the blocks sharing rows of the gathered operand (and halo rows of
// neighbouring tiles) share an XCD; otherwise the launch order (m tile fastest).
struct TileId {
  int mt, nt, ph;
};
__device__ __forceinline__ TileId tile_id(bool remap) {
  if (!remap) return TileId{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
  const uint32_t gx = gridDim.x, gy = gridDim.y;  // m tiles, n tiles
  const uint32_t lg = xcd_remap(blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z), gx * gy * gridDim.z);
  return TileId{(int)((lg / gy) % gx), (int)(lg % gy), (int)(lg / (gx * gy))};
}

// The per-phase geometry a block needs, read from the kernel arguments once at entry
// (the phase is chosen by the block index, so every field access would otherwise be a
// dependent scalar load)
struct Geo {
  int m, gh, gw;
  FastDiv div_gw, div_ghw;
  int doff_h, doff_w;
  int tw, th, dh0, dw0, tsh, tsw;
};
__device__ __forceinline__ Geo load_geo(const GemmPhase& P) {
  Geo g;
  g.m = P.m;
  g.gh = P.gh;
  g.gw = P.gw;
  g.div_gw = P.div_gw;
  g.div_ghw = P.div_ghw;
  g.doff_h = P.doff_h;
  g.doff_w = P.doff_w;
  g.tw = P.tw;
  g.th = P.th;
  g.dh0 = P.dh0;
  g.dw0 = P.dw0;
  g.tsh = P.tsh;
  g.tsw = P.tsw;
  return g;
}
__device__ __forceinline__ void geo_pos(uint32_t m, const Geo& G, uint32_t& img, uint32_t& gi, uint32_t& gj) {
  img = fdiv(m, G.div_ghw);
  const uint32_t rem = m - img * (uint32_t)(G.gh * G.gw);
  gi = fdiv(rem, G.div_gw);
  gj = rem - gi * (uint32_t)G.gw;
}

// destination element offset of GEMM row m (-1 past the phase's rows)
__device__ __forceinline__ int64_t dst_offset(const ConvGemmArgs& a, const Geo& G, int m) {
  if (m >= G.m) return -1;
  uint32_t img, gi, gj;
  geo_pos((uint32_t)m, G, img, gi, gj);
  return (((int64_t)img * a.hd + (int)gi * a.dstep_h + G.doff_h) * a.wd + (int)gj * a.dstep_w + G.doff_w) *
         a.dst_pix;
}

// Byte offset (from the tile's gather base, without the halo) of GEMM row m's anchor
// pixel, and the bitmask of its taps that fall inside the image.  The taps form a grid
// (rows of tw taps with constant steps), so the mask is the outer product of the grid
// rows that stay inside the image height and the grid columns inside its width.
__device__ __forceinline__ void row_gather(const ConvGemmArgs& a, const Geo& G, int m, uint32_t img0,
                                           uint32_t& vrow, uint32_t& vmask) {
  vrow = 0;
  vmask = 0;
  if (m >= G.m) return;
  uint32_t img, gi, gj;
  geo_pos((uint32_t)m, G, img, gi, gj);
  const int ih0 = (int)gi * a.gstride_h, iw0 = (int)gj * a.gstride_w;
  vrow = (uint32_t)((((int64_t)(img - img0) * a.hs + ih0) * a.ws + iw0) * (a.src_pix * 2));
  // (kernel sides are at most 5: fixed-trip, branch-free loops)
  uint32_t cols = 0;
#pragma unroll
  for (int j = 0; j < 5; ++j) {
    const int iw = iw0 + G.dw0 + j * G.tsw;
    cols |= (j < G.tw && (unsigned)iw < (unsigned)a.ws ? 1u : 0u) << j;
  }
  uint32_t mk = 0;
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    const int ih = ih0 + G.dh0 + i * G.tsh;
    mk |= (i < G.th && (unsigned)ih < (unsigned)a.hs ? cols : 0u) << (i * G.tw);
  }
  vmask = mk;  // bits >= taps stay clear, so a walk past the last tap reads zeros
}

// Shared epilogue: per-channel (mean, M2) partials of the tile's rows (phase 0, when
// requested) and the bf16 output, staged through LDS as fp32 and written as 16-byte
// vectors of 8 channels.  Accumulator register r of a lane sits on wave row
// 8*(r/4) + 4*(lane/32) + (r%4) of its 32-row block, column lane%32 of its 32-column block.
// sum of the NW waves' partials of column c, in a fixed pairwise order
template <int NW>
__device__ __forceinline__ float wave_sum(const float* r, int ld, int c) {
  const float s4 = (r[c] + r[ld + c]) + (r[2 * ld + c] + r[3 * ld + c]);
  if constexpr (NW == 4) return s4;
  else return s4 + ((r[4 * ld + c] + r[5 * ld + c]) + (r[6 * ld + c] + r[7 * ld + c]));
}

// `active` false: a wave that holds no accumulators of its own (the second half of a
// block whose halves split the reduction) and only takes the block's barriers.
template <int TM, int TN, int NW = 4>
__device__ __forceinline__ void gemm_epilogue(const ConvGemmArgs& a, const GemmPhase& P, const TileId& T,
                                              f32x16 (&acc)[TM][TN], int m0, int n0, unsigned char* smem,
                                              const int64_t* s_dst, float (*s_red)[TN * 32], float* s_mean,
                                              bool active = true) {
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  using S = GemmShape<TM, TN, NW>;
  constexpr int BM = S::BM, BN = S::BN, WTM = S::WTM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  float* stage = reinterpret_cast<float*>(smem);
  __syncthreads();  // the main loop's last LDS reads are done before staging reuses LDS
  // ---- per-channel (mean, M2) of this tile's rows from the fp32 accumulators (phase 0)
  if (a.stats_part != nullptr && T.ph == 0) {
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
      if (lane < 32 && active) s_red[wave][j * 32 + lane] = s;
    }
    __syncthreads();
    if (tid < BN) s_mean[tid] = wave_sum<NW>(&s_red[0][0], BN, tid) / (float)count;
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
      if (lane < 32 && active) s_red[wave][j * 32 + lane] = q;
    }
    __syncthreads();
    if (tid < BN && n0 + tid < a.nout) {
      const float q = wave_sum<NW>(&s_red[0][0], BN, tid);
      a.stats_part[(int64_t)T.mt * a.nout + n0 + tid] = make_float2(s_mean[tid], q);
    }
  }

  // ---- inference epilogue constants: per column a scale and a shift (bias: 1, bias[n];
  // eval-mode BN: gamma rstd, beta - mean gamma rstd), in s_red rows 0 and 1 (the
  // statistics, which share that space, are never asked for with them)
  const int post = a.post;
  if (post != kPostNone) {
    __syncthreads();
    if (tid < BN) {
      const int col = n0 + tid;
      float sc = 1.f, sh = 0.f;
      if (col < a.nout) {
        if (post == kPostBias) {
          sh = a.post_bias[col];
        } else {
          sc = a.post_gamma[col] * (1.0f / sqrtf(a.post_var[col] + a.post_eps));
          sh = a.post_beta[col] - a.post_mean[col] * sc;
        }
      }
      s_red[0][tid] = sc;
      s_red[1][tid] = sh;
    }
    __syncthreads();
  }
  auto post_op = [&](float (&f)[8], int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float z = __builtin_fmaf(f[e], s_red[0][c0 + e], s_red[1][c0 + e]);
      f[e] = post == kPostBnSilu ? z * sigmoidf_fast(z) : z;
    }
  };

  // ---- output
  if (!active) return;  // (no block barrier follows)
  if ((a.nout & 7) == 0) {
    // stage 8 rows per wave in LDS as fp32 (register group g = r/4 of every 32-row block),
    // then write 16-byte vectors of 8 channels
    float* st = stage + wave * 8 * S::STAGE_LD;
    constexpr int VPR = BN / 8;  // vectors per staged row
    // (the staging rows are private to the wave, and one wave's LDS accesses complete in
    // issue order, so the rounds need no barrier)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) st[(4 * half + e) * S::STAGE_LD + j * 32 + l32] = acc[i][j][4 * g + e];
        __builtin_amdgcn_wave_barrier();
        for (int v = lane; v < 8 * VPR; v += 64) {
          const int r = v / VPR, c8 = v - r * VPR;
          const int col = n0 + c8 * 8;
          const int64_t d = s_dst[wave * WTM + i * 32 + 8 * g + r];
          if (col < a.nout && d >= 0) {
            const float4 lo = *reinterpret_cast<const float4*>(&st[r * S::STAGE_LD + c8 * 8]);
            const float4 hi = *reinterpret_cast<const float4*>(&st[r * S::STAGE_LD + c8 * 8 + 4]);
            float f[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            uint4* p = reinterpret_cast<uint4*>(a.dst + d + col);
            if (post != kPostNone) post_op(f, c8 * 8);
            if (a.accumulate) {
              float o[8];
              unpack8(*p, o);
#pragma unroll
              for (int e = 0; e < 8; ++e) f[e] += o[e];
            }
            // (non-temporal: the tile is written once and read by a later kernel; measured
            // 3-12% faster across the conv layers than a default store)
            const uint4 v = pack8(f);
            __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4*>(p));
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
            if (post != kPostNone) {
              v = __builtin_fmaf(v, s_red[0][j * 32 + l32], s_red[1][j * 32 + l32]);
              if (post == kPostBnSilu) v = v * sigmoidf_fast(v);
            }
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

  const TileId T = tile_id(a.remap != 0);
  const GemmPhase& P = a.ph[T.ph];
  const int m0 = T.mt * BM;
  if (m0 >= P.m) return;  // this phase has fewer tiles; uniform exit before any barrier
  const int n0 = T.nt * BN;
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

  gemm_epilogue<TM, TN>(a, P, T, acc, m0, n0, smem, s_dst, s_red, s_mean);
}

// ---------------------------------------------------------------------------
// Fast path for source channel counts that are multiples of 16 and at least 32 (every
// layer of the detector except the 3-channel image).
//
// Both operands are staged through LDS and the gathered operand is loaded coalesced: a
// thread always loads the same 16-byte chunk (8 channels) of the step's reduction
// elements, and the threads with the same row cover the row's contiguous bytes, so one
// wave instruction reads whole rows -- 8 or 16 of them.  (Gathering MFMA fragments
// straight from global memory reads 32 rows per instruction; the L1 path's cost grows
// with the rows, not the bytes, an instruction touches, and that design stalled on it.)
//
// Loads are raw buffer loads.  The gather base sits halo_px pixels before the first
// image of the tile, so every in-image address is a non-negative 32-bit offset: row
// offset (fixed for the whole reduction) + the thread's tap-and-channel offset.  A tap
// outside the image swaps the offset for one past the buffer's range, which the hardware
// answers with zeros; so does a weight row past nout or a reduction index past ktot.
// Each thread walks its own reduction position (tap, channel) with adds and selects:
// 16-multiple channel counts never split a chunk between taps, and with 32 or more
// channels a step of up to 64 elements crosses at most two tap boundaries.
constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every range below
constexpr int kRecords = 0x7ffffff0;    // buffer range (bytes); in-range offsets stay below kOob - 2^24

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  // raw buffer, stride 0, range kRecords; word 3 = 0x00020000 (32-bit data format, the
  // setting for linear loads on this architecture)
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, kRecords, 0x00020000);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS variant of the staged fast path.  The loads of both operands write LDS
// themselves (buffer_load ... lds: lane i of a wave instruction deposits its 16 bytes
// at the instruction's LDS base + 16*i), so a pipeline step costs no VGPR staging and no
// LDS store instructions, and the prefetch depth lives in LDS stages instead of a
// register ring.  A stage holds BK reduction elements (64 or 32) of every row, in
// unpadded rows of 2*BK bytes; a wave instruction fills 1 KiB of consecutive rows.
// Bank conflicts on the 16-byte fragment reads (16 lanes, 16 rows, one 256-byte bank
// window) are avoided by storing 16-byte chunk k of row r in slot k ^ ((r / W) % C),
// with W rows per bank window and C chunks per row: rows sharing a window differ in
// their byte offset, rows of different windows in their slot.  A load lane picks the
// chunk its fixed LDS slot needs, so the swizzle costs nothing per step.
//
// Stage s of each operand is its own LDS object, so the compiler can tell the stages
// apart when it counts the loads an LDS read must wait for; every step issues the same
// loads (past the end of K they read zeros), and a step begins with a wait for its own
// loads (the later stages stay in flight) and a barrier, after which the stage it frees
// is refilled before its multiply.
template <int TM, int TN, int S, int BK, int NW, bool BT>
struct DmaShape {
  using G = GemmShape<TM, TN, NW>;
  static constexpr int ROWB = 2 * BK;               // bytes per LDS row
  static constexpr int CPR = BK / 8;                // 16-byte chunks per row
  static constexpr int RPI = 1024 / ROWB;           // rows per wave load instruction
  static constexpr int WIN = 256 / ROWB;            // rows per 256-byte bank window
  static constexpr int AI = G::BM / RPI / NW;       // A load instructions per wave per step
  // B load instructions per step (all waves): BN rows of BK elements, or (transposed B)
  // BK rows of BN elements
  static constexpr int BI = BT ? BK * G::BN * 2 / 1024 : (G::BN + RPI - 1) / RPI;
  static constexpr int BI_MIN = BI / NW;                 // ... issued by every wave
  static constexpr int BI_MAX = (BI + NW - 1) / NW;      // ... issued by the first waves
  static constexpr int A_ELEMS = G::BM * BK, B_ELEMS = BI * 512;
  // stage 0 of A doubles as the epilogue's staging area
  static constexpr int A0_ELEMS = 2 * A_ELEMS >= G::STAGE_BYTES ? A_ELEMS : G::STAGE_BYTES / 2;
  // loads still in flight when a step's own are done (every wave issues at least
  // AI + BI_MIN loads per step; a wave that issues more waits a little longer)
  static constexpr int PENDING = (S - 2) * (AI + BI_MIN);
  static_assert(G::BM % (NW * RPI) == 0, "A rows per step split evenly over the waves");
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef unsigned v2u_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// Transposed B stage ([BK reduction rows][BN columns], rows of 2*BN bytes): 16-byte chunk
// c of row r sits in slot c ^ bt_swizzle(r).  A transposing read (ds_read_b64_tr_b16)
// of a 16-lane group covers 4 consecutive rows x 32 bytes; the swizzle puts those 4
// segments in distinct quarters of the 256-byte bank window (rows of 192 or 64 bytes
// already do).
template <int BN>
__device__ __forceinline__ int bt_swizzle(int r) {
  return (BN == 64 || BN == 192) ? 4 * ((r >> 1) & 1) : BN == 128 ? 4 * (r & 3) : 0;
}

template <int TM, int TN, int S, int BK, int NW, bool BT>
__global__ __launch_bounds__(NW * 64) void convdma_kernel(ConvGemmArgs a) {
  using G = GemmShape<TM, TN, NW>;
  using Sh = DmaShape<TM, TN, S, BK, NW, BT>;
  constexpr int BM = G::BM, BN = G::BN, WTM = G::WTM;
  constexpr int AI = Sh::AI, BI = Sh::BI, BI_MAX = Sh::BI_MAX, RPI = Sh::RPI, CPR = Sh::CPR, WIN = Sh::WIN;
  static_assert(S >= 2 && S <= 6, "2..6 LDS stages");
  static_assert(BK == 32 || BK == 64, "stage depth");
  static_assert(Sh::PENDING <= 63, "load counter range");
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");

  __shared__ __attribute__((aligned(16))) bf16_t sA0[Sh::A0_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sA1[Sh::A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sA2[Sh::A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sA3[Sh::A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sA4[S > 4 ? Sh::A_ELEMS : 8];
  __shared__ __attribute__((aligned(16))) bf16_t sA5[S > 5 ? Sh::A_ELEMS : 8];
  __shared__ __attribute__((aligned(16))) bf16_t sB0[Sh::B_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sB1[Sh::B_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sB2[Sh::B_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sB3[Sh::B_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sB4[S > 4 ? Sh::B_ELEMS : 8];
  __shared__ __attribute__((aligned(16))) bf16_t sB5[S > 5 ? Sh::B_ELEMS : 8];
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[NW][BN];
  __shared__ float s_mean[BN];
  auto stage_a = [&](auto sc) __attribute__((always_inline)) -> bf16_t* {
    constexpr int s = decltype(sc)::value;
    if constexpr (s == 0) return sA0;
    else if constexpr (s == 1) return sA1;
    else if constexpr (s == 2) return sA2;
    else if constexpr (s == 3) return sA3;
    else if constexpr (s == 4) return sA4;
    else return sA5;
  };
  auto stage_b = [&](auto sc) __attribute__((always_inline)) -> bf16_t* {
    constexpr int s = decltype(sc)::value;
    if constexpr (s == 0) return sB0;
    else if constexpr (s == 1) return sB1;
    else if constexpr (s == 2) return sB2;
    else if constexpr (s == 3) return sB3;
    else if constexpr (s == 4) return sB4;
    else return sB5;
  };

  // (launch order: the XCD-aware order measured no faster for these GEMMs; a constant
  // keeps the block's first loads from waiting on a kernel argument)
  const TileId T = tile_id(false);
  const GemmPhase& P = a.ph[T.ph];
  const Geo Ge = load_geo(P);
  {
    // every kernel argument the prologue needs, loaded at once and completed before the
    // early-exit test (otherwise the compiler splits them into dependent rounds after it)
    const bf16_t* src = a.src;
    const bf16_t* wt = P.wt;
    const int64_t spx = a.src_pix;
    const int hs = a.hs, ws = a.ws, cs = a.cs, nout = a.nout, halo = a.halo_px, gsh = a.gstride_h,
              gsw = a.gstride_w, kt = P.ktot, tw = P.tw, t0 = P.toff0, cst = P.cstep, rst = P.rstep;
    asm volatile("" ::"s"(src), "s"(wt), "s"(spx), "s"(hs), "s"(ws), "s"(cs), "s"(nout), "s"(halo), "s"(gsh),
                 "s"(gsw), "s"(kt), "s"(tw), "s"(t0), "s"(cst), "s"(rst), "s"(Ge.m), "s"(Ge.gh), "s"(Ge.gw),
                 "s"(Ge.th), "s"(Ge.dh0), "s"(Ge.dw0), "s"(Ge.tsh), "s"(Ge.tsw), "s"(Ge.div_gw.mul),
                 "s"(Ge.div_gw.shift), "s"(Ge.div_ghw.mul), "s"(Ge.div_ghw.shift));
  }
  const int m0 = T.mt * BM;
  if (m0 >= Ge.m) return;  // this phase has fewer tiles; uniform exit before any barrier
  const int n0 = T.nt * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  // Load instruction q of this wave fills rows (NW*q + wave)*RPI .. +RPI; the lane's LDS
  // slot is lane % CPR of row lane / CPR in it, which holds chunk slot ^ ((row / WIN) % CPR)
  // (the same for every q)
  const int lrow = lane / CPR;
  const int kc = (lane % CPR) ^ (((wave * RPI + lrow) / WIN) % CPR);

  const uint32_t img0 = fdiv((uint32_t)m0, Ge.div_ghw);
  const __amdgpu_buffer_rsrc_t rsA =
      buffer_rsrc(a.src + ((int64_t)img0 * a.hs * a.ws - a.halo_px) * a.src_pix);
  uint32_t vrow[AI], vmask[AI];  // the rows this thread loads
#pragma unroll
  for (int q = 0; q < AI; ++q) row_gather(a, Ge, m0 + (NW * q + wave) * RPI + lrow, img0, vrow[q], vmask[q]);
  const __amdgpu_buffer_rsrc_t rsB = buffer_rsrc(P.wt);
  const int p_tw = P.tw, p_ktot = P.ktot, p_taps = P.taps, cs = a.cs;
  const uint32_t p_cstep = (uint32_t)P.cstep, p_rstep = (uint32_t)P.rstep;
  uint32_t voffb[BI_MAX];
  // transposed B (OHWI weights read in place): instruction j of this lane covers stage row
  // brw[j] (reduction index kb + brw[j] = (tap, o)), 16-byte column chunk bch[j]; the
  // walk keeps o, the tap's grid column and the byte offset of (o, tap) per instruction
  int bo[BT ? BI_MAX : 1], btap[BT ? BI_MAX : 1], btc[BT ? BI_MAX : 1];
  const uint32_t w_ostep = (uint32_t)P.wostep, w_cstep = (uint32_t)P.wcstep, w_rstep = (uint32_t)P.wrstep;
  if constexpr (!BT) {
#pragma unroll
    for (int j = 0; j < BI_MAX; ++j) {
      const int row = (NW * j + wave) * RPI + lrow, o = n0 + row;
      voffb[j] = (row < BN && o < a.nout) ? (uint32_t)(((int64_t)o * p_ktot + kc * 8) * 2) : kOob;
    }
  } else {
#pragma unroll
    for (int j = 0; j < BI_MAX; ++j) {
      const int byte = (NW * j + wave) * 1024 + lane * 16;
      const int row = byte / (2 * BN), slot = (byte % (2 * BN)) / 16;
      const int chunk = slot ^ bt_swizzle<BN>(row);
      const bool colok = n0 + chunk * 8 < a.nout;
      // reduction index row = tap * cs + o (row < BK <= 2 * cs: at most two wraps)
      int o = row, tp = 0, tc = 0;
      uint32_t off = (uint32_t)P.wtoff0 + (uint32_t)((n0 + chunk * 8) * 2);
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const bool wrap = o >= cs;
        o = wrap ? o - cs : o;
        tp += wrap ? 1 : 0;
        tc += wrap ? 1 : 0;
        const bool rw = tc == p_tw;
        tc = rw ? 0 : tc;
        off += wrap ? (rw ? w_rstep : w_cstep) : 0u;
      }
      bo[j] = o;
      btap[j] = colok ? tp : 31;  // a chunk past nout never loads
      btc[j] = tc;
      voffb[j] = off;
    }
  }
  int ch = kc * 8, tap = 0, tcol = 0;
  uint32_t toff = (uint32_t)P.toff0;
  auto wrap_taps = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      const bool wrap = ch >= cs;
      ch = wrap ? ch - cs : ch;
      tap += wrap ? 1 : 0;
      tcol += wrap ? 1 : 0;
      const bool rw = tcol == p_tw;
      tcol = rw ? 0 : tcol;
      toff += wrap ? (rw ? p_rstep : p_cstep) : 0u;
    }
  };
  wrap_taps();
  const int nk = (p_ktot + BK - 1) / BK;

  // issue the loads of step kt into stage s; the A walk advances by one step
  auto issue = [&](auto sc, int kt) __attribute__((always_inline)) {
    bf16_t* A = stage_a(sc);
    bf16_t* B = stage_b(sc);
    const uint32_t lo = toff + 2u * (uint32_t)ch;
    const int tq = tap < 31 ? tap : 31;  // past the last tap: bit 31 is clear
#pragma unroll
    for (int q = 0; q < AI; ++q) {
      const uint32_t t = (uint32_t)__builtin_amdgcn_sbfe((int)vmask[q], tq, 1);
      const uint32_t vo = (t & (vrow[q] + lo)) | (~t & kOob);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (lds_void_t*)(A + (NW * q + wave) * RPI * BK), 16, vo, 0, 0, 0);
    }
    if constexpr (!BT) {
      const int kb = kt * BK;
      const bool kin = kb + kc * 8 < p_ktot;
#pragma unroll
      for (int j = 0; j < BI_MAX; ++j) {
        if (NW * j + wave < BI) {  // wave-uniform
          // (the select stays out of the builtin's argument list: written inline, the host
          // pass drops the kernel's launch stub)
          const uint32_t vb = kin ? voffb[j] : kOob;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, (lds_void_t*)(B + (NW * j + wave) * 512), 16, vb,
                                                   (uint32_t)kb * 2, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < BI_MAX; ++j) {
        if (NW * j + wave < BI) {  // wave-uniform
          const uint32_t vb = btap[j] < p_taps ? voffb[j] + (uint32_t)bo[j] * w_ostep : kOob;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, (lds_void_t*)(B + (NW * j + wave) * 512), 16, vb, 0, 0, 0);
          // next step: o advances by BK, wrapping into later taps
          int o = bo[j] + BK, tp = btap[j], tc = btc[j];
          uint32_t off = voffb[j];
#pragma unroll
          for (int w = 0; w < 2; ++w) {
            const bool wrap = o >= cs;
            o = wrap ? o - cs : o;
            tp += wrap ? 1 : 0;
            tc += wrap ? 1 : 0;
            const bool rw = tc == p_tw;
            tc = rw ? 0 : tc;
            off += wrap ? (rw ? w_rstep : w_cstep) : 0u;
          }
          bo[j] = o;
          btap[j] = tp;
          btc[j] = tc;
          voffb[j] = off;
        }
      }
    }
    ch += BK;
    wrap_taps();
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // fragment byte offsets: row (wave rows + l32) of A, l32 of B; k-slice ks sits in chunk
  // 2*ks + half, stored in slot (2*ks + half) ^ ((l32 / WIN) % CPR)
  const int sw = (l32 / WIN) % CPR;
  const uint32_t arow = (uint32_t)(wave * WTM + l32) * (BK * 2), brow = (uint32_t)l32 * (BK * 2);
  uint32_t koff[BK / 16];
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) koff[ks] = (uint32_t)(((2 * ks + half) ^ sw) * 16);
  // transposed B: lane l = 16 g + 4 e + q reads 4 columns (8 bytes) of rows 8 (g / 2) + e
  // and that + 4 of the 16-row slice, columns 32 j + 16 (g % 2) + 4 q ..; the read hands
  // each lane 4 consecutive rows of one column, two reads make its fragment
  uint32_t btoff[BT ? TN : 1];
  if constexpr (BT) {
    const int g = lane >> 4, e = (lane & 15) >> 2, q = lane & 3;
    const int r0 = 8 * (g >> 1) + e;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int c = 4 * j + 2 * (g & 1) + (q >> 1);
      btoff[j] = (uint32_t)(r0 * 2 * BN + (c ^ bt_swizzle<BN>(r0)) * 16 + (q & 1) * 8);
    }
  }
  auto compute = [&](auto sc) __attribute__((always_inline)) {
    const unsigned char* A = reinterpret_cast<const unsigned char*>(stage_a(sc));
    const unsigned char* B = reinterpret_cast<const unsigned char*>(stage_b(sc));
    u32x4 af[2][TM], bf[2][TN];
    auto rd = [&](int ks, u32x4 (&xa)[TM], u32x4 (&xb)[TN]) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < TM; ++i) xa[i] = *reinterpret_cast<const u32x4*>(A + arow + i * 32 * BK * 2 + koff[ks]);
      if constexpr (!BT) {
#pragma unroll
        for (int j = 0; j < TN; ++j) xb[j] = *reinterpret_cast<const u32x4*>(B + brow + j * 32 * BK * 2 + koff[ks]);
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const unsigned char* pb = B + btoff[j] + ks * 16 * 2 * BN;
          const v4s_t r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)pb);
          const v4s_t r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(pb + 4 * 2 * BN));
          const v2u_t lo = __builtin_bit_cast(v2u_t, r0), hi = __builtin_bit_cast(v2u_t, r1);
          xb[j][0] = lo.x;
          xb[j][1] = lo.y;
          xb[j][2] = hi.x;
          xb[j][3] = hi.y;
        }
      }
    };
    rd(0, af[0], bf[0]);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      if (ks + 1 < BK / 16) rd(ks + 1, af[(ks + 1) & 1], bf[(ks + 1) & 1]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(af[ks & 1][i], bf[ks & 1][j], acc[i][j]);
    }
  };
  // this wave's loads of the current step are done (the later stages' stay in flight),
  // then every wave's: the stage is complete in LDS and the stage read last step is free
  auto sync = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(Sh::PENDING) : "memory");
  };
  // step kt reads stage u = kt mod S and refills stage (kt - 1) mod S with step kt + S - 1
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    sync();
    issue(Ic<(u + S - 1) % S>{}, kt + S - 1);
    compute(uc);
  };
  if (nk > 0) static_for_ic<0, S - 1>([&](auto ic) { issue(ic, decltype(ic)::value); });
  // destination offsets of the tile's rows, needed only by the epilogue: computed while
  // the first stages load (the first step's barrier publishes them)
  for (int r = tid; r < BM; r += NW * 64) s_dst[r] = dst_offset(a, Ge, m0 + r);
  int kb = 0;
  for (; kb + S <= nk; kb += S) static_for_ic<0, S>([&](auto ic) { step(ic, kb + decltype(ic)::value); });
  static_for_ic<0, S - 1>([&](auto ic) {
    if (kb + decltype(ic)::value < nk) step(ic, kb + decltype(ic)::value);
  });
  // the loads issued past the last step land in LDS before stage 0 becomes staging space
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  gemm_epilogue<TM, TN, NW>(a, P, T, acc, m0, n0, reinterpret_cast<unsigned char*>(sA0), s_dst, s_red, s_mean);
}

// ---------------------------------------------------------------------------
// Forward convolution of a narrow input (fewer than 8 channels: the RGB image).  The
// reduction k = (tap, channel) is packed densely (K = taps * ci, e.g. 27, padded to a
// multiple of 16), so an MFMA A fragment -- 8 consecutive k of one output pixel -- is
// gathered element by element: a per-k table in LDS holds each k's offset from the
// pixel's anchor and its tap, and a tap outside the image reads a zero.  The weights
// (OHWI is already [o][k]) sit in LDS for the whole block.  One pass over K, then the
// shared epilogue (statistics partials, 16-byte output vectors).
template <int TM, int TN>
struct NarrowShape {
  using G = GemmShape<TM, TN>;
  static constexpr int KMAX = ((kMaxTaps * 7 + 15) / 16) * 16;  // 176
  static constexpr int BROW = KMAX + 8;                           // bf16 per weight row (odd multiple of 16 bytes)
  static constexpr int B_BYTES = G::BN * BROW * 2;
  static constexpr int SM = B_BYTES > G::STAGE_BYTES ? B_BYTES : G::STAGE_BYTES;
};

template <int TM, int TN>
__global__ __launch_bounds__(256) void convnarrow_kernel(ConvGemmArgs a) {
  using G = GemmShape<TM, TN>;
  using Sh = NarrowShape<TM, TN>;
  constexpr int BM = G::BM, BN = G::BN, WTM = G::WTM, BROW = Sh::BROW;
  __shared__ __attribute__((aligned(16))) unsigned char smem[Sh::SM];
  __shared__ int32_t s_koff[Sh::KMAX];  // element offset of k from the pixel's anchor
  __shared__ int32_t s_ktap[Sh::KMAX];  // tap of k (31 past K: bit 31 of a tap mask is clear)
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[4][BN];
  __shared__ float s_mean[BN];
  bf16_t* Bs = reinterpret_cast<bf16_t*>(smem);

  const TileId T{(int)blockIdx.x, (int)blockIdx.y, 0};
  const GemmPhase& P = a.ph[0];
  const int m0 = T.mt * BM, n0 = T.nt * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int ktot = P.ktot, nks = (ktot + 15) / 16, kp = nks * 16;

  for (int k = tid; k < kp; k += 256) {
    int off = 0, tap = 31;
    if (k < ktot) {
      tap = k / a.cs;
      const int c = k - tap * a.cs;
      const int o = P.off[tap];
      off = (int)(((int16_t)(o & 0xffff) * a.ws + (o >> 16)) * a.src_pix) + c;
    }
    s_koff[k] = off;
    s_ktap[k] = tap;
  }
  for (int e = tid; e < BN * kp; e += 256) {
    const int r = e / kp, k = e - r * kp, o = n0 + r;
    Bs[r * BROW + k] = (o < a.nout && k < ktot) ? P.wt[(int64_t)o * ktot + k] : (bf16_t)0;
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
  // this lane's rows: anchor element (the tap (0, 0) pixel before padding) and the taps
  // inside the image
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
  __syncthreads();

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  const bf16_t* zp = reinterpret_cast<const bf16_t*>(&kZero16);
  for (int ks = 0; ks < nks; ++ks) {
    const int kb = ks * 16 + half * 8;
    int koff[8];
    uint32_t ktap[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      koff[e] = s_koff[kb + e];
      ktap[e] = (uint32_t)s_ktap[kb + e];
    }
    u32x4 af[TM], bf[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      uint32_t h[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = (rmask[i] >> ktap[e]) & 1u;
        h[e] = (uint32_t)*(ok ? rowp[i] + koff[e] : zp);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) af[i][q] = h[2 * q] | (h[2 * q + 1] << 16);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) bf[j] = *reinterpret_cast<const u32x4*>(&Bs[(j * 32 + l32) * BROW + kb]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
  }
  gemm_epilogue<TM, TN>(a, P, T, acc, m0, n0, smem, s_dst, s_red, s_mean);
}

// ---------------------------------------------------------------------------
// Forward convolution of the RGB image layer (3 channels, 3x3, stride 2, padding 1;
// output rows a multiple of 4 and columns of 64): a block computes a 4 x 64 patch of
// output pixels.  The 9 x 129 input pixels it reads are loaded once into LDS, each
// padded to 4 channels (8 bytes, the fourth zero), and the reduction is ordered as
// k = 16 r + 4 s + c (tap row r, tap column s, channel c; zero weights at c = 3 and
// past s = 2), so the 8 consecutive k of an MFMA fragment are 16 aligned bytes of one
// input row (s = 0, 1), or 8 bytes (s = 2) and four zeros.  Wave w owns output row w of
// the patch.  The weights, as [o][k], stay in LDS; then the shared epilogue.
constexpr int kStemCols = 129, kStemPitch = 130;  // input pixels per patch row, LDS pitch (pixels)
constexpr int kStemKp = 56;                       // bf16 per weight row (48 + 8)

__global__ __launch_bounds__(256) void convstem_kernel(ConvGemmArgs a) {
  using G = GemmShape<2, 2>;
  constexpr int BN = G::BN;
  constexpr int PATCH = 9 * kStemPitch * 8;  // bytes
  constexpr int SM = PATCH > G::STAGE_BYTES ? PATCH : G::STAGE_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SM];
  __shared__ __attribute__((aligned(16))) bf16_t s_w[BN * kStemKp];
  __shared__ int64_t s_dst[256];
  __shared__ float s_red[4][BN];
  __shared__ float s_mean[BN];
  const GemmPhase& P = a.ph[0];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  // tile: blockIdx.x = patch column, blockIdx.y = patch row, blockIdx.z = image
  const int oj0 = blockIdx.x * 64, oi0 = blockIdx.y * 4, img = blockIdx.z;
  const int ntc = P.gw >> 6, ntr = P.gh >> 2;
  const TileId T{(int)((img * ntr + blockIdx.y) * ntc + blockIdx.x), 0, 0};
  const int m0 = T.mt * 256;

  // input patch: rows 2 oi0 - 1 + pr, columns 2 oj0 - 1 + pc; all loads first
  constexpr int kPix = 9 * kStemCols, kRounds = (kPix + 255) / 256;
  uint32_t lo[kRounds], hi[kRounds];
#pragma unroll
  for (int u = 0; u < kRounds; ++u) {
    const int e = tid + 256 * u;
    const int pr = e / kStemCols, pc = e - pr * kStemCols;
    const int ih = 2 * oi0 - 1 + pr, iw = 2 * oj0 - 1 + pc;
    lo[u] = hi[u] = 0u;
    if (e < kPix && (unsigned)ih < (unsigned)a.hs && (unsigned)iw < (unsigned)a.ws) {
      const bf16_t* px = a.src + (((int64_t)img * a.hs + ih) * a.ws + iw) * a.src_pix;
      lo[u] = (uint32_t)px[0] | ((uint32_t)px[1] << 16);
      hi[u] = (uint32_t)px[2];
    }
  }
  // weights [o][k = 16 r + 4 s + c] from OHWI [o][r][s][c]: zeros first, then the
  // tensor read contiguously (2-byte elements, loads issued before the stores)
  for (int e = tid; e < BN * kStemKp / 2; e += 256) reinterpret_cast<uint32_t*>(s_w)[e] = 0u;
  constexpr int kWRounds = 64 * 27 / 256 + 1;
  bf16_t wv[kWRounds];
  const int nwt = a.nout * 27;
#pragma unroll
  for (int u = 0; u < kWRounds; ++u) {
    const int e = tid + 256 * u;
    wv[u] = e < nwt ? P.wt[e] : (bf16_t)0;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kWRounds; ++u) {
    const int e = tid + 256 * u;
    if (e < nwt) {
      const int o = e / 27, k = e - o * 27;
      const int r = k / 9, sc = k - r * 9, s = sc / 3, c = sc - s * 3;
      s_w[o * kStemKp + r * 16 + s * 4 + c] = wv[u];
    }
  }
  for (int r = tid; r < 256; r += 256) {
    const int oi = oi0 + (r >> 6), oj = oj0 + (r & 63);
    s_dst[r] = (((int64_t)img * a.hd + oi) * a.wd + oj) * a.dst_pix;
  }
#pragma unroll
  for (int u = 0; u < kRounds; ++u) {
    const int e = tid + 256 * u;
    if (e < kPix) {
      const int pr = e / kStemCols, pc = e - pr * kStemCols;
      *reinterpret_cast<uint2*>(smem + (pr * kStemPitch + pc) * 8) = make_uint2(lo[u], hi[u]);
    }
  }
  __syncthreads();

  // A fragment of output pixel (row wave, column 32 i + l32), tap row ks: input patch row
  // 2 wave + ks, columns 2 oj + half * 2 (16 bytes: s = 0, 1) or + 2 (8 bytes: s = 2)
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
#pragma unroll
  for (int ks = 0; ks < 3; ++ks) {
    u32x4 af[2], bf[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const unsigned char* px = smem + ((2 * wave + ks) * kStemPitch + 2 * (32 * i + l32)) * 8;
      if (half == 0) {
        af[i] = *reinterpret_cast<const u32x4*>(px);
      } else {
        const uint2 v = *reinterpret_cast<const uint2*>(px + 16);
        af[i] = u32x4{v.x, v.y, 0u, 0u};
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) bf[j] = *reinterpret_cast<const u32x4*>(&s_w[(j * 32 + l32) * kStemKp + ks * 16 + half * 8]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
  }
  gemm_epilogue<2, 2>(a, P, T, acc, m0, 0, smem, s_dst, s_red, s_mean);
}

// ---------------------------------------------------------------------------
// 3x3, stride-1, padding-1 convolutions (the forward and, with the weights read in place
// and flipped, the data gradient): the input halo of a tile is staged in LDS once per
// 32-channel chunk and all nine taps are read out of it.  A tile is BM consecutive output
// pixels (linear over image, row, column); the source pixels its taps reach are the
// contiguous linear range [m0 - W - 1, m0 + BM + W + 1), because tap (r, s) of output
// pixel m reads source pixel m + (r - 1) W + (s - 1) whenever that pixel is inside the
// image (taps that leave the image read zeros instead: each lane keeps the LDS address of
// every tap of its rows, pointing at a zero row for the taps outside the image).  Per
// chunk the tile loads about BM + 2W pixels instead of 9 BM, so the loads are mostly the
// weights.
//
// Pipeline: one step is KT taps (1, or a whole tap row of 3) of one chunk, 32 reduction
// elements per tap: the weights of those taps (BN rows of 64 bytes per tap, or for the
// data gradient 32 rows of BN columns read with transposing LDS reads) in one of SB
// stages (prefetch distance SB - 1 steps), and the chunk's halo, two deep: the next
// chunk's halo is issued at the first step of the current one.  The waits are exact: at
// step s the loads issued after the weights of s are the later steps' weights, plus the
// next halo on the steps right after a chunk's first.  Every step issues the same loads;
// past the end of K they read zeros.  Halo buffers and weight stages are distinct LDS
// objects selected at compile time (two chunks per loop trip), so the compiler can tell an
// in-flight load's target from the buffer being read.
template <int TM, int TN, int HI, int KT, int SB, bool BT, int TC>
struct HaloShape {
  using G = GemmShape<TM, TN, 4>;
  static constexpr int NW = 4;
  static constexpr int SPC = 9 / KT;                   // steps per chunk
  static constexpr int HPAD = HI * NW * 16;            // halo pixels per buffer (16 per load instruction)
  static constexpr int HBYTES = (HPAD + 1) * 64;       // + one zero row read by out-of-image taps
  static constexpr int H0BYTES = HBYTES >= G::STAGE_BYTES ? HBYTES : G::STAGE_BYTES;  // buffer 0 stages the epilogue
  static constexpr int TBYTES = G::BN * 64;            // the weights of one tap: BN x 32 elements
  static constexpr int BI = KT * G::BN / 16;           // weight load instructions per step (all waves)
  static constexpr int BI_MIN = BI / NW, BI_MAX = (BI + NW - 1) / NW;
  static_assert(KT == 1 || KT == 3, "one tap or one tap row per step");
  static_assert((2 * SPC) % SB == 0, "stage of a step known at compile time over two chunks");
  static_assert(SB >= 2 && SB - 1 <= SPC, "prefetch within one chunk");
  // two-dimensional tiles (TC > 0): TR x TC output pixels of one image, whose padded halo of
  // (TR + 2) x (TC + 2) pixels fits the buffer
  static constexpr int TR = TC > 0 ? G::BM / TC : 0;
  static_assert(TC == 0 || (G::BM % TC == 0 && (TR + 2) * (TC + 2) <= HPAD), "2D tile and its halo");
  // waves of the plain kernel: 128-row tiles take two reduction halves of four waves (the
  // first halo buffer holds their exchange), 256-row tiles four waves
  static constexpr int KV = (TM == 1 && H0BYTES >= 4 * 64 * 64) ? 2 : 1;
};

// KV = 2: eight waves in two halves of four; half 0 issues every load, half k multiplies
// reduction slice k (16 channels) of every tap, and the halves add their sums through LDS
// before the epilogue (twice the waves per SIMD to cover a step's latencies, same LDS).
//
// PRO (kProFwd, kProBwd): an element-wise prologue on each 32-channel chunk of the staged
// halo, once per element, before any tap reads it; its per-channel constants sit in dynamic
// LDS (2 or 4 floats per source channel, sized at launch), and the loading lanes transform
// their own chunks between their load wait and the barrier.  kProBwd (the data gradient,
// four waves): the halo holds g, each lane also loads y for its own halo chunks (into
// registers, a chunk ahead), and dy = BN + SiLU backward (g, y) replaces g in place; dy of
// the tile's own pixels is also stored (first column tile only).
template <int TM, int TN, int HI, int KT, int SB, bool BT, int TC, int PRO, int KV>
__global__ __launch_bounds__(256 * KV) void convhalo_kernel(ConvGemmArgs a) {
  using G = GemmShape<TM, TN, 4>;
  using Sh = HaloShape<TM, TN, HI, KT, SB, BT, TC>;
  constexpr int TR = Sh::TR;
  constexpr int BM = G::BM, BN = G::BN, WTM = G::WTM, NW = 4, SPC = Sh::SPC, D = SB - 1;
  constexpr int BI = Sh::BI, BI_MIN = Sh::BI_MIN, BI_MAX = Sh::BI_MAX, TBYTES = Sh::TBYTES;
  // memory operations a chunk's first step issues besides the weights: the next halo, and
  // with the backward prologue also the chunk's dy stores and the next chunk's y loads
  constexpr int XB = PRO == kProBwd ? 3 * HI : HI;
  static_assert((D - 1) * BI_MIN + XB <= 60, "load counter range");

  __shared__ __attribute__((aligned(16))) unsigned char sH0[Sh::H0BYTES];
  __shared__ __attribute__((aligned(16))) unsigned char sH1[Sh::HBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char sB0[KT * TBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char sB1[KT * TBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char sB2[SB > 2 ? KT * TBYTES : 16];
  __shared__ __attribute__((aligned(16))) unsigned char sB3[SB > 3 ? KT * TBYTES : 16];
  __shared__ __attribute__((aligned(16))) unsigned char sB4[SB > 4 ? KT * TBYTES : 16];
  __shared__ __attribute__((aligned(16))) unsigned char sB5[SB > 5 ? KT * TBYTES : 16];
  __shared__ int64_t s_dst[BM];
  __shared__ float s_red[NW][BN];
  __shared__ float s_mean[BN];
  // prologue constants, [2 or 4][cs]: forward scale, shift; backward a, b, c, d (bn_bwd_fold)
  extern __shared__ __attribute__((aligned(16))) float s_pro[];
  static_assert(PRO != kProFwd || !BT, "the BN + SiLU prologue is a forward's");
  static_assert(PRO != kProBwd || (BT && KV == 1), "the BN + SiLU backward prologue: a data gradient, four waves");
  static_assert(KV == 1 || KV == 2, "one or two reduction halves");
  auto hbuf = [&](auto hc) __attribute__((always_inline)) -> unsigned char* {
    if constexpr (decltype(hc)::value == 0) return sH0;
    else return sH1;
  };
  auto bstage = [&](auto bc) __attribute__((always_inline)) -> unsigned char* {
    constexpr int b = decltype(bc)::value;
    if constexpr (b == 0) return sB0;
    else if constexpr (b == 1) return sB1;
    else if constexpr (b == 2) return sB2;
    else if constexpr (b == 3) return sB3;
    else if constexpr (b == 4) return sB4;
    else return sB5;
  };

  const TileId T{(int)blockIdx.x, (int)blockIdx.y, 0};
  const GemmPhase& P = a.ph[0];
  const Geo Ge = load_geo(P);
  const int m0 = T.mt * BM;
  const int n0 = T.nt * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wave = KV == 2 ? (wv & 3) : wv;  // the wave's rows (and load slots)
  const int kh = KV == 2 ? (wv >> 2) : 0;     // its reduction half
  const int l32 = lane & 31, half = lane >> 5;
  const int W = a.ws, H = a.hs, cs = a.cs, nout = a.nout;
  const int64_t pix2 = a.src_pix * 2;
  const int64_t npix = (int64_t)a.nimg * H * W;
  // a two-dimensional tile: image img2, output rows h0 .. h0 + TR, columns w0 .. w0 + TC
  // (the host checks that TR divides H and TC divides W, so every tile is whole)
  int img2 = 0, h0 = 0, w0 = 0;
  if constexpr (TC > 0) {
    const int ncol = W / TC, nrow = H / TR;
    img2 = T.mt / (nrow * ncol);
    const int rem = T.mt - img2 * nrow * ncol;
    const int tr = rem / ncol;
    h0 = tr * TR;
    w0 = (rem - tr * ncol) * TC;
  }

  // zero rows read by out-of-image taps (never a load target)
  if (tid < 4) {
    *reinterpret_cast<u32x4*>(sH0 + Sh::HPAD * 64 + tid * 16) = u32x4{0u, 0u, 0u, 0u};
    *reinterpret_cast<u32x4*>(sH1 + Sh::HPAD * 64 + tid * 16) = u32x4{0u, 0u, 0u, 0u};
  }
  // prologue: the BN constants of every source channel (published by the barrier below,
  // before any halo is transformed)
  if constexpr (PRO == kProFwd) {
    for (int ch = tid; ch < cs; ch += NW * 64 * KV)
      bn_fold(a.pro_gamma[ch], a.pro_beta[ch], a.pro_mean[ch], a.pro_var[ch], a.pro_eps, s_pro[ch], s_pro[cs + ch]);
    __syncthreads();
  } else if constexpr (PRO == kProBwd) {
    for (int ch = tid; ch < cs; ch += NW * 64 * KV)
      bn_bwd_fold(a.pro_gamma[ch], a.pro_beta[ch], a.pro_mean[ch], a.pro_rstd[ch], a.pro_dgamma[ch],
                  a.pro_dbeta[ch], a.pro_m, s_pro[ch], s_pro[cs + ch], s_pro[2 * cs + ch], s_pro[3 * cs + ch]);
    __syncthreads();
  }

  // ---- halo loads: instruction q of this wave fills pixels (q*NW + wave)*16 .. +16; the
  // lane's slot is lane % 4 of pixel lane / 4, holding chunk slot ^ ((pixel >> 2) & 3).
  // Linear tiles: halo pixel j is source pixel m0 - W - 1 + j.  Two-dimensional tiles:
  // halo pixel j is (row j / (TC + 2), column j % (TC + 2)) of the padded window whose
  // corner is (h0 - 1, w0 - 1); its pixels outside the image load zeros (the padding).
  const int64_t hbase_px =
      TC > 0 ? ((int64_t)img2 * H + h0 - 1) * W + w0 - 1 : (int64_t)m0 - W - 1;
  const __amdgpu_buffer_rsrc_t rsA = buffer_rsrc(a.src + hbase_px * a.src_pix);
  uint32_t hoff[HI];
  int hc8[HI];  // channel of the lane's chunk within a 32-channel chunk
#pragma unroll
  for (int q = 0; q < HI; ++q) {
    const int j = (q * NW + wave) * 16 + (lane >> 2);
    const int lc = (lane & 3) ^ ((j >> 2) & 3);
    if constexpr (TC > 0) {
      const int hr = j / (TC + 2), hcol = j - hr * (TC + 2);
      const bool ok = j < (TR + 2) * (TC + 2) && (unsigned)(h0 - 1 + hr) < (unsigned)H &&
                      (unsigned)(w0 - 1 + hcol) < (unsigned)W;
      hoff[q] = ok ? (uint32_t)(((int64_t)hr * W + hcol) * pix2 + lc * 16) : kOob;
      hc8[q] = ok ? lc * 8 : (1 << 20);
    } else {
      const int64_t src_px = hbase_px + j;
      const bool ok = src_px >= 0 && src_px < npix && j < BM + 2 * W + 2;
      hoff[q] = ok ? (uint32_t)(j * pix2 + lc * 16) : kOob;
      hc8[q] = ok ? lc * 8 : (1 << 20);
    }
  }
  // backward prologue: byte offset of the lane's chunk of halo instruction q in a tensor of
  // pixel stride pix (relative to that tensor's halo base pixel; valid where hoff[q] is),
  // and whether its pixel is one of the tile's own output pixels (the halo's interior)
  auto chunk_off = [&](int q, int64_t pix) __attribute__((always_inline)) -> uint32_t {
    const int j = (q * NW + wave) * 16 + (lane >> 2);
    const int lc = (lane & 3) ^ ((j >> 2) & 3);
    if constexpr (TC > 0) {
      const int hr = j / (TC + 2), hcol = j - hr * (TC + 2);
      return (uint32_t)(((int64_t)hr * W + hcol) * pix * 2 + lc * 16);
    } else {
      return (uint32_t)(j * pix * 2 + lc * 16);
    }
  };
  auto interior = [&](int q) __attribute__((always_inline)) -> bool {
    const int j = (q * NW + wave) * 16 + (lane >> 2);
    if constexpr (TC > 0) {
      const int hr = j / (TC + 2), hcol = j - hr * (TC + 2);
      return hr >= 1 && hr <= TR && hcol >= 1 && hcol <= TC;
    } else {
      return j >= W + 1 && j < W + 1 + BM;
    }
  };
  const __amdgpu_buffer_rsrc_t rsY = buffer_rsrc(PRO == kProBwd ? a.pro_y + hbase_px * a.pro_y_pix : a.src);
  const __amdgpu_buffer_rsrc_t rsD = buffer_rsrc(PRO == kProBwd ? a.pro_dy + hbase_px * a.pro_dy_pix : a.dst);
  u32x4 yv[PRO == kProBwd ? HI : 1];  // y of the lane's chunks of the next chunk to transform

  // ---- weight loads: instruction u of a step covers 1 KiB of tap u / (BI / KT)'s stage
  const __amdgpu_buffer_rsrc_t rsB = buffer_rsrc(P.wt);
  constexpr int BPT = BN / 16;  // load instructions per tap
  uint32_t boff[BI_MAX];
  int bch[BI_MAX];  // non-transposed: channel of the lane's chunk; transposed: o row of the stage
  int btap[BI_MAX];  // tap of the step (0 .. KT-1) the instruction loads
#pragma unroll
  for (int j = 0; j < BI_MAX; ++j) {
    const int u = j * NW + wave;     // instruction index within the step
    const int tp = u / BPT, v = u % BPT;
    btap[j] = tp;
    if constexpr (!BT) {
      // stage row = output channel n0 + row, 64 bytes = 32 channels of one tap
      const int row = v * 16 + (lane >> 2), o = n0 + row;
      const int lc = (lane & 3) ^ ((row >> 2) & 3);
      const bool ok = u < BI && o < nout;
      boff[j] = ok ? (uint32_t)(((int64_t)o * 9 * cs + tp * cs + lc * 8) * 2) : kOob;
      bch[j] = ok ? lc * 8 : (1 << 20);
    } else {
      // stage row = reduction channel o (of the 32-channel chunk), 2*BN bytes = output
      // channels n0 .. n0 + BN of one (flipped) tap
      const int byte = v * 1024 + lane * 16;
      const int row = byte / (2 * BN), slot = (byte % (2 * BN)) / 16;
      const int ch = slot ^ bt_swizzle<BN>(row);
      const bool ok = u < BI && n0 + ch * 8 < nout;
      boff[j] = ok ? (uint32_t)(((int64_t)row * 9 * nout + n0 + ch * 8) * 2) : kOob;
      bch[j] = ok ? row : (1 << 20);
    }
  }
  const int nchunk = (cs + 31) / 32;
  const int nsteps = SPC * nchunk;

  auto issue_halo = [&](auto hc, int c) __attribute__((always_inline)) {
    if (KV == 2 && kh != 0) return;
    unsigned char* Hb = hbuf(hc);
    const int cb = 32 * c;
#pragma unroll
    for (int q = 0; q < HI; ++q) {
      const uint32_t v = cb + hc8[q] < cs ? hoff[q] : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (lds_void_t*)(Hb + (q * NW + wave) * 1024), 16, v,
                                               (uint32_t)(cb * 2), 0, 0);
    }
  };
  // weights of step s (chunk s / SPC, taps KT * (s % SPC) ..) into stage bc
  auto issue_b = [&](auto bc, int s) __attribute__((always_inline)) {
    if (KV == 2 && kh != 0) return;
    unsigned char* Bb = bstage(bc);
    const int c = s / SPC, t0 = KT * (s - SPC * c), cb = 32 * c;
    const bool live = s < nsteps;
    uint32_t so;
    if constexpr (!BT) so = (uint32_t)((t0 * cs + cb) * 2);
    else so = (uint32_t)(((int64_t)cb * 9 + 8 - t0) * nout * 2);  // the flipped tap 8 - t
#pragma unroll
    for (int j = 0; j < BI_MAX; ++j) {
      if (j * NW + wave < BI) {  // wave-uniform
        const uint32_t v = (live && cb + bch[j] < cs) ? boff[j] : kOob;
        // (transposed: tap t0 + btap is 8 - t0 - btap, btap rows of weights lower)
        const uint32_t sv = BT ? so - (uint32_t)(btap[j] * nout * 2) : so;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, (lds_void_t*)(Bb + (j * NW + wave) * 1024), 16, v, sv, 0, 0);
      }
    }
  };

  // ---- this lane's A rows: the LDS address of every tap of its rows (linear tiles: the
  // zero row for taps outside the image; two-dimensional tiles: the padded window holds
  // those zeros itself)
  uint32_t aaddr[TM][9];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int prow = wave * WTM + i * 32 + l32;
    if constexpr (TC > 0) {
      const int ir = prow / TC, ic = prow - ir * TC;
#pragma unroll
      for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s = 0; s < 3; ++s) {
          const int p = (ir + r) * (TC + 2) + ic + s;
          aaddr[i][3 * r + s] = (uint32_t)(p * 64 + (((half) ^ ((p >> 2) & 3)) << 4));
        }
      continue;
    }
    const int m = m0 + prow;
    uint32_t mask = 0;
    if (m < Ge.m) {
      uint32_t img, oh, ow;
      geo_pos((uint32_t)m, Ge, img, oh, ow);
#pragma unroll
      for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s = 0; s < 3; ++s) {
          const bool in = (unsigned)((int)oh + r - 1) < (unsigned)H && (unsigned)((int)ow + s - 1) < (unsigned)W;
          mask |= (in ? 1u : 0u) << (3 * r + s);
        }
    }
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        const int p = prow + r * W + s;
        const uint32_t ad = (uint32_t)(p * 64 + (((half) ^ ((p >> 2) & 3)) << 4));
        const uint32_t zr = (uint32_t)(Sh::HPAD * 64 + half * 16);
        aaddr[i][3 * r + s] = ((mask >> (3 * r + s)) & 1u) ? ad : zr;
      }
  }
  // transposed B reads (see convdma_kernel): lane l = 16 g + 4 e + q reads 4 columns of
  // rows 8 (g / 2) + e and that + 4 of each 16-row slice
  uint32_t btoff[BT ? TN : 1];
  if constexpr (BT) {
    const int g = lane >> 4, e = (lane & 15) >> 2, q = lane & 3;
    const int r0 = 8 * (g >> 1) + e;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int c = 4 * j + 2 * (g & 1) + (q >> 1);
      btoff[j] = (uint32_t)(r0 * 2 * BN + (c ^ bt_swizzle<BN>(r0)) * 16 + (q & 1) * 8);
    }
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // the backward prologue on a tile whose plain kernel has two reduction halves: the second
  // 16-channel slice of every step goes to accumulators of its own, added last, so the sums
  // (and dx) equal the plain kernel's bit for bit
  constexpr bool SPLIT = PRO == kProBwd && Sh::KV == 2;
  f32x16 acc2[SPLIT ? TM : 1][SPLIT ? TN : 1];
  if constexpr (SPLIT) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc2[i][j][r] = 0.f;
  }

  // multiply one tap (t, within the step's stage at tap slot tk) from halo buffer hc
  auto compute_tap = [&](const unsigned char* Hb, const unsigned char* Bb, auto tc, auto khc)
                         __attribute__((always_inline)) {
    constexpr int t = decltype(tc)::value, KH = decltype(khc)::value;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (KV == 2 && ks != KH) continue;  // (compile-time after unrolling)
      u32x4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const u32x4*>(Hb + (aaddr[i][t] ^ (uint32_t)(32 * ks)));
      if constexpr (!BT) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int row = j * 32 + l32;
          bf[j] = *reinterpret_cast<const u32x4*>(Bb + row * 64 + ((((2 * ks + half) ^ ((row >> 2) & 3))) << 4));
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const unsigned char* pb = Bb + btoff[j] + ks * 16 * 2 * BN;
          const v4s_t r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)pb);
          const v4s_t r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(pb + 4 * 2 * BN));
          const v2u_t lo = __builtin_bit_cast(v2u_t, r0), hi = __builtin_bit_cast(v2u_t, r1);
          bf[j][0] = lo.x;
          bf[j][1] = lo.y;
          bf[j][2] = hi.x;
          bf[j][3] = hi.y;
        }
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          if constexpr (SPLIT) {
            if (ks == 0) acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
            else acc2[SPLIT ? i : 0][SPLIT ? j : 0] = mfma32x32x16(af[i], bf[j], acc2[SPLIT ? i : 0][SPLIT ? j : 0]);
          } else {
            acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
          }
        }
    }
  };
  // wait for this wave's loads of the step (N later loads stay in flight), then every wave's
  auto sync = [&](auto nc) __attribute__((always_inline)) {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(decltype(nc)::value) : "memory");
  };
  // backward prologue: y of this lane's chunks of chunk c, into registers (zeros past the
  // channels and outside the image)
  auto issue_y = [&](int c) __attribute__((always_inline)) {
    if constexpr (PRO == kProBwd) {
      const int cb = 32 * c;
#pragma unroll
      for (int q = 0; q < HI; ++q) {
        const uint32_t v = (hoff[q] != kOob && cb + hc8[q] < cs) ? chunk_off(q, a.pro_y_pix) : kOob;
        yv[q] = __builtin_amdgcn_raw_buffer_load_b128(rsY, v, (uint32_t)(cb * 2), 0);
      }
    }
  };
  // backward prologue: the chunks of chunk c's halo that halo wave `wave` loaded (landed
  // and visible) become dy in place, from g there and y in yv.  A lane's chunks are the same
  // 8 channels for every halo instruction (slot (lane & 3) ^ ((lane >> 4) & 3)); they are
  // done in two passes of 4 channels, each with its 16 constants in registers (the
  // accumulators stay live, so the working set is kept small), the second pass storing the
  // whole chunk.  One dy store per halo instruction, issued by every wave whatever its
  // lanes hold (out of range where the chunk is not the tile's own pixel, or in another
  // column tile's block), so the wave's count of memory operations is fixed.
  auto transform_bwd = [&](auto hc, int c) __attribute__((always_inline)) {
    unsigned char* Hb = hbuf(hc);
    const int cb = 32 * c;
    const int c8 = 8 * ((lane & 3) ^ ((lane >> 4) & 3));
    const int ch = cb + c8 < cs ? cb + c8 : 0;
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      float ka[4], kb[4], kc[4], kd[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ka[e] = s_pro[ch + 4 * ps + e];
        kb[e] = s_pro[cs + ch + 4 * ps + e];
        kc[e] = s_pro[2 * cs + ch + 4 * ps + e];
        kd[e] = s_pro[3 * cs + ch + 4 * ps + e];
      }
#pragma unroll
      for (int q = 0; q < HI; ++q) {
        const bool live = hoff[q] != kOob && cb + hc8[q] < cs;
        unsigned char* p = Hb + (q * NW + wave) * 1024 + lane * 16;
        // pass 0: the first 4 channels; pass 1: the last 4, with the first 4 as pass 0 left them
        u32x4 v;
        if (ps == 0) {
          const uint2 h = *reinterpret_cast<const uint2*>(p);
          v = u32x4{h.x, h.y, 0u, 0u};
        } else {
          v = *reinterpret_cast<const u32x4*>(p);
        }
        const uint32_t g0 = v[2 * ps], g1 = v[2 * ps + 1];
        const uint32_t y0 = yv[q][2 * ps], y1 = yv[q][2 * ps + 1];
        const float o0 = bn_silu_bwd_apply(bf2f(g0 & 0xffffu), bf2f(y0 & 0xffffu), ka[0], kb[0], kc[0], kd[0]);
        const float o1 = bn_silu_bwd_apply(bf2f(g0 >> 16), bf2f(y0 >> 16), ka[1], kb[1], kc[1], kd[1]);
        const float o2 = bn_silu_bwd_apply(bf2f(g1 & 0xffffu), bf2f(y1 & 0xffffu), ka[2], kb[2], kc[2], kd[2]);
        const float o3 = bn_silu_bwd_apply(bf2f(g1 >> 16), bf2f(y1 >> 16), ka[3], kb[3], kc[3], kd[3]);
        const uint2 oh = make_uint2(pack2(o0, o1), pack2(o2, o3));
        if (live) *reinterpret_cast<uint2*>(p + 8 * ps) = oh;
        if (ps == 1) {
          const uint32_t so = (live && T.nt == 0 && interior(q)) ? chunk_off(q, a.pro_dy_pix) : kOob;
          __builtin_amdgcn_raw_buffer_store_b128(u32x4{v[0], v[1], oh.x, oh.y}, rsD, so, (uint32_t)(cb * 2), 0);
          // wait states before anything rewrites the store's data registers: with the
          // scheduling barrier right after it, the compiler issued a VALU write to the first
          // data register on the next cycle, and about one 16-byte store in 20000 then wrote
          // that register's new value (measured; none with this pause)
          asm volatile("s_nop 4");
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  // prologue: this lane's own 16-byte chunks of chunk c's halo (landed: the wait before
  // this covers them) become the previous layer's activations, SiLU(BN(y)), in place;
  // chunks that loaded zeros (padding, past the image or the channels) stay zero
  auto transform = [&](auto hc, int c) __attribute__((always_inline)) {
    if constexpr (PRO != kProFwd) return;
    if (KV == 2 && kh != 0) return;  // (the chunks are half 0's loads)
    unsigned char* Hb = hbuf(hc);
    const int cb = 32 * c;
#pragma unroll
    for (int q = 0; q < HI; ++q) {
      if (hoff[q] != kOob && cb + hc8[q] < cs) {
        u32x4* p = reinterpret_cast<u32x4*>(Hb + (q * NW + wave) * 1024 + lane * 16);
        const u32x4 v = *p;
        float f[8];
        unpack8(uint4{v[0], v[1], v[2], v[3]}, f);
        const int ch = cb + hc8[q];
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = bn_silu_apply(f[e], s_pro[ch + e], s_pro[cs + ch + e]);
        const uint4 o = pack8(f);
        *p = u32x4{o.x, o.y, o.z, o.w};
      }
    }
  };
  // step k (0 .. SPC-1) of a chunk c of parity h (halo buffer h): wait, issue the next
  // halo (k = 0) and the weights D steps ahead, multiply the step's KT taps
  auto step = [&](auto hc, auto kc, int c, auto khc) __attribute__((always_inline)) {
    constexpr int h = decltype(hc)::value, k = decltype(kc)::value;
    constexpr int sl = h * SPC + k;  // step index within the two-chunk trip
    constexpr int waitn = (D - 1) * BI_MIN + ((k >= 1 && k <= D - 1) ? XB : 0);
    if constexpr (PRO == kProFwd && k == 0) {
      // the chunk's halo has landed for this wave: transform this lane's part, then publish
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(waitn) : "memory");
      transform(hc, c);
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    } else if constexpr (PRO == kProBwd && k == 0) {
      // as the forward's (the wait also covers this chunk's y, loaded before its halo), then
      // this wave's y loads of the next chunk
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(waitn) : "memory");
      transform_bwd(hc, c);
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      issue_y(c + 1);
    } else {
      sync(Ic<waitn>{});
    }
    if constexpr (k == 0) issue_halo(Ic<1 - h>{}, c + 1);
    issue_b(Ic<(sl + D) % SB>{}, SPC * c + k + D);
    const unsigned char* Hb = hbuf(hc);
    const unsigned char* Bb = bstage(Ic<sl % SB>{});
#pragma unroll
    for (int tt = 0; tt < KT; ++tt) {
      // (compile-time tap index: KT * k + tt)
      if constexpr (KT == 1) compute_tap(Hb, Bb, Ic<k>{}, khc);
      else {
        if (tt == 0) compute_tap(Hb, Bb, Ic<3 * k + 0>{}, khc);
        if (tt == 1) compute_tap(Hb, Bb + TBYTES, Ic<3 * k + 1>{}, khc);
        if (tt == 2) compute_tap(Hb, Bb + 2 * TBYTES, Ic<3 * k + 2>{}, khc);
      }
    }
  };
  auto chunk = [&](auto hc, int c, auto khc) __attribute__((always_inline)) {
    step(hc, Ic<0>{}, c, khc);
    step(hc, Ic<1>{}, c, khc);
    step(hc, Ic<2>{}, c, khc);
    if constexpr (SPC == 9) {
      step(hc, Ic<3>{}, c, khc);
      step(hc, Ic<4>{}, c, khc);
      step(hc, Ic<5>{}, c, khc);
      step(hc, Ic<6>{}, c, khc);
      step(hc, Ic<7>{}, c, khc);
      step(hc, Ic<8>{}, c, khc);
    }
  };

  issue_y(0);  // (before the halo, as at every chunk's first step)
  issue_halo(Ic<0>{}, 0);
  issue_b(Ic<0>{}, 0);
  if constexpr (D >= 2) issue_b(Ic<1>{}, 1);
  if constexpr (D >= 3) issue_b(Ic<2>{}, 2);
  if constexpr (D >= 4) issue_b(Ic<3>{}, 3);
  if constexpr (D >= 5) issue_b(Ic<4>{}, 4);
  // destination offsets of the tile's rows (the epilogue's), under the first loads
  for (int r = tid; r < BM; r += NW * 64) {
    const int m = TC > 0 ? (img2 * H + h0 + r / (TC > 0 ? TC : 1)) * W + w0 + r % (TC > 0 ? TC : 1) : m0 + r;
    s_dst[r] = dst_offset(a, Ge, m);
  }
  // the main loop, one copy per reduction half (a compile-time slice choice)
  auto main_loop = [&](auto khc) __attribute__((always_inline)) {
    int c = 0;
    for (; c + 2 <= nchunk; c += 2) {
      chunk(Ic<0>{}, c, khc);
      chunk(Ic<1>{}, c + 1, khc);
    }
    if (c < nchunk) chunk(Ic<0>{}, c, khc);
  };
  if (KV == 1 || kh == 0) main_loop(Ic<0>{});
  else main_loop(Ic<1>{});
  // the loads issued past the last step land before the halo buffer becomes staging space
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  if constexpr (KV == 2) {
    // half 1 hands its sums to half 0, one 32 x 32 block of each wave at a time through
    // halo buffer 0 (16 KiB: 4 waves x 64 lanes x 16 floats); the sum is half 0 + half 1
    f32x4* xb = reinterpret_cast<f32x4*>(sH0);
    static_assert(Sh::H0BYTES >= 4 * 64 * 64, "exchange space");
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        if (kh == 1) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            f32x4 v;
            v[0] = acc[i][j][4 * q];
            v[1] = acc[i][j][4 * q + 1];
            v[2] = acc[i][j][4 * q + 2];
            v[3] = acc[i][j][4 * q + 3];
            xb[(wave * 4 + q) * 64 + lane] = v;
          }
        }
        __syncthreads();
        if (kh == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = xb[(wave * 4 + q) * 64 + lane];
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
          }
        }
        __syncthreads();
      }
  }
  if constexpr (SPLIT) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += acc2[SPLIT ? i : 0][SPLIT ? j : 0][r];
  }
  gemm_epilogue<TM, TN, NW>(a, P, T, acc, m0, n0, sH0, s_dst, s_red, s_mean, kh == 0);
}

template <int TN>
hipError_t launch_narrow(const ConvGemmArgs& a, hipStream_t s) {
  using G = GemmShape<2, TN>;
  dim3 grid((unsigned)((a.ph[0].m + G::BM - 1) / G::BM), (unsigned)((a.nout + G::BN - 1) / G::BN), 1);
  NUMBAT_LAUNCH((convnarrow_kernel<2, TN>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

struct GInst {
  int tm, tn, d;  // 32-row tiles per wave (4 waves along M), 32-col tiles, prefetch depth (generic kernel)
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


template <int TM, int TN, int S, int BK, int NW>
void launch_dma(const ConvGemmArgs& a, int mmax, hipStream_t s) {
  using Sh = GemmShape<TM, TN, NW>;
  dim3 grid((unsigned)((mmax + Sh::BM - 1) / Sh::BM), (unsigned)((a.nout + Sh::BN - 1) / Sh::BN), (unsigned)a.nphase);
  if (a.bt)
    NUMBAT_LAUNCH((convdma_kernel<TM, TN, S, BK, NW, true>), grid, dim3(NW * 64), 0, s, a);
  else
    NUMBAT_LAUNCH((convdma_kernel<TM, TN, S, BK, NW, false>), grid, dim3(NW * 64), 0, s, a);
}

template <int I>
hipError_t launch_g(const ConvGemmArgs& a, int variant, hipStream_t s) {
  constexpr GInst c = kG[I];
  using Sh = GemmShape<c.tm, c.tn>;
  int mmax = 0;
  for (int p = 0; p < a.nphase; ++p) mmax = a.ph[p].m > mmax ? a.ph[p].m : mmax;
  if (variant == kVariantDma3)
    launch_dma<c.tm, c.tn, 3, 64, 4>(a, mmax, s);
  else if (variant == kVariantDma2)
    launch_dma<c.tm, c.tn, 2, 64, 4>(a, mmax, s);
  else if (variant == kVariantDma32)
    launch_dma<c.tm, c.tn, 3, 32, 4>(a, mmax, s);
  else if (variant == kVariantDma3W8 && c.tn <= 4)
    launch_dma<1, c.tn <= 4 ? c.tn : 4, 3, 64, 8>(a, mmax, s);
#ifdef NUMBAT_TUNING
  else if (variant == 6)
    launch_dma<c.tm, c.tn, 4, 32, 4>(a, mmax, s);
  else if (variant == 8 && c.tn <= 4)
    launch_dma<1, c.tn <= 4 ? c.tn : 4, 2, 64, 8>(a, mmax, s);
  else if (variant == 9 && c.tn <= 4)
    launch_dma<1, c.tn <= 4 ? c.tn : 4, 4, 32, 8>(a, mmax, s);
  else if (variant == 10 && c.tn <= 4)
    launch_dma<1, c.tn <= 4 ? c.tn : 4, 3, 32, 8>(a, mmax, s);
  else if (variant == 12 && c.tm == 1 && c.tn <= 3)
    launch_dma<1, c.tn <= 3 ? c.tn : 3, 5, 64, 4>(a, mmax, s);
  else if (variant == 13 && c.tm == 1 && c.tn <= 2)
    launch_dma<1, c.tn <= 2 ? c.tn : 2, 6, 64, 4>(a, mmax, s);
  else if (variant == 14 && c.tm == 1)
    launch_dma<1, c.tn, 6, 32, 4>(a, mmax, s);
#endif
  else {
    dim3 grid((unsigned)((mmax + Sh::BM - 1) / Sh::BM), (unsigned)((a.nout + Sh::BN - 1) / Sh::BN),
              (unsigned)a.nphase);
    NUMBAT_LAUNCH((convgemm_kernel<c.tm, c.tn, c.d>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// halo kernel instantiations: (32-row tiles per wave, 32-column tiles, halo load
// instructions per wave, taps per step, weight stages, tile columns); a linear BM-row tile
// (tile columns 0) of a W-wide image needs BM + 2 W + 2 halo pixels, a two-dimensional
// TR x TC tile (TC tile columns) (TR + 2) x (TC + 2), 16 per instruction
struct HInst {
  int tm, tn, hi, kt, sb, tc;
};
constexpr HInst kH[] = {
    {1, 3, 4, 3, 2, 0},   // 0: 128 x 96, W <= 63, a tap row per step, two weight stages
    {2, 3, 7, 1, 3, 0},   // 1: 256 x 96, W <= 95, one tap per step, three weight stages
    {1, 2, 4, 3, 2, 0},   // 2: 128 x 64, W <= 63
    {2, 2, 7, 1, 3, 0},   // 3: 256 x 64, W <= 95
    {2, 3, 6, 1, 3, 32},  // 4: 256 x 96 on 8 x 32 output pixels (a 10 x 34 halo), one tap per step
    {2, 2, 6, 1, 3, 32},  // 5: 256 x 64 on 8 x 32
#ifdef NUMBAT_TUNING
    {1, 3, 4, 1, 3, 0},   // 6..
    {1, 3, 5, 1, 3, 0},
    {2, 3, 6, 1, 3, 0},
    {1, 2, 8, 1, 3, 0},
    {2, 2, 10, 1, 3, 0},
    {1, 3, 4, 1, 6, 0},
    {1, 3, 4, 3, 3, 0},
    {2, 3, 6, 1, 6, 0},
    {2, 3, 6, 3, 2, 0},
    {1, 3, 5, 1, 6, 0},
    {1, 3, 5, 3, 2, 0},
    {2, 3, 7, 1, 6, 0},
    {2, 3, 7, 3, 2, 0},
    {1, 2, 4, 1, 3, 32},  // 19..: two-dimensional tiles
    {1, 2, 3, 3, 2, 16},
    {1, 3, 3, 3, 2, 16},
    {1, 3, 4, 3, 2, 32},
    {1, 2, 4, 3, 2, 32},
#endif
};
constexpr int kNumH = sizeof(kH) / sizeof(kH[0]);

template <int I>
hipError_t launch_h(const ConvGemmArgs& a, hipStream_t s) {
  if constexpr (I < kNumH) {
    constexpr HInst c = kH[I];
    using G = GemmShape<c.tm, c.tn, 4>;
    dim3 grid((unsigned)((a.ph[0].m + G::BM - 1) / G::BM), (unsigned)((a.nout + G::BN - 1) / G::BN), 1);
    constexpr int KV = HaloShape<c.tm, c.tn, c.hi, c.kt, c.sb, false, c.tc>::KV;
    // the backward prologue keeps four waves: its y registers and transform do not fit the
    // eight-wave form's 128 registers per lane
    const dim3 block(256 * KV);
    // the prologue's per-channel constants (dynamic LDS, sized to the channels so that the
    // blocks per CU stay those of the plain kernel wherever the channels allow)
    const size_t fwd_smem = (size_t)2 * a.cs * sizeof(float), bwd_smem = (size_t)4 * a.cs * sizeof(float);
#ifdef NUMBAT_TUNING
    if (KV == 2 && getenv("NUMBAT_HALO_KV1") && a.pro_kind != kProBwd) {
      if (a.bt)
        NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, true, c.tc, kProNone, 1>), grid, dim3(256), 0, s, a);
      else if (a.pro_kind == kProFwd)
        NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, false, c.tc, kProFwd, 1>), grid, dim3(256),
                      fwd_smem, s, a);
      else
        NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, false, c.tc, kProNone, 1>), grid, dim3(256), 0, s, a);
      return hipGetLastError();
    }
#endif
    if (a.bt && a.pro_kind == kProBwd)
      NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, true, c.tc, kProBwd, 1>), grid, dim3(256), bwd_smem,
                    s, a);
    else if (a.bt)
      NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, true, c.tc, kProNone, KV>), grid, block, 0, s, a);
    else if (a.pro_kind == kProFwd)
      NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, false, c.tc, kProFwd, KV>), grid, block, fwd_smem, s,
                    a);
    else
      NUMBAT_LAUNCH((convhalo_kernel<c.tm, c.tn, c.hi, c.kt, c.sb, false, c.tc, kProNone, KV>), grid, block, 0, s, a);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int I>
hipError_t launch_h_id(int id, const ConvGemmArgs& a, hipStream_t s) {
  if constexpr (I >= kNumH) return hipErrorInvalidValue;
  else return id == I ? launch_h<I>(a, s) : launch_h_id<I + 1>(id, a, s);
}

int tap_dh(int32_t off) { return (int)(int16_t)(off & 0xffff); }
int tap_dw(int32_t off) { return off >> 16; }

// Fills in the tap walk of the fast path (tw, toff0, cstep, rstep, halo_px) and reports
// whether the fast path applies: 16-multiple source channels (at least 32), taps forming a grid with
// unit steps, and every gathered byte of a tile within 32-bit buffer offsets.
bool prepare_fast(ConvGemmArgs& a, int bm) {
  if (a.cs % 16 != 0 || a.cs < 32) return false;
  const int64_t pix2 = a.src_pix * 2;
  int halo = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const GemmPhase& P = a.ph[p];
    for (int t = 0; t < P.taps; ++t) {
      const int lin = tap_dh(P.off[t]) * a.ws + tap_dw(P.off[t]);
      halo = -lin > halo ? -lin : halo;
    }
  }
  a.halo_px = halo;
  int64_t worst = 0;
  for (int p = 0; p < a.nphase; ++p) {
    GemmPhase& P = a.ph[p];
    int tw = 1;
    while (tw < P.taps && tap_dh(P.off[tw]) == tap_dh(P.off[0])) ++tw;
    if (P.taps % tw != 0) return false;
    const int sw = tw > 1 ? tap_dw(P.off[1]) - tap_dw(P.off[0]) : 0;
    const int sh = P.taps > tw ? tap_dh(P.off[tw]) - tap_dh(P.off[0]) : 0;
    int64_t maxlin = 0;
    for (int t = 0; t < P.taps; ++t) {
      const int i = t / tw, j = t % tw;
      if (tap_dh(P.off[t]) != tap_dh(P.off[0]) + i * sh || tap_dw(P.off[t]) != tap_dw(P.off[0]) + j * sw) return false;
      const int64_t lin = (int64_t)tap_dh(P.off[t]) * a.ws + tap_dw(P.off[t]) + halo;
      maxlin = lin > maxlin ? lin : maxlin;
    }
    if ((int64_t)a.nout * P.ktot * 2 >= (int64_t)kRecords) return false;  // weight offsets are 32-bit too
    P.tw = tw;
    P.th = P.taps / tw;
    P.dh0 = tap_dh(P.off[0]);
    P.dw0 = tap_dw(P.off[0]);
    P.tsh = sh;
    P.tsw = sw;
    P.toff0 = (int32_t)(((int64_t)tap_dh(P.off[0]) * a.ws + tap_dw(P.off[0]) + halo) * pix2);
    P.cstep = (int32_t)((int64_t)sw * pix2);
    P.rstep = (int32_t)(((int64_t)sh * a.ws - (int64_t)(tw - 1) * sw) * pix2);
    // a tile's rows span at most bm / (gh*gw) + 2 images
    const int64_t imgs = bm / ((int64_t)P.gh * P.gw) + 2;
    const int64_t span = (imgs * a.hs * a.ws + halo + maxlin) * pix2 + (int64_t)a.cs * 2 + 16;
    worst = span > worst ? span : worst;
  }
  return worst < (int64_t)kOob - (1 << 24);
}

}  // namespace

// Tile and kernel choice, fitted to timings of every (kernel, tile, stages) choice over
// the forward and data-gradient GEMMs of the detector's layers at batch 16, weighted by
// how often each shape occurs (within 1% of the per-layer best in total):
//  * forward (K-major weights): N tile the least padding among 128, 96 and 64 columns
//    (ties to the wider; 64 when fewer than 400 blocks of 128 rows); more than 32768
//    rows, three stages of 32 reduction elements (three blocks per CU for 128-row tiles),
//    256-row tiles when the reduction is 768 or longer, 64 columns when it is shorter
//    than 512 and 64 divides N; 8193..32768 rows, two stages of 64 (two blocks per CU) on
//    128 x 96 tiles when 96 divides N <= 192, else 128 x 64; up to 8192 rows, reductions
//    of 3000 or more into N >= 256: three stages of 64 on 128 x 96 (else x 128) tiles
//    when one block per CU covers the grid; otherwise 128 x 64 tiles, two stages of 64
//    when the grid exceeds 256 blocks, else three;
//  * data gradient (weights read in place through transposing LDS reads, which favour
//    64-column tiles): more than 32768 rows as the forward, with 64 columns on 128-row
//    tiles; 8193..32768 rows, eight waves on 256 x 96 (or x 64) tiles with three stages
//    of 64 when the reduction is 1000 or longer and one such block per CU covers the
//    grid, else 128 x 64 with three stages of 32; up to 8192 rows, 128 x 64 with two
//    stages of 64 when the grid holds 300 blocks or more, else three;
//  * generic kernel (narrow or 8-multiple channels): 256-row tiles unless that leaves
//    fewer than 512 blocks.
TileCfg convgemm_pick(int64_t m_max, int nout, int cs, int ktot, int nphase, bool bt) {
  const int bns[4] = {128, 96, 64, 32};
  const int ncand = nout <= 32 ? 4 : 3;
  int bn = 128;
  int64_t waste = INT64_MAX;
  for (int i = 0; i < ncand; ++i) {
    const int64_t w = ((nout + bns[i] - 1) / bns[i]) * bns[i] - nout;
    if (w < waste) {
      waste = w;
      bn = bns[i];
    }
  }
  const bool fast = cs % 16 == 0 && cs >= 32;
  int bm, variant;
  if (fast && !bt) {
    const int64_t mt = (m_max + 127) / 128;
    const int64_t blocks128 = mt * ((nout + bn - 1) / bn);
    if (blocks128 < 400 && bn > 64) bn = 64;
    bm = 128;
    if (m_max > 32768) {
      variant = kVariantDma32;
      bm = ktot >= 768 ? 256 : 128;
      if (ktot < 512 && nout % 64 == 0) bn = 64;
    } else if (m_max > 8192) {
      variant = kVariantDma2;
      bn = (nout % 96 == 0 && nout <= 192) ? 96 : 64;
    } else if (ktot >= 3000 && nout >= 256) {
      // long reductions: one 128 x 96 (or x 128) block per CU with three 64-deep stages,
      // when the grid fits one round
      variant = kVariantDma3;
      bn = (nout % 96 == 0 && mt * (nout / 96) <= 256) ? 96 : mt * ((nout + 127) / 128) <= 256 ? 128 : 64;
    } else {
      bn = 64;
      variant = mt * ((nout + 63) / 64) > 256 ? kVariantDma2 : kVariantDma3;
    }
  } else if (fast) {
    const int bn64 = bn < 64 ? bn : 64;
    bm = 128;
    if (m_max > 32768) {
      variant = kVariantDma32;
      if (ktot >= 768) bm = 256;
      else bn = bn64;
    } else if (m_max > 8192) {
      const int bn8 = nout % 96 == 0 ? 96 : bn64;
      const int64_t blocks8 = ((m_max + 255) / 256) * ((nout + bn8 - 1) / bn8) * nphase;
      if (ktot >= 1000 && blocks8 <= 256) {
        variant = kVariantDma3W8;
        bm = 256;
        bn = bn8;
      } else {
        variant = kVariantDma32;
        bn = bn64;
      }
    } else {
      bn = bn64;
      const int64_t blocks = ((m_max + 127) / 128) * ((nout + bn - 1) / bn) * nphase;
      variant = blocks >= 300 ? kVariantDma2 : kVariantDma3;
    }
  } else {
    const int64_t blocks256 = ((m_max + 255) / 256) * ((nout + bn - 1) / bn);
    bm = blocks256 < 512 ? 128 : 256;
    variant = kVariantGeneric;
  }
  int id = (bm == 128 ? 4 : 0) + (bn == 128 ? 0 : bn == 96 ? 1 : bn == 64 ? 2 : 3);
#ifdef NUMBAT_TUNING
  // timing sweeps only: force the instantiation and kernel
  if (const char* e = getenv("NUMBAT_TILE")) id = atoi(e);
  if (const char* e = getenv("NUMBAT_VARIANT")) variant = fast ? atoi(e) : kVariantGeneric;
  if (variant >= kVariantDma3W8 && variant <= 10) id &= 3;  // eight waves of 32 rows: the 256-row instantiations
  bm = kG[id].tm * 128;
  bn = kG[id].tn * 32;
#endif
  return TileCfg{bm, bn, id, variant};
}

// narrow input (ci < 8): 256-row tiles, 32 or 64 columns
TileCfg narrow_pick(int nout) { return TileCfg{256, nout <= 32 ? 32 : 64, -1, kVariantGeneric}; }

// the RGB image layer's shape: 3 channels, 3x3 taps at offsets -1..1, stride 2, at most
// 64 output channels, output rows a multiple of 4 and columns of 64, 256-row tiles
bool stem_shape(const ConvGemmArgs& a, const TileCfg& t) {
  const GemmPhase& P = a.ph[0];
  if (a.nphase != 1 || a.cs != 3 || P.taps != 9 || a.gstride_h != 2 || a.gstride_w != 2 || a.nout > 64 ||
      t.bm != 256 || P.gh % 4 != 0 || P.gw % 64 != 0 || a.nimg > 65535 || P.gh / 4 > 65535)
    return false;
  for (int r = 0; r < 3; ++r)
    for (int q = 0; q < 3; ++q)
      if (P.off[r * 3 + q] != (int32_t)((uint32_t)(uint16_t)(int16_t)(r - 1) | ((uint32_t)(q - 1) << 16))) return false;
  return true;
}

hipError_t convnarrow_launch(const ConvGemmArgs& a, const TileCfg& t, hipStream_t s) {
  if (a.nphase != 1 || a.ph[0].ktot > NarrowShape<2, 2>::KMAX || a.ph[0].taps > kMaxTaps)
    return hipErrorInvalidValue;
  if (stem_shape(a, t)) {
    trace_begin(KC_CONV_FWD);
    dim3 grid((unsigned)(a.ph[0].gw / 64), (unsigned)(a.ph[0].gh / 4), (unsigned)a.nimg);
    NUMBAT_LAUNCH(convstem_kernel, grid, dim3(256), 0, s, a);
    trace_end(KC_CONV_FWD);
    return hipGetLastError();
  }
  trace_begin(KC_CONV_FWD);
  const hipError_t e = t.bn == 32 ? launch_narrow<1>(a, s) : launch_narrow<2>(a, s);
  trace_end(KC_CONV_FWD);
  return e;
}

bool convgemm_direct(ConvGemmArgs a, const TileCfg& t) {
  return t.variant != kVariantGeneric && prepare_fast(a, t.bm);
}

hipError_t convgemm_launch(ConvGemmArgs a, const TileCfg& t, hipStream_t s, int cls) {
  // a problem the fast paths cannot take runs the generic kernel on the same tile
  const int variant = (t.variant != kVariantGeneric && prepare_fast(a, t.bm)) ? t.variant : kVariantGeneric;
  if (a.bt && variant == kVariantGeneric) return hipErrorInvalidValue;  // needs K-major B
  a.remap = 0;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_REMAP_CONV")) a.remap = atoi(e);
#endif
  trace_begin(cls);
  hipError_t e;
  switch (t.id) {
    case 0: e = launch_g<0>(a, variant, s); break;
    case 1: e = launch_g<1>(a, variant, s); break;
    case 2: e = launch_g<2>(a, variant, s); break;
    case 3: e = launch_g<3>(a, variant, s); break;
    case 4: e = launch_g<4>(a, variant, s); break;
    case 5: e = launch_g<5>(a, variant, s); break;
    case 6: e = launch_g<6>(a, variant, s); break;
    default: e = launch_g<7>(a, variant, s); break;
  }
  trace_end(cls);
  return e;
}

// 3x3, stride 1, padding 1, 16-multiple source channels (at least 32), one phase
bool convhalo_shape(const ConvGemmArgs& a) {
  const GemmPhase& P = a.ph[0];
  if (a.nphase != 1 || a.cs % 16 != 0 || a.cs < 32 || P.taps != 9 || a.gstride_h != 1 || a.gstride_w != 1 ||
      a.dstep_h != 1 || a.dstep_w != 1 || P.gh != a.hs || P.gw != a.ws || a.hd != a.hs || a.wd != a.ws)
    return false;
  if (!a.bt)
    for (int r = 0; r < 3; ++r)
      for (int q = 0; q < 3; ++q)
        if (P.off[r * 3 + q] != (int32_t)((uint32_t)(uint16_t)(int16_t)(r - 1) | ((uint32_t)(q - 1) << 16)))
          return false;
  // weight offsets of one step are 32-bit
  return (int64_t)a.nout * 9 * a.cs * 2 < (int64_t)kRecords;
}

// the halo pixels a tile needs: a linear BM-row tile (tc 0) of a w-wide image, or a
// two-dimensional (BM / tc) x tc one
static int halo_pixels(int bm, int tc, int w) { return tc > 0 ? (bm / tc + 2) * (tc + 2) : bm + 2 * w + 2; }

// Halo kernel tile, from a sweep of the instantiations over the detector's 3x3 stride-1
// layers at batch 16 (each layer alone): 96 columns when 96 divides the channel count, else
// 64; images up to 63 pixels wide on 128-row tiles with a whole tap row (three taps) per
// step and two weight stages (40 x 40, 192 channels: forward 33.6 -> 29.6 us, data
// gradient 29.4 -> 24.0), up to 95 wide on 256-row tiles with one tap per step and three
// stages (80 x 80, 96 channels: 35.4 -> 28.3 and 28.9 -> 22.6 us); wider images on
// two-dimensional tiles of 8 x 32 output pixels with one tap per step and three stages,
// when 32 divides the width and 8 the height (160 x 160, 48 channels: forward 54.5 -> 51.1,
// data gradient 44.2 -> 39.3 us against the direct-to-LDS kernel; a linear tile of a
// 160-wide image needs 2.5 image rows of halo and measured 30-80% slower, 4 x 32 tiles
// with a tap row per step 10-20% slower, and 8 x 16 tiles on the 80-wide layers 13-18%
// slower than their linear 256-row tiles).  Forward grids of fewer than 256 tiles (20 x 20,
// 288 channels: 23.6 -> 26.1 us) keep the direct-to-LDS kernel.  Returns variant
// kVariantGeneric when the halo kernel is not used.
TileCfg convhalo_pick(int64_t m, int nout, int h, int w, bool bt, bool any_grid) {
  const int tn = nout % 96 == 0 ? 3 : 2;
  int tm = w <= 63 ? 1 : 2, kt = w <= 63 ? 3 : 1, sb = w <= 63 ? 2 : 3, tc = 0;
  if (w > 95) {
    tm = 2;
    kt = 1;
    sb = 3;
    tc = 32;
  }
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_HALO_TM")) tm = atoi(e);
  if (const char* e = getenv("NUMBAT_HALO_KT")) kt = atoi(e);
  if (const char* e = getenv("NUMBAT_HALO_SB")) sb = atoi(e);
  if (const char* e = getenv("NUMBAT_HALO_TC")) tc = atoi(e);
#endif
  const TileCfg none{0, 0, -1, kVariantGeneric};
  if (tc > 0 && (w % tc != 0 || (128 * tm) % tc != 0 || h % (128 * tm / tc) != 0)) return none;
  const int64_t tiles = ((m + 128 * tm - 1) / (128 * tm)) * ((nout + 32 * tn - 1) / (32 * tn));
  if (!bt && !any_grid && tiles < 256) return none;
  int best = -1;
  for (int i = 0; i < kNumH; ++i) {
    const HInst& c = kH[i];
    if (c.tm != tm || c.tn != tn || c.kt != kt || c.sb != sb || c.tc != tc) continue;
    if (c.hi * 64 < halo_pixels(128 * tm, tc, w)) continue;
    if (best < 0 || c.hi < kH[best].hi) best = i;
  }
  if (best < 0) return none;
  return TileCfg{128 * kH[best].tm, 32 * kH[best].tn, best, kVariantHalo};
}

hipError_t convhalo_launch(const ConvGemmArgs& a, const TileCfg& t, hipStream_t s, int cls) {
  if (t.variant != kVariantHalo || t.id < 0 || t.id >= kNumH || !convhalo_shape(a)) return hipErrorInvalidValue;
  if (a.pro_kind == kProFwd && (a.bt || a.cs > kProMaxC || a.pro_mean == nullptr)) return hipErrorInvalidValue;
  if (a.pro_kind == kProBwd && (!a.bt || a.cs > kProMaxC || a.pro_y == nullptr || a.pro_dy == nullptr))
    return hipErrorInvalidValue;
  if (a.pro_kind != kProNone && a.pro_kind != kProFwd && a.pro_kind != kProBwd) return hipErrorInvalidValue;
  const HInst& c = kH[t.id];
  if (c.hi * 64 < halo_pixels(t.bm, c.tc, a.ws)) return hipErrorInvalidValue;
  // a two-dimensional tile must divide the image (every tile whole)
  if (c.tc > 0 && (a.ws % c.tc != 0 || a.hs % (t.bm / c.tc) != 0)) return hipErrorInvalidValue;
  trace_begin(cls);
  const hipError_t e = launch_h_id<0>(t.id, a, s);
  trace_end(cls);
  return e;
}

}  // namespace numbat

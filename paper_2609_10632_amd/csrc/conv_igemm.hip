// Implicit-GEMM convolution on gfx950 MFMA (bf16 in, fp32 accumulate).
//
// One kernel serves the forward convolution and every stride phase of the data
// gradient: both are GEMMs whose A operand is gathered from an NHWC tensor at a
// per-tap spatial offset (zero outside the image) and whose B operand is a dense
// [N][K] weight matrix with K contiguous.  Tiles of A and B are staged through LDS
// with a two-buffer pipeline (global loads for step k+1 are in flight while MFMAs
// consume step k); each wave owns a (TM*16) x (TN*16) block of accumulators built
// from 16x16x32 bf16 MFMAs.  The epilogue rounds to bf16 and, for the forward,
// reduces the fp32 accumulators of the tile into per-channel (mean, M2) partials
// for the batch statistics of the following BatchNorm.
#include "kernels.h"

namespace numbat {

namespace {

constexpr int BK = 64;             // reduction elements per pipeline step
constexpr int LDS_ROW = BK + 8;    // bf16 per LDS row: 16 B of padding against bank conflicts

template <int WM, int WN, int TM, int TN, bool SMALLC>
__global__ __launch_bounds__(256) void igemm_kernel(IgemmArgs a) {
  constexpr int BM = WM * TM * 16;
  constexpr int BN = WN * TN * 16;
  constexpr int AV = BM / 32;         // A vectors (16 B) per thread per step
  constexpr int BV = (BN + 31) / 32;  // B vectors per thread per step
  static_assert(WM * WN == 4, "four waves");
  static_assert(BM % 32 == 0, "BM multiple of 32");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][LDS_ROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][LDS_ROW];
  __shared__ int32_t s_off[kMaxTaps];
  __shared__ float s_red[WM][BN];
  __shared__ float s_mean[BN];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int cv = tid & 7;    // which 16-byte column of the BK-wide tile this thread loads
  const int rbase = tid >> 3;  // first tile row this thread loads

  if (tid < kMaxTaps) s_off[tid] = a.off[tid];

  // per-row gather state for the A operand
  int64_t abase[AV];
  int aih[AV], aiw[AV];
#pragma unroll
  for (int i = 0; i < AV; ++i) {
    const int64_t m = m0 + rbase + 32 * i;
    if (m < a.m) {
      const uint32_t mm = (uint32_t)m;
      const uint32_t img = fdiv(mm, a.div_ghw);
      const uint32_t rem = mm - img * (uint32_t)(a.gh * a.gw);
      const uint32_t gi = fdiv(rem, a.div_gw);
      const uint32_t gj = rem - gi * (uint32_t)a.gw;
      abase[i] = (int64_t)img * a.hs * a.ws;
      aih[i] = (int)gi * a.gstride_h;
      aiw[i] = (int)gj * a.gstride_w;
    } else {
      abase[i] = 0;
      aih[i] = -(1 << 28);  // never inside the image
      aiw[i] = 0;
    }
  }
  // reduction position of this thread's A/B column
  int tapA = 0, cA = 0;
  if (!SMALLC) {
    tapA = (cv * 8) / a.cs;
    cA = (cv * 8) - tapA * a.cs;
  }
  __syncthreads();

  uint4 ra[AV], rb[BV];
  const int nk = (a.ktot + BK - 1) / BK;

  auto load_tiles = [&](int kt) {
    const int kb = kt * BK + cv * 8;
    if (!SMALLC) {
      int off = 0;
      const bool tap_ok = tapA < a.taps;
      if (tap_ok) off = s_off[tapA];
      const int dh = (int)(int16_t)(off & 0xffff), dw = off >> 16;
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        uint4 v = make_uint4(0, 0, 0, 0);
        const int ih = aih[i] + dh, iw = aiw[i] + dw;
        if (tap_ok && (unsigned)ih < (unsigned)a.hs && (unsigned)iw < (unsigned)a.ws)
          v = *reinterpret_cast<const uint4*>(a.src + ((abase[i] + (int64_t)ih * a.ws + iw) * a.src_pix + cA));
        ra[i] = v;
      }
      cA += BK;
      while (cA >= a.cs) {
        cA -= a.cs;
        ++tapA;
      }
    } else {
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        uint32_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          h[e] = 0;
          const int k = kb + e;
          if (k < a.ktot) {
            const int tap = k / a.cs;
            const int c = k - tap * a.cs;
            const int off = s_off[tap];
            const int ih = aih[i] + (int)(int16_t)(off & 0xffff), iw = aiw[i] + (off >> 16);
            if ((unsigned)ih < (unsigned)a.hs && (unsigned)iw < (unsigned)a.ws)
              h[e] = a.src[(abase[i] + (int64_t)ih * a.ws + iw) * a.src_pix + c];
          }
        }
        ra[i] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
      }
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int row = rbase + 32 * i;
      const int o = n0 + row;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < BN && o < a.nout) {
        if (!SMALLC) {
          if (kb < a.ktot) v = *reinterpret_cast<const uint4*>(a.wt + (int64_t)o * a.ktot + kb);
        } else {
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = (kb + e < a.ktot) ? a.wt[(int64_t)o * a.ktot + kb + e] : 0u;
          v = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
        }
      }
      rb[i] = v;
    }
  };

  auto store_tiles = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AV; ++i) *reinterpret_cast<uint4*>(&As[buf][rbase + 32 * i][cv * 8]) = ra[i];
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int row = rbase + 32 * i;
      if (row < BN) *reinterpret_cast<uint4*>(&Bs[buf][row][cv * 8]) = rb[i];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tiles(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      uint4 af[TM], bfr[TN];
      const int kc = ks * 32 + (lane >> 4) * 8;
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
    if (kt + 1 < nk) store_tiles(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: bf16 output
  const int colbase = n0 + wn * TN * 16 + (lane & 15);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = wm * TM * 16 + i * 16 + 4 * (lane >> 4) + e;
      const int64_t m = m0 + row;
      if (m >= a.m) continue;
      const uint32_t mm = (uint32_t)m;
      const uint32_t img = fdiv(mm, a.div_ghw);
      const uint32_t rem = mm - img * (uint32_t)(a.gh * a.gw);
      const uint32_t gi = fdiv(rem, a.div_gw);
      const uint32_t gj = rem - gi * (uint32_t)a.gw;
      const int64_t pix = ((int64_t)img * a.hd + (int)gi * a.dstep_h + a.doff_h) * a.wd + (int)gj * a.dstep_w + a.doff_w;
      bf16_t* drow = a.dst + pix * a.dst_pix;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = colbase + j * 16;
        if (col < a.nout) {
          float v = acc[i][j][e];
          if (a.accumulate) v += bf2f(drow[col]);
          drow[col] = (bf16_t)f2bf(v);
        }
      }
    }
  }

  // ---- epilogue: per-channel (mean, M2) of this tile's rows, from the fp32 accumulators
  if (a.stats_part != nullptr) {
    const int64_t left = (int64_t)a.m - m0;
    const int count = left < BM ? (int)left : BM;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i) s += (acc[i][j][0] + acc[i][j][1]) + (acc[i][j][2] + acc[i][j][3]);
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (lane < 16) s_red[wm][wn * TN * 16 + j * 16 + lane] = s;
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
      const float mu = s_mean[wn * TN * 16 + j * 16 + (lane & 15)];
      float q = 0.f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = wm * TM * 16 + i * 16 + 4 * (lane >> 4) + e;
          const float d = acc[i][j][e] - mu;
          q += (row < count) ? d * d : 0.f;
        }
      q += __shfl_xor(q, 16);
      q += __shfl_xor(q, 32);
      if (lane < 16) s_red[wm][wn * TN * 16 + j * 16 + lane] = q;
    }
    __syncthreads();
    if (tid < BN && n0 + tid < a.nout) {
      float q = 0.f;
#pragma unroll
      for (int w = 0; w < WM; ++w) q += s_red[w][tid];
      a.stats_part[(int64_t)blockIdx.x * a.nout + n0 + tid] = make_float2(s_mean[tid], q);
    }
  }
}

// Tile instantiations: (waves along M, waves along N, 16-row tiles per wave, 16-col tiles per wave)
struct Inst {
  int wm, wn, tm, tn;
};
constexpr Inst kInst[] = {
    {2, 2, 4, 4},  // 0: 128 x 128
    {4, 1, 2, 3},  // 1: 128 x 48
    {2, 2, 4, 3},  // 2: 128 x 96
    {2, 2, 4, 2},  // 3: 128 x 64
    {4, 1, 2, 5},  // 4: 128 x 80
    {4, 1, 1, 1},  // 5: 64 x 16 (tiny N)
};

template <int I, bool S>
hipError_t launch_inst(const IgemmArgs& a, hipStream_t s) {
  constexpr Inst c = kInst[I];
  constexpr int BM = c.wm * c.tm * 16, BN = c.wn * c.tn * 16;
  dim3 grid((unsigned)((a.m + BM - 1) / BM), (unsigned)((a.nout + BN - 1) / BN));
  hipLaunchKernelGGL((igemm_kernel<c.wm, c.wn, c.tm, c.tn, S>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <bool S>
hipError_t launch_any(const IgemmArgs& a, int id, hipStream_t s) {
  switch (id) {
    case 0: return launch_inst<0, S>(a, s);
    case 1: return launch_inst<1, S>(a, s);
    case 2: return launch_inst<2, S>(a, s);
    case 3: return launch_inst<3, S>(a, s);
    case 4: return launch_inst<4, S>(a, s);
    default: return launch_inst<5, S>(a, s);
  }
}

}  // namespace

TileCfg igemm_pick(int64_t m, int nout, int cs) {
  (void)m;
  (void)cs;
  // smallest padding waste on N; M tile fixed
  struct Opt {
    int id, bm, bn;
  };
  const Opt opts[] = {{0, 128, 128}, {2, 128, 96}, {4, 128, 80}, {3, 128, 64}, {1, 128, 48}};
  if (nout <= 16) return TileCfg{64, 16, 5};
  int best = 0;
  int64_t best_waste = INT64_MAX;
  for (int i = 0; i < 5; ++i) {
    const int64_t tiles = (nout + opts[i].bn - 1) / opts[i].bn;
    const int64_t waste = tiles * opts[i].bn - nout;
    // prefer wider tiles when waste ties
    if (waste < best_waste) {
      best_waste = waste;
      best = i;
    }
  }
  return TileCfg{opts[best].bm, opts[best].bn, opts[best].id};
}

hipError_t igemm_launch(const IgemmArgs& a, const TileCfg& t, hipStream_t s, int cls) {
  const bool smallc = (a.cs % 8) != 0;
  trace_begin(cls, s);
  const hipError_t e = smallc ? launch_any<true>(a, t.id, s) : launch_any<false>(a, t.id, s);
  trace_end(cls, s);
  return e;
}

// ---------------------------------------------------------------------------
// Merge of per-tile (mean, M2) partials into the batch mean and biased variance, in
// fp64 and a fixed order.  With K the first tile's mean (a shift shared by every thread
// of a channel), each thread sums n_t (mean_t - K), n_t (mean_t - K)^2 and M2_t over the
// tiles g, g+G, g+2G, ...; the G partial sums are added in index order, and
//   mean = K + S1 / N,   M2 = sum M2_t + S2 - N (S1 / N)^2
// (the pairwise update of Chan et al. written as sums, with no division per tile).

namespace {

// 8 channels per block, 32 groups of tiles per channel: consecutive lanes read the
// partials of consecutive channels (64-byte segments) and each lane keeps several loads
// in flight.
constexpr int kMergeCh = 8, kMergeGroups = 32;

__global__ __launch_bounds__(kMergeCh * kMergeGroups) void stats_merge_kernel(const float2* part, int mtiles,
                                                                              int tile_rows, int64_t m, int c,
                                                                              float* mean_var) {
  __shared__ double s1s[kMergeGroups][kMergeCh], s2s[kMergeGroups][kMergeCh], m2s[kMergeGroups][kMergeCh];
  const int cl = threadIdx.x % kMergeCh;
  const int g = threadIdx.x / kMergeCh;
  const int ch = blockIdx.x * kMergeCh + cl;
  double s1 = 0, s2 = 0, m2 = 0;
  double K = 0;
  if (ch < c) {
    K = (double)part[ch].x;
    // every tile but the last holds tile_rows rows
    const int full = (int)((m / tile_rows) < mtiles ? (m / tile_rows) : mtiles);
    const double nt = (double)tile_rows;
    int t = g;
#pragma unroll 8
    for (; t < full; t += kMergeGroups) {
      const float2 p = part[(int64_t)t * c + ch];
      const double d = (double)p.x - K;
      s1 += nt * d;
      s2 += nt * d * d;
      m2 += (double)p.y;
    }
    for (; t < mtiles; t += kMergeGroups) {
      const double cnt = (double)(m - (int64_t)t * tile_rows);
      const float2 p = part[(int64_t)t * c + ch];
      const double d = (double)p.x - K;
      s1 += cnt * d;
      s2 += cnt * d * d;
      m2 += (double)p.y;
    }
  }
  s1s[g][cl] = s1;
  s2s[g][cl] = s2;
  m2s[g][cl] = m2;
  __syncthreads();
  if (g == 0 && ch < c) {
    for (int k = 1; k < kMergeGroups; ++k) {
      s1 += s1s[k][cl];
      s2 += s2s[k][cl];
      m2 += m2s[k][cl];
    }
    const double n = (double)m;
    const double dm = s1 / n;
    mean_var[ch] = (float)(K + dm);
    const double v = (m2 + s2 - n * dm * dm) / n;
    mean_var[c + ch] = (float)(v > 0 ? v : 0);
  }
}

}  // namespace

hipError_t stats_merge_launch(const float2* part, int mtiles, int tile_rows, int64_t m, int c, float* mean_var,
                              hipStream_t s) {
  trace_begin(KC_STATS_MERGE, s);
  hipLaunchKernelGGL(stats_merge_kernel, dim3((c + kMergeCh - 1) / kMergeCh), dim3(kMergeCh * kMergeGroups), 0, s,
                     part, mtiles, tile_rows, m, c, mean_var);
  trace_end(KC_STATS_MERGE, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Data-gradient weight re-layout.  Phase f gathers the taps (r, s) that reach the
// input rows/cols of that stride phase; its B matrix is wt[c][t][o] = w[o][r_t][s_t][c]
// (N = c_in rows, K = taps * c_out contiguous).

namespace {

struct PhaseTable {
  int nphase;
  int first[16];  // element offset of each phase's matrix inside wt
  int count[16];
  int r[16][kMaxTaps], s[16][kMaxTaps];
};

__global__ void dgrad_weights_kernel(const bf16_t* w, bf16_t* wt, int co, int kh, int kw, int ci, PhaseTable tab) {
  const int64_t total = (int64_t)co * kh * kw * ci;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    // i enumerates the destination: find phase, then (c, t, o)
    int f = 0;
    while (f + 1 < tab.nphase && i >= tab.first[f + 1]) ++f;
    const int64_t j = i - tab.first[f];
    const int T = tab.count[f];
    const int o = (int)(j % co);
    const int64_t ct = j / co;
    const int t = (int)(ct % T);
    const int c = (int)(ct / T);
    const int r = tab.r[f][t], s = tab.s[f][t];
    wt[i] = w[(((int64_t)o * kh + r) * kw + s) * ci + c];
  }
}

}  // namespace

hipError_t dgrad_weights_launch(const bf16_t* w, bf16_t* wt, int co, int kh, int kw, int ci, const int* phase_first,
                                const PhaseTaps* phases, int nphase, hipStream_t s) {
  PhaseTable tab;
  tab.nphase = nphase;
  for (int f = 0; f < nphase; ++f) {
    tab.first[f] = phase_first[f];
    tab.count[f] = phases[f].count;
    for (int t = 0; t < phases[f].count; ++t) {
      tab.r[f][t] = phases[f].r[t];
      tab.s[f][t] = phases[f].s[t];
    }
  }
  const int64_t total = (int64_t)co * kh * kw * ci;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  trace_begin(KC_DGRAD_WEIGHTS, s);
  hipLaunchKernelGGL(dgrad_weights_kernel, dim3(blocks), dim3(256), 0, s, w, wt, co, kh, kw, ci, tab);
  trace_end(KC_DGRAD_WEIGHTS, s);
  return hipGetLastError();
}

}  // namespace numbat

// Auxiliary kernels of the convolution passes on gfx950: the fixed-order merge of the
// forward's per-tile batch-statistics partials, the data-gradient weight re-layout, and
// the 8-channel repacking that lets a 3-channel image input use the vectorized kernels.
#include "kernels.h"

namespace numbat {

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
  int first[16];       // element offset of each phase's matrix inside wt
  int item_first[16];  // first work item of each phase (items are (tap, 8 o's, c) triples)
  int count[16];
  int r[16][kMaxTaps], s[16][kMaxTaps];
};

// One thread writes 8 consecutive output channels (16 bytes) of one destination row
// (phase f, channel c, tap t): wt[f][c][t][o..o+7] = w[o..o+7][r][s][c], zero for the
// padding channels c >= ci.  Consecutive threads take consecutive c, so each of the 8
// source reads is coalesced across the wave.
__global__ void dgrad_weights_kernel(const bf16_t* w, uint4* wt, int co, int kh, int kw, int ci, int cpad, int nitems,
                                     PhaseTable tab) {
  const int cpr = co / 8;  // 8-channel chunks per destination row
  const int64_t ostride = (int64_t)kh * kw * ci;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < nitems; i += gridDim.x * blockDim.x) {
    int f = 0;
    while (f + 1 < tab.nphase && i >= tab.item_first[f + 1]) ++f;
    const int T = tab.count[f];
    const int j = i - tab.item_first[f];
    const int c = j % cpad, q = j / cpad;
    const int oc = q % cpr, t = q / cpr;
    uint32_t h[8];
    if (c < ci) {
      const bf16_t* src = w + (int64_t)(oc * 8) * ostride + ((int64_t)tab.r[f][t] * kw + tab.s[f][t]) * ci + c;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = src[e * ostride];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = 0u;
    }
    const int64_t dst = (tab.first[f] + ((int64_t)c * T + t) * co) / 8 + oc;
    wt[dst] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  }
}

}  // namespace

hipError_t dgrad_weights_launch(const bf16_t* w, bf16_t* wt, int co, int kh, int kw, int ci, int cpad,
                                const int* phase_first, const PhaseTaps* phases, int nphase, hipStream_t s) {
  PhaseTable tab;
  tab.nphase = nphase;
  int items = 0;
  for (int f = 0; f < nphase; ++f) {
    tab.first[f] = phase_first[f];
    tab.item_first[f] = items;
    tab.count[f] = phases[f].count;
    items += cpad * phases[f].count * (co / 8);
    for (int t = 0; t < phases[f].count; ++t) {
      tab.r[f][t] = phases[f].r[t];
      tab.s[f][t] = phases[f].s[t];
    }
  }
  const int nitems = items;
  int blocks = (nitems + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  trace_begin(KC_DGRAD_WEIGHTS, s);
  hipLaunchKernelGGL(dgrad_weights_kernel, dim3(blocks), dim3(256), 0, s, w, reinterpret_cast<uint4*>(wt), co, kh, kw,
                     ci, cpad, nitems, tab);
  trace_end(KC_DGRAD_WEIGHTS, s);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// 8-channel repacking: dst[i][0..7] = (src[i*src_pix + c] for c < ci, then zeros).  Used
// for the image input (ci = 3) and its weights, so the forward and the weight gradient
// run on the 16-byte-vector kernels.

namespace {

__global__ void pack8_kernel(const bf16_t* src, int64_t src_pix, int ci, int64_t n, uint4* dst) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    uint32_t h[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) h[c] = c < ci ? (uint32_t)src[i * src_pix + c] : 0u;
    dst[i] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  }
}

__global__ void unpack_dw_kernel(const float* dw8, float* dw, int64_t rows, int ci, int accumulate) {
  const int64_t total = rows * ci;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / ci;
    const int c = (int)(i - r * ci);
    const float v = dw8[r * 8 + c];
    dw[i] = accumulate ? dw[i] + v : v;
  }
}

// dst[i*dst_pix + c] (+)= src[i][c] for c < ci: the narrow channels of an 8-channel bf16
// tensor (the data gradient of a 3-channel input, which the GEMM writes padded to 8)
__global__ void unpack8_kernel(const uint4* src, int ci, int64_t n, bf16_t* dst, int64_t dst_pix) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint4 v = src[i];
    const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (c < ci) dst[i * dst_pix + c] = (bf16_t)(wd[c >> 1] >> (16 * (c & 1)));
  }
}

int blocks_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 16384) b = 16384;
  return (int)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t pack8_launch(const bf16_t* src, int64_t src_pix, int ci, int64_t n, bf16_t* dst, hipStream_t s) {
  trace_begin(KC_PACK, s);
  hipLaunchKernelGGL(pack8_kernel, dim3(blocks_for(n)), dim3(256), 0, s, src, src_pix, ci, n, reinterpret_cast<uint4*>(dst));
  trace_end(KC_PACK, s);
  return hipGetLastError();
}

hipError_t unpack8_launch(const bf16_t* src8, int ci, int64_t n, bf16_t* dst, int64_t dst_pix, hipStream_t s) {
  trace_begin(KC_PACK, s);
  hipLaunchKernelGGL(unpack8_kernel, dim3(blocks_for(n)), dim3(256), 0, s, reinterpret_cast<const uint4*>(src8), ci, n, dst,
                     dst_pix);
  trace_end(KC_PACK, s);
  return hipGetLastError();
}

hipError_t unpack_dw_launch(const float* dw8, float* dw, int64_t rows, int ci, int accumulate, hipStream_t s) {
  trace_begin(KC_PACK, s);
  hipLaunchKernelGGL(unpack_dw_kernel, dim3(blocks_for(rows * ci)), dim3(256), 0, s, dw8, dw, rows, ci, accumulate);
  trace_end(KC_PACK, s);
  return hipGetLastError();
}

}  // namespace numbat

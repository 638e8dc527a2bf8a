// Auxiliary kernels of the convolution passes on gfx950: the fixed-order merge of the
// forward's per-tile batch-statistics partials, the data-gradient weight re-layouts, the
// 8-channel repacking that lets a 3-channel image input use the weight-gradient kernel,
// and the direct data gradient of such an input.
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

// 8 channels per block, 128 groups of tiles per channel: consecutive lanes read the
// partials of consecutive channels (64-byte segments) and each lane keeps several loads
// in flight; the group sums are combined by a fixed pairwise tree.  (With 32 groups the
// 6400 tiles of the image-input layer took 25 dependent rounds of loads.)
constexpr int kMergeCh = 8, kMergeGroups = 128;

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
#pragma unroll
  for (int h = kMergeGroups / 2; h > 0; h >>= 1) {
    if (g < h) {
      s1s[g][cl] += s1s[g + h][cl];
      s2s[g][cl] += s2s[g + h][cl];
      m2s[g][cl] += m2s[g + h][cl];
    }
    __syncthreads();
  }
  if (g == 0 && ch < c) {
    s1 = s1s[0][cl];
    s2 = s2s[0][cl];
    m2 = m2s[0][cl];
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
// for the image input (ci = 3) of the weight gradient, so it runs on the 16-byte-vector
// kernel; unpack_dw_kernel then keeps the ci real columns of the 8-column result.

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

hipError_t unpack_dw_launch(const float* dw8, float* dw, int64_t rows, int ci, int accumulate, hipStream_t s) {
  trace_begin(KC_PACK, s);
  hipLaunchKernelGGL(unpack_dw_kernel, dim3(blocks_for(rows * ci)), dim3(256), 0, s, dw8, dw, rows, ci, accumulate);
  trace_end(KC_PACK, s);
  return hipGetLastError();
}



// ---------------------------------------------------------------------------
// Data gradient of a narrow input (ci < 8: the RGB image).  As a GEMM its N would be ci
// (padded to a 32-column tile), so one thread computes the ci channels of one input
// pixel directly:
//   dx[p][c] = sum over taps (r, s) and o of dy[q(p, r, s)][o] * W[o][r][s][c].
// Threads are grouped by stride phase (blockIdx.y), so every lane of a wave walks the
// same taps and weight indices: the weights are read with wave-uniform addresses
// (scalar loads) and dy with 16-byte vectors of 8 output channels.  The sum is formed
// in fp32 (plus the existing dx when accumulating) and rounded once.
namespace {

// (the tensors are separate restrict-qualified arguments so the compiler knows the
// weights are not written by the kernel and reads them with scalar loads)
constexpr int kNarrowChunk = 64;

// weights as fp32 [kh][kw][co][ci]: the weights of one tap and 8 output channels are
// 8 * ci consecutive aligned words, which scalar loads fetch whole
__global__ void narrow_weights_kernel(const bf16_t* w, float* wf, int co, int kh, int kw, int ci) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // ((r * kw + s) * co + o) * ci + c
  const int64_t total = (int64_t)kh * kw * co * ci;
  if (i >= total) return;
  const int c = (int)(i % ci);
  const int64_t ro = i / ci;
  const int o = (int)(ro % co);
  const int rs = (int)(ro / co);
  wf[i] = bf2f(w[((int64_t)o * kh * kw + rs) * ci + c]);
}

template <int CI>
__global__ __launch_bounds__(256) void dgrad_narrow_kernel(NarrowDgradArgs a, const bf16_t* __restrict__ dy,
                                                           const float* __restrict__ wf,
                                                           bf16_t* __restrict__ dx) {
  // Each wave computes 64 consecutive pixels of one phase row (one per lane).  A pass is
  // one tap and up to CH output channels: the wave reads the 64 dy pixels that tap needs
  // -- contiguous memory -- with 1 KiB wave loads, writes them to its own LDS rows (odd
  // pitch in 16-byte units: conflict-free row reads), and each lane reads its pixel's
  // channels back.  (A per-lane 16-byte gather of the same data touches 64 cache lines
  // per load instruction.)  The loads of the next pass are in flight in registers while
  // the current pass is multiplied.
  constexpr int CH = kNarrowChunk;  // channels per pass (8 chunks of 8)
  constexpr int P16 = CH / 8 + 1;   // LDS row pitch in 16-byte units (odd)
  __shared__ uint4 s_px[4][64 * P16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sh = a.sh, sw = a.sw;
  const int pa = (int)blockIdx.y / sw, pb = (int)blockIdx.y - pa * sw;
  const int gh = pa < a.h ? (a.h - pa + sh - 1) / sh : 0;
  const int gw = pb < a.w ? (a.w - pb + sw - 1) / sw : 0;
  const int segs = (gw + 63) / 64;  // 64-pixel segments per phase row
  const int64_t seg = (int64_t)blockIdx.x * 4 + wave;
  const int64_t per_img = (int64_t)gh * segs;
  if (seg >= (int64_t)a.n * per_img) return;  // wave-uniform
  const int img = (int)(seg / per_img);
  const int rem = (int)(seg - (int64_t)img * per_img);
  const int i = rem / segs, j0 = (rem - i * segs) * 64;
  uint4* rows = s_px[wave];
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(dy), (short)0, 0x7ffffff0,
                                                                      0x00020000);
  // the phase's taps in order: (r, s) with sh | (pa + ph - r) and sw | (pb + pw - s)
  auto next_tap = [&](int& r, int& s) -> bool {
    for (;;) {
      if (++s >= a.kw) {
        s = 0;
        if (++r >= a.kh) return false;
      }
      if ((pa + a.ph - r) % sh == 0 && (pb + a.pw - s) % sw == 0) return true;
    }
  };
  u32x4 buf[8];
  // issue the loads of pass (r, s, cc): instruction k covers pixels 8k..8k+7, lane
  // (pixel 8k + lane/8, chunk lane%8), so a pixel's channels are consecutive bytes; a
  // chunk past the pass, or a pixel outside the image or past the phase row, reads zeros
  const int lpx = lane >> 3, lck = lane & 7;
  auto fetch = [&](int r, int s, int cc) __attribute__((always_inline)) {
    const int oh = i + (pa + a.ph - r) / sh, ow0 = j0 + (pb + a.pw - s) / sw;
    const int nch = (a.co - cc < CH ? a.co - cc : CH) / 8;
    const bool rok = (unsigned)oh < (unsigned)a.ho && lck < nch;
    const int64_t rowbase = ((int64_t)img * a.ho + oh) * a.wo;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int px = 8 * k + lpx, ow = ow0 + px;
      const bool ok = rok && (unsigned)ow < (unsigned)a.wo && j0 + px < gw;
      const uint32_t vo = ok ? (uint32_t)((rowbase + ow) * a.dy_pix * 2 + (int64_t)(cc + lck * 8) * 2) : 0x80000000u;
      buf[k] = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, 0u, 0);
    }
  };
  auto stage = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < 8; ++k) rows[(8 * k + lpx) * P16 + lck] = make_uint4(buf[k][0], buf[k][1], buf[k][2], buf[k][3]);
  };
  float acc[CI];
#pragma unroll
  for (int c = 0; c < CI; ++c) acc[c] = 0.f;
  int r = 0, s = -1, cc = 0;
  bool have = next_tap(r, s);
  if (have) fetch(r, s, cc);
  while (have) {  // wave-uniform
    stage();
    // (one wave's LDS accesses complete in issue order: the rows written above are read
    // below, and overwritten by the next pass, without a barrier)
    __builtin_amdgcn_wave_barrier();
    int nr = r, ns = s, ncc = cc + CH;
    bool nhave = true;
    if (ncc >= a.co) {
      ncc = 0;
      nhave = next_tap(nr, ns);
    }
    if (nhave) fetch(nr, ns, ncc);
    const float* wrs = wf + (((int64_t)r * a.kw + s) * a.co + cc) * CI;  // W[o][r][s][c] = wrs[(o - cc) * CI + c]
    const int nch = (a.co - cc < CH ? a.co - cc : CH) / 8;
    for (int ck = 0; ck < nch; ++ck) {
      float f[8];
      unpack8(rows[lane * P16 + ck], f);
      const float* wk = wrs + ck * 8 * CI;
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int c = 0; c < CI; ++c) acc[c] += f[e] * wk[e * CI + c];
    }
    __builtin_amdgcn_wave_barrier();
    r = nr;
    s = ns;
    cc = ncc;
    have = nhave;
  }
  const int j = j0 + lane;
  if (j >= gw) return;
  bf16_t* dst = dx + (((int64_t)img * a.h + pa + sh * i) * a.w + pb + sw * j) * a.dx_pix;
#pragma unroll
  for (int c = 0; c < CI; ++c) {
    const float v = a.accumulate ? acc[c] + bf2f(dst[c]) : acc[c];
    dst[c] = (bf16_t)f2bf(v);
  }
}

}  // namespace

hipError_t dgrad_narrow_launch(const NarrowDgradArgs& a, int ci, float* wf, hipStream_t s) {
  const int ghm = (a.h + a.sh - 1) / a.sh, gwm = (a.w + a.sw - 1) / a.sw;
  const int64_t blocks = ((int64_t)a.n * ghm * ((gwm + 63) / 64) + 3) / 4;  // 4 waves of 64 pixels
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t wn = (int64_t)a.kh * a.kw * a.co * ci;
  trace_begin(KC_DGRAD_WEIGHTS, s);
  hipLaunchKernelGGL(narrow_weights_kernel, dim3((unsigned)((wn + 255) / 256)), dim3(256), 0, s, a.wt, wf, a.co, a.kh,
                     a.kw, ci);
  trace_end(KC_DGRAD_WEIGHTS, s);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)blocks, (unsigned)(a.sh * a.sw), 1);
  trace_begin(KC_CONV_DGRAD, s);
  switch (ci) {
    case 1: hipLaunchKernelGGL(dgrad_narrow_kernel<1>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 2: hipLaunchKernelGGL(dgrad_narrow_kernel<2>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 3: hipLaunchKernelGGL(dgrad_narrow_kernel<3>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 4: hipLaunchKernelGGL(dgrad_narrow_kernel<4>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 5: hipLaunchKernelGGL(dgrad_narrow_kernel<5>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 6: hipLaunchKernelGGL(dgrad_narrow_kernel<6>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 7: hipLaunchKernelGGL(dgrad_narrow_kernel<7>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    default: trace_end(KC_CONV_DGRAD, s); return hipErrorInvalidValue;
  }
  trace_end(KC_CONV_DGRAD, s);
  return hipGetLastError();
}

}  // namespace numbat

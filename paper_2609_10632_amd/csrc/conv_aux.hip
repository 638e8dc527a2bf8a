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
// in flight; the group sums are combined in a fixed order (shuffles within a wave, then
// a pairwise tree over the waves).  (With 32 groups the
// 6400 tiles of the image-input layer took 25 dependent rounds of loads.)
constexpr int kMergeCh = 8, kMergeGroups = 128;

__global__ __launch_bounds__(kMergeCh * kMergeGroups) void stats_merge_kernel(const float2* part, int mtiles,
                                                                              int tile_rows, int64_t m, int c,
                                                                              float* mean_var) {
  __shared__ double s1s[kMergeCh * kMergeGroups / 64][kMergeCh], s2s[kMergeCh * kMergeGroups / 64][kMergeCh],
      m2s[kMergeCh * kMergeGroups / 64][kMergeCh];
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
  // lanes 8 apart hold the same channel of neighbouring groups: shuffles combine the 8
  // groups of a wave, then one thread per channel adds the 16 wave sums pairwise
#pragma unroll
  for (int d = 8; d < 64; d *= 2) {
    s1 += __shfl_xor(s1, d);
    s2 += __shfl_xor(s2, d);
    m2 += __shfl_xor(m2, d);
  }
  const int wave = threadIdx.x / 64;
  if ((threadIdx.x & 63) < kMergeCh) {
    s1s[wave][cl] = s1;
    s2s[wave][cl] = s2;
    m2s[wave][cl] = m2;
  }
  __syncthreads();
  if (g == 0 && ch < c) {
    constexpr int NWv = kMergeCh * kMergeGroups / 64;  // 16 waves
    double a1[NWv], a2[NWv], a3[NWv];
#pragma unroll
    for (int w = 0; w < NWv; ++w) {
      a1[w] = s1s[w][cl];
      a2[w] = s2s[w][cl];
      a3[w] = m2s[w][cl];
    }
#pragma unroll
    for (int h = NWv / 2; h > 0; h >>= 1)
#pragma unroll
      for (int w = 0; w < h; ++w) {
        a1[w] += a1[w + h];
        a2[w] += a2[w + h];
        a3[w] += a3[w + h];
      }
    s1 = a1[0];
    s2 = a2[0];
    m2 = a3[0];
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
  trace_begin(KC_STATS_MERGE);
  NUMBAT_LAUNCH(stats_merge_kernel, dim3((c + kMergeCh - 1) / kMergeCh), dim3(kMergeCh * kMergeGroups), 0, s,
                     part, mtiles, tile_rows, m, c, mean_var);
  trace_end(KC_STATS_MERGE);
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
  trace_begin(KC_DGRAD_WEIGHTS);
  NUMBAT_LAUNCH(dgrad_weights_kernel, dim3(blocks), dim3(256), 0, s, w, reinterpret_cast<uint4*>(wt), co, kh, kw,
                     ci, cpad, nitems, tab);
  trace_end(KC_DGRAD_WEIGHTS);
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
  trace_begin(KC_PACK);
  NUMBAT_LAUNCH(pack8_kernel, dim3(blocks_for(n)), dim3(256), 0, s, src, src_pix, ci, n, reinterpret_cast<uint4*>(dst));
  trace_end(KC_PACK);
  return hipGetLastError();
}

hipError_t unpack_dw_launch(const float* dw8, float* dw, int64_t rows, int ci, int accumulate, hipStream_t s) {
  trace_begin(KC_PACK);
  NUMBAT_LAUNCH(unpack_dw_kernel, dim3(blocks_for(rows * ci)), dim3(256), 0, s, dw8, dw, rows, ci, accumulate);
  trace_end(KC_PACK);
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

// ---------------------------------------------------------------------------
// Data gradient of a narrow input on MFMA, for c_out a multiple of 16 up to 64 and
// kh*kw*ci <= 32 (the RGB image layer).  Per output-gradient pixel q the products with
// every (tap, channel) form one small GEMM row,
//   Z[q][(r, s, c)] = sum over o of dy[q][o] * W[o][r][s][c]   (N = kh*kw*ci <= 32, K = c_out),
// and each input pixel p then sums the Z entries of the (q, r, s) that reach it:
//   dx[p][c] = sum over (r, s) with p = q*stride - pad + (r, s) of Z[q][(r, s, c)].
// A block owns a TH x TW patch of dx and loads the dy pixels its taps reach (the patch
// plus a halo) once: [q][c_out] bf16 rows in LDS, the weights as [n = (r,s,c)][o].  Each
// wave multiplies 32-row blocks of q with 32x32x16 MFMAs, the fp32 Z replaces dy in LDS,
// and each thread sums the ci channels of its dx pixels (fp32, rounded once).
constexpr int kNqMax = 192;   // dy pixels per block (six 32-row MFMA blocks)
constexpr int kNarrowKp = 72; // bf16 per LDS row of dy and of the weights (c_out <= 64, odd multiple of 16 bytes)
constexpr int kZp = 33;       // fp32 per LDS row of Z

__device__ __forceinline__ int floordiv(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// Patch geometry: image, first input row and column, and the dy rows/columns reached.
struct NarrowPatch {
  int img, i0, j0, i1, j1, qr0, qc0, nqc, nq;
};
__device__ __forceinline__ NarrowPatch narrow_patch(const NarrowDgradArgs& a, int pid, int th, int lgtw, int ntw,
                                                    int nth, int kh, int kw, int sh, int sw) {
  NarrowPatch P;
  const int tj = pid % ntw, r = pid / ntw;
  const int ti = r % nth;
  P.img = r / nth;
  P.i0 = ti * th;
  P.j0 = tj << lgtw;
  P.i1 = min(P.i0 + th, a.h);
  P.j1 = min(P.j0 + (1 << lgtw), a.w);
  const int qr0 = max(floordiv(P.i0 + a.ph - kh + 1 + sh - 1, sh), 0);
  const int qc0 = max(floordiv(P.j0 + a.pw - kw + 1 + sw - 1, sw), 0);
  const int qr1 = min(floordiv(P.i1 - 1 + a.ph, sh), a.ho - 1);
  const int qc1 = min(floordiv(P.j1 - 1 + a.pw, sw), a.wo - 1);
  P.qr0 = qr0;
  P.qc0 = qc0;
  P.nqc = max(qc1 - qc0 + 1, 0);
  P.nq = max(qr1 - qr0 + 1, 0) * P.nqc;  // <= kNqMax (the host sizes the patch)
  return P;
}

// Each block walks patches blockIdx.x, + gridDim.x, ...; the dy loads of its next patch
// are in flight while it multiplies and sums the current one.  KS (square kernel side),
// SS (square stride), TH, LGTW (patch rows, log2 patch columns) and CO are compile-time
// for the RGB image layer and 0 (taken from the arguments) otherwise: the index
// arithmetic, not the data, bounds this kernel.
template <int CI, int KS, int SS, int TH, int LGTW, int CO>
__global__ __launch_bounds__(256) void dgrad_narrow_mfma_kernel(NarrowDgradArgs a, int th_, int lgtw_, int ntw,
                                                                int nth, int npatch) {
  const int kh = KS ? KS : a.kh, kw = KS ? KS : a.kw, sh = SS ? SS : a.sh, sw = SS ? SS : a.sw;
  const int th = TH ? TH : th_, lgtw = LGTW ? LGTW : lgtw_;
  const int tw = 1 << lgtw;
  __shared__ __attribute__((aligned(16))) unsigned char s_buf[kNqMax * kNarrowKp * 2 > kNqMax * kZp * 4
                                                                  ? kNqMax * kNarrowKp * 2
                                                                  : kNqMax * kZp * 4];
  __shared__ __attribute__((aligned(16))) bf16_t s_w[32 * kNarrowKp];
  bf16_t* s_dy = reinterpret_cast<bf16_t*>(s_buf);
  float* s_z = reinterpret_cast<float*>(s_buf);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int nn = kh * kw * CI;
  const int co = CO ? CO : a.co, cch = co >> 3, nks = co >> 4;
  constexpr int kWLoads = 32 * 64 / 2 / 256;  // nn * co / 2 <= 1024 words
  constexpr int kQLoads = kNqMax / 32;        // pixel rounds of 32
  const int c8 = tid & 7;

  // dy rows of a patch's reached pixels, 16-byte chunks: thread t loads chunk t % 8 of
  // pixels t / 8, + 32, + 64, ... (walked without division)
  auto load_dy = [&](const NarrowPatch& P, uint4 (&dv)[kQLoads]) __attribute__((always_inline)) {
    const int nqc = max(P.nqc, 1);
    int q = tid >> 3, qi = q / nqc, qj = q - qi * nqc;
#pragma unroll
    for (int u = 0; u < kQLoads; ++u) {
      dv[u] = make_uint4(0u, 0u, 0u, 0u);
      if (c8 < cch && q < P.nq)
        dv[u] = *reinterpret_cast<const uint4*>(a.dy + (((int64_t)P.img * a.ho + P.qr0 + qi) * a.wo + P.qc0 + qj) *
                                                           a.dy_pix +
                                                c8 * 8);
      q += 32;
      qj += 32;
      while (qj >= nqc) {
        qj -= nqc;
        ++qi;
      }
    }
  };

  int pid = blockIdx.x;
  NarrowPatch P = narrow_patch(a, pid, th, lgtw, ntw, nth, kh, kw, sh, sw);
  uint4 dv[kQLoads];
  load_dy(P, dv);
  // weights as [n][o] (zero rows past nn): the OHWI tensor [o][n] is read contiguously
  // (4-byte words: nn * co is even since co is) and scattered into LDS
  {
    const int nw = (nn * co) >> 1;
    uint32_t wv[kWLoads];
#pragma unroll
    for (int u = 0; u < kWLoads; ++u) {
      const int e = tid + 256 * u;
      wv[u] = e < nw ? reinterpret_cast<const uint32_t*>(a.wt)[e] : 0u;
    }
    for (int e = tid; e < (32 - nn) * (kNarrowKp / 2); e += 256)
      reinterpret_cast<uint32_t*>(s_w + nn * kNarrowKp)[e] = 0u;
#pragma unroll
    for (int u = 0; u < kWLoads; ++u) {
      const int e = tid + 256 * u;
      if (e < nw) {
        const int o = (2 * e) / nn, n = 2 * e - o * nn;
        s_w[n * kNarrowKp + o] = (bf16_t)(wv[u] & 0xffffu);
        const int n1 = n + 1 < nn ? n + 1 : 0, o1 = n + 1 < nn ? o : o + 1;
        s_w[n1 * kNarrowKp + o1] = (bf16_t)(wv[u] >> 16);
      }
    }
  }

  for (; pid < npatch; pid += gridDim.x) {
    const int nqp = (P.nq + 31) & ~31;
#pragma unroll
    for (int u = 0; u < kQLoads; ++u) {
      const int q = (tid >> 3) + 32 * u;
      if (c8 < cch && q < nqp) *reinterpret_cast<uint4*>(&s_dy[q * kNarrowKp + c8 * 8]) = dv[u];
    }
    __syncthreads();
    const int nxt = pid + (int)gridDim.x;
    const NarrowPatch Pn = narrow_patch(a, nxt < npatch ? nxt : pid, th, lgtw, ntw, nth, kh, kw, sh, sw);
    if (nxt < npatch) load_dy(Pn, dv);

    // Z blocks: wave w takes 32-row blocks w and w + 4 (all fragments read before the
    // first multiply; rows past the patch's pixels are zero)
    f32x16 acc[2];
    const int nblk = nqp >> 5;
    u32x4 bfr[4], af[2][4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      if (ks < nks) bfr[ks] = *reinterpret_cast<const u32x4*>(&s_w[l32 * kNarrowKp + ks * 16 + half * 8]);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = min(wave + 4 * u, kNqMax / 32 - 1) * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        if (ks < nks) af[u][ks] = *reinterpret_cast<const u32x4*>(&s_dy[row * kNarrowKp + ks * 16 + half * 8]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[u][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        if (ks < nks) acc[u] = mfma32x32x16(af[u][ks], bfr[ks], acc[u]);
    }
    __syncthreads();  // every dy read is done before Z overwrites it
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int blk = wave + 4 * u;
      if (blk < nblk) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = blk * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          s_z[row * kZp + l32] = acc[u][r];
        }
      }
    }
    __syncthreads();

    if constexpr (SS == 2 && TH > 0 && LGTW > 0) {
      // stride 2: wave w sums the input pixels of parity class (w / 2, w % 2), which all
      // take the same taps (rows r = (i + ph) mod 2, + 2; columns alike), so the loops
      // are uniform and every Z read of a pixel is issued before the first add (an
      // out-of-range tap reads a clamped entry and adds nothing)
      constexpr int TWC = (1 << LGTW) / 2, THC = TH / 2, RG = 64 / TWC;
      static_assert(64 % TWC == 0, "class columns divide the wave");
      const int ca = wave >> 1, cb = wave & 1;
      const int r0 = (ca + a.ph) & 1, s0 = (cb + a.pw) & 1;
      const int j = P.j0 + cb + 2 * (lane % TWC);
      const int qlast = P.nq > 0 ? P.nq - 1 : 0;
      for (int ri = lane / TWC; ri < THC; ri += RG) {
        const int i = P.i0 + ca + 2 * ri;
        if (i >= P.i1 || j >= P.j1) continue;
        float zv[(KS + 1) / 2][(KS + 1) / 2][CI];
        bool ok[(KS + 1) / 2][(KS + 1) / 2];
#pragma unroll
        for (int dr = 0; dr < (KS + 1) / 2; ++dr)
#pragma unroll
          for (int ds = 0; ds < (KS + 1) / 2; ++ds) {
            const int r = r0 + 2 * dr, s = s0 + 2 * ds;
            const int qi = (i + a.ph - r) >> 1, qj = (j + a.pw - s) >> 1;
            ok[dr][ds] = r < KS && s < KS && qi >= 0 && qi < a.ho && qj >= 0 && qj < a.wo;
            int q = (qi - P.qr0) * P.nqc + (qj - P.qc0);
            q = ok[dr][ds] ? q : 0;
            q = q < qlast ? q : qlast;
            const int n = ok[dr][ds] ? (r * KS + s) * CI : 0;
#pragma unroll
            for (int c = 0; c < CI; ++c) zv[dr][ds][c] = s_z[q * kZp + n + c];
          }
        float sum[CI];
#pragma unroll
        for (int c = 0; c < CI; ++c) {
          sum[c] = 0.f;
#pragma unroll
          for (int dr = 0; dr < (KS + 1) / 2; ++dr)
#pragma unroll
            for (int ds = 0; ds < (KS + 1) / 2; ++ds) sum[c] += ok[dr][ds] ? zv[dr][ds][c] : 0.f;
        }
        bf16_t* d = a.dx + (((int64_t)P.img * a.h + i) * a.w + j) * a.dx_pix;
#pragma unroll
        for (int c = 0; c < CI; ++c) {
          const float v = a.accumulate ? sum[c] + bf2f(d[c]) : sum[c];
          d[c] = (bf16_t)f2bf(v);
        }
      }
    } else {
      // each thread sums the CI channels of the input pixels of one patch column, in rows
      // tid / tw, + 256 / tw, ...: the taps that reach row i are r = (i + ph) mod sh, + sh,
      // ..., reading dy rows (i + ph) div sh, - 1, ... (columns alike)
      {
        const int jj = tid & (tw - 1);
        const int j = P.j0 + jj, uj = j + a.pw;
        const int qj0 = uj / sw, sj0 = uj - qj0 * sw;
        const int rstep = 256 >> lgtw;
        for (int i = P.i0 + (tid >> lgtw); i < P.i1 && j < P.j1; i += rstep) {
          float sum[CI];
#pragma unroll
          for (int c = 0; c < CI; ++c) sum[c] = 0.f;
          const int ui = i + a.ph;
          const int qi0 = ui / sh, ri0 = ui - qi0 * sh;
          for (int r = ri0, qi = qi0; r < kh && qi >= 0; r += sh, --qi) {
            if (qi >= a.ho) continue;
            const float* zr = s_z + (qi - P.qr0) * P.nqc * kZp + r * kw * CI;
            for (int s = sj0, qj = qj0; s < kw && qj >= 0; s += sw, --qj) {
              if (qj >= a.wo) continue;
              const float* z = zr + (qj - P.qc0) * kZp + s * CI;
#pragma unroll
              for (int c = 0; c < CI; ++c) sum[c] += z[c];
            }
          }
          bf16_t* d = a.dx + (((int64_t)P.img * a.h + i) * a.w + j) * a.dx_pix;
#pragma unroll
          for (int c = 0; c < CI; ++c) {
            const float v = a.accumulate ? sum[c] + bf2f(d[c]) : sum[c];
            d[c] = (bf16_t)f2bf(v);
          }
        }
      }
    }
    __syncthreads();  // Z reads are done before the next patch's dy is stored
    P = Pn;
  }
}

hipError_t dgrad_narrow_launch(const NarrowDgradArgs& a, int ci, float* wf, hipStream_t s) {
  // MFMA path: c_out a multiple of 16 up to 64, kh*kw*ci <= 32, 16-byte dy rows, 4-byte
  // aligned weights; the patch is the largest of these whose reached dy pixels fit the block
  if (a.co % 16 == 0 && a.co <= 64 && a.kh * a.kw * ci <= 32 && a.dy_pix % 8 == 0 &&
      (reinterpret_cast<uintptr_t>(a.dy) & 15) == 0 && (reinterpret_cast<uintptr_t>(a.wt) & 3) == 0 && a.n <= 65535) {
    static const int cand[][3] = {{8, 64, 6}, {4, 64, 6}, {8, 32, 5}, {4, 32, 5}, {8, 16, 4},
                                  {4, 16, 4},  {2, 16, 4}, {2, 8, 3},  {1, 8, 3}};
    int th = 0, tw = 0, lgtw = 0;
    for (const auto& c : cand) {
      const int qr = (c[0] - 1 + a.kh - 1) / a.sh + 1, qc = (c[1] - 1 + a.kw - 1) / a.sw + 1;
      if (qr * qc <= kNqMax) {
        th = c[0];
        tw = c[1];
        lgtw = c[2];
        break;
      }
    }
    const int ntw = tw > 0 ? (a.w + tw - 1) / tw : 0, nth = th > 0 ? (a.h + th - 1) / th : 0;
    const int64_t npatch = (int64_t)ntw * nth * a.n;
    if (npatch > 0 && npatch < 0x7fffffff) {
      dim3 grid((unsigned)(npatch < 1280 ? npatch : 1280));  // five blocks per CU
      trace_begin(KC_CONV_DGRAD);
      const int np = (int)npatch;
      if (ci == 3 && a.kh == 3 && a.kw == 3 && a.sh == 2 && a.sw == 2 && a.co == 48 && th == 8 && lgtw == 6) {
        NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<3, 3, 2, 8, 6, 48>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np);
      } else {
        switch (ci) {
          case 1: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<1, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 2: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<2, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 3: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<3, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 4: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<4, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 5: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<5, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 6: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<6, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          case 7: NUMBAT_LAUNCH((dgrad_narrow_mfma_kernel<7, 0, 0, 0, 0, 0>), grid, dim3(256), 0, s, a, th, lgtw, ntw, nth, np); break;
          default: trace_end(KC_CONV_DGRAD); return hipErrorInvalidValue;
        }
      }
      trace_end(KC_CONV_DGRAD);
      return hipGetLastError();
    }
  }
  const int ghm = (a.h + a.sh - 1) / a.sh, gwm = (a.w + a.sw - 1) / a.sw;
  const int64_t blocks = ((int64_t)a.n * ghm * ((gwm + 63) / 64) + 3) / 4;  // 4 waves of 64 pixels
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t wn = (int64_t)a.kh * a.kw * a.co * ci;
  trace_begin(KC_DGRAD_WEIGHTS);
  NUMBAT_LAUNCH(narrow_weights_kernel, dim3((unsigned)((wn + 255) / 256)), dim3(256), 0, s, a.wt, wf, a.co, a.kh,
                     a.kw, ci);
  trace_end(KC_DGRAD_WEIGHTS);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)blocks, (unsigned)(a.sh * a.sw), 1);
  trace_begin(KC_CONV_DGRAD);
  switch (ci) {
    case 1: NUMBAT_LAUNCH(dgrad_narrow_kernel<1>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 2: NUMBAT_LAUNCH(dgrad_narrow_kernel<2>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 3: NUMBAT_LAUNCH(dgrad_narrow_kernel<3>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 4: NUMBAT_LAUNCH(dgrad_narrow_kernel<4>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 5: NUMBAT_LAUNCH(dgrad_narrow_kernel<5>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 6: NUMBAT_LAUNCH(dgrad_narrow_kernel<6>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    case 7: NUMBAT_LAUNCH(dgrad_narrow_kernel<7>, grid, dim3(256), 0, s, a, a.dy, wf, a.dx); break;
    default: trace_end(KC_CONV_DGRAD); return hipErrorInvalidValue;
  }
  trace_end(KC_CONV_DGRAD);
  return hipGetLastError();
}

}  // namespace numbat

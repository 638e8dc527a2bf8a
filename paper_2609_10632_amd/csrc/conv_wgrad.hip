// Weight gradient dW[o][k] = sum_m dy[m][o] * X[m][k] on gfx950 MFMA, where m runs over
// the n*ho*wo output pixels and X[m][(tap, c)] is the input pixel that tap reads.
//
// In NHWC both operands are contiguous along o / k and strided along the reduction
// dimension m, while an MFMA lane needs 8 consecutive reduction elements.  Each thread
// therefore loads an 8-pixel x 8-channel unit (eight 16-byte buffer loads, 8 channels of
// 8 consecutive pixels), transposes it in registers with byte permutes and writes eight
// 16-byte rows of [channel][pixel] into LDS; the MFMAs (32x32x16) read both operands
// from there.  Loads run a register ring several steps ahead of the multiply.  Buffer
// loads answer padding taps, pixels past the split and channels past the tile with
// zeros (offsets past the buffer range), so every step issues the same loads.  The
// reduction over m is split into fixed contiguous ranges, one per blockIdx.z, whose fp32
// partial sums are added afterwards in split order, so the result does not depend on
// scheduling.
#include <cstdlib>
#include <type_traits>

#include "kernels.h"

namespace numbat {

namespace {

template <int V>
using Ic = std::integral_constant<int, V>;

constexpr int BR = 64;           // reduction pixels per step
constexpr int LROW = BR + 8;     // bf16 per LDS row (144 bytes: conflict-free fragment reads)
constexpr int BNK = 128;         // k columns per tile
constexpr uint32_t kOobW = 0x80000000u;
constexpr int kRecW = 0x7ffffff0;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t wrsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, kRecW, 0x00020000);
}

__device__ __forceinline__ uint32_t lo_pair(uint32_t p0, uint32_t p1) {
  return __builtin_amdgcn_perm(p1, p0, 0x05040100u);  // (p0.lo16, p1.lo16)
}
__device__ __forceinline__ uint32_t hi_pair(uint32_t p0, uint32_t p1) {
  return __builtin_amdgcn_perm(p1, p0, 0x07060302u);  // (p0.hi16, p1.hi16)
}

// in: P[j] = 8 channels of pixel j.  out: Q[ch] = 8 pixels of channel ch.
__device__ __forceinline__ void transpose8x8(const u32x4 (&P)[8], u32x4 (&Q)[8]) {
#pragma unroll
  for (int ch = 0; ch < 8; ++ch) {
    const int wi = ch >> 1;
    u32x4 q;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t x0 = P[2 * k][wi], x1 = P[2 * k + 1][wi];
      q[k] = (ch & 1) ? hi_pair(x0, x1) : lo_pair(x0, x1);
    }
    Q[ch] = q;
  }
}

// Tile BMO = 64*TMO output channels x BNK = 128 k columns; 2 x 2 waves of
// (32*TMO) x 64.  Threads [0, BMO) load dy units, [BMO, BMO + 128) x units.
template <int TMO, int D>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a, FastDiv div_wo, FastDiv div_howo) {
  constexpr int BMO = 64 * TMO;
  constexpr int TM = TMO, TN = 2;
  constexpr int UDY = BMO, UX = 128;
  static_assert(D >= 1 && D <= 4, "prefetch depth 1..4");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BMO][LROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNK][LROW];
  __shared__ __attribute__((aligned(16))) uint2 s_pix[2][BR];  // per pixel of a step: (byte offset, tap mask)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, half = lane >> 5;
  // logical tile (o tile fastest, then k tile, then split): the blocks of one split read
  // the same pixels and are kept on one XCD
  const uint32_t gx = gridDim.x, gy = gridDim.y;
  const uint32_t lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const uint32_t lg = a.remap ? xcd_remap(lin, gx * gy * gridDim.z) : lin;
  const int bx = (int)(lg % gx), by = (int)((lg / gx) % gy), bz = (int)(lg / (gx * gy));
  const int o0 = bx * BMO;
  const int k0 = by * BNK;
  const int64_t rbeg = (int64_t)bz * a.rows_per_split;
  int64_t rend = rbeg + a.rows_per_split;
  if (rend > a.m) rend = a.m;
  const int nsteps = rend > rbeg ? (int)((rend - rbeg + BR - 1) / BR) : 0;

  // this thread's unit: channel group grp (8 output channels, or 8 k columns of one tap)
  // and pixel block pb (8 consecutive pixels of the step).  8 lanes share a channel
  // group and cover the step's 8 pixel blocks: a load instruction reads 8 pixels x 128
  // contiguous bytes, and the transposed LDS rows they write are 128 contiguous bytes
  // (lanes of the next group land in the other half of the banks).
  // the role is the same for the whole wave (UDY is a multiple of 64); deriving it from the
  // wave index read into a scalar register lets the compiler keep the buffer descriptor
  // selected by it in scalar registers
  const bool isx = __builtin_amdgcn_readfirstlane(wave) * 64 >= UDY;
  const uint32_t xsel = 0u - (uint32_t)isx;  // all ones for the x role
  const bool has = tid < UDY + UX;
  const int v = isx ? tid - UDY : tid;
  const int grp = v >> 3;
  const int pb = v & 7;
  bool uok;
  uint32_t ucol;  // dy: byte offset of the 8 channels; x: tap offset + channel offset (bytes)
  int utap = 31;  // x: tap of the unit's k group (31: none; bit 31 of a tap mask is clear)
  const uint32_t dpix2 = (uint32_t)a.dy_pix * 2, xpix2 = (uint32_t)a.x_pix * 2;
  if (!isx) {
    const int o = o0 + grp * 8;
    uok = has && o < a.co;
    ucol = (uint32_t)o * 2;
  } else {
    const int k = k0 + grp * 8;
    uok = has && k < a.ktot;
    const int tap = k / a.ci, c = k - tap * a.ci;
    const int r = tap / a.kw, q = tap - r * a.kw;
    ucol = (uint32_t)(r * a.w + q) * xpix2 + (uint32_t)c * 2;
    utap = uok ? tap : 31;
  }
  const int howo = a.ho * a.wo;
  const int halo_px = a.ph * a.w + a.pw;  // the x gather base sits this many pixels before an image

  // x gather base of step st: the image of its first pixel, moved back by the halo
  auto step_img = [&](int st) __attribute__((always_inline)) -> uint32_t {
    const int64_t p0 = rbeg + (int64_t)st * BR;
    return p0 < a.m ? fdiv((uint32_t)p0, div_howo) : 0u;
  };
  // The 64 pixels of a step are decoded once, by threads 0..63, into table slot st & 1:
  // the byte offset of the pixel's top-left tap from the step's gather base and the mask
  // of its taps inside the image (0 past the split)
  auto decode = [&](int st) __attribute__((always_inline)) {
    if (tid >= BR) return;
    const int64_t px = rbeg + (int64_t)st * BR + tid;
    uint2 e = make_uint2(0u, 0u);
    if (px < rend) {
      const uint32_t img_s = step_img(st);
      const uint32_t img = fdiv((uint32_t)px, div_howo);
      const uint32_t rem = (uint32_t)px - img * (uint32_t)howo;
      const uint32_t p = fdiv(rem, div_wo), q = rem - p * (uint32_t)a.wo;
      const int ih0 = (int)p * a.sh - a.ph, iw0 = (int)q * a.sw - a.pw;
      e.x = (uint32_t)((((int)(img - img_s) * a.h + ih0) * a.w + iw0 + halo_px)) * xpix2;
      // kernel sides are at most 5 (25 taps): fixed-trip loops, so no loop sits inside
      // the main loop (a loop there would make the load counters wait for everything)
      uint32_t cols = 0;
#pragma unroll
      for (int j = 0; j < 5; ++j)
        cols |= (j < a.kw && (unsigned)(iw0 + j) < (unsigned)a.w ? 1u : 0u) << j;
      uint32_t mk = 0;
#pragma unroll
      for (int i = 0; i < 5; ++i)
        mk |= (i < a.kh && (unsigned)(ih0 + i) < (unsigned)a.h ? cols : 0u) << (i * a.kw);
      e.y = mk;
    }
    s_pix[st & 1][tid] = e;
  };

  // Every thread runs the same load code -- the dy and the x offset are both formed and
  // the role selects one -- so the loads are never under divergent control flow and the
  // compiler's load counters wait for exactly the ring slot being staged.
  auto load = [&](int st, u32x4 (&xr)[8]) __attribute__((always_inline)) {
    const int64_t p0 = rbeg + (int64_t)st * BR;  // first pixel of the step
    const __amdgpu_buffer_rsrc_t r =
        isx ? wrsrc(a.x + ((int64_t)step_img(st) * a.h * a.w - halo_px) * a.x_pix) : wrsrc(a.dy + p0 * a.dy_pix);
    const uint4* tab = reinterpret_cast<const uint4*>(&s_pix[st & 1][pb * 8]);
    // pixels of the step inside the split (a 32-bit scalar: a 64-bit per-lane compare
    // here was turned into a branch around one load)
    const int64_t left64 = rend - p0;
    const int left = left64 <= 0 ? 0 : (left64 >= BR ? BR : (int)left64);
#pragma unroll
    for (int j2 = 0; j2 < 4; ++j2) {
      const uint4 e = tab[j2];  // two pixels
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int j = 2 * j2 + h;
        const uint32_t base = h ? e.z : e.x, mask = h ? e.w : e.y;
        // branch-free selects (bit masks): the compiler otherwise turns one of them into
        // control flow around a load
        const uint32_t t = (uint32_t)__builtin_amdgcn_sbfe((int)mask, utap, 1);
        const uint32_t xo = (t & (base + ucol)) | (~t & kOobW);
        const uint32_t d = 0u - (uint32_t)(uok && pb * 8 + j < left);
        const uint32_t dofs = (d & ((uint32_t)(pb * 8 + j) * dpix2 + ucol)) | (~d & kOobW);
        xr[j] = __builtin_amdgcn_raw_buffer_load_b128(r, (xsel & xo) | (~xsel & dofs), 0u, 0);
      }
    }
  };
  auto store = [&](int buf, const u32x4 (&xr)[8]) __attribute__((always_inline)) {
    if (!has) return;
    u32x4 Q[8];
    transpose8x8(xr, Q);
    const int col = pb * 8;
    if (!isx) {
#pragma unroll
      for (int c = 0; c < 8; ++c) *reinterpret_cast<u32x4*>(&As[buf][grp * 8 + c][col]) = Q[c];
    } else {
#pragma unroll
      for (int c = 0; c < 8; ++c) *reinterpret_cast<u32x4*>(&Bs[buf][grp * 8 + c][col]) = Q[c];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < BR / 16; ++ks) {
      u32x4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const u32x4*>(&As[buf][wm * 32 * TM + i * 32 + l32][ks * 16 + half * 8]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *reinterpret_cast<const u32x4*>(&Bs[buf][wn * 64 + j * 32 + l32][ks * 16 + half * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
    }
  };

  // Step kt: stage step kt+1 in LDS, issue the loads of step kt+1+D (their pixels were
  // decoded during step kt-1), decode the pixels of step kt+2+D, multiply step kt.  The
  // barrier ending the step publishes both the staged tiles and the decoded pixels.
  u32x4 ring[D][8];
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    constexpr int nxt = (u + 1) % D;
    compute(kt & 1);
    store((kt + 1) & 1, ring[nxt]);
    load(kt + 1 + D, ring[nxt]);
    decode(kt + 2 + D);
    __syncthreads();
  };
  // prologue in the steady state's issue order (step 0 to LDS, steps 1..D in flight)
  if (nsteps > 0) {
    decode(0);
    __syncthreads();
    load(0, ring[0]);
    store(0, ring[0]);
    __syncthreads();  // step 0's table slot is reused by step 2
#pragma unroll
    for (int st = 1; st <= D; ++st) {
      decode(st);
      __syncthreads();
      load(st, ring[st % D]);
    }
    decode(D + 1);
    __syncthreads();
  }
  int kb = 0;
  for (; kb + D <= nsteps; kb += D) {
    step(Ic<0>{}, kb);
    if constexpr (D > 1) step(Ic<1 % D>{}, kb + 1);
    if constexpr (D > 2) step(Ic<2 % D>{}, kb + 2);
    if constexpr (D > 3) step(Ic<3 % D>{}, kb + 3);
  }
  if constexpr (D > 1) {
    if (kb < nsteps) step(Ic<0>{}, kb);
  }
  if constexpr (D > 2) {
    if (kb + 1 < nsteps) step(Ic<1 % D>{}, kb + 1);
  }
  if constexpr (D > 3) {
    if (kb + 2 < nsteps) step(Ic<2 % D>{}, kb + 2);
  }

  // epilogue: accumulator register r of a lane is output channel row 8*(r/4) +
  // 4*(lane/32) + (r%4) of its 32-row block, k column lane%32
  float* out = a.out + (a.splits > 1 ? (int64_t)bz * a.co * a.ktot : 0);
  const bool acc_in = a.splits == 1 && a.accumulate;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int k = k0 + wn * 64 + j * 32 + l32;
      if (k >= a.ktot) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = o0 + wm * 32 * TM + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (o >= a.co) continue;
        float* p = out + (int64_t)o * a.ktot + k;
        const float val = acc[i][j][r];
        *p = acc_in ? *p + val : val;
      }
    }
}

template <int TMO>
hipError_t launch_w(const WgradArgs& a, hipStream_t s) {
  constexpr int BMO = 64 * TMO;
  dim3 grid((a.co + BMO - 1) / BMO, (a.ktot + BNK - 1) / BNK, a.splits);
  const FastDiv dwo = make_fastdiv((uint32_t)a.wo), dhw = make_fastdiv((uint32_t)(a.ho * a.wo));
  trace_begin(KC_WGRAD, s);
  hipLaunchKernelGGL((wgrad_kernel<TMO, 3>), grid, dim3(256), 0, s, a, dwo, dhw);
  trace_end(KC_WGRAD, s);
  return hipGetLastError();
}

// dw = [dw +] sum over splits, four consecutive outputs per thread.  The splits are cut
// into G contiguous groups summed by G threads in split order; the G group sums are then
// added in group order.  The order depends only on (splits, G), so the result is bitwise
// reproducible.  A block holds 256/G outputs (float4) x G groups.
template <int G>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float4* part, int splits, int64_t count4, float* dw,
                                                            int accumulate) {
  constexpr int OPB = 256 / G;  // float4 outputs per block
  __shared__ float4 s_sum[G][OPB];
  const int g = threadIdx.x / OPB, lo = threadIdx.x % OPB;
  const int64_t i = blockIdx.x * (int64_t)OPB + lo;
  const int s0 = (int)((int64_t)splits * g / G), s1 = (int)((int64_t)splits * (g + 1) / G);
  float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < count4) {
    for (int k = s0; k < s1; ++k) {
      const float4 u = part[(int64_t)k * count4 + i];
      t.x += u.x;
      t.y += u.y;
      t.z += u.z;
      t.w += u.w;
    }
  }
  s_sum[g][lo] = t;
  __syncthreads();
  if (g != 0 || i >= count4) return;
  float4 r = s_sum[0][lo];
#pragma unroll
  for (int k = 1; k < G; ++k) {
    const float4 u = s_sum[k][lo];
    r.x += u.x;
    r.y += u.y;
    r.z += u.z;
    r.w += u.w;
  }
  float* o = dw + 4 * i;
  if (accumulate) {
    r.x = o[0] + r.x;
    r.y = o[1] + r.y;
    r.z = o[2] + r.z;
    r.w = o[3] + r.w;
  }
  o[0] = r.x;
  o[1] = r.y;
  o[2] = r.z;
  o[3] = r.w;
}

}  // namespace

// output-channel tile: 128 rows (twice the multiply per loaded x tile of 64 rows, which
// outweighs the padding of channel counts like 192), 64 when one such tile covers c_out
int wgrad_bmo(int co) { return co <= 64 ? 64 : 128; }

int wgrad_pick_splits(int64_t m, int co, int ktot, int64_t* rows_per_split) {
  const int bmo = wgrad_bmo(co);
  const int tiles = (int)(((co + bmo - 1) / bmo) * ((ktot + BNK - 1) / BNK));
  const int64_t steps = (m + BR - 1) / BR;
  // Two blocks fit per CU (LDS), 512 on the chip: as many splits as keep the grid within
  // one such round (a few blocks past it would cost a whole second round); at least 16
  // steps per split, at most 256 splits, partials at most 64 MiB
  int64_t splits = tiles < 512 ? 512 / tiles : 1;
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

hipError_t wgrad_launch(const WgradArgs& args, hipStream_t s) {
  WgradArgs a = args;
  a.remap = 0;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_REMAP_WG")) a.remap = atoi(e);
#endif
  return wgrad_bmo(a.co) == 64 ? launch_w<1>(a, s) : launch_w<2>(a, s);
}

hipError_t splitk_reduce_launch(const float* part, int splits, int64_t count, float* dw, int accumulate,
                                hipStream_t s) {
  // count = c_out * k_total is a multiple of 8 (c_out is).  Split groups: enough to give
  // ~1024 blocks (each thread then sums a handful of splits), at most one per split.
  const int64_t count4 = count / 4;
  int G = 1;
  while (G < 64 && G < splits && (count4 * G) / 256 < 1024) G *= 2;
  const float4* p4 = reinterpret_cast<const float4*>(part);
  const int opb = 256 / G;
  const unsigned blocks = (unsigned)((count4 + opb - 1) / opb);
  trace_begin(KC_SPLITK_REDUCE, s);
  switch (G) {
    case 1: hipLaunchKernelGGL(splitk_reduce_kernel<1>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 2: hipLaunchKernelGGL(splitk_reduce_kernel<2>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 4: hipLaunchKernelGGL(splitk_reduce_kernel<4>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 8: hipLaunchKernelGGL(splitk_reduce_kernel<8>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 16: hipLaunchKernelGGL(splitk_reduce_kernel<16>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 32: hipLaunchKernelGGL(splitk_reduce_kernel<32>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    default: hipLaunchKernelGGL(splitk_reduce_kernel<64>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
  }
  trace_end(KC_SPLITK_REDUCE, s);
  return hipGetLastError();
}

}  // namespace numbat

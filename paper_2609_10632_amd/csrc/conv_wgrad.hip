// Weight gradient dW[o][k] = sum_m dy[m][o] * X[m][k] on gfx950 MFMA, where m runs over
// the n*ho*wo output pixels and X[m][(tap, c)] is the input pixel that tap reads: the
// general kernel (every shape; the 3x3 stride-1 and 1x1 layers whose sizes suit it take
// the patch-staged kernel of conv_wgrad_halo.hip instead), the image layer's kernel and the
// split reduction.
//
// In NHWC both operands are contiguous along o / k and strided along the reduction
// dimension m, while an MFMA lane needs 8 consecutive reduction elements.  The loads
// write LDS directly in the tensors' own [pixel][channel] layout and the MFMA operands
// are read out of LDS with transposing reads, so no transpose runs in registers (the
// kernel below).  Buffer loads answer padding taps, pixels past the split and channels
// past the tile with zeros (offsets past the buffer range), so every step issues the
// same loads.  The reduction over m is split into fixed contiguous ranges, one per
// blockIdx.z, whose fp32 partial sums are added afterwards in split order, so the result
// does not depend on scheduling.
#include <cstdlib>
#include <type_traits>

#include "kernels.h"

namespace numbat {

namespace {

template <int V>
using Ic = std::integral_constant<int, V>;

constexpr int kSplitQuantum = 64;  // pixel splits are whole multiples of this
constexpr int BNK = 128;         // k columns per tile
constexpr uint32_t kOobW = 0x80000000u;
constexpr int kRecW = 0x7ffffff0;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t wrsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, kRecW, 0x00020000);
}

// The loads write LDS themselves (buffer_load ... lds: lane i of a wave instruction
// deposits its 16 bytes at the instruction's LDS base + 16*i) in the tensors' own
// layout, [pixel][64 channels] sub-tiles of 128-byte rows, and the MFMA operands -- 8 consecutive pixels of one channel per lane -- come out of LDS
// through transposing reads (ds_read_b64_tr_b16): within each 16-lane group, lane j
// reads 4 channels of one pixel and lane i receives 4 pixels of channel i; two reads make
// a fragment.  So a step costs no register transposes and no LDS store instructions.
// The 16-byte chunk c of pixel row r sits in slot c ^ (4 * ((r >> 1) & 1)), which makes
// the transposing reads of 32 lanes cover all 64 banks once; a load lane picks the chunk
// its fixed slot needs.  Each stage is its own LDS object (exact load waits, as in the
// convolution's direct-to-LDS kernel); a step begins with a wait for its own loads and a
// barrier, refills the stage read last step, decodes the pixels of a later step and
// multiplies.
typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef unsigned v2u_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void wlds_void_t;
typedef __attribute__((address_space(3))) v4s_t wlds_v4s_t;

// An LDS read of one pixel-table entry that completes before it returns.  Written as
// plain code, the compiler cannot tell the table from the stages the direct-to-LDS loads
// are filling and waits for every load in flight before it; this read waits for LDS
// only.
__device__ __forceinline__ v2u_t table_read(const uint2* p) {
  const uint32_t addr = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
  v2u_t r;
  asm volatile("ds_read_b64 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(addr) : "memory");
  return r;
}

// Output-channel tiles of BMO = 64, 128 or 192 rows take the four waves as 2 (o) x 2 (k),
// each wave BMO/2 rows x 64 columns; 96-row tiles take them as 1 x 4, each wave all 96
// rows x 32 columns.  dy is staged in DS = ceil(BMO / 64) sub-tiles of 64 channels (the
// upper half of a 96-row tile's second sub-tile loads zeros).
template <int BMO, int S, int BR>
struct WgDmaShape {
  static constexpr int DS = (BMO + 63) / 64;
  static constexpr int WM = BMO == 96 ? 1 : 2, WN = 4 / WM;  // waves along o, along k
  static constexpr int TM = BMO / 32 / WM, TN = BNK / 32 / WN;  // 32 x 32 blocks per wave
  static constexpr int D_ELEMS = DS * BR * 64;   // dy: DS sub-tiles of [BR px][64 ch]
  static constexpr int X_ELEMS = 2 * BR * 64;    // x: 2 sub-tiles of [BR px][64 k]
  static constexpr int RBW = BR / 32;            // 8-pixel row blocks per wave per sub-tile
  static constexpr int LOADS = (DS + 2) * RBW;   // load instructions per thread per step
  static constexpr int PENDING = (S - 2) * LOADS;
  static constexpr int LDS_BYTES = S * (D_ELEMS + X_ELEMS) * 2 + 2 * BR * 8;
  static_assert(BMO == 64 || BMO == 96 || BMO == 128 || BMO == 192, "output-channel tile");
};

template <int BMO, int S, int BR>
__global__ __launch_bounds__(256) void wgrad_dma_kernel(WgradArgs a, FastDiv div_wo, FastDiv div_howo) {
  using Sh = WgDmaShape<BMO, S, BR>;
  constexpr int DS = Sh::DS, TM = Sh::TM, TN = Sh::TN, RBW = Sh::RBW;
  static_assert(BR == 32 || BR == 64, "pixels per step");
  static_assert(S >= 2 && S <= 4, "2..4 LDS stages");
  static_assert(Sh::PENDING <= 63, "load counter range");

  __shared__ __attribute__((aligned(16))) bf16_t sD0[Sh::D_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sD1[Sh::D_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sD2[Sh::D_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sD3[Sh::D_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sX0[Sh::X_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sX1[Sh::X_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sX2[Sh::X_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t sX3[Sh::X_ELEMS];
  __shared__ __attribute__((aligned(16))) uint2 s_pix[2][BR];  // per pixel of a step: (x byte offset, tap mask)
  auto stage_d = [&](auto sc) __attribute__((always_inline)) -> bf16_t* {
    constexpr int s = decltype(sc)::value;
    if constexpr (s == 0) return sD0;
    else if constexpr (s == 1) return sD1;
    else if constexpr (s == 2) return sD2;
    else return sD3;
  };
  auto stage_x = [&](auto sc) __attribute__((always_inline)) -> bf16_t* {
    constexpr int s = decltype(sc)::value;
    if constexpr (s == 0) return sX0;
    else if constexpr (s == 1) return sX1;
    else if constexpr (s == 2) return sX2;
    else return sX3;
  };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = Sh::WM == 1 ? 0 : (wave & 1), wn = Sh::WM == 1 ? wave : (wave >> 1);
  const int half = lane >> 5;
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

  // Load instruction t of this wave fills rows 8*(wave + 4*(t & 1)) .. +8 of sub-tile t/2
  // (dy sub-tiles first, then x): lane loads chunk ck of pixel row 8*rowblock + lane/8.
  const int ck = (lane & 7) ^ (4 * ((lane >> 4) & 1));
  const int prow = lane >> 3;  // pixel row within the 8-row block
  const uint32_t dpix2 = (uint32_t)a.dy_pix * 2, xpix2 = (uint32_t)a.x_pix * 2;
  uint32_t dcol[DS];  // dy: byte offset of this lane's 8 channels in sub-tile h (kOobW past the tile or c_out)
#pragma unroll
  for (int h = 0; h < DS; ++h) {
    const int ol = 64 * h + 8 * ck, o = o0 + ol;
    dcol[h] = (o < a.co && ol < BMO) ? (uint32_t)o * 2 : kOobW;
  }
  uint32_t xcol[2];  // x: tap offset + channel offset (bytes) of this lane's 8 k columns
  int xtap[2];       // their tap (31: past k_total; bit 31 of a tap mask is clear)
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = k0 + 64 * h + 8 * ck;
    const int tap = k / a.ci, c = k - tap * a.ci;
    const int r = tap / a.kw, q = tap - r * a.kw;
    xcol[h] = (uint32_t)(r * a.w + q) * xpix2 + (uint32_t)c * 2;
    xtap[h] = k < a.ktot ? tap : 31;
  }
  const int howo = a.ho * a.wo;
  const int halo_px = a.ph * a.w + a.pw;

  auto step_img = [&](int st) __attribute__((always_inline)) -> uint32_t {
    const int64_t p0 = rbeg + (int64_t)st * BR;
    return p0 < a.m ? fdiv((uint32_t)p0, div_howo) : 0u;
  };
  // the 64 pixels of a step, decoded once by threads 0..63 into table slot st & 1
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

  // issue the loads of step st into stage s
  auto issue = [&](auto sc, int st) __attribute__((always_inline)) {
    bf16_t* D = stage_d(sc);
    bf16_t* X = stage_x(sc);
    const int64_t p0 = rbeg + (int64_t)st * BR;
    const __amdgpu_buffer_rsrc_t rx = wrsrc(a.x + ((int64_t)step_img(st) * a.h * a.w - halo_px) * a.x_pix);
    const __amdgpu_buffer_rsrc_t rd = wrsrc(a.dy + p0 * a.dy_pix);
    const int64_t left64 = rend - p0;
    const int left = left64 <= 0 ? 0 : (left64 >= BR ? BR : (int)left64);
    v2u_t e[RBW];
#pragma unroll
    for (int u = 0; u < RBW; ++u) e[u] = table_read(&s_pix[st & 1][(wave + 4 * u) * 8 + prow]);
#pragma unroll
    for (int h = 0; h < DS; ++h)
#pragma unroll
      for (int u = 0; u < RBW; ++u) {
        const int rb = wave + 4 * u;  // row block
        const int px = rb * 8 + prow;  // pixel of the step
        const uint32_t ok = 0u - (uint32_t)(px < left);
        const uint32_t vo = (ok & ((uint32_t)px * dpix2 + dcol[h])) | (~ok & kOobW);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (wlds_void_t*)(D + h * BR * 64 + rb * 8 * 64), 16, vo, 0, 0, 0);
      }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int u = 0; u < RBW; ++u) {
        const int rb = wave + 4 * u;
        const uint32_t tb = (uint32_t)__builtin_amdgcn_sbfe((int)e[u].y, xtap[h], 1);
        const uint32_t vo = (tb & (e[u].x + xcol[h])) | (~tb & kOobW);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (wlds_void_t*)(X + h * BR * 64 + rb * 8 * 64), 16, vo, 0, 0, 0);
      }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // transposing-read addresses: lane j of a 16-lane group reads 4 channels (8 bytes) of
  // pixel row 4*rd + (j / 4) of the slice's half; its 32-channel block jb sits in chunks
  // 4*jb + 2*((lane >> 4) & 1) + ((lane >> 1) & 1), swizzled by the row
  const uint32_t rbase = (uint32_t)((8 * half + ((lane & 15) >> 2)) * 128 + (lane & 1) * 8);
  const uint32_t slot0 = (uint32_t)((2 * ((lane >> 4) & 1) + ((lane >> 1) & 1)) ^ (4 * ((lane >> 3) & 1)));
  const uint32_t aoff[2] = {rbase + slot0 * 16, rbase + (slot0 ^ 4u) * 16};
  auto frag = [&](const unsigned char* T, int sub, int jb, int ks) __attribute__((always_inline)) -> u32x4 {
    const unsigned char* p = T + sub * BR * 128 + aoff[jb] + ks * 16 * 128;
    const v4s_t r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wlds_v4s_t*)p);
    const v4s_t r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wlds_v4s_t*)(p + 4 * 128));
    const v2u_t lo = __builtin_bit_cast(v2u_t, r0), hi = __builtin_bit_cast(v2u_t, r1);
    u32x4 f;
    f[0] = lo.x;
    f[1] = lo.y;
    f[2] = hi.x;
    f[3] = hi.y;
    return f;
  };
  auto compute = [&](auto sc) __attribute__((always_inline)) {
    const unsigned char* D = reinterpret_cast<const unsigned char*>(stage_d(sc));
    const unsigned char* X = reinterpret_cast<const unsigned char*>(stage_x(sc));
#pragma unroll
    for (int ks = 0; ks < BR / 16; ++ks) {
      u32x4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int ol = wm * 32 * TM + i * 32;  // first output channel of the fragment
        af[i] = frag(D, ol >> 6, (ol >> 5) & 1, ks);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int cb = wn * TN + j;  // 32-column block of the tile
        bf[j] = frag(X, cb >> 1, cb & 1, ks);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(af[i], bf[j], acc[i][j]);
    }
  };
  auto sync = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(Sh::PENDING) : "memory");
  };
  // step kt reads stage u = kt mod S, refills stage (kt - 1) mod S with step kt + S - 1
  // (pixels decoded last step) and decodes step kt + S
  auto step = [&](auto uc, int kt) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    sync();
    issue(Ic<(u + S - 1) % S>{}, kt + S - 1);
    decode(kt + S);
    compute(uc);
  };
  // prologue: steps 0..S-2 in flight (a plain barrier: the decoded table is LDS data, and
  // the loads already issued need not land yet)
  auto table_barrier = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  if (nsteps > 0) {
    decode(0);
    table_barrier();
    issue(Ic<0>{}, 0);
    decode(1);
    if constexpr (S > 2) {
      table_barrier();
      issue(Ic<1>{}, 1);
      decode(2);
    }
    if constexpr (S > 3) {
      table_barrier();
      issue(Ic<2>{}, 2);
      decode(3);
    }
  }
  int kb = 0;
  for (; kb + S <= nsteps; kb += S) {
    step(Ic<0>{}, kb);
    step(Ic<1>{}, kb + 1);
    if constexpr (S > 2) step(Ic<2 % S>{}, kb + 2);
    if constexpr (S > 3) step(Ic<3 % S>{}, kb + 3);
  }
  if (kb < nsteps) step(Ic<0>{}, kb);
  if constexpr (S > 2) {
    if (kb + 1 < nsteps) step(Ic<1>{}, kb + 1);
  }
  if constexpr (S > 3) {
    if (kb + 2 < nsteps) step(Ic<2>{}, kb + 2);
  }
  // loads issued past the last step must land before the block ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  float* out = a.out + (a.splits > 1 ? (int64_t)bz * a.co * a.ktot : 0);
  const bool acc_in = a.splits == 1 && a.accumulate;
  const int l32 = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int k = k0 + (wn * TN + j) * 32 + l32;
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
    // (unrolled: the loads of several partials in flight, the sums still in split order)
#pragma unroll 8
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

// Kernel configuration for a weight gradient: output-channel tile bmo (64, 96, 128 or
// 192), pixels per step br (32 or 64), LDS stages.  Chosen from the problem only, so the
// workspace size and the launch agree.
struct WgCfg {
  int bmo, stages, br;
};
// splits of the pixel range for `tiles` output tiles over `steps` 64-pixel quanta: as many
// as fill 448 block slots, at least 16 quanta per split, at most 256 splits.  The weight
// gradients run beside the backward's main chain on a second stream, and a grid that
// leaves that chain some CUs made the two-stream step faster though the kernels alone are
// slower: 512 slots (two blocks per CU) 8.925 ms per step, 448 8.82, 384 8.80, 256 8.81 ms
// (weight-gradient kernels alone 2.24, 2.37, 2.62, 3.15 ms); 768 slots were slower still.
static int64_t wgrad_splits_for(int64_t tiles, int64_t steps) {
  int64_t slots = 448;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_WG_SLOTS")) slots = atoi(e);
#endif
  int64_t splits = tiles < slots ? slots / tiles : 1;
  const int64_t max_by_steps = steps / 16 > 0 ? steps / 16 : 1;
  if (splits > max_by_steps) splits = max_by_steps;
  if (splits > 256) splits = 256;
  return splits < 1 ? 1 : splits;
}
static WgCfg wgrad_cfg(int64_t m, int co, int ktot) {
  // The output-channel tile among 64, 96 and 128 rows: where the split grid of a tile
  // leaves it under 350 blocks (small pixel counts cap the splits), the one with the most
  // blocks; otherwise the one that pads c_out least, then has the fewest tiles (fewer
  // re-reads of x).  Two stages of 64 pixels.  Measured over the detector's layer shapes
  // at batch 16 against 64 / 128-row tiles alone: 3% less weight-gradient time (96-row
  // tiles on the 96-, 192- and 288-channel 3x3 layers and the stride-2 576-channel one);
  // 32 pixels per step, three stages and 192-row tiles lost everywhere.
  const int64_t steps = (m + kSplitQuantum - 1) / kSplitQuantum;
  const int64_t kt = (ktot + BNK - 1) / BNK;
  int best = 64;
  int64_t bkey[3] = {INT64_MAX, INT64_MAX, INT64_MAX};
  for (const int b : {64, 96, 128}) {
    const int64_t ot = (co + b - 1) / b, tiles = ot * kt;
    const int64_t blocks = tiles * wgrad_splits_for(tiles, steps);
    const bool under = blocks < 350;
    const int64_t key[3] = {under ? 1 : 0, under ? -blocks : ot * b - co, tiles};
    if (key[0] < bkey[0] || (key[0] == bkey[0] && (key[1] < bkey[1] || (key[1] == bkey[1] && key[2] < bkey[2])))) {
      best = b;
      bkey[0] = key[0];
      bkey[1] = key[1];
      bkey[2] = key[2];
    }
  }
  WgCfg c{best, 2, 64};
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_WG_BMO")) c.bmo = atoi(e);
  if (const char* e = getenv("NUMBAT_WG_OLD")) {  // 64 / 128-row tiles alone
    const bool wide = co > 64 && (co + 127) / 128 * 128 == (co + 63) / 64 * 64;
    if (atoi(e)) c.bmo = wide ? 128 : 64;
  }
  if (const char* e = getenv("NUMBAT_WG_STAGES")) c.stages = atoi(e);
  if (const char* e = getenv("NUMBAT_WG_BR")) c.br = atoi(e);
#endif
  return c;
}
int wgrad_pick_splits(int64_t m, int co, int ktot, int64_t* rows_per_split) {
  const WgCfg c = wgrad_cfg(m, co, ktot);
  const int bmo = c.bmo;
  const int tiles = (int)(((co + bmo - 1) / bmo) * ((ktot + BNK - 1) / BNK));
  const int64_t steps = (m + kSplitQuantum - 1) / kSplitQuantum;
  int64_t splits = wgrad_splits_for(tiles, steps);
  // partials at most 64 MiB
  const int64_t part_bytes = (int64_t)co * ktot * 4;
  while (splits > 1 && splits * part_bytes > (64ll << 20)) --splits;
  if (splits < 1) splits = 1;
  const int64_t steps_per = (steps + splits - 1) / splits;
  *rows_per_split = steps_per * kSplitQuantum;
  splits = (int)((m + *rows_per_split - 1) / *rows_per_split);
  return (int)(splits < 1 ? 1 : splits);
}

namespace {
template <int BMO, int S, int BR>
hipError_t launch_w(const WgradArgs& a, hipStream_t s) {
  dim3 grid((a.co + BMO - 1) / BMO, (a.ktot + BNK - 1) / BNK, a.splits);
  const FastDiv dwo = make_fastdiv((uint32_t)a.wo), dhw = make_fastdiv((uint32_t)(a.ho * a.wo));
  NUMBAT_LAUNCH((wgrad_dma_kernel<BMO, S, BR>), grid, dim3(256), 0, s, a, dwo, dhw);
  return hipGetLastError();
}
template <int BMO>
hipError_t launch_w_bmo(const WgradArgs& a, const WgCfg& c, hipStream_t s) {
  if (c.br == 32) return c.stages == 3 ? launch_w<BMO, 3, 32>(a, s) : launch_w<BMO, 2, 32>(a, s);
  return c.stages == 3 ? launch_w<BMO, 3, 64>(a, s) : launch_w<BMO, 2, 64>(a, s);
}
}  // namespace

hipError_t wgrad_launch(const WgradArgs& args, hipStream_t s) {
  WgradArgs a = args;
  // XCD-aware tile order: the tiles of one pixel split share an XCD and its L2 (9% less
  // weight-gradient time over the detector's layers than the launch order)
  a.remap = 1;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_REMAP_WG")) a.remap = atoi(e);
#endif
  const WgCfg c = wgrad_cfg(a.m, a.co, a.ktot);
  trace_begin(KC_WGRAD);
  hipError_t e;
  if (c.bmo == 64) e = launch_w_bmo<64>(a, c, s);
  else if (c.bmo == 96) e = launch_w_bmo<96>(a, c, s);
  else if (c.bmo == 192) e = launch_w_bmo<192>(a, c, s);
  else e = launch_w_bmo<128>(a, c, s);
  trace_end(KC_WGRAD);
  return e;
}

hipError_t splitk_reduce_launch(const float* part, int splits, int64_t count, float* dw, int accumulate,
                                hipStream_t s) {
  // count = c_out * k_total is a multiple of 8 (c_out is).  Split groups: enough to give
  // ~256 blocks, at most one per split.  The reduction runs beside the main chain's
  // kernels; a grid of one block per CU left them more of the GPU than ~1024 blocks
  // (0.7% faster two-stream step; one group per output, the smallest grid, 2.5% slower).
  const int64_t count4 = count / 4;
  int G = 1;
  while (G < 64 && G < splits && (count4 * G) / 256 < 256) G *= 2;
  const float4* p4 = reinterpret_cast<const float4*>(part);
  const int opb = 256 / G;
  const unsigned blocks = (unsigned)((count4 + opb - 1) / opb);
  trace_begin(KC_SPLITK_REDUCE);
  switch (G) {
    case 1: NUMBAT_LAUNCH(splitk_reduce_kernel<1>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 2: NUMBAT_LAUNCH(splitk_reduce_kernel<2>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 4: NUMBAT_LAUNCH(splitk_reduce_kernel<4>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 8: NUMBAT_LAUNCH(splitk_reduce_kernel<8>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 16: NUMBAT_LAUNCH(splitk_reduce_kernel<16>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    case 32: NUMBAT_LAUNCH(splitk_reduce_kernel<32>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
    default: NUMBAT_LAUNCH(splitk_reduce_kernel<64>, dim3(blocks), dim3(256), 0, s, p4, splits, count4, dw, accumulate); break;
  }
  trace_end(KC_SPLITK_REDUCE);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient of the RGB image layer (3 channels, 3x3, stride 2, padding 1, at most
// 64 output channels, a multiple of 8; output rows a multiple of 4 and columns of 64):
//   dW[o][(r, s, c)] = sum over q of dy[q][o] * x[2 qi - 1 + r][2 qj - 1 + s][c].
// A block walks 4 x 64 patches of q (the next patch's loads in flight): dy rows and the
// 9 x 129 input pixels the patch reaches go to LDS once; the input pixels, padded to 4
// channels, are expanded into the patch's reduction rows X[q][16 r + 4 s + c] (zero at
// c = 3 and past s = 2), and dy^T X accumulates on 32x32x16 MFMAs whose operands come
// out of the [q][64] tiles through transposing reads (the q-major layout and swizzle of
// the general kernel).  Each wave takes a quarter of the patch's q; the waves' sums are
// added in a fixed order and each block writes one partial [o][27] for the split
// reduction.
namespace {
constexpr int kStemXCols = 129, kStemXPitch = 130;  // input pixels per patch row, LDS pitch

__global__ __launch_bounds__(256) void wgrad_stem_kernel(WgradArgs a, int npatch, float* part) {
  __shared__ __attribute__((aligned(16))) unsigned char s_tiles[2 * 256 * 128];  // dy, X; then wave sums
  __shared__ __attribute__((aligned(16))) unsigned char s_x[9 * kStemXPitch * 8];
  unsigned char* s_dy = s_tiles;
  unsigned char* s_col = s_tiles + 256 * 128;
  float* s_red = reinterpret_cast<float*>(s_tiles);  // [4][64][48]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5;
  const int ntc = a.wo >> 6, ntr = a.ho >> 2;
  const int cch = a.co >> 3;  // 16-byte dy chunks per pixel

  // global loads of patch pid: dy chunk (q = tid / 8 + 32 u, chunk tid % 8), input pixels
  // e = tid + 256 u of the 9 x 129 patch (three 2-byte channels each)
  constexpr int kDyRounds = 256 * 8 / 256, kXPix = 9 * kStemXCols, kXRounds = (kXPix + 255) / 256;
  uint4 dv[kDyRounds];
  uint32_t xlo[kXRounds], xhi[kXRounds];
  auto load = [&](int pid) __attribute__((always_inline)) {
    const int tj = pid % ntc, rr = pid / ntc;
    const int ti = rr % ntr, img = rr / ntr;
    const int oi0 = ti * 4, oj0 = tj * 64;
    const int c = tid & 7;
#pragma unroll
    for (int u = 0; u < kDyRounds; ++u) {
      const int q = (tid >> 3) + 32 * u;
      dv[u] = make_uint4(0u, 0u, 0u, 0u);
      if (c < cch)
        dv[u] = *reinterpret_cast<const uint4*>(a.dy + (((int64_t)img * a.ho + oi0 + (q >> 6)) * a.wo + oj0 + (q & 63)) *
                                                           a.dy_pix +
                                                c * 8);
    }
#pragma unroll
    for (int u = 0; u < kXRounds; ++u) {
      const int e = tid + 256 * u;
      const int pr = e / kStemXCols, pc = e - pr * kStemXCols;
      const int ih = 2 * oi0 - 1 + pr, iw = 2 * oj0 - 1 + pc;
      xlo[u] = xhi[u] = 0u;
      if (e < kXPix && (unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w) {
        const bf16_t* px = a.x + (((int64_t)img * a.h + ih) * a.w + iw) * a.x_pix;
        xlo[u] = (uint32_t)px[0] | ((uint32_t)px[1] << 16);
        xhi[u] = (uint32_t)px[2];
      }
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // transposing-read offsets (the general kernel's): lane j of a 16-lane group reads 4
  // channels of q row 4 rd + j / 4 of the slice's half; 32-channel block jb
  const uint32_t rbase = (uint32_t)((8 * half + ((lane & 15) >> 2)) * 128 + (lane & 1) * 8);
  const uint32_t slot0 = (uint32_t)((2 * ((lane >> 4) & 1) + ((lane >> 1) & 1)) ^ (4 * ((lane >> 3) & 1)));
  const uint32_t toff[2] = {rbase + slot0 * 16, rbase + (slot0 ^ 4u) * 16};
  auto frag = [&](const unsigned char* T, int jb, int ks) __attribute__((always_inline)) -> u32x4 {
    const unsigned char* p = T + toff[jb] + ks * 16 * 128;
    const v4s_t r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wlds_v4s_t*)p);
    const v4s_t r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wlds_v4s_t*)(p + 4 * 128));
    const v2u_t lo = __builtin_bit_cast(v2u_t, r0), hi = __builtin_bit_cast(v2u_t, r1);
    u32x4 f;
    f[0] = lo.x;
    f[1] = lo.y;
    f[2] = hi.x;
    f[3] = hi.y;
    return f;
  };

  int pid = blockIdx.x;
  if (pid < npatch) load(pid);
  for (; pid < npatch; pid += gridDim.x) {
    // stage: dy chunk c of row q in slot c ^ 4 ((q >> 1) & 1); input pixels padded to 4 channels
    {
      const int c = tid & 7;
#pragma unroll
      for (int u = 0; u < kDyRounds; ++u) {
        const int q = (tid >> 3) + 32 * u;
        if (c < cch) *reinterpret_cast<uint4*>(s_dy + q * 128 + ((c ^ (4 * ((q >> 1) & 1))) * 16)) = dv[u];
      }
#pragma unroll
      for (int u = 0; u < kXRounds; ++u) {
        const int e = tid + 256 * u;
        if (e < kXPix) {
          const int pr = e / kStemXCols, pc = e - pr * kStemXCols;
          *reinterpret_cast<uint2*>(s_x + (pr * kStemXPitch + pc) * 8) = make_uint2(xlo[u], xhi[u]);
        }
      }
    }
    __syncthreads();
    if (pid + (int)gridDim.x < npatch) load(pid + (int)gridDim.x);
    // reduction rows: X[q][chunk 2r] = input pixels (2 qi + r, 2 qj .. 2 qj + 1),
    // X[q][chunk 2r + 1] = pixel (2 qi + r, 2 qj + 2) and four zeros
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      const int e = tid + 256 * u;  // (q, r) pairs: 768
      const int q = e / 3, r = e - q * 3;
      const unsigned char* src = s_x + ((2 * (q >> 6) + r) * kStemXPitch + 2 * (q & 63)) * 8;
      const u32x4 v0 = *reinterpret_cast<const u32x4*>(src);
      const uint2 v1 = *reinterpret_cast<const uint2*>(src + 16);
      const int sw = 4 * ((q >> 1) & 1);
      *reinterpret_cast<u32x4*>(s_col + q * 128 + (((2 * r) ^ sw) * 16)) = v0;
      *reinterpret_cast<u32x4*>(s_col + q * 128 + (((2 * r + 1) ^ sw) * 16)) = u32x4{v1.x, v1.y, 0u, 0u};
    }
    __syncthreads();
    // wave w: q slices w, w + 4, w + 8, w + 12 (16 q each)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int ks = wave + 4 * k;
      const u32x4 a0 = frag(s_dy, 0, ks), a1 = frag(s_dy, 1, ks);
      const u32x4 b0 = frag(s_col, 0, ks), b1 = frag(s_col, 1, ks);
      acc[0][0] = mfma32x32x16(a0, b0, acc[0][0]);
      acc[0][1] = mfma32x32x16(a0, b1, acc[0][1]);
      acc[1][0] = mfma32x32x16(a1, b0, acc[1][0]);
      acc[1][1] = mfma32x32x16(a1, b1, acc[1][1]);
    }
    __syncthreads();  // tiles are free for the next patch
  }
  // wave sums [o][n' < 48] in LDS, then a fixed-order sum over the waves per output
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = i * 32 + 8 * (r >> 2) + 4 * half + (r & 3), n = j * 32 + (lane & 31);
        if (n < 48) s_red[(wave * 64 + o) * 48 + n] = acc[i][j][r];
      }
  __syncthreads();
  const int nout = a.co * 27;
  for (int e = tid; e < nout; e += 256) {
    const int o = e / 27, k = e - o * 27;
    const int r = k / 9, sc = k - r * 9, s = sc / 3, c = sc - s * 3;
    const int n = 16 * r + 4 * s + c;
    const float v = (s_red[(0 * 64 + o) * 48 + n] + s_red[(1 * 64 + o) * 48 + n]) +
                    (s_red[(2 * 64 + o) * 48 + n] + s_red[(3 * 64 + o) * 48 + n]);
    part[(int64_t)blockIdx.x * nout + e] = v;
  }
}
}  // namespace

bool wgrad_stem_shape(const WgradArgs& a) {
  return a.ci == 3 && a.kh == 3 && a.kw == 3 && a.sh == 2 && a.sw == 2 && a.ph == 1 && a.pw == 1 && a.co <= 64 &&
         a.co % 8 == 0 && a.ho % 4 == 0 && a.wo % 64 == 0 && a.dy_pix % 8 == 0 &&
         (reinterpret_cast<uintptr_t>(a.dy) & 15) == 0;
}

int wgrad_stem_blocks(const WgradArgs& a) {
  const int64_t npatch = (int64_t)a.n * (a.ho / 4) * (a.wo / 64);
  return (int)(npatch < 512 ? npatch : 512);  // two blocks per CU
}

hipError_t wgrad_stem_launch(const WgradArgs& a, float* part, hipStream_t s) {
  const int64_t npatch = (int64_t)a.n * (a.ho / 4) * (a.wo / 64);
  if (!wgrad_stem_shape(a) || npatch <= 0 || npatch >= 0x7fffffff) return hipErrorInvalidValue;
  const int nb = wgrad_stem_blocks(a);
  trace_begin(KC_WGRAD);
  NUMBAT_LAUNCH(wgrad_stem_kernel, dim3((unsigned)nb), dim3(256), 0, s, a, (int)npatch, part);
  trace_end(KC_WGRAD);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return splitk_reduce_launch(part, nb, (int64_t)a.co * 27, a.out, a.accumulate, s);
}

}  // namespace numbat
